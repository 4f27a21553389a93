// General fp32 path: any c_z <= 256, H <= 16, d <= 64, H*d <= 128, with s and
// z in fp32 or bf16. Plain vector-ALU kernels with fp32 arithmetic throughout
// (two-pass LayerNorm, expf), for the small and odd shapes the fused bf16
// kernels do not cover. Partial states use natural-log units.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "dcp_internal.h"

namespace dcp {
namespace {

__device__ __forceinline__ float load_act(const void* p, int bf16, int64_t idx) {
  if (bf16) return __uint_as_float((uint32_t)static_cast<const uint16_t*>(p)[idx] << 16);
  return static_cast<const float*>(p)[idx];
}

// One thread per (token, output) of the four projections; grid-stride.
__global__ void __launch_bounds__(256) gen_proj_kernel(GenProjArgs a) {
  const int64_t per_kv = a.n_tok * a.hd, per_q = a.n_q * a.hd;
  const int64_t total = 2 * per_kv + 2 * per_q;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    int which;
    int64_t r;
    if (t < per_kv) {
      which = 1;
      r = t;
    } else if (t < 2 * per_kv) {
      which = 2;
      r = t - per_kv;
    } else if (t < 2 * per_kv + per_q) {
      which = 0;
      r = t - 2 * per_kv;
    } else {
      which = 3;
      r = t - 2 * per_kv - per_q;
    }
    const int64_t row = r / a.hd;
    const int o = (int)(r - row * a.hd);
    const int64_t tok = (which == 0 || which == 3) ? a.q_row0 + row : row;
    const float* w = which == 0 ? a.w_q : which == 1 ? a.w_k : which == 2 ? a.w_v : a.w_g;
    float acc = 0.0f;
    for (int c = 0; c < a.c_s; ++c) acc = fmaf(w[(int64_t)o * a.c_s + c], load_act(a.s, a.s_bf16, tok * a.c_s + c), acc);
    float* dst = which == 0 ? a.q : which == 1 ? a.k : which == 2 ? a.v : a.g;
    dst[r] = which == 3 ? 1.0f / (1.0f + expf(-acc)) : acc;
  }
}

// LayerNorm statistics of one pair in fp32, two passes.
__device__ __forceinline__ void ln_stats(const void* z, int bf16, int64_t off, int c_z, float eps, float& mu,
                                         float& rstd) {
  float s = 0.0f;
  for (int c = 0; c < c_z; ++c) s += load_act(z, bf16, off + c);
  mu = s / (float)c_z;
  float v = 0.0f;
  for (int c = 0; c < c_z; ++c) {
    const float t = load_act(z, bf16, off + c) - mu;
    v = fmaf(t, t, v);
  }
  rstd = 1.0f / sqrtf(v / (float)c_z + eps);
}

// grid (n_q rows, n_kb parts), one wave. Each lane owns keys start+lane,
// start+lane+64, ... with its own online-softmax state in LDS; the 64 states
// are then merged in lane order.
__global__ void __launch_bounds__(64) gen_attn_kernel(GenAttnArgs a) {
  __shared__ float wg[kGenMaxH * kGenMaxCz];  // W_b * gamma
  __shared__ float st_m[64][kGenMaxH];
  __shared__ float st_l[64][kGenMaxH];
  __shared__ float st_acc[64][kGenMaxHD];
  const int lane = threadIdx.x;
  const int64_t row = blockIdx.x;
  const int part = blockIdx.y;
  const int H = a.n_heads, d = a.head_dim, hd = H * d, c_z = a.c_z;
  for (int x = lane; x < H * c_z; x += 64) wg[x] = a.w_b[x] * (a.gamma ? a.gamma[x % c_z] : 1.0f);
  for (int h = 0; h < H; ++h) {
    st_m[lane][h] = -INFINITY;
    st_l[lane][h] = 0.0f;
  }
  for (int x = 0; x < hd; ++x) st_acc[lane][x] = 0.0f;
  __syncthreads();

  int64_t size, start;
  chunk_of(a.k_len, a.n_kb, part, &size, &start);
  start += a.k_lo;
  const float scale = 1.0f / sqrtf((float)d);
  const float* qr = a.q + row * hd;
  for (int64_t j = start + lane; j < start + size; j += 64) {
    if (a.mask && a.mask[j] == 0) continue;
    const int64_t off = (row * a.n_tok + j) * c_z;
    float mu, rstd;
    ln_stats(a.z, a.z_bf16, off, c_z, a.eps, mu, rstd);
    for (int h = 0; h < H; ++h) {
      float b = 0.0f;
      for (int c = 0; c < c_z; ++c) b = fmaf(wg[h * c_z + c], (load_act(a.z, a.z_bf16, off + c) - mu) * rstd, b);
      float dot = 0.0f;
      for (int e = 0; e < d; ++e) dot = fmaf(qr[h * d + e], a.k[j * hd + h * d + e], dot);
      const float lg = dot * scale + b;
      const float mo = st_m[lane][h];
      const float mn = fmaxf(mo, lg);
      const float al = expf(mo - mn);  // 0 when mo = -inf
      const float p = expf(lg - mn);
      st_l[lane][h] = st_l[lane][h] * al + p;
      for (int e = 0; e < d; ++e)
        st_acc[lane][h * d + e] = fmaf(p, a.v[j * hd + h * d + e], st_acc[lane][h * d + e] * al);
      st_m[lane][h] = mn;
    }
  }
  __syncthreads();
  for (int x = lane; x < hd; x += 64) {
    const int h = x / d;
    float mx = -INFINITY;
    for (int t = 0; t < 64; ++t) mx = fmaxf(mx, st_m[t][h]);
    float l = 0.0f, acc = 0.0f;
    if (mx != -INFINITY)
      for (int t = 0; t < 64; ++t) {
        if (st_m[t][h] == -INFINITY) continue;
        const float sc = expf(st_m[t][h] - mx);
        l = fmaf(sc, st_l[t][h], l);
        acc = fmaf(sc, st_acc[t][x], acc);
      }
    a.acc_parts[((int64_t)part * a.n_q + row) * hd + x] = acc;
    if (x % d == 0) {
      a.m_parts[((int64_t)part * H + h) * a.n_q + row] = mx;
      a.l_parts[((int64_t)part * H + h) * a.n_q + row] = l;
    }
  }
}

// One thread per pair: the full bias with the LayerNorm affine and b_b.
__global__ void __launch_bounds__(256) gen_bias_kernel(GenBiasArgs a) {
  const int64_t total = a.n_rows * a.n_cols;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / a.n_cols, c = t - r * a.n_cols;
    const int64_t off = r * a.row_stride + c * a.c_z;
    float mu, rstd;
    ln_stats(a.z, a.z_bf16, off, a.c_z, a.eps, mu, rstd);
    for (int h = 0; h < a.n_heads; ++h) {
      float b = a.b_b ? a.b_b[h] : 0.0f;
      for (int k = 0; k < a.c_z; ++k) {
        const float ln = (load_act(a.z, a.z_bf16, off + k) - mu) * rstd * (a.gamma ? a.gamma[k] : 1.0f) +
                         (a.beta ? a.beta[k] : 0.0f);
        b = fmaf(a.w_b[(int64_t)h * a.c_z + k], ln, b);
      }
      a.out[t * a.n_heads + h] = b;
    }
  }
}

int grid_for(int64_t items) {
  int64_t g = (items + 255) / 256;
  if (g > 8192) g = 8192;
  return (int)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_gen_proj(const GenProjArgs& a, hipStream_t st) {
  const int64_t total = 2 * a.n_tok * a.hd + 2 * a.n_q * a.hd;
  hipLaunchKernelGGL(gen_proj_kernel, dim3(grid_for(total)), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gen_attn(const GenAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(gen_attn_kernel, dim3((unsigned)a.n_q, (unsigned)a.n_kb), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gen_bias(const GenBiasArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(gen_bias_kernel, dim3(grid_for(a.n_rows * a.n_cols)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
