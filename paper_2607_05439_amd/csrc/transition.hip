// Pair transition on gfx950 (CDNA4): z <- z + W3 (SiLU(W1 LN z) * W2 LN z)
// per pair (Appendix "Manual SwiGLU decomposition"). The paper's memory
// device (free each 4x-expanded tensor as soon as it is used) becomes, on one
// GPU, a fused kernel in which no expanded tensor ever leaves the registers.
//
// bf16 path, c_z = 128, hidden = 512 (matrix cores):
//   trans_prep_kernel  folds gamma into W1 and W2 (beta into per-unit biases),
//                      rounds the weights to bf16 and writes them as
//                      matrix-core operand tiles, 12 KB per 16 hidden units
//                      (W1, W2 for v_mfma_f32_16x16x32_bf16, W3 for
//                      v_mfma_f32_16x16x16_bf16, its rows permuted so the
//                      output accumulator lines up with the z channels a lane
//                      holds).
//   trans_kernel       one workgroup (4 waves) per CU, persistent over groups
//                      of 256 pairs (64 per wave). Per group: z loaded once
//                      (B operands: lane (pair n, group g) holds channels
//                      32 ks + 8g .. +7), LayerNorm in registers; then for each
//                      16 hidden units: A = W1' N + b1 and B = W2' N + b2 as
//                      transposed products (hidden x pairs), h = SiLU(A) * B in
//                      registers, which is exactly the B operand layout of the
//                      second product out^T += W3' h^T; finally z + out, bf16,
//                      stored where z was read. Weight tiles stream through two
//                      48 KB LDS buffers by direct-to-LDS loads, one chunk of
//                      64 hidden units ahead.
// fp32 path (any c_z <= 256, hidden <= 1024): one wave per pair, plain fp32.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kCz = kTransCz;       // 128
constexpr int kHid = kTransHidden;  // 512
constexpr int kHt = kHid / 16;      // hidden tiles of 16 units
constexpr int kTileBytes = 12 * 1024;  // per hidden tile: W1 4 KB, W2 4 KB, W3 4 KB
constexpr int kChunkTiles = 4;          // hidden tiles per LDS chunk (two tile pairs)
constexpr int kChunks = kHt / kChunkTiles;
constexpr int kChunkBytes = kChunkTiles * kTileBytes;  // 48 KB
constexpr int kDmaPerWave = kChunkBytes / 4 / 1024;    // 1 KB DMA instructions per wave per chunk
constexpr float kLog2e = 1.44269504088896340736f;

// Output channel held at accumulator row r (0..15) of output tile ct: tiles
// 2ks and 2ks+1 cover channels 32ks .. 32ks+31 so that lane group g holds
// channels 32ks + 8g .. 32ks + 8g + 7, the ones it loaded as a B operand.
__host__ __device__ inline int out_channel(int ct, int r) { return 32 * (ct >> 1) + 8 * (r >> 2) + 4 * (ct & 1) + (r & 3); }

// ----------------------------------------------------------------------------- weight preparation
// Scaling: W1 (and its bias) carry a factor -log2(e), so the kernel's
// A' = -log2(e) A gives sigmoid(A) = 1 / (1 + 2^A') with no extra multiply, and
// SiLU(A) B = A B sigmoid(A) = -ln(2) A' B / (1 + 2^A'); the factor -ln(2)
// goes into W3. Layout per pair of hidden tiles (32 units, 24 KB):
//   W1 and W2 A operands of v_mfma_f32_16x16x32_bf16 for each of the two
//   tiles: [tile][mat][ks][lane] 16 B (row = unit, k-slots = channels
//   32 ks + 8 (lane/16) .. +7), 16 KB;
//   W3 A operands of v_mfma_f32_16x16x32_bf16 over the 32 units: [ct][lane]
//   16 B (row = channel out_channel(ct, lane%16), k-slot j of lane group g =
//   unit 4g + j of the first tile for j < 4, of the second for j >= 4, the
//   order in which the lane holds SiLU(A) B), 8 KB.
constexpr int kPairBytes = 2 * kTileBytes;
__global__ void __launch_bounds__(256) trans_prep_kernel(TransArgs a) {
  const float s1 = -kLog2e, s3 = -0.69314718055994530942f;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int per_pair = 2 * 2 * 4 * 64 + 8 * 64;  // 16-byte fragments per tile pair
  if (t < (kHt / 2) * per_pair) {
    const int hp = t / per_pair, f = t % per_pair;
    char* base = static_cast<char*>(a.w_prep) + (size_t)hp * kPairBytes;
    bf16x8 v;
    if (f < 1024) {
      const int tile = f / 512, mat = (f / 256) % 2, ks = (f / 64) % 4, lane = f % 64;
      const float* w = mat ? a.w2 : a.w1;
      const float sc = mat ? 1.0f : s1;
      const int unit = 16 * (2 * hp + tile) + (lane & 15), c0 = 32 * ks + 8 * (lane >> 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = (__bf16)(w[unit * kCz + c0 + i] * (a.gamma ? a.gamma[c0 + i] : 1.0f) * sc);
      *reinterpret_cast<u32x4*>(base + tile * 8192 + mat * 4096 + ks * 1024 + lane * 16) = __builtin_bit_cast(u32x4, v);
    } else {
      const int f3 = f - 1024, ct = f3 / 64, lane = f3 % 64, g = lane >> 4;
      const int ch = out_channel(ct, lane & 15);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int unit = 16 * (2 * hp + (j >> 2)) + 4 * g + (j & 3);
        v[j] = (__bf16)(a.w3[ch * kHid + unit] * s3);
      }
      *reinterpret_cast<u32x4*>(base + 16384 + ct * 1024 + lane * 16) = __builtin_bit_cast(u32x4, v);
    }
  }
  // biases b1 = -log2(e) W1 beta, b2 = W2 beta (fp32, per hidden unit)
  const int u = t - (kHt / 2) * per_pair;
  if (u >= 0 && u < 2 * kHid) {
    const int mat = u / kHid, unit = u % kHid;
    const float* w = mat ? a.w2 : a.w1;
    float s = 0.0f;
    if (a.beta)
      for (int c = 0; c < kCz; ++c) s = fmaf(w[unit * kCz + c], a.beta[c], s);
    a.b_prep[u] = mat ? s : s * s1;
  }
}

// ----------------------------------------------------------------------------- fused transition
__global__ void __launch_bounds__(256, 1) trans_kernel(TransArgs a) {
  __shared__ __attribute__((aligned(16))) char s_w[2][kChunkBytes];  // 96 KB
  __shared__ __attribute__((aligned(16))) float s_b[2 * kHid];        // b1, b2
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t n_groups = (a.n_pairs + 255) / 256;
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(a.w_prep, 0, kHt * kTileBytes, kRawBufferFlags);
  // chunk c of the weights (48 KB) into LDS buffer b: this wave's 12 KB quarter
  auto chunk_dma = [&](int c, int b) {
    const uint32_t base = lds_addr(&s_w[b][0]) + (uint32_t)(wave * kDmaPerWave * 1024);
#pragma unroll
    for (int i = 0; i < kDmaPerWave; ++i)
      dma_b128(wres, c * kChunkBytes + (wave * kDmaPerWave + i) * 1024 + lane * 16, base + (uint32_t)(i * 1024));
  };

  int64_t grp = blockIdx.x;
  if (grp >= n_groups) return;  // whole workgroup, before any barrier
  // biases in LDS, so the chunk loop issues no global loads of its own (their
  // waits would also wait for the weight loads in flight)
  for (int i = tid; i < 2 * kHid; i += 256) s_b[i] = a.b_prep[i];
  __syncthreads();
  chunk_dma(0, 0);
  int seq = 0;  // chunk sequence number across groups (buffer = seq & 1)
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  for (; grp < n_groups; grp += gridDim.x) {
    const bool last_group = grp + gridDim.x >= n_groups;
    // z of this wave's 4 pair tiles: lane (n, g) holds pair 16p + n, channels 32 ks + 8g .. +7
    const int64_t pair0 = grp * 256 + wave * 64;
    // z is read twice: here for the LayerNorm and again for the residual at
    // the end of the group (a few microseconds later, from L2), so that its
    // registers are free while the products run
    auto load_z = [&](u32x4 (&zz)[4][4]) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int64_t pr = min(pair0 + 16 * p + n, a.n_pairs - 1);
        const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.z_in) + pr * kCz + 8 * g);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) zz[p][ks] = src[4 * ks];
      }
    };
    u32x4 zr[4][4];
    load_z(zr);
    // LayerNorm (two passes over the pair's 128 channels: 32 per lane, 4 lanes)
    bf16x8 nv[4][4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      float x[4][8], s = 0.0f;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t w = zr[p][ks][i >> 1];
          x[ks][i] = __uint_as_float((i & 1) ? (w & 0xFFFF0000u) : (w << 16));
          s += x[ks][i];
        }
      const float mu = sum4(s) * (1.0f / kCz);
      float v = 0.0f;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          x[ks][i] -= mu;
          v = fmaf(x[ks][i], x[ks][i], v);
        }
      const float rstd = __builtin_amdgcn_rsqf(sum4(v) * (1.0f / kCz) + a.eps);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) nv[p][ks][i] = (__bf16)(x[ks][i] * rstd);
    }
    f32x4 acc[8][4];  // out^T: output tile ct, pair tile p
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int p = 0; p < 4; ++p) acc[ct][p] = zero;

    auto run_chunk = [&](int c, bool last_chunk, u32x4 (&zres)[4][4]) {
      const int b = seq & 1;
      barrier_lds();  // every wave is done with buffer b ^ 1 (the previous chunk)
      const bool more = c + 1 < kChunks || !last_group;
      if (more) chunk_dma((c + 1) % kChunks, b ^ 1);
      if (more)
        wait_vm<kDmaPerWave>();  // this wave's loads of chunk c have landed
      else
        wait_vm<0>();
      barrier_lds();  // and every other wave's
      const char* chunk = s_w[b];
      // first products of tile pair q: A' = W1' N + b1', B = W2' N + b2
      // (rows: hidden units 16 ht + 4g + i; columns: pairs), tiles ht = 2q', 2q'+1
      auto first = [&](int q, f32x4 (&ha)[2][4], f32x4 (&hb)[2][4]) {
        const char* pr = chunk + q * kPairBytes;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const int ht = (c * kChunkTiles / 2 + q) * 2 + tt;
          const float4 b1 = *reinterpret_cast<const float4*>(s_b + 16 * ht + 4 * g);
          const float4 b2 = *reinterpret_cast<const float4*>(s_b + kHid + 16 * ht + 4 * g);
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            ha[tt][p] = f32x4{b1.x, b1.y, b1.z, b1.w};
            hb[tt][p] = f32x4{b2.x, b2.y, b2.z, b2.w};
          }
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            const bf16x8 w1 = as_bf16x8(*reinterpret_cast<const u32x4*>(pr + tt * 8192 + ks * 1024 + lane * 16));
            const bf16x8 w2 = as_bf16x8(*reinterpret_cast<const u32x4*>(pr + tt * 8192 + 4096 + ks * 1024 + lane * 16));
#pragma unroll
            for (int p = 0; p < 4; ++p) {
              ha[tt][p] = mfma32(w1, nv[p][ks], ha[tt][p]);
              hb[tt][p] = mfma32(w2, nv[p][ks], hb[tt][p]);
            }
          }
        }
      };
      // h' = A' B / (1 + 2^A') as the B operand over the 32 units of the pair
      // (k-slot j: unit 4g + j of tile 0 for j < 4, of tile 1 for j >= 4), then
      // out^T += W3'' h'^T
      auto second = [&](int q, const f32x4 (&ha)[2][4], const f32x4 (&hb)[2][4]) {
        bf16x8 hv[4];
#pragma unroll
        for (int p = 0; p < 4; ++p)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float x = ha[j >> 2][p][j & 3];
            hv[p][j] = (__bf16)(x * hb[j >> 2][p][j & 3] * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x)));
          }
        const char* pr = chunk + q * kPairBytes + 16384;
#pragma unroll
        for (int ct = 0; ct < 8; ++ct) {
          const bf16x8 w3 = as_bf16x8(*reinterpret_cast<const u32x4*>(pr + ct * 1024 + lane * 16));
#pragma unroll
          for (int p = 0; p < 4; ++p) acc[ct][p] = mfma32(w3, hv[p], acc[ct][p]);
        }
      };
      f32x4 ha0[2][4], hb0[2][4], ha1[2][4], hb1[2][4];
      first(0, ha0, hb0);
      first(1, ha1, hb1);
      if (last_chunk) load_z(zres);  // the residual's z, issued once the normalised z is dead
      second(0, ha0, hb0);
      second(1, ha1, hb1);
      ++seq;
    };
    u32x4 zres[4][4];
    for (int c = 0; c < kChunks - 1; ++c) run_chunk(c, false, zres);
    run_chunk(kChunks - 1, true, zres);
    // residual and store: accumulator (ct = 2 ks + s, register i) is channel
    // 32 ks + 8g + 4s + i, element 4s + i of the lane's loaded chunk ks
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int64_t pr = pair0 + 16 * p + n;
      if (pr >= a.n_pairs) continue;
      u32x4* dst = reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.z_out) + pr * kCz + 8 * g);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t w = zres[p][ks][e >> 1];
          const float zin = __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
          o[e] = (__bf16)(zin + acc[2 * ks + (e >> 2)][p][e & 3]);
        }
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, o), dst + 4 * ks);
      }
    }
  }
  wait_vm<0>();
}

// ----------------------------------------------------------------------------- fp32 path
// One wave per pair: LayerNorm, then 8+ hidden units per lane, h in LDS, then
// the output channels per lane; fp32 throughout.
__global__ void __launch_bounds__(256) trans_gen_kernel(TransGenArgs a) {
  __shared__ float s_n[4][kGenMaxCz];
  __shared__ float s_h[4][kTransGenMaxHidden];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t p = (int64_t)blockIdx.x * 4 + wave;
  if (p >= a.n_pairs) return;
  const float* z = a.z_in + p * a.c_z;
  float s = 0.0f;
  for (int c = lane; c < a.c_z; c += 64) s += z[c];
  for (int m = 32; m > 0; m >>= 1) s += __shfl_xor(s, m);
  const float mu = s / (float)a.c_z;
  float v = 0.0f;
  for (int c = lane; c < a.c_z; c += 64) v = fmaf(z[c] - mu, z[c] - mu, v);
  for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m);
  const float rstd = 1.0f / sqrtf(v / (float)a.c_z + a.eps);
  float* nn = s_n[wave];
  for (int c = lane; c < a.c_z; c += 64)
    nn[c] = (a.gamma ? a.gamma[c] : 1.0f) * ((z[c] - mu) * rstd) + (a.beta ? a.beta[c] : 0.0f);
  __builtin_amdgcn_wave_barrier();
  float* hh = s_h[wave];
  for (int u = lane; u < a.hidden; u += 64) {
    float x = 0.0f, y = 0.0f;
    for (int c = 0; c < a.c_z; ++c) {
      x = fmaf(a.w1[(int64_t)u * a.c_z + c], nn[c], x);
      y = fmaf(a.w2[(int64_t)u * a.c_z + c], nn[c], y);
    }
    hh[u] = x / (1.0f + expf(-x)) * y;
  }
  __builtin_amdgcn_wave_barrier();
  for (int c = lane; c < a.c_z; c += 64) {
    float t = 0.0f;
    for (int u = 0; u < a.hidden; ++u) t = fmaf(a.w3[(int64_t)c * a.hidden + u], hh[u], t);
    a.z_out[p * a.c_z + c] = z[c] + t;
  }
}

}  // namespace

size_t trans_prep_bytes() { return (size_t)kHt * kTileBytes + 2 * kHid * sizeof(float); }

hipError_t launch_transition(const TransArgs& a, hipStream_t st) {
  const int prep_threads = (kHt / 2) * (2 * 2 * 4 * 64 + 8 * 64) + 2 * kHid;
  hipLaunchKernelGGL(trans_prep_kernel, dim3((prep_threads + 255) / 256), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_groups = (a.n_pairs + 255) / 256;
  const int64_t grid = n_groups < 256 ? n_groups : 256;
  hipLaunchKernelGGL(trans_kernel, dim3((unsigned)grid), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_transition_gen(const TransGenArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(trans_gen_kernel, dim3((unsigned)((a.n_pairs + 3) / 4)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
