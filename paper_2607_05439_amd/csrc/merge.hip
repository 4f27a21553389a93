// Online-softmax merge of partial states (the combine of the paper's ring
// steps: Appendix "Q/K/V layout and the ring loop"), then out = gate*acc/l.
// One thread per (row, h*d + e), or per four channels of one head when the
// head size allows; parts are folded in increasing order.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "dcp_internal.h"

namespace dcp {
namespace {

__global__ void __launch_bounds__(256) merge_kernel(MergeArgs a) {
  const int hd = a.n_heads * a.head_dim;
  const int64_t total = a.n_rows * hd;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = t / hd;
    const int x = (int)(t - r * hd);
    const int h = x / a.head_dim;
    float mx = -INFINITY;
    for (int p = 0; p < a.n_parts; ++p) mx = fmaxf(mx, a.m[((int64_t)p * a.n_heads + h) * a.n_rows + r]);
    float l = 0.0f, acc = 0.0f;
    if (mx != -INFINITY) {
      for (int p = 0; p < a.n_parts; ++p) {
        const float mp = a.m[((int64_t)p * a.n_heads + h) * a.n_rows + r];
        if (mp == -INFINITY) continue;
        // base-2 partials have integer maxima: the factor is an exact power of two
        const float sc = a.log2_units ? ldexpf(1.0f, (int)(mp - mx)) : expf(mp - mx);
        l = fmaf(sc, a.l[((int64_t)p * a.n_heads + h) * a.n_rows + r], l);
        acc = fmaf(sc, a.acc[((int64_t)p * a.n_rows + r) * hd + x], acc);
      }
    }
    if (a.acc_out) a.acc_out[t] = acc;
    if (x % a.head_dim == 0) {
      if (a.m_out)
        a.m_out[(int64_t)h * a.n_rows + r] =
            (a.log2_units && a.m_natural && mx != -INFINITY) ? mx * 0.69314718055994530942f : mx;
      if (a.l_out) a.l_out[(int64_t)h * a.n_rows + r] = l;
    }
    if (a.out) {
      const float gt = a.gate ? a.gate[t] : 1.0f;
      const float o = l > 0.0f ? gt * (acc / l) : 0.0f;
      if (a.out_bf16)
        static_cast<__bf16*>(a.out)[t] = (__bf16)o;
      else
        static_cast<float*>(a.out)[t] = o;
    }
  }
}

// The same merge, four consecutive channels of one head per thread (16-byte
// loads of the partial accumulators and the gate), 32-bit index arithmetic.
// Used when the head size is a multiple of 4 and the element count fits.
__global__ void __launch_bounds__(256) merge4_kernel(MergeArgs a) {
  const uint32_t d4 = (uint32_t)a.head_dim >> 2, hd4 = (uint32_t)a.n_heads * d4, hd = 4 * hd4;
  const uint32_t nr = (uint32_t)a.n_rows, total = nr * hd4;
  for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < total; t += gridDim.x * 256u) {
    const uint32_t r = t / hd4, x4 = t - r * hd4, h = x4 / d4;
    const float* m = a.m + (size_t)h * nr + r;
    const float* l_in = a.l + (size_t)h * nr + r;
    const size_t part = (size_t)nr * hd, pm = (size_t)a.n_heads * nr;
    float mx = -INFINITY;
    for (int p = 0; p < a.n_parts; ++p) mx = fmaxf(mx, m[p * pm]);
    float l = 0.0f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (mx != -INFINITY) {
      const float4* ap = reinterpret_cast<const float4*>(a.acc + (size_t)r * hd) + x4;
      // four parts' loads at a time (a part past the end repeats the last
      // one and is skipped), folded in increasing order
      for (int p0 = 0; p0 < a.n_parts; p0 += 4) {
        float mv[4], lv[4];
        float4 vv[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int p = min(p0 + j, a.n_parts - 1);
          mv[j] = m[p * pm];
          lv[j] = l_in[p * pm];
          vv[j] = ap[p * part / 4];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (p0 + j >= a.n_parts || mv[j] == -INFINITY) continue;
          const float sc = a.log2_units ? ldexpf(1.0f, (int)(mv[j] - mx)) : expf(mv[j] - mx);
          l = fmaf(sc, lv[j], l);
          acc.x = fmaf(sc, vv[j].x, acc.x);
          acc.y = fmaf(sc, vv[j].y, acc.y);
          acc.z = fmaf(sc, vv[j].z, acc.z);
          acc.w = fmaf(sc, vv[j].w, acc.w);
        }
      }
    }
    const size_t e0 = (size_t)t * 4;  // = r * hd + 4 * x4
    if (a.acc_out) *reinterpret_cast<float4*>(a.acc_out + e0) = acc;
    if (x4 == h * d4) {
      if (a.m_out)
        a.m_out[(size_t)h * nr + r] = (a.log2_units && a.m_natural && mx != -INFINITY) ? mx * 0.69314718055994530942f : mx;
      if (a.l_out) a.l_out[(size_t)h * nr + r] = l;
    }
    if (a.out) {
      const float4 gt = a.gate ? *reinterpret_cast<const float4*>(a.gate + e0) : make_float4(1.f, 1.f, 1.f, 1.f);
      const bool any = l > 0.0f;
      const float o[4] = {any ? gt.x * (acc.x / l) : 0.0f, any ? gt.y * (acc.y / l) : 0.0f,
                          any ? gt.z * (acc.z / l) : 0.0f, any ? gt.w * (acc.w / l) : 0.0f};
      if (a.out_bf16) {
        __bf16* dst = static_cast<__bf16*>(a.out) + e0;
        const __bf16 b[4] = {(__bf16)o[0], (__bf16)o[1], (__bf16)o[2], (__bf16)o[3]};
        *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(b);
      } else {
        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + e0) = make_float4(o[0], o[1], o[2], o[3]);
      }
    }
  }
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t st) {
  const int64_t total = a.n_rows * (int64_t)a.n_heads * a.head_dim;
  const uintptr_t align = reinterpret_cast<uintptr_t>(a.acc) | reinterpret_cast<uintptr_t>(a.acc_out) |
                          reinterpret_cast<uintptr_t>(a.gate) | reinterpret_cast<uintptr_t>(a.out);
  if (a.head_dim % 4 == 0 && total / 4 < (int64_t)INT32_MAX && (align & 15) == 0) {
    int64_t g = (total / 4 + 255) / 256;
    if (g > 16384) g = 16384;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(merge4_kernel, dim3((unsigned)g), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  int64_t g = (total + 255) / 256;
  if (g > 16384) g = 16384;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)g), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
