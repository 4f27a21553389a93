// Online-softmax merge of partial states (the combine of the paper's ring
// steps: Appendix "Q/K/V layout and the ring loop"), then out = gate*acc/l.
// One thread per (row, h*d + e), or per four (two, on small layers) channels
// of one head when the head size allows; parts are folded in increasing order.
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

// V consecutive floats, 16 or 8 bytes, as one access
template <int V>
__device__ __forceinline__ void load_vec(const float* p, float (&x)[V]) {
  if constexpr (V == 4) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    x[0] = v.x, x[1] = v.y, x[2] = v.z, x[3] = v.w;
  } else {
    const float2 v = *reinterpret_cast<const float2*>(p);
    x[0] = v.x, x[1] = v.y;
  }
}
template <int V>
__device__ __forceinline__ void store_vec(float* p, const float (&x)[V]) {
  if constexpr (V == 4)
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  else
    *reinterpret_cast<float2*>(p) = make_float2(x[0], x[1]);
}

// The same merge, V (4 or 2) consecutive channels of one head per thread
// (16- or 8-byte loads of the partial accumulators and the gate), 32-bit index
// arithmetic. Used when the head size is a multiple of V and the element count
// fits; V = 2 doubles the threads (and so the loads in flight) on small layers.
template <int V>
__device__ __forceinline__ void merge_vec(const MergeArgs& a) {
  const uint32_t dv = (uint32_t)a.head_dim / V, hdv = (uint32_t)a.n_heads * dv, hd = V * hdv;
  const uint32_t nr = (uint32_t)a.n_rows, total = nr * hdv;
  for (uint32_t t = blockIdx.x * 256u + threadIdx.x; t < total; t += gridDim.x * 256u) {
    const uint32_t r = t / hdv, xv = t - r * hdv, h = xv / dv;
    const float* m = a.m + (size_t)h * nr + r;
    const float* l_in = a.l + (size_t)h * nr + r;
    const size_t part = (size_t)nr * hd, pm = (size_t)a.n_heads * nr;
    float mx = -INFINITY;
    for (int p = 0; p < a.n_parts; ++p) mx = fmaxf(mx, m[p * pm]);
    float l = 0.0f;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.0f;
    if (mx != -INFINITY) {
      const float* ap = a.acc + (size_t)r * hd + (size_t)V * xv;
      // four parts' loads at a time (a part past the end repeats the last
      // one and is skipped), folded in increasing order
      for (int p0 = 0; p0 < a.n_parts; p0 += 4) {
        float mv[4], lv[4], vv[4][V];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int p = min(p0 + j, a.n_parts - 1);
          mv[j] = m[p * pm];
          lv[j] = l_in[p * pm];
          load_vec<V>(ap + p * part, vv[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (p0 + j >= a.n_parts || mv[j] == -INFINITY) continue;
          const float sc = a.log2_units ? ldexpf(1.0f, (int)(mv[j] - mx)) : expf(mv[j] - mx);
          l = fmaf(sc, lv[j], l);
#pragma unroll
          for (int i = 0; i < V; ++i) acc[i] = fmaf(sc, vv[j][i], acc[i]);
        }
      }
    }
    const size_t e0 = (size_t)t * V;  // = r * hd + V * xv
    if (a.acc_out) store_vec<V>(a.acc_out + e0, acc);
    if (xv == h * dv) {
      if (a.m_out)
        a.m_out[(size_t)h * nr + r] = (a.log2_units && a.m_natural && mx != -INFINITY) ? mx * 0.69314718055994530942f : mx;
      if (a.l_out) a.l_out[(size_t)h * nr + r] = l;
    }
    if (a.out) {
      const bool any = l > 0.0f;
      float gt[V], o[V];
      if (a.gate)
        load_vec<V>(a.gate + e0, gt);
      else
#pragma unroll
        for (int i = 0; i < V; ++i) gt[i] = 1.0f;
#pragma unroll
      for (int i = 0; i < V; ++i) o[i] = any ? gt[i] * (acc[i] / l) : 0.0f;
      if (a.out_bf16) {
        __bf16 b[V];
#pragma unroll
        for (int i = 0; i < V; ++i) b[i] = (__bf16)o[i];
        if constexpr (V == 4)
          *reinterpret_cast<uint2*>(static_cast<__bf16*>(a.out) + e0) = *reinterpret_cast<const uint2*>(b);
        else
          *reinterpret_cast<uint32_t*>(static_cast<__bf16*>(a.out) + e0) = *reinterpret_cast<const uint32_t*>(b);
      } else {
        store_vec<V>(static_cast<float*>(a.out) + e0, o);
      }
    }
  }
}

__global__ void __launch_bounds__(256) merge4_kernel(MergeArgs a) { merge_vec<4>(a); }
__global__ void __launch_bounds__(256) merge2_kernel(MergeArgs a) { merge_vec<2>(a); }

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t st) {
  const int64_t total = a.n_rows * (int64_t)a.n_heads * a.head_dim;
  const uintptr_t align = reinterpret_cast<uintptr_t>(a.acc) | reinterpret_cast<uintptr_t>(a.acc_out) |
                          reinterpret_cast<uintptr_t>(a.gate) | reinterpret_cast<uintptr_t>(a.out);
  if (a.head_dim % 4 == 0 && total / 4 < (int64_t)INT32_MAX && (align & 15) == 0) {
    // two channels per thread where four would leave fewer than 2^18 threads
    // (small layers: twice the loads in flight, the same arithmetic)
    if (total / 4 < (1 << 18)) {
      int64_t g = (total / 2 + 255) / 256;
      if (g < 1) g = 1;
      hipLaunchKernelGGL(merge2_kernel, dim3((unsigned)g), dim3(256), 0, st, a);
      return hipGetLastError();
    }
    int64_t g = (total / 4 + 255) / 256;
    if (g > 16384) g = 16384;
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
