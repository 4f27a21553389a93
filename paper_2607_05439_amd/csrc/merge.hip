// Online-softmax merge of partial states (the combine of the paper's ring
// steps: Appendix "Q/K/V layout and the ring loop"), then out = gate*acc/l.
// One thread per (row, h*d + e); parts are folded in increasing order.
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

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t st) {
  const int64_t total = a.n_rows * (int64_t)a.n_heads * a.head_dim;
  int64_t g = (total + 255) / 256;
  if (g > 16384) g = 16384;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)g), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
