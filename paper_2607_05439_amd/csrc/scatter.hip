// Deterministic atom -> token mean pooling on gfx950.
//
// Appendix "Non-determinism guard" and the 2D pooling boundary: atom features
// are averaged per token; a floating-point atomic index_reduce("mean") gives
// results that depend on scheduling, so the paper broadcasts one rank's
// result (1D) or uses a deterministic collective (2D). Here the reduction is
// deterministic by construction on any device: every feature is converted to a
// 64-bit fixed-point integer (value * 2^32, rounded to nearest), and integer
// addition is associative, so the per-token sums do not depend on the order in
// which atoms are added, whatever the index pattern.
//
//   scatter_zero_kernel   clears the fixed-point sums and the counts (a fill
//                         kernel, so the call can be captured in a graph)
//   scatter_accum_kernel  one wave per run of 64 consecutive atoms, lanes over
//                         channels: runs of atoms with the same token are summed
//                         in registers (exact), and each run adds its sum with
//                         one 64-bit atomic per channel and one count atomic;
//                         with atoms ordered by token that is about one atomic
//                         per (token, channel)
//   scatter_final_kernel  out = sum * 2^-32 / count (0 for a token without atoms)
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kRun = 64;  // atoms per wave (longer runs: fewer token boundaries, fewer atomics)
constexpr double kFix = 4294967296.0;  // 2^32
constexpr double kFixMax = 1073741824.0;  // |feature| clamp: 2^30

__global__ void __launch_bounds__(256) scatter_zero_kernel(ScatterArgs a) {
  const int64_t n = a.n_tokens * a.c;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) a.acc[i] = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < a.n_tokens; i += (int64_t)gridDim.x * 256) a.cnt[i] = 0;
}

__device__ __forceinline__ long long to_fixed(float x) {
  double v = (double)x;
  v = v > kFixMax ? kFixMax : (v < -kFixMax ? -kFixMax : v);  // NaN passes through as NaN
  return __double2ll_rn(v * kFix);
}

template <bool kBf16, int CPL>
__global__ void __launch_bounds__(256) scatter_accum_kernel(ScatterArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t run = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t i0 = run * kRun;
  if (i0 >= a.n_atoms) return;
  const int64_t i1 = min(i0 + kRun, a.n_atoms);
  long long sum[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) sum[j] = 0;
  int32_t cur = -1;
  uint32_t seg = 0;
  auto flush = [&]() {
    if (seg != 0 && cur >= 0 && (int64_t)cur < a.n_tokens) {
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int ch = lane + 64 * j;
        if (ch < a.c)
          atomicAdd(reinterpret_cast<unsigned long long*>(a.acc) + (int64_t)cur * a.c + ch,
                    (unsigned long long)sum[j]);
      }
      if (lane == 0) atomicAdd(a.cnt + cur, seg);
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) sum[j] = 0;
    seg = 0;
  };
  constexpr int kU = 8;  // atoms whose index and features are loaded together
  for (int64_t ib = i0; ib < i1; ib += kU) {
    int32_t tv[kU];
    float xv[kU][CPL];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = min(ib + u, i1 - 1);  // a clamped repeat past the end is skipped below
      tv[u] = __builtin_amdgcn_readfirstlane(a.tok_idx[i]);
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int ch = min(lane + 64 * j, a.c - 1);
        if constexpr (kBf16)
          xv[u][j] = __uint_as_float((uint32_t)static_cast<const uint16_t*>(a.a)[i * a.c + ch] << 16);
        else
          xv[u][j] = static_cast<const float*>(a.a)[i * a.c + ch];
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (ib + u >= i1) break;
      if (tv[u] != cur) {
        flush();
        cur = tv[u];
      }
#pragma unroll
      for (int j = 0; j < CPL; ++j) sum[j] += to_fixed(xv[u][j]);
      ++seg;
    }
  }
  flush();
}

__global__ void __launch_bounds__(256) scatter_final_kernel(ScatterArgs a) {
  const int64_t n = a.n_tokens * a.c;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / a.c;
    const uint32_t k = a.cnt[t];
    const float v = k ? (float)((double)a.acc[i] / kFix / (double)k) : 0.0f;
    if (a.out_bf16)
      static_cast<__bf16*>(a.out)[i] = (__bf16)v;
    else
      static_cast<float*>(a.out)[i] = v;
  }
}

unsigned grid_of(int64_t items) {
  int64_t g = (items + 255) / 256;
  if (g > 16384) g = 16384;
  return (unsigned)(g < 1 ? 1 : g);
}

template <bool kBf16>
void launch_accum(const ScatterArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.n_atoms + 4 * kRun - 1) / (4 * kRun))), block(256);
  if (a.c <= 64)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 1>), grid, block, 0, st, a);
  else if (a.c <= 128)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 2>), grid, block, 0, st, a);
  else if (a.c <= 256)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 4>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 8>), grid, block, 0, st, a);
}

}  // namespace

hipError_t launch_scatter_mean(const ScatterArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(scatter_zero_kernel, dim3(grid_of(a.n_tokens * a.c)), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.n_atoms > 0) {
    if (a.a_bf16)
      launch_accum<true>(a, st);
    else
      launch_accum<false>(a, st);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(scatter_final_kernel, dim3(grid_of(a.n_tokens * a.c)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
