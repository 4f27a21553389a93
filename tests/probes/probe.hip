// In-bounds checks of the gfx950 builtins' lane layouts that the fused kernels
// rely on (matrix-core accumulator layout, cross-lane swaps, the bias-tile
// transpose). Each kernel is one wave of 64 lanes writing 64 x K floats.
#include <hip/hip_runtime.h>

#include "cdna4.h"

namespace {
using namespace dcp;

__global__ void __launch_bounds__(64) k_mfma32(float* out) {
  const int L = threadIdx.x, n = L & 15, g = L >> 4;
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    const int k = 8 * g + i;
    a[i] = (__bf16)(k == n ? 1.0f : 0.0f);
    b[i] = (__bf16)(k < 16 ? (float)(k * 16 + n) : 0.0f);
  }
  const f32x4 d = mfma32(a, b, f32x4{0.f, 0.f, 0.f, 0.f});
  for (int i = 0; i < 4; ++i) out[L * 4 + i] = d[i];
}

__global__ void __launch_bounds__(64) k_mfma16(float* out) {
  const int L = threadIdx.x, n = L & 15, g = L >> 4;
  bf16x4 a, b;
  for (int i = 0; i < 4; ++i) {
    const int k = 4 * g + i;
    a[i] = (__bf16)(k == n ? 1.0f : 0.0f);
    b[i] = (__bf16)(float)(k * 16 + n);
  }
  const f32x4 d = mfma16(a, b, f32x4{0.f, 0.f, 0.f, 0.f});
  for (int i = 0; i < 4; ++i) out[L * 4 + i] = d[i];
}

__global__ void __launch_bounds__(64) k_swaps(float* out) {
  const int L = threadIdx.x;
  float x = (float)L, y = (float)(100 + L);
  swap32(x, y);
  out[L * 6 + 0] = x;
  out[L * 6 + 1] = y;
  float u = (float)L, v = (float)(100 + L);
  swap16(u, v);
  out[L * 6 + 2] = u;
  out[L * 6 + 3] = v;
  out[L * 6 + 4] = sum4((float)L);
  out[L * 6 + 5] = max4((float)((L * 37) % 64));
}

__global__ void __launch_bounds__(64) k_transpose(float* out) {
  const int L = threadIdx.x;
  float b[16][4];
  for (int k = 0; k < 16; ++k)
    for (int i = 0; i < 4; ++i) b[k][i] = (float)(L * 64 + k * 4 + i);
  transpose_bias(b);
  for (int k = 0; k < 16; ++k)
    for (int i = 0; i < 4; ++i) out[L * 64 + k * 4 + i] = b[k][i];
}

__global__ void __launch_bounds__(64) k_exp2(const float* in, float* out, int n) {
  for (int t = threadIdx.x; t < n; t += 64) out[t] = __builtin_amdgcn_exp2f(in[t]);
}

// Direct-to-LDS loads: per-lane source offsets, destinations below and above
// 64 KB of LDS, and one load with an out-of-range offset.
__global__ void __launch_bounds__(256) k_dma(const u32x4* g, u32x4* out) {
  __shared__ u32x4 lds[10240];  // 160 KB
  for (int i = threadIdx.x; i < 10240; i += 256) lds[i] = u32x4{0xDEAD0000u | (uint32_t)i, 1u, 2u, 3u};
  __syncthreads();
  const int L = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void*)g, 0, 192 * 16, kRawBufferFlags);
  if (wave == 0) {
    dma_b128(r, 16 * (L ^ 5), lds_addr(&lds[0]));
    dma_b128(r, 1024 + 16 * (L ^ 9), lds_addr(&lds[71680 / 16]));
    dma_b128(r, kOutOfRange, lds_addr(&lds[102400 / 16]));
    dma_b128(r, 2048 + 16 * (L ^ 3), lds_addr(&lds[154624 / 16]));
    wait_vm<0>();
  }
  __syncthreads();
  if (wave == 0) {
    out[L] = lds[L];
    out[64 + L] = lds[71680 / 16 + L];
    out[128 + L] = lds[102400 / 16 + L];
    out[192 + L] = lds[154624 / 16 + L];
  }
}

}  // namespace

extern "C" {
int probe_dma(const void* g, void* out) { hipLaunchKernelGGL(k_dma, dim3(1), dim3(256), 0, 0, (const u32x4*)g, (u32x4*)out); return hipDeviceSynchronize(); }
int probe_mfma32(float* out) { hipLaunchKernelGGL(k_mfma32, dim3(1), dim3(64), 0, 0, out); return hipDeviceSynchronize(); }
int probe_mfma16(float* out) { hipLaunchKernelGGL(k_mfma16, dim3(1), dim3(64), 0, 0, out); return hipDeviceSynchronize(); }
int probe_swaps(float* out) { hipLaunchKernelGGL(k_swaps, dim3(1), dim3(64), 0, 0, out); return hipDeviceSynchronize(); }
int probe_transpose(float* out) { hipLaunchKernelGGL(k_transpose, dim3(1), dim3(64), 0, 0, out); return hipDeviceSynchronize(); }
int probe_exp2(const float* in, float* out, int n) { hipLaunchKernelGGL(k_exp2, dim3(1), dim3(64), 0, 0, in, out, n); return hipDeviceSynchronize(); }
}
