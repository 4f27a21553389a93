// Sparse (kNN) pair-biased gated attention over atoms on gfx950 (CDNA4).
//
// Paper, Methods, "RFDiffusion 3 preliminaries and notation": atom attention
// is sparse, each query atom attending to k neighbours, with the bias
// projected from the pair track P gathered at those neighbours. Appendix
// "Distributed kNN for sparse atom attention": per ring step, the neighbour
// indices are filtered to the visited column block, K, V and the bias are
// gathered there, and the logits are merged into the running softmax.
//
// Two kernels:
//   atom_proj_kernel   q, k, v, g projections of the atom single track on the
//                      matrix cores (bf16 activations; fp32 weights as a bf16
//                      hi+lo pair). The fp32 path uses the general projection.
//   sparse_attn_kernel one wave per query atom. Per key block present among
//                      its neighbours, in increasing block order:
//                        compact the block's slots into an LDS list;
//                        bias: 4 lanes per slot read the 16 pair channels,
//                        LayerNorm statistics and the 16 -> 4 projection with
//                        quad reductions;
//                        logits: each K row (4 heads x 32) is gathered by a
//                        run of lanes with 16-byte loads, one lane per 16
//                        bytes, dot products reduced across the head's lanes;
//                        online softmax in base 2 with integer block maxima
//                        (rescaling by exact powers of two);
//                        values: V rows gathered the same way, weights fp32.
//                      Gathers whose slot is past the list end use an
//                      out-of-range buffer offset: no traffic, no branch.
// The work is bound by the latency and cache bandwidth of the K/V gathers
// (neighbours of nearby atoms overlap, so most gathers hit L2); the pair
// slices are the only data read once from HBM, with the non-temporal hint.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kH = kSparseH, kD = kSparseD, kHD = kSparseH * kSparseD, kCap = kSparseCap;
constexpr int kWaves = 4;  // waves (query atoms) per workgroup
constexpr float kLog2e = 1.44269504088896340736f;
constexpr uint32_t kNt = 2;  // cache-policy bit of a buffer load: non-temporal

// ----------------------------------------------------------------------------- projections
constexpr int kProjTiles = 4;  // 16-atom tiles per wave (share the weight operands)

// grid (groups of 4 tiles of 16 atoms, head h, projection {q, k, v, g}); one
// wave each. Weight rows of head h are the A operand (rows e = 16 et + n), the
// atoms the B operand: the accumulator holds outputs 16 et + 4g + i of atom n.
__global__ void __launch_bounds__(64) atom_proj_kernel(SparseProjArgs a) {
  const int lane = threadIdx.x, n = lane & 15, g = lane >> 4;
  const int h = blockIdx.y, which = blockIdx.z;  // 0 q, 1 k, 2 v, 3 g
  const bool is_query = (which == 0 || which == 3);
  const int64_t rows = is_query ? a.n_q : a.n_atoms;
  const int64_t base = is_query ? a.q_row0 : 0;
  const int64_t tile0 = (int64_t)blockIdx.x * kProjTiles;
  if (tile0 * 16 >= rows) return;
  const float* w = which == 0 ? a.w_q : which == 1 ? a.w_k : which == 2 ? a.w_v : a.w_g;

  const uint16_t* arow[kProjTiles];
#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) {
    const int64_t row = min((tile0 + u) * 16 + n, rows - 1);  // rows past the end are not stored
    arow[u] = a.a + (base + row) * a.c_atom + 8 * g;
  }
  f32x4 acc[kProjTiles][2];
#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) acc[u][0] = acc[u][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < a.c_atom; k0 += 32) {
    bf16x8 whi[2], wlo[2];
#pragma unroll
    for (int et = 0; et < 2; ++et) {
      const float4* wp = reinterpret_cast<const float4*>(w + (int64_t)(h * kD + 16 * et + n) * a.c_atom + k0 + 8 * g);
      const float4 x0 = wp[0], x1 = wp[1];
      const float xs[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const __bf16 hv = (__bf16)xs[i];
        whi[et][i] = hv;
        wlo[et][i] = (__bf16)(xs[i] - (float)hv);
      }
    }
#pragma unroll
    for (int u = 0; u < kProjTiles; ++u) {
      const bf16x8 av = as_bf16x8(*reinterpret_cast<const u32x4*>(arow[u] + k0));
#pragma unroll
      for (int et = 0; et < 2; ++et) {
        acc[u][et] = mfma32(whi[et], av, acc[u][et]);
        acc[u][et] = mfma32(wlo[et], av, acc[u][et]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) {
    const int64_t row = (tile0 + u) * 16 + n;
    if (row >= rows) continue;
#pragma unroll
    for (int et = 0; et < 2; ++et) {
      const int o = h * kD + 16 * et + 4 * g;  // outputs o .. o+3
      if (which == 1 || which == 2) {
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (__bf16)acc[u][et][i];
        *reinterpret_cast<u32x2*>((which == 1 ? a.k : a.v) + row * kHD + o) = __builtin_bit_cast(u32x2, v);
      } else {
        float4 v;
        if (which == 0) {
          v = make_float4(acc[u][et][0], acc[u][et][1], acc[u][et][2], acc[u][et][3]);
        } else {
          v.x = 1.0f / (1.0f + __expf(-acc[u][et][0]));
          v.y = 1.0f / (1.0f + __expf(-acc[u][et][1]));
          v.z = 1.0f / (1.0f + __expf(-acc[u][et][2]));
          v.w = 1.0f / (1.0f + __expf(-acc[u][et][3]));
        }
        *reinterpret_cast<float4*>((which == 0 ? a.q : a.g) + row * kHD + o) = v;
      }
    }
  }
}

// ----------------------------------------------------------------------------- cross-lane helpers
// x combined with lane L ^ M (M = 1, 2: DPP quad permutes; 4, 8: swizzles).
template <int M>
__device__ __forceinline__ float xor_lane(float x) {
  const int xi = __float_as_int(x);
  if constexpr (M == 1) return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, true));
  if constexpr (M == 2) return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, true));
  if constexpr (M == 4) return __int_as_float(__builtin_amdgcn_ds_swizzle(xi, 0x101F));
  if constexpr (M == 8) return __int_as_float(__builtin_amdgcn_ds_swizzle(xi, 0x201F));
}

// Sum over the LANES consecutive lanes of an aligned group (1, 2, 4 or 8);
// every lane of the group gets the same bits.
template <int LANES>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (LANES >= 2) x += xor_lane<1>(x);
  if constexpr (LANES >= 4) x += xor_lane<2>(x);
  if constexpr (LANES >= 8) x += xor_lane<4>(x);
  return x;
}

// Sum / max over lanes L, L ^ 32 (GROUPS = 2) or L, L ^ 16, L ^ 32, L ^ 48 (GROUPS = 4).
template <int GROUPS>
__device__ __forceinline__ float across_sum(float x) {
  if constexpr (GROUPS == 4) return sum4(x);
  float a = x, b = x;
  swap32(a, b);
  return a + b;
}
template <int GROUPS>
__device__ __forceinline__ float across_max(float x) {
  if constexpr (GROUPS == 4) return max4(x);
  float a = x, b = x;
  swap32(a, b);
  return fmaxf(a, b);
}

__device__ __forceinline__ int wave_min(int x) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) x = min(x, __shfl_xor(x, m));
  return x;
}

// LDS written by some lanes of this wave is read by others next: keep the
// compiler from moving the accesses across this point (the LDS queue of one
// wave is in order, so no hardware wait is needed).
__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// Element e of a 16-byte chunk as fp32: bf16 pairs or fp32.
template <bool kBf16>
__device__ __forceinline__ float chunk_elem(const u32x4& w, int e) {
  if constexpr (kBf16) {
    const uint32_t x = w[e >> 1];
    return __uint_as_float((e & 1) ? (x & 0xFFFF0000u) : (x << 16));
  } else {
    return __uint_as_float(w[e]);
  }
}

// Key block of atom j under the chunk rule (block p holds floor(L/P) atoms,
// plus one for p < L mod P).
__device__ __forceinline__ int block_of(uint32_t j, uint32_t q, uint32_t rem) {
  const uint32_t big = rem * (q + 1);
  return j < big ? (int)(j / (q + 1)) : (int)(rem + (j - big) / q);
}

// ----------------------------------------------------------------------------- attention
template <bool kBf16, int KMAX>
__global__ void __launch_bounds__(64 * kWaves) sparse_attn_kernel(SparseAttnArgs a) {
  constexpr int EB = kBf16 ? 2 : 4;  // bytes per element of P, K and V
  constexpr int EPL = 16 / EB;       // K/V elements per lane per 16-byte load
  constexpr int LPN = kHD / EPL;     // lanes per K/V row (16 | 32)
  constexpr int NPI = 64 / LPN;      // rows per load instruction (4 | 2)
  constexpr int LPH = kD / EPL;      // lanes per head (4 | 8)
  constexpr int KS = KMAX / 64;      // slots per lane in slot order
  constexpr int CPL = kCap / 4;      // pair channels per lane in the bias phase
  constexpr int kUnroll = 8;
  __shared__ uint32_t s_list[kWaves][KMAX];  // (atom << 8) | slot, compacted
  __shared__ float s_lg[kWaves][KMAX][kH];   // bias, then logits (base-2 units)

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // The hardware deals workgroups to the 8 XCDs in turn; renumber them so each
  // XCD (its own L2) gets a contiguous run of query atoms, whose neighbour
  // lists overlap.
  const int64_t per = (int64_t)gridDim.x / 8;
  const int64_t lwg = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
  const int64_t r = lwg * kWaves + wave;
  if (r >= a.n_q) return;

  const int c = lane % LPN;  // 16-byte chunk of a K/V row held by this lane
  const int hl = c / LPH;    // its head
  float qv[EPL];
  {
    const float qs = kLog2e * 0.17677669529663688110f;  // log2(e) / sqrt(32)
    const float4* qp = reinterpret_cast<const float4*>(a.q + r * kHD + c * EPL);
#pragma unroll
    for (int e4 = 0; e4 < EPL / 4; ++e4) {
      const float4 t = qp[e4];
      qv[4 * e4 + 0] = t.x * qs;
      qv[4 * e4 + 1] = t.y * qs;
      qv[4 * e4 + 2] = t.z * qs;
      qv[4 * e4 + 3] = t.w * qs;
    }
  }
  // bias weights for this lane's 4 pair channels: log2(e) W_b[h, ch] gamma[ch]
  const int cq = lane & 3;
  float wb[kH][CPL];
#pragma unroll
  for (int h = 0; h < kH; ++h)
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int ch = CPL * cq + i;
      wb[h][i] = a.w_b[h * kCap + ch] * (a.gamma ? a.gamma[ch] : 1.0f) * kLog2e;
    }

  // neighbour slots in slot order: lane holds slots 64u + lane
  const uint32_t bq = (uint32_t)(a.n_atoms / a.n_kb), brem = (uint32_t)(a.n_atoms % a.n_kb);
  int32_t jn[KS];
  int blk[KS];
#pragma unroll
  for (int u = 0; u < KS; ++u) {
    const int t = 64 * u + lane;
    const int32_t j = t < a.k_slots ? a.nbr[r * a.k_slots + t] : -1;
    const bool valid = j >= 0 && (int64_t)j < a.n_atoms;
    jn[u] = j;
    blk[u] = valid ? block_of((uint32_t)j, bq, brem) : INT32_MAX;
  }

  const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(static_cast<const char*>(a.p)) + r * a.p_row_elems * EB, 0, (int)(a.p_row_elems * EB),
      kRawBufferFlags);
  const int kv_bytes = (int)(a.n_atoms * kHD * EB);
  const __amdgpu_buffer_rsrc_t kres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.k), 0, kv_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t vres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.v), 0, kv_bytes, kRawBufferFlags);
  uint32_t* list = s_list[wave];
  float(*lgs)[kH] = s_lg[wave];

  float m_run = -INFINITY, l_run = 0.0f;  // head hl; l_run over this lane's rows only
  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.0f;

  int b = INT32_MAX;
#pragma unroll
  for (int u = 0; u < KS; ++u) b = min(b, blk[u]);
  b = __builtin_amdgcn_readfirstlane(wave_min(b));
  while (b != INT32_MAX) {
    // 1. compact the slots of block b
    int count = 0;
#pragma unroll
    for (int u = 0; u < KS; ++u) {
      const bool sel = blk[u] == b;
      const uint64_t mask = __ballot(sel);
      const int pos = count + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
      if (sel) list[pos] = ((uint32_t)jn[u] << 8) | (uint32_t)(64 * u + lane);
      count += __popcll(mask);
    }
    wave_lds_sync();

    // 2. bias of each listed slot: 4 lanes per slot, 16 slots per pass
    for (int p0 = 0; p0 < count; p0 += 16) {
      const int pos = p0 + (lane >> 2);
      const bool ok = pos < count;
      const uint32_t ent = list[ok ? pos : 0];
      const uint32_t idx = a.p_gathered ? (ent & 255u) : (ent >> 8);
      const int voff = ok ? (int)(idx * (uint32_t)(kCap * EB) + (uint32_t)(cq * CPL * EB)) : kOutOfRange;
      float x[CPL];
      if constexpr (kBf16) {
        const u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(pres, voff, 0, kNt);
        x[0] = __uint_as_float(w[0] << 16);
        x[1] = __uint_as_float(w[0] & 0xFFFF0000u);
        x[2] = __uint_as_float(w[1] << 16);
        x[3] = __uint_as_float(w[1] & 0xFFFF0000u);
      } else {
        const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(pres, voff, 0, kNt);
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(w[i]);
      }
      const float mu = group_sum<4>((x[0] + x[1]) + (x[2] + x[3])) * (1.0f / kCap);
      float dv[CPL], ss = 0.0f;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        dv[i] = x[i] - mu;
        ss = fmaf(dv[i], dv[i], ss);
      }
      const float rstd = __builtin_amdgcn_rsqf(group_sum<4>(ss) * (1.0f / kCap) + a.eps);
      float hp[kH];
#pragma unroll
      for (int h = 0; h < kH; ++h) {
        float t = 0.0f;
#pragma unroll
        for (int i = 0; i < CPL; ++i) t = fmaf(wb[h][i], dv[i], t);
        hp[h] = group_sum<4>(t);
      }
      const float mine = cq == 0 ? hp[0] : cq == 1 ? hp[1] : cq == 2 ? hp[2] : hp[3];
      if (ok) lgs[pos][cq] = rstd * mine;
    }
    wave_lds_sync();

    // 3. logits: K rows, NPI per load instruction, lane chunk c
    const int n_ins = (count + NPI - 1) / NPI;
    float mx = -INFINITY;
    for (int i0 = 0; i0 < n_ins; i0 += kUnroll) {
      u32x4 kw[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int pos = NPI * (i0 + u) + lane / LPN;
        const bool ok = pos < count;
        const uint32_t j = list[ok ? pos : 0] >> 8;
        kw[u] = __builtin_amdgcn_raw_buffer_load_b128(kres, ok ? (int)(j * (uint32_t)(kHD * EB) + 16u * c) : kOutOfRange,
                                                      0, 0);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int pos = NPI * (i0 + u) + lane / LPN;
        const bool ok = pos < count;
        float dot = 0.0f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) dot = fmaf(qv[e], chunk_elem<kBf16>(kw[u], e), dot);
        dot = group_sum<LPH>(dot);
        if (ok) {
          const float lg = dot + lgs[pos][hl];
          if ((lane % LPH) == 0) lgs[pos][hl] = lg;
          mx = fmaxf(mx, lg);
        }
      }
    }
    mx = across_max<NPI>(mx);
    const float mb = ceilf(mx);  // integer block maximum (or -inf)
    const float m_new = fmaxf(m_run, mb);
    const float sr = m_run == -INFINITY ? 0.0f : ldexpf(1.0f, (int)(m_run - m_new));
    l_run *= sr;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] *= sr;
    m_run = m_new;
    wave_lds_sync();

    // 4. values: V rows, weights exp2(logit - m)
    for (int i0 = 0; i0 < n_ins; i0 += kUnroll) {
      u32x4 vw[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int pos = NPI * (i0 + u) + lane / LPN;
        const bool ok = pos < count;
        const uint32_t j = list[ok ? pos : 0] >> 8;
        vw[u] = __builtin_amdgcn_raw_buffer_load_b128(vres, ok ? (int)(j * (uint32_t)(kHD * EB) + 16u * c) : kOutOfRange,
                                                      0, 0);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int pos = NPI * (i0 + u) + lane / LPN;
        const bool ok = pos < count && m_new != -INFINITY;
        const float p = ok ? __builtin_amdgcn_exp2f(lgs[pos < count ? pos : 0][hl] - m_new) : 0.0f;
        l_run += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = fmaf(p, chunk_elem<kBf16>(vw[u], e), acc[e]);
      }
    }

    // next block present among the neighbours
    int nb = INT32_MAX;
#pragma unroll
    for (int u = 0; u < KS; ++u) nb = min(nb, blk[u] > b ? blk[u] : INT32_MAX);
    b = __builtin_amdgcn_readfirstlane(wave_min(nb));
    wave_lds_sync();
  }

  const float l = across_sum<NPI>(l_run);
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = across_sum<NPI>(acc[e]);
  if (lane < LPN) {
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
    const float4* gp = reinterpret_cast<const float4*>(a.g + r * kHD + c * EPL);
    float o[EPL];
#pragma unroll
    for (int e4 = 0; e4 < EPL / 4; ++e4) {
      const float4 t = gp[e4];
      o[4 * e4 + 0] = t.x * (acc[4 * e4 + 0] * inv);
      o[4 * e4 + 1] = t.y * (acc[4 * e4 + 1] * inv);
      o[4 * e4 + 2] = t.z * (acc[4 * e4 + 2] * inv);
      o[4 * e4 + 3] = t.w * (acc[4 * e4 + 3] * inv);
    }
    if (a.out_bf16) {
      __bf16* op = static_cast<__bf16*>(a.out) + r * kHD + c * EPL;
#pragma unroll
      for (int e = 0; e < EPL; ++e) op[e] = (__bf16)o[e];
    } else {
      float4* op = reinterpret_cast<float4*>(static_cast<float*>(a.out) + r * kHD + c * EPL);
#pragma unroll
      for (int e4 = 0; e4 < EPL / 4; ++e4)
        op[e4] = make_float4(o[4 * e4 + 0], o[4 * e4 + 1], o[4 * e4 + 2], o[4 * e4 + 3]);
    }
  }
}

template <bool kBf16, int KMAX>
hipError_t launch_attn(const SparseAttnArgs& a, hipStream_t st) {
  const int64_t n_wg = (a.n_q + kWaves - 1) / kWaves;
  const int64_t grid = (n_wg + 7) / 8 * 8;
  hipLaunchKernelGGL((sparse_attn_kernel<kBf16, KMAX>), dim3((unsigned)grid), dim3(64 * kWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_proj(const SparseProjArgs& a, hipStream_t st) {
  const int64_t rows = a.n_atoms > a.n_q ? a.n_atoms : a.n_q;
  const int64_t groups = ((rows + 15) / 16 + kProjTiles - 1) / kProjTiles;
  hipLaunchKernelGGL(atom_proj_kernel, dim3((unsigned)groups, kH, 4), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, bool bf16, hipStream_t st) {
  if (a.k_slots <= 128) return bf16 ? launch_attn<true, 128>(a, st) : launch_attn<false, 128>(a, st);
  return bf16 ? launch_attn<true, 256>(a, st) : launch_attn<false, 256>(a, st);
}

}  // namespace dcp
