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
// bf16 path: logits in base-2 units are offset by this constant (through the
// bias), so every logit of moderate size lies in [128, 256), on one fp32 grid
// (2^-16). With integer running maxima the subtraction logit - max is then
// exact, and the bf16-rounded softmax weights do not depend on how the slots
// are split into key blocks (rescaling is by exact powers of two).
constexpr float kShift = 192.0f;

// ----------------------------------------------------------------------------- projections
constexpr int kProjTiles = 4;  // 16-atom tiles per wave (share the weight operands)

// Any c_atom (a multiple of 32). grid (groups of 4 tiles of 16 atoms, head h,
// projection {q, k, v, g}); one wave each. Weight rows of head h are the A
// operand (rows e = 16 et + n), the atoms the B operand: the accumulator holds
// outputs 16 et + 4g + i of atom n.
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

// c_atom = 128 (the paper's atom width). blockIdx.y picks the projection
// (0 q, 1 k, 2 v, 3 g; q and g over the query rows, k and v over all atoms).
// Its weight matrix is converted once per workgroup into matrix-core A
// operands in LDS (bf16 hi + lo, 64 KB, so two workgroups share a CU); each
// wave then takes 4 tiles of 16 atoms at a time, holds their B operands in
// registers, and runs all 128 outputs against them.
constexpr int kP128Ks = 4;  // 32-channel k-steps
struct ProjOperands {
  u32x4 w[8][kP128Ks][2][64];  // [output tile][k-step][hi, lo][lane]
};

__global__ void __launch_bounds__(256, 2) atom_proj128_kernel(SparseProjArgs a) {
  __shared__ ProjOperands ops;
  const int which = blockIdx.y;
  const bool query = which == 0 || which == 3;
  const int64_t rows = query ? a.n_q : a.n_atoms;
  const int64_t base = query ? a.q_row0 : 0;
  const int64_t n_groups = (rows + 63) / 64;
  if ((int64_t)blockIdx.x * 4 >= n_groups) return;  // whole workgroup, before any barrier
  const float* wsrc = which == 0 ? a.w_q : which == 1 ? a.w_k : which == 2 ? a.w_v : a.w_g;
  constexpr int kEntries = 8 * kP128Ks * 64;  // 8 per thread, 4 at a time with their loads in flight
  for (int i0 = threadIdx.x; i0 < kEntries; i0 += 4 * 256) {
    float4 x[4][2];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int idx = i0 + 256 * v;
      const int ln = idx & 63, ks = (idx >> 6) % kP128Ks, ot = (idx >> 6) / kP128Ks;
      const float4* wp = reinterpret_cast<const float4*>(wsrc + (16 * ot + (ln & 15)) * kHD + 32 * ks + 8 * (ln >> 4));
      x[v][0] = wp[0];
      x[v][1] = wp[1];
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int idx = i0 + 256 * v;
      const int ln = idx & 63, ks = (idx >> 6) % kP128Ks, ot = (idx >> 6) / kP128Ks;
      const float xs[8] = {x[v][0].x, x[v][0].y, x[v][0].z, x[v][0].w, x[v][1].x, x[v][1].y, x[v][1].z, x[v][1].w};
      bf16x8 hi, lo;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        hi[i] = (__bf16)xs[i];
        lo[i] = (__bf16)(xs[i] - (float)hi[i]);
      }
      ops.w[ot][ks][0][ln] = __builtin_bit_cast(u32x4, hi);
      ops.w[ot][ks][1][ln] = __builtin_bit_cast(u32x4, lo);
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int64_t grp = (int64_t)blockIdx.x * 4 + wave; grp < n_groups; grp += (int64_t)gridDim.x * 4) {
    u32x4 av[4][kP128Ks];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t row = min(grp * 64 + 16 * u + n, rows - 1);  // rows past the end are not stored
      const u32x4* ap = reinterpret_cast<const u32x4*>(a.a + (base + row) * kHD + 8 * g);
#pragma unroll
      for (int ks = 0; ks < kP128Ks; ++ks) av[u][ks] = ap[4 * ks];
    }
#pragma unroll 2
    for (int ot = 0; ot < 8; ++ot) {
      f32x4 acc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < kP128Ks; ++ks) {
        const bf16x8 hi = as_bf16x8(ops.w[ot][ks][0][lane]);
        const bf16x8 lo = as_bf16x8(ops.w[ot][ks][1][lane]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc[u] = mfma32(hi, as_bf16x8(av[u][ks]), acc[u]);
          acc[u] = mfma32(lo, as_bf16x8(av[u][ks]), acc[u]);
        }
      }
      const int o = 16 * ot + 4 * g;  // outputs o .. o+3 of the atom row
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t row = grp * 64 + 16 * u + n;
        if (row >= rows) continue;
        if (which == 1 || which == 2) {
          bf16x4 v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = (__bf16)acc[u][i];
          *reinterpret_cast<u32x2*>((which == 1 ? a.k : a.v) + row * kHD + o) = __builtin_bit_cast(u32x2, v);
        } else if (which == 0) {
          *reinterpret_cast<float4*>(a.q + row * kHD + o) = make_float4(acc[u][0], acc[u][1], acc[u][2], acc[u][3]);
        } else {
          float4 v;
          v.x = 1.0f / (1.0f + __expf(-acc[u][0]));
          v.y = 1.0f / (1.0f + __expf(-acc[u][1]));
          v.z = 1.0f / (1.0f + __expf(-acc[u][2]));
          v.w = 1.0f / (1.0f + __expf(-acc[u][3]));
          *reinterpret_cast<float4*>(a.g + row * kHD + o) = v;
        }
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
// Maximum of two floats as one v_max_f32: fmaxf would first canonicalise
// operands that come from cross-lane moves (two more instructions each); the
// instruction itself already returns the other operand for a NaN one.
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
template <int GROUPS>
__device__ __forceinline__ float across_max(float x) {
  float a = x, b = x;
  swap32(a, b);
  x = vmax(a, b);
  if constexpr (GROUPS == 4) {
    a = x;
    b = x;
    swap16(a, b);
    x = vmax(a, b);
  }
  return x;
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
// Bias operands of the 16x16x16 matrix-core form (bf16 path): row h < 4 holds
// W''[h, c] = log2(e) W_b[h, c] gamma_c, centred over c (then sum_c W''[h,c] p_c
// = sum_c W''[h,c] (p_c - mean p)), split into bf16 hi + lo; row 4 holds ones
// in hi (the row sum of the pair vector); other rows are zero. Lane L: row
// L % 16, channels 4g .. 4g+3 with g = L / 16.
__device__ __forceinline__ void bias_operands(const float* __restrict__ w_b, const float* __restrict__ gamma, int lane,
                                              bf16x4& hi, bf16x4& lo) {
  const int n = lane & 15, g = lane >> 4;
  float w[4], rs = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = 4 * g + i;
    w[i] = n < kH ? w_b[n * kCap + ch] * (gamma ? gamma[ch] : 1.0f) * kLog2e : 0.0f;
    rs += w[i];
  }
  const float mean = sum4(rs) * (1.0f / kCap);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float cw = w[i] - mean;
    const __bf16 x = (__bf16)cw;
    hi[i] = n < kH ? x : (n == kH ? (__bf16)1.0f : (__bf16)0.0f);
    lo[i] = n < kH ? (__bf16)(cw - (float)x) : (__bf16)0.0f;
  }
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(a), as_bf16x2(b), c, false);
}

template <bool kBf16, int KMAX>
__global__ void __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(kBf16 && KMAX == 128 ? 5 : 1)))
sparse_attn_kernel(SparseAttnArgs a) {
  constexpr int EB = kBf16 ? 2 : 4;  // bytes per element of P, K and V
  constexpr int EPL = 16 / EB;       // K/V elements per lane per 16-byte load
  constexpr int LPN = kHD / EPL;     // lanes per K/V row (16 | 32)
  constexpr int NPI = 64 / LPN;      // rows per load instruction (4 | 2)
  constexpr int LPH = kD / EPL;      // lanes per head (4 | 8)
  constexpr int KS = KMAX / 64;      // slots per lane in slot order
  constexpr int kUnroll = 2;         // K (and V) loads per lane per batch (few: more waves fit)
  constexpr int kBatch = NPI * kUnroll;  // slots per batch (8 | 4)
  constexpr int kPad = 32;           // list length granularity
  constexpr int kPasses = KMAX / 16; // bias passes of 16 slots
  static_assert(kPad % 16 == 0 && kPad % kBatch == 0 && KMAX % kPad == 0, "list padding");
  __shared__ uint32_t s_kv[kWaves][KMAX + kBatch];  // byte offset of the K/V row, or out of range (padding)
  __shared__ uint32_t s_p[kWaves][KMAX];   // byte offset of the pair vector in this query's P row
  __shared__ __attribute__((aligned(16))) float s_b[kWaves][KMAX][kH];  // bias (base-2 units), -inf for padding

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // The hardware deals workgroups to the 8 XCDs in turn; renumber them so each
  // XCD (its own L2) gets a contiguous run of query atoms, whose neighbour
  // lists overlap.
  const int64_t per = (int64_t)gridDim.x / 8;
  const int64_t lwg = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
  const int64_t r = lwg * kWaves + wave;
  if (r >= a.n_q) return;

  const int c = lane % LPN;    // 16-byte chunk of a K/V row held by this lane
  const int grp = lane / LPN;  // which of the NPI rows of a load
  const int hl = c / LPH;      // head of the chunk
  // q slice, scaled into base-2 logit units (log2(e) / sqrt(32))
  float qv[EPL];
  {
    const float qs = kLog2e * 0.17677669529663688110f;
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
  uint32_t qhi[4], qlo[4];  // bf16 path: q as a bf16 hi + lo pair, packed by element pairs
  if constexpr (kBf16) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      qhi[w] = pack_bf16(qv[2 * w], qv[2 * w + 1]);
      const bf16x2 h = as_bf16x2(qhi[w]);
      qlo[w] = pack_bf16(qv[2 * w] - (float)h[0], qv[2 * w + 1] - (float)h[1]);
    }
  }
  bf16x4 whi, wlo;       // bf16 path: bias operands
  float wb[kH][4] = {};  // fp32 path: log2(e) W_b[h, ch] gamma[ch] for this lane's 4 channels
  float wsum[kH] = {};   // bf16 path: per-head sums of the hi + lo operands (wave-uniform)
  if constexpr (kBf16) {
    bias_operands(a.w_b, a.gamma, lane, whi, wlo);
    bf16x4 ones;
#pragma unroll
    for (int i = 0; i < 4; ++i) ones[i] = (__bf16)1.0f;
    f32x4 r = {0.f, 0.f, 0.f, 0.f};
    r = mfma16(whi, ones, r);
    r = mfma16(wlo, ones, r);  // rows 0..3 (the heads) of every column, in lane group 0
#pragma unroll
    for (int h = 0; h < kH; ++h) wsum[h] = __builtin_amdgcn_readfirstlane(r[h]);
  } else {
#pragma unroll
    for (int h = 0; h < kH; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ch = 4 * (lane & 3) + i;
        wb[h][i] = a.w_b[h * kCap + ch] * (a.gamma ? a.gamma[ch] : 1.0f) * kLog2e;
      }
  }

  // neighbour slots in slot order: lane holds slots 64u + lane
  const uint32_t bq = (uint32_t)(a.n_atoms / a.n_kb), brem = (uint32_t)(a.n_atoms % a.n_kb);
  uint32_t kvo[KS], po[KS];
  int blk[KS];
#pragma unroll
  for (int u = 0; u < KS; ++u) {
    const int t = 64 * u + lane;
    const int32_t j = t < a.k_slots ? a.nbr[r * a.k_slots + t] : -1;
    const bool valid = j >= 0 && (int64_t)j < a.n_atoms;
    blk[u] = valid ? block_of((uint32_t)j, bq, brem) : INT32_MAX;
    kvo[u] = (uint32_t)j * (uint32_t)(kHD * EB);
    po[u] = (a.p_gathered ? (uint32_t)t : (uint32_t)j) * (uint32_t)(kCap * EB);
  }

  const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(static_cast<const char*>(a.p)) + r * a.p_row_elems * EB, 0, (int)(a.p_row_elems * EB),
      kRawBufferFlags);
  const int kv_bytes = (int)(a.n_atoms * kHD * EB);
  const __amdgpu_buffer_rsrc_t kres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.k), 0, kv_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t vres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.v), 0, kv_bytes, kRawBufferFlags);
  uint32_t* lkv = s_kv[wave];
  uint32_t* lp = s_p[wave];
  float(*lb)[kH] = s_b[wave];

  // running softmax state of head hl: integer maximum m (base-2 units), and
  // this lane's share of l and acc (summed over the NPI row groups at the end)
  float m_run = -INFINITY, l_run = 0.0f;
  float acc[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) acc[e] = 0.0f;

  // one register buffer of K rows and one of V rows per batch; the next
  // batch's K rows are requested as soon as this batch's logits are formed and
  // its V rows as soon as this batch's weighted sum is done (more buffers cost
  // occupancy, which hides the gather latency better)
  u32x4 kw[1][kUnroll], vw[1][kUnroll];
  auto offsets = [&](int b0, int (&off)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) off[u] = (int)(lkv[b0 + NPI * u + grp] + 16u * c);
  };
  auto issue_k = [&](int buf, const int (&off)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) kw[buf][u] = __builtin_amdgcn_raw_buffer_load_b128(kres, off[u], 0, 0);
  };
  auto issue_v = [&](int buf, const int (&off)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) vw[buf][u] = __builtin_amdgcn_raw_buffer_load_b128(vres, off[u], 0, 0);
  };
  // one batch: logits (the only use of the K rows) ...
  auto logits = [&](int buf, int b0, float (&lg)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      float dot = 0.0f;
      if constexpr (kBf16) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          dot = dot2(qhi[w], kw[buf][u][w], dot);
          dot = dot2(qlo[w], kw[buf][u][w], dot);
        }
      } else {
#pragma unroll
        for (int e = 0; e < EPL; ++e) dot = fmaf(qv[e], __uint_as_float(kw[buf][u][e]), dot);
      }
      lg[u] = group_sum<LPH>(dot) + lb[b0 + NPI * u + grp][hl];
    }
  };
  // ... then the online softmax (integer maxima, exact power-of-two
  // rescaling) and the weighted V
  auto weigh = [&](int buf, const float (&lg)[kUnroll]) {
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) mx = vmax(mx, lg[u]);
    mx = across_max<NPI>(mx);
    const float m_new = fmaxf(m_run, ceilf(mx));
    if (m_new != m_run) {  // lane-varying (per head); only a rescale of the state
      const float sr = m_run == -INFINITY ? 0.0f : ldexpf(1.0f, (int)(m_run - m_new));
      l_run *= sr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] *= sr;
      m_run = m_new;
    }
    const float m_use = m_run == -INFINITY ? 0.0f : m_run;
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const float p = __builtin_amdgcn_exp2f(lg[u] - m_use);
      if constexpr (kBf16) {
        // the weight as bf16 pairs (p, 0) and (0, p): one dot2 per element (no
        // constant operands in the dot2: an inline constant is not read as a
        // packed bf16 pair)
        const uint32_t plo = pack_bf16(p, 0.0f), phi = plo << 16;
        l_run += __uint_as_float(phi);  // bf16(p) as fp32: the weight the numerator uses
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          acc[2 * w] = dot2(plo, vw[buf][u][w], acc[2 * w]);
          acc[2 * w + 1] = dot2(phi, vw[buf][u][w], acc[2 * w + 1]);
        }
      } else {
        l_run += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = fmaf(p, __uint_as_float(vw[buf][u][e]), acc[e]);
      }
    }
  };

  int b = INT32_MAX;
#pragma unroll
  for (int u = 0; u < KS; ++u) b = min(b, blk[u]);
  b = __builtin_amdgcn_readfirstlane(wave_min(b));
  while (b != INT32_MAX) {
    // 1. compact the slots of block b; pad the list to a multiple of kPad with
    //    out-of-range offsets (those loads move no data)
    int count = 0;
#pragma unroll
    for (int u = 0; u < KS; ++u) {
      const bool sel = blk[u] == b;
      const uint64_t mask = __ballot(sel);
      const int pos = count + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
      if (sel) {
        lkv[pos] = kvo[u];
        lp[pos] = po[u];
      }
      count += __popcll(mask);
    }
    const int count_pad = (count + kPad - 1) / kPad * kPad;
    if (lane < count_pad - count) lp[count + lane] = (uint32_t)kOutOfRange;
    if (lane < count_pad - count + kBatch) lkv[count + lane] = (uint32_t)kOutOfRange;  // and one more batch
    wave_lds_sync();

    // 2. every pair-vector load of the list, then the first batch's K rows, so
    //    the bias work below overlaps their latency
    if constexpr (kBf16) {
      // 16 slots per pass on the matrix cores: lane (n, g) holds channels
      // 4g..4g+3 of slot n; W''.p gives the heads (rows 0..3) and the row sum
      // (row 4); the diagonal of the Gram tile p.p^T the sums of squares.
      const int n = lane & 15, g = lane >> 4;
      u32x2 pw[kPasses];
#pragma unroll
      for (int ps = 0; ps < kPasses; ++ps) {
        const int off = 16 * ps < count_pad ? (int)(lp[16 * ps + n] + 8u * g) : kOutOfRange;
        pw[ps] = __builtin_amdgcn_raw_buffer_load_b64(pres, off, 0, kNt);
      }
      {  // the first batch's K rows; its V rows follow the bias work
        int o0[kUnroll];
        offsets(0, o0);
        issue_k(0, o0);
      }
#pragma unroll
      for (int ps = 0; ps < kPasses; ++ps) {
        if (16 * ps >= count_pad) break;
        const int pos = 16 * ps + n;
        const bf16x4 pv = as_bf16x4(pw[ps]);
        const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
        f32x4 hb = mfma16(whi, pv, zero);
        hb = mfma16(wlo, pv, hb);
        const f32x4 gram = mfma16(pv, pv, zero);
        // diagonal entry of column n: row n sits in lane group n/4, register n%4
        const float t0 = (n & 1) ? gram[1] : gram[0];
        const float t1 = (n & 1) ? gram[3] : gram[2];
        float d = (n & 2) ? t1 : t0;
        const int tg = n >> 2;
        float x0 = d, x1 = d;
        swap32(x0, x1);
        d = (tg & 2) ? x1 : x0;
        x0 = d;
        x1 = d;
        swap16(x0, x1);
        const float s2 = (tg & 1) ? x1 : x0;
        // row sum: row 4 is register 0 of lane group 1; bring it to group 0
        float y0 = hb[0], y1 = hb[0];
        swap16(y0, y1);
        const float mu = y1 * (1.0f / kCap);
        // one rounding of s2/c - mu^2 (the square exact inside the fma), and the
        // operands' own per-head sums times mu removed: exact centring even
        // when the channel mean is large against the spread
        const float var = fmaxf(fmaf(-mu, mu, s2 * (1.0f / kCap)), 0.0f);
        const float rstd = __builtin_amdgcn_rsqf(var + a.eps);
        if (g == 0) {
          const bool ok = pos < count;
          float hc[kH];
#pragma unroll
          for (int h = 0; h < kH; ++h) hc[h] = fmaf(-mu, wsum[h], hb[h]);
          *reinterpret_cast<float4*>(lb[pos]) =
              ok ? make_float4(fmaf(rstd, hc[0], kShift), fmaf(rstd, hc[1], kShift), fmaf(rstd, hc[2], kShift),
                               fmaf(rstd, hc[3], kShift))
                 : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        }
      }
    } else {
      // 4 lanes per slot, 16 slots per pass; quad reductions
      const int cq = lane & 3;
      u32x4 pw[kPasses];
#pragma unroll
      for (int ps = 0; ps < kPasses; ++ps) {
        const int off = 16 * ps < count_pad ? (int)(lp[16 * ps + (lane >> 2)] + 16u * cq) : kOutOfRange;
        pw[ps] = __builtin_amdgcn_raw_buffer_load_b128(pres, off, 0, kNt);
      }
      {  // the first batch's K rows; its V rows follow the bias work
        int o0[kUnroll];
        offsets(0, o0);
        issue_k(0, o0);
      }
#pragma unroll
      for (int ps = 0; ps < kPasses; ++ps) {
        if (16 * ps >= count_pad) break;
        const int pos = 16 * ps + (lane >> 2);
        float x[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(pw[ps][i]);
        const float mu = group_sum<4>((x[0] + x[1]) + (x[2] + x[3])) * (1.0f / kCap);
        float dv[4], ss = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dv[i] = x[i] - mu;
          ss = fmaf(dv[i], dv[i], ss);
        }
        const float rstd = __builtin_amdgcn_rsqf(group_sum<4>(ss) * (1.0f / kCap) + a.eps);
        float hp[kH];
#pragma unroll
        for (int h = 0; h < kH; ++h) {
          float t = 0.0f;
#pragma unroll
          for (int i = 0; i < 4; ++i) t = fmaf(wb[h][i], dv[i], t);
          hp[h] = group_sum<4>(t);
        }
        const float mine = cq == 0 ? hp[0] : cq == 1 ? hp[1] : cq == 2 ? hp[2] : hp[3];
        lb[pos][cq] = pos < count ? rstd * mine : -INFINITY;
      }
    }
    wave_lds_sync();

    // 3. batches of K/V rows; the requests for the batch after the last one
    //    read the extra padding of the list (no data), which keeps the number
    //    of loads in flight the same on every path
    int prev[kUnroll];  // addresses of the V loads in flight
    offsets(0, prev);
    issue_v(0, prev);
    for (int b0 = 0; b0 < count_pad; b0 += kBatch) {
      int off[kUnroll];
      offsets(b0 + kBatch, off);
      // the loads in flight read their addresses from prev: keep those
      // registers until the next addresses are in others
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) asm volatile("" ::"v"(prev[u]));
      float lg[kUnroll];
      logits(0, b0, lg);
      issue_k(0, off);
      weigh(0, lg);
      issue_v(0, off);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) prev[u] = off[u];
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
  if (a.c_atom == kHD) {
    int64_t wgs = ((rows + 63) / 64 + 3) / 4;
    if (wgs > 128) wgs = 128;  // 4 x 128 workgroups, two per CU (64 KB of LDS each); waves loop over atom groups
    hipLaunchKernelGGL(atom_proj128_kernel, dim3((unsigned)wgs, 4), dim3(256), 0, st, a);
    return hipGetLastError();
  }
  const int64_t groups = ((rows + 15) / 16 + kProjTiles - 1) / kProjTiles;
  hipLaunchKernelGGL(atom_proj_kernel, dim3((unsigned)groups, kH, 4), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sparse_attn(const SparseAttnArgs& a, bool bf16, hipStream_t st) {
  if (a.k_slots <= 128) return bf16 ? launch_attn<true, 128>(a, st) : launch_attn<false, 128>(a, st);
  return bf16 ? launch_attn<true, 256>(a, st) : launch_attn<false, 256>(a, st);
}

}  // namespace dcp
