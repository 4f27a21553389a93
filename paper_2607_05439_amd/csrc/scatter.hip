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
// Two paths add the same integers, so they give the same bits:
//
// Atoms ordered by token (the model's layout), no atomics and no clearing:
//   scatter_plan_kernel   one wave per tile of 64 atom positions: checks the
//                         tile's indices for a decrease (one flag per
//                         workgroup, written whatever its value, so nothing
//                         needs clearing first) and, where there is none,
//                         writes each token's first and one-past-last atom to
//                         a plan: the lane at a token boundary writes the end
//                         of the run before it and the start of the run after
//                         it (both at the boundary for a token without atoms),
//                         so no lane scans a long token's atoms
//   scatter_sum_kernel    if no flag is set: consecutive tokens go to groups of
//                         lanes, a group covering a feature row in 16-byte
//                         chunks; each group loads all its token's rows at
//                         once, sums them and writes the mean. If a flag is
//                         set, the kernel clears the sums and counts of the
//                         general path instead.
// Any order (run when a flag is set, or when rows are not 16-byte aligned):
//   scatter_accum_kernel  one wave per run of 64 consecutive atoms, lanes over
//                         channels: runs of atoms with the same token are
//                         summed in registers, and each run adds its sum with
//                         one 64-bit atomic per channel and one count atomic
//   scatter_final_kernel  out = sum * 2^-32 / count (0 for a token without atoms)
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kRun = 64;  // atoms per wave of the general path
constexpr double kFix = 4294967296.0;  // 2^32
constexpr int kSlots = 4;              // atom rows per lane group in flight (few: more waves fit)
constexpr uint32_t kNt = 2;            // cache-policy bit of a buffer load: non-temporal
constexpr int kGatedBlocks = 1024;     // grid cap of the general path's accumulation and division

// 1.5 * 2^52 and its bits: for |y| < 2^51, y + 1.5 * 2^52 rounded to fp64 is
// round-half-even(y) + 1.5 * 2^52, whose bits are those of the constant plus
// the integer.
constexpr double kMagic = 6755399441055744.0;
constexpr uint64_t kMagicBits = 0x4338000000000000ull;

// s += round-half-even(clamp(x, -2^30, 2^30) * 2^32) + kMagicBits (mod 2^64).
// The integer part h of the clamped x contributes h * 2^32 exactly; the
// fraction x - h (exact in fp32, |.| < 1) is scaled by 2^32 and rounded to an
// integer with the constant above, in one fma. Rounding the whole equals the
// integer part plus the rounded fraction because h * 2^32 is an even integer.
// The caller subtracts kMagicBits once per addition.
__device__ __forceinline__ void add_fixed(uint64_t& s, float x) {
  const float xc = fminf(fmaxf(x, -1073741824.0f), 1073741824.0f);
  const float h = truncf(xc);
  const double t = fma((double)(xc - h), kFix, kMagic);
  s += (uint64_t)__double_as_longlong(t) + ((uint64_t)(uint32_t)(int32_t)h << 32);
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef int64_t i64x2 __attribute__((ext_vector_type(2)));

// round-half-even(x * 2^32) + kMagicBits for |x| < 2^19: x * 2^32 is exact in
// fp64 and below 2^51, so one fma rounds it to an integer
__device__ __forceinline__ uint64_t fixed_small(float x) {
  return (uint64_t)__double_as_longlong(fma((double)x, kFix, kMagic));
}

// 2^32 in an SGPR pair the compiler cannot fold into a literal operand
__device__ __forceinline__ double opaque_two32() {
  uint32_t hi;
  asm volatile("s_mov_b32 %0, 0x41f00000" : "=s"(hi));
  return __builtin_bit_cast(double, (uint64_t)hi << 32);
}

// 1/k in fp64, correctly rounded (a table for the usual counts)
struct InvCount {
  double v[257];
};
constexpr InvCount make_inv_count() {
  InvCount t{};
  for (int k = 1; k < 257; ++k) t.v[k] = 1.0 / k;
  return t;
}
__constant__ const InvCount kInvCount = make_inv_count();

// the mean of k features whose fixed-point sum is sum: sum * 2^-32 * (1/k) in
// fp64, rounded to fp32 (both paths use exactly this, so they agree bit for bit)
__device__ __forceinline__ double mean_scale(uint32_t k) {
  return (k <= 256 ? kInvCount.v[k] : 1.0 / (double)k) * (1.0 / kFix);
}
__device__ __forceinline__ float mean_of(int64_t sum, uint32_t k) {
  return k ? (float)((double)sum * mean_scale(k)) : 0.0f;
}


// feature c of a chunk of a feature row: bf16 pairs (channel 2j in the low half
// of dword j) or fp32
template <bool kBf16, typename T>
__device__ __forceinline__ float elem(const T& x, int c) {
  if constexpr (kBf16)
    return __uint_as_float((c & 1) ? (x[c >> 1] & 0xFFFF0000u) : (x[c >> 1] << 16));
  else
    return __uint_as_float(x[c]);
}

// out[t, EPL * q .. EPL * q + EPL) = o (zeros when o is NULL), fp32 or bf16
template <int EPL>
__device__ __forceinline__ void store_mean(const ScatterArgs& a, int64_t t, int q, const float* o) {
  float z[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) z[e] = o ? o[e] : 0.0f;
  const int64_t i = t * a.c + (int64_t)q * EPL;
  if (a.out_bf16) {
    uint32_t w[(EPL + 1) / 2];
#pragma unroll
    for (int e = 0; e < EPL; e += 2) {
      const uint32_t lo = __builtin_bit_cast(uint16_t, (__bf16)z[e]);
      const uint32_t hi = e + 1 < EPL ? (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)z[e + 1]) : 0u;
      w[e / 2] = lo | (hi << 16);
    }
    __bf16* dst = static_cast<__bf16*>(a.out) + i;
    if constexpr (EPL == 1)
      *reinterpret_cast<uint16_t*>(dst) = (uint16_t)w[0];
    else if constexpr (EPL == 2)
      *reinterpret_cast<uint32_t*>(dst) = w[0];
    else if constexpr (EPL == 4)
      *reinterpret_cast<u32x2*>(dst) = u32x2{w[0], w[1]};
    else
      *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
  } else {
    float* dst = static_cast<float*>(a.out) + i;
    if constexpr (EPL == 1)
      *dst = z[0];
    else if constexpr (EPL == 2)
      *reinterpret_cast<float2*>(dst) = make_float2(z[0], z[1]);
    else
#pragma unroll
      for (int e = 0; e < EPL; e += 4) *reinterpret_cast<f32x4*>(dst + e) = f32x4{z[e], z[e + 1], z[e + 2], z[e + 3]};
  }
}

// any flag of the order check set (wave-uniform)
__device__ __forceinline__ bool out_of_order(const int32_t* flags, int n_flags) {
  int32_t any = 0;
  for (int f = (int)(threadIdx.x & 63); f < n_flags; f += 64) any |= flags[f];
  return __ballot(any != 0) != 0;
}

// plan[2t] = first atom of token t, plan[2t + 1] = one past its last, for
// indices ordered by token. Each run boundary writes the end of the run before
// it and the start of the run after it, so every entry is written once, by the
// tile that holds the boundary; a token without atoms gets both at the
// position after the gap, so first atoms never decrease along the tokens.
__global__ void __launch_bounds__(1024) scatter_plan_kernel(ScatterArgs a) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t n = a.n_atoms, tiles = n / 64 + 1;  // positions 0..n (n: the end of the last token)
  int bad = 0;
  for (int64_t tile = (int64_t)blockIdx.x * 16 + wave; tile < tiles; tile += (int64_t)gridDim.x * 16) {
    const int64_t p = tile * 64 + lane;
    const int32_t cur = p < n ? a.tok_idx[p] : 0;
    const int32_t prv = (p >= 1 && p <= n) ? a.tok_idx[p - 1] : -1;
    if (__ballot(p >= 1 && p < n && prv > cur)) {  // out of order: no plan (it is never read)
      bad = 1;
      continue;
    }
    // a boundary at p: p = 0, p = n, or a token change between p - 1 and p
    int64_t g0 = 0, g1 = 0;
    if (p <= n && (p == 0 || p == n || prv != cur)) {
      if (p > 0 && prv >= 0 && (int64_t)prv < a.n_tokens) a.plan[2 * (int64_t)prv + 1] = p;
      if (p < n && cur >= 0 && (int64_t)cur < a.n_tokens) a.plan[2 * (int64_t)cur] = p;
      // the tokens strictly between the two runs' tokens have no atoms
      g0 = (p == 0 ? -1 : max((int64_t)prv, (int64_t)-1)) + 1;
      g1 = p == n ? a.n_tokens : min((int64_t)cur, a.n_tokens);
    }
    // gaps are filled by the whole wave, one at a time
    for (uint64_t m = __ballot(g1 > g0); m; m &= m - 1) {
      const int l = __builtin_ctzll(m);
      const int64_t t0 = __shfl(g0, l), t1 = __shfl(g1, l), at = tile * 64 + l;
      for (int64_t t = t0 + lane; t < t1; t += 64) {
        a.plan[2 * t] = at;
        a.plan[2 * t + 1] = at;
      }
    }
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) a.flags[blockIdx.x] = bad;
}

__device__ void clear_general(const ScatterArgs& a) {
  const int64_t nth = (int64_t)gridDim.x * gridDim.y * 256;
  const int64_t id = ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * 256 + threadIdx.x;
  const int64_t n = a.n_tokens * a.c;
  for (int64_t i = id; i < n; i += nth) a.acc[i] = 0;
  for (int64_t i = id; i < a.n_tokens; i += nth) a.cnt[i] = 0;
}

// Waves take 64 / G consecutive tokens, one per group of G lanes; a group
// covers one feature row in 16-byte chunks (blockIdx.y selects a slice of G
// chunks when a row has more than 64). The tokens' rows are
// consecutive, so one buffer resource from the first token's first row serves
// the wave.
template <bool kBf16, int G>
__global__ void __launch_bounds__(256) scatter_sum_kernel(ScatterArgs a) {
  constexpr int R = 64 / G;          // groups (tokens) per wave
  constexpr int CH = kBf16 ? 8 : 4;  // channels per 16-byte chunk
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = lane / G;
  const int64_t t0 = ((int64_t)blockIdx.x * 4 + wave) * R, t = t0 + grp;
  const bool act = t < a.n_tokens;
  // the plan is loaded before the order flags are known
  int64_t b = 0, cnt = 0;
  if (act) {
    const i64x2 e = *reinterpret_cast<const i64x2*>(a.plan + 2 * t);
    b = e[0];
    cnt = e[1] - e[0];
  }
  if (out_of_order(a.flags, a.n_flags)) {
    clear_general(a);
    return;
  }
  if (t0 >= a.n_tokens) return;
  const int q = (int)blockIdx.y * G + lane % G;  // this lane's chunk of a row
  const int nch = a.c * (kBf16 ? 2 : 4) / 16;
  const bool qok = q < nch;
  const uint32_t row = (uint32_t)a.c * (kBf16 ? 2u : 4u);

  // the rows of the wave's tokens: b_lo .. b_hi
  int kmax = (int)(cnt < INT32_MAX ? cnt : INT32_MAX);
#pragma unroll
  for (int s = G; s < 64; s <<= 1) kmax = max(kmax, __shfl_xor(kmax, s));
  const int last = (int)min((int64_t)R - 1, a.n_tokens - 1 - t0) * G;
  const int64_t b_lo = ((int64_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const int64_t b_hi = ((int64_t)__builtin_amdgcn_readlane((uint32_t)((b + cnt) >> 32), last) << 32) |
                       (uint32_t)__builtin_amdgcn_readlane((uint32_t)(b + cnt), last);
  const double two32 = opaque_two32();  // in SGPRs: lets the fma take its 3-operand form
  const double magic = kMagic;
  uint64_t acc[CH];
#pragma unroll
  for (int e = 0; e < CH; ++e) acc[e] = 0;
  if ((b_hi - b_lo) * (int64_t)row <= (1ll << 30)) {
    const uint32_t rel = (uint32_t)(b - b_lo);
    for (int s0 = 0; s0 < kmax; s0 += kSlots) {
      // rows from b_lo + s0 on; a slot past its token's rows, or a lane past
      // the row's chunks, reads beyond the record: zeros, no traffic
      const int64_t rb = b_lo + s0, rem = (b_hi - rb) * (int64_t)row;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char*>(static_cast<const char*>(a.a)) + rb * (int64_t)row, 0, (int)(rem > 0 ? rem : 0),
          kRawBufferFlags);
      u32x4 v[kSlots];
#pragma unroll
      for (int u = 0; u < kSlots; ++u) {
        const int off = (qok && s0 + u < cnt) ? (int)((rel + u) * row + 16u * (uint32_t)q) : kOutOfRange;
        v[u] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kNt);
      }
      // features below 2^19 in magnitude (all of them, in practice) take the
      // one-fma conversion: x * 2^32 is exact in fp64 and below 2^51
      u16x2 mx2 = {0, 0};
      uint32_t mx = 0;
#pragma unroll
      for (int u = 0; u < kSlots; ++u)
        if (s0 + u < kmax)  // wave-uniform: rows past every group's count are zeros
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            if constexpr (kBf16)
              mx2 = __builtin_elementwise_max(mx2, __builtin_bit_cast(u16x2, v[u][w] & 0x7FFF7FFFu));
            else
              mx = max(mx, v[u][w] & 0x7FFFFFFFu);
          }
      const bool big = kBf16 ? (mx2[0] >= 0x4900u || mx2[1] >= 0x4900u)  // bf16 bits of 2^19
                             : mx >= 0x49000000u;                       // fp32 bits of 2^19
      if (__ballot(big) == 0) {
#pragma unroll
        for (int u = 0; u < kSlots; ++u)
          if (s0 + u < kmax)  // wave-uniform: skips rows no group of the wave has
#pragma unroll
            for (int e = 0; e < CH; ++e)
              acc[e] += (uint64_t)__double_as_longlong(fma((double)elem<kBf16>(v[u], e), two32, magic));
      } else {
#pragma unroll
        for (int u = 0; u < kSlots; ++u)
          if (s0 + u < kmax)
#pragma unroll
            for (int e = 0; e < CH; ++e) add_fixed(acc[e], elem<kBf16>(v[u], e));
      }
    }
  } else {
    // rows spread over more than 2^30 bytes (tokens of millions of atoms): one
    // row at a time, 64-bit addresses
    for (int s0 = 0; s0 < kmax; ++s0) {
      u32x4 x = {0, 0, 0, 0};
      if (qok && s0 < cnt)
        x = *reinterpret_cast<const u32x4*>(static_cast<const char*>(a.a) + (b + s0) * (int64_t)row + 16 * q);
#pragma unroll
      for (int e = 0; e < CH; ++e) add_fixed(acc[e], elem<kBf16>(x, e));
    }
  }
  if (act && qok) {
    // every lane added kmax rows (zeros past its own count); a token without
    // atoms gets zeros
    const uint64_t bias = (uint64_t)kmax * kMagicBits;
    float o[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) o[e] = mean_of((int64_t)(acc[e] - bias), (uint32_t)cnt);
    store_mean<CH>(a, t, q, o);
  }
}

__global__ void __launch_bounds__(256) scatter_zero_kernel(ScatterArgs a) { clear_general(a); }

// one run of kRun consecutive atoms [i0, i1)
template <bool kBf16, int CPL>
__device__ void accum_run(const ScatterArgs& a, int64_t i0, int64_t i1) {
  const int lane = threadIdx.x & 63;
  uint64_t sum[CPL];
#pragma unroll
  for (int j = 0; j < CPL; ++j) sum[j] = 0;
  int32_t cur = -1;
  uint32_t seg = 0;
  auto flush = [&]() {
    if (seg != 0 && cur >= 0 && (int64_t)cur < a.n_tokens) {
      const uint64_t bias = (uint64_t)seg * kMagicBits;
#pragma unroll
      for (int j = 0; j < CPL; ++j) {
        const int ch = lane + 64 * j;
        if (ch < a.c)
          atomicAdd(reinterpret_cast<unsigned long long*>(a.acc) + (int64_t)cur * a.c + ch,
                    (unsigned long long)(sum[j] - bias));
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
      for (int j = 0; j < CPL; ++j) add_fixed(sum[j], xv[u][j]);
      ++seg;
    }
  }
  flush();
}

// grid-stride over the runs, so a small grid serves (its launch is short when
// the ordered path already wrote the output)
template <bool kBf16, int CPL>
__global__ void __launch_bounds__(256) scatter_accum_kernel(ScatterArgs a) {
  if (a.flags && !out_of_order(a.flags, a.n_flags)) return;  // the ordered path wrote the output
  const int64_t runs = (a.n_atoms + kRun - 1) / kRun;
  for (int64_t run = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); run < runs;
       run += (int64_t)gridDim.x * 4)
    accum_run<kBf16, CPL>(a, run * kRun, min((run + 1) * kRun, a.n_atoms));
}

__global__ void __launch_bounds__(256) scatter_final_kernel(ScatterArgs a) {
  if (a.flags && !out_of_order(a.flags, a.n_flags)) return;
  const int64_t n = a.n_tokens * a.c;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / a.c;
    const float v = mean_of(a.acc[i], a.cnt[t]);
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
  int64_t blocks = (a.n_atoms + 4 * kRun - 1) / (4 * kRun);
  if (blocks > kGatedBlocks) blocks = kGatedBlocks;
  const dim3 grid((unsigned)blocks), block(256);
  if (a.c <= 64)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 1>), grid, block, 0, st, a);
  else if (a.c <= 128)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 2>), grid, block, 0, st, a);
  else if (a.c <= 256)
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 4>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((scatter_accum_kernel<kBf16, 8>), grid, block, 0, st, a);
}

template <bool kBf16>
void launch_sum(const ScatterArgs& a, hipStream_t st) {
  const int nch = a.c * (kBf16 ? 2 : 4) / 16;
  int g = 1;
  while (g < nch && g < 64) g *= 2;
  const int64_t token_blocks = (a.n_tokens + 4 * (64 / g) - 1) / (4 * (64 / g));
  // in the out-of-order case the same grid clears the general path's sums
  int64_t clear_blocks = (a.n_tokens * a.c + 2047) / 2048;
  if (clear_blocks > 1024) clear_blocks = 1024;
  const dim3 grid((unsigned)(token_blocks > clear_blocks ? token_blocks : clear_blocks), (unsigned)((nch + g - 1) / g)),
      block(256);
  switch (g) {
    case 1: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 1>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 2>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 4>), grid, block, 0, st, a); break;
    case 8: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 8>), grid, block, 0, st, a); break;
    case 16: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 16>), grid, block, 0, st, a); break;
    case 32: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 32>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((scatter_sum_kernel<kBf16, 64>), grid, block, 0, st, a); break;
  }
}

}  // namespace

int scatter_order_flags(int64_t n_atoms) {
  const int64_t f = (n_atoms / 64 + 1 + 15) / 16;  // plan workgroups: 16 tiles of 64 positions each
  return (int)(f < 1 ? 1 : (f > kScatterFlags ? kScatterFlags : f));
}

hipError_t launch_scatter_mean(const ScatterArgs& in, hipStream_t st) {
  ScatterArgs a = in;
  const int eb = a.a_bf16 ? 2 : 4, ob = a.out_bf16 ? 2 : 4;
  const int chunk = 16 / eb;  // channels per 16-byte chunk of a feature row
  // the ordered path loads 16-byte chunks of feature rows and stores chunk * ob
  // bytes (at most 16 per instruction)
  const size_t store_align = chunk * ob < 16 ? (size_t)(chunk * ob) : 16;
  const bool ordered = a.n_atoms > 0 && a.flags && a.c % chunk == 0 &&
                       reinterpret_cast<uintptr_t>(a.a) % 16 == 0 && reinterpret_cast<uintptr_t>(a.out) % store_align == 0;
  hipError_t e;
  if (ordered) {
    a.n_flags = scatter_order_flags(a.n_atoms);
    hipLaunchKernelGGL(scatter_plan_kernel, dim3((unsigned)a.n_flags), dim3(1024), 0, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.a_bf16)
      launch_sum<true>(a, st);
    else
      launch_sum<false>(a, st);
  } else {
    a.flags = nullptr;
    a.n_flags = 0;
    hipLaunchKernelGGL(scatter_zero_kernel, dim3(grid_of(a.n_tokens * a.c)), dim3(256), 0, st, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.n_atoms > 0) {
    if (a.a_bf16)
      launch_accum<true>(a, st);
    else
      launch_accum<false>(a, st);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // grid-stride, with a grid small enough that the launch is short when the
  // ordered path already wrote the output
  const unsigned fg = grid_of(a.n_tokens * a.c);
  hipLaunchKernelGGL(scatter_final_kernel, dim3(fg < (unsigned)kGatedBlocks ? fg : (unsigned)kGatedBlocks), dim3(256), 0,
                     st, a);
  return hipGetLastError();
}

}  // namespace dcp
