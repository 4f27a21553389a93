// k nearest neighbours of atoms and the top-k merge on gfx950 (CDNA4).
//
// Appendix "Distributed kNN for sparse atom attention": every query atom keeps
// the k atoms closest to it; the distances are taken block by block (never the
// whole [L, L] matrix) and the running top-k of each query is merged with each
// block's candidates (the ring top-k combine). Order: squared distance in fp32,
// ((dx*dx) + (dy*dy)) + (dz*dz) with every operation rounded, ties by the
// smaller candidate index. The 64-bit key (d2 bits << 32) | index orders
// exactly that way (d2 >= 0).
//
// knn_prep_kernel: one pass over the candidates writes each as a 16-byte
// entry (x, y, z, then |c|^2, or the group in the group modes) and, for every
// step of 128 consecutive candidates, its bounding box (low and high corner),
// into the caller's workspace.
// knn_kernel: a workgroup of 8 independent waves serves 32 consecutive query
// rows, 4 per wave (their coordinates and thresholds are wave-uniform
// scalars). A wave visits the candidates in groups of 16 steps (2048
// candidates), starting at the group that holds the queries themselves when
// they are candidates (their sequence neighbours are close in space, which
// makes the thresholds tight early; the result does not depend on the order).
// Per group it tests the 16 boxes against its 4 queries (the next group's
// boxes are loaded meanwhile) and skips a step whose box distance (computed in
// the definition's rounded operations, which bound every member's distance
// from below) exceeds the current k-th distance of all 4 queries: an exact
// exclusion, not a heuristic. Only the candidates of the remaining steps are
// read, straight from the workspace (L2-resident): a lane takes two per step
// and tests them against the 4 queries with a cheap conservative bound (|c|^2
// - 2 c.q by three multiply-adds against a per-query limit derived from the
// current k-th distance with a proven rounding margin): no candidate that
// could enter is rejected. Only where some lane passes does the step compute
// the distances of the definition; the exact 64-bit key test then picks the
// candidates that enter the query's 64-entry LDS buffer. The sorted top-k
// lives in registers (entry 64s + lane in slot s); a full buffer is sorted
// (bitonic network across lanes) and merged slot by slot: the lane-wise
// minimum of a sorted slot and the reversed sorted carry is a bitonic sequence
// that holds the 64 smallest of the two, the maximum holds the other 64, and
// one bitonic merge pass sorts each.
// topk_merge_kernel: one wave per row, a rank merge of two sorted lists.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kKnnWaves = 8;
constexpr int kKnnQ = 4;                          // query rows per wave
constexpr int kKnnRows = kKnnWaves * kKnnQ;       // query rows per workgroup
constexpr uint64_t kNoKey = ~0ULL;

// Value of lane (lane ^ M).
template <int M>
__device__ __forceinline__ uint32_t xor_lane(uint32_t x) {
  if constexpr (M == 1) return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, true);
  if constexpr (M == 2) return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, true);
  if constexpr (M == 4) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x101F);
  if constexpr (M == 8) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x201F);
  if constexpr (M == 16) return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x401F);
  if constexpr (M >= 32) return (uint32_t)__shfl_xor((int)x, M);
}

template <int M>
__device__ __forceinline__ uint64_t xor_lane64(uint64_t v) {
  const uint32_t lo = xor_lane<M>((uint32_t)v), hi = xor_lane<M>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// One compare-exchange stage of a bitonic network over the wave: lanes whose
// bit M is clear keep the minimum of the pair when `up`, else the maximum.
template <int SIZE, int M>
__device__ __forceinline__ uint64_t bitonic_stage(uint64_t v, int lane) {
  const uint64_t p = xor_lane64<M>(v);
  const bool up = SIZE >= 64 || (lane & SIZE) == 0;
  const bool keep_min = ((lane & M) == 0) == up;
  // the partner's key where it is the one to keep: one comparison per stage
  // (equal keys are the same either way)
  return ((p < v) == keep_min) ? p : v;
}

// Merge pass of size SIZE: sorts every bitonic run of SIZE lanes (ascending
// runs where bit SIZE of the lane is clear; the whole wave ascending at 64).
template <int SIZE>
__device__ __forceinline__ uint64_t bitonic_pass(uint64_t v, int lane) {
  if constexpr (SIZE > 32) v = bitonic_stage<SIZE, 32>(v, lane);
  if constexpr (SIZE > 16) v = bitonic_stage<SIZE, 16>(v, lane);
  if constexpr (SIZE > 8) v = bitonic_stage<SIZE, 8>(v, lane);
  if constexpr (SIZE > 4) v = bitonic_stage<SIZE, 4>(v, lane);
  if constexpr (SIZE > 2) v = bitonic_stage<SIZE, 2>(v, lane);
  return bitonic_stage<SIZE, 1>(v, lane);
}

// Ascending sort of one key per lane across the wave.
__device__ __forceinline__ uint64_t wave_sort(uint64_t v, int lane) {
  v = bitonic_pass<2>(v, lane);
  v = bitonic_pass<4>(v, lane);
  v = bitonic_pass<8>(v, lane);
  v = bitonic_pass<16>(v, lane);
  v = bitonic_pass<32>(v, lane);
  return bitonic_pass<64>(v, lane);
}

__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// a wave-uniform value, held in a scalar register
__device__ __forceinline__ float uniform(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

// State of one query row: its sorted top-k (KS slots of 64 keys), the number
// of valid entries, the k-th key, and the LDS buffer of pending keys.
template <int KS>
struct QueryTopk {
  uint64_t top[KS];
  uint64_t tau;  // keys below tau may enter (kNoKey until k entries exist)
  int count, bcount;
  uint64_t* buf;
  float x, y, z;
  int32_t g;
  float mx, my, mz;  // -2 x, -2 y, -2 z (exact)
  float qq, qn;      // |q|^2 and |q|
  float lim;         // prefilter bound on |c|^2 - 2 c.q for candidates that may still enter

  // The prefilter computes e = |c|^2 - 2 c.q with three multiply-adds; the
  // exact distance is |c - q|^2 = e + |q|^2 up to rounding. If the rounded
  // distance of the definition is at most T (the k-th key's distance), then
  // the true distance D is at most T (1 + 6u) (u = 2^-24), so |c| <= |q| +
  // 1.001 sqrt(T) =: rho, and e is within 6u (|c|^2 + |c||q|) <= 12u rho^2 of
  // its true value D - |q|^2. So every candidate that may enter has
  // e <= T - |q|^2 + 6uT + 12u rho^2; the bound below adds 32u (T + rho^2),
  // which also covers the rounding of |q|^2 (3u rho^2) and of the bound
  // itself (about 2u (T + rho^2)). With no
  // finite k-th distance yet the bound is +inf or NaN, and the test
  // "not above the bound" lets every candidate through.
  __device__ __forceinline__ void set_limit() {
    const float T = __uint_as_float((uint32_t)(tau >> 32));
    const float rho = qn + 1.001f * __builtin_sqrtf(T);
    lim = uniform((T - qq) + 0x1p-19f * (T + rho * rho));
  }

  __device__ __forceinline__ void init(uint64_t* b) {
#pragma unroll
    for (int s = 0; s < KS; ++s) top[s] = kNoKey;
    tau = kNoKey;
    count = 0;
    bcount = 0;
    buf = b;
  }

  // merge the bcount pending keys into the sorted top-k
  __device__ __forceinline__ void flush(int lane, int k) {
    uint64_t carry = lane < bcount ? buf[lane] : kNoKey;
    carry = wave_sort(carry, lane);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint64_t r = xor_lane64<63>(carry);  // reversed: descending
      const uint64_t lo = r < top[s] ? r : top[s];
      const uint64_t hi = r < top[s] ? top[s] : r;
      top[s] = bitonic_pass<64>(lo, lane);
      if (s + 1 < KS) carry = bitonic_pass<64>(hi, lane);
    }
    count = min(k, count + bcount);
    bcount = 0;
    uint64_t last = top[0];  // slot of entry k - 1, chosen without dynamic register indexing
#pragma unroll
    for (int s = 1; s < KS; ++s)
      if (s == ((k - 1) >> 6)) last = top[s];
    tau = count == k ? readlane64(last, (k - 1) & 63) : kNoKey;
    set_limit();
    wave_lds_sync();  // the buffer has been read before it is refilled
  }

  // the exact test and the append of one 64-candidate step
  template <int MODE>
  __device__ __forceinline__ void offer(uint32_t d2bits, uint32_t index, bool valid, int32_t g_c, int lane,
                                        int k) {
    const uint64_t key = ((uint64_t)d2bits << 32) | index;
    bool take = valid && key < tau;
    if constexpr (MODE == 1) take = take && g_c == g;
    if constexpr (MODE == 2) take = take && g_c != g;
    const uint64_t mask = __ballot(take);
    if (mask == 0) return;
    const int n_new = __popcll(mask);
    if (bcount + n_new > 64) flush(lane, k);
    const int pos = bcount + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
    if (take) buf[pos] = key;
    wave_lds_sync();
    bcount += n_new;
  }
};

__device__ __forceinline__ float norm2(float4 c) { return fmaf(c.x, c.x, fmaf(c.y, c.y, c.z * c.z)); }

__device__ __forceinline__ float dist2(float qx, float qy, float qz, float4 c) {
  // the distance is part of the definition: each operation rounded, in this
  // order, never fused into multiply-adds
#pragma clang fp contract(off)
  const float dx = qx - c.x, dy = qy - c.y, dz = qz - c.z;
  return (dx * dx + dy * dy) + dz * dz;
}

constexpr int kStep = 128;   // candidates per bounding box
constexpr int kGroup = 2048;  // candidates per group of 16 steps (one skip test per lane)
constexpr int kSeedWords = 64;  // steps whose seed bit a wave keeps: 64 x 64

// one wave per step of 128 candidates, two per lane
template <int MODE>
__global__ void __launch_bounds__(256) knn_prep_kernel(KnnArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t st = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (st * kStep >= a.n_c) return;
  float4* c4 = static_cast<float4*>(a.cand);
  float4* box = static_cast<float4*>(a.box);
  float lx = __builtin_inff(), ly = lx, lz = lx, hx = -lx, hy = -lx, hz = -lx;
  for (int h = 0; h < 2; ++h) {
    const int64_t i = st * kStep + 64 * h + lane;
    if (i < a.n_c) {
      const float* p = a.x_c + 3 * i;
      float4 v = make_float4(p[0], p[1], p[2], 0.f);
      v.w = MODE ? __int_as_float(a.group_c[i]) : norm2(v);
      c4[i] = v;
      lx = fminf(lx, v.x); ly = fminf(ly, v.y); lz = fminf(lz, v.z);
      hx = fmaxf(hx, v.x); hy = fmaxf(hy, v.y); hz = fmaxf(hz, v.z);
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    lx = fminf(lx, __shfl_xor(lx, m));
    ly = fminf(ly, __shfl_xor(ly, m));
    lz = fminf(lz, __shfl_xor(lz, m));
    hx = fmaxf(hx, __shfl_xor(hx, m));
    hy = fmaxf(hy, __shfl_xor(hy, m));
    hz = fmaxf(hz, __shfl_xor(hz, m));
  }
  if (lane == 0) {
    box[2 * st] = make_float4(lx, ly, lz, 0.f);
    box[2 * st + 1] = make_float4(hx, hy, hz, 0.f);
  }
}

template <int KS, int MODE>
__global__ void __launch_bounds__(64 * kKnnWaves) __attribute__((amdgpu_waves_per_eu(KS == 2 ? 6 : 1))) knn_kernel(KnnArgs a) {
  __shared__ uint64_t s_buf[kKnnWaves][kKnnQ][64];
  __shared__ uint64_t s_seed[kKnnWaves][kSeedWords];
  const float4* c4 = static_cast<const float4*>(a.cand);
  const float4* box = static_cast<const float4*>(a.box);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r0 = (int64_t)blockIdx.x * kKnnRows;
  const int64_t rw = r0 + wave * kKnnQ;
  const int k = a.k;
  QueryTopk<KS> q[kKnnQ];
#pragma unroll
  for (int j = 0; j < kKnnQ; ++j) {
    const int64_t rr = min(rw + j, a.n_q - 1);  // rows past n_q repeat the last one and are not written
    q[j].init(s_buf[wave][j]);
    q[j].x = a.x_q[3 * rr];
    q[j].y = a.x_q[3 * rr + 1];
    q[j].z = a.x_q[3 * rr + 2];
    q[j].g = MODE ? a.group_q[rr] : 0;
    q[j].mx = uniform(-2.0f * q[j].x);
    q[j].my = uniform(-2.0f * q[j].y);
    q[j].mz = uniform(-2.0f * q[j].z);
    q[j].qq = uniform(fmaf(q[j].x, q[j].x, fmaf(q[j].y, q[j].y, q[j].z * q[j].z)));
    q[j].qn = uniform(__builtin_sqrtf(q[j].qq));
    q[j].set_limit();
  }
  const int64_t n_steps = (a.n_c + kStep - 1) / kStep;
  const int64_t n_groups = (a.n_c + kGroup - 1) / kGroup;
  int64_t t0 = 0;
  if (a.q_self0 >= 0 && n_groups > 0) t0 = ((a.q_self0 + r0) / kGroup) % n_groups;
  const int jq = lane >> 4;
  // lane l holds the box of step l % 16 of a group (the group's last step
  // where it has fewer: those bits are never used)
  auto box_of = [&](int64_t grp, float4& lo, float4& hi) {
    const int64_t st = min(grp * (kGroup / kStep) + (lane & 15), n_steps - 1);
    lo = box[2 * st];
    hi = box[2 * st + 1];
  };
  // One step: 128 candidates from c0s, two per lane (entries past the n_s
  // candidates take no part), the prefilter against the 4 queries, and the
  // exact test and append where some lane passes it.
  auto visit = [&](int64_t c0s, int n_s) {
    const bool va = lane < n_s, vb = 64 + lane < n_s;
    const float4 ca = c4[c0s + (va ? lane : 0)], cb = c4[c0s + (vb ? 64 + lane : 0)];
    const float cca = MODE ? norm2(ca) : ca.w, ccb = MODE ? norm2(cb) : cb.w;
    uint64_t ma[kKnnQ], mb[kKnnQ], any = 0;
#pragma unroll
    for (int j = 0; j < kKnnQ; ++j) {
      const float ea = fmaf(ca.x, q[j].mx, fmaf(ca.y, q[j].my, fmaf(ca.z, q[j].mz, cca)));
      const float eb = fmaf(cb.x, q[j].mx, fmaf(cb.y, q[j].my, fmaf(cb.z, q[j].mz, ccb)));
      ma[j] = __ballot(va && !(ea > q[j].lim));
      mb[j] = __ballot(vb && !(eb > q[j].lim));
      any |= ma[j] | mb[j];
    }
    if (any == 0) return;
    // the exact distances and keys decide; a flush lowers tau after the
    // prefilter, so the masks stay a superset
    const uint32_t index0 = (uint32_t)(a.c_index0 + c0s);
#pragma unroll
    for (int j = 0; j < kKnnQ; ++j) {
      if (ma[j])
        q[j].template offer<MODE>(__float_as_uint(dist2(q[j].x, q[j].y, q[j].z, ca)), index0 + lane, va,
                                  __float_as_int(ca.w), lane, k);
      if (mb[j])
        q[j].template offer<MODE>(__float_as_uint(dist2(q[j].x, q[j].y, q[j].z, cb)), index0 + 64 + lane, vb,
                                  __float_as_int(cb.w), lane, k);
    }
  };

  // Seeds: the steps (among the first 64 x 64) whose box holds one of the
  // wave's queries. They are visited first, the one that holds the queries
  // themselves (as candidates) before the others, so that the k-th distances
  // are small before the bulk of the candidates is tested; the full pass below
  // then leaves them out. Only the visiting order changes, never the result.
  const int64_t seed_steps = min(n_steps, (int64_t)kSeedWords * 64);
  for (int64_t w0 = 0; w0 < seed_steps; w0 += 64) {
    const int64_t st = w0 + lane;
    bool in = false;
    if (st < seed_steps) {
      const float4 lo = box[2 * st], hi = box[2 * st + 1];
#pragma unroll
      for (int j = 0; j < kKnnQ; ++j)
        in = in || (q[j].x >= lo.x && q[j].x <= hi.x && q[j].y >= lo.y && q[j].y <= hi.y && q[j].z >= lo.z &&
                    q[j].z <= hi.z);
    }
    const uint64_t m = __ballot(in);
    if (lane == 0) s_seed[wave][w0 >> 6] = m;
  }
  wave_lds_sync();
  {
    int64_t own = -1;
    if (a.q_self0 >= 0) {
      own = (a.q_self0 + rw) / kStep;
      if (own < seed_steps && ((s_seed[wave][own >> 6] >> (own & 63)) & 1u))
        visit(own * kStep, (int)min((int64_t)kStep, a.n_c - own * kStep));
      else
        own = -1;
    }
    for (int wd = 0; wd < (int)((seed_steps + 63) >> 6); ++wd) {
      uint64_t m = s_seed[wave][wd];
      m = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(m >> 32)) << 32) |
          (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)m);
      while (m) {
        const int64_t st = ((int64_t)wd << 6) + __builtin_ctzll(m);
        m &= m - 1;
        if (st != own) visit(st * kStep, (int)min((int64_t)kStep, a.n_c - st * kStep));
      }
    }
  }

  float4 blo, bhi;
  if (n_groups > 0) box_of(t0, blo, bhi);
  for (int64_t tt = 0; tt < n_groups; ++tt) {
    const int64_t grp = (t0 + tt) % n_groups;
    const int64_t c0 = grp * kGroup;
    const int n_here = (int)min((int64_t)kGroup, a.n_c - c0);
    const float4 lo = blo, hi = bhi;
    if (tt + 1 < n_groups) box_of((t0 + tt + 1) % n_groups, blo, bhi);  // in flight during this group
    // Steps no candidate of which can enter any of the wave's 4 top-k lists:
    // lane l tests step l % 16 against query l / 16. For a candidate c in the
    // box, |x_q - x_c| >= the box distance bx per axis, and the definition's
    // rounded operations are monotone, so with bx, by, bz computed as rounded
    // differences and d = ((bx*bx) + (by*by)) + (bz*bz) in the definition's
    // order, the candidate's distance is at least d. A candidate enters only
    // with distance <= the current k-th distance T, so d > T excludes the
    // whole step. (T only decreases, so the test stays valid for the group;
    // with fewer than k entries T is NaN and nothing is excluded.) Seeds,
    // already visited, are left out too.
    uint32_t skip;
    {
      float qx = q[0].x, qy = q[0].y, qz = q[0].z, T = __uint_as_float((uint32_t)(q[0].tau >> 32));
#pragma unroll
      for (int j = 1; j < kKnnQ; ++j)
        if (jq == j) {
          qx = q[j].x; qy = q[j].y; qz = q[j].z;
          T = __uint_as_float((uint32_t)(q[j].tau >> 32));
        }
      float d;
      {
#pragma clang fp contract(off)
        const float bx = fmaxf(fmaxf(lo.x - qx, qx - hi.x), 0.0f);
        const float by = fmaxf(fmaxf(lo.y - qy, qy - hi.y), 0.0f);
        const float bz = fmaxf(fmaxf(lo.z - qz, qz - hi.z), 0.0f);
        d = (bx * bx + by * by) + bz * bz;
      }
      const uint64_t far = __ballot(d > T);
      skip = (uint32_t)(far & (far >> 16) & (far >> 32) & (far >> 48) & 0xFFFFull);
      const int64_t st0 = grp * (kGroup / kStep);  // a multiple of 16: its seeds are 16 bits of one word
      if (st0 < seed_steps) {
        const uint64_t sw = s_seed[wave][st0 >> 6];
        skip |= (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)((sw >> (st0 & 63)) & 0xFFFFull));
      }
    }
    // In the group that holds the wave's own queries the steps start just
    // before them and wrap around, so their sequence neighbours come first.
    const int n_pairs = (n_here + kStep - 1) / kStep;
    int pr = 0;
    if (a.q_self0 >= 0) {
      const int64_t self = a.q_self0 + rw - c0;
      if (self >= 0 && self < n_here) pr = max(0, (int)(self >> 7) - 1);
    }
    for (int t = 0; t < n_pairs; ++t, pr = pr + 1 == n_pairs ? 0 : pr + 1) {
      if ((skip >> pr) & 1u) continue;
      visit(c0 + pr * kStep, min(kStep, n_here - pr * kStep));
    }
  }
#pragma unroll
  for (int j = 0; j < kKnnQ; ++j) {
    const int64_t r = rw + j;
    if (r >= a.n_q) break;
    if (q[j].bcount > 0) q[j].flush(lane, k);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int i = 64 * s + lane;
      if (i < k) {
        const bool have = i < q[j].count;
        const uint64_t t = q[j].top[s];
        a.idx_out[r * k + i] = have ? (int32_t)(uint32_t)t : -1;
        if (a.d2_out) a.d2_out[r * k + i] = have ? __uint_as_float((uint32_t)(t >> 32)) : __builtin_inff();
      }
    }
  }
}

// Number of entries of the sorted a[0, n) that are < x (or <= x when `or_equal`).
__device__ __forceinline__ int rank_in(const uint64_t* a, int n, uint64_t x, bool or_equal) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const uint64_t m = a[mid];
    if (m < x || (or_equal && m == x))
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// One wave per row: the k smallest keys of two sorted lists (index -1 = empty).
template <int KMAX>
__global__ void __launch_bounds__(256) topk_merge_kernel(TopkMergeArgs a) {
  __shared__ uint64_t s_a[4][KMAX], s_b[4][KMAX];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r = (int64_t)blockIdx.x * 4 + wave;
  if (r >= a.n_rows) return;
  const int k = a.k;
  uint64_t* la = s_a[wave];
  uint64_t* lb = s_b[wave];
  for (int i = lane; i < k; i += 64) {
    const int32_t ia = a.idx_a[r * k + i], ib = a.idx_b[r * k + i];
    la[i] = ia < 0 ? kNoKey : ((uint64_t)__float_as_uint(a.d2_a[r * k + i]) << 32) | (uint32_t)ia;
    lb[i] = ib < 0 ? kNoKey : ((uint64_t)__float_as_uint(a.d2_b[r * k + i]) << 32) | (uint32_t)ib;
  }
  wave_lds_sync();
  for (int i = lane; i < k; i += 64) {
    const uint64_t x = la[i], y = lb[i];
    const int pa = i + rank_in(lb, k, x, false);  // ties: a's entry first
    const int pb = i + rank_in(la, k, y, true);
    if (pa < k) {
      a.idx_out[r * k + pa] = x == kNoKey ? -1 : (int32_t)(uint32_t)x;
      a.d2_out[r * k + pa] = x == kNoKey ? __builtin_inff() : __uint_as_float((uint32_t)(x >> 32));
    }
    if (pb < k) {
      a.idx_out[r * k + pb] = y == kNoKey ? -1 : (int32_t)(uint32_t)y;
      a.d2_out[r * k + pb] = y == kNoKey ? __builtin_inff() : __uint_as_float((uint32_t)(y >> 32));
    }
  }
}

template <int KS>
hipError_t launch_knn_k(const KnnArgs& a, hipStream_t st) {
  if (a.n_c > 0) {
    const dim3 pg((unsigned)(((a.n_c + kStep - 1) / kStep + 3) / 4)), pb(256);
    if (a.group_mode) hipLaunchKernelGGL((knn_prep_kernel<1>), pg, pb, 0, st, a);
    else hipLaunchKernelGGL((knn_prep_kernel<0>), pg, pb, 0, st, a);
  }
  const dim3 grid((unsigned)((a.n_q + kKnnRows - 1) / kKnnRows)), block(64 * kKnnWaves);
  if (a.group_mode == 1)
    hipLaunchKernelGGL((knn_kernel<KS, 1>), grid, block, 0, st, a);
  else if (a.group_mode == 2)
    hipLaunchKernelGGL((knn_kernel<KS, 2>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((knn_kernel<KS, 0>), grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace

size_t knn_workspace_bytes(int64_t n_c, size_t* box_offset) {
  const size_t cand = ((size_t)n_c * 16 + 255) / 256 * 256;
  if (box_offset) *box_offset = cand;
  return cand + (size_t)((n_c + kStep - 1) / kStep) * 32;
}

hipError_t launch_knn(const KnnArgs& a, hipStream_t st) {
  return a.k <= 128 ? launch_knn_k<2>(a, st) : launch_knn_k<4>(a, st);
}

hipError_t launch_topk_merge(const TopkMergeArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.n_rows + 3) / 4)), block(256);
  if (a.k <= 128)
    hipLaunchKernelGGL(topk_merge_kernel<128>, grid, block, 0, st, a);
  else
    hipLaunchKernelGGL(topk_merge_kernel<256>, grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
