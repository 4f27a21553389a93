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
// knn_kernel: a workgroup of 16 waves serves 16 consecutive query rows, one per
// wave. Candidates are staged through LDS in tiles of 2048 (structure of
// arrays) shared by the 16 waves, visited starting at the tile that holds the
// queries themselves when they are candidates (their sequence neighbours are
// close in space, which makes the running threshold tight early; the result
// does not depend on the order). Per 64 candidates a wave computes the keys,
// keeps those below its current k-th key in a 64-entry LDS buffer, and when the
// buffer would overflow merges it into its sorted top-k (bitonic sort of the
// buffer across lanes, then both lists placed by rank with binary searches).
// topk_merge_kernel: one wave per row, the same rank merge of two sorted lists.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kKnnWaves = 16;
constexpr int kTile = 2048;  // candidates per LDS tile
constexpr uint64_t kNoKey = ~0ULL;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
  const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

// Ascending bitonic sort of one key per lane across the wave.
__device__ __forceinline__ uint64_t wave_sort(uint64_t v, int lane) {
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const uint64_t p = shfl_xor_u64(v, stride);
      const bool up = (lane & size) == 0 || size == 64;
      const bool lower = (lane & stride) == 0;
      v = (lower == up) ? (p < v ? p : v) : (p > v ? p : v);
    }
  }
  return v;
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

__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

template <int KMAX, int MODE>
__global__ void __launch_bounds__(64 * kKnnWaves) knn_kernel(KnnArgs a) {
  __shared__ float s_x[kTile], s_y[kTile], s_z[kTile];
  __shared__ int32_t s_g[MODE ? kTile : 1];
  __shared__ uint64_t s_top[kKnnWaves][2][KMAX];
  __shared__ uint64_t s_buf[kKnnWaves][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t r0 = (int64_t)blockIdx.x * kKnnWaves;
  const int64_t r = r0 + wave;
  const bool active = r < a.n_q;
  const int64_t rr = active ? r : a.n_q - 1;
  const float qx = a.x_q[3 * rr], qy = a.x_q[3 * rr + 1], qz = a.x_q[3 * rr + 2];
  const int32_t qg = MODE ? a.group_q[rr] : 0;
  const int k = a.k;

  int cur = 0, count = 0, bcount = 0;
  uint64_t tau = kNoKey;  // keys below tau may enter the top-k
  uint64_t* buf = s_buf[wave];

  // merge the buffer (bcount unsorted keys) into the sorted top-k
  auto flush = [&]() {
    uint64_t v = lane < bcount ? buf[lane] : kNoKey;
    v = wave_sort(v, lane);
    wave_lds_sync();
    buf[lane] = v;
    wave_lds_sync();
    const uint64_t* top = s_top[wave][cur];
    uint64_t* nxt = s_top[wave][cur ^ 1];
    if (lane < bcount) {
      const int pos = lane + rank_in(top, count, v, false);
      if (pos < k) nxt[pos] = v;
    }
    for (int i = lane; i < count; i += 64) {
      const uint64_t t = top[i];
      const int pos = i + rank_in(buf, bcount, t, true);
      if (pos < k) nxt[pos] = t;
    }
    wave_lds_sync();
    count = min(k, count + bcount);
    bcount = 0;
    cur ^= 1;
    tau = count == k ? s_top[wave][cur][k - 1] : kNoKey;
  };

  const int64_t n_tiles = (a.n_c + kTile - 1) / kTile;
  int64_t t0 = 0;
  if (a.q_self0 >= 0 && n_tiles > 0) t0 = ((a.q_self0 + r0) / kTile) % n_tiles;
  for (int64_t tt = 0; tt < n_tiles; ++tt) {
    const int64_t tile = (t0 + tt) % n_tiles;
    const int64_t c0 = tile * kTile;
    const int n_here = (int)min((int64_t)kTile, a.n_c - c0);
    __syncthreads();  // the previous tile has been read by every wave
    for (int i = threadIdx.x; i < n_here; i += 64 * kKnnWaves) {
      const float* p = a.x_c + 3 * (c0 + i);
      s_x[i] = p[0];
      s_y[i] = p[1];
      s_z[i] = p[2];
      if constexpr (MODE != 0) s_g[i] = a.group_c[c0 + i];
    }
    __syncthreads();
    if (!active) continue;
    // 64 candidates per step, no branch on the tile tail: lanes past n_here
    // read stale LDS (inside the tile) and are masked out of `take`
    auto step = [&](int s) {
      const int i = s + lane;
      float d2;
      {
        // the distance is part of the definition: each operation rounded, in
        // this order, never fused into multiply-adds
#pragma clang fp contract(off)
        const float dx = qx - s_x[i], dy = qy - s_y[i], dz = qz - s_z[i];
        d2 = (dx * dx + dy * dy) + dz * dz;
      }
      const uint64_t key = ((uint64_t)__float_as_uint(d2) << 32) | (uint32_t)(a.c_index0 + c0 + i);
      bool take = key < tau && i < n_here;
      if constexpr (MODE == 1) take = take && s_g[i] == qg;
      if constexpr (MODE == 2) take = take && s_g[i] != qg;
      const uint64_t mask = __ballot(take);
      if (mask == 0) return;
      const int n_new = __popcll(mask);
      if (bcount + n_new > 64) flush();
      const int pos = bcount + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
      if (take) buf[pos] = key;
      wave_lds_sync();
      bcount += n_new;
    };
    for (int s = 0; s < n_here; s += 128) {
      step(s);
      if (s + 64 < n_here) step(s + 64);
    }
  }
  if (!active) return;
  if (bcount > 0) flush();
  const uint64_t* top = s_top[wave][cur];
  for (int i = lane; i < k; i += 64) {
    const bool have = i < count;
    const uint64_t t = have ? top[i] : kNoKey;
    a.idx_out[r * k + i] = have ? (int32_t)(uint32_t)t : -1;
    if (a.d2_out) a.d2_out[r * k + i] = have ? __uint_as_float((uint32_t)(t >> 32)) : __builtin_inff();
  }
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

template <int KMAX>
hipError_t launch_knn_k(const KnnArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.n_q + kKnnWaves - 1) / kKnnWaves)), block(64 * kKnnWaves);
  if (a.group_mode == 1)
    hipLaunchKernelGGL((knn_kernel<KMAX, 1>), grid, block, 0, st, a);
  else if (a.group_mode == 2)
    hipLaunchKernelGGL((knn_kernel<KMAX, 2>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((knn_kernel<KMAX, 0>), grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_knn(const KnnArgs& a, hipStream_t st) {
  return a.k <= 128 ? launch_knn_k<128>(a, st) : launch_knn_k<256>(a, st);
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
