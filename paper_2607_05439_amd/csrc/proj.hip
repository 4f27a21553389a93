// q, k, v, g projections of the single track for the fused bf16 path
// (c_z = 128, H = 16, d = 24) on gfx950: matrix-core products with the fp32
// weights split into a bf16 hi + lo pair, written in the layouts the attention
// kernel's operands want (fast.hip):
//   q  [H][nq_pad][32] bf16, scaled by log2(e) / sqrt(d), zero-padded
//   k  [H][n_pad][32] bf16, zero for masked and padding keys
//   vt [H][n_pad / 16][64][2][4] bf16: V^T tiles in (lane, M-tile) order, with
//      a row of ones at e = 24 for valid keys (the softmax denominator)
//   g  [n_q][H d] fp32, sigmoid applied
//   tile_valid [n_pad / 16]: bit i = key 16 t + i exists and attends
// Matrix-core operand layouts as in fast.hip (v_mfma_f32_16x16x32_bf16).
//
// Two kernels:
//   proj_split_kernel  the four weight matrices, split into bf16 hi + lo and
//                      laid out as matrix-core operands: for projection p,
//                      16-output tile j (rows 16 j .. 16 j + 15 of W_p, which
//                      are the outputs h d + e in order) and k-step s
//                      (channels 32 s .. 32 s + 31), 1 KB of hi then 1 KB of
//                      lo, lane L holding row 16 j + L % 16, channels
//                      32 s + 8 (L / 16) .. + 7. A wave's weight load is then
//                      1 KB of consecutive bytes, where rows of W read in
//                      place give 16 half cache lines per load.
//   proj_kernel        the products. The 384 outputs of a projection are 24
//                      tiles of 16 with no padding (a tile may hold the end
//                      of one head and the start of the next); each wave
//                      takes two tiles over 128 tokens (64 or 32 on small
//                      layers, so that the launch still fills the chip).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kH = kFastH, kD = kFastD, kDp = kFastDp;
constexpr int kHD = kH * kD;         // 384 outputs per projection
constexpr int kOutTiles = kHD / 16;  // 24 output tiles per projection
constexpr float kLog2e = 1.44269504088896340736f;

constexpr int kProjWaves = 8;                                   // waves per workgroup, two output tiles each
constexpr int kProjSideWgs = 2 * kOutTiles / (2 * kProjWaves);  // workgroups per token group and side (3)
constexpr int kProjChunk = 64;                                  // s channels staged in LDS at a time (2 k-steps)
constexpr int kProjRowChunks = kProjChunk / 8;                  // 16-byte chunks per staged row

// byte offset of the split weights of projection p, output tile j, k-step s
__device__ __forceinline__ int split_offset(int p, int j, int s, int n_ks) {
  return ((p * kOutTiles + j) * n_ks + s) * 2048;
}

// One thread per 4 consecutive weights of a row of W_p (reads in row order,
// 16 bytes per thread): element (o, c), o = 16 j + n, c = 32 s + 8 g + i,
// goes to lane 16 g + n, slot i of (p, j, s); 8 bytes of hi and 8 of lo out.
__global__ void __launch_bounds__(256) proj_split_kernel(FastProjArgs a) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int q4 = a.c_s / 4;  // float4s per row
  if (t >= (int64_t)4 * kHD * q4) return;
  const int p = (int)(t / ((int64_t)kHD * q4));
  const int o = (int)(t / q4 % kHD), c = 4 * (int)(t % q4);
  const float* w = p == 0 ? a.w_q : p == 1 ? a.w_k : p == 2 ? a.w_v : a.w_g;
  const float4 x = *reinterpret_cast<const float4*>(w + (int64_t)o * a.c_s + c);
  const float xs[4] = {x.x, x.y, x.z, x.w};
  bf16x4 hi, lo;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const __bf16 hv = (__bf16)xs[i];
    hi[i] = hv;
    lo[i] = (__bf16)(xs[i] - (float)hv);
  }
  const int j = o / 16, n = o % 16, s = c / 32, g = c % 32 / 8, i0 = c % 8;
  char* dst = reinterpret_cast<char*>(a.w_split) + split_offset(p, j, s, a.c_s / 32) + 16 * (16 * g + n) + 2 * i0;
  *reinterpret_cast<bf16x4*>(dst) = hi;
  *reinterpret_cast<bf16x4*>(dst + 1024) = lo;
}

// One workgroup = TILES x 16 tokens (128 when TILES = 8; fewer tiles per
// workgroup, and so more workgroups, when the token count is small) x one side (query: q and g of the stripe's rows;
// key: k and v of all tokens) x 16 of the side's 48 output tiles; wave w of
// workgroup b takes tiles 2 (8 b + w) and the next, of the side's first
// projection for 8 b + w < 12, else its second. The group's s rows are staged
// in LDS, 64 channels at a time and double-buffered, so each s row is read
// from memory once per workgroup; every wave then reads its matrix-core
// operands from LDS (16-byte chunks of a row XOR-swizzled by row / 2, so the
// 16 rows of one operand read cover all banks once). Per 32-channel k-step a
// wave loads its two tiles' split weights (one k-step ahead) and applies them
// to the TILES token tiles: 4 TILES products per 4 KB of weights. The three workgroups
// of a (side, token group) run on the same XCD (dispatch gives workgroup i to
// XCD i % 8), which then fetches the group's s rows once into its L2. Every
// accumulator holds [output][token]; v's tiles are transposed at the end.
template <int TILES>
__global__ void __launch_bounds__(64 * kProjWaves) __attribute__((amdgpu_waves_per_eu(4))) proj_kernel(FastProjArgs a) {
  constexpr int kProjTiles = TILES;                           // 16-token tiles per workgroup
  constexpr int kBlocks = kProjTiles * 2;                     // blocks of 8 staged rows
  constexpr int kProjStage = (kBlocks + kProjWaves - 1) / kProjWaves;  // LDS copies per wave per chunk
  __shared__ __attribute__((aligned(16))) u32x4 s_s[2][kProjTiles * 16][kProjRowChunks];  // 2 x 2 TILES KB
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int64_t item = (int64_t)(slot / kProjSideWgs) * 8 + xcd;  // key groups first, then query groups
  const int pair = (slot % kProjSideWgs) * kProjWaves + wave;     // 0..23 within the side
  const int64_t key_groups = (a.n_pad / 16 + kProjTiles - 1) / kProjTiles;
  const int64_t query_groups = (a.nq_pad / 16 + kProjTiles - 1) / kProjTiles;
  if (item >= key_groups + query_groups) return;  // the whole workgroup, before any barrier
  const bool is_query = item >= key_groups;
  const int64_t grp = is_query ? item - key_groups : item;
  const bool second = pair >= kOutTiles / 2;                          // g or v
  const int which = is_query ? (second ? 3 : 0) : (second ? 2 : 1);  // 0 q, 1 k, 2 v, 3 g
  const int j0 = 2 * (pair % (kOutTiles / 2));                        // first of the wave's two output tiles
  const int64_t limit = is_query ? a.nq_pad : a.n_pad;
  const int64_t n_valid = is_query ? a.n_q : a.n_tok;
  const int64_t base_tok = is_query ? a.q_row0 : 0;
  const int64_t tile0 = grp * kProjTiles;

  // Staging goes straight to LDS (16 bytes per lane): the workgroup's 2 TILES KB
  // per chunk are 2 TILES blocks of 8 rows, block b copied by wave b % 8; lane i of
  // a block fills row 8 b + i / 8, swizzled chunk i % 8, i.e. channel chunk
  // (i % 8) ^ ((row >> 1) & 7) of the 64. Rows past the valid tokens repeat
  // the last one (their outputs are zeroed); c_s is a multiple of 32, so a
  // chunk's upper half past c_s repeats the last 8 channels, whose products
  // with the zero weights there (out-of-range loads) add nothing.
  const int64_t rows_left = min(n_valid - tile0 * 16, (int64_t)(kProjTiles * 16));
  const __amdgpu_buffer_rsrc_t sres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.s + (base_tok + tile0 * 16) * a.c_s), 0, (int)(rows_left * a.c_s * 2),
      kRawBufferFlags);
  const int n_chunks = (a.c_s + kProjChunk - 1) / kProjChunk;
  const int last_row = (int)rows_left - 1;
  auto stage = [&](int kc, int buf) {
#pragma unroll
    for (int m = 0; m < kProjStage; ++m) {
      if (kBlocks % kProjWaves != 0 && wave + kProjWaves * m >= kBlocks) break;  // wave-uniform
      const int row = 8 * (wave + kProjWaves * m) + lane / 8;
      const int ch = min(kc * kProjChunk + 8 * ((lane % 8) ^ ((row >> 1) & 7)), a.c_s - 8);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          sres, (__attribute__((address_space(3))) void*)&s_s[buf][8 * (wave + kProjWaves * m)][0], 16,
          (min(row, last_row) * a.c_s + ch) * 2, 0, 0, 0);
    }
  };

  // the two tiles' split weights of a k-step: hi and lo of tile j0, then of
  // tile j0 + 1, one k-step ahead in two register buffers (k-step ks of a
  // chunk uses buffer ks & 1; a chunk holds an even number of k-steps, so the
  // parity carries over). Loads past the last k-step read out of range: zeros.
  const int n_ks = a.c_s / 32;
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(a.w_split, 0, split_offset(4, 0, 0, n_ks), kRawBufferFlags);
  const int wbase = split_offset(which, j0, 0, n_ks) + 16 * lane;
  u32x4 wbuf[2][4];
  auto load_w = [&](int ks, u32x4 (&dst)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      dst[q] = __builtin_amdgcn_raw_buffer_load_b128(
          wres, ks < n_ks ? wbase + (q >> 1) * n_ks * 2048 + ks * 2048 + (q & 1) * 1024 : kOutOfRange, 0, 0);
  };

  f32x4 acc[kProjTiles][2];
#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) acc[u][0] = acc[u][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  stage(0, 0);
  load_w(0, wbuf[0]);
  for (int kc = 0; kc < n_chunks; ++kc) {
    // chunk kc is in buffer kc & 1 (the barrier waits for this wave's copies
    // into it); nobody still reads the other buffer, which takes chunk kc + 1
    __syncthreads();
    if (kc + 1 < n_chunks) stage(kc + 1, (kc + 1) & 1);
#pragma unroll
    for (int ks = 0; ks < kProjChunk / 32; ++ks) {
      const bf16x8 whi0 = as_bf16x8(wbuf[ks & 1][0]), wlo0 = as_bf16x8(wbuf[ks & 1][1]);
      const bf16x8 whi1 = as_bf16x8(wbuf[ks & 1][2]), wlo1 = as_bf16x8(wbuf[ks & 1][3]);
      load_w(kc * (kProjChunk / 32) + ks + 1, wbuf[(ks + 1) & 1]);  // in flight during this k-step's products
      __builtin_amdgcn_sched_barrier(0);  // (issued here, not sunk towards their use)
#pragma unroll
      for (int u = 0; u < kProjTiles; ++u) {
        const int row = 16 * u + n;
        const bf16x8 sv = as_bf16x8(s_s[kc & 1][row][(4 * ks + g) ^ ((row >> 1) & 7)]);
        acc[u][0] = mfma32(whi0, sv, acc[u][0]);
        acc[u][1] = mfma32(whi1, sv, acc[u][1]);
        acc[u][0] = mfma32(wlo0, sv, acc[u][0]);
        acc[u][1] = mfma32(wlo1, sv, acc[u][1]);
      }
      // keep the next k-step's weight use (which waits for its loads) after
      // this k-step's products
      __builtin_amdgcn_sched_barrier(0);
    }
  }

#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) {
    const int64_t tile = tile0 + u;
    if (tile * 16 >= limit) break;
    const int64_t t0 = tile * 16;
#pragma unroll
    for (int jt = 0; jt < 2; ++jt) {
      const int j = j0 + jt;
      if (which == 2) {
        // transposed through the matrix cores: the accumulator's registers as
        // an A operand of the k = 16 product hold the tile's transpose, and
        // times the identity that lands in the accumulator layout (exact: the
        // bf16 values times 1). Then vt[i] = v[token t0 + 4g + i][output
        // 16 j + n]: for its head h and e = output % 24, the V^T operand item
        // (lane 16 g + e % 16, M-tile e / 16) of keys 4g .. 4g + 3. Rows
        // e >= 16 also write row e + 8: the ones row (e + 8 = 24) or a zero row.
        bf16x4 av, id;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          av[i] = (__bf16)acc[u][jt][i];
          id[i] = (__bf16)(4 * g + i == n ? 1.0f : 0.0f);
        }
        const f32x4 vt = mfma16(av, id, f32x4{0.f, 0.f, 0.f, 0.f});
        const int o = 16 * j + n, h = o / kD, e = o % kD;
        bf16x4 val, pad;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t tok = t0 + 4 * g + i;
          const bool valid = tok < a.n_tok && (a.mask == nullptr || a.mask[tok] != 0);
          val[i] = (__bf16)(valid ? vt[i] : 0.0f);
          pad[i] = (__bf16)(valid && e == 16 ? 1.0f : 0.0f);
        }
        u32x2* dst = reinterpret_cast<u32x2*>(a.vt) + (((int64_t)h * (a.n_pad / 16) + tile) * 64 + 16 * g) * 2;
        dst[(e % 16) * 2 + e / 16] = __builtin_bit_cast(u32x2, val);
        if (e >= 16) dst[(e - 8) * 2 + 1] = __builtin_bit_cast(u32x2, pad);
        continue;
      }
      // acc[u][jt][i] = proj[output 16 j + 4g + i][token t0 + n]; the four
      // outputs lie in one head (24 is a multiple of 4)
      const int64_t tok = t0 + n;
      const int o = 16 * j + 4 * g, h = o / kD, e = o % kD;
      if (which == 3) {
        if (tok >= a.n_q) continue;
        f32x4 sg;
#pragma unroll
        for (int i = 0; i < 4; ++i) sg[i] = 1.0f / (1.0f + __expf(-acc[u][jt][i]));
        *reinterpret_cast<f32x4*>(a.g + tok * kHD + o) = sg;
        continue;
      }
      if (which == 1 && j == 0) {
        // per-tile key mask: bit i = token t0 + i exists and attends
        const bool kv_valid = tok < a.n_tok && (a.mask == nullptr || a.mask[tok] != 0);
        const uint32_t bits = (uint32_t)(__ballot(kv_valid) & 0xFFFFull);
        if (lane == 0) a.tile_valid[tile] = bits;
      }
      bool valid;
      float scale;
      uint16_t* dst;
      if (which == 0) {
        valid = tok < a.n_q;
        scale = kLog2e * 0.20412414523193150818f;  // log2(e) / sqrt(24)
        dst = a.q + ((int64_t)h * a.nq_pad + tok) * kDp;
      } else {
        valid = tok < a.n_tok && (a.mask == nullptr || a.mask[tok] != 0);
        scale = 1.0f;
        dst = a.k + ((int64_t)h * a.n_pad + tok) * kDp;
      }
      bf16x4 val;
#pragma unroll
      for (int i = 0; i < 4; ++i) val[i] = (__bf16)(valid ? acc[u][jt][i] * scale : 0.0f);
      *reinterpret_cast<u32x2*>(dst + e) = __builtin_bit_cast(u32x2, val);
      if (e == kD - 4) *reinterpret_cast<u32x4*>(dst + kD) = u32x4{0u, 0u, 0u, 0u};  // e = 24 .. 31
    }
  }
}

}  // namespace

size_t fast_proj_split_bytes(int32_t c_s) { return (size_t)4 * kOutTiles * (c_s / 32) * 2048; }

hipError_t launch_fast_proj(const FastProjArgs& a, hipStream_t st) {
  const int64_t split_threads = (int64_t)4 * kHD * (a.c_s / 4);
  hipLaunchKernelGGL(proj_split_kernel, dim3((unsigned)((split_threads + 255) / 256)), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // (side, token group) items, rounded up to whole sets of 8 (one per XCD),
  // 3 workgroups each. 128-token groups when that fills the chip twice;
  // else 64 if that fills it once, else 32 (small layers: a 1024-token layer
  // 0.106 -> 0.093 ms, a 4800-token one -0.8%; each wave's weights are then
  // applied to fewer tokens, which costs more than it saves on larger layers).
  auto workgroups = [&](int tiles) {
    const int64_t items = (a.n_pad / 16 + tiles - 1) / tiles + (a.nq_pad / 16 + tiles - 1) / tiles;
    return (items + 7) / 8 * 8 * kProjSideWgs;
  };
  const int64_t w8 = workgroups(8), w4 = workgroups(4), w2 = workgroups(2);
  if (w8 >= 512)
    hipLaunchKernelGGL(proj_kernel<8>, dim3((unsigned)w8), dim3(64 * kProjWaves), 0, st, a);
  else if (w4 >= 256)
    hipLaunchKernelGGL(proj_kernel<4>, dim3((unsigned)w4), dim3(64 * kProjWaves), 0, st, a);
  else
    hipLaunchKernelGGL(proj_kernel<2>, dim3((unsigned)w2), dim3(64 * kProjWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
