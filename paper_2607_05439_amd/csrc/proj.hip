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
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kH = kFastH, kD = kFastD, kDp = kFastDp;
constexpr float kLog2e = 1.44269504088896340736f;

// ----------------------------------------------------------------------------- projections
constexpr int kProjTiles = 8;                   // 16-token tiles per workgroup (128 tokens)
constexpr int kProjWaves = 8;                   // waves per workgroup, one head each
constexpr int kProjHalves = kH / kProjWaves;    // workgroups per (token group, projection)
constexpr int kProjChunk = 64;                  // s channels staged in LDS at a time (2 k-steps)
constexpr int kProjRowChunks = kProjChunk / 8;  // 16-byte chunks per staged row
constexpr int kProjStage = kProjTiles * 16 * kProjRowChunks / (64 * kProjWaves);  // loads per thread

// One workgroup = 128 tokens x one projection {q, k, v, g} x 8 heads; wave w
// computes head 8 * half + w. The group's s rows are staged in LDS, 64
// channels at a time and double-buffered, so each s row is read from memory
// once per workgroup; every wave then reads its matrix-core operands from
// LDS (16-byte chunks of a row XOR-swizzled by row / 2, so the 16 rows of one
// operand read cover all banks once). Per 32-channel k-step a wave converts
// its head's fp32 weight rows to bf16 hi + lo (loaded one k-step ahead) and
// applies them to the 8 tiles: 32 products per weight load. Workgroups are
// numbered so that the 8 workgroups of a token group (4 projections x 2 head
// halves) run on the same XCD (dispatch gives workgroup i to XCD i % 8), which
// then fetches the group's s rows once into its L2.
__global__ void __launch_bounds__(64 * kProjWaves) __attribute__((amdgpu_waves_per_eu(4))) proj_kernel(FastProjArgs a) {
  __shared__ __attribute__((aligned(16))) u32x4 s_s[2][kProjTiles * 16][kProjRowChunks];  // 2 x 16 KB
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int64_t grp = (int64_t)(slot / (4 * kProjHalves)) * 8 + xcd;
  const int sub = slot % (4 * kProjHalves);
  const int which = sub / kProjHalves;  // 0 q, 1 k, 2 v, 3 g
  const int h = (sub % kProjHalves) * kProjWaves + wave;
  const bool is_query = (which == 0 || which == 3);
  const int64_t limit = is_query ? a.nq_pad : a.n_pad;
  const int64_t tile0 = grp * kProjTiles;
  if (tile0 * 16 >= limit) return;  // the whole workgroup, before any barrier
  const int64_t n_valid = is_query ? a.n_q : a.n_tok;
  const int64_t base_tok = is_query ? a.q_row0 : 0;
  const float* w = which == 0 ? a.w_q : which == 1 ? a.w_k : which == 2 ? a.w_v : a.w_g;

  // All loads are unconditional buffer loads; a load past the end of its
  // buffer returns zeros and moves no data (the compiler then knows how many
  // loads are in flight on every path and can wait for exactly the old ones).
  // Staging: load m of thread t moves 16 bytes, item i = t + 512 m: row i / 8
  // (rows past the valid tokens repeat the last one; their outputs are
  // zeroed), chunk i % 8 of the 64 channels.
  const int64_t rows_left = min(n_valid - tile0 * 16, (int64_t)(kProjTiles * 16));
  const __amdgpu_buffer_rsrc_t sres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.s + (base_tok + tile0 * 16) * a.c_s), 0, (int)(rows_left * a.c_s * 2),
      kRawBufferFlags);
  int st_off[kProjStage];
#pragma unroll
  for (int m = 0; m < kProjStage; ++m) {
    const int i = tid + 64 * kProjWaves * m, row = i / kProjRowChunks, c = i % kProjRowChunks;
    st_off[m] = (int)(min((int64_t)row, rows_left - 1) * a.c_s * 2) + 16 * c;
  }
  const int n_chunks = (a.c_s + kProjChunk - 1) / kProjChunk;
  auto stage_load = [&](int kc, u32x4 (&v)[kProjStage]) {
#pragma unroll
    for (int m = 0; m < kProjStage; ++m) {
      const int c = (tid + 64 * kProjWaves * m) % kProjRowChunks;
      const bool in = kc * kProjChunk + 8 * c < a.c_s;
      v[m] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(sres, in ? st_off[m] + kc * kProjChunk * 2 : kOutOfRange, 0, 0));
    }
  };
  auto stage_store = [&](int buf, const u32x4 (&v)[kProjStage]) {
#pragma unroll
    for (int m = 0; m < kProjStage; ++m) {
      const int i = tid + 64 * kProjWaves * m, row = i / kProjRowChunks, c = i % kProjRowChunks;
      s_s[buf][row][c ^ ((row >> 1) & 7)] = v[m];
    }
  };

  // weight rows e = 16 et + n of head h (zero for e >= 24), k-slots 8g .. 8g+7,
  // one k-step ahead in two register buffers (k-step ks uses buffer ks & 1;
  // a chunk holds an even number of k-steps, so the parity carries over)
  float4 wbuf[2][2][2];
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(w), 0, kH * kD * a.c_s * 4, kRawBufferFlags);
  auto load_w = [&](int k0, float4 (&dst)[2][2]) {
#pragma unroll
    for (int et = 0; et < 2; ++et) {
      const int e = 16 * et + n;
      const int off = (e < kD && k0 < a.c_s) ? ((h * kD + e) * a.c_s + k0 + 8 * g) * 4 : kOutOfRange;
      dst[et][0] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(wres, off, 0, 0));
      dst[et][1] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(wres, off + 16, 0, 0));
    }
  };

  f32x4 acc[kProjTiles][2];
#pragma unroll
  for (int u = 0; u < kProjTiles; ++u) acc[u][0] = acc[u][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the product loop, instantiated per operand orientation (swap: v, whose
  // accumulator is [token][e]; the others [e][token]) so the loop body has no
  // branches
  auto products = [&](auto swap_tag) {
    constexpr bool kSwap = decltype(swap_tag)::value;
    {
      u32x4 first[kProjStage];
      stage_load(0, first);
      stage_store(0, first);
    }
    load_w(0, wbuf[0]);
    for (int kc = 0; kc < n_chunks; ++kc) {
      __syncthreads();  // chunk kc is in buffer kc & 1; nobody still reads the other buffer
      const bool more = kc + 1 < n_chunks;
      u32x4 nxt[kProjStage];
      stage_load(more ? kc + 1 : kc, nxt);
      // every chunk runs its 2 k-steps: channels past c_s are zeros on both
      // sides (out-of-range loads), which add nothing
#pragma unroll
      for (int ks = 0; ks < kProjChunk / 32; ++ks) {
        const int k0 = kc * kProjChunk + 32 * ks;
        bf16x8 whi[2], wlo[2];
#pragma unroll
        for (int et = 0; et < 2; ++et) {
          const float4 w0 = wbuf[ks & 1][et][0], w1 = wbuf[ks & 1][et][1];
          const float xs[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const __bf16 hv = (__bf16)xs[i];
            whi[et][i] = hv;
            wlo[et][i] = (__bf16)(xs[i] - (float)hv);
          }
        }
        load_w(k0 + 32, wbuf[(ks + 1) & 1]);  // the next k-step, in flight during this one's products
        __builtin_amdgcn_sched_barrier(0);     // (issued here, not sunk towards their use)
#pragma unroll
        for (int u = 0; u < kProjTiles; ++u) {
          const int row = 16 * u + n;
          const bf16x8 sv = as_bf16x8(s_s[kc & 1][row][(4 * ks + g) ^ ((row >> 1) & 7)]);
#pragma unroll
          for (int et = 0; et < 2; ++et) {
            if constexpr (kSwap) {
              acc[u][et] = mfma32(sv, whi[et], acc[u][et]);
              acc[u][et] = mfma32(sv, wlo[et], acc[u][et]);
            } else {
              acc[u][et] = mfma32(whi[et], sv, acc[u][et]);
              acc[u][et] = mfma32(wlo[et], sv, acc[u][et]);
            }
          }
        }
        // keep the next k-step's conversion (which waits for its loads) after
        // this k-step's products
        __builtin_amdgcn_sched_barrier(0);
      }
      if (more) stage_store((kc + 1) & 1, nxt);
    }
  };
  if (which == 2)
    products(std::integral_constant<bool, true>{});
  else
    products(std::integral_constant<bool, false>{});

  {
#pragma unroll
    for (int u = 0; u < kProjTiles; ++u) {
      const int64_t tile = tile0 + u;
      if (tile * 16 >= limit) break;
      const int64_t t0 = tile * 16;
      if (which == 2) {
        // acc[u][et][i] = v[token t0 + 4g + i][e = 16 et + n]: exactly the
        // V^T tile operand (lane L, slot i) of rows e = 16 et + n, keys 4g + i.
#pragma unroll
        for (int et = 0; et < 2; ++et) {
          const int e = 16 * et + n;
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int64_t tok = t0 + 4 * g + i;
            const bool valid = tok < a.n_tok && (a.mask == nullptr || a.mask[tok] != 0);
            float val = valid ? acc[u][et][i] : 0.0f;
            if (e == kD) val = valid ? 1.0f : 0.0f;  // row of ones: the softmax denominator
            o[i] = (__bf16)val;
          }
          u32x2* dst = reinterpret_cast<u32x2*>(a.vt) + ((((int64_t)h * (a.n_pad / 16) + tile) * 64 + lane) * 2 + et);
          *dst = __builtin_bit_cast(u32x2, o);
        }
        continue;
      }
      // acc[u][et][i] = proj[e = 16 et + 4g + i][token t0 + n]
      const int64_t tok = t0 + n;
      if (which == 3) {
        if (tok >= a.n_q) continue;
#pragma unroll
        for (int et = 0; et < 2; ++et) {
          const int e0 = 16 * et + 4 * g;
          if (e0 >= kD) continue;
          float4 o;
          o.x = 1.0f / (1.0f + __expf(-acc[u][et][0]));
          o.y = 1.0f / (1.0f + __expf(-acc[u][et][1]));
          o.z = 1.0f / (1.0f + __expf(-acc[u][et][2]));
          o.w = 1.0f / (1.0f + __expf(-acc[u][et][3]));
          *reinterpret_cast<float4*>(a.g + tok * (kH * kD) + h * kD + e0) = o;
        }
        continue;
      }
      if (which == 1 && h == 0) {
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
#pragma unroll
      for (int et = 0; et < 2; ++et) {
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (__bf16)(valid ? acc[u][et][i] * scale : 0.0f);  // rows >= 24 are 0
        *reinterpret_cast<u32x2*>(dst + 16 * et + 4 * g) = __builtin_bit_cast(u32x2, o);
      }
    }
  }
}

}  // namespace

hipError_t launch_fast_proj(const FastProjArgs& a, hipStream_t st) {
  // token groups rounded up to whole sets of 8 (one per XCD), 4 projections x
  // 2 head halves each
  const int64_t tiles = (a.n_pad > a.nq_pad ? a.n_pad : a.nq_pad) / 16;
  const int64_t groups = (tiles + kProjTiles - 1) / kProjTiles;
  const int64_t sets = (groups + 7) / 8;
  hipLaunchKernelGGL(proj_kernel, dim3((unsigned)(sets * 8 * 4 * kProjHalves)), dim3(64 * kProjWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
