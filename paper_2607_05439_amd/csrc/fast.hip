// Fused bf16 path for c_z = 128, H = 16, d = 24 on gfx950 (CDNA4).
//
// Kernels (the q, k, v, g projections that feed them are in proj.hip):
//   attn_kernel  the hot loop: one wave owns 16 query rows and one key range
//                (a ring step of the paper's 2D scheme, or a slice of one). Per
//                key it reads the 16 rows' pair vectors z[i, j, :] once from
//                HBM, forms LayerNorm statistics and the c_z -> H bias
//                projection on the matrix cores, then per 16-key tile runs
//                QK^T and PV on the matrix cores with an fp32 online softmax.
//                It writes one partial state (m, l, acc) per (row, head).
//   bias_ring_kernel  the pair bias alone, materialised (dcp_bias_project):
//                the same z stream, one column per step, whole-line stores
//                (bias_kernel, with z loaded straight into registers, serves
//                row strides too long for 32-bit offsets).
//
// Matrix-core operand layouts (v_mfma_f32_16x16x32_bf16, 64 lanes, lane L,
// n = L % 16, g = L / 16): A holds row n with k-slots 8g..8g+7, B holds
// column n with the same k-slots, and the accumulator holds rows 4g..4g+3 of
// column n. The 16x16x16 form holds k-slots 4g..4g+3. Because A and B share
// the k-slot numbering, the channel order inside k is free; it is chosen so
// each lane's loads are contiguous.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kCz = kFastCz, kH = kFastH, kD = kFastD, kDp = kFastDp;
constexpr int kPre = 4;  // keys of z in flight per wave (registers)
constexpr float kLog2e = 1.44269504088896340736f;
// Logits in base-2 units are offset by this constant inside the QK^T
// accumulator, so every logit of moderate size lands in [128, 256) and is
// rounded to a multiple of 2^-16 there. With integer running maxima, the
// subtraction logit - max is then exact, the softmax weights do not depend on
// which keys were seen before, and rescaling factors are exact powers of two:
// key blocks of any size give the same weights.
constexpr float kShift = kFastShift;

// Bias weights as A operands: row = head (lane % 16), k-step s holds channels
// 32s + 8g .. 32s + 8g + 7. W' = scale * W_b * diag(gamma), centred per head
// (subtracting its mean over channels makes sum_c W''_hc z_c = sum_c W'_hc
// (z_c - mean z)), then split into bf16 hi + lo so the pair carries about 16
// significant bits.
// w_b and gamma are 16-byte aligned (checked on the host): each lane reads its
// 8 consecutive channels per k-step as two 16-byte loads, and the absence of
// gamma is one wave-uniform branch, not one per element.
__device__ void bias_weights(const float* __restrict__ w_b, const float* __restrict__ gamma, float scale, int lane,
                             bf16x8 (&hi)[4], bf16x8 (&lo)[4]) {
  const int h = lane & 15, g = lane >> 4;
  float w[4][8];
  const float4* wr = reinterpret_cast<const float4*>(w_b + h * kCz + 8 * g);  // channel 32 s + 8 g + i: float4 8 s + i / 4
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const float4 a = wr[8 * s], b = wr[8 * s + 1];
    w[s][0] = a.x, w[s][1] = a.y, w[s][2] = a.z, w[s][3] = a.w;
    w[s][4] = b.x, w[s][5] = b.y, w[s][6] = b.z, w[s][7] = b.w;
  }
  if (gamma) {
    const float4* gr = reinterpret_cast<const float4*>(gamma + 8 * g);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const float4 a = gr[8 * s], b = gr[8 * s + 1];
      const float gm[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) w[s][i] *= gm[i];
    }
  }
  float rs = 0.f;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      w[s][i] *= scale;
      rs += w[s][i];
    }
  const float mean = sum4(rs) * (1.0f / kCz);
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float c = w[s][i] - mean;
      const __bf16 x = (__bf16)c;
      hi[s][i] = x;
      lo[s][i] = (__bf16)(c - (float)x);
    }
}

// One key for the wave's 16 rows: z B operands (k-step s = channels 32s+8g..+7
// of row n) -> rstd of the pair and the unnormalised projection acc[i] =
// sum_c W''[4g+i, c] z_c (accumulator rows = heads 4g..4g+3, column = row n).
// The LayerNorm statistics come from the matrix cores as well: ones . z gives
// the row sum in every accumulator register, and the diagonal of the Gram tile
// z . z^T (row n at lane group n/4, register n%4) gives the sum of squares;
// bf16 products are exact in fp32.
__device__ __forceinline__ void pair_bias(const u32x4 (&zb)[4], const bf16x8 (&whi)[4], const bf16x8 (&wlo)[4],
                                          const f32x4& wsum, float eps, int n, f32x4& acc, float& rstd) {
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (__bf16)1.0f;
  f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, gram = {0.f, 0.f, 0.f, 0.f};
  acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const bf16x8 zv = as_bf16x8(zb[s]);
    acc = mfma32(whi[s], zv, acc);
    s1 = mfma32(ones, zv, s1);
    acc = mfma32(wlo[s], zv, acc);
    gram = mfma32(zv, zv, gram);
  }
  // diagonal of the Gram tile: pick register n%4, then fetch it from lane group n/4
  const float t0 = (n & 1) ? gram[1] : gram[0];
  const float t1 = (n & 1) ? gram[3] : gram[2];
  float d = (n & 2) ? t1 : t0;        // (row 4g + n%4, column n)
  const int tg = n >> 2;               // the lane group holding row n
  float lo = d, hi = d;
  swap32(lo, hi);                      // lo: group g&1, hi: group (g&1)|2
  d = (tg & 2) ? hi : lo;              // group (g&1) | (tg&2)
  lo = d;
  hi = d;
  swap16(lo, hi);                      // lo: even group of the pair, hi: odd group
  const float s2 = (tg & 1) ? hi : lo; // group tg: the diagonal entry
  const float mu = s1[0] * (1.0f / kCz);
  // s2/c_z - mu^2 with the square formed exactly inside the fma: one rounding
  // of the exact difference, so a large channel mean (|mu| >> sigma) does not
  // cancel away the variance's significant bits
  const float var = fmaxf(fmaf(-mu, mu, s2 * (1.0f / kCz)), 0.0f);
  rstd = __builtin_amdgcn_rsqf(var + eps);
  // the bf16 hi + lo weights sum to wsum (not exactly 0) per head; remove
  // wsum * mu so the projection is that of z - mu even when mu is large
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = fmaf(-mu, wsum[i], acc[i]);
}

// Per-head sums of the bias weight operands, sum_c (hi + lo)[h, c], in the
// accumulator layout of pair_bias (heads 4g..4g+3 in every column): W'' . 1
// on the matrix cores.
__device__ __forceinline__ f32x4 bias_weight_sums(const bf16x8 (&whi)[4], const bf16x8 (&wlo)[4]) {
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (__bf16)1.0f;
  f32x4 r = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    r = mfma32(whi[s], ones, r);
    r = mfma32(wlo[s], ones, r);
  }
  return r;
}

// ----------------------------------------------------------------------------- attention
constexpr int kWaves = 4;           // waves per workgroup: 4 query tiles sharing one key range
constexpr int kRing = 8;            // z slots per wave (LDS ring)
constexpr int kAhead = kRing - 1;   // keys of z in flight ahead of the one being used
constexpr int kKvDma = 8;           // DMA loads per wave per K/V tile (4 heads x K, V)

// One key's z for a wave's 16 rows: [row][16-byte chunk], chunk index XOR row
// (so the 16 rows of one operand read hit 16 different bank groups).
struct ZSlot {
  u32x4 c[16][16];
};
// K and V^T of one 16-key tile for all heads, in matrix-core operand order:
// k[h][L] = lane L's QK^T A operand; v[h][L] = lane L's PV A operands (M-tile 0
// in .xy, M-tile 1 in .zw).
struct KvTile {
  u32x4 k[kH][64];
  u32x4 v[kH][64];
};

typedef const __attribute__((address_space(4))) uint32_t* const_u32_ptr;

// Valid keys of tile t: the per-tile key mask, restricted to [start, end). The
// mask is read-only during the attention kernel, so it is read through the
// constant address space (a scalar load, outside the vector-memory queue).
__device__ __forceinline__ uint32_t tile_valid_bits(const_u32_ptr tv, int64_t t, int64_t start, int64_t end) {
  const int64_t lo = max(start - t * 16, (int64_t)0), hi = min(end - t * 16, (int64_t)16);
  if (hi <= lo) return 0u;
  const uint32_t range = (hi >= 16 ? 0xFFFFu : ((1u << hi) - 1u)) & ~((1u << lo) - 1u);
  return tv[t] & range;
}

// Outstanding DMA loads allowed when waiting for key kk of a tile: the z loads
// of the kAhead - 1 keys issued after it, plus the K/V tile loads when those
// were issued after it (for the first kAhead keys, whose z was issued during
// the previous tile).
template <int KK>
__device__ __forceinline__ void wait_key() {
  wait_vm<4 * (kAhead - 1) + (KK < kAhead ? kKvDma : 0)>();
}

// One workgroup = 4 waves = 4 tiles of 16 query rows over the same key range
// (one internal part). Each wave streams its rows' z through its own LDS ring
// with direct-to-LDS loads issued kAhead keys ahead; an invalid (masked or
// out-of-range) key gets an out-of-range offset, so its load moves no data and
// every load is unconditional. K/V tiles are loaded into LDS one tile ahead,
// each wave fetching 4 heads, into one LDS buffer; two barriers per tile (the
// second, after the compute-only attention phase, frees the buffer).
__global__ void __launch_bounds__(256, 1) attn_kernel(FastAttnArgs a) {
  __shared__ ZSlot zring[kWaves][kRing];  // 128 KB
  __shared__ KvTile kv;                   // 32 KB
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t n_qt = a.nq_pad / kTileQ;
  // Workgroup -> (row group, part). The hardware deals workgroups to the 8
  // XCDs in turn (workgroup i to XCD i % 8). By default row groups vary
  // fastest, so the resident workgroups of every XCD stream the same part.
  // With xcd_order (layers of at least 256 row groups), XCD x takes the row
  // groups rg = x (mod 8), all parts of them, one part after another starting
  // at part x mod P: each XCD's L2 still serves one part's K/V at a time while
  // the XCDs stream z at different key positions.
  int64_t rg;
  int part;
  if (a.xcd_order) {
    const int P = a.n_kb * a.n_seg;
    const int64_t n_rg = (n_qt + kWaves - 1) / kWaves;
    const int x = blockIdx.x & 7;
    const int64_t k = blockIdx.x >> 3;
    const int64_t cnt = (n_rg - x + 7) / 8;  // row groups of this XCD
    if (k >= cnt * P) return;                // whole workgroup, before any barrier
    rg = x + 8 * (k % cnt);
    part = (int)((x + k / cnt) % P);
  } else {
    rg = blockIdx.x;
    part = blockIdx.y;
  }
  const int64_t qt = rg * kWaves + wave;
  const bool active = qt < n_qt;
  const int64_t q0 = (active ? qt : n_qt - 1) * kTileQ;
  int64_t start, end;
  part_range(a.k_len, a.n_kb, a.n_seg, part, &start, &end);
  start += a.k_lo;
  end += a.k_lo;
  const int64_t t_begin = start >> 4, t_end = (end + 15) >> 4;
  const int64_t n_tiles_all = a.n_pad / 16;

  bf16x8 whi[4], wlo[4];
  bias_weights(a.w_b, a.gamma, kLog2e, lane, whi, wlo);
  const f32x4 wsum = bias_weight_sums(whi, wlo);
  bf16x8 qreg[kH];
#pragma unroll
  for (int h = 0; h < kH; ++h)
    qreg[h] = as_bf16x8(*(reinterpret_cast<const u32x4*>(a.q) + ((int64_t)h * a.nq_pad + q0 + n) * 4 + g));

  float m[kH];
  f32x4 o[kH][2];
#pragma unroll
  for (int h = 0; h < kH; ++h) {
    m[h] = -INFINITY;
    o[h][0] = f32x4{0.f, 0.f, 0.f, 0.f};
    o[h][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // z rows q0 .. q0+15 of this wave: one buffer resource, 32-bit byte offsets.
  const int64_t rows_here = min((int64_t)kTileQ, a.n_q - q0);
  const int row_bytes = (int)(a.n_tok * (kCz * 2));
  const __amdgpu_buffer_rsrc_t zres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.z) + q0 * a.n_tok * kCz, 0, (int)(rows_here * row_bytes), kRawBufferFlags);
  // DMA instruction i of a key fills slot rows 4i..4i+3; lane L writes row
  // 4i + L/16, physical chunk L%16, which holds logical chunk (L%16) ^ row.
  int zoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * i + (lane >> 4);
    zoff[i] = row * row_bytes + 16 * ((lane & 15) ^ row);
  }
  const uint32_t ring_base = lds_addr(&zring[wave][0]);
  // one M0 per key: the instruction offset 1024 i, which moves the LDS and the
  // global address alike, selects load i's quarter of the slot, so its vector
  // offset is that of its rows minus 1024 i
#pragma unroll
  for (int i = 0; i < 4; ++i) zoff[i] -= 1024 * i;
  auto z_dma = [&](int64_t j, bool valid, int slot) {
    const int jo = (int)j * (kCz * 2);
    dma_key_stream(zres, valid ? zoff[0] + jo : kOutOfRange, valid ? zoff[1] + jo : kOutOfRange,
                   valid ? zoff[2] + jo : kOutOfRange, valid ? zoff[3] + jo : kOutOfRange,
                   ring_base + (uint32_t)slot * (uint32_t)sizeof(ZSlot));
  };
  // K/V tiles: this wave fetches heads 4*wave .. 4*wave+3.
  const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.k), 0, (int)(kH * a.n_pad * kDp * 2), kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.vt), 0, (int)(kH * a.n_pad * kDp * 2), kRawBufferFlags);
  auto kv_dma = [&](int64_t t) {
    const uint32_t base = lds_addr(&kv);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * wave + i;
      dma_b128(kres, (int)((((int64_t)h * a.n_pad + t * 16 + n) * kDp + 8 * g) * 2),
               base + (uint32_t)offsetof(KvTile, k) + (uint32_t)(h * 64 * 16));
      dma_b128(vres, (int)((((int64_t)h * n_tiles_all + t) * 64 + lane) * 16),
               base + (uint32_t)offsetof(KvTile, v) + (uint32_t)(h * 64 * 16));
    }
  };

  const const_u32_ptr tvres = (const_u32_ptr)(a.tile_valid);
  uint32_t bits = t_begin < t_end ? tile_valid_bits(tvres, t_begin, start, end) : 0u;
  if (t_begin < t_end) {
    // same issue order as the steady state: the first kAhead keys, then K/V
#pragma unroll
    for (int p = 0; p < kAhead; ++p) z_dma(t_begin * 16 + p, (bits >> p) & 1u, (int)((t_begin * 16 + p) % kRing));
    kv_dma(t_begin);
  }

  for (int64_t t = t_begin; t < t_end; ++t) {
    const uint32_t bits_next = (t + 1 < t_end) ? tile_valid_bits(tvres, t + 1, start, end) : 0u;
    const int slot0 = (int)((t * 16) % kRing);
    float b[16][4];
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      int slot = slot0 + kk % kRing;
      if (slot >= kRing) slot -= kRing;
      if (kk < kAhead)
        wait_key<0>();
      else
        wait_key<kAhead>();
      if ((bits >> kk) & 1u) {
        const ZSlot& zs = zring[wave][slot];
        u32x4 zb[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) zb[st] = zs.c[n][(4 * st + g) ^ n];
        f32x4 acc;
        float rstd;
        pair_bias(zb, whi, wlo, wsum, a.eps, n, acc, rstd);
#pragma unroll
        for (int i = 0; i < 4; ++i) b[kk][i] = fmaf(acc[i], rstd, kShift);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) b[kk][i] = -INFINITY;
      }
      const int nk = kk + kAhead;
      int nslot = slot + kAhead;
      if (nslot >= kRing) nslot -= kRing;
      if (nk < 16)
        z_dma(t * 16 + nk, (bits >> nk) & 1u, nslot);
      else
        z_dma((t + 1) * 16 + (nk - 16), (bits_next >> (nk - 16)) & 1u, nslot);
    }
    // K/V tile t is complete in this wave (its loads precede the last key's);
    // after the barrier, in every wave.
    barrier_lds();
    const KvTile& cur = kv;
    transpose_bias(b);

    // heads in pairs: two independent QK^T / softmax chains and one vote per
    // pair on rescaling (a factor of exactly 1 leaves a head unchanged)
    constexpr int kG = 2;
#pragma unroll
    for (int h0 = 0; h0 < kH; h0 += kG) {
      f32x4 x[kG];
      float mnew[kG], muse[kG], alpha[kG];
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        const int h = h0 + j, ha = h >> 2, hi = h & 3;
        const f32x4 cin = {b[4 * ha + 0][hi], b[4 * ha + 1][hi], b[4 * ha + 2][hi], b[4 * ha + 3][hi]};
        const u32x4 kt = cur.k[h][lane];
        // x[r]: logit (base 2, + kShift) of row n, key 4g + r
        x[j] = mfma32(as_bf16x8(kt), qreg[h], cin);
      }
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        const int h = h0 + j;
        const float tmax = max4(fmaxf(fmaxf(x[j][0], x[j][1]), fmaxf(x[j][2], x[j][3])));
        mnew[j] = fmaxf(m[h], ceilf(tmax));
        muse[j] = (mnew[j] == -INFINITY) ? 0.0f : mnew[j];
        alpha[j] = (m[h] == -INFINITY) ? 0.0f : ldexpf(1.0f, (int)(m[h] - muse[j]));
      }
      bf16x4 p[kG];
#pragma unroll
      for (int j = 0; j < kG; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) p[j][r] = (__bf16)__builtin_amdgcn_exp2f(x[j][r] - muse[j]);
      // the running maximum is an integer and rarely moves, so most pairs skip this
      bool mv = false;
#pragma unroll
      for (int j = 0; j < kG; ++j) mv = mv || alpha[j] != 1.0f;
      if (__any(mv)) {
#pragma unroll
        for (int j = 0; j < kG; ++j) {
          o[h0 + j][0] *= alpha[j];
          o[h0 + j][1] *= alpha[j];
        }
      }
#pragma unroll
      for (int j = 0; j < kG; ++j) {
        const int h = h0 + j;
        const u32x4 vv = cur.v[h][lane];
        o[h][0] = mfma16(as_bf16x4(u32x2{vv[0], vv[1]}), p[j], o[h][0]);
        o[h][1] = mfma16(as_bf16x4(u32x2{vv[2], vv[3]}), p[j], o[h][1]);
        m[h] = mnew[j];
      }
    }
    // every wave is done with K/V tile t: load tile t+1 into the same buffer
    barrier_lds();
    if (t + 1 < t_end) kv_dma(t + 1);
    bits = bits_next;
  }
  wait_vm<0>();  // the last tile's look-ahead loads (no data) before exit

  // Partial state of rows q0 + n: o[h][0][i] = acc e = 4g+i, o[h][1][i] = acc
  // e = 16+4g+i (e = 24 is the denominator l).
  const int64_t row = q0 + n;
  if (!active || row >= a.n_q) return;
#pragma unroll
  for (int h = 0; h < kH; ++h) {
    const float l = o[h][1][0];  // valid in lane group 2 (e = 24)
    if (g == 2) {
      const bool empty = !(l > 0.0f);
      a.m_parts[((int64_t)part * kH + h) * a.n_q + row] = empty ? -INFINITY : m[h] - kShift;
      a.l_parts[((int64_t)part * kH + h) * a.n_q + row] = empty ? 0.0f : l;
    }
    float* accp = a.acc_parts + (((int64_t)part * a.n_q + row) * kH + h) * kD;
    *reinterpret_cast<float4*>(accp + 4 * g) = make_float4(o[h][0][0], o[h][0][1], o[h][0][2], o[h][0][3]);
    if (g < 2)
      *reinterpret_cast<float4*>(accp + 16 + 4 * g) = make_float4(o[h][1][0], o[h][1][1], o[h][1][2], o[h][1][3]);
  }
}

// ----------------------------------------------------------------------------- bias only
// Per-head constant sum_c W_b[h,c] beta_c + b_b[h] for heads 4g..4g+3. Lane
// (n, g) forms the partial sums over channels 8n .. 8n+7 (all its loads issued
// at once: one memory round trip, not one per 16 channels), then the 16 lanes
// of the group add them in a fixed butterfly, which leaves the same bits in
// every lane of the group. w_b and beta are 16-byte aligned (host-checked).
__device__ __forceinline__ void bias_constants(const FastBiasArgs& a, int n, int g, float (&cst)[4]) {
  float part[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (a.beta) {
    const float4* bp = reinterpret_cast<const float4*>(a.beta + 8 * n);
    const float4 b0 = bp[0], b1 = bp[1];
    const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4* wp = reinterpret_cast<const float4*>(a.w_b + (4 * g + i) * kCz + 8 * n);
      const float4 w0 = wp[0], w1 = wp[1];
      const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
      for (int k = 0; k < 8; ++k) part[i] = fmaf(wv[k], bv[k], part[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int m = 8; m >= 1; m >>= 1) part[i] += __shfl_xor(part[i], m, 16);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) cst[i] = (a.b_b ? a.b_b[4 * g + i] : 0.0f) + part[i];
}

constexpr int kBiasRing = 8;               // z slots per wave: 128 KB per workgroup, one per CU
constexpr int kBiasAhead = kBiasRing - 1;  // columns of z in flight ahead of the one being used

// grid (groups of 64 rows, column chunks of an even length); 4 waves of 16
// rows. Each wave streams its rows' z through an LDS ring by direct-to-LDS
// loads, 4 rows x 256 B per load (the pair tensor's fast read pattern), and
// computes the bias of one column per step on the matrix cores. Every two
// columns the results are regrouped across lanes so that each non-temporal
// store writes 8 rows x one whole 128-byte line (a row's two columns); half
// lines written by separate streaming stores would each go to memory alone.
__global__ void __launch_bounds__(64 * kWaves, 1) bias_ring_kernel(FastBiasArgs a) {
  __shared__ ZSlot ring[kWaves][kBiasRing];
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t r0 = ((int64_t)blockIdx.x * kWaves + wave) * 16;
  if (r0 >= a.n_rows) return;  // whole wave; nothing below synchronises waves
  const int64_t c_begin = (int64_t)blockIdx.y * a.cols_per_wave;
  const int64_t c_end = min(c_begin + (int64_t)a.cols_per_wave, a.n_cols);
  bf16x8 whi[4], wlo[4];
  bias_weights(a.w_b, a.gamma, 1.0f, lane, whi, wlo);
  const f32x4 wsum = bias_weight_sums(whi, wlo);
  float cst[4];
  bias_constants(a, n, g, cst);

  // rows r0 .. r0+15 (those past n_rows fall outside the record range: no data)
  const int64_t rows_here = min((int64_t)16, a.n_rows - r0);
  const int row_bytes = (int)(a.row_stride * 2);
  const __amdgpu_buffer_rsrc_t zres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.z) + r0 * a.row_stride, 0, (int)((rows_here - 1) * row_bytes + a.n_cols * (kCz * 2)),
      kRawBufferFlags);
  // load i of a column fills slot rows 4i..4i+3 (lane L: row 4i + L/16, chunk
  // (L%16) ^ row); the instruction offset 1024 i selects the slot quarter
  int zoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * i + (lane >> 4);
    zoff[i] = row * row_bytes + 16 * ((lane & 15) ^ row) - 1024 * i;
  }
  const uint32_t ring_base = lds_addr(&ring[wave][0]);
  auto z_dma = [&](int64_t c) {
    const bool valid = c < c_end;
    const int jo = (int)c * (kCz * 2);
    dma_key_stream(zres, valid ? zoff[0] + jo : kOutOfRange, valid ? zoff[1] + jo : kOutOfRange,
                   valid ? zoff[2] + jo : kOutOfRange, valid ? zoff[3] + jo : kOutOfRange,
                   ring_base + (uint32_t)((c - c_begin) & (kBiasRing - 1)) * (uint32_t)sizeof(ZSlot));
  };
#pragma unroll
  for (int p = 0; p < kBiasAhead; ++p) z_dma(c_begin + p);

  // store lane L of store q: row 8q + L/8, bytes 16 (L%8) of the row's 128
  // bytes for columns c0, c0+1, i.e. head chunk (L%8)%4 of column c0 + (L%8)/4,
  // held by lane (row, group (L%8)%4)
  const int orow = lane >> 3, ochunk = lane & 7;
  for (int64_t c0 = c_begin; c0 < c_end; c0 += 2) {
    float o[2][4];  // o[k][i]: column c0 + k, head 4g + i
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int64_t c = c0 + k;
      // column c has landed: the loads issued after it are the next kBiasAhead - 1
      // columns (loads complete in issue order; stores in between only make this stricter)
      wait_vm<4 * (kBiasAhead - 1)>();
      const ZSlot& zs = ring[wave][(c - c_begin) & (kBiasRing - 1)];
      u32x4 zb[4];
#pragma unroll
      for (int st = 0; st < 4; ++st) zb[st] = zs.c[n][(4 * st + g) ^ n];
      f32x4 acc;
      float rstd;
      pair_bias(zb, whi, wlo, wsum, a.eps, n, acc, rstd);
#pragma unroll
      for (int i = 0; i < 4; ++i) o[k][i] = fmaf(acc[i], rstd, cst[i]);
      z_dma(c + kBiasAhead);  // into column c-1's slot (the wait inside covers this step's reads too)
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int src = (8 * q + orow) + 16 * (ochunk & 3);
      f32x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float lo = __int_as_float(__builtin_amdgcn_ds_bpermute(4 * src, __float_as_int(o[0][i])));
        const float hi = __int_as_float(__builtin_amdgcn_ds_bpermute(4 * src, __float_as_int(o[1][i])));
        v[i] = ochunk < 4 ? lo : hi;
      }
      const int64_t orw = r0 + 8 * q + orow;
      const int64_t oc = c0 + (ochunk >> 2);
      if (orw < a.n_rows && oc < c_end)
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(a.out + (orw * a.n_cols + oc) * kH + 4 * (ochunk & 3)));
    }
  }
  wait_vm<0>();  // the look-ahead loads past the chunk (no data) before exit
}

// The same for row strides too long for 32-bit buffer offsets over 16 rows:
// grid (tiles of 16 rows, column chunks); one wave each, z loaded straight into
// the operand registers.
__global__ void __launch_bounds__(64) bias_kernel(FastBiasArgs a) {
  const int lane = threadIdx.x, n = lane & 15, g = lane >> 4;
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  const int64_t c_begin = (int64_t)blockIdx.y * a.cols_per_wave;
  const int64_t c_end = min(c_begin + (int64_t)a.cols_per_wave, a.n_cols);
  bf16x8 whi[4], wlo[4];
  bias_weights(a.w_b, a.gamma, 1.0f, lane, whi, wlo);
  const f32x4 wsum = bias_weight_sums(whi, wlo);
  float cst[4];
  bias_constants(a, n, g, cst);
  const int64_t row = r0 + n;
  const int64_t rr = min(row, a.n_rows - 1);
  const u32x4* zrow = reinterpret_cast<const u32x4*>(a.z + rr * a.row_stride) + g;
  auto load = [&](int64_t c, u32x4 (&zb)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) zb[s] = __builtin_nontemporal_load(zrow + c * 16 + 4 * s);
  };
  auto column = [&](int64_t c, const u32x4 (&zb)[4]) {
    f32x4 acc;
    float rstd;
    pair_bias(zb, whi, wlo, wsum, a.eps, n, acc, rstd);
    if (row < a.n_rows) {
      float4 o;
      o.x = fmaf(acc[0], rstd, cst[0]);
      o.y = fmaf(acc[1], rstd, cst[1]);
      o.z = fmaf(acc[2], rstd, cst[2]);
      o.w = fmaf(acc[3], rstd, cst[3]);
      *reinterpret_cast<float4*>(a.out + (row * a.n_cols + c) * kH + 4 * g) = o;
    }
  };
  // Two buffers, two columns per iteration, the next column's z always in
  // flight while one is computed. The loads are unconditional (past the end
  // they repeat the last column, unused), so every wait is for the older
  // buffer only, the same on every path into the loop.
  u32x4 za[4], zb[4];
  load(c_begin, za);
  for (int64_t c = c_begin; c < c_end; c += 2) {
    load(min(c + 1, c_end - 1), zb);
    column(c, za);
    load(min(c + 2, c_end - 1), za);
    if (c + 1 < c_end) column(c + 1, zb);
  }
}

}  // namespace

hipError_t launch_fast_attn(const FastAttnArgs& a, hipStream_t st) {
  const int64_t n_qt = a.nq_pad / kTileQ;
  const int64_t n_rg = (n_qt + kWaves - 1) / kWaves;
  const int64_t parts = (int64_t)a.n_kb * a.n_seg;
  FastAttnArgs b = a;
  // numbered per XCD only where every XCD then holds at least 32 row groups
  // (a round of its CUs) of each part, which keeps the XCDs evenly loaded
  b.xcd_order = n_rg >= 256 && parts > 1;
  if (b.xcd_order)
    hipLaunchKernelGGL(attn_kernel, dim3((unsigned)(8 * ((n_rg + 7) / 8) * parts)), dim3(64 * kWaves), 0, st, b);
  else
    hipLaunchKernelGGL(attn_kernel, dim3((unsigned)n_rg, (unsigned)parts), dim3(64 * kWaves), 0, st, b);
  return hipGetLastError();
}

hipError_t launch_fast_bias(const FastBiasArgs& a, hipStream_t st) {
  // 16 rows of the tile must be addressable with 32-bit offsets (plus one slot quarter)
  if ((int64_t)16 * a.row_stride * 2 + 4096 <= INT32_MAX) {
    FastBiasArgs b = a;
    const int64_t groups = (a.n_rows + 16 * kWaves - 1) / (16 * kWaves);
    // about 1024 workgroups (four rounds of one per CU), at least 16 columns each
    int64_t chunks = (1024 + groups - 1) / groups;
    chunks = max((int64_t)1, min(chunks, (a.n_cols + 15) / 16));
    int64_t per = (a.n_cols + chunks - 1) / chunks;
    per += per & 1;  // even: column pairs start on 128-byte lines when n_cols is even
    b.cols_per_wave = (int32_t)per;
    const int64_t ct = (a.n_cols + per - 1) / per;
    hipLaunchKernelGGL(bias_ring_kernel, dim3((unsigned)groups, (unsigned)ct), dim3(64 * kWaves), 0, st, b);
    return hipGetLastError();
  }
  const int64_t rt = (a.n_rows + 15) / 16;
  const int64_t ct = (a.n_cols + a.cols_per_wave - 1) / a.cols_per_wave;
  hipLaunchKernelGGL(bias_kernel, dim3((unsigned)rt, (unsigned)ct), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
