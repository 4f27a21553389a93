// Pair transition on gfx950 (CDNA4): z <- z + W3 (SiLU(W1 LN z) * W2 LN z)
// per pair (Appendix "Manual SwiGLU decomposition"). The paper's memory
// device (free each 4x-expanded tensor as soon as it is used) becomes, on one
// GPU, a fused kernel in which no expanded tensor ever leaves the registers.
//
// bf16 path, c_z = 128, hidden = 512 (matrix cores):
//   trans_prep_kernel  rounds the weights to bf16 and writes them as
//                      matrix-core operand tiles, 24 KB per 32 hidden units
//                      (W1, W2 and W3 for v_mfma_f32_16x16x32_bf16, W3's rows
//                      permuted so the output accumulator lines up with the z
//                      channels a lane holds), and gamma, beta as fp32.
//   trans_kernel       one workgroup of 8 waves per CU (two per SIMD),
//                      persistent over groups of 256 pairs, 32 per wave. Per
//                      group: z (B operands: lane (pair n, group g) holds
//                      channels 32 ks + 8g .. +7), LayerNorm with gamma and
//                      beta in registers; then for each 32 hidden units:
//                      A = W1' N and B = W2 N as transposed products (hidden x
//                      pairs), h = SiLU(A) * B in registers, which is exactly
//                      the B operand layout of the second product
//                      out^T += W3' h^T; finally z + out, bf16, stored where z
//                      was read. Weight tiles stream through two 48 KB LDS
//                      buffers by direct-to-LDS loads, one chunk of 64 hidden
//                      units ahead, and reach the registers through a short
//                      queue of LDS reads issued a few products early; the
//                      next group's z is staged into the other 64 KB of LDS
//                      the same way while this group computes. On this chip
//                      every 1 KB LDS read also costs matrix-core issue time,
//                      which is why each weight fragment serves two pair tiles.
// fp32 path (any c_z <= 256, hidden <= 1024): one wave per pair, plain fp32.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "cdna4.h"
#include "dcp_internal.h"

namespace dcp {
namespace {

constexpr int kCz = kTransCz;       // 128
constexpr int kHid = kTransHidden;  // 512
constexpr int kHt = kHid / 16;      // hidden tiles of 16 units
constexpr int kTileBytes = 12 * 1024;  // per hidden tile: W1 4 KB, W2 4 KB, W3 4 KB
constexpr int kChunkTiles = 4;          // hidden tiles per LDS chunk (two tile pairs)
constexpr int kChunks = kHt / kChunkTiles;
constexpr int kChunkBytes = kChunkTiles * kTileBytes;  // 48 KB
constexpr int kWaves = 8;                              // per workgroup, two per SIMD
constexpr int kWavePairs = 32;                         // pairs per wave: two tiles of 16
constexpr int kGroupPairs = kWaves * kWavePairs;       // 256
constexpr int kDmaPerWave = kChunkBytes / 1024 / kWaves;  // 1 KB DMA instructions per wave per chunk
constexpr float kLog2e = 1.44269504088896340736f;

// Output channel held at accumulator row r (0..15) of output tile ct: tiles
// 2ks and 2ks+1 cover channels 32ks .. 32ks+31 so that lane group g holds
// channels 32ks + 8g .. 32ks + 8g + 7, the ones it loaded as a B operand.
__host__ __device__ inline int out_channel(int ct, int r) { return 32 * (ct >> 1) + 8 * (r >> 2) + 4 * (ct & 1) + (r & 3); }

// ----------------------------------------------------------------------------- weight preparation
// Scaling: W1 carries a factor -log2(e), so the kernel's A' = -log2(e) A gives
// sigmoid(A) = 1 / (1 + 2^A') with no extra multiply, and
// SiLU(A) B = A B sigmoid(A) = -ln(2) A' B / (1 + 2^A'); the factor -ln(2)
// goes into W3. Layout per pair of hidden tiles (32 units, 24 KB):
//   W1 and W2 A operands of v_mfma_f32_16x16x32_bf16 for each of the two
//   tiles: [tile][mat][ks][lane] 16 B (row = unit, k-slots = channels
//   32 ks + 8 (lane/16) .. +7), 16 KB;
//   W3 A operands of v_mfma_f32_16x16x32_bf16 over the 32 units: [ct][lane]
//   16 B (row = channel out_channel(ct, lane%16), k-slot j of lane group g =
//   unit 4g + j of the first tile for j < 4, of the second for j >= 4, the
//   order in which the lane holds SiLU(A) B), 8 KB.
// After the tiles: gamma and beta (fp32, 1 and 0 when absent).
constexpr int kPairBytes = 2 * kTileBytes;
constexpr int kPrepFragments = (kHt / 2) * (2 * 2 * 4 * 64 + 8 * 64);  // 16-byte fragments
__global__ void __launch_bounds__(256) trans_prep_kernel(TransArgs a) {
  const float s1 = -kLog2e, s3 = -0.69314718055994530942f;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int per_pair = 2 * 2 * 4 * 64 + 8 * 64;
  if (t < kPrepFragments) {
    const int hp = t / per_pair, f = t % per_pair;
    char* base = static_cast<char*>(a.w_prep) + (size_t)hp * kPairBytes;
    bf16x8 v;
    if (f < 1024) {
      const int tile = f / 512, mat = (f / 256) % 2, ks = (f / 64) % 4, lane = f % 64;
      const float* w = mat ? a.w2 : a.w1;
      const float sc = mat ? 1.0f : s1;
      const int unit = 16 * (2 * hp + tile) + (lane & 15), c0 = 32 * ks + 8 * (lane >> 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = (__bf16)(w[unit * kCz + c0 + i] * sc);
      *reinterpret_cast<u32x4*>(base + tile * 8192 + mat * 4096 + ks * 1024 + lane * 16) = __builtin_bit_cast(u32x4, v);
    } else {
      const int f3 = f - 1024, ct = f3 / 64, lane = f3 % 64, g = lane >> 4;
      const int ch = out_channel(ct, lane & 15);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int unit = 16 * (2 * hp + (j >> 2)) + 4 * g + (j & 3);
        v[j] = (__bf16)(a.w3[ch * kHid + unit] * s3);
      }
      *reinterpret_cast<u32x4*>(base + 16384 + ct * 1024 + lane * 16) = __builtin_bit_cast(u32x4, v);
    }
  }
  const int u = t - kPrepFragments;
  if (u >= 0 && u < 2 * kCz)
    a.gb_prep[u] = u < kCz ? (a.gamma ? a.gamma[u] : 1.0f) : (a.beta ? a.beta[u - kCz] : 0.0f);
}

// ----------------------------------------------------------------------------- fused transition
__global__ void __launch_bounds__(64 * kWaves) trans_kernel(TransArgs a) {
  __shared__ __attribute__((aligned(16))) char s_w[2][kChunkBytes];        // 96 KB of weights
  __shared__ __attribute__((aligned(16))) u32x4 s_z[kWaves][8][64];        // 64 KB: next group's z
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t n_groups = (a.n_pairs + kGroupPairs - 1) / kGroupPairs;
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(a.w_prep, 0, kHt * kTileBytes, kRawBufferFlags);
  // chunk c of the weights (48 KB) into LDS buffer b: this wave's 6 KB eighth
  auto chunk_dma = [&](int c, int b) {
    const uint32_t base = lds_addr(&s_w[b][0]) + (uint32_t)(wave * kDmaPerWave * 1024);
#pragma unroll
    for (int i = 0; i < kDmaPerWave; ++i)
      dma_b128(wres, c * kChunkBytes + (wave * kDmaPerWave + i) * 1024 + lane * 16, base + (uint32_t)(i * 1024));
  };
  // z of this wave's 32 pairs of group gr, slot i = 4p + ks: lane (n, g) gets
  // pair 16p + n, channels 32 ks + 8g .. +7 (the B operand it needs), at
  // s_z[wave][i][lane]; pairs past n_pairs read as zeros (buffer range check)
  auto z_rsrc = [&](int64_t gr) {
    const int64_t pair0 = gr * kGroupPairs + wave * kWavePairs;
    const int64_t left = (a.n_pairs - pair0) * (int64_t)(kCz * 2);  // negative past the end: no records
    const uint32_t bytes = (uint32_t)max((int64_t)0, min(left, (int64_t)(kWavePairs * kCz * 2)));
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(static_cast<const uint16_t*>(a.z_in) + pair0 * kCz), 0, (int)bytes, kRawBufferFlags);
  };
  auto z_dma = [&](__amdgpu_buffer_rsrc_t zr, int i) {
    const int p = i >> 2, ks = i & 3;
    dma_b128(zr, (16 * p + n) * (kCz * 2) + (32 * ks + 8 * g) * 2, lds_addr(&s_z[wave][i][0]));
  };

  int64_t grp = blockIdx.x;
  if (grp >= n_groups) return;  // whole workgroup, before any barrier
  {
    const __amdgpu_buffer_rsrc_t zr = z_rsrc(grp);
#pragma unroll
    for (int i = 0; i < 8; ++i) z_dma(zr, i);
  }
  chunk_dma(0, 0);
  wait_vm<kDmaPerWave>();  // the first group's z has landed (each wave reads only its own slots)
  int seq = 0;  // chunk sequence number across groups (buffer = seq & 1)
  for (; grp < n_groups; grp += gridDim.x) {
    const bool last_group = grp + gridDim.x >= n_groups;
    const int64_t pair0 = grp * kGroupPairs + wave * kWavePairs;
    // LayerNorm of the staged z (two passes over the pair's 128 channels: 32
    // per lane, 4 lanes), then gamma and beta (from global memory: small and
    // cached)
    // The output accumulators start at z itself (the residual): accumulator
    // (ct = 2 ks + s, register i) is channel 32 ks + 8g + 4s + i, element
    // 4s + i of the lane's staged chunk ks, so z never has to be read again.
    f32x4 acc[8][2];  // out^T: output tile ct, pair tile p
    bf16x8 nv[2][4];
    {
      float x[2][4][8], rstd[2];
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float s = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const u32x4 zz = s_z[wave][4 * p + ks][lane];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint32_t w = zz[i >> 1];
            x[p][ks][i] = __uint_as_float((i & 1) ? (w & 0xFFFF0000u) : (w << 16));
            acc[2 * ks + (i >> 2)][p][i & 3] = x[p][ks][i];
            s += x[p][ks][i];
          }
        }
        const float mu = sum4(s) * (1.0f / kCz);
        float v = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            x[p][ks][i] -= mu;
            v = fmaf(x[p][ks][i], x[p][ks][i], v);
          }
        rstd[p] = __builtin_amdgcn_rsqf(sum4(v) * (1.0f / kCz) + a.eps);
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c0 = 32 * ks + 8 * g;
        const float4 ga = *reinterpret_cast<const float4*>(a.gb_prep + c0);
        const float4 gb = *reinterpret_cast<const float4*>(a.gb_prep + c0 + 4);
        const float4 ba = *reinterpret_cast<const float4*>(a.gb_prep + kCz + c0);
        const float4 bb = *reinterpret_cast<const float4*>(a.gb_prep + kCz + c0 + 4);
        const float gm[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
        const float bt[8] = {ba.x, ba.y, ba.z, ba.w, bb.x, bb.y, bb.z, bb.w};
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int i = 0; i < 8; ++i) nv[p][ks][i] = (__bf16)fmaf(x[p][ks][i] * rstd[p], gm[i], bt[i]);
      }
    }
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};

    bf16x8 hv[2];
    // h' = A' B / (1 + 2^A') of one tile pair, as the B operand over its 32
    // units (k-slot j: unit 4g + j of tile 0 for j < 4, of tile 1 for j >= 4)
    auto silu = [&](const f32x4 (&ha)[2][2], const f32x4 (&hb)[2][2]) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float x = ha[j >> 2][p][j & 3];
          hv[p][j] = (__bf16)(x * hb[j >> 2][p][j & 3] * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x)));
        }
    };
    const bool stage_next = !last_group;
    const __amdgpu_buffer_rsrc_t znext = z_rsrc(stage_next ? grp + gridDim.x : grp);
    f32x4 h[2][2][2];  // first products of one tile pair: [W1' | W2][tile][pair tile]
    for (int c = 0; c < kChunks; ++c) {
      const int b = seq & 1;
      barrier_lds();  // every wave is done with buffer b ^ 1 (the previous chunk)
      const bool more = c + 1 < kChunks || !last_group;
      if (more) chunk_dma((c + 1) % kChunks, b ^ 1);
      // the next group's z, staged over chunks 0..6 (two slots in chunk 0),
      // after this chunk's weight loads so that the wait below does not
      // include it; everything staged has landed by chunk 7's wait
      if (stage_next && c < 7) {
        if (c == 0) z_dma(znext, 0);
        z_dma(znext, c + 1);
      }
      if (!more)
        wait_vm<0>();
      else if (stage_next && c == 0)
        wait_vm<kDmaPerWave + 2>();  // this wave's loads of chunk c have landed
      else if (stage_next && c < 7)
        wait_vm<kDmaPerWave + 1>();
      else
        wait_vm<kDmaPerWave>();
      barrier_lds();  // and every other wave's
      const char* chunk = s_w[b];
      // The chunk's 48 weight fragments (1 KB per wave each) in use order:
      // per tile pair q, 16 first-product fragments (tile tt, k-step ks,
      // matrix W1'/W2), then 8 W3'' fragments (output tile ct). They are
      // read from LDS kAhead fragments before their products, through a
      // queue of registers, so the LDS latency stays off the critical path.
      constexpr int kFrags = 2 * 24;
      constexpr int kAhead = 4;
      auto frag = [&](int f) {
        const int q = f / 24, r = f % 24;
        const int off = r < 16 ? (r >> 3) * 8192 + (r & 1) * 4096 + ((r >> 1) & 3) * 1024 : 16384 + (r - 16) * 1024;
        return *reinterpret_cast<const u32x4*>(chunk + q * kPairBytes + off + lane * 16);
      };
      u32x4 wq[kAhead];
#pragma unroll
      for (int f = 0; f < kAhead; ++f) wq[f] = frag(f);
#pragma unroll
      for (int f = 0; f < kFrags; ++f) {
        const bf16x8 w = as_bf16x8(wq[f % kAhead]);
        if (f + kAhead < kFrags) wq[f % kAhead] = frag(f + kAhead);
        const int r = f % 24;
        if (r < 16) {
          // A' = W1' N or B = W2 N (rows: hidden units 16 ht + 4g + i; columns: pairs)
          const int tt = r >> 3, ks = (r >> 1) & 3, m = r & 1;
#pragma unroll
          for (int p = 0; p < 2; ++p) h[m][tt][p] = mfma32(w, nv[p][ks], ks == 0 ? zero : h[m][tt][p]);
        } else {
          if (r == 16) silu(h[0], h[1]);
          // out^T += W3'' h'^T
#pragma unroll
          for (int p = 0; p < 2; ++p) acc[r - 16][p] = mfma32(w, hv[p], acc[r - 16][p]);
        }
        // keep each step's read where it is: the compiler would otherwise
        // move the reads next to their uses
        __builtin_amdgcn_sched_barrier(0);
      }
      ++seq;
    }
    // store. Accumulator (ct = 2 ks + s, register i) is channel 32 ks + 8g +
    // 4s + i of pair 16p + n: lane (n, g) holds bytes 64 ks + 16 g .. +15 of
    // the pair's 256-byte row for each ks. Those are regrouped across lanes so
    // that each store instruction writes 8 pairs x one whole 128-byte line
    // (lane L: pair 8 half + L / 8, bytes 128 line + 16 (L % 8)); half lines
    // written by separate streaming stores were each sent to memory on their own.
    {
      uint32_t o[2][4][4];  // [pair tile][ks][dword]: bf16 pairs of the lane's chunk
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          bf16x8 v;
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = (__bf16)acc[2 * ks + (e >> 2)][p][e & 3];  // z + W3'' h'
          const u32x4 w = __builtin_bit_cast(u32x4, v);
#pragma unroll
          for (int d = 0; d < 4; ++d) o[p][ks][d] = w[d];
        }
      const bool upper = (lane & 4) != 0;  // chunk L % 8 >= 4: the second 64 bytes of the line
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int src = 8 * half + (lane >> 3) + 16 * (lane & 3);  // lane (n, g) holding the bytes
#pragma unroll
          for (int line = 0; line < 2; ++line) {
            u32x4 v;
#pragma unroll
            for (int d = 0; d < 4; ++d) {
              const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(4 * src, (int)o[p][2 * line][d]);
              const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(4 * src, (int)o[p][2 * line + 1][d]);
              v[d] = upper ? hi : lo;
            }
            const int64_t pr = pair0 + 16 * p + 8 * half + (lane >> 3);
            if (pr < a.n_pairs) {
              u32x4* dst = reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.z_out) + pr * kCz) + 8 * line + (lane & 7);
              __builtin_nontemporal_store(v, dst);
            }
          }
        }
    }
  }
  wait_vm<0>();
}

// ----------------------------------------------------------------------------- fp32 path
// One wave per pair: LayerNorm, then 8+ hidden units per lane, h in LDS, then
// the output channels per lane; fp32 throughout.
__global__ void __launch_bounds__(256) trans_gen_kernel(TransGenArgs a) {
  __shared__ float s_n[4][kGenMaxCz];
  __shared__ float s_h[4][kTransGenMaxHidden];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t p = (int64_t)blockIdx.x * 4 + wave;
  if (p >= a.n_pairs) return;
  const float* z = a.z_in + p * a.c_z;
  float s = 0.0f;
  for (int c = lane; c < a.c_z; c += 64) s += z[c];
  for (int m = 32; m > 0; m >>= 1) s += __shfl_xor(s, m);
  const float mu = s / (float)a.c_z;
  float v = 0.0f;
  for (int c = lane; c < a.c_z; c += 64) v = fmaf(z[c] - mu, z[c] - mu, v);
  for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m);
  const float rstd = 1.0f / sqrtf(v / (float)a.c_z + a.eps);
  float* nn = s_n[wave];
  for (int c = lane; c < a.c_z; c += 64)
    nn[c] = (a.gamma ? a.gamma[c] : 1.0f) * ((z[c] - mu) * rstd) + (a.beta ? a.beta[c] : 0.0f);
  __builtin_amdgcn_wave_barrier();
  float* hh = s_h[wave];
  for (int u = lane; u < a.hidden; u += 64) {
    float x = 0.0f, y = 0.0f;
    for (int c = 0; c < a.c_z; ++c) {
      x = fmaf(a.w1[(int64_t)u * a.c_z + c], nn[c], x);
      y = fmaf(a.w2[(int64_t)u * a.c_z + c], nn[c], y);
    }
    hh[u] = x / (1.0f + expf(-x)) * y;
  }
  __builtin_amdgcn_wave_barrier();
  for (int c = lane; c < a.c_z; c += 64) {
    float t = 0.0f;
    for (int u = 0; u < a.hidden; ++u) t = fmaf(a.w3[(int64_t)c * a.hidden + u], hh[u], t);
    a.z_out[p * a.c_z + c] = z[c] + t;
  }
}

}  // namespace

size_t trans_prep_bytes() { return (size_t)kHt * kTileBytes + 2 * kCz * sizeof(float); }

hipError_t launch_transition(const TransArgs& a, hipStream_t st) {
  const int prep_threads = kPrepFragments + 2 * kCz;
  hipLaunchKernelGGL(trans_prep_kernel, dim3((prep_threads + 255) / 256), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n_groups = (a.n_pairs + kGroupPairs - 1) / kGroupPairs;
  const int64_t grid = n_groups < 256 ? n_groups : 256;  // one persistent workgroup per CU
  hipLaunchKernelGGL(trans_kernel, dim3((unsigned)grid), dim3(64 * kWaves), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_transition_gen(const TransGenArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(trans_gen_kernel, dim3((unsigned)((a.n_pairs + 3) / 4)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace dcp
