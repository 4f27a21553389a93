// Internal launch interface between the C-ABI layer (dcp_api.hip) and the
// kernels. Not installed; the public interface is include/dcp.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcp {

// Shape of the fused MFMA path.
constexpr int kFastCz = 128;   // pair channels
constexpr int kFastH = 16;     // heads
constexpr int kFastD = 24;     // head dim
// Logits of the fused path are in base-2 units plus this offset inside the
// kernel (exact power-of-two rescaling); its partial maxima are written
// without it
constexpr float kFastShift = 192.0f;
constexpr int kFastDp = 32;    // head dim padded to the MFMA k width
constexpr int kTileQ = 16;     // query rows per wave
constexpr int kTileK = 16;     // keys per tile
// 16 rows of z must be addressable with 31-bit byte offsets: 16 * N * 256 < 2^31
constexpr int64_t kFastMaxTokens = 500000;

// Limits of the general fp32 path.
constexpr int kGenMaxCz = 256;
constexpr int kGenMaxH = 16;
constexpr int kGenMaxHD = 128;
constexpr int kGenMaxD = 64;
constexpr int kMaxCs = 4096;

// The paper's chunk rule (Appendix "Chunk distribution algorithm"): part p of
// `total` items over `parts` parts has floor(total/parts) items, plus one when
// p < total mod parts, and starts at p*floor(total/parts) + min(p, total mod parts).
__host__ __device__ inline void chunk_of(int64_t total, int64_t parts, int64_t p, int64_t* size, int64_t* start) {
  const int64_t q = total / parts, r = total % parts;
  *size = q + (p < r ? 1 : 0);
  *start = p * q + (p < r ? p : r);
}

// Key range of internal part `part` = (block b, segment s): the keys are split
// into n_kb blocks by the chunk rule, and each block into n_seg segments by the
// same rule. Parts are ordered block-major, so merging them in index order
// merges the blocks in increasing order.
__host__ __device__ inline void part_range(int64_t n_tok, int n_kb, int n_seg, int part, int64_t* start,
                                           int64_t* end) {
  const int b = part / n_seg, s = part % n_seg;
  int64_t bs, b0, ss, s0;
  chunk_of(n_tok, n_kb, b, &bs, &b0);
  chunk_of(bs, n_seg, s, &ss, &s0);
  *start = b0 + s0;
  *end = b0 + s0 + ss;
}

struct FastProjArgs {
  const uint16_t* s;  // [N, c_s] bf16
  const float *w_q, *w_k, *w_v, *w_g;
  const uint8_t* mask;  // [N] or null
  int64_t n_tok, q_row0, n_q, nq_pad, n_pad;
  int32_t c_s;
  uint16_t* q;   // [H][nq_pad][32] bf16, scaled by log2(e)/sqrt(d)
  uint16_t* k;   // [H][n_pad][32] bf16
  uint16_t* vt;  // [H][n_pad/16][64][2][4] bf16: V^T tiles (lane, M-tile) with a row of ones at e = 24
  float* g;      // [n_q][H*d] fp32, sigmoid applied
  uint32_t* tile_valid;  // [n_pad/16]: bit i = key 16t+i exists and is not masked
  void* w_split;         // fast_proj_split_bytes(c_s): the weights as bf16 hi + lo matrix-core operands
};

struct FastAttnArgs {
  const uint16_t* z;  // [n_q][N][128] bf16
  const uint8_t* mask;
  const float *w_b, *gamma;
  const uint16_t *q, *k, *vt;
  const uint32_t* tile_valid;
  int64_t n_tok, n_q, nq_pad, n_pad;
  int64_t k_lo, k_len;  // keys [k_lo, k_lo + k_len), split into n_kb blocks x n_seg segments
  int32_t n_kb, n_seg;
  float eps;
  float *m_parts, *l_parts, *acc_parts;  // [P][H][n_q], [P][H][n_q], [P][n_q][H][d]
  int32_t xcd_order;                     // set by the launcher: workgroup numbering (attn_kernel)
};

struct FastBiasArgs {
  const uint16_t* z;
  const float *w_b, *b_b, *gamma, *beta;
  int64_t n_rows, n_cols, row_stride;
  int32_t cols_per_wave;
  float eps;
  float* out;  // [n_rows][n_cols][16]
};

struct GenProjArgs {
  const void* s;
  int32_t s_bf16;
  const float *w_q, *w_k, *w_v, *w_g;
  int64_t n_tok, q_row0, n_q;
  int32_t c_s, hd;
  float *q, *k, *v, *g;  // q, g: [n_q][hd]; k, v: [N][hd]; g holds the sigmoid
};

struct GenAttnArgs {
  const void* z;
  int32_t z_bf16;
  const uint8_t* mask;
  const float *w_b, *gamma;
  const float *q, *k, *v;
  int64_t n_tok, n_q;
  int64_t k_lo, k_len;  // keys [k_lo, k_lo + k_len), split into n_kb blocks
  int32_t c_z, n_heads, head_dim, n_kb;
  float eps;
  float *m_parts, *l_parts, *acc_parts;
};

struct GenBiasArgs {
  const void* z;
  int32_t z_bf16;
  const float *w_b, *b_b, *gamma, *beta;
  int64_t n_rows, n_cols, row_stride;
  int32_t c_z, n_heads;
  float eps;
  float* out;
};

struct MergeArgs {
  int32_t n_parts, n_heads, head_dim;
  int64_t n_rows;
  const float *m, *l, *acc, *gate;
  float *m_out, *l_out, *acc_out;
  void* out;
  int32_t out_bf16;
  int32_t log2_units;  // 1: m is in base-2 units with integer differences (the fused path)
  int32_t m_natural;   // with log2_units: write m_out in natural-log units
};

// Sparse (kNN) atom attention: the paper's atom-attention shape (4 heads of
// 32, 16 pair channels), up to 256 neighbour slots per query.
constexpr int kSparseH = 4;
constexpr int kSparseD = 32;
constexpr int kSparseCap = 16;
constexpr int kSparseMaxK = 256;
// Neighbour indices are packed with their slot number into 32 bits (24 + 8),
// and an fp32 K or V array of this many atoms stays below 2^31 bytes.
constexpr int64_t kSparseMaxAtoms = 4000000;

struct SparseProjArgs {
  const uint16_t* a;  // [L, c_atom] bf16
  const float *w_q, *w_k, *w_v, *w_g;
  int64_t n_atoms, q_row0, n_q;
  int32_t c_atom;
  float *q, *g;       // [n_q][128] fp32 (g after the sigmoid)
  uint16_t *k, *v;    // [L][128] bf16
};

struct SparseAttnArgs {
  const void* p;          // pair rows of the query stripe (dense [n_q][L][16] or gathered [n_q][k][16])
  const int32_t* nbr;     // [n_q][k]
  const float *w_b, *gamma;
  const float *q, *g;     // [n_q][128] fp32
  const void *k, *v;      // [L][128] in the activation dtype
  int64_t n_atoms, n_q;
  int64_t p_row_elems;    // elements per query row of p
  int32_t k_slots, n_kb, p_gathered, out_bf16;
  float eps;
  void* out;              // [n_q][128]
};

// k nearest neighbours: up to 256 per query; candidate indices fit in int32.
constexpr int kKnnMaxK = 256;

struct KnnArgs {
  const float* x_q;       // [n_q][3]
  const float* x_c;       // [n_c][3]
  const int32_t *group_q, *group_c;
  int64_t n_q, n_c, c_index0, q_self0;
  int32_t k, group_mode;
  int32_t* idx_out;       // [n_q][k]
  float* d2_out;          // [n_q][k] or null
  void *cand, *box;       // workspace: [n_c] float4 candidates, [ceil(n_c / 128)][2] float4 boxes
};

struct TopkMergeArgs {
  int64_t n_rows;
  int32_t k;
  const int32_t *idx_a, *idx_b;
  const float *d2_a, *d2_b;
  int32_t* idx_out;
  float* d2_out;
};

// Pair transition: the matrix-core path serves c_z = 128 with a 4x expansion;
// the fp32 path c_z <= 256 and hidden <= 1024.
constexpr int kTransCz = 128;
constexpr int kTransHidden = 512;
constexpr int kTransGenMaxHidden = 1024;

struct TransArgs {
  int64_t n_pairs;
  const float *w1, *w2, *w3, *gamma, *beta;
  const void* z_in;    // [n_pairs][128] bf16
  void* z_out;         // may equal z_in
  void* w_prep;        // operand tiles (trans_prep_bytes(): tiles, then gamma and beta)
  float* gb_prep;      // [2][128] gamma, beta inside w_prep
  float eps;
};

struct TransGenArgs {
  int64_t n_pairs;
  int32_t c_z, hidden;
  const float *w1, *w2, *w3, *gamma, *beta;
  const float* z_in;
  float* z_out;        // may equal z_in
  float eps;
};

size_t trans_prep_bytes();

// Atom -> token mean: up to 512 channels.
constexpr int kScatterMaxC = 512;
constexpr int kScatterFlags = 256;  // most order-check flags of one pooling call

struct ScatterArgs {
  int64_t n_atoms, n_tokens;
  int32_t c, a_bf16, out_bf16;
  const void* a;          // [n_atoms][c]
  const int32_t* tok_idx; // [n_atoms]
  int64_t* acc;           // [n_tokens][c] fixed-point sums (workspace)
  uint32_t* cnt;          // [n_tokens] (workspace)
  void* out;              // [n_tokens][c]
  int32_t* flags;         // [kScatterFlags] order-check flags (workspace); NULL: general path only
  int32_t n_flags;        // flags written by this call (set by the launcher)
  int64_t* plan;          // [n_tokens][2] first atom and one past the last of each token (workspace)
};

size_t fast_proj_split_bytes(int32_t c_s);
hipError_t launch_fast_proj(const FastProjArgs& a, hipStream_t st);
hipError_t launch_fast_attn(const FastAttnArgs& a, hipStream_t st);
hipError_t launch_fast_bias(const FastBiasArgs& a, hipStream_t st);
hipError_t launch_gen_proj(const GenProjArgs& a, hipStream_t st);
hipError_t launch_gen_attn(const GenAttnArgs& a, hipStream_t st);
hipError_t launch_gen_bias(const GenBiasArgs& a, hipStream_t st);
hipError_t launch_merge(const MergeArgs& a, hipStream_t st);
hipError_t launch_sparse_proj(const SparseProjArgs& a, hipStream_t st);
hipError_t launch_sparse_attn(const SparseAttnArgs& a, bool bf16, hipStream_t st);
size_t knn_workspace_bytes(int64_t n_c, size_t* box_offset);
hipError_t launch_knn(const KnnArgs& a, hipStream_t st);
hipError_t launch_topk_merge(const TopkMergeArgs& a, hipStream_t st);
hipError_t launch_transition(const TransArgs& a, hipStream_t st);
hipError_t launch_transition_gen(const TransGenArgs& a, hipStream_t st);
hipError_t launch_scatter_mean(const ScatterArgs& a, hipStream_t st);
int scatter_order_flags(int64_t n_atoms);  // plan workgroups (one flag each) for n_atoms (<= kScatterFlags)

}  // namespace dcp
