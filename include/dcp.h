/* dcp.h -- pair-biased, gated multi-head attention on one AMD MI355X (gfx950).
 *
 * The operation (paper: Design-CP, arXiv 2607.05439):
 *   Methods, "RFDiffusion 3 preliminaries and notation": inside every
 *   token-level attention block a learned projection of the pair track Z gives
 *   a per-head bias B that is added to the logits, softmax(Q K^T / sqrt(d) + B).
 *   Methods, "1D row-sharding", Eq. (cross_attn): a stripe of query rows
 *   attends to keys and values projected from the full single track S, with
 *   the bias drawn from the stripe's own rows of Z.
 *   Methods, "2D grid context parallelism", and Appendix "Q/K/V layout and the
 *   ring loop": keys are visited block by block and each block's partial
 *   result is folded into a running total with an online softmax.
 * Readings where the paper is silent: the projection is
 *   b[i,j,h] = sum_c W_b[h,c] LayerNorm(z[i,j,:])_c + b_b[h]
 * (biased variance, eps inside the square root, affine gamma/beta over c_z),
 * and the output is gated, out_i = sigmoid(W_g s_i) * attention_i.
 *
 * For query rows i in [q_row0, q_row0 + n_q) and heads h (flat index h*d + e):
 *   q_i = W_q s_i, k_j = W_k s_j, v_j = W_v s_j, g_i = sigmoid(W_g s_i),
 *   l[h,i,j] = q_{i,h} . k_{j,h} / sqrt(d) + b[i,j,h]   (-inf for a masked key),
 *   out[i - q_row0, h*d + e] = g_i[h*d+e] * sum_j softmax_j(l[h,i,:]) v_{j,h,e};
 *   a row whose keys are all masked gives 0.
 *
 * Conventions for every entry point:
 *  - Tensor pointers are DEVICE pointers owned by the caller; the descriptor
 *    structs are host memory read during the call only. The library never
 *    allocates or frees memory: scratch comes from `workspace`.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*, NULL =
 *    the null stream) and never synchronise. All arguments are validated on
 *    the host before anything is launched; a non-OK status means nothing was
 *    launched (DCP_ERR_HIP: a launch failed after validation) and
 *    dcp_last_error() describes it. No C++ exception crosses this interface.
 *  - Layouts are row-major and contiguous; weights are fp32 in nn.Linear layout
 *    [out_features, in_features].
 *  - NaN or Inf in unmasked inputs propagate to the outputs; masked keys' s and
 *    z are never read into the result.
 *  - Results are deterministic: the same call on the same inputs gives the
 *    same bits (no atomics, fixed reduction order).
 */
#ifndef DCP_H
#define DCP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { DCP_F32 = 0, DCP_BF16 = 1 } dcp_dtype;

enum {
  DCP_OK = 0,
  DCP_ERR_INVALID_ARGUMENT = -1, /* null/misaligned pointer, bad size or range      */
  DCP_ERR_UNSUPPORTED = -2,      /* shape/dtype combination not built (see below)  */
  DCP_ERR_WORKSPACE = -3,        /* workspace missing, misaligned or too small     */
  DCP_ERR_HIP = -4               /* a kernel launch failed                         */
};

typedef struct {
  int64_t n_tokens;  /* N: rows of s, number of keys, columns of z                */
  int32_t c_s;       /* single-track channels                                     */
  int32_t c_z;       /* pair-track channels                                       */
  int32_t n_heads;   /* H                                                         */
  int32_t head_dim;  /* d                                                         */
  int32_t act_dtype; /* dcp_dtype of s and z                                      */
  int32_t out_dtype; /* dcp_dtype of out                                          */
  float ln_eps;      /* LayerNorm epsilon (PyTorch default 1e-5), >= 0            */
} dcp_shape;

typedef struct {
  const float* w_q;      /* [H*d, c_s]                                            */
  const float* w_k;      /* [H*d, c_s]                                            */
  const float* w_v;      /* [H*d, c_s]                                            */
  const float* w_g;      /* [H*d, c_s]                                            */
  const float* w_b;      /* [H, c_z]                                              */
  const float* b_b;      /* [H] or NULL (= 0)                                     */
  const float* ln_gamma; /* [c_z] or NULL (= 1)                                   */
  const float* ln_beta;  /* [c_z] or NULL (= 0)                                   */
} dcp_weights;
/* On the fused bf16 path below (attention and dcp_bias_project), w_q, w_k,
 * w_v, w_g, w_b and ln_gamma (and, for dcp_bias_project, ln_beta) must be
 * 16-byte aligned (DCP_ERR_INVALID_ARGUMENT otherwise); the general fp32 path
 * needs 4-byte alignment only. */

/* Supported shapes. A fused MFMA path serves act_dtype = BF16 with c_z = 128,
 * H = 16, d = 24 and c_s a multiple of 32 (at most 4096). A general fp32 path
 * serves every other combination with c_z <= 256, H <= 16, d <= 64,
 * H*d <= 128 and c_s <= 4096, for either act_dtype. Anything else returns
 * DCP_ERR_UNSUPPORTED. */

/* Workspace bytes that dcp_pair_bias_attention needs for these arguments
 * (written to *bytes). Host-only; launches nothing. */
int dcp_workspace_size(const dcp_shape* shape, int64_t n_q, int32_t n_key_blocks, size_t* bytes);

/* The same query returning the size itself (Methods, "1D row-sharding",
 * Eq. (cross_attn): the scratch of one stripe call). Returns 0 and sets
 * dcp_last_error() when the arguments are invalid or the shape is not
 * supported; a valid call with n_q = 0 also returns 0 (no workspace needed)
 * and leaves dcp_last_error() empty. Host-only; launches nothing. */
size_t dcp_workspace_bytes(const dcp_shape* shape, int64_t n_q, int32_t n_key_blocks);

/* Pair-biased gated attention of the query stripe [q_row0, q_row0 + n_q)
 * against all N keys (Methods, Eq. (cross_attn)).
 *   s           [N, c_s] act_dtype, 16-byte aligned
 *   z_rows      [n_q, N, c_z] act_dtype: the stripe's rows of z, i.e.
 *               &z[q_row0, 0, 0] of a contiguous z[N, N, c_z]; 16-byte aligned
 *   key_mask    [N] uint8, 1 = attend, 0 = masked; NULL = every key attends
 *   n_q         0 <= n_q, q_row0 >= 0, q_row0 + n_q <= N (n_q = 0 is a no-op)
 *   n_key_blocks in [1, N]: keys are split into this many blocks by the
 *               paper's chunk rule (Appendix "Chunk distribution algorithm":
 *               block p has floor(N/P) + [p < N mod P] keys) and the blocks'
 *               partial states are merged in increasing order, as the ring
 *               steps of the paper's 2D scheme do. Any value gives the same
 *               result up to fp32 rounding order.
 *   out         [n_q, H*d] out_dtype, 16-byte aligned
 *   workspace   device scratch of at least dcp_workspace_size() bytes,
 *               256-byte aligned; contents on entry are ignored.
 * The gate and softmax statistics are fp32. On the fused bf16 path, z, s and
 * the projected q, k, v, the softmax weights and the bias weights enter the
 * matrix cores as bf16 (the bias weights as a bf16 hi+lo pair) with fp32
 * accumulation. */
int dcp_pair_bias_attention(const dcp_shape* shape, const dcp_weights* weights, const void* s,
                            const void* z_rows, const uint8_t* key_mask, int64_t q_row0, int64_t n_q,
                            int32_t n_key_blocks, void* out, void* workspace, size_t workspace_bytes,
                            void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call as dcp_pair_bias_attention, with the same arguments, kernels and
 * results, but its scratch comes from a library-owned device array of
 * DCP_NOALLOC_SCRATCH_BYTES on each GPU (held from the first call on that GPU
 * until the process ends) instead of a workspace argument. It allocates and
 * frees nothing and calls no allocating routine. A call whose
 * dcp_workspace_size() exceeds DCP_NOALLOC_SCRATCH_BYTES returns
 * DCP_ERR_WORKSPACE before anything is launched (split the query rows into
 * stripes). The array used is the current device's; `stream` must belong to
 * the current device (DCP_ERR_INVALID_ARGUMENT otherwise). Every call on one
 * GPU shares that array: calls that overlap in time on one GPU (different
 * streams, or host threads) race and give undefined results; calls ordered on
 * one stream do not. Nothing in the array needs clearing: every byte a call
 * reads is first written by the same call. */
#define DCP_NOALLOC_SCRATCH_BYTES (128u << 20) /* 128 MiB */
int dcp_pair_bias_attention_noalloc(const dcp_shape* shape, const dcp_weights* weights, const void* s,
                                    const void* z_rows, const uint8_t* key_mask, int64_t q_row0, int64_t n_q,
                                    int32_t n_key_blocks, void* out, void* stream);

/* One ring step (Appendix "Q/K/V layout and the ring loop": a query stripe
 * against the key block visiting this rank; the 2D scheme's inner loop): the
 * partial attention state of query rows [q_row0, q_row0 + n_q) over the keys
 * [k0, k1) only, for merging with dcp_block_merge. Arguments as for
 * dcp_pair_bias_attention, with k0, k1 in place of n_key_blocks and:
 *   m_out    [H, n_q] fp32: a reference logit in natural-log units, at least
 *            the largest logit of the row and head over the range (the fused
 *            path rounds it up to a whole number of base-2 units); -inf when
 *            the range holds no unmasked key
 *   l_out    [H, n_q] fp32: sum over the range of exp(logit - m)
 *   acc_out  [n_q, H, d] fp32: sum over the range of exp(logit - m) v_j
 *   gate_out [n_q, H*d] fp32 sigmoid(W_g s_i), or NULL
 * Merging the partials of ranges that cover [0, N) with gate_out as the gate
 * gives dcp_pair_bias_attention's output. Needs dcp_workspace_size(shape,
 * n_q, 1) bytes of workspace. 0 <= k0 <= k1 <= N; k0 = k1 gives the empty
 * state (-inf, 0, 0). The output buffers must not overlap the inputs or the
 * workspace. */
int dcp_pair_bias_attention_partial(const dcp_shape* shape, const dcp_weights* weights, const void* s,
                                    const void* z_rows, const uint8_t* key_mask, int64_t q_row0, int64_t n_q,
                                    int64_t k0, int64_t k1, float* m_out, float* l_out, float* acc_out,
                                    float* gate_out, void* workspace, size_t workspace_bytes, void* stream);

/* The pair bias alone (Methods, "RFDiffusion 3 preliminaries and notation":
 * B = f_B(Z)), materialised: bias_out[r, c, h] = sum_k W_b[h,k] LN(z_tile[r, c, :])_k + b_b[h]
 * including gamma, beta and b_b, for r < n_rows, c < n_cols. Pair (r, c) is
 * read at z_tile + (r*row_stride_elems + c*c_z) elements (row_stride_elems >=
 * n_cols*c_z; it is N*c_z for a tile of a full z). bias_out is fp32 [n_rows,
 * n_cols, H], contiguous and 16-byte aligned. Only w_b, b_b, ln_gamma and
 * ln_beta of `weights` are read; c_s, head_dim, out_dtype and n_tokens of
 * `shape` are ignored. Needs no workspace. n_rows = 0 or n_cols = 0 is a no-op. */
int dcp_bias_project(const dcp_shape* shape, const dcp_weights* weights, const void* z_tile, int64_t n_rows,
                     int64_t n_cols, int64_t row_stride_elems, float* bias_out, void* stream);

/* Online-softmax merge of partial attention states, in increasing part order
 * (Appendix "Q/K/V layout and the ring loop": each ring step's partial output
 * is merged into a running total; Related Work, "IO-efficient attention").
 * A partial over a key subset K_p holds m = max_{j in K_p} l_j (natural log
 * units), l = sum exp(l_j - m) and acc = sum exp(l_j - m) v_j; (-inf, 0, 0) is
 * the empty partial.
 *   m_parts, l_parts  [n_parts, H, n_rows] fp32
 *   acc_parts         [n_parts, n_rows, H, d] fp32
 *   m_out, l_out      [H, n_rows] fp32, or NULL
 *   acc_out           [n_rows, H, d] fp32 (unnormalised), or NULL
 *   gate              [n_rows, H*d] fp32 (already sigmoid), or NULL (= 1)
 *   out               [n_rows, H*d] out_dtype = gate * acc / l (0 where l = 0), or NULL
 * Limits: 1 <= n_parts, 1 <= H, 1 <= d, H*d <= 4096. n_rows = 0 is a no-op.
 * Output buffers must not overlap the inputs. */
int dcp_block_merge(int32_t n_parts, int64_t n_rows, int32_t n_heads, int32_t head_dim, const float* m_parts,
                    const float* l_parts, const float* acc_parts, float* m_out, float* l_out, float* acc_out,
                    const float* gate, void* out, int32_t out_dtype, void* stream);

/* ---------------------------------------------------------------------------
 * Sparse (kNN) pair-biased gated attention over atoms.
 *
 * Paper, Methods, "RFDiffusion 3 preliminaries and notation": atoms carry a
 * single track A[L, c_atom] and a pair track P[L, L, c_ap]; the atom-level
 * attention is not dense: every query atom sees only k neighbour atoms, whose
 * entries of P are gathered and projected per head into the bias.
 * Appendix "Distributed kNN for sparse atom attention": per ring step the
 * neighbour indices are filtered to the visited column block, K, V and the
 * bias are gathered there, and the logits are merged into the running softmax.
 * Readings as for the token path: b = Linear(LayerNorm(p)) over the c_ap
 * channels of one gathered pair, output gated by sigmoid(W_g a_i).
 *
 * For query atoms i = q_row0 + r, r < n_q, and slots t < k with neighbour
 * j_t = nbr[r, t] (a slot whose index is outside [0, L) is empty):
 *   b[r,t,h] = sum_c W_b[h,c] LayerNorm(P[i, j_t, :])_c + b_b[h],
 *   l[h,r,t] = (W_q a_i)_h . (W_k a_{j_t})_h / sqrt(d) + b[r,t,h]   (-inf if empty),
 *   out[r, h*d+e] = sigmoid(W_g a_i)[h*d+e] * sum_t softmax_t(l[h,r,:]) (W_v a_{j_t})_{h,e};
 *   a query whose slots are all empty gives 0. A neighbour listed twice is two keys.
 * ------------------------------------------------------------------------- */
typedef struct {
  int64_t n_atoms;    /* L: rows of a, neighbour index range                     */
  int32_t c_atom;     /* atom single-track channels                              */
  int32_t c_ap;       /* atom pair channels                                      */
  int32_t n_heads;    /* H                                                       */
  int32_t head_dim;   /* d                                                       */
  int32_t k;          /* neighbour slots per query atom                          */
  int32_t act_dtype;  /* dcp_dtype of a and p                                    */
  int32_t out_dtype;  /* dcp_dtype of out                                        */
  int32_t p_gathered; /* 0: p holds dense rows of P; 1: p holds gathered slices  */
  float ln_eps;       /* LayerNorm epsilon, >= 0                                 */
} dcp_sparse_shape;

/* Supported: H = 4, d = 32, c_ap = 16 (the paper's atom attention), k <= 256,
 * L <= 4,000,000, c_atom <= 4096 (a multiple of 32 when act_dtype = BF16).
 * Other shapes return DCP_ERR_UNSUPPORTED. */

/* Workspace bytes for dcp_sparse_pair_bias_attention (written to *bytes). Host-only. */
int dcp_sparse_workspace_size(const dcp_sparse_shape* shape, int64_t n_q, size_t* bytes);

/* Sparse pair-biased gated attention of the query atoms [q_row0, q_row0 + n_q).
 *   a           [L, c_atom] act_dtype, 16-byte aligned
 *   p           p_gathered = 0: [n_q, L, c_ap], the stripe's rows of P, i.e.
 *               &P[q_row0, 0, 0] of a contiguous P[L, L, c_ap];
 *               p_gathered = 1: [n_q, k, c_ap], P[i, nbr[r, t], :] already
 *               gathered (the paper's P_sparse; empty slots are not read);
 *               act_dtype, 16-byte aligned
 *   nbr         [n_q, k] int32 neighbour atom indices; -1 (or any index
 *               outside [0, L)) marks an empty slot; 4-byte aligned
 *   n_q         0 <= n_q, q_row0 >= 0, q_row0 + n_q <= L (n_q = 0 is a no-op)
 *   n_key_blocks in [1, L]: the atoms are split into this many column blocks
 *               by the paper's chunk rule, and each query's slots are
 *               processed block by block in increasing order, folded into a
 *               running softmax (the ring steps). Any value gives the same
 *               result up to fp32 rounding.
 *   out         [n_q, H*d] out_dtype, 16-byte aligned
 *   workspace   at least dcp_sparse_workspace_size() bytes, 256-byte aligned
 * Only w_q, w_k, w_v, w_g ([H*d, c_atom]), w_b ([H, c_ap]) and ln_gamma
 * ([c_ap] or NULL) of `weights` are read: ln_beta and b_b add a per-head
 * constant to every logit of a query and do not change the result. Softmax
 * statistics, weights and accumulation are fp32; with BF16 activations the
 * projected k and v are stored as bf16 and the projections run on the matrix
 * cores (weights as a bf16 hi+lo pair). */
int dcp_sparse_pair_bias_attention(const dcp_sparse_shape* shape, const dcp_weights* weights, const void* a,
                                   const void* p, const int32_t* nbr, int64_t q_row0, int64_t n_q,
                                   int32_t n_key_blocks, void* out, void* workspace, size_t workspace_bytes,
                                   void* stream);

/* ---------------------------------------------------------------------------
 * k nearest neighbours of atoms (Appendix "Distributed kNN for sparse atom
 * attention": each query atom keeps the k closest atoms; distances are taken
 * block by block, never as a whole [L, L] matrix, and the running top-k of each
 * query is merged with every block's candidates, the ring top-k combine;
 * Methods, "Atom-level kNN attention budget": k = 128, intra- and inter-chain
 * budgets).
 *
 * Order: squared Euclidean distance computed in fp32 as
 * ((dx*dx) + (dy*dy)) + (dz*dz), dx = x_q - x_c, every operation rounded to
 * fp32; ties go to the smaller candidate index. The result is therefore exact
 * and deterministic: it does not depend on blocking or on the visiting order.
 * NaN coordinates give an unspecified order.
 * ------------------------------------------------------------------------- */

/* The k nearest candidates of each query.
 *   x_q        [n_q, 3] fp32 query coordinates
 *   x_c        [n_c, 3] fp32 candidate coordinates (may be NULL when n_c = 0);
 *              candidate j has the global index c_index0 + j
 *              (c_index0 + n_c <= INT32_MAX)
 *   q_self0    when the queries are themselves candidates, the position in x_c
 *              of query 0 (then query r is candidate q_self0 + r); else -1.
 *              Only the visiting order depends on it, never the result.
 *   group_q, group_c  [n_q], [n_c] int32 group ids (chains), used when
 *              group_mode = 1 (same group only) or 2 (other groups only);
 *              may be NULL with group_mode = 0 (every candidate admissible)
 *   k          1 <= k <= 256
 *   idx_out    [n_q, k] int32 global indices, nearest first; -1 past the
 *              number of admissible candidates
 *   d2_out     [n_q, k] fp32 squared distances (+inf past the end), or NULL
 *   workspace  at least dcp_knn_workspace_size(n_c) bytes of device memory,
 *              256-byte aligned (may be NULL when n_c = 0): the candidates
 *              re-laid out and the bounding box of every 128 of them, written
 *              by this call; owned by the caller, contents undefined after
 * Device pointers, 4-byte aligned. n_q = 0 is a no-op. A workspace that is
 * missing, misaligned or too small returns DCP_ERR_WORKSPACE. */
int dcp_knn_topk(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, int64_t c_index0, int64_t q_self0,
                 const int32_t* group_q, const int32_t* group_c, int32_t group_mode, int32_t k, int32_t* idx_out,
                 float* d2_out, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes that dcp_knn_topk needs for n_c candidates (written to
 * *bytes): 16 per candidate plus 32 per 128 candidates. Host-only; launches
 * nothing. */
int dcp_knn_workspace_size(int64_t n_c, size_t* bytes);

/* The ring top-k combine: per row, the k smallest entries of the union of two
 * lists sorted as dcp_knn_topk returns them ([n_rows, k] each; index -1 =
 * empty). Equal entries in both lists are both kept (a's first). Outputs must
 * not overlap the inputs. */
int dcp_topk_merge(int64_t n_rows, int32_t k, const int32_t* idx_a, const float* d2_a, const int32_t* idx_b,
                   const float* d2_b, int32_t* idx_out, float* d2_out, void* stream);

/* ---------------------------------------------------------------------------
 * Pair transition (Appendix "Manual SwiGLU decomposition"): the SwiGLU
 * feed-forward update of the pair track with its residual, per pair,
 *   N = LayerNorm(z),  z <- z + W3 (SiLU(W1 N) * W2 N),  SiLU(a) = a / (1 + e^-a),
 * W1, W2: [hidden, c_z], W3: [c_z, hidden] (fp32, nn.Linear layout, no bias);
 * LayerNorm over c_z with optional gamma, beta ([c_z] fp32, NULL = 1 / 0),
 * biased variance, eps inside the square root.
 * ------------------------------------------------------------------------- */

/* Workspace bytes for dcp_pair_transition (written to *bytes). Host-only. */
int dcp_transition_workspace_size(int32_t c_z, int32_t hidden, int32_t act_dtype, size_t* bytes);

/* The transition of n_pairs consecutive pairs z[n_pairs, c_z] (any stripe of
 * rows of a contiguous pair tensor). z_out may equal z_in (in place) or must
 * not overlap it; both 16-byte aligned, act_dtype.
 * act_dtype = BF16: c_z = 128 and hidden = 512 only; the weights (gamma folded
 * into W1 and W2, beta into per-unit biases), the normalised pair vector and
 * SiLU(A) * B enter the matrix cores as bf16 with fp32 accumulation; the
 * result is rounded to bf16. Needs dcp_transition_workspace_size() bytes of
 * workspace (256-byte aligned; prepared weights, rewritten on every call).
 * act_dtype = F32: c_z <= 256, hidden <= 1024, fp32 throughout, no workspace
 * (workspace may be NULL). n_pairs = 0 is a no-op. */
int dcp_pair_transition(int64_t n_pairs, int32_t c_z, int32_t hidden, int32_t act_dtype, float ln_eps,
                        const float* w1, const float* w2, const float* w3, const float* ln_gamma,
                        const float* ln_beta, const void* z_in, void* z_out, void* workspace, size_t workspace_bytes,
                        void* stream);

/* ---------------------------------------------------------------------------
 * Atom -> token mean pooling (Appendix "Non-determinism guard" and the 2D
 * pooling boundary): out[t, :] = mean of a[i, :] over the atoms i with
 * tok_idx[i] = t; a token without atoms gives 0; an index outside
 * [0, n_tokens) belongs to no token.
 *
 * Deterministic for any index pattern and on any device: features are summed
 * as 64-bit fixed-point integers (value * 2^32, rounded to nearest), whose
 * addition does not depend on order, then scaled by 2^-32 and by the count's
 * reciprocal (1/count rounded to fp64) in fp64 and rounded to out_dtype, so
 * any permutation of the atoms gives the same bits. Each feature is clamped to
 * |x| <= 2^30 and each token's sum must stay below 2^31 in magnitude; the
 * absolute rounding of a feature is at most 2^-33. NaN features give
 * unspecified values for their token.
 *
 * Atoms ordered by token (tok_idx non-decreasing, the model's layout) take a
 * path without atomics that reads each feature once; the order is checked on
 * the device, and any other order takes a path with 64-bit integer atomics.
 * ------------------------------------------------------------------------- */

/* Workspace bytes for dcp_scatter_mean (written to *bytes). Host-only. */
int dcp_scatter_mean_workspace_size(int64_t n_tokens, int32_t c, size_t* bytes);

/*   a        [n_atoms, c] in_dtype (may be NULL when n_atoms = 0)
 *   tok_idx  [n_atoms] int32 token of each atom (any order)
 *   out      [n_tokens, c] out_dtype
 *   c        1 <= c <= 512
 * Device pointers aligned to their element size; workspace of at least
 * dcp_scatter_mean_workspace_size() bytes, 256-byte aligned. n_tokens = 0 is a
 * no-op. */
int dcp_scatter_mean(int64_t n_atoms, int64_t n_tokens, int32_t c, int32_t in_dtype, int32_t out_dtype, const void* a,
                     const int32_t* tok_idx, void* out, void* workspace, size_t workspace_bytes, void* stream);

/* Optional timing hook: when both are non-NULL hipEvent_t handles, the calling
 * thread's next dcp_pair_bias_attention, dcp_sparse_pair_bias_attention,
 * dcp_knn_topk, dcp_pair_transition and dcp_scatter_mean calls record
 * `start` just before and
 * `stop` just after the main kernel (after any projections; around the
 * weight preparation and the transition kernel of a transition; around all
 * kernels of a pooling), on that call's stream. Pass NULL, NULL to clear.
 * Host-only. */
int dcp_set_timing_events(void* start_event, void* stop_event);

/* Message for the calling thread's last non-OK status ("" if none). */
const char* dcp_last_error(void);

/* Library version string. */
const char* dcp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DCP_H */
