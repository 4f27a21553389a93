/* oracle.c -- plain fp64 CPU oracle for pair-biased, gated multi-head attention.
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may load or call this library. It shares no code, header,
 * table or helper with the GPU path, and the GPU path never calls it.
 *
 * What it computes (every formula is evaluated exactly as written, in fp64, on
 * the exact input values; bf16 and fp32 inputs convert to fp64 without error):
 *
 *   Paper, Methods, "RFDiffusion 3 preliminaries and notation": every
 *   token-level attention block adds a per-head pair bias B = f_B(Z), a
 *   learned projection of the pair track, to the logits before the softmax,
 *   softmax(Q K^T / sqrt(d) + B).
 *   Paper, Methods, "1D row-sharding", Eq. (cross_attn): a stripe of query
 *   rows attends to keys and values projected from the full single track S,
 *   with the bias taken from the stripe's own rows of Z.
 *   The projection f_B is read as Linear(LayerNorm(z)) over the c_z channels
 *   of one pair (biased variance, eps inside the square root, affine gamma and
 *   beta), and the output is gated elementwise by sigmoid(W_g s_i); the paper
 *   states neither, so both are readings.
 *
 *   q_i = W_q s_i, k_j = W_k s_j, v_j = W_v s_j, g_i = sigmoid(W_g s_i), each
 *   reshaped [H, d] with flat index h*d + e;
 *   b[i,j,h] = sum_c W_b[h,c] (gamma_c (z[i,j,c] - mu) / sqrt(var + eps) + beta_c) + b_b[h];
 *   l[h,i,j] = q_{i,h} . k_{j,h} / sqrt(d) + b[i,j,h], or -inf for a masked key;
 *   out[i, h*d+e] = g_i[h*d+e] * sum_j softmax_j(l[h,i,:]) v_{j,h,e}; a row
 *   with every key masked gives 0.
 *
 *   Blocked form (self-tests only), Paper, Methods, "2D grid context
 *   parallelism" and Appendix "Q/K/V layout and the ring loop": keys are split
 *   into blocks by the chunk rule of Appendix "Chunk distribution algorithm";
 *   each block yields a partial state (m, l, acc) with m the block's maximum
 *   logit, l = sum exp(l - m) and acc = sum exp(l - m) v, and the partials are
 *   folded one by one, in increasing block order, into a running total with the
 *   online-softmax rule (Related Work, "IO-efficient attention": running
 *   softmax statistics).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Appendix "Chunk distribution algorithm": part p of `total` items over
 * `parts` parts has floor(total/parts) items plus one when p < total mod parts,
 * and starts at p*floor(total/parts) + min(p, total mod parts). */
void oracle_chunk(int64_t total, int64_t parts, int64_t p, int64_t* size, int64_t* start) {
  const int64_t q = total / parts, r = total % parts;
  *size = q + (p < r ? 1 : 0);
  *start = p * q + (p < r ? p : r);
}

/* Input decoding: element idx of a buffer holding fp32 (dtype 0) or bf16 (dtype 1). */
static double load_elem(const void* buf, int dtype, int64_t idx) {
  if (dtype == 0) return (double)((const float*)buf)[idx];
  uint32_t bits = (uint32_t)((const uint16_t*)buf)[idx] << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* y[t, o] = sum_c w[o, c] x[t, c]  (nn.Linear layout, no bias). */
void oracle_linear(int64_t n_tok, int n_in, int n_out, const double* x, const double* w, double* y) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n_tok; ++t)
    for (int o = 0; o < n_out; ++o) {
      double acc = 0.0;
      for (int c = 0; c < n_in; ++c) acc += w[(int64_t)o * n_in + c] * x[t * n_in + c];
      y[t * n_out + o] = acc;
    }
}

/* LayerNorm of one pair's c_z channels, then the linear map to H heads. */
static void pair_bias(const void* z, int dtype, int64_t off, int c_z, int n_heads, const double* w_b,
                      const double* b_b, const double* gamma, const double* beta, double eps, double* ln,
                      double* b_out) {
  double mu = 0.0;
  for (int c = 0; c < c_z; ++c) mu += load_elem(z, dtype, off + c);
  mu /= c_z;
  double var = 0.0;
  for (int c = 0; c < c_z; ++c) {
    const double t = load_elem(z, dtype, off + c) - mu;
    var += t * t;
  }
  var /= c_z;
  const double inv = 1.0 / sqrt(var + eps);
  for (int c = 0; c < c_z; ++c) {
    const double xhat = (load_elem(z, dtype, off + c) - mu) * inv;
    ln[c] = (gamma ? gamma[c] : 1.0) * xhat + (beta ? beta[c] : 0.0);
  }
  for (int h = 0; h < n_heads; ++h) {
    double acc = 0.0;
    for (int c = 0; c < c_z; ++c) acc += w_b[(int64_t)h * c_z + c] * ln[c];
    b_out[h] = acc + (b_b ? b_b[h] : 0.0);
  }
}

/* bias[r, c, h] for pairs z[r*row_stride + c*c_z + ...], r < n_rows, c < n_cols. */
int oracle_bias(int64_t n_rows, int64_t n_cols, int c_z, int n_heads, const void* z, int dtype,
                int64_t row_stride, const double* w_b, const double* b_b, const double* gamma,
                const double* beta, double eps, double* out) {
  if (!z || !w_b || !out || c_z <= 0 || n_heads <= 0) return -1;
#pragma omp parallel
  {
    double* ln = (double*)malloc(sizeof(double) * (size_t)c_z);
#pragma omp for schedule(static)
    for (int64_t r = 0; r < n_rows; ++r)
      for (int64_t c = 0; c < n_cols; ++c)
        pair_bias(z, dtype, r * row_stride + c * c_z, c_z, n_heads, w_b, b_b, gamma, beta, eps, ln,
                  out + (r * n_cols + c) * n_heads);
    free(ln);
  }
  return 0;
}

/* Logits of one query row for head h over keys [k0, k1); masked keys get -inf. */
static void row_logits(int64_t k0, int64_t k1, int n_heads, int d, int h, const double* q_row,
                       const double* k, const double* bias_row, const uint8_t* mask, double* logit) {
  const int hd = n_heads * d;
  const double scale = 1.0 / sqrt((double)d);
  for (int64_t j = k0; j < k1; ++j) {
    if (mask && !mask[j]) {
      logit[j - k0] = -INFINITY;
      continue;
    }
    double dot = 0.0;
    for (int e = 0; e < d; ++e) dot += q_row[h * d + e] * k[j * hd + h * d + e];
    logit[j - k0] = dot * scale + bias_row[j * n_heads + h];
  }
}

/* Plain softmax attention of one query row against all n_tok keys, then the gate. */
static void attend_row(int64_t n_tok, int n_heads, int d, const double* q_row, const double* k,
                       const double* v, const double* bias_row, const uint8_t* mask, const double* g_row,
                       double* logit, double* out_row) {
  for (int h = 0; h < n_heads; ++h) {
    row_logits(0, n_tok, n_heads, d, h, q_row, k, bias_row, mask, logit);
    double mx = -INFINITY;
    for (int64_t j = 0; j < n_tok; ++j)
      if (logit[j] > mx) mx = logit[j];
    for (int e = 0; e < d; ++e) out_row[h * d + e] = 0.0;
    if (mx == -INFINITY) continue; /* every key masked: output 0 */
    double den = 0.0;
    for (int64_t j = 0; j < n_tok; ++j) den += exp(logit[j] - mx);
    for (int e = 0; e < d; ++e) {
      double num = 0.0;
      for (int64_t j = 0; j < n_tok; ++j)
        num += exp(logit[j] - mx) * v[j * (int64_t)n_heads * d + h * d + e];
      out_row[h * d + e] = g_row[h * d + e] * (num / den);
    }
  }
}

/* Attention given every ingredient: q, g_pre (pre-sigmoid gate) [n_rows, H*d],
 * k, v [n_tok, H*d], bias [n_rows, n_tok, H], mask [n_tok] or NULL. */
int oracle_attend(int64_t n_rows, int64_t n_tok, int n_heads, int d, const double* q, const double* k,
                  const double* v, const double* g_pre, const double* bias, const uint8_t* mask,
                  double* out) {
  if (!q || !k || !v || !g_pre || !bias || !out) return -1;
  const int hd = n_heads * d;
#pragma omp parallel
  {
    double* logit = (double*)malloc(sizeof(double) * (size_t)n_tok);
    double* g_row = (double*)malloc(sizeof(double) * (size_t)hd);
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; ++r) {
      for (int x = 0; x < hd; ++x) g_row[x] = sigmoid(g_pre[r * hd + x]);
      attend_row(n_tok, n_heads, d, q + r * hd, k, v, bias + r * n_tok * n_heads, mask, g_row, logit,
                 out + r * hd);
    }
    free(logit);
    free(g_row);
  }
  return 0;
}

/* Partial state of one query row over keys [k0, k1): m[h], l[h], acc[h*d+e]. */
static void partial_row(int64_t k0, int64_t k1, int n_heads, int d, const double* q_row, const double* k,
                        const double* v, const double* bias_row, const uint8_t* mask, double* logit,
                        double* m, double* l, double* acc) {
  for (int h = 0; h < n_heads; ++h) {
    row_logits(k0, k1, n_heads, d, h, q_row, k, bias_row, mask, logit);
    double mx = -INFINITY;
    for (int64_t j = 0; j < k1 - k0; ++j)
      if (logit[j] > mx) mx = logit[j];
    m[h] = mx;
    l[h] = 0.0;
    for (int e = 0; e < d; ++e) acc[h * d + e] = 0.0;
    if (mx == -INFINITY) continue;
    for (int64_t j = 0; j < k1 - k0; ++j) {
      const double w = exp(logit[j] - mx);
      l[h] += w;
      for (int e = 0; e < d; ++e) acc[h * d + e] += w * v[(k0 + j) * (int64_t)n_heads * d + h * d + e];
    }
  }
}

/* Online-softmax fold of one partial (mb, lb, accb) into the running total (m, l, acc). */
static void fold(int d, double* m, double* l, double* acc, double mb, double lb, const double* accb) {
  if (mb == -INFINITY) return; /* empty partial: the identity */
  if (*m == -INFINITY) {
    *m = mb;
    *l = lb;
    for (int e = 0; e < d; ++e) acc[e] = accb[e];
    return;
  }
  const double mn = mb > *m ? mb : *m;
  const double a = exp(*m - mn), b = exp(mb - mn);
  *l = a * *l + b * lb;
  for (int e = 0; e < d; ++e) acc[e] = a * acc[e] + b * accb[e];
  *m = mn;
}

/* Merge n_parts partial states, in increasing part order.
 * m, l: [n_parts, H, n_rows]; acc: [n_parts, n_rows, H, d]; gate: [n_rows, H*d] post-sigmoid or NULL.
 * Outputs (each may be NULL): m_out, l_out [H, n_rows]; acc_out [n_rows, H, d];
 * out [n_rows, H*d] = gate * acc / l (0 where l == 0). */
int oracle_merge(int n_parts, int64_t n_rows, int n_heads, int d, const double* m, const double* l,
                 const double* acc, const double* gate, double* m_out, double* l_out, double* acc_out,
                 double* out) {
  if (n_parts < 1 || !m || !l || !acc) return -1;
  const int hd = n_heads * d;
#pragma omp parallel
  {
    double* run = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(static)
    for (int64_t r = 0; r < n_rows; ++r)
      for (int h = 0; h < n_heads; ++h) {
        double rm = -INFINITY, rl = 0.0;
        for (int e = 0; e < d; ++e) run[e] = 0.0;
        for (int p = 0; p < n_parts; ++p)
          fold(d, &rm, &rl, run, m[((int64_t)p * n_heads + h) * n_rows + r], l[((int64_t)p * n_heads + h) * n_rows + r],
               acc + (((int64_t)p * n_rows + r) * n_heads + h) * d);
        if (m_out) m_out[(int64_t)h * n_rows + r] = rm;
        if (l_out) l_out[(int64_t)h * n_rows + r] = rl;
        for (int e = 0; e < d; ++e) {
          if (acc_out) acc_out[(r * n_heads + h) * d + e] = run[e];
          if (out) out[r * hd + h * d + e] = rl > 0.0 ? (gate ? gate[r * hd + h * d + e] : 1.0) * run[e] / rl : 0.0;
        }
      }
    free(run);
  }
  return 0;
}

/* The whole definition for the query tokens rows[0..n_rows): projections, LN
 * bias from each row's z (z_rows[r] = z[rows[r], :, :]), attention, gate.
 * s [n_tok, c_s]; weights fp64 in nn.Linear layout; gamma, beta, b_b may be NULL.
 * n_blocks == 1: the plain softmax; n_blocks > 1: the blocked form, and the
 * per-block partials are returned when m_parts/l_parts/acc_parts are non-NULL
 * (layout as in oracle_merge, with n_rows rows). */
int oracle_attention(int64_t n_tok, int c_s, int c_z, int n_heads, int d, const double* s, const void* z_rows,
                     int z_dtype, const int64_t* rows, int64_t n_rows, const uint8_t* mask, const double* w_q,
                     const double* w_k, const double* w_v, const double* w_g, const double* w_b,
                     const double* b_b, const double* gamma, const double* beta, double eps, int n_blocks,
                     double* out, double* m_parts, double* l_parts, double* acc_parts) {
  if (!s || !z_rows || !rows || !w_q || !w_k || !w_v || !w_g || !w_b || !out) return -1;
  if (n_tok <= 0 || n_rows < 0 || n_blocks < 1 || n_blocks > n_tok) return -1;
  const int hd = n_heads * d;
  double* k = (double*)malloc(sizeof(double) * (size_t)(n_tok * hd));
  double* v = (double*)malloc(sizeof(double) * (size_t)(n_tok * hd));
  double* sq = (double*)malloc(sizeof(double) * (size_t)((n_rows ? n_rows : 1) * c_s));
  double* q = (double*)malloc(sizeof(double) * (size_t)((n_rows ? n_rows : 1) * hd));
  double* gp = (double*)malloc(sizeof(double) * (size_t)((n_rows ? n_rows : 1) * hd));
  for (int64_t r = 0; r < n_rows; ++r) memcpy(sq + r * c_s, s + rows[r] * c_s, sizeof(double) * (size_t)c_s);
  oracle_linear(n_tok, c_s, hd, s, w_k, k);
  oracle_linear(n_tok, c_s, hd, s, w_v, v);
  oracle_linear(n_rows, c_s, hd, sq, w_q, q);
  oracle_linear(n_rows, c_s, hd, sq, w_g, gp);
  double* pm = m_parts ? m_parts : (n_blocks > 1 ? (double*)malloc(sizeof(double) * (size_t)(n_blocks * n_heads * n_rows)) : NULL);
  double* pl = l_parts ? l_parts : (n_blocks > 1 ? (double*)malloc(sizeof(double) * (size_t)(n_blocks * n_heads * n_rows)) : NULL);
  double* pa = acc_parts ? acc_parts : (n_blocks > 1 ? (double*)malloc(sizeof(double) * (size_t)(n_blocks * n_rows * hd)) : NULL);
#pragma omp parallel
  {
    double* bias_row = (double*)malloc(sizeof(double) * (size_t)(n_tok * n_heads));
    double* logit = (double*)malloc(sizeof(double) * (size_t)n_tok);
    double* ln = (double*)malloc(sizeof(double) * (size_t)c_z);
    double* g_row = (double*)malloc(sizeof(double) * (size_t)hd);
    double* bm = (double*)malloc(sizeof(double) * (size_t)n_heads);
    double* bl = (double*)malloc(sizeof(double) * (size_t)n_heads);
    double* ba = (double*)malloc(sizeof(double) * (size_t)hd);
#pragma omp for schedule(dynamic, 1)
    for (int64_t r = 0; r < n_rows; ++r) {
      const int64_t zoff = r * n_tok * (int64_t)c_z;
      for (int64_t j = 0; j < n_tok; ++j)
        pair_bias(z_rows, z_dtype, zoff + j * c_z, c_z, n_heads, w_b, b_b, gamma, beta, eps, ln,
                  bias_row + j * n_heads);
      for (int x = 0; x < hd; ++x) g_row[x] = sigmoid(gp[r * hd + x]);
      if (n_blocks == 1) {
        attend_row(n_tok, n_heads, d, q + r * hd, k, v, bias_row, mask, g_row, logit, out + r * hd);
        continue;
      }
      for (int b = 0; b < n_blocks; ++b) {
        int64_t size, start;
        oracle_chunk(n_tok, n_blocks, b, &size, &start);
        partial_row(start, start + size, n_heads, d, q + r * hd, k, v, bias_row, mask, logit, bm, bl, ba);
        for (int h = 0; h < n_heads; ++h) {
          pm[((int64_t)b * n_heads + h) * n_rows + r] = bm[h];
          pl[((int64_t)b * n_heads + h) * n_rows + r] = bl[h];
          for (int e = 0; e < d; ++e) pa[(((int64_t)b * n_rows + r) * n_heads + h) * d + e] = ba[h * d + e];
        }
      }
    }
    free(bias_row);
    free(logit);
    free(ln);
    free(g_row);
    free(bm);
    free(bl);
    free(ba);
  }
  if (n_blocks > 1) {
    double* gate = (double*)malloc(sizeof(double) * (size_t)((n_rows ? n_rows : 1) * hd));
    for (int64_t x = 0; x < n_rows * hd; ++x) gate[x] = sigmoid(gp[x]);
    oracle_merge(n_blocks, n_rows, n_heads, d, pm, pl, pa, gate, NULL, NULL, NULL, out);
    free(gate);
    if (!m_parts) free(pm);
    if (!l_parts) free(pl);
    if (!acc_parts) free(pa);
  }
  free(k);
  free(v);
  free(sq);
  free(q);
  free(gp);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Sparse (kNN) pair-biased atom attention.
 *
 * Paper, Methods, "RFDiffusion 3 preliminaries and notation": the atom-level
 * attention is not dense; every query atom looks at a fixed number k of
 * neighbour atoms only, and the bias for those k keys comes from the matching
 * entries of the atom pair track P, gathered and projected per head. Appendix "Distributed kNN for sparse atom attention":
 * at each ring step the indices are filtered to the visited column block, K, V
 * and B are gathered there, and the logits are merged into the running
 * softmax. Readings as for the token path (LayerNorm over the c_ap channels of
 * one gathered pair, sigmoid gate); every neighbour slot is one key, and a slot
 * whose index is not an atom (-1, or any value outside [0, L)) is empty.
 *
 *   q_i = W_q a_i, k_j = W_k a_j, v_j = W_v a_j, g_i = sigmoid(W_g a_i)
 *   b[i,t,h] = sum_c W_b[h,c] LN(p[i,t,:])_c + b_b[h]   (p[i,t,:] = P[i, nbr[i,t], :])
 *   l[h,i,t] = q_{i,h} . k_{nbr[i,t],h} / sqrt(d) + b[i,t,h]   (-inf for an empty slot)
 *   (a query whose slots are all empty gives 0)
 *   out[i, h*d+e] = g_i[h*d+e] * sum_t softmax_t(l[h,i,:]) v_{nbr[i,t],h,e}
 *
 * a [L, c_atom] fp64; p_rows [n_rows, k, c_ap] (fp32 or bf16 bits); nbr
 * [n_rows, k] int32; rows[r] is the atom index of query r. n_blocks == 1: the
 * plain softmax over all slots; n_blocks > 1: slots grouped by the chunk of
 * [0, L) their neighbour index falls in, one partial per block, folded in
 * increasing block order.
 * ------------------------------------------------------------------------- */
int oracle_sparse_attention(int64_t n_atoms, int c_atom, int c_ap, int n_heads, int d, int k, const double* a,
                            const void* p_rows, int p_dtype, const int32_t* nbr, const int64_t* rows, int64_t n_rows,
                            const double* w_q, const double* w_k, const double* w_v, const double* w_g,
                            const double* w_b, const double* b_b, const double* gamma, const double* beta, double eps,
                            int n_blocks, double* out) {
  if (!a || !p_rows || !nbr || !rows || !w_q || !w_k || !w_v || !w_g || !w_b || !out) return -1;
  if (n_atoms <= 0 || k <= 0 || n_blocks < 1 || n_blocks > n_atoms) return -1;
  const int hd = n_heads * d;
  double* kk = (double*)malloc(sizeof(double) * (size_t)(n_atoms * hd));
  double* vv = (double*)malloc(sizeof(double) * (size_t)(n_atoms * hd));
  oracle_linear(n_atoms, c_atom, hd, a, w_k, kk);
  oracle_linear(n_atoms, c_atom, hd, a, w_v, vv);
  const double scale = 1.0 / sqrt((double)d);
#pragma omp parallel
  {
    double* ai = (double*)malloc(sizeof(double) * (size_t)c_atom);
    double* q = (double*)malloc(sizeof(double) * (size_t)hd);
    double* gp = (double*)malloc(sizeof(double) * (size_t)hd);
    double* ln = (double*)malloc(sizeof(double) * (size_t)c_ap);
    double* bias = (double*)malloc(sizeof(double) * (size_t)(k * n_heads));
    double* logit = (double*)malloc(sizeof(double) * (size_t)k);
    double* accb = (double*)malloc(sizeof(double) * (size_t)d);
    double* run = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 16)
    for (int64_t r = 0; r < n_rows; ++r) {
      const int64_t i = rows[r];
      memcpy(ai, a + i * c_atom, sizeof(double) * (size_t)c_atom);
      oracle_linear(1, c_atom, hd, ai, w_q, q);
      oracle_linear(1, c_atom, hd, ai, w_g, gp);
      for (int t = 0; t < k; ++t)
        pair_bias(p_rows, p_dtype, (r * k + t) * (int64_t)c_ap, c_ap, n_heads, w_b, b_b, gamma, beta, eps, ln,
                  bias + t * n_heads);
      for (int h = 0; h < n_heads; ++h) {
        double rm = -INFINITY, rl = 0.0;
        for (int e = 0; e < d; ++e) run[e] = 0.0;
        for (int blk = 0; blk < n_blocks; ++blk) {
          int64_t bsize, bstart;
          oracle_chunk(n_atoms, n_blocks, blk, &bsize, &bstart);
          /* logits of the slots whose neighbour lies in this block */
          double mx = -INFINITY;
          for (int t = 0; t < k; ++t) {
            const int32_t j = nbr[r * k + t];
            logit[t] = -INFINITY;
            if (j < 0 || j >= n_atoms || j < bstart || j >= bstart + bsize) continue;
            double dot = 0.0;
            for (int e = 0; e < d; ++e) dot += q[h * d + e] * kk[(int64_t)j * hd + h * d + e];
            logit[t] = dot * scale + bias[t * n_heads + h];
            if (logit[t] > mx) mx = logit[t];
          }
          if (mx == -INFINITY) continue; /* empty partial */
          double lb = 0.0;
          for (int e = 0; e < d; ++e) accb[e] = 0.0;
          for (int t = 0; t < k; ++t) {
            if (logit[t] == -INFINITY) continue;
            const double w = exp(logit[t] - mx);
            lb += w;
            for (int e = 0; e < d; ++e) accb[e] += w * vv[(int64_t)nbr[r * k + t] * hd + h * d + e];
          }
          fold(d, &rm, &rl, run, mx, lb, accb);
        }
        for (int e = 0; e < d; ++e) {
          const double o = rl > 0.0 ? run[e] / rl : 0.0;
          out[r * hd + h * d + e] = sigmoid(gp[h * d + e]) * o;
        }
      }
    }
    free(ai);
    free(q);
    free(gp);
    free(ln);
    free(bias);
    free(logit);
    free(accb);
    free(run);
  }
  free(kk);
  free(vv);
  return 0;
}

/* ---------------------------------------------------------------------------
 * k nearest neighbours of atoms (Appendix "Distributed kNN for sparse atom
 * attention"; Methods, "Atom-level kNN attention budget"): for every query
 * atom, the k candidate atoms closest in Euclidean distance, never forming the
 * whole [L, L] distance matrix: the candidates are visited in blocks, each
 * block's top-k is taken, and the running top-k is merged with it (the ring
 * top-k combine).
 *
 * Readings: the order is by squared distance, computed in fp32 as
 * ((dx*dx) + (dy*dy)) + (dz*dz) with dx = x_q - x_c and every operation
 * rounded to fp32, ties broken by the smaller candidate index; a query's own
 * atom (distance 0) counts. group_mode 1 admits only candidates of the query's
 * group, 2 only candidates of other groups (the paper's intra- and
 * inter-chain budgets); 0 admits all. Fewer than k admissible candidates
 * leave index -1 and d2 +inf at the end of the list.
 * ------------------------------------------------------------------------- */
typedef struct {
  float d2;
  int64_t j;
} knn_key;

static int knn_less(knn_key a, knn_key b) { return a.d2 < b.d2 || (a.d2 == b.d2 && a.j < b.j); }

static int knn_cmp(const void* pa, const void* pb) {
  const knn_key a = *(const knn_key*)pa, b = *(const knn_key*)pb;
  return knn_less(a, b) ? -1 : (knn_less(b, a) ? 1 : 0);
}

static float knn_d2(const float* a, const float* b) {
  const float dx = a[0] - b[0], dy = a[1] - b[1], dz = a[2] - b[2];
  const float xx = dx * dx, yy = dy * dy, zz = dz * dz;
  const float s = xx + yy;
  return s + zz;
}

/* Top-k of each query against candidates [0, n_c) (global index c_index0 + j). */
int oracle_knn(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, int64_t c_index0, const int32_t* group_q,
               const int32_t* group_c, int group_mode, int k, int32_t* idx_out, float* d2_out) {
  if (!x_q || !x_c || !idx_out || k < 1 || n_c < 0 || n_q < 0) return -1;
  if (group_mode != 0 && (!group_q || !group_c)) return -1;
#pragma omp parallel
  {
    knn_key* keys = (knn_key*)malloc(sizeof(knn_key) * (size_t)(n_c > 0 ? n_c : 1));
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < n_q; ++r) {
      int64_t n = 0;
      for (int64_t j = 0; j < n_c; ++j) {
        if (group_mode == 1 && group_c[j] != group_q[r]) continue;
        if (group_mode == 2 && group_c[j] == group_q[r]) continue;
        keys[n].d2 = knn_d2(x_q + 3 * r, x_c + 3 * j);
        keys[n].j = c_index0 + j;
        ++n;
      }
      qsort(keys, (size_t)n, sizeof(knn_key), knn_cmp);
      for (int t = 0; t < k; ++t) {
        idx_out[r * k + t] = t < n ? (int32_t)keys[t].j : -1;
        if (d2_out) d2_out[r * k + t] = t < n ? keys[t].d2 : INFINITY;
      }
    }
    free(keys);
  }
  return 0;
}

/* The ring top-k combine: per row, the k smallest entries of the union of two
 * sorted candidate lists (index -1 entries are empty and sort last). */
int oracle_topk_merge(int64_t n_rows, int k, const int32_t* idx_a, const float* d2_a, const int32_t* idx_b,
                      const float* d2_b, int32_t* idx_out, float* d2_out) {
  if (!idx_a || !d2_a || !idx_b || !d2_b || !idx_out || !d2_out || k < 1) return -1;
  for (int64_t r = 0; r < n_rows; ++r) {
    knn_key* u = (knn_key*)malloc(sizeof(knn_key) * (size_t)(2 * k));
    int n = 0;
    for (int t = 0; t < k; ++t) {
      if (idx_a[r * k + t] >= 0) {
        u[n].d2 = d2_a[r * k + t];
        u[n].j = idx_a[r * k + t];
        ++n;
      }
      if (idx_b[r * k + t] >= 0) {
        u[n].d2 = d2_b[r * k + t];
        u[n].j = idx_b[r * k + t];
        ++n;
      }
    }
    qsort(u, (size_t)n, sizeof(knn_key), knn_cmp);
    for (int t = 0; t < k; ++t) {
      idx_out[r * k + t] = t < n ? (int32_t)u[t].j : -1;
      d2_out[r * k + t] = t < n ? u[t].d2 : INFINITY;
    }
    free(u);
  }
  return 0;
}

/* Blocked form (self-tests): candidates split into n_blocks by the chunk rule,
 * each block's top-k taken, merged into the running top-k in block order. */
int oracle_knn_blocked(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, const int32_t* group_q,
                       const int32_t* group_c, int group_mode, int k, int n_blocks, int32_t* idx_out, float* d2_out) {
  if (n_blocks < 1 || n_blocks > n_c) return -1;
  const size_t cells = (size_t)(n_q * k);
  int32_t* bi = (int32_t*)malloc(sizeof(int32_t) * cells);
  float* bd = (float*)malloc(sizeof(float) * cells);
  int32_t* ri = (int32_t*)malloc(sizeof(int32_t) * cells);
  float* rd = (float*)malloc(sizeof(float) * cells);
  for (size_t c = 0; c < cells; ++c) {
    ri[c] = -1;
    rd[c] = INFINITY;
  }
  for (int b = 0; b < n_blocks; ++b) {
    int64_t size, start;
    oracle_chunk(n_c, n_blocks, b, &size, &start);
    oracle_knn(x_q, n_q, x_c + 3 * start, size, start, group_q, group_c ? group_c + start : NULL, group_mode, k, bi, bd);
    oracle_topk_merge(n_q, k, ri, rd, bi, bd, idx_out, d2_out);
    memcpy(ri, idx_out, sizeof(int32_t) * cells);
    memcpy(rd, d2_out, sizeof(float) * cells);
  }
  free(bi);
  free(bd);
  free(ri);
  free(rd);
  return 0;
}

/* ---------------------------------------------------------------------------
 * Pair transition (Appendix "Manual SwiGLU decomposition", Eq. for
 * Transition(Z) and Alg. alg:swiglu-decomp): the SwiGLU feed-forward update of
 * the pair track with its residual,
 *   N = LayerNorm(z),  A = W1 N,  B = W2 N,  T = W3 (SiLU(A) * B),  z <- z + T,
 * SiLU(a) = a / (1 + exp(-a)), W1, W2: c_z -> hidden, W3: hidden -> c_z
 * (nn.Linear layout [out, in], no bias), evaluated per pair; the LayerNorm
 * is the one read for the attention bias (biased variance, eps inside the
 * square root, affine gamma and beta; NULL = 1 and 0).
 * z: [n_pairs, c_z] fp32 (dtype 0) or bf16 (1); out: [n_pairs, c_z] fp64.
 * ------------------------------------------------------------------------- */
int oracle_transition(int64_t n_pairs, int c_z, int hidden, const void* z, int dtype, const double* w1, const double* w2,
                      const double* w3, const double* gamma, const double* beta, double eps, double* out) {
  if (!z || !w1 || !w2 || !w3 || !out || c_z <= 0 || hidden <= 0) return -1;
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)c_z);
    double* n = (double*)malloc(sizeof(double) * (size_t)c_z);
    double* h = (double*)malloc(sizeof(double) * (size_t)hidden);
#pragma omp for schedule(static)
    for (int64_t p = 0; p < n_pairs; ++p) {
      double mu = 0.0, var = 0.0;
      for (int c = 0; c < c_z; ++c) {
        x[c] = load_elem(z, dtype, p * c_z + c);
        mu += x[c];
      }
      mu /= c_z;
      for (int c = 0; c < c_z; ++c) var += (x[c] - mu) * (x[c] - mu);
      var /= c_z;
      const double inv = 1.0 / sqrt(var + eps);
      for (int c = 0; c < c_z; ++c) n[c] = (gamma ? gamma[c] : 1.0) * ((x[c] - mu) * inv) + (beta ? beta[c] : 0.0);
      for (int u = 0; u < hidden; ++u) {
        double a = 0.0, b = 0.0;
        for (int c = 0; c < c_z; ++c) {
          a += w1[(int64_t)u * c_z + c] * n[c];
          b += w2[(int64_t)u * c_z + c] * n[c];
        }
        h[u] = a / (1.0 + exp(-a)) * b;
      }
      for (int c = 0; c < c_z; ++c) {
        double t = 0.0;
        for (int u = 0; u < hidden; ++u) t += w3[(int64_t)c * hidden + u] * h[u];
        out[p * c_z + c] = x[c] + t;
      }
    }
    free(x);
    free(n);
    free(h);
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Atom -> token mean pooling (Appendix "Non-determinism guard" and the 2D
 * pooling boundary: atom-level features are averaged per token; the paper
 * replaces a non-deterministic atomic index_reduce("mean") by a deterministic
 * reduction): out[t, :] = mean of a[i, :] over the atoms i with tok_idx[i] = t,
 * summed in increasing atom order in fp64; a token without atoms gives 0; an
 * index outside [0, n_tokens) belongs to no token.
 * a: [n_atoms, c] fp32 (dtype 0) or bf16 (1); out: [n_tokens, c] fp64.
 * ------------------------------------------------------------------------- */
int oracle_scatter_mean(int64_t n_atoms, int64_t n_tokens, int c, const void* a, int dtype, const int32_t* tok_idx,
                        double* out) {
  if (!a || !tok_idx || !out || c <= 0 || n_tokens < 0 || n_atoms < 0) return -1;
  int64_t* cnt = (int64_t*)calloc((size_t)(n_tokens > 0 ? n_tokens : 1), sizeof(int64_t));
  for (int64_t t = 0; t < n_tokens * c; ++t) out[t] = 0.0;
  for (int64_t i = 0; i < n_atoms; ++i) {
    const int64_t t = tok_idx[i];
    if (t < 0 || t >= n_tokens) continue;
    cnt[t] += 1;
    for (int k = 0; k < c; ++k) out[t * c + k] += load_elem(a, dtype, i * c + k);
  }
  for (int64_t t = 0; t < n_tokens; ++t)
    for (int k = 0; k < c; ++k) out[t * c + k] = cnt[t] > 0 ? out[t * c + k] / (double)cnt[t] : 0.0;
  free(cnt);
  return 0;
}
