/* Calls every entry point of the fp64 oracle on small inputs, including edge
 * cases (masked keys, empty neighbour slots, out-of-range indices, k larger
 * than the candidate set, bf16 inputs), so that a build with AddressSanitizer
 * and UndefinedBehaviorSanitizer checks the oracle's memory accesses and
 * arithmetic. Exits non-zero if an entry point rejects valid arguments or
 * returns a non-finite value where the definition gives a finite one. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_chunk(int64_t total, int64_t parts, int64_t p, int64_t* size, int64_t* start);
void oracle_linear(int64_t n_tok, int n_in, int n_out, const double* x, const double* w, double* y);
int oracle_bias(int64_t n_rows, int64_t n_cols, int c_z, int n_heads, const void* z, int dtype, int64_t row_stride,
                const double* w_b, const double* b_b, const double* gamma, const double* beta, double eps, double* out);
int oracle_attend(int64_t n_rows, int64_t n_tok, int n_heads, int d, const double* q, const double* k,
                  const double* v, const double* g_pre, const double* bias, const uint8_t* mask, double* out);
int oracle_merge(int n_parts, int64_t n_rows, int n_heads, int d, const double* m, const double* l,
                 const double* acc, const double* gate, double* m_out, double* l_out, double* acc_out, double* out);
int oracle_attention(int64_t n_tok, int c_s, int c_z, int n_heads, int d, const double* s, const void* z_rows,
                     int z_dtype, const int64_t* rows, int64_t n_rows, const uint8_t* mask, const double* w_q,
                     const double* w_k, const double* w_v, const double* w_g, const double* w_b, const double* b_b,
                     const double* gamma, const double* beta, double eps, int n_blocks, double* out, double* m_parts,
                     double* l_parts, double* acc_parts);
int oracle_sparse_attention(int64_t n_atoms, int c_atom, int c_ap, int n_heads, int d, int k, const double* a,
                            const void* p_rows, int p_dtype, const int32_t* nbr, const int64_t* rows, int64_t n_rows,
                            const double* w_q, const double* w_k, const double* w_v, const double* w_g,
                            const double* w_b, const double* b_b, const double* gamma, const double* beta, double eps,
                            int n_blocks, double* out);
int oracle_knn(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, int64_t c_index0, const int32_t* group_q,
               const int32_t* group_c, int group_mode, int k, int32_t* idx_out, float* d2_out);
int oracle_topk_merge(int64_t n_rows, int k, const int32_t* idx_a, const float* d2_a, const int32_t* idx_b,
                      const float* d2_b, int32_t* idx_out, float* d2_out);
int oracle_knn_blocked(const float* x_q, int64_t n_q, const float* x_c, int64_t n_c, const int32_t* group_q,
                       const int32_t* group_c, int group_mode, int k, int n_blocks, int32_t* idx_out, float* d2_out);
int oracle_transition(int64_t n_pairs, int c_z, int hidden, const void* z, int dtype, const double* w1,
                      const double* w2, const double* w3, const double* gamma, const double* beta, double eps,
                      double* out);
int oracle_scatter_mean(int64_t n_atoms, int64_t n_tokens, int c, const void* a, int dtype, const int32_t* tok_idx,
                        double* out);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static double uni(void) { /* xorshift64*, in [-1, 1) */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (double)((state * 0x2545F4914F6CDD1Dull) >> 11) / 4503599627370496.0 - 1.0;
}
static double* vec(size_t n) {
  double* p = (double*)malloc(n * sizeof(double));
  for (size_t i = 0; i < n; ++i) p[i] = uni();
  return p;
}
static float* vecf(size_t n) {
  float* p = (float*)malloc(n * sizeof(float));
  for (size_t i = 0; i < n; ++i) p[i] = (float)uni();
  return p;
}
static uint16_t* vecb(size_t n) { /* bf16 bit patterns of values in [-1, 1) */
  uint16_t* p = (uint16_t*)malloc(n * sizeof(uint16_t));
  for (size_t i = 0; i < n; ++i) {
    const float f = (float)uni();
    uint32_t u;
    memcpy(&u, &f, 4);
    p[i] = (uint16_t)(u >> 16);
  }
  return p;
}
static int failures = 0;
static void check(int ok, const char* what) {
  if (!ok) {
    fprintf(stderr, "FAILED: %s\n", what);
    ++failures;
  }
}
static int finite(const double* p, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(p[i])) return 0;
  return 1;
}

int main(void) {
  /* chunk rule */
  for (int64_t total = 0; total < 20; ++total)
    for (int64_t parts = 1; parts <= 6; ++parts) {
      int64_t sum = 0;
      for (int64_t p = 0; p < parts; ++p) {
        int64_t size, start;
        oracle_chunk(total, parts, p, &size, &start);
        check(start == sum, "chunk start");
        sum += size;
      }
      check(sum == total, "chunk sizes");
    }
  /* linear, bias, attend, merge */
  {
    double *x = vec(6 * 5), *w = vec(4 * 5), y[6 * 4];
    oracle_linear(6, 5, 4, x, w, y);
    check(finite(y, 24), "linear");
    free(x), free(w);
  }
  for (int dt = 0; dt < 2; ++dt) {
    const int rows = 3, cols = 5, cz = 6, h = 2;
    void* z = dt ? (void*)vecb(rows * cols * cz) : (void*)vecf(rows * cols * cz);
    double *wb = vec(h * cz), *bb = vec(h), *g = vec(cz), *b = vec(cz), out[3 * 5 * 2];
    check(oracle_bias(rows, cols, cz, h, z, dt, cols * cz, wb, bb, g, b, 1e-5, out) == 0, "bias rc");
    check(finite(out, rows * cols * h), "bias");
    check(oracle_bias(rows, cols, cz, h, z, dt, cols * cz, wb, NULL, NULL, NULL, 1e-5, out) == 0, "bias rc 2");
    free(z), free(wb), free(bb), free(g), free(b);
  }
  {
    const int nr = 3, nt = 7, h = 2, d = 3;
    double *q = vec(nr * h * d), *k = vec(nt * h * d), *v = vec(nt * h * d), *g = vec(nr * h * d);
    double *bias = vec(nr * nt * h), out[3 * 6];
    uint8_t mask[7] = {1, 0, 1, 1, 0, 1, 1}, none[7] = {0};
    check(oracle_attend(nr, nt, h, d, q, k, v, g, bias, mask, out) == 0 && finite(out, nr * h * d), "attend");
    check(oracle_attend(nr, nt, h, d, q, k, v, g, bias, NULL, out) == 0 && finite(out, nr * h * d), "attend nomask");
    check(oracle_attend(nr, nt, h, d, q, k, v, g, bias, none, out) == 0 && finite(out, nr * h * d), "attend masked");
    free(q), free(k), free(v), free(g), free(bias);
    const int np = 3;
    double *m = vec(np * h * nr), *l = vec(np * h * nr), *acc = vec(np * nr * h * d), *gate = vec(nr * h * d);
    for (int i = 0; i < np * h * nr; ++i) l[i] = fabs(l[i]) + 0.1;
    m[0] = -INFINITY;
    l[0] = 0.0;
    double mo[2 * 3], lo[2 * 3], ao[3 * 2 * 3], o2[3 * 6];
    check(oracle_merge(np, nr, h, d, m, l, acc, gate, mo, lo, ao, o2) == 0 && finite(o2, nr * h * d), "merge");
    free(m), free(l), free(acc), free(gate);
  }
  /* the whole dense definition, both z dtypes, blocked and not */
  for (int dt = 0; dt < 2; ++dt) {
    const int nt = 7, cs = 5, cz = 6, h = 2, d = 3, nb = 3;
    const int64_t rows[3] = {0, 3, 6};
    void* z = dt ? (void*)vecb(3 * nt * cz) : (void*)vecf(3 * nt * cz);
    double *s = vec(nt * cs), *wq = vec(h * d * cs), *wk = vec(h * d * cs), *wv = vec(h * d * cs);
    double *wg = vec(h * d * cs), *wb = vec(h * cz), *bb = vec(h), *g = vec(cz), *b = vec(cz);
    uint8_t mask[7] = {1, 1, 0, 1, 1, 0, 1};
    double out[3 * 6], mp[3 * 2 * 3], lp[3 * 2 * 3], ap[3 * 3 * 2 * 3];
    check(oracle_attention(nt, cs, cz, h, d, s, z, dt, rows, 3, mask, wq, wk, wv, wg, wb, bb, g, b, 1e-5, nb, out, mp,
                           lp, ap) == 0 && finite(out, 18), "attention blocked");
    check(oracle_attention(nt, cs, cz, h, d, s, z, dt, rows, 3, NULL, wq, wk, wv, wg, wb, NULL, NULL, NULL, 1e-5, 1,
                           out, NULL, NULL, NULL) == 0 && finite(out, 18), "attention");
    free(z), free(s), free(wq), free(wk), free(wv), free(wg), free(wb), free(bb), free(g), free(b);
  }
  /* sparse atom attention: empty and out-of-range slots, a repeated neighbour */
  for (int dt = 0; dt < 2; ++dt) {
    const int na = 9, ca = 5, cap = 4, h = 2, d = 3, k = 4;
    const int64_t rows[2] = {1, 4};
    const int32_t nbr[2 * 4] = {0, 2, -1, 2, 8, 9, -1, 3};
    void* p = dt ? (void*)vecb(2 * k * cap) : (void*)vecf(2 * k * cap);
    double *a = vec(na * ca), *wq = vec(h * d * ca), *wk = vec(h * d * ca), *wv = vec(h * d * ca);
    double *wg = vec(h * d * ca), *wb = vec(h * cap), *bb = vec(h), *g = vec(cap), *b = vec(cap), out[2 * 6];
    check(oracle_sparse_attention(na, ca, cap, h, d, k, a, p, dt, nbr, rows, 2, wq, wk, wv, wg, wb, bb, g, b, 1e-5, 2,
                                  out) == 0 && finite(out, 12), "sparse attention");
    const int32_t empty[2 * 4] = {-1, -1, -1, 99, -1, -1, -1, -1};
    check(oracle_sparse_attention(na, ca, cap, h, d, k, a, p, dt, empty, rows, 2, wq, wk, wv, wg, wb, NULL, NULL,
                                  NULL, 1e-5, 1, out) == 0 && finite(out, 12), "sparse attention, no neighbours");
    free(p), free(a), free(wq), free(wk), free(wv), free(wg), free(wb), free(bb), free(g), free(b);
  }
  /* kNN, the top-k merge and the blocked form; k above the candidate count */
  {
    const int nq = 5, nc = 11;
    float *xq = vecf(nq * 3), *xc = vecf(nc * 3);
    int32_t gq[5] = {0, 1, 0, 1, 2}, gc[11] = {0, 0, 1, 1, 2, 2, 0, 1, 2, 0, 1};
    for (int mode = 0; mode < 3; ++mode)
      for (int k = 1; k <= 20; k += 6) {
        int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * nq * k);
        float* d2 = (float*)malloc(sizeof(float) * nq * k);
        check(oracle_knn(xq, nq, xc, nc, 100, mode ? gq : NULL, mode ? gc : NULL, mode, k, idx, d2) == 0, "knn");
        int32_t* idx2 = (int32_t*)malloc(sizeof(int32_t) * nq * k);
        float* d22 = (float*)malloc(sizeof(float) * nq * k);
        check(oracle_knn_blocked(xq, nq, xc, nc, mode ? gq : NULL, mode ? gc : NULL, mode, k, 3, idx2, d22) == 0,
              "knn blocked");
        int32_t* io = (int32_t*)malloc(sizeof(int32_t) * nq * k);
        float* dout = (float*)malloc(sizeof(float) * nq * k);
        check(oracle_topk_merge(nq, k, idx, d2, idx2, d22, io, dout) == 0, "topk merge");
        free(idx), free(d2), free(idx2), free(d22), free(io), free(dout);
      }
    free(xq), free(xc);
  }
  /* transition, both dtypes, with and without the LayerNorm affine */
  for (int dt = 0; dt < 2; ++dt) {
    const int np = 5, cz = 6, hid = 10;
    void* z = dt ? (void*)vecb(np * cz) : (void*)vecf(np * cz);
    double *w1 = vec(hid * cz), *w2 = vec(hid * cz), *w3 = vec(cz * hid), *g = vec(cz), *b = vec(cz), out[5 * 6];
    check(oracle_transition(np, cz, hid, z, dt, w1, w2, w3, g, b, 1e-5, out) == 0 && finite(out, np * cz),
          "transition");
    check(oracle_transition(np, cz, hid, z, dt, w1, w2, w3, NULL, NULL, 1e-5, out) == 0 && finite(out, np * cz),
          "transition plain");
    free(z), free(w1), free(w2), free(w3), free(g), free(b);
  }
  /* pooling: out-of-range indices, a token without atoms, no atoms */
  for (int dt = 0; dt < 2; ++dt) {
    const int na = 9, nt = 4, c = 3;
    void* a = dt ? (void*)vecb(na * c) : (void*)vecf(na * c);
    const int32_t idx[9] = {0, 0, 1, -1, 3, 3, 4, 1, 0};
    double out[4 * 3];
    check(oracle_scatter_mean(na, nt, c, a, dt, idx, out) == 0 && finite(out, nt * c), "scatter mean");
    check(out[2 * c] == 0.0, "token without atoms");
    check(oracle_scatter_mean(0, nt, c, a, dt, idx, out) == 0 && finite(out, nt * c), "scatter mean, no atoms");
    free(a);
  }
  if (failures) return 1;
  printf("oracle driver: all entry points ran\n");
  return 0;
}
