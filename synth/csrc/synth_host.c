/* Seeded synthetic inputs, host side (plain C).
 *
 * This file generates test and benchmark inputs only. It holds none of the
 * attention arithmetic: it is shared by the fp64 oracle's tests and by the GPU
 * path's tests and benchmark, so that both read the same values.
 *
 * Definition (identical in synth/__init__.py and synth/csrc/synth_dev.hip):
 *   fin(x)        SplitMix64 output function (Steele, Lea, Flood 2014):
 *                 x ^= x>>30; x *= 0xBF58476D1CE4E5B9; x ^= x>>27;
 *                 x *= 0x94D049BB133111EB; x ^= x>>31
 *   key(seed,t)   fin(fin(seed + G) + t*G), G = 0x9E3779B97F4A7C15
 *   word(k,n)     fin(k + (n+1)*G)              (counter-based SplitMix64)
 *   normal(k,e)   Irwin-Hall(12): the twelve 16-bit fields of word(k,3e),
 *                 word(k,3e+1), word(k,3e+2) summed to S, then
 *                 (S - 393210) / 65536. Mean 0, variance 1 - 2^-32; the value
 *                 is an exact fp32 number, so no rounding mode enters.
 *   bf16(x)       round-to-nearest-even of the fp32 bits to the top 16.
 *   structured z  z[i,j,c] = bf16(fl32(base[i%P, j%P, c] + fl32(0.1f*noise[i,j,c])))
 *                 evaluated as two separately rounded fp32 operations.
 */
#include <stdint.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define SM_G 0x9E3779B97F4A7C15ULL

static inline uint64_t sm_fin(uint64_t x) {
  x ^= x >> 30;
  x *= 0xBF58476D1CE4E5B9ULL;
  x ^= x >> 27;
  x *= 0x94D049BB133111EBULL;
  x ^= x >> 31;
  return x;
}

uint64_t synth_key(uint64_t seed, uint64_t tensor_id) {
  return sm_fin(sm_fin(seed + SM_G) + tensor_id * SM_G);
}

uint64_t synth_word(uint64_t key, uint64_t n) { return sm_fin(key + (n + 1) * SM_G); }

static inline float sm_normal(uint64_t key, uint64_t e) {
  int32_t s = 0;
  for (int k = 0; k < 3; ++k) {
    uint64_t w = sm_fin(key + (3 * e + (uint64_t)k + 1) * SM_G);
    s += (int32_t)(w & 0xFFFF) + (int32_t)((w >> 16) & 0xFFFF) +
         (int32_t)((w >> 32) & 0xFFFF) + (int32_t)((w >> 48) & 0xFFFF);
  }
  return (float)(s - 393210) * (1.0f / 65536.0f);
}

static inline uint16_t sm_bf16(float x) {
  uint32_t b;
  memcpy(&b, &x, 4);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

/* out[i] = normal(key, start + i), i < count. */
void synth_normal_f32(uint64_t key, uint64_t start, int64_t count, float* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = sm_normal(key, start + (uint64_t)i);
}

/* out[i] = bf16(normal(key, start + i)). */
void synth_normal_bf16(uint64_t key, uint64_t start, int64_t count, uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = sm_bf16(sm_normal(key, start + (uint64_t)i));
}

/* Rows `rows[r]` of the pair tensor z[N, N, c_z] into out[r, N, c_z].
 * period == 0: z[i,j,c] = normal(key_z, (i*N + j)*c_z + c).
 * period  > 0: structured form above with base element index
 *              ((i%period)*period + j%period)*c_z + c and noise index (i*N+j)*c_z + c.
 * out_bf16 != 0 writes bf16 bits (uint16), else fp32. */
void synth_z_rows(uint64_t key_z, uint64_t key_base, int64_t period, int64_t n_tok, int32_t c_z,
                  const int64_t* rows, int64_t n_rows, int32_t out_bf16, void* out) {
  const int64_t row_elems = n_tok * (int64_t)c_z;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t r = 0; r < n_rows; ++r) {
    for (int64_t j = 0; j < n_tok; ++j) {
      const int64_t i = rows[r];
      for (int32_t c = 0; c < c_z; ++c) {
        const uint64_t e = ((uint64_t)i * (uint64_t)n_tok + (uint64_t)j) * (uint64_t)c_z + (uint64_t)c;
        float v;
        if (period > 0) {
          const uint64_t eb = ((uint64_t)(i % period) * (uint64_t)period + (uint64_t)(j % period)) *
                                  (uint64_t)c_z + (uint64_t)c;
          volatile float t = 0.1f * sm_normal(key_z, e); /* volatile: keep two roundings */
          v = sm_normal(key_base, eb) + t;
        } else {
          v = sm_normal(key_z, e);
        }
        const int64_t o = r * row_elems + j * c_z + c;
        if (out_bf16)
          ((uint16_t*)out)[o] = sm_bf16(v);
        else
          ((float*)out)[o] = v;
      }
    }
  }
}

/* Neighbour lists for sparse atom attention, nbr[r, t] for query atoms
 * i = row0 + r (r < n_rows), slots t < k; -1 marks an empty slot.
 *
 * Stand-in for the paper's kNN budget (query atom plus flanking residues in
 * sequence, then spatial neighbours, with an inter-chain quota when there are
 * more than three chains), made without coordinates:
 *   atoms are grouped into residues of `per_res` atoms and chains of
 *   `per_chain` atoms (the last chain may be shorter); atom i lies in chain
 *   c = i / per_chain, at residue r = (i % per_chain) / per_res;
 *   1. sequence-local: every atom of residues r-1, r, r+1 of the same chain,
 *      in index order;
 *   2. intra-chain: atoms drawn uniformly from residues r-win .. r+win of the
 *      same chain, skipping repeats, until k - q_inter slots are filled;
 *   3. inter-chain (only with more than three chains): q_inter atoms drawn
 *      uniformly from residues r-win .. r+win of chains c+1, c-1 (cyclic, in
 *      turn), skipping repeats;
 *   draws use word(key, i*8192 + a), a the attempt number (attempts 0..4095
 *   for step 2, 4096..8191 for step 3); unfilled slots stay -1.
 *   ragged != 0: rows with word(key2, i) % 8 == 0 then empty their last
 *   word(key2, i) / 8 % (k/2) slots (budgets not filled). */
static int64_t nb_window(int64_t chain0, int64_t chain_len, int64_t per_res, int64_t r_lo, int64_t r_hi,
                         int64_t* lo) {
  int64_t a = chain0 + (r_lo < 0 ? 0 : r_lo) * per_res;
  int64_t b = chain0 + (r_hi + 1) * per_res;
  if (b > chain0 + chain_len) b = chain0 + chain_len;
  *lo = a;
  return b > a ? b - a : 0;
}

static int nb_has(const int32_t* row, int n, int32_t j) {
  for (int t = 0; t < n; ++t)
    if (row[t] == j) return 1;
  return 0;
}

void synth_neighbours(uint64_t key, uint64_t key2, int64_t n_atoms, int32_t per_res, int32_t per_chain, int32_t k,
                      int32_t win, int32_t q_inter, int64_t row0, int64_t n_rows, int32_t ragged, int32_t* out) {
  const int64_t n_chains = (n_atoms + per_chain - 1) / per_chain;
  const int32_t quota = n_chains > 3 ? (q_inter < k ? q_inter : k) : 0;
#pragma omp parallel for schedule(static)
  for (int64_t rr = 0; rr < n_rows; ++rr) {
    const int64_t i = row0 + rr;
    int32_t* row = out + rr * k;
    for (int t = 0; t < k; ++t) row[t] = -1;
    const int64_t c = i / per_chain, c0 = c * per_chain;
    const int64_t clen = (c0 + per_chain <= n_atoms) ? per_chain : n_atoms - c0;
    const int64_t r = (i - c0) / per_res;
    int n = 0;
    int64_t lo, cnt;
    cnt = nb_window(c0, clen, per_res, r - 1, r + 1, &lo);
    for (int64_t j = lo; j < lo + cnt && n < k; ++j) row[n++] = (int32_t)j;
    cnt = nb_window(c0, clen, per_res, r - win, r + win, &lo);
    for (uint64_t a = 0; a < 4096 && n < k - quota && cnt > 0; ++a) {
      const int32_t j = (int32_t)(lo + (int64_t)(synth_word(key, (uint64_t)i * 8192 + a) % (uint64_t)cnt));
      if (!nb_has(row, n, j)) row[n++] = j;
    }
    const int target = n + quota < k ? n + quota : k;
    for (uint64_t a = 0; a < 4096 && n < target; ++a) {
      const int64_t cc = (a & 1) ? (c + n_chains - 1) % n_chains : (c + 1) % n_chains;
      const int64_t cc0 = cc * per_chain;
      const int64_t cclen = (cc0 + per_chain <= n_atoms) ? per_chain : n_atoms - cc0;
      cnt = nb_window(cc0, cclen, per_res, r - win, r + win, &lo);
      if (cnt <= 0) continue;
      const int32_t j = (int32_t)(lo + (int64_t)(synth_word(key, (uint64_t)i * 8192 + 4096 + a) % (uint64_t)cnt));
      if (!nb_has(row, n, j)) row[n++] = j;
    }
    if (ragged) {
      const uint64_t w = synth_word(key2, (uint64_t)i);
      if (w % 8 == 0) {
        const int drop = (int)((w / 8) % (uint64_t)(k / 2 > 0 ? k / 2 : 1));
        for (int t = k - drop; t < k; ++t) row[t] = -1;
      }
    }
  }
}

/* Atom coordinates of a synthetic assembly, out[L, 3] fp32 (Angstrom).
 * Chains of `per_chain` atoms (residues of `per_res` atoms) are random walks:
 * residue r sits 3.8 A from residue r-1 along the direction of a normal vector;
 * each chain is centred on its mean and moved to point c of a Fibonacci sphere
 * of radius 12 * sqrt(n_chains) A (neighbouring chains touch); atoms scatter
 * around their residue with N(0, 1.5 A) per axis. Normals: direction noise normal(key, (c * n_res + r) * 3 + axis),
 * atom offsets normal(key, 2^40 + 3 * atom + axis). Computed in fp64, stored
 * rounded to fp32. */
void synth_coords(uint64_t key, int64_t n_atoms, int32_t per_res, int32_t per_chain, float* out) {
  const int64_t n_chains = (n_atoms + per_chain - 1) / per_chain;
  const int64_t n_res = (per_chain + per_res - 1) / per_res;
  const double radius = 12.0 * sqrt((double)n_chains);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t c = 0; c < n_chains; ++c) {
    double* res = (double*)malloc(sizeof(double) * (size_t)(3 * n_res));
    double dir[3], p[3] = {0.0, 0.0, 0.0}, mean[3] = {0.0, 0.0, 0.0};
    for (int64_t r = 0; r < n_res; ++r) {
      double nd[3], nn = 0.0;
      for (int a = 0; a < 3; ++a) {
        nd[a] = (double)sm_normal(key, (uint64_t)((c * n_res + r) * 3 + a));
        nn += nd[a] * nd[a];
      }
      nn = sqrt(nn);
      for (int a = 0; a < 3; ++a) {
        dir[a] = nd[a] / nn;
        if (r > 0) p[a] += 3.8 * dir[a];
        res[3 * r + a] = p[a];
        mean[a] += p[a];
      }
    }
    /* Fibonacci sphere point c of n_chains */
    const double golden = 2.39996322972865332; /* pi (3 - sqrt 5) */
    const double y = n_chains > 1 ? 1.0 - 2.0 * ((double)c + 0.5) / (double)n_chains : 0.0;
    const double rr = sqrt(1.0 - y * y), th = golden * (double)c;
    const double centre[3] = {radius * rr * cos(th), radius * y, radius * rr * sin(th)};
    for (int64_t t = 0; t < per_chain; ++t) {
      const int64_t atom = c * per_chain + t;
      if (atom >= n_atoms) break;
      const int64_t r = t / per_res;
      for (int a = 0; a < 3; ++a) {
        const double off = 1.5 * (double)sm_normal(key, (1ULL << 40) + (uint64_t)(3 * atom + a));
        out[3 * atom + a] = (float)(res[3 * r + a] - mean[a] / (double)n_res + centre[a] + off);
      }
    }
    free(res);
  }
}
