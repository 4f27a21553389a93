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
