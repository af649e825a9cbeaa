/*
 * Host twin of the synthetic-input generator (the device twin lives in the
 * library as sevo_fill_normal_bf16).  It is pure input generation: seeded,
 * counter-based, and free of any arithmetic of the decode step.
 *
 * Element e of a tensor with key k:
 *   r   = mix64(k + (e + 1) * 0x9E3779B97F4A7C15)        (SplitMix64, Steele,
 *         Lea & Flood, "Fast splittable pseudorandom number generators",
 *         OOPSLA 2014; finaliser as in java.util.SplittableRandom)
 *   s   = sum of the four 16-bit fields of r              (Irwin-Hall, n = 4)
 *   val = fp32(s - 131070) * mul  [+ add]                 (each op rounded once)
 *   out = bf16 bits of val, round-to-nearest-even
 * mul = std / sqrt((2^32 - 1) / 3) rounded to fp32 by the caller.
 *
 * Build: gcc -O3 -fopenmp -ffp-contract=off -shared -fPIC
 */
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

uint64_t synth_mix64(uint64_t z) { return mix64(z); }

/* out[i] = bf16(normal_approx(key, offset + i) * mul + add), i < count */
void synth_fill_bf16(uint16_t* out, int64_t count, uint64_t key, int64_t offset,
                     float mul, float add, int use_add) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    uint64_t r = mix64(key + (uint64_t)(offset + i + 1) * 0x9E3779B97F4A7C15ULL);
    int32_t s = (int32_t)(r & 0xFFFF) + (int32_t)((r >> 16) & 0xFFFF) +
                (int32_t)((r >> 32) & 0xFFFF) + (int32_t)(r >> 48);
    volatile float v = (float)(s - 131070) * mul;
    float w = use_add ? (float)(v + add) : (float)v;
    out[i] = f32_to_bf16_rne(w);
  }
}

/* Same values as fp32 (bf16-representable), for host consumers. */
void synth_fill_bf16_as_f32(float* out, int64_t count, uint64_t key, int64_t offset,
                            float mul, float add, int use_add) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) {
    uint64_t r = mix64(key + (uint64_t)(offset + i + 1) * 0x9E3779B97F4A7C15ULL);
    int32_t s = (int32_t)(r & 0xFFFF) + (int32_t)((r >> 16) & 0xFFFF) +
                (int32_t)((r >> 32) & 0xFFFF) + (int32_t)(r >> 48);
    volatile float v = (float)(s - 131070) * mul;
    float w = use_add ? (float)(v + add) : (float)v;
    uint32_t b = ((uint32_t)f32_to_bf16_rne(w)) << 16;
    memcpy(&out[i], &b, 4);
  }
}

/* Selected pages of a paged tensor: out[j * per_page + i] = the fp32 value of
 * element pages[j] * per_page + i, for j < n_sel and i < per_page. */
void synth_fill_pages_as_f32(float* out, const int64_t* pages, int64_t n_sel, int64_t per_page,
                             uint64_t key, float mul, float add, int use_add) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n_sel; ++j)
    for (int64_t i = 0; i < per_page; ++i) {
      const int64_t el = pages[j] * per_page + i;
      uint64_t r = mix64(key + (uint64_t)(el + 1) * 0x9E3779B97F4A7C15ULL);
      int32_t s = (int32_t)(r & 0xFFFF) + (int32_t)((r >> 16) & 0xFFFF) +
                  (int32_t)((r >> 32) & 0xFFFF) + (int32_t)(r >> 48);
      volatile float v = (float)(s - 131070) * mul;
      float w = use_add ? (float)(v + add) : (float)v;
      uint32_t b = ((uint32_t)f32_to_bf16_rne(w)) << 16;
      memcpy(&out[j * per_page + i], &b, 4);
    }
}
