/*
 * oracle/wgen.c -- TEST INFRASTRUCTURE ONLY (the CPU oracle).  Only tests/,
 * __graft_entry__.smoke() and bench.py's cpu_baseline leg may load this file's
 * library.  The product path never does.
 *
 * Counter-based weight generator for the random-init Llama-2-shaped models.
 * The paper runs pretrained Llama-2 (Methodology section); no weights ship, so
 * every matrix is drawn N(0, 0.02) from a seed and all norm gains are 1.  The
 * draw has to be identical on CPU and GPU, so it is defined with integer
 * arithmetic and single correctly-rounded IEEE operations only:
 *
 *   SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
 *   generators", OOPSLA 2014): gamma = 0x9E3779B97F4A7C15 and the finaliser
 *     mix(z): z ^= z>>30; z *= 0xBF58476D1CE4E5B9; z ^= z>>27;
 *             z *= 0x94D049BB133111EB; z ^= z>>31.
 *   The n-th output (n >= 1) of a stream seeded with s is mix(s + n*gamma).
 *
 *   stream key    s_tl = output (1 + 256*t + l) of the stream seeded with `seed`
 *                 (t = tensor id < 16, l = layer < 256)
 *   element e     (row-major flat index of the logical [out][in] matrix):
 *                 r0 = output 2e+1, r1 = output 2e+2 of the stream s_tl
 *   S             sum of the four 16-bit lanes of r0 and the four of r1
 *                 (Irwin-Hall sum of 8 uniforms on [0, 65535]; mean 262140)
 *   value         fp32(S - 262140) * C, one RNE fp32 multiply, with
 *                 C = RNE_fp32(0.02 / sqrt(8 * (65536^2 - 1) / 12))
 *                   = 0x1.91530cp-22, so the value has std 0.02
 *   bf16 models   the fp32 value rounded to nearest-even bf16.
 *
 * The result is exact; it is returned widened to fp64 for the numpy oracle.
 */
#include <stdint.h>
#include <string.h>

#define SM_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t sm_mix(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ULL;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return z;
}

/* n-th output (n >= 1) of the SplitMix64 stream seeded with s */
uint64_t oracle_splitmix_output(uint64_t s, uint64_t n) { return sm_mix(s + n * SM_GAMMA); }

uint64_t oracle_stream_key(uint64_t seed, int tensor, int layer) {
  return oracle_splitmix_output(seed, 1u + 256u * (uint64_t)tensor + (uint64_t)layer);
}

static inline float to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  u &= 0xFFFF0000u;
  memcpy(&f, &u, 4);
  return f;
}

static inline float element_value(uint64_t key, uint64_t e, int bf16) {
  uint64_t r0 = oracle_splitmix_output(key, 2 * e + 1);
  uint64_t r1 = oracle_splitmix_output(key, 2 * e + 2);
  int64_t s = 0;
  for (int i = 0; i < 4; ++i) {
    s += (int64_t)((r0 >> (16 * i)) & 0xFFFF);
    s += (int64_t)((r1 >> (16 * i)) & 0xFFFF);
  }
  const float c = 0x1.91530cp-22f;
  float v = (float)(s - 262140) * c;
  return bf16 ? to_bf16_rne(v) : v;
}

/* Writes rows [row0, row0 + nrows) of the logical n_rows x n_cols matrix
 * (tensor, layer) into out (row-major, nrows x n_cols doubles). */
void oracle_wgen_rows(uint64_t seed, int tensor, int layer, int64_t n_cols, int64_t row0,
                      int64_t nrows, int bf16, double* out) {
  const uint64_t key = oracle_stream_key(seed, tensor, layer);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < nrows; ++r) {
    const uint64_t base = (uint64_t)(row0 + r) * (uint64_t)n_cols;
    double* o = out + r * n_cols;
    for (int64_t c = 0; c < n_cols; ++c) o[c] = (double)element_value(key, base + (uint64_t)c, bf16);
  }
}

/* Same values as fp32 (exact), for bit-level comparisons. */
void oracle_wgen_rows_f32(uint64_t seed, int tensor, int layer, int64_t n_cols, int64_t row0,
                          int64_t nrows, int bf16, float* out) {
  const uint64_t key = oracle_stream_key(seed, tensor, layer);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < nrows; ++r) {
    const uint64_t base = (uint64_t)(row0 + r) * (uint64_t)n_cols;
    float* o = out + r * n_cols;
    for (int64_t c = 0; c < n_cols; ++c) o[c] = element_value(key, base + (uint64_t)c, bf16);
  }
}
