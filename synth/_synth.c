/* Seeded synthetic inputs shared by the oracle and the GPU path.
 *
 * Counter-based generator: element i of the stream with key k is
 *   z = mix64(k + (i + 1) * GAMMA)
 * where mix64 is the SplitMix64 finaliser (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014) and
 * GAMMA = 0x9e3779b97f4a7c15.  The top 24 bits u of z give the symmetric
 * uniform w = (2u + 1 - 2^24) / 2^24 in (-1, 1), exact in binary32.
 * A value is offset + scale * w, rounded once per operation in binary32
 * (this file is built with -ffp-contract=off so no FMA merges the two),
 * and optionally rounded to bfloat16 with round-to-nearest-even.
 *
 * This library holds no arithmetic of the decoding method: it only fills
 * buffers.  synth/gen.py has a numpy twin of every routine; a CPU test
 * checks that the two agree bit for bit.
 */
#include <stdint.h>

#define GAMMA 0x9e3779b97f4a7c15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

static inline float uniform_value(uint64_t key, uint64_t i, float scale, float offset) {
  uint64_t z = mix64(key + (i + 1) * GAMMA);
  int32_t u = (int32_t)(z >> 40);                 /* 24 bits */
  float w = (float)(2 * u + 1 - 16777216) / 16777216.0f;
  float s = scale * w;
  return offset + s;
}

static inline uint16_t to_bf16_rne(float f) {
  union { float f; uint32_t u; } v;
  v.f = f;
  uint32_t lsb = (v.u >> 16) & 1u;
  return (uint16_t)((v.u + 0x7fffu + lsb) >> 16);
}

uint64_t synth_mix64(uint64_t z) { return mix64(z); }

void synth_uniform_f32(uint64_t key, uint64_t start, int64_t n, float scale, float offset, float *out) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = uniform_value(key, start + (uint64_t)j, scale, offset);
}

void synth_uniform_bf16(uint64_t key, uint64_t start, int64_t n, float scale, float offset, uint16_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = to_bf16_rne(uniform_value(key, start + (uint64_t)j, scale, offset));
}

/* Tokens uniform over [0, vocab): multiply-shift of the high 32 bits. */
void synth_tokens(uint64_t key, uint64_t start, int64_t n, uint32_t vocab, int32_t *out) {
  for (int64_t j = 0; j < n; ++j) {
    uint64_t z = mix64(key + (start + (uint64_t)j + 1) * GAMMA);
    out[j] = (int32_t)(((z >> 32) * (uint64_t)vocab) >> 32);
  }
}

/* Exact widening of bfloat16 bit patterns to binary64 (used to hand the
 * oracle the very values the GPU streams). */
void synth_bf16_to_f64(const uint16_t *in, int64_t n, double *out) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    union { float f; uint32_t u; } v;
    v.u = ((uint32_t)in[j]) << 16;
    out[j] = (double)v.f;
  }
}
