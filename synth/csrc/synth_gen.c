/*
 * Seeded synthetic-input generator (host C, OpenMP).
 *
 * This file produces the *inputs* of the verification path (weights, KV-cache
 * contents, logits for accept-only tests).  It holds none of the method's
 * arithmetic.  Both the CPU oracle and the GPU path consume the bytes it writes.
 *
 * Generator: counter-based SplitMix64 (Steele, Lea & Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  The i-th 64-bit word of the
 * stream with key K is  mix64(K + (i + 1) * GOLDEN)  -- exactly the i-th output
 * of a SplitMix64 generator seeded with K -- so any element can be produced
 * independently and the fill parallelises without changing values.
 * Stream key:  K(seed, stream) = mix64(mix64(seed) ^ (stream * GOLDEN2)).
 * Uniform:     U = ((w >> 11) + 0.5) * 2^-53, in (0, 1).
 * Normal:      Box-Muller on words (2p, 2p+1):  r = sqrt(-2 ln U0),
 *              z_{2p} = r cos(2 pi U1),  z_{2p+1} = r sin(2 pi U1)   (fp64, libm).
 * Outputs are scaled in fp64, rounded to fp32 (C cast, nearest-even) and, for
 * bf16, rounded once more from fp32 to bf16 with nearest-even.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL
#define GOLDEN2 0xD1B54A32D192ED03ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_stream_key(uint64_t seed, uint64_t stream) {
  return mix64(mix64(seed) ^ (stream * GOLDEN2));
}

static inline uint64_t word_at(uint64_t key, uint64_t i) { return mix64(key + (i + 1) * GOLDEN); }

static inline double unif(uint64_t w) { return ((double)(w >> 11) + 0.5) * (1.0 / 9007199254740992.0); }

static inline uint16_t f32_to_bf16_rne(float f) {
  union { float f; uint32_t u; } v; v.f = f;
  uint32_t u = v.u;
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

void synth_words(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, uint64_t* out) {
  uint64_t key = synth_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (size_t i = 0; i < n; ++i) out[i] = word_at(key, offset + i);
}

/* Fill out[0..n) with mean + std * z_{offset + i}; each Box-Muller pair is evaluated once. */
#define NORMAL_FILL(NAME, T, CONVERT)                                                            \
  void NAME(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, double mean, double std, T* out) { \
    uint64_t key = synth_stream_key(seed, stream);                                               \
    if (n == 0) return;                                                                          \
    uint64_t p0 = offset >> 1, p1 = (offset + n - 1) >> 1;                                       \
    _Pragma("omp parallel for schedule(static)")                                                 \
    for (uint64_t p = p0; p <= p1; ++p) {                                                        \
      double u0 = unif(word_at(key, 2 * p)), u1 = unif(word_at(key, 2 * p + 1));                 \
      double r = sqrt(-2.0 * log(u0)), t = 6.283185307179586 * u1;                               \
      double z[2] = {r * cos(t), r * sin(t)};                                                    \
      for (int h = 0; h < 2; ++h) {                                                              \
        uint64_t i = 2 * p + h;                                                                  \
        if (i < offset || i >= offset + n) continue;                                             \
        out[i - offset] = CONVERT(mean + std * z[h]);                                            \
      }                                                                                          \
    }                                                                                            \
  }

#define CONV_F64(x) (x)
#define CONV_F32(x) ((float)(x))
#define CONV_BF16(x) f32_to_bf16_rne((float)(x))
NORMAL_FILL(synth_normal_f64, double, CONV_F64)
NORMAL_FILL(synth_normal_f32, float, CONV_F32)
NORMAL_FILL(synth_normal_bf16, uint16_t, CONV_BF16)

/* Uniform integers in [0, high): w mod high (bias < high / 2^64, negligible). */
void synth_randint(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, uint64_t high, int32_t* out) {
  uint64_t key = synth_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (size_t i = 0; i < n; ++i) out[i] = (int32_t)(word_at(key, offset + i) % high);
}

void synth_uniform_f64(uint64_t seed, uint64_t stream, uint64_t offset, size_t n, double* out) {
  uint64_t key = synth_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (size_t i = 0; i < n; ++i) out[i] = unif(word_at(key, offset + i));
}
