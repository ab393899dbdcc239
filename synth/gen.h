/*
 * Seeded synthetic input values, shared by the device fill kernel and the
 * CPU oracle.  This header holds no part of the layout transform: it only
 * says which number sits at position `idx` of a buffer.
 *
 * Definition (counter based, so any element can be recomputed on its own):
 *   mix(z)       = SplitMix64 output finalizer (Steele, Lea & Flood,
 *                  "Fast splittable pseudorandom number generators",
 *                  OOPSLA 2014): z ^= z>>30; z *= 0xBF58476D1CE4E5B9;
 *                  z ^= z>>27; z *= 0x94D049BB133111EB; z ^= z>>31.
 *   bits(s,t,i)  = mix(s ^ mix(t) ^ ((i+1) * 0x9E3779B97F4A7C15))  (mod 2^64)
 *   real64(b)    = 2 * ((b >> 11) * 2^-53) - 1        uniform on [-1, 1),
 *                  a multiple of 2^-52, computed exactly, never -0.
 *   real32(b)    = 2 * ((b >> 40) * 2^-24) - 1        the same on a 2^-23 grid.
 *   complex      : real part from counter 2*i, imaginary part from 2*i+1.
 *
 * The stream number names the buffer: synth_stream(role, item, rank).
 */
#ifndef SYNTH_GEN_H
#define SYNTH_GEN_H

#include <stdint.h>

#if defined(__HIPCC__)
#define SYNTH_FN static inline __host__ __device__
#else
#define SYNTH_FN static inline
#endif

#define SYNTH_GOLDEN 0x9E3779B97F4A7C15ULL

/* Roles of the buffers a test or a benchmark fills. */
#define SYNTH_ROLE_B 1u  /* source matrix B            */
#define SYNTH_ROLE_A 2u  /* initial target matrix A_0  */

SYNTH_FN uint64_t synth_mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ULL;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBULL;
  z ^= z >> 31;
  return z;
}

SYNTH_FN uint64_t synth_bits(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_mix64(seed ^ synth_mix64(stream) ^ ((idx + 1u) * SYNTH_GOLDEN));
}

/* stream = role * 2^32 + item * 2^16 + rank  (item < 2^16, rank < 2^16) */
SYNTH_FN uint64_t synth_stream(uint32_t role, uint32_t item, uint32_t rank) {
  return ((uint64_t)role << 32) | ((uint64_t)(item & 0xFFFFu) << 16) | (uint64_t)(rank & 0xFFFFu);
}

SYNTH_FN double synth_real64(uint64_t b) {
  return 2.0 * ((double)(b >> 11) * 0x1.0p-53) - 1.0;
}

SYNTH_FN float synth_real32(uint64_t b) {
  return 2.0f * ((float)(uint32_t)(b >> 40) * 0x1.0p-24f) - 1.0f;
}

/* Value of element idx of a real buffer. */
SYNTH_FN double synth_f64(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real64(synth_bits(seed, stream, idx));
}
SYNTH_FN float synth_f32(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real32(synth_bits(seed, stream, idx));
}
/* Real and imaginary parts of element idx of a complex buffer. */
SYNTH_FN double synth_c128_re(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real64(synth_bits(seed, stream, 2u * idx));
}
SYNTH_FN double synth_c128_im(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real64(synth_bits(seed, stream, 2u * idx + 1u));
}
SYNTH_FN float synth_c64_re(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real32(synth_bits(seed, stream, 2u * idx));
}
SYNTH_FN float synth_c64_im(uint64_t seed, uint64_t stream, uint64_t idx) {
  return synth_real32(synth_bits(seed, stream, 2u * idx + 1u));
}

/* Uniform integer in [0, n) by rejection (no modulo bias); `*ctr` advances
 * once per draw, including rejected draws.  n >= 1. */
SYNTH_FN uint64_t synth_below(uint64_t seed, uint64_t stream, uint64_t* ctr, uint64_t n) {
  const uint64_t lim = (~(uint64_t)0) - ((~(uint64_t)0) % n + 1u) % n; /* largest multiple of n, minus 1 */
  for (;;) {
    uint64_t b = synth_bits(seed, stream, (*ctr)++);
    if (b <= lim) return b % n;
  }
}

#endif /* SYNTH_GEN_H */
