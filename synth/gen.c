/*
 * Seeded synthetic input generator shared by the library tests, the benchmark
 * and the oracle checks.  It holds none of the method's arithmetic: it only
 * turns (seed, tensor id, element index) into a value and stores it in the
 * requested element type.
 *
 * Generator: splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
 * number generators", OOPSLA 2014; the 64-bit finaliser published with it) used
 * in counter mode.  Normal deviates come from the Box-Muller transform (Box and
 * Muller, 1958).  Every value depends only on its counter, so the contents of a
 * tensor are the same whatever the thread count.
 *
 * Element types: 0 = IEEE binary16, 1 = bfloat16, 2 = binary32.  The 16-bit
 * encodings are round-to-nearest-even from binary32.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t sm64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t tensor_id) {
  return sm64(seed ^ sm64(tensor_id * 0xD1B54A32D192ED03ull));
}

static inline uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* binary32 -> binary16, round to nearest even, with subnormals, inf and NaN. */
static uint16_t enc_f16(float f) {
  uint32_t u = f32_bits(f);
  uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  uint32_t exp = (u >> 23) & 0xFFu, man = u & 0x7FFFFFu;
  if (exp == 0xFFu) return sign | 0x7C00u | (man ? 0x200u : 0u);
  int e = (int)exp - 127 + 15;
  if (e >= 31) return sign | 0x7C00u;
  if (e <= 0) {                       /* subnormal or zero in binary16 */
    if (e < -10) return sign;
    uint32_t m = man | 0x800000u;     /* 24-bit significand */
    int shift = 14 - e;               /* keep 10 - (1 - e) bits */
    uint32_t q = m >> shift, rem = m & ((1u << shift) - 1u), half = 1u << (shift - 1);
    if (rem > half || (rem == half && (q & 1u))) q++;
    return sign | (uint16_t)q;
  }
  uint32_t q = ((uint32_t)e << 10) | (man >> 13), rem = man & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) q++;   /* may carry into inf */
  return sign | (uint16_t)q;
}

/* binary32 -> bfloat16, round to nearest even; NaN stays NaN. */
static uint16_t enc_bf16(float f) {
  uint32_t u = f32_bits(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline void store(void* dst, int dtype, int64_t i, float v) {
  if (dtype == 0) ((uint16_t*)dst)[i] = enc_f16(v);
  else if (dtype == 1) ((uint16_t*)dst)[i] = enc_bf16(v);
  else ((float*)dst)[i] = v;
}

/* dst[i] = mean + std * N(0,1) for i in [0, n).  Pair p = i/2 draws one 64-bit
 * counter value; its high and low halves give the two Box-Muller uniforms. */
int synth_fill_normal(void* dst, int64_t n, int dtype, uint64_t seed, uint64_t tensor_id,
                      double mean, double std) {
  if (!dst || n < 0 || dtype < 0 || dtype > 2) return -1;
  const uint64_t key = stream_key(seed, tensor_id);
  const int64_t npairs = (n + 1) / 2;
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < npairs; ++p) {
    uint64_t r = sm64(key + (uint64_t)p);
    double u1 = ((double)(r >> 32) + 1.0) * (1.0 / 4294967296.0);   /* (0, 1] */
    double u2 = (double)(r & 0xFFFFFFFFull) * (1.0 / 4294967296.0); /* [0, 1) */
    double rad = sqrt(-2.0 * log(u1));
    double z0 = rad * cos(two_pi * u2), z1 = rad * sin(two_pi * u2);
    store(dst, dtype, 2 * p, (float)(mean + std * z0));
    if (2 * p + 1 < n) store(dst, dtype, 2 * p + 1, (float)(mean + std * z1));
  }
  return 0;
}

/* dst[i] = uniform integer in [lo, hi] (inclusive), stored exactly. */
int synth_fill_int(void* dst, int64_t n, int dtype, uint64_t seed, uint64_t tensor_id,
                   int lo, int hi) {
  if (!dst || n < 0 || dtype < 0 || dtype > 2 || hi < lo) return -1;
  const uint64_t key = stream_key(seed, tensor_id);
  const uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint64_t r = sm64(key + (uint64_t)i);
    int v = lo + (int)((r >> 11) % span);
    store(dst, dtype, i, (float)v);
  }
  return 0;
}

/* Encode n binary32 values into dtype (used to build structured fixtures). */
int synth_encode(const float* src, void* dst, int64_t n, int dtype) {
  if (!src || !dst || n < 0 || dtype < 0 || dtype > 2) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) store(dst, dtype, i, src[i]);
  return 0;
}
