/*
 * ORACLE - test infrastructure only.  Nothing in the library calls, links or
 * loads this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.
 *
 * What the heterogeneous Linear computes (HeteGen, Sec. 3.1 "Parallelism
 * Strategy", Fig. 3a and Eq. 2; Sec. 4.2 "Hybrid Heterogeneous Parallelism",
 * Fig. 5a): the weight of one linear module is partitioned between the CPU and
 * the GPU, each device computes its part of the output and the parts are joined.
 * The partition changes who computes which output, not the result, so the
 * oracle is the plain definition of the module:
 *
 *     y[b, j] = sum_{k=0}^{K-1} x[b, k] * W[j, k]  +  bias[j]
 *
 * in binary32, products and partial sums rounded to binary32 in the order
 * k = 0, 1, ..., K-1, the bias added after the last product.  Inputs are
 * decoded from their 16-bit encodings exactly (every binary16 and bfloat16
 * value is a binary32 value).  The decoders below are written from the
 * IEEE 754-2008 binary16 layout (1 sign, 5 exponent bits with bias 15,
 * 10 fraction bits, subnormals, inf, NaN) and the bfloat16 layout (the upper
 * 16 bits of a binary32).  They share nothing with the library.
 *
 * Element type codes: 0 = binary16, 1 = bfloat16, 2 = binary32.
 * Layouts: x [B, K] row stride ldx; W [N, K] row-major (PyTorch nn.Linear
 * weight layout); bias [N] or NULL; y [B, N] binary32, row stride ldy.
 *
 * The parallel loop over output features only splits independent outputs
 * among threads (for timing); each output is computed by one thread in the
 * order stated above, so the result does not depend on the thread count.
 */
#include <stdint.h>
#include <string.h>

float oracle_decode_f16(uint16_t h) {
  uint32_t sign = (uint32_t)(h >> 15) << 31;
  uint32_t e = (h >> 10) & 0x1Fu, f = h & 0x3FFu, bits;
  if (e == 0x1Fu) {
    bits = sign | 0x7F800000u | (f << 13);           /* inf or NaN */
  } else if (e != 0) {
    bits = sign | ((e - 15u + 127u) << 23) | (f << 13); /* normal */
  } else if (f == 0) {
    bits = sign;                                      /* signed zero */
  } else {
    /* subnormal: value = f * 2^-24; renormalise */
    int exp = -14;
    while (!(f & 0x400u)) { f <<= 1; --exp; }
    f &= 0x3FFu;
    bits = sign | ((uint32_t)(exp + 127) << 23) | (f << 13);
  }
  float out;
  memcpy(&out, &bits, 4);
  return out;
}

float oracle_decode_bf16(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float out;
  memcpy(&out, &bits, 4);
  return out;
}

static float load(const void* p, int dtype, int64_t i) {
  if (dtype == 0) return oracle_decode_f16(((const uint16_t*)p)[i]);
  if (dtype == 1) return oracle_decode_bf16(((const uint16_t*)p)[i]);
  return ((const float*)p)[i];
}

/* Decode n elements of dtype into binary32 (used by tests to read outputs). */
int oracle_decode(const void* src, int dtype, int64_t n, float* dst) {
  if (!src || !dst || n < 0 || dtype < 0 || dtype > 2) return -1;
  for (int64_t i = 0; i < n; ++i) dst[i] = load(src, dtype, i);
  return 0;
}

/* One output: sequential binary32 dot product, bias last. */
static float dot_row(const void* x, int64_t xoff, const void* W, int64_t woff, int K, int dtype,
                     const void* bias, int64_t j) {
  float acc = 0.0f;
  for (int k = 0; k < K; ++k) {
    float p = load(x, dtype, xoff + k) * load(W, dtype, woff + k);
    acc = acc + p;
  }
  if (bias) acc = acc + load(bias, dtype, j);
  return acc;
}

/* Full output y[B, N]. */
int oracle_linear_f32(const void* x, int ldx, int B, int K, const void* W, int N, int dtype,
                      const void* bias, float* y, int ldy) {
  if (!x || !W || !y || B < 0 || K < 0 || N < 0 || dtype < 0 || dtype > 2 || ldx < K || ldy < N)
    return -1;
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < N; ++j)
    for (int b = 0; b < B; ++b)
      y[(int64_t)b * ldy + j] = dot_row(x, (int64_t)b * ldx, W, j * (int64_t)K, K, dtype, bias, j);
  return 0;
}

/* Selected outputs only: out[i] = y[rows_b[i], rows_j[i]] for i in [0, n). */
int oracle_linear_sample(const void* x, int ldx, int B, int K, const void* W, int N, int dtype,
                         const void* bias, const int* rows_b, const int64_t* rows_j, int64_t n,
                         float* out) {
  if (!x || !W || !out || !rows_b || !rows_j || K < 0 || ldx < K) return -1;
  for (int64_t i = 0; i < n; ++i)
    if (rows_b[i] < 0 || rows_b[i] >= B || rows_j[i] < 0 || rows_j[i] >= N) return -1;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    out[i] = dot_row(x, (int64_t)rows_b[i] * ldx, W, rows_j[i] * (int64_t)K, K, dtype, bias, rows_j[i]);
  return 0;
}
