// gfx950 kernels of the heterogeneous Linear: the GPU-share GEMV and the small
// glue kernels around it.
//
// GEMV (HeteGen Sec. 4.2: the GPU computes its share of the module's output
// once its weight rows are in device memory).  At batch 1..8 a linear reads each
// weight element once and does 2B flops on it, i.e. B flop per byte of fp16/bf16
// weight: far below the ridge point of the vector ALUs, so the kernel is bound by
// HBM bandwidth and uses no matrix cores.  Design:
//  * one wavefront (64 lanes) owns R output rows at a time; a lane loads 16 bytes
//    (8 elements) of each row per step, so one load instruction reads 1 KiB of a
//    row, fully coalesced; U steps are unrolled so U*R 16-byte loads per lane are
//    in flight;
//  * x [B, K] is staged once per workgroup in LDS (in K tiles when it does not fit)
//    and every lane reads its 8 elements per batch row with ds_read_b128, reused for
//    the R rows it holds;
//  * products accumulate in binary32 through v_dot2 (fp16 pairs or bf16 pairs with
//    binary32 accumulation);
//  * the 64 lane partials of each (row, batch) pair are summed with DPP row
//    permutations and four readlanes;
//  * workgroups walk the row groups in a grid-stride loop, so x is staged once per
//    workgroup rather than once per row group;
//  * the epilogue adds the bias, applies ReLU or a residual sum and rounds to the
//    activation type (or stores binary32), so the decode step needs no separate
//    elementwise kernels; an optional LayerNorm prologue normalises x while staging it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace hg {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kLnEps = 1e-5f;

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte weight load (read once: marked non-temporal).
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

struct F16 {
  static __device__ __forceinline__ float dot2(uint32_t w, uint32_t x, float acc) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, w), __builtin_bit_cast(f16x2, x), acc, false);
  }
  static __device__ __forceinline__ float lo(uint32_t v) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v & 0xFFFFu));
  }
  static __device__ __forceinline__ float hi(uint32_t v) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v >> 16));
  }
  static __device__ __forceinline__ float to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
  static __device__ __forceinline__ uint16_t from_f32(float v) { return __builtin_bit_cast(uint16_t, (_Float16)v); }
};

struct BF16 {
  static __device__ __forceinline__ float dot2(uint32_t w, uint32_t x, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), __builtin_bit_cast(bf16x2, x), acc,
                                           false);
  }
  static __device__ __forceinline__ float lo(uint32_t v) { return __builtin_bit_cast(float, v << 16); }
  static __device__ __forceinline__ float hi(uint32_t v) { return __builtin_bit_cast(float, v & 0xFFFF0000u); }
  static __device__ __forceinline__ float to_f32(uint16_t h) { return __builtin_bit_cast(float, (uint32_t)h << 16); }
  static __device__ __forceinline__ uint16_t from_f32(float v) { return __builtin_bit_cast(uint16_t, (__bf16)v); }
};

template <class T>
__device__ __forceinline__ float dot8(const uint4& w, const uint4& x, float acc) {
  acc = T::dot2(w.x, x.x, acc);
  acc = T::dot2(w.y, x.y, acc);
  acc = T::dot2(w.z, x.z, acc);
  acc = T::dot2(w.w, x.w, acc);
  return acc;
}

template <class T>
__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  f[0] = T::lo(v.x); f[1] = T::hi(v.x); f[2] = T::lo(v.y); f[3] = T::hi(v.y);
  f[4] = T::lo(v.z); f[5] = T::hi(v.z); f[6] = T::lo(v.w); f[7] = T::hi(v.w);
}

template <class T>
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return (uint32_t)T::from_f32(a) | ((uint32_t)T::from_f32(b) << 16);
}

// Sum over the 64 lanes of a wavefront; every lane returns the total.
__device__ __forceinline__ float wave_sum(float v) {
  int iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x141, 0xF, 0xF, false)); // row_half_mirror
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x140, 0xF, 0xF, false)); // row_mirror
  iv = __builtin_bit_cast(int, v);
  // each 16-lane row now holds its row sum in every lane
  float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 0));
  float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 16));
  float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 32));
  float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(iv, 48));
  return (r0 + r1) + (r2 + r3);
}

// LayerNorm statistics of B rows of x [B, K] for one 256-thread workgroup, two
// passes (mean, then the mean of squared deviations).  The reduction order is
// fixed by the thread mapping, so every workgroup of every kernel that calls this
// gets bit-identical statistics.
template <class T, int B>
__device__ __forceinline__ void ln_stats(const uint16_t* __restrict__ x, long long ldx, int K, float* mean,
                                         float* rstd, float (*red)[8][kWaves]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n8 = K >> 3;
  float s[B];
#pragma unroll
  for (int b = 0; b < B; ++b) {
    s[b] = 0.f;
    for (int c = tid; c < n8; c += kThreads) {
      uint4 v = *(const uint4*)(x + b * ldx + (long long)c * 8);
      float f[8];
      unpack8<T>(v, f);
      s[b] += ((f[0] + f[1]) + (f[2] + f[3])) + ((f[4] + f[5]) + (f[6] + f[7]));
    }
    s[b] = wave_sum(s[b]);
    if (lane == 0) red[0][b][wave] = s[b];
  }
  __syncthreads();
#pragma unroll
  for (int b = 0; b < B; ++b) mean[b] = ((red[0][b][0] + red[0][b][1]) + (red[0][b][2] + red[0][b][3])) / (float)K;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    s[b] = 0.f;
    for (int c = tid; c < n8; c += kThreads) {
      uint4 v = *(const uint4*)(x + b * ldx + (long long)c * 8);
      float f[8];
      unpack8<T>(v, f);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float d = f[e] - mean[b];
        acc += d * d;
      }
      s[b] += acc;
    }
    s[b] = wave_sum(s[b]);
    if (lane == 0) red[1][b][wave] = s[b];
  }
  __syncthreads();
#pragma unroll
  for (int b = 0; b < B; ++b) {
    float var = ((red[1][b][0] + red[1][b][1]) + (red[1][b][2] + red[1][b][3])) / (float)K;
    rstd[b] = 1.0f / sqrtf(var + kLnEps);
  }
}

template <class T>
__device__ __forceinline__ uint4 normalize8(const uint4& v, float mean, float rstd) {
  float f[8];
  unpack8<T>(v, f);
  uint4 o;
  o.x = pack2<T>((f[0] - mean) * rstd, (f[1] - mean) * rstd);
  o.y = pack2<T>((f[2] - mean) * rstd, (f[3] - mean) * rstd);
  o.z = pack2<T>((f[4] - mean) * rstd, (f[5] - mean) * rstd);
  o.w = pack2<T>((f[6] - mean) * rstd, (f[7] - mean) * rstd);
  return o;
}

template <class T>
__device__ __forceinline__ void finish(float v, int epi, int y_f32, void* y, long long yi, const void* resid,
                                       long long ri) {
  if (epi == EPI_RELU) v = fmaxf(v, 0.f);
  else if (epi == EPI_RESID) v = v + T::to_f32(((const uint16_t*)resid)[ri]);
  if (y_f32) ((float*)y)[yi] = v;
  else ((uint16_t*)y)[yi] = T::from_f32(v);
}

// Stage tile [k0, k0 + kn) of x (optionally normalised) into LDS as [B][ktile].
template <class T, int B>
__device__ __forceinline__ void stage_x(const GemvParams& p, uint4* xs, int k0, int kn, const float* mean,
                                        const float* rstd, bool write_h) {
  const uint16_t* x = (const uint16_t*)p.x;
  const int n8 = kn >> 3, kt8 = p.ktile >> 3;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    for (int c = threadIdx.x; c < n8; c += kThreads) {
      uint4 v = *(const uint4*)(x + b * p.ldx + k0 + (long long)c * 8);
      if (p.ln) {
        v = normalize8<T>(v, mean[b], rstd[b]);
        if (write_h) *(uint4*)((uint16_t*)p.h_out + b * p.ldh + k0 + (long long)c * 8) = v;
      }
      xs[b * kt8 + c] = v;
    }
  }
}

template <class T, int B, int R, int U>
__global__ __launch_bounds__(kThreads) void gemv_kernel(GemvParams p) {
  extern __shared__ uint4 xs[];
  __shared__ float red[2][8][kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int K = p.K, ktile = p.ktile, kt8 = ktile >> 3;
  const int ntiles = (K + ktile - 1) / ktile;
  float mean[B], rstd[B];
#pragma unroll
  for (int b = 0; b < B; ++b) { mean[b] = 0.f; rstd[b] = 1.f; }
  if (p.ln) ln_stats<T, B>((const uint16_t*)p.x, p.ldx, K, mean, rstd, red);
  const bool wg_writes_h = p.ln && p.h_out != nullptr && blockIdx.x == 0;
  if (ntiles == 1) {
    stage_x<T, B>(p, xs, 0, K, mean, rstd, wg_writes_h);
    __syncthreads();
  }
  const int nrg = (p.rows + R - 1) / R;
  const uint16_t* W = (const uint16_t*)p.W;
  const uint16_t* bias = (const uint16_t*)p.bias;
  bool first = true;
  for (int rg0 = blockIdx.x * kWaves; rg0 < nrg; rg0 += gridDim.x * kWaves) {
    const int rg = rg0 + wave;
    const bool valid = rg < nrg;  // uniform per wavefront
    const int row0 = rg * R;
    const uint4* wp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      int row = min(row0 + r, p.rows - 1);
      wp[r] = (const uint4*)(W + (long long)row * K);
    }
    float acc[R][B];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int b = 0; b < B; ++b) acc[r][b] = 0.f;
    for (int t = 0; t < ntiles; ++t) {
      const int k0 = t * ktile, kn = min(ktile, K - k0);
      if (ntiles > 1) {
        __syncthreads();
        stage_x<T, B>(p, xs, k0, kn, mean, rstd, wg_writes_h && first);
        __syncthreads();
      }
      if (valid) {
        const int n8 = kn >> 3, c0 = k0 >> 3;
        int c = lane;
        for (; c + 64 * (U - 1) < n8; c += 64 * U) {
          uint4 w[U][R];
          uint4 xv[U][B];
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) w[u][r] = load_stream(wp[r] + c0 + c + 64 * u);
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int b = 0; b < B; ++b) xv[u][b] = xs[b * kt8 + c + 64 * u];
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
              for (int b = 0; b < B; ++b) acc[r][b] = dot8<T>(w[u][r], xv[u][b], acc[r][b]);
        }
        for (; c < n8; c += 64) {
          uint4 w[R];
#pragma unroll
          for (int r = 0; r < R; ++r) w[r] = load_stream(wp[r] + c0 + c);
#pragma unroll
          for (int b = 0; b < B; ++b) {
            uint4 xv = xs[b * kt8 + c];
#pragma unroll
            for (int r = 0; r < R; ++r) acc[r][b] = dot8<T>(w[r], xv, acc[r][b]);
          }
        }
      }
    }
    if (valid) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
          float s = wave_sum(acc[r][b]);
          const int row = row0 + r;
          if (lane == 0 && row < p.rows) {
            if (bias) s += T::to_f32(bias[row]);
            finish<T>(s, p.epi, p.y_f32, p.y, b * p.ldy + row, p.resid, b * p.ldr + row);
          }
        }
      }
    }
    first = false;
  }
}

template <class T, int B>
__global__ __launch_bounds__(kThreads) void layernorm_kernel(const uint16_t* __restrict__ x, long long ldx, int K,
                                                             uint16_t* __restrict__ h, long long ldh,
                                                             float* __restrict__ h_host) {
  __shared__ float red[2][8][kWaves];
  float mean[B], rstd[B];
  ln_stats<T, B>(x, ldx, K, mean, rstd, red);
  const int n8 = K >> 3;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    for (int c = blockIdx.x * kThreads + threadIdx.x; c < n8; c += gridDim.x * kThreads) {
      uint4 v = normalize8<T>(*(const uint4*)(x + b * ldx + (long long)c * 8), mean[b], rstd[b]);
      *(uint4*)(h + b * ldh + (long long)c * 8) = v;
      if (h_host) {
        float f[8];
        unpack8<T>(v, f);
        float4* dst = (float4*)(h_host + (long long)b * K + (long long)c * 8);
        dst[0] = make_float4(f[0], f[1], f[2], f[3]);
        dst[1] = make_float4(f[4], f[5], f[6], f[7]);
      }
    }
  }
}

template <class T>
__global__ __launch_bounds__(kThreads) void export_kernel(const uint16_t* __restrict__ x, long long ldx, int B, int K,
                                                          float* __restrict__ dst) {
  const int n8 = K >> 3;
  const long long total = (long long)B * n8;
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < total; i += (long long)gridDim.x * kThreads) {
    const int b = (int)(i / n8), c = (int)(i - (long long)b * n8);
    float f[8];
    unpack8<T>(*(const uint4*)(x + b * ldx + (long long)c * 8), f);
    float4* d = (float4*)(dst + (long long)b * K + (long long)c * 8);
    d[0] = make_float4(f[0], f[1], f[2], f[3]);
    d[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
}

template <class T>
__global__ __launch_bounds__(kThreads) void import_kernel(const float* __restrict__ src, int B, int n, int epi,
                                                          void* __restrict__ y, long long ldy, int y_f32,
                                                          const void* __restrict__ resid, long long ldr) {
  const long long total = (long long)B * n;
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < total; i += (long long)gridDim.x * kThreads) {
    const int b = (int)(i / n), c = (int)(i - (long long)b * n);
    finish<T>(src[i], epi, y_f32, y, b * ldy + c, resid, b * ldr + c);
  }
}

// Per-batch tiling: rows per wavefront R and unrolled steps U (U*R loads in flight).
template <int B> struct Tile;
template <> struct Tile<1> { static constexpr int R = 1, U = 8; };
template <> struct Tile<2> { static constexpr int R = 2, U = 4; };
template <> struct Tile<3> { static constexpr int R = 2, U = 4; };
template <> struct Tile<4> { static constexpr int R = 2, U = 4; };
template <> struct Tile<5> { static constexpr int R = 4, U = 2; };
template <> struct Tile<6> { static constexpr int R = 4, U = 2; };
template <> struct Tile<7> { static constexpr int R = 4, U = 2; };
template <> struct Tile<8> { static constexpr int R = 4, U = 2; };

constexpr int kLdsBudget = 32768;  // bytes of LDS for the x tile per workgroup
constexpr int kDefaultGridCap = 1024;

template <class T, int B>
hipError_t launch_gemv_b(GemvParams p, hipStream_t s, int grid_cap) {
  constexpr int R = Tile<B>::R, U = Tile<B>::U;
  int kt = kLdsBudget / (2 * B);
  kt -= kt % 512;
  if (p.K <= kt) kt = p.K;
  p.ktile = kt;
  const int nrg = (p.rows + R - 1) / R;
  int grid = (nrg + kWaves - 1) / kWaves;
  const int cap = grid_cap > 0 ? grid_cap : kDefaultGridCap;
  if (grid > cap) grid = cap;
  const size_t lds = (size_t)B * kt * 2;
  hipLaunchKernelGGL((gemv_kernel<T, B, R, U>), dim3(grid), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

template <class T>
hipError_t launch_gemv_t(const GemvParams& p, int B, hipStream_t s, int cap) {
  switch (B) {
    case 1: return launch_gemv_b<T, 1>(p, s, cap);
    case 2: return launch_gemv_b<T, 2>(p, s, cap);
    case 3: return launch_gemv_b<T, 3>(p, s, cap);
    case 4: return launch_gemv_b<T, 4>(p, s, cap);
    case 5: return launch_gemv_b<T, 5>(p, s, cap);
    case 6: return launch_gemv_b<T, 6>(p, s, cap);
    case 7: return launch_gemv_b<T, 7>(p, s, cap);
    case 8: return launch_gemv_b<T, 8>(p, s, cap);
  }
  return hipErrorInvalidValue;
}

template <class T, int B>
hipError_t launch_ln_b(const void* x, long long ldx, int K, void* h, long long ldh, float* hh, hipStream_t s) {
  const int n8 = K >> 3;
  int grid = (n8 + kThreads * 4 - 1) / (kThreads * 4);
  if (grid < 1) grid = 1;
  if (grid > 16) grid = 16;
  hipLaunchKernelGGL((layernorm_kernel<T, B>), dim3(grid), dim3(kThreads), 0, s, (const uint16_t*)x, ldx, K,
                     (uint16_t*)h, ldh, hh);
  return hipGetLastError();
}

template <class T>
hipError_t launch_ln_t(const void* x, long long ldx, int B, int K, void* h, long long ldh, float* hh, hipStream_t s) {
  switch (B) {
    case 1: return launch_ln_b<T, 1>(x, ldx, K, h, ldh, hh, s);
    case 2: return launch_ln_b<T, 2>(x, ldx, K, h, ldh, hh, s);
    case 3: return launch_ln_b<T, 3>(x, ldx, K, h, ldh, hh, s);
    case 4: return launch_ln_b<T, 4>(x, ldx, K, h, ldh, hh, s);
    case 5: return launch_ln_b<T, 5>(x, ldx, K, h, ldh, hh, s);
    case 6: return launch_ln_b<T, 6>(x, ldx, K, h, ldh, hh, s);
    case 7: return launch_ln_b<T, 7>(x, ldx, K, h, ldh, hh, s);
    case 8: return launch_ln_b<T, 8>(x, ldx, K, h, ldh, hh, s);
  }
  return hipErrorInvalidValue;
}

int small_grid(long long work_items) {
  long long g = (work_items + kThreads - 1) / kThreads;
  if (g < 1) g = 1;
  if (g > 256) g = 256;
  return (int)g;
}

}  // namespace

hipError_t launch_gemv(GemvParams p, int dtype, int B, hipStream_t stream, int grid_cap) {
  if (p.rows <= 0) return hipSuccess;
  return dtype == 1 ? launch_gemv_t<BF16>(p, B, stream, grid_cap) : launch_gemv_t<F16>(p, B, stream, grid_cap);
}

hipError_t launch_layernorm(const void* x, long long ldx, int B, int K, int dtype, void* h, long long ldh,
                            float* h_host_f32, hipStream_t stream) {
  return dtype == 1 ? launch_ln_t<BF16>(x, ldx, B, K, h, ldh, h_host_f32, stream)
                    : launch_ln_t<F16>(x, ldx, B, K, h, ldh, h_host_f32, stream);
}

hipError_t launch_export_f32(const void* x, long long ldx, int B, int K, int dtype, float* dst, hipStream_t stream) {
  const int grid = small_grid((long long)B * (K >> 3));
  if (dtype == 1)
    hipLaunchKernelGGL(export_kernel<BF16>, dim3(grid), dim3(kThreads), 0, stream, (const uint16_t*)x, ldx, B, K, dst);
  else
    hipLaunchKernelGGL(export_kernel<F16>, dim3(grid), dim3(kThreads), 0, stream, (const uint16_t*)x, ldx, B, K, dst);
  return hipGetLastError();
}

hipError_t launch_import_rows(const float* src, int B, int n, int dtype, int epi, void* y, long long ldy, int y_f32,
                              const void* resid, long long ldr, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int grid = small_grid((long long)B * n);
  if (dtype == 1)
    hipLaunchKernelGGL(import_kernel<BF16>, dim3(grid), dim3(kThreads), 0, stream, src, B, n, epi, y, ldy, y_f32,
                       resid, ldr);
  else
    hipLaunchKernelGGL(import_kernel<F16>, dim3(grid), dim3(kThreads), 0, stream, src, B, n, epi, y, ldy, y_f32,
                       resid, ldr);
  return hipGetLastError();
}

}  // namespace hg
