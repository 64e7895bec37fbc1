// gfx950 kernels of the heterogeneous Linear: the GPU-share GEMV and the small
// glue kernels around it.
//
// GEMV (HeteGen Sec. 4.2: the GPU computes its share of the module's output
// once its weight rows are in device memory).  At batch 1..8 a linear reads each
// weight element once and does 2B flops on it, i.e. B flop per byte of fp16/bf16
// weight: far below the ridge point of the vector ALUs, so the kernel is bound by
// HBM bandwidth and uses no matrix cores.  Design of the main kernel:
//  * a workgroup (4 wavefronts) owns a contiguous block of output rows; a
//    wavefront takes R rows at a time and walks them in "tasks" of 64*U 16-byte
//    chunks per row: a lane loads 16 bytes (8 elements) of each row per step, so
//    one load instruction reads 1 KiB of a row, fully coalesced, and U*R loads per
//    lane are in flight;
//  * the loads of the next task are issued before the current task is computed
//    (two register buffers), so a wavefront never waits on an empty memory pipe,
//    and the weights of the first task are requested before the prologue;
//  * weight loads are non-temporal: the weights are read once per step and should
//    not evict x or the outputs from the caches;
//  * x [B, K] is staged once per workgroup in LDS (and normalised there when a
//    LayerNorm is fused) and read with ds_read_b128, reused for the R rows;
//  * products accumulate in binary32 through v_dot2 (fp16 pairs or bf16 pairs);
//  * the 64 lane partials of each (row, batch) pair are summed with DPP row
//    permutations and four readlanes;
//  * bias and residual of the block are staged in LDS in the prologue, outputs are
//    gathered in LDS and stored per block with contiguous stores; the epilogue adds
//    the bias, applies ReLU or a residual sum and rounds to the activation type (or
//    stores binary32), so the decode step needs no elementwise kernels.
// x may use the device's whole LDS per workgroup (160 KiB on gfx950, opted in above the
// default 64 KiB, with the grid capped at the workgroups that fit at once); when it
// does not fit even so (large B*K), a K-tiled variant restages x per tile.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>

#include "kernels.h"

namespace hg {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kX1MaxRows = 64;  // rows per wavefront the x-direct GEMV keeps bias/residual for
constexpr float kLnEps = 1e-5f;

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Global-memory view of a pointer.  Pointers read from a device-side table are
// generic to the compiler; generic (flat) loads also count against the LDS
// counter, so every LDS wait would drain the weight stream.
template <class T>
__device__ __forceinline__ const __attribute__((address_space(1))) T* gmem(const T* p) {
  return (const __attribute__((address_space(1))) T*)p;
}

// Cached 16-byte global load.
__device__ __forceinline__ uint4 load_g16(const uint4* p) {
  u32x4 v = *gmem((const u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Streaming 16-byte weight load (read once: marked non-temporal).
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  u32x4 v = __builtin_nontemporal_load(gmem((const u32x4*)p));
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

// Sum over each row of 16 lanes (lanes 16 r .. 16 r + 15); every lane of the row returns
// its row's total, formed in a fixed order.
__device__ __forceinline__ float row16_sum(float v) {
  int iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x141, 0xF, 0xF, false)); // row_half_mirror
  iv = __builtin_bit_cast(int, v);
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, iv, 0x140, 0xF, 0xF, false)); // row_mirror
  return v;
}

// LayerNorm statistics of B rows of x (16-byte chunk c of row b read by get(b, c))
// for one 256-thread workgroup, two passes (mean, then the mean of squared
// deviations).  Chunk c is always summed by thread c % 256 in increasing c and the
// partials are combined in a fixed tree, so every workgroup of every kernel that
// calls this gets bit-identical statistics, whether x is read from global memory
// or from LDS.
template <class T, int B, class Get>
__device__ __forceinline__ void ln_stats(Get get, int K, float* mean, float* rstd, float (*red)[8][kWaves]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n8 = K >> 3;
  // the B rows are read side by side (B loads in flight per chunk); each row's
  // partial still adds its chunks in increasing c
  float s[B];
#pragma unroll
  for (int b = 0; b < B; ++b) s[b] = 0.f;
#pragma unroll 2
  for (int c = tid; c < n8; c += kThreads) {
    uint4 v[B];
#pragma unroll
    for (int b = 0; b < B; ++b) v[b] = get(b, c);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float f[8];
      unpack8<T>(v[b], f);
      s[b] += ((f[0] + f[1]) + (f[2] + f[3])) + ((f[4] + f[5]) + (f[6] + f[7]));
    }
  }
#pragma unroll
  for (int b = 0; b < B; ++b) s[b] = wave_sum(s[b]);
  if (lane == 0)
#pragma unroll
    for (int b = 0; b < B; ++b) red[0][b][wave] = s[b];
  __syncthreads();
#pragma unroll
  for (int b = 0; b < B; ++b) {
    mean[b] = ((red[0][b][0] + red[0][b][1]) + (red[0][b][2] + red[0][b][3])) / (float)K;
    s[b] = 0.f;
  }
#pragma unroll 2
  for (int c = tid; c < n8; c += kThreads) {
    uint4 v[B];
#pragma unroll
    for (int b = 0; b < B; ++b) v[b] = get(b, c);
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float f[8];
      unpack8<T>(v[b], f);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float d = f[e] - mean[b];
        acc += d * d;
      }
      s[b] += acc;
    }
  }
#pragma unroll
  for (int b = 0; b < B; ++b) s[b] = wave_sum(s[b]);
  if (lane == 0)
#pragma unroll
    for (int b = 0; b < B; ++b) red[1][b][wave] = s[b];
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
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    f[e] = (f[e] - mean) * rstd;
    // the binary32 value is materialised before it is rounded to the activation type:
    // otherwise instruction selection may fold the scaling into a mixed-precision
    // multiply-add that rounds once to 16 bits, and results at ties would depend on
    // the surrounding code (the kernels that fuse this must agree bit for bit)
    asm volatile("" : "+v"(f[e]));
  }
  uint4 o;
  o.x = pack2<T>(f[0], f[1]);
  o.y = pack2<T>(f[2], f[3]);
  o.z = pack2<T>(f[4], f[5]);
  o.w = pack2<T>(f[6], f[7]);
  return o;
}

// ReLU or residual sum on a binary32 value (bias already added).
__device__ __forceinline__ float apply_epi(float v, int epi, float resid) {
  if (epi == EPI_RELU) return fmaxf(v, 0.f);
  if (epi == EPI_RESID) return v + resid;
  return v;
}

// A binary32 result rounded to the activation type.  The value is materialised first
// so that it is rounded once from binary32 in every kernel (instruction selection
// could otherwise fold the last add into a mixed-precision operation that rounds
// straight to 16 bits, which differs at ties).
template <class T>
__device__ __forceinline__ uint16_t round_act(float v) {
  asm volatile("" : "+v"(v));
  return T::from_f32(v);
}

template <class T>
__device__ __forceinline__ void store_y(void* y, long long i, int y_f32, float v) {
  if (y_f32) ((float*)y)[i] = v;
  else ((uint16_t*)y)[i] = round_act<T>(v);
}

// ---------------------------------------------------------------------------
// Coherent accesses for data produced by other workgroups of the same kernel
// (the persistent decode step): buffer loads/stores with sc0 sc1, which bypass
// the non-coherent cache levels, so no L2 writeback/invalidate is needed between
// linears.  Word 3 of the buffer descriptor is the gfx9 raw-buffer format.
// ---------------------------------------------------------------------------
constexpr int kBufWord3 = 0x00020000;
constexpr int kCoherent = 1 | 16;  // sc0 | sc1
constexpr uint32_t kXPast = 0x80000000u;  // a buffer offset past every descriptor the GEMVs build

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufWord3);
}

// The descriptor base must be wave-uniform (it lives in scalar registers): pass
// the row base and a per-lane byte offset; `bytes` bounds the row.
template <bool COH>
__device__ __forceinline__ uint4 load_act16(const uint16_t* row, uint32_t bytes, uint32_t off) {
  if (COH) {
    u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rsrc(row, bytes), (int)off, 0, kCoherent);
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  return *(const uint4*)((const char*)row + off);
}

template <bool COH>
__device__ __forceinline__ uint16_t load_act1(const uint16_t* row, uint32_t bytes, uint32_t off) {
  if (COH) return (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(rsrc(row, bytes), (int)off, 0, kCoherent);
  return *(const uint16_t*)((const char*)row + off);
}

// y row base (wave-uniform) and element index within the row.
template <class T, bool COH>
__device__ __forceinline__ void store_y_c(void* yrow, uint32_t n, uint32_t i, int y_f32, float v) {
  if (COH) {
    if (y_f32)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rsrc(yrow, n * 4), (int)(i * 4), 0,
                                            kCoherent);
    else
      __builtin_amdgcn_raw_buffer_store_b16(round_act<T>(v), rsrc(yrow, n * 2), (int)(i * 2), 0, kCoherent);
    return;
  }
  store_y<T>(yrow, i, y_f32, v);
}

// 16-byte group col of row `row` in the segment-major layout of a [rows, K] weight.
__device__ __forceinline__ const uint4* seg_addr(const uint4* W, int rows, int row, int col) {
  constexpr int G = kSegElems / 8;  // 16-byte groups per segment
  return W + ((long long)(col / G) * rows + row) * G + (col % G);
}

// ---------------------------------------------------------------------------
// Main GEMV, one workgroup's block of rows (x fits in LDS).  Dynamic LDS layout:
//   xs [B][K/8] uint4 | bias [rpw] f32 | resid [B][rpw] f32 | out [B][rpw] f32
// The first task of every wavefront is requested before `wait()` and the
// prologue, so its weights stream in while the block waits for its inputs.
// ---------------------------------------------------------------------------
template <class T, int B, int R, int U, bool COH_LOAD, bool COH_STORE, class Wait>
__device__ __forceinline__ void gemv_block(const GemvParams& p, int blk, uint4* smem, float (*red)[8][kWaves],
                                           Wait wait) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = p.K, k8 = K >> 3, rpw = p.rpw;
  uint4* xs = smem;
  float* sb = (float*)(smem + (size_t)B * k8);
  float* sr = sb + rpw;
  float* sy = sr + B * rpw;
  const int row_begin = blk * rpw;
  const int nrows = max(0, min(rpw, p.rows - row_begin));
  constexpr int SEG = 64 * U;  // 16-byte chunks per task and row
  const int nseg = (k8 + SEG - 1) / SEG;
  const int nrg = (nrows + R - 1) / R;
  const int my_rg = nrg > wave ? (nrg - wave + kWaves - 1) / kWaves : 0;
  const int ntask = my_rg * nseg;
  const uint16_t* W = (const uint16_t*)p.W;

  // task t of this wavefront: row group j = t / nseg (local rows (wave + j*kWaves)*R ..), segment t % nseg
  auto load = [&](int t, uint4 (&w)[U][R]) {
    const int j = t / nseg, seg = t - j * nseg;
    const int lr0 = (wave + j * kWaves) * R;
    const int c0 = seg * SEG + lane;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int row = row_begin + min(lr0 + r, nrows - 1);
      const uint4* wr = (const uint4*)(W + (long long)row * K);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // unconditional load (clamped address): no branch, so the compiler can keep
        // later tasks' loads in flight; lanes past the row end reread its last
        // chunk (same cache line, no extra traffic) and skip it in compute()
        const int col = min(c0 + 64 * u, k8 - 1);
        w[u][r] = load_stream(p.segmajor ? seg_addr((const uint4*)W, p.rows, row, col) : wr + col);
      }
    }
  };
  auto compute = [&](int t, const uint4 (&w)[U][R], float (&acc)[R][B]) {
    const int j = t / nseg, seg = t - j * nseg;
    const int c0 = seg * SEG + lane;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + 64 * u;
      if (c < k8) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const uint4 xv = xs[b * k8 + c];
#pragma unroll
          for (int r = 0; r < R; ++r) acc[r][b] = dot8<T>(w[u][r], xv, acc[r][b]);
        }
      }
    }
    if (seg == nseg - 1) {  // row group complete: reduce and finish into LDS
      const int lr0 = (wave + j * kWaves) * R;
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const float s = wave_sum(acc[r][b]);
          acc[r][b] = 0.f;
          const int lr = lr0 + r;
          if (lane == 0 && lr < nrows) sy[b * rpw + lr] = apply_epi(s + sb[lr], p.epi, sr[b * rpw + lr]);
        }
      }
    }
  };

  uint4 wa[U][R], wb[U][R];
  float acc[R][B];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[r][b] = 0.f;
  if (ntask > 0) load(0, wa);

  wait();

  // prologue: x, bias and residual of the block into LDS
  {
    const uint16_t* x = (const uint16_t*)p.x;
#pragma unroll 2
    for (int c = tid; c < k8; c += kThreads) {
      uint4 v[B];
#pragma unroll
      for (int b = 0; b < B; ++b) v[b] = load_act16<COH_LOAD>(x + b * p.ldx, (uint32_t)K * 2, (uint32_t)c * 16);
#pragma unroll
      for (int b = 0; b < B; ++b) xs[b * k8 + c] = v[b];
    }
    const uint16_t* bias = (const uint16_t*)p.bias;
    for (int i = tid; i < nrows; i += kThreads) sb[i] = bias ? T::to_f32(gmem(bias)[row_begin + i]) : 0.f;
    if (p.epi == EPI_RESID) {
      const uint16_t* res = (const uint16_t*)p.resid;
#pragma unroll
      for (int b = 0; b < B; ++b) {
        const uint16_t* rrow = res + b * p.ldr + row_begin;
        for (int lr = tid; lr < nrows; lr += kThreads)
          sr[b * rpw + lr] = T::to_f32(load_act1<COH_LOAD>(rrow, (uint32_t)nrows * 2, (uint32_t)lr * 2));
      }
    }
    __syncthreads();
    if (p.ln) {
      float mean[B], rstd[B];
      ln_stats<T, B>([&](int b, int c) { return xs[b * k8 + c]; }, K, mean, rstd, red);
      const bool write_h = p.h_out != nullptr && blk == 0;
      for (int c = tid; c < k8; c += kThreads) {  // each thread rewrites only the chunks it summed
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const uint4 v = normalize8<T>(xs[b * k8 + c], mean[b], rstd[b]);
          xs[b * k8 + c] = v;
          if (write_h) *(uint4*)((uint16_t*)p.h_out + b * p.ldh + (long long)c * 8) = v;
        }
      }
      __syncthreads();
    }
  }

  // main loop, two register buffers: loads of task t+1 are in flight while t is
  // computed.  The loop body issues its loads unconditionally; the last one or two
  // tasks are peeled.
  int t = 0;
  for (; t + 2 < ntask; t += 2) {
    load(t + 1, wb);
    compute(t, wa, acc);
    load(t + 2, wa);
    compute(t + 1, wb, acc);
  }
  if (t + 1 < ntask) {
    load(t + 1, wb);
    compute(t, wa, acc);
    compute(t + 1, wb, acc);
  } else if (t < ntask) {
    compute(t, wa, acc);
  }

  // block outputs: contiguous stores
  __syncthreads();
  const size_t ys = p.y_f32 ? 4 : 2;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    void* yrow = (char*)p.y + ((size_t)b * p.ldy + row_begin) * ys;
    for (int lr = tid; lr < nrows; lr += kThreads)
      store_y_c<T, COH_STORE>(yrow, (uint32_t)nrows, (uint32_t)lr, p.y_f32, sy[b * rpw + lr]);
  }
}

template <class T, int B, int R, int U>
__global__ __launch_bounds__(kThreads) void gemv_kernel(GemvParams p) {
  extern __shared__ uint4 smem[];
  __shared__ float red[2][8][kWaves];
  gemv_block<T, B, R, U, false, false>(p, blockIdx.x, smem, red, [] {});
}

// ---------------------------------------------------------------------------
// GEMV of NB <= 2 batch rows without a fused LayerNorm: x is read straight from
// L1/L2 inside the task loop (it is the same NB*2*K bytes for every wavefront, so
// it stays cached), which removes the LDS prologue and its barrier; the bias and residual
// of a wavefront's rows are loaded once, ahead of its weight stream, into that
// wavefront's slice of LDS, and lane 0 stores each finished row.  Each
// lane accumulates its chunks in the same order as gemv_block, so both kernels
// give bit-identical results.
// ---------------------------------------------------------------------------
template <class T, int U, int NB>
__global__ __launch_bounds__(kThreads) void gemv_x1_kernel(GemvParams p) {
  // per wavefront: bias and residual of its rows (row j of the wave: local row wave + j*kWaves)
  __shared__ float sbias[kWaves][kX1MaxRows], sres[kWaves][NB][kX1MaxRows];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int K = p.K, k8 = K >> 3, rpw = p.rpw;
  const int row_begin = blockIdx.x * rpw;
  const int nrows = min(rpw, p.rows - row_begin);  // >= 1: the grid covers rows exactly
  constexpr int SEG = 64 * U;
  static_assert(SEG * 8 == kSegElems, "a request segment is one segment of the segment-major layout");
  const int nseg = (k8 + SEG - 1) / SEG;
  const int my_rg = nrows > wave ? (nrows - wave + kWaves - 1) / kWaves : 0;  // <= kX1MaxRows (launcher)
  const int ntask = my_rg * nseg;
  const uint16_t* W = (const uint16_t*)p.W;
  const uint16_t* bias = (const uint16_t*)p.bias;
  const uint16_t* res = (const uint16_t*)p.resid;
  // bias and residual first: waiting for them later does not wait for the weights
  float bj = 0.f, rj[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) rj[b] = 0.f;
  if (lane < my_rg) {
    const int row = row_begin + wave + lane * kWaves;
    if (bias) bj = T::to_f32(gmem(bias)[row]);
    if (p.epi == EPI_RESID)
#pragma unroll
      for (int b = 0; b < NB; ++b) rj[b] = T::to_f32(gmem(res)[(long long)b * p.ldr + row]);
  }
  struct Buf {
    uint4 w[U], x[NB][U];
  };
  auto load = [&](int t, Buf& f) {
    const int j = t / nseg, seg = t - j * nseg;
    const int row = row_begin + wave + j * kWaves;
    // segment-major: segment seg of this row at (seg * rows + row) * SEG 16-byte groups
    const uint4* wr = p.segmajor ? (const uint4*)W + ((long long)seg * p.rows + row) * SEG - (long long)seg * SEG
                                 : (const uint4*)(W + (long long)row * K);
    const int c0 = seg * SEG + lane;
#pragma unroll
    for (int u = 0; u < U; ++u) f.w[u] = load_stream(wr + min(c0 + 64 * u, k8 - 1));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const uint4* xb = (const uint4*)((const uint16_t*)p.x + (long long)b * p.ldx);
#pragma unroll
      for (int u = 0; u < U; ++u) f.x[b][u] = load_g16(xb + min(c0 + 64 * u, k8 - 1));
    }
  };
  Buf fa, fb;
  if (ntask > 0) load(0, fa);
  if (lane < my_rg) {
    sbias[wave][lane] = bj;
#pragma unroll
    for (int b = 0; b < NB; ++b) sres[wave][b][lane] = rj[b];
  }
  float acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = 0.f;
  auto compute = [&](int t, const Buf& f) {
    const int j = t / nseg, seg = t - j * nseg;
    const int c0 = seg * SEG + lane;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c0 + 64 * u < k8)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[b] = dot8<T>(f.w[u], f.x[b][u], acc[b]);
    if (seg == nseg - 1) {
      const int row = row_begin + wave + j * kWaves;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float s = wave_sum(acc[b]);
        acc[b] = 0.f;
        if (lane == 0)
          store_y<T>(p.y, (long long)b * p.ldy + row, p.y_f32, apply_epi(s + sbias[wave][j], p.epi, sres[wave][b][j]));
      }
    }
  };
  int t = 0;
  for (; t + 2 < ntask; t += 2) {
    load(t + 1, fb);
    compute(t, fa);
    load(t + 2, fa);
    compute(t + 1, fb);
  }
  if (t + 1 < ntask) {
    load(t + 1, fb);
    compute(t, fa);
    compute(t + 1, fb);
  } else if (t < ntask) {
    compute(t, fa);
  }
}

// ---------------------------------------------------------------------------
// Batch-1 GEMV with a fused LayerNorm for K = 512 * NC (NC <= 14): every wavefront
// loads the whole input row into registers (lane l holds the 16-byte chunks
// l + 64u, exactly the chunks it multiplies in every row), normalises it there and
// keeps it for all its rows: no LDS staging and no workgroup barrier.  The
// statistics are summed in the order of ln_stats and the products in the order of
// gemv_block, so the result is bit-identical to the workgroup kernels.
// ---------------------------------------------------------------------------
template <class T, int NC>
__device__ __forceinline__ void ln_stats_wave(const uint4 (&xv)[NC], int K, float& mean, float& rstd) {
  // "thread" t = 64 w + l of ln_stats sums chunks t + 256 i, i.e. chunks u = w + 4 i of lane l
  float part[kWaves];
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    float s = 0.f;
#pragma unroll
    for (int u = w; u < NC; u += kWaves) {
      float f[8];
      unpack8<T>(xv[u], f);
      s += ((f[0] + f[1]) + (f[2] + f[3])) + ((f[4] + f[5]) + (f[6] + f[7]));
    }
    part[w] = wave_sum(s);
  }
  mean = ((part[0] + part[1]) + (part[2] + part[3])) / (float)K;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    float s = 0.f;
#pragma unroll
    for (int u = w; u < NC; u += kWaves) {
      float f[8];
      unpack8<T>(xv[u], f);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float d = f[e] - mean;
        acc += d * d;
      }
      s += acc;
    }
    part[w] = wave_sum(s);
  }
  const float var = ((part[0] + part[1]) + (part[2] + part[3])) / (float)K;
  rstd = 1.0f / sqrtf(var + kLnEps);
}

template <class T, int NC>
__global__ __launch_bounds__(kThreads) void gemv_ln1_kernel(GemvParams p) {
  __shared__ float sbias[kWaves][kX1MaxRows], sres[kWaves][kX1MaxRows];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int K = p.K, rpw = p.rpw;  // K == 512 * NC (launcher)
  const int row_begin = blockIdx.x * rpw;
  const int nrows = min(rpw, p.rows - row_begin);  // >= 1: the grid covers rows exactly
  const int my_rg = nrows > wave ? (nrows - wave + kWaves - 1) / kWaves : 0;  // <= kX1MaxRows (launcher)
  const uint16_t* W = (const uint16_t*)p.W;
  const uint16_t* bias = (const uint16_t*)p.bias;
  const uint16_t* res = (const uint16_t*)p.resid;
  float bj = 0.f, rj = 0.f;
  if (lane < my_rg) {
    const int row = row_begin + wave + lane * kWaves;
    if (bias) bj = T::to_f32(gmem(bias)[row]);
    if (p.epi == EPI_RESID) rj = T::to_f32(gmem(res)[row]);
  }
  auto load = [&](int j, uint4 (&w)[NC]) {
    const uint4* wr = (const uint4*)(W + (long long)(row_begin + wave + j * kWaves) * K);
#pragma unroll
    for (int u = 0; u < NC; ++u) w[u] = load_stream(wr + lane + 64 * u);
  };
  uint4 wa[NC], wb[NC], xn[NC];
  if (my_rg > 0) load(0, wa);
  const uint4* x = (const uint4*)p.x;
#pragma unroll
  for (int u = 0; u < NC; ++u) xn[u] = load_g16(x + lane + 64 * u);
  if (lane < my_rg) {
    sbias[wave][lane] = bj;
    sres[wave][lane] = rj;
  }
  float mean, rstd;
  ln_stats_wave<T, NC>(xn, K, mean, rstd);
#pragma unroll
  for (int u = 0; u < NC; ++u) xn[u] = normalize8<T>(xn[u], mean, rstd);
  if (p.h_out && blockIdx.x == 0 && wave == 0)
#pragma unroll
    for (int u = 0; u < NC; ++u) *(uint4*)((uint16_t*)p.h_out + (long long)(lane + 64 * u) * 8) = xn[u];
  auto compute = [&](int j, const uint4 (&w)[NC]) {
    float acc = 0.f;
#pragma unroll
    for (int u = 0; u < NC; ++u) acc = dot8<T>(w[u], xn[u], acc);
    const float s = wave_sum(acc);
    if (lane == 0)
      store_y<T>(p.y, row_begin + wave + j * kWaves, p.y_f32, apply_epi(s + sbias[wave][j], p.epi, sres[wave][j]));
  };
  int j = 0;
  for (; j + 2 < my_rg; j += 2) {
    load(j + 1, wb);
    compute(j, wa);
    load(j + 2, wa);
    compute(j + 1, wb);
  }
  if (j + 1 < my_rg) {
    load(j + 1, wb);
    compute(j, wa);
    compute(j + 1, wb);
  } else if (j < my_rg) {
    compute(j, wa);
  }
}

// ---------------------------------------------------------------------------
// Matrix-core GEMV on tile-ordered weights (batches 1..8).  A linear is a product of
// B <= 8 activation rows with N weight rows; v_mfma_f32_16x16x32 takes one 1 KiB tile
// of 16 weight rows x 32 columns as its 16-row operand (one 16-byte load per lane,
// the whole tile in one coalesced instruction) and the matching 32 columns of x as its
// 16-column operand (batch row b in lanes b, b + 16, b + 32, b + 48; the columns past
// B repeat row B - 1 and their results are dropped).  The products and their fp32 sums
// happen in the matrix core, so no lane reduction is needed and the instruction cost
// per weight byte does not grow with B: the kernel stays bound by HBM at every batch
// size, where the vector GEMV becomes bound by its dot products and LDS reads of x.
//
// Workgroup (row tile rt, split g) of 4 wavefronts takes k-tiles of split g of the
// 16 rows; wavefront w a contiguous quarter of them, U tiles per step with the next
// step's loads in flight.  The four 16x16 partial tiles are summed in LDS in wavefront
// order.  With G > 1 splits, each workgroup stores its partial (coherent stores to
// memory: the splits run on different XCDs with their own L2) and the last of the G to
// arrive (an arrival counter, no waiting) adds the G partials in split order, so the
// result does not depend on timing.  Column order inside a tile is free (both
// operands use the same one), so every lane's x fragment is 16 contiguous bytes.
//
// LayerNorm without a launch of its own (LN = true): the linear that produced x (out or
// fc2, this kernel with ln_out) left per-16-row partials of its output; the consumer
// combines them in its prologue, while its first weight tiles are in flight, and
// normalises each x fragment as it multiplies it (one fused multiply-add per element).
// ---------------------------------------------------------------------------
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <class T> struct Mma;
template <> struct Mma<F16> {
  static __device__ __forceinline__ f32x4 run(const uint4& w, const uint4& x, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, w), __builtin_bit_cast(f16x8, x), c, 0, 0,
                                                  0);
  }
};
template <> struct Mma<BF16> {
  static __device__ __forceinline__ f32x4 run(const uint4& w, const uint4& x, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), __builtin_bit_cast(bf16x8, x), c, 0,
                                                   0, 0);
  }
};

// (x - mean) * rstd for 8 packed elements as one fused multiply-add x * a + c (a = rstd,
// c = -mean * rstd), rounded to the activation type: for fp16 a mixed-precision fma that
// reads the halves of a register and writes one half (v_fma_mix{lo,hi}_f16, 8
// instructions), for bf16 fp32 fmas and packed conversions (v_cvt_pk_bf16_f32).  A GEMV
// that normalises every x fragment it multiplies does this once per weight tile.
template <class T> struct NormFma;
template <> struct NormFma<F16> {
  static __device__ __forceinline__ uint32_t two(uint32_t w, float a, float c) {
    const f16x2 h = __builtin_bit_cast(f16x2, w);
    const f16x2 r = {(_Float16)__builtin_fmaf((float)h.x, a, c), (_Float16)__builtin_fmaf((float)h.y, a, c)};
    return __builtin_bit_cast(uint32_t, r);
  }
};
template <> struct NormFma<BF16> {
  static __device__ __forceinline__ uint32_t two(uint32_t w, float a, float c) {
    const f32x2 f = {__builtin_fmaf(__builtin_bit_cast(float, w << 16), a, c),
                     __builtin_fmaf(__builtin_bit_cast(float, w & 0xFFFF0000u), a, c)};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
  }
};
template <class T>
__device__ __forceinline__ uint4 normalize8_fma(const uint4& v, float a, float c) {
  return make_uint4(NormFma<T>::two(v.x, a, c), NormFma<T>::two(v.y, a, c), NormFma<T>::two(v.z, a, c),
                    NormFma<T>::two(v.w, a, c));
}

constexpr int kTileRows = 16, kTileK = 32;
// K-split choice of the matrix-core GEMV (mfma_splits)
constexpr double kMaxUneven = 1.15;  // busiest CU's workgroups over the mean, tolerated unsplit
constexpr int kMaxSplits = 8, kMinSplitTiles = 32;
constexpr int kMaxDevices = 64, kDefaultCus = 256;
constexpr int kMaxKmajorPerCu = 4;  // mfma_kmajor
constexpr int kLnGroup = 16;    // elements per LayerNorm partial
constexpr int kLnSlots = 8;     // batch rows per partial group (the largest batch)
constexpr int kLnMaxGroups = kMaxLnK / kLnGroup;

// LayerNorm statistics of B rows from their partials (see ln_partials_floats): the mean
// is the sum of the group sums over K, and the variance combines each group's squared
// deviations with its count times the squared distance of its mean from the row mean
// (the pairwise combination of Chan, Golub and LeVeque), so no large sums of squares
// are subtracted.  Wavefront w owns batch rows 2w and 2w + 1 (one 16-byte load per
// group holds both rows' pairs): lane l takes groups l + 64 i in increasing i, and the
// lanes are combined in a fixed DPP tree, so every workgroup gets the same bits with no
// reduction across wavefronts; one barrier publishes the statistics.
constexpr int kLnGroupsPerLane = kLnMaxGroups / 64;

template <int B>
__device__ __forceinline__ void ln_partials_load(const float* __restrict__ pt, int K,
                                                 f32x4 (&v)[kLnGroupsPerLane]) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int QG = (K + kLnGroup - 1) / kLnGroup, rounds = (QG + 63) / 64;  // the same for the workgroup
  if (2 * wave >= B) return;
  // a lane past the last group of a round rereads it (the reduction drops it); slot 2w + 1
  // past B holds nothing this launch uses
#pragma unroll
  for (int i = 0; i < kLnGroupsPerLane; ++i)
    if (i < rounds) {
      const int q = min(lane + 64 * i, QG - 1);
      v[i] = *gmem((const f32x4*)(pt + ((size_t)q * kLnSlots + 2 * wave) * 2));
    }
}

template <int B>
__device__ __forceinline__ void ln_partials_reduce(const f32x4 (&v)[kLnGroupsPerLane], int K,
                                                   float (*st)[2]) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int QG = (K + kLnGroup - 1) / kLnGroup, rounds = (QG + 63) / 64;
  if (2 * wave < B) {
    const float inv_k = 1.0f / (float)K;
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int i = 0; i < kLnGroupsPerLane; ++i)
      if (i < rounds && lane + 64 * i < QG) {
        s0 += v[i].x;
        s1 += v[i].z;
      }
    const float m0 = wave_sum(s0) * inv_k, m1 = wave_sum(s1) * inv_k;
    float t0 = 0.f, t1 = 0.f;
#pragma unroll
    for (int i = 0; i < kLnGroupsPerLane; ++i) {
      const int q = lane + 64 * i;
      if (i < rounds && q < QG) {
        // a group holds 16 elements, or 8 (the last one when K % 16 == 8; K % 8 == 0): its
        // mean is its sum times an exact power-of-two reciprocal
        const bool full = K - kLnGroup * q >= kLnGroup;
        const float n = full ? (float)kLnGroup : 8.f, inv_n = full ? 1.f / kLnGroup : 0.125f;
        const float d0 = v[i].x * inv_n - m0, d1 = v[i].z * inv_n - m1;
        t0 += v[i].y + n * d0 * d0;
        t1 += v[i].w + n * d1 * d1;
      }
    }
    t0 = wave_sum(t0);
    t1 = wave_sum(t1);
    if (lane == 0) {
      st[2 * wave][0] = m0;
      st[2 * wave][1] = 1.0f / sqrtf(t0 * inv_k + kLnEps);
      if (2 * wave + 1 < B) {
        st[2 * wave + 1][0] = m1;
        st[2 * wave + 1][1] = 1.0f / sqrtf(t1 * inv_k + kLnEps);
      }
    }
  }
  __syncthreads();
}

template <class T, int B, int U, bool LN>
__global__ __launch_bounds__(kThreads) void gemv_mfma_kernel(GemvParams p, int G) {
  __shared__ float part[kWaves][4][64];
  __shared__ float lnst[kLnSlots][2];  // LN: mean and 1 / sqrt(var + eps) of each batch row
  __shared__ int last;
  // the wavefront index through a scalar register: every tile bound below is then
  // wave-uniform and the skipped products are skipped by a branch.  A condition the
  // compiler cannot prove uniform becomes an execution mask, which matrix-core
  // instructions do not obey (they would run for every skipped tile).
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int K = p.K, KT = (K + kTileK - 1) / kTileK;
  const int rt = blockIdx.x / G, gi = blockIdx.x - rt * G;
  const int kg = (KT + G - 1) / G;
  const int kb = min(KT, gi * kg), ke = min(KT, kb + kg);
  const int pw = (ke - kb + kWaves - 1) / kWaves;
  const int k0 = min(ke, kb + wave * pw), k1 = min(ke, k0 + pw);
  const int nst = (k1 - k0 + U - 1) / U;
  // k-tile kt of row tile rt: tile rt * KT + kt (row-tile order) or kt * RT + rt (k-major)
  const size_t RT = (size_t)((p.rows + kTileRows - 1) / kTileRows);
  const uint4* wp = (const uint4*)p.W + (p.korder ? (size_t)rt : (size_t)rt * KT) * 64 + lane;
  const size_t kstride = p.korder ? RT * 64 : 64;
  const int b = min(lane & 15, B - 1), grp = lane >> 4;
  // x fragments through a buffer descriptor over rows [0, B) of x: a lane whose result
  // column is past B (its products are never read), a group past K and the repeated tile
  // of a step past k1 get an offset past the descriptor's size, for which the load
  // returns zeros without a memory access; at B = 8 that halves the x fragments' share of
  // the load pipeline, and no branch is needed (a branch around the loads makes the
  // compiler wait for the weights in flight)
  const auto xrs = rsrc(p.x, (uint32_t)(((long long)(B - 1) * p.ldx + K) * 2));
  const bool xlane = (lane & 15) < B;
  const uint32_t xrow = (uint32_t)((long long)b * p.ldx * 2);
  struct Buf {
    uint4 w[U], x[U];
  };
  auto load = [&](int st, Buf& f) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = min(k0 + st * U + u, k1 - 1);
      f.w[u] = load_stream(wp + (size_t)kt * kstride);
      const int kx = kt * kTileK + 8 * grp;  // K % 8 == 0: a group is wholly inside or past K
      const bool in = xlane & (kx < K) & (k0 + st * U + u < k1);  // no short circuit: no branch
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(xrs, in ? xrow + 2u * kx : kXPast, 0, 0);
      f.x[u] = make_uint4(v.x, v.y, v.z, v.w);
    }
  };
  // LayerNorm of x on the fly: xn = x * ln_a + ln_c for this lane's batch row
  float ln_a = 0.f, ln_c = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int st, const Buf& f) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = k0 + st * U + u;
      if (kt < k1) {
        uint4 xv = f.x[u];
        if (LN) {
          xv = normalize8_fma<T>(xv, ln_a, ln_c);
          // columns past K (only in the last k-tile when K % 32 != 0) multiply zeros
          if ((K & (kTileK - 1)) && kt == KT - 1 && kt * kTileK + 8 * grp >= K) xv = make_uint4(0u, 0u, 0u, 0u);
        }
        acc = Mma<T>::run(f.w[u], xv, acc);
      }
    }
  };
  Buf fa, fb;
  // the LayerNorm partials are requested before the first weights, so that waiting for
  // them leaves the weight loads in flight
  f32x4 lnv[LN ? kLnGroupsPerLane : 1];
  if constexpr (LN) {
    ln_partials_load<B>(p.ln_in, K, lnv);
    __builtin_amdgcn_sched_barrier(0);  // keep them ahead of the weight loads
  }
  // (with the LayerNorm the first loads are unconditional, for the same reason; a
  // wavefront without tiles rereads tile k1 - 1 >= 0 and computes nothing)
  if (LN || nst > 0) load(0, fa);
  if constexpr (LN) {
    ln_partials_reduce<B>(lnv, K, lnst);
    ln_a = lnst[b][1];
    ln_c = -lnst[b][0] * lnst[b][1];
    if (p.h_out && blockIdx.x == 0) {
      // the normalised input, for a caller that records it
      const int n8 = K >> 3;
      for (int c = threadIdx.x; c < B * n8; c += kThreads) {
        const int r = c / n8, cc = c - r * n8;
        const uint4 xv = load_g16((const uint4*)((const uint16_t*)p.x + (long long)r * p.ldx + 8 * cc));
        *(uint4*)((uint16_t*)p.h_out + (long long)r * p.ldh + 8 * cc) =
            normalize8_fma<T>(xv, lnst[r][1], -lnst[r][0] * lnst[r][1]);
      }
    }
  }
  int st = 0;
  for (; st + 2 < nst; st += 2) {
    load(st + 1, fb);
    compute(st, fa);
    load(st + 2, fa);
    compute(st + 1, fb);
  }
  if (st + 1 < nst) {
    load(st + 1, fb);
    compute(st, fa);
    compute(st + 1, fb);
  } else if (st < nst) {
    compute(st, fa);
  }
  // lane l of the result holds rows 4 (l / 16) + v, v < 4, of column l % 16
#pragma unroll
  for (int v = 0; v < 4; ++v) part[wave][v][lane] = acc[v];
  __syncthreads();
  const int t = threadIdx.x, i = t & 15, j = t >> 4;  // row i of the tile, batch row j
  const bool mine = t < 16 * B;
  const int l = j + 16 * (i >> 2), v = i & 3;
  float s = 0.f;
  if (mine) s = (part[0][v][l] + part[1][v][l]) + (part[2][v][l] + part[3][v][l]);
  if (G > 1) {
    const uint32_t pbytes = (uint32_t)(G * 16 * B * sizeof(float));
    const auto rs = rsrc(p.ws + (size_t)rt * G * 16 * B, pbytes);
    if (mine)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, s), rs, (gi * 16 * B + t) * 4, 0,
                                            kCoherent);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's partial store has completed
    __syncthreads();
    if (t == 0) {
      const uint32_t prev = __hip_atomic_fetch_add(p.cnt + rt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last = prev == (uint32_t)(G - 1);
      if (last) __hip_atomic_store(p.cnt + rt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next launch
    }
    __syncthreads();
    if (!last) return;
    if (mine) {
      s = 0.f;
      for (int q = 0; q < G; ++q)
        s += __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (q * 16 * B + t) * 4, 0, kCoherent));
    }
  }
  const int row = rt * kTileRows + i;
  const bool valid = mine && row < p.rows;
  float yv = 0.f;
  if (valid) {
    const uint16_t* bias = (const uint16_t*)p.bias;
    const float y = s + (bias ? T::to_f32(bias[row]) : 0.f);
    const float rv = p.epi == EPI_RESID ? T::to_f32(((const uint16_t*)p.resid)[j * p.ldr + row]) : 0.f;
    yv = apply_epi(y, p.epi, rv);
    store_y<T>(p.y, j * p.ldy + row, p.y_f32, yv);
  }
  // LayerNorm partials of this row tile's outputs for the next linear: a row of 16
  // lanes holds the 16 rows of one batch row (lanes past 16 B hold none)
  if (!p.ln_out || wave * 64 >= 16 * B) return;
  const float n = (float)min(kTileRows, p.rows - rt * kTileRows);
  const float a = valid ? T::to_f32(round_act<T>(yv)) : 0.f;
  const float s1 = row16_sum(a);
  const float d = valid ? a - s1 / n : 0.f;
  const float m2 = row16_sum(d * d);
  if (mine && i == 0) *(f32x2*)(p.ln_out + ((size_t)rt * kLnSlots + j) * 2) = f32x2{s1, m2};
}

// Tile order of W [rows, K]: one 16-byte group per thread (see tiled_bytes in kernels.h).
__global__ __launch_bounds__(kThreads) void tile_kernel(const uint16_t* __restrict__ W, long long ldw, int rows,
                                                        int K, uint4* __restrict__ dst, long long groups, int korder) {
  const int KT = (K + kTileK - 1) / kTileK;
  const long long RT = (rows + kTileRows - 1) / kTileRows;
  for (long long q = (long long)blockIdx.x * kThreads + threadIdx.x; q < groups;
       q += (long long)gridDim.x * kThreads) {
    const int l = (int)(q & 63);
    const long long tile = q >> 6;
    const int kt = korder ? (int)(tile / RT) : (int)(tile % KT);
    const long long rt = korder ? tile % RT : tile / KT;
    const long long row = rt * kTileRows + (l & 15);
    const int k = kt * kTileK + 8 * (l >> 4);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < rows && k < K) v = *(const uint4*)(W + row * ldw + k);
    dst[q] = v;
  }
}

// ---------------------------------------------------------------------------
// Persistent decode step: one cooperative launch runs every linear of the step,
// each workgroup taking the same row block of every linear, with a grid barrier
// between dependent linears.  A workgroup requests the weights of its first
// task of linear i+1 before it waits at the barrier of linear i, so HBM keeps
// streaming through the barrier and the next prologue.
// Barrier: workgroups arrive on one of `ngroups` counters (blockIdx % ngroups);
// the last arrival of a group bumps the top counter, which the waiting
// workgroups poll.  Counters only grow (wrap-safe comparisons); barrier n of the
// model's lifetime completes when the top counter reaches (n + 1) * ngroups.
// The wait gives up after a bounded number of polls, records the failure in
// `err` and lets the kernel run to its end, so the grid always drains.
// ---------------------------------------------------------------------------
constexpr int kCounterStride = 64;  // uint32 words: one 256-byte line per counter

__device__ __forceinline__ bool reached(uint32_t v, uint32_t target) { return (int32_t)(v - target) >= 0; }

__device__ __forceinline__ void grid_arrive(const StepArgs& a, uint32_t n) {
  // every thread's output stores have completed (coherent stores: visible device-wide)
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int g = blockIdx.x % a.ngroups;
    const uint32_t gsize = gridDim.x / a.ngroups + ((uint32_t)g < gridDim.x % a.ngroups ? 1u : 0u);
    const uint32_t old =
        __hip_atomic_fetch_add(a.counters + g * kCounterStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1u == (n + 1u) * gsize)
      __hip_atomic_fetch_add(a.counters + a.ngroups * kCounterStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ void grid_wait(const StepArgs& a, uint32_t n) {
  if (threadIdx.x == 0) {
    const uint32_t target = (n + 1u) * (uint32_t)a.ngroups;
    const uint32_t* top = a.counters + a.ngroups * kCounterStride;
    uint32_t spins = 0;
    while (!reached(__hip_atomic_load(top, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), target)) {
      if (++spins > a.spin_limit) {
        __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  __syncthreads();
}

template <class T, int B, int R, int U>
__global__ __launch_bounds__(kThreads) void step_kernel(StepArgs a) {
  extern __shared__ uint4 smem[];
  __shared__ float red[2][8][kWaves];
  for (int i = 0; i < a.nlin; ++i) {
    const StepLinear& d = a.lin[i];
    GemvParams p{};
    p.x = d.x_in ? a.x_in : d.x;
    p.ldx = d.ldx;
    p.W = d.W;
    p.bias = d.bias;
    p.y = d.y_out ? a.out : d.y;
    p.ldy = d.ldy;
    p.resid = d.resid_in ? a.x_in : d.resid;
    p.ldr = d.ldr;
    p.rows = d.rows;
    p.K = d.K;
    p.epi = d.epi;
    p.ln = d.ln;
    p.rpw = d.rpw;
    p.segmajor = d.segmajor;
    const uint32_t n = a.barrier_base + (uint32_t)i;
    gemv_block<T, B, R, U, true, true>(p, blockIdx.x, smem, red, [&] {
      if (i > 0) grid_wait(a, n - 1u);
    });
    grid_arrive(a, n);
  }
}

// ---------------------------------------------------------------------------
// K-tiled GEMV for x that does not fit in LDS: x is restaged per K tile and row
// group (grid-stride over row groups).  No fused LayerNorm: a LayerNorm input fits in
// LDS at the batches that fuse it (B <= 4, hidden size <= kMaxLnK).
// ---------------------------------------------------------------------------
template <int B>
__device__ __forceinline__ void stage_x_tile(const GemvParams& p, uint4* xs, int k0, int kn) {
  const uint16_t* x = (const uint16_t*)p.x;
  const int n8 = kn >> 3, kt8 = p.ktile >> 3;
  for (int c = threadIdx.x; c < n8; c += kThreads) {
    uint4 v[B];
#pragma unroll
    for (int b = 0; b < B; ++b) v[b] = *(const uint4*)(x + b * p.ldx + k0 + (long long)c * 8);
#pragma unroll
    for (int b = 0; b < B; ++b) xs[b * kt8 + c] = v[b];
  }
}

template <class T, int B, int R, int U>
__global__ __launch_bounds__(kThreads) void gemv_tiled_kernel(GemvParams p) {
  extern __shared__ uint4 xs[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int K = p.K, ktile = p.ktile, kt8 = ktile >> 3;
  const int ntiles = (K + ktile - 1) / ktile;
  const int nrg = (p.rows + R - 1) / R;
  const uint16_t* W = (const uint16_t*)p.W;
  const uint16_t* bias = (const uint16_t*)p.bias;
  for (int rg0 = blockIdx.x * kWaves; rg0 < nrg; rg0 += gridDim.x * kWaves) {
    const int rg = rg0 + wave;
    const bool valid = rg < nrg;  // uniform per wavefront
    const int row0 = rg * R;
    const uint4* wp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) wp[r] = (const uint4*)(W + (long long)min(row0 + r, p.rows - 1) * K);
    float acc[R][B];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int b = 0; b < B; ++b) acc[r][b] = 0.f;
    for (int t = 0; t < ntiles; ++t) {
      const int k0 = t * ktile, kn = min(ktile, K - k0);
      __syncthreads();
      stage_x_tile<B>(p, xs, k0, kn);
      __syncthreads();
      if (valid) {
        const int n8 = kn >> 3, c0 = k0 >> 3;
        int c = lane;
        for (; c + 64 * (U - 1) < n8; c += 64 * U) {
          uint4 w[U][R];
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) w[u][r] = load_stream(wp[r] + c0 + c + 64 * u);
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int b = 0; b < B; ++b) {
              const uint4 xv = xs[b * kt8 + c + 64 * u];
#pragma unroll
              for (int r = 0; r < R; ++r) acc[r][b] = dot8<T>(w[u][r], xv, acc[r][b]);
            }
        }
        for (; c < n8; c += 64) {
          uint4 w[R];
#pragma unroll
          for (int r = 0; r < R; ++r) w[r] = load_stream(wp[r] + c0 + c);
#pragma unroll
          for (int b = 0; b < B; ++b) {
            const uint4 xv = xs[b * kt8 + c];
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
            const float rv = p.epi == EPI_RESID ? T::to_f32(((const uint16_t*)p.resid)[b * p.ldr + row]) : 0.f;
            store_y<T>(p.y, b * p.ldy + row, p.y_f32, apply_epi(s, p.epi, rv));
          }
        }
      }
    }
  }
}

// LayerNorm of a materialised input, one batch row per blockIdx.y (the statistics of a
// row are the same bits whatever the batch), the row held in registers (thread t keeps
// chunks t + 256 i, the chunks ln_stats gives it, for i < NI): every sum is formed in
// ln_stats' order, so the bits are those of the GEMVs that fuse the LayerNorm.
template <class T, int NI>
__global__ __launch_bounds__(kThreads) void layernorm_regs_kernel(const uint16_t* __restrict__ x, long long ldx,
                                                                  int K, uint16_t* __restrict__ h, long long ldh,
                                                                  float* __restrict__ h_host) {
  __shared__ float red[2][kWaves];
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint16_t* xr = x + b * ldx;
  const int n8 = K >> 3;  // <= kThreads * NI (launcher)
  uint4 v[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = tid + kThreads * i;
    v[i] = c < n8 ? *(const uint4*)(xr + (long long)c * 8) : make_uint4(0u, 0u, 0u, 0u);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    if (tid + kThreads * i < n8) {
      float f[8];
      unpack8<T>(v[i], f);
      s += ((f[0] + f[1]) + (f[2] + f[3])) + ((f[4] + f[5]) + (f[6] + f[7]));
    }
  }
  s = wave_sum(s);
  if (lane == 0) red[0][wave] = s;
  __syncthreads();
  const float mean = ((red[0][0] + red[0][1]) + (red[0][2] + red[0][3])) / (float)K;
  s = 0.f;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    if (tid + kThreads * i < n8) {
      float f[8];
      unpack8<T>(v[i], f);
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float d = f[e] - mean;
        acc += d * d;
      }
      s += acc;
    }
  }
  s = wave_sum(s);
  if (lane == 0) red[1][wave] = s;
  __syncthreads();
  const float var = ((red[1][0] + red[1][1]) + (red[1][2] + red[1][3])) / (float)K;
  const float rstd = 1.0f / sqrtf(var + kLnEps);
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int c = tid + kThreads * i;
    if (c < n8) {
      const uint4 o = normalize8<T>(v[i], mean, rstd);
      *(uint4*)(h + b * ldh + (long long)c * 8) = o;
      if (h_host) {
        float f[8];
        unpack8<T>(o, f);
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
    const float rv = epi == EPI_RESID ? T::to_f32(((const uint16_t*)resid)[b * ldr + c]) : 0.f;
    store_y<T>(y, b * ldy + c, y_f32, apply_epi(src[i], epi, rv));
  }
}

// Per-batch tiling: rows per wavefront R and 16-byte steps per task U (U*R loads in flight).
template <int B> struct Tile;
// (Measured on OPT-6.7B/13B shapes: one row per wavefront up to B = 4, two from B = 5.)
template <> struct Tile<1> { static constexpr int R = 1, U = 8; };
template <> struct Tile<2> { static constexpr int R = 1, U = 8; };
template <> struct Tile<3> { static constexpr int R = 1, U = 4; };
template <> struct Tile<4> { static constexpr int R = 1, U = 4; };
template <> struct Tile<5> { static constexpr int R = 2, U = 2; };
template <> struct Tile<6> { static constexpr int R = 2, U = 2; };
template <> struct Tile<7> { static constexpr int R = 2, U = 2; };
template <> struct Tile<8> { static constexpr int R = 2, U = 2; };

constexpr size_t kLdsMain = 65536 - 1024;  // dynamic LDS of the persistent step (x, bias, residual, outputs)

// LDS a workgroup of the per-linear main GEMV may use on this device (gfx950: 160 KiB
// per CU, all of it addressable by one workgroup), less a margin for the static
// arrays; and the LDS of one CU, which bounds the co-resident workgroups.
struct LdsInfo {
  size_t per_block = 65536, per_cu = 65536;
  int cus = 1;
};
const LdsInfo& lds_info() {
  static const LdsInfo info = [] {
    LdsInfo i;
    int dev = 0, blk = 0, cu = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&blk, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess &&
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && blk > 0 && cu > 0 &&
        n > 0) {
      i.per_block = (size_t)blk;
      i.per_cu = (size_t)cu;
      i.cus = n;
    }
    (void)hipGetLastError();
    return i;
  }();
  return info;
}
constexpr int kTiledLdsBudget = 32768;  // bytes of x per tile in the K-tiled kernel
constexpr int kDefaultGridCap = 1024;

// Batches up to this size run linears without a fused LayerNorm on gemv_x1_kernel (x
// read per wavefront from L1/L2) rather than staging x in LDS per workgroup (OPT-6.7B
// shapes at B = 2: out 9.3 -> 8.6 us, fc2 25.9 -> 25.3 us; slower from B = 3 on, and
// the register LayerNorm kernel only pays at B = 1).
constexpr int kX1MaxB = 2;

template <class T, int B>
hipError_t launch_gemv_b(GemvParams p, hipStream_t s, int grid_cap) {
  constexpr int R = Tile<B>::R, U = Tile<B>::U;
  const int cap = grid_cap > 0 ? grid_cap : kDefaultGridCap;
  if constexpr (B <= kX1MaxB) {
    // K = 512 * NC for the NC instantiated below (hidden sizes of OPT-350M .. OPT-30B); at
    // NC = 18 (9216) the row no longer fits the registers well and the LDS kernel is as fast
    const int nc = p.K % 512 == 0 ? p.K / 512 : 0;
    const bool ln_regs = B == 1 && p.ln && (nc == 1 || nc == 2 || nc == 4 || nc == 5 || nc == 8 || nc == 10 || nc == 14);
    // segment-major weights: gemv_x1_kernel and gemv_block (below) read them, the register
    // LayerNorm kernel does not
    if (p.segmajor && ln_regs) return hipErrorInvalidValue;
    if (!p.ln || ln_regs) {
      const long long units = (p.rows + kWaves - 1) / kWaves;
      const long long per = std::min<long long>((units + cap - 1) / cap, kX1MaxRows);
      p.rpw = (int)(per * kWaves);
      const int grid = (int)((p.rows + p.rpw - 1) / p.rpw);
      if (!p.ln) hipLaunchKernelGGL((gemv_x1_kernel<T, 4, B>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 1) hipLaunchKernelGGL((gemv_ln1_kernel<T, 1>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 2) hipLaunchKernelGGL((gemv_ln1_kernel<T, 2>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 4) hipLaunchKernelGGL((gemv_ln1_kernel<T, 4>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 5) hipLaunchKernelGGL((gemv_ln1_kernel<T, 5>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 8) hipLaunchKernelGGL((gemv_ln1_kernel<T, 8>), dim3(grid), dim3(kThreads), 0, s, p);
      else if (nc == 10) hipLaunchKernelGGL((gemv_ln1_kernel<T, 10>), dim3(grid), dim3(kThreads), 0, s, p);
      else hipLaunchKernelGGL((gemv_ln1_kernel<T, 14>), dim3(grid), dim3(kThreads), 0, s, p);
      return hipGetLastError();
    }
  }
  // contiguous row blocks of a multiple of R*kWaves rows, at most `cap` blocks; a block
  // that needs much LDS also caps the grid at the workgroups that fit at once (more
  // would run in a second round)
  const int unit = R * kWaves;
  const long long units = (p.rows + unit - 1) / unit;
  const LdsInfo& li = lds_info();
  const size_t lds_max = li.per_block - 1024;
  auto block_lds = [&](int c) {
    const long long per = (units + c - 1) / c;
    return (size_t)B * p.K * 2 + (size_t)(1 + 2 * B) * (size_t)(per * unit) * 4;  // gemv_lds_bytes
  };
  int cap_b = cap;
  const size_t lds0 = block_lds(cap_b);
  if (lds0 <= lds_max) {
    const long long fit = (long long)li.cus * (long long)std::max<size_t>(1, li.per_cu / lds0);
    if (fit < cap_b && block_lds((int)std::max<long long>(1, fit)) <= lds_max)
      cap_b = (int)std::max<long long>(1, fit);
    const long long per = (units + cap_b - 1) / cap_b;
    const int rpw = (int)(per * unit);
    const size_t lds = block_lds(cap_b);
    if (lds > 65536) {  // beyond the default dynamic LDS: opt in once per kernel
      static const hipError_t opt = hipFuncSetAttribute((const void*)gemv_kernel<T, B, R, U>,
                                                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_max);
      if (opt != hipSuccess) return opt;
    }
    p.rpw = rpw;
    p.ktile = p.K;
    const int grid = (int)((p.rows + rpw - 1) / rpw);
    hipLaunchKernelGGL((gemv_kernel<T, B, R, U>), dim3(grid), dim3(kThreads), lds, s, p);
    return hipGetLastError();
  }
  if (p.ln) return hipErrorInvalidValue;  // not reached: see gemv_tiled_kernel
  if (p.segmajor) return hipErrorInvalidValue;  // gemv_tiled_kernel reads row-major weights
  int kt = kTiledLdsBudget / (2 * B);
  kt -= kt % 512;
  p.ktile = kt;
  const int nrg = (p.rows + R - 1) / R;
  int grid = (nrg + kWaves - 1) / kWaves;
  if (grid > cap) grid = cap;
  hipLaunchKernelGGL((gemv_tiled_kernel<T, B, R, U>), dim3(grid), dim3(kThreads), (size_t)B * kt * 2, s, p);
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

template <class T, int NI>
hipError_t launch_ln_regs(int B, const uint16_t* x, long long ldx, int K, uint16_t* h, long long ldh, float* hh,
                          hipStream_t s) {
  hipLaunchKernelGGL((layernorm_regs_kernel<T, NI>), dim3(1, B), dim3(kThreads), 0, s, x, ldx, K, h, ldh, hh);
  return hipGetLastError();
}

template <class T>
hipError_t launch_ln_t(const void* x, long long ldx, int B, int K, void* h, long long ldh, float* hh, hipStream_t s) {
  if (B < 1 || B > 8) return hipErrorInvalidValue;
  const int n8 = K >> 3;
  // rows of up to 8 * kThreads * 8 elements (hidden sizes up to kMaxLnK) stay in registers
  const int ni = (n8 + kThreads - 1) / kThreads;
  const uint16_t* xx = (const uint16_t*)x;
  uint16_t* hp = (uint16_t*)h;
  switch (ni) {
    case 1: return launch_ln_regs<T, 1>(B, xx, ldx, K, hp, ldh, hh, s);
    case 2: return launch_ln_regs<T, 2>(B, xx, ldx, K, hp, ldh, hh, s);
    case 3: return launch_ln_regs<T, 3>(B, xx, ldx, K, hp, ldh, hh, s);
    case 4: return launch_ln_regs<T, 4>(B, xx, ldx, K, hp, ldh, hh, s);
    case 5: return launch_ln_regs<T, 5>(B, xx, ldx, K, hp, ldh, hh, s);
    case 6:
    case 7:
    case 8: return launch_ln_regs<T, 8>(B, xx, ldx, K, hp, ldh, hh, s);
    default: return hipErrorInvalidValue;  // K > kMaxLnK
  }
}

// The persistent step runs the row-major copy, which only batch 1 uses (models created for
// larger batches run batches from 2 on their matrix-core tiles; the batch-2 instance is
// not launched by the library).
template <class T>
const void* step_fn(int B) {
  switch (B) {
    case 1: return (const void*)step_kernel<T, 1, Tile<1>::R, Tile<1>::U>;
    case 2: return (const void*)step_kernel<T, 2, Tile<2>::R, Tile<2>::U>;
  }
  return nullptr;
}

int small_grid(long long work_items) {
  long long g = (work_items + kThreads - 1) / kThreads;
  if (g < 1) g = 1;
  if (g > 256) g = 256;
  return (int)g;
}

}  // namespace

int gemv_rows_unit(int B) {
  static const int r[9] = {0, Tile<1>::R, Tile<2>::R, Tile<3>::R, Tile<4>::R,
                           Tile<5>::R, Tile<6>::R, Tile<7>::R, Tile<8>::R};
  return (B >= 1 && B <= 8) ? r[B] : 0;
}

size_t gemv_lds_bytes(int B, int K, int rows_per_block) {
  return (size_t)B * K * 2 + (size_t)(1 + 2 * B) * rows_per_block * 4;
}

size_t gemv_lds_limit() { return kLdsMain; }

// Measured on OPT-6.7B shapes: from B = 5 on, normalising x once per workgroup in the
// prologue costs more than a separate LayerNorm launch.
bool gemv_fuses_ln(int B) { return B <= 4; }

int step_blocks_per_cu(int dtype, int B, size_t lds) {
  const void* f = dtype == 1 ? step_fn<BF16>(B) : step_fn<F16>(B);
  if (!f) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, kThreads, lds) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return n;
}

hipError_t launch_step(const StepArgs& a, int dtype, int B, int grid, size_t lds, hipStream_t stream) {
  const void* f = dtype == 1 ? step_fn<BF16>(B) : step_fn<F16>(B);
  if (!f) return hipErrorInvalidValue;
  StepArgs args = a;
  void* kargs[] = {(void*)&args};
  return hipLaunchCooperativeKernel(f, dim3(grid), dim3(kThreads), kargs, (unsigned)lds, stream);
}

hipError_t launch_gemv(GemvParams p, int dtype, int B, hipStream_t stream, int grid_cap) {
  if (p.rows <= 0) return hipSuccess;
  if (p.segmajor && (B != 1 || p.K % kSegElems)) return hipErrorInvalidValue;
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

size_t tiled_bytes(int rows, int K) {
  if (rows <= 0 || K <= 0) return 0;
  return (size_t)((rows + kTileRows - 1) / kTileRows) * (size_t)((K + kTileK - 1) / kTileK) * 1024;
}

// Segment-major copy (see launch_segmajor): one 16-byte group per thread.
__global__ __launch_bounds__(kThreads) void segmajor_kernel(const uint4* __restrict__ W, int rows, int k8,
                                                            uint4* __restrict__ dst, long long n) {
  constexpr int SEG = kSegElems / 8;
  for (long long q = (long long)blockIdx.x * kThreads + threadIdx.x; q < n; q += (long long)gridDim.x * kThreads) {
    const long long s = q / ((long long)rows * SEG), rem = q - s * rows * SEG, r = rem / SEG, i = rem - r * SEG;
    dst[q] = W[r * k8 + s * SEG + i];
  }
}

hipError_t launch_segmajor(const void* W, int rows, int K, void* dst, hipStream_t stream) {
  if (rows <= 0 || K <= 0 || K % kSegElems) return hipErrorInvalidValue;
  const long long n = (long long)rows * (K / 8);
  long long g = std::min<long long>((n + kThreads - 1) / kThreads, 4096);
  hipLaunchKernelGGL(segmajor_kernel, dim3((unsigned)g), dim3(kThreads), 0, stream, (const uint4*)W, rows, K / 8,
                     (uint4*)dst, n);
  return hipGetLastError();
}

hipError_t launch_tile(const void* W, long long ldw, int rows, int K, void* dst, hipStream_t stream, int korder) {
  const long long groups = (long long)(tiled_bytes(rows, K) / 16);
  if (groups == 0) return hipSuccess;
  long long g = (groups + kThreads - 1) / kThreads;
  if (g > 4096) g = 4096;
  hipLaunchKernelGGL(tile_kernel, dim3((unsigned)g), dim3(kThreads), 0, stream, (const uint16_t*)W, ldw, rows, K,
                     (uint4*)dst, groups, korder);
  return hipGetLastError();
}

// Compute units of the current device (read once per device).
static int device_cus() {
  static std::atomic<int> cus[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return kDefaultCus;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c < 1) c = kDefaultCus;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// How unevenly `wgs` equal workgroups load `cus` compute units: the busiest unit's
// workgroups over the mean (1 when wgs is a multiple of cus).
static double uneven(long long wgs, int cus) {
  const long long per = (wgs + cus - 1) / cus;
  return (double)(per * cus) / (double)wgs;
}

// One row tile per workgroup unless that loads the CUs unevenly (more than 1.15x the
// mean on the busiest); then the fewest splits that do not, each at least 32 k-tiles
// long, or else the most even split.  Splitting a balanced grid only adds the merge:
// OPT-6.7B fc2 [4096, 16384] (256 row tiles) at B = 8 takes 23.9 us unsplit against
// 26.2 us in 4 splits; OPT-13B fc2 [5120, 20480] (320 row tiles) 49.4 unsplit against
// 39.1 us in 4 splits.  Over the 16 linear shapes of OPT-6.7B/13B/30B/66B at B = 1, 2, 3
// and 8 the rule picks the fastest split count but at B = 8 for OPT-13B out [5120, 5120]
// (4 splits: 15.5 against 14.8 us with 2) and OPT-66B fc2 [9216, 36864] (2 splits: 117.3
// against 114.0 us with 4).  The choice does not depend on B, so a batch row's bits do not
// either.
int mfma_splits(int rows, int K) {
  if (rows <= 0 || K <= 0) return 1;
  const int KT = (K + kTileK - 1) / kTileK, RT = (rows + kTileRows - 1) / kTileRows, cus = device_cus();
  double best_u = uneven(RT, cus);
  if (best_u <= kMaxUneven) return 1;
  int best = 1;
  for (int g = 2; g <= kMaxSplits && KT / g >= kMinSplitTiles; g *= 2) {
    const double u = uneven((long long)RT * g, cus);
    if (u <= kMaxUneven) return g;
    if (u < best_u) {
      best = g;
      best_u = u;
    }
  }
  return best;
}

// k-major tiles when the grid puts the same number of workgroups, 1 to 4, on every CU: all
// of them then start together and walk K side by side, and in row-tile order their loads
// would fall on the same offsets of blocks a fixed multiple of 16 rows apart, crowding a few
// memory channels (OPT-6.7B fc2 [4096, 16384] at B = 8: 23.9 against 25.5 us in a decode
// step, and the whole step 2.42 against 2.49 ms); k-major, the walk reads one contiguous
// window.  With more workgroups per CU, or uneven ones, they drift apart and k-major
// scatters the loads instead (OPT-30B fc1 [28672, 7168], 7 per CU: 72.8 against 70.5 us).
int mfma_kmajor(int rows, int K) {
  if (rows <= 0 || K <= 0) return 0;
  const long long wgs = (long long)((rows + kTileRows - 1) / kTileRows) * mfma_splits(rows, K);
  const int cus = device_cus();
  return wgs % cus == 0 && wgs / cus <= kMaxKmajorPerCu ? 1 : 0;
}

size_t mfma_ws_floats(int rows, int K, int B) {
  const int G = mfma_splits(rows, K);
  if (G == 1 || rows <= 0) return 0;
  return (size_t)((rows + kTileRows - 1) / kTileRows) * G * kTileRows * B;
}

size_t mfma_cnt_words(int rows, int K) {
  if (mfma_splits(rows, K) == 1 || rows <= 0) return 0;
  return (size_t)((rows + kTileRows - 1) / kTileRows);
}

// Tiles per request: 4 in split launches and with the LayerNorm prologue (fewer registers)
// from B = 2 on or when the grid puts more than 3 workgroups on a CU (142-146 VGPRs with 8
// allow 3 wavefronts per SIMD); 8 otherwise.  Measured on OPT-6.7B shapes: fc2 [4096,
// 16384] took 4 while every lane of the product loaded x (24.6 against 23.9 us at B = 8),
// and 8 since lanes of columns past B load none (whole steps 2.354-2.357 against
// 2.383-2.385 ms at B = 8; OPT-30B fc2 [7168, 28672] unchanged); qkv with the prologue at
// B = 8 with 8: 2.370-2.374 against 2.356-2.357 ms per step; at B = 1 on tiles (a model
// without the row-major copy), 8 for every unsplit linear but fc1 (4 workgroups per CU):
// 2.260-2.265 against 2.279-2.282 ms.  Each wavefront sums its k-tiles in order either way:
// the bits are the same.
template <class T, int B, bool LN>
hipError_t launch_mfma_ln(const GemvParams& p, int G, hipStream_t s) {
  const int grid = ((p.rows + kTileRows - 1) / kTileRows) * G;
  const int cus = device_cus();
  const bool u4 = G > 1 || (LN && (B > 1 || (grid + cus - 1) / cus > 3));
  if (u4) hipLaunchKernelGGL((gemv_mfma_kernel<T, B, 4, LN>), dim3(grid), dim3(kThreads), 0, s, p, G);
  else if (LN) hipLaunchKernelGGL((gemv_mfma_kernel<T, 1, 8, true>), dim3(grid), dim3(kThreads), 0, s, p, 1);
  else hipLaunchKernelGGL((gemv_mfma_kernel<T, B, 8, false>), dim3(grid), dim3(kThreads), 0, s, p, 1);
  return hipGetLastError();
}

template <class T, int B>
hipError_t launch_mfma_b(const GemvParams& p, int G, hipStream_t s) {
  return p.ln ? launch_mfma_ln<T, B, true>(p, G, s) : launch_mfma_ln<T, B, false>(p, G, s);
}

template <class T>
hipError_t launch_mfma_t(const GemvParams& p, int B, int G, hipStream_t s) {
  switch (B) {
    case 1: return launch_mfma_b<T, 1>(p, G, s);
    case 2: return launch_mfma_b<T, 2>(p, G, s);
    case 3: return launch_mfma_b<T, 3>(p, G, s);
    case 4: return launch_mfma_b<T, 4>(p, G, s);
    case 5: return launch_mfma_b<T, 5>(p, G, s);
    case 6: return launch_mfma_b<T, 6>(p, G, s);
    case 7: return launch_mfma_b<T, 7>(p, G, s);
    case 8: return launch_mfma_b<T, 8>(p, G, s);
  }
  return hipErrorInvalidValue;
}

size_t ln_partials_floats(int n) { return n > 0 ? (size_t)((n + kLnGroup - 1) / kLnGroup) * kLnSlots * 2 : 0; }

hipError_t launch_gemv_mfma(GemvParams p, int dtype, int B, hipStream_t stream) {
  if (p.rows <= 0) return hipSuccess;
  if (p.K < 8 || p.K % 8 || B < 1 || B > kLnSlots) return hipErrorInvalidValue;
  if (p.ln && (!p.ln_in || p.K > kMaxLnK)) return hipErrorInvalidValue;
  if (p.ln_out && p.y_f32) return hipErrorInvalidValue;
  if (p.ldx < p.K || ((long long)(B - 1) * p.ldx + p.K) * 2 >= (long long)kXPast) return hipErrorInvalidValue;
  const int G = mfma_splits(p.rows, p.K);
  if (G > 1 && (!p.ws || !p.cnt || p.ws_floats < mfma_ws_floats(p.rows, p.K, B) ||
                p.cnt_words < mfma_cnt_words(p.rows, p.K)))
    return hipErrorInvalidValue;
  return dtype == 1 ? launch_mfma_t<BF16>(p, B, G, stream) : launch_mfma_t<F16>(p, B, G, stream);
}

}  // namespace hg
