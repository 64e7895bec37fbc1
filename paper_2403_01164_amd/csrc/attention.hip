// gfx950 decode attention over a KV cache (HeteGen Sec. 2.1, Eq. 1: at a decode
// step the new token's key and value are appended to the cached ones and its
// query attends to every cached position).  Batch b, head h, position pos:
//
//   s_j = (q . K_j) / sqrt(D)  for j <= pos,   out = sum_j softmax(s)_j V_j,
//
// with K_pos, V_pos the new token's key and value (taken from the qkv output and
// written into the cache by this kernel).  Everything is read once, so the kernel
// is bound by HBM bandwidth (2 * (pos + 1) * D * 2 bytes per (b, h)), not by
// arithmetic; no matrix cores.
//
// Split over positions: workgroup (c, h, b) takes the 64 positions of chunk c (128
// from 2048 cached positions on: fewer partials to merge, 13-35 % faster at 2048 and
// 4096 positions, slower below at batch 8; the size depends on the position alone, so a
// batch row's bits do not depend on the batch size), 4 wavefronts x 64 / (D / 8) positions
// per round (D / 8 lanes hold one 16-byte
// slice each of a key or value row, so a load instruction reads whole 256-byte
// rows, coalesced).  It keeps (max score, sum of exponentials, weighted sum of V)
// of its chunk; the last workgroup of (b, h) to finish (an arrival counter, no
// waiting) merges the chunks in chunk order and writes the output rounded to the
// activation type.  Every reduction has a fixed order, so results are
// deterministic.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "attention.h"

namespace hg {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 64;       // positions per workgroup, short caches
constexpr int kLongChunk = 128;  // positions per workgroup from kLongFrom positions on
constexpr int kLongFrom = 2048;
constexpr int kMaxChunks = 256;  // chunks the merge holds in LDS (positions <= 16384)
constexpr int kMergeRegs = 16;   // chunks whose partial outputs the merge requests at once

struct F16 {
  static __device__ __forceinline__ float to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
  static __device__ __forceinline__ uint16_t from_f32(float v) { return __builtin_bit_cast(uint16_t, (_Float16)v); }
};

struct BF16 {
  static __device__ __forceinline__ float to_f32(uint16_t h) { return __builtin_bit_cast(float, (uint32_t)h << 16); }
  static __device__ __forceinline__ uint16_t from_f32(float v) { return __builtin_bit_cast(uint16_t, (__bf16)v); }
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <class T>
__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = T::to_f32((uint16_t)(w[i] & 0xFFFFu));
    f[2 * i + 1] = T::to_f32((uint16_t)(w[i] >> 16));
  }
}

// 16-byte load through the global address space (a generic load would also count
// against the LDS counter); `stream`: read once, non-temporal.
template <bool STREAM>
__device__ __forceinline__ uint4 load16(const uint16_t* p) {
  const __attribute__((address_space(1))) u32x4* g = (const __attribute__((address_space(1))) u32x4*)p;
  const u32x4 v = STREAM ? __builtin_nontemporal_load(g) : *g;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Partials of the chunk merge cross workgroups on different XCDs (separate L2s):
// they are written and read with sc0 sc1 buffer accesses, which go to memory, so
// no cache-wide writeback or invalidate is needed.  The descriptor base is
// wave-uniform; word 3 is the gfx9 raw-buffer format.
constexpr int kCoherent = 1 | 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ float wave_add(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <class T, int D, int CH>
__global__ __launch_bounds__(kThreads) void attn_kernel(AttnParams a) {
  constexpr int LP = D / 8;          // lanes per key/value row
  constexpr int PPW = 64 / LP;       // rows per wavefront per round
  constexpr int PPR = PPW * kWaves;  // rows per workgroup per round
  constexpr int ROUNDS = CH / PPR;
  constexpr int SPL = CH / 64;       // scores per lane of the softmax wavefront
  __shared__ float sp[CH];
  __shared__ float sacc[kWaves][D];
  __shared__ float sml[2];
  __shared__ float s_m[kMaxChunks], s_l[kMaxChunks];
  __shared__ int s_last;

  const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LP, grp = lane / LP;
  const int H = a.heads * D;
  const uint16_t* qkv = (const uint16_t*)a.qkv + (size_t)b * a.ldq;
  const uint16_t* knew = qkv + H + h * D;
  const uint16_t* vnew = qkv + 2 * H + h * D;
  const size_t head = ((size_t)b * a.heads + h) * a.max_seq;
  uint16_t* Kc = (uint16_t*)a.kc + head * D;
  uint16_t* Vc = (uint16_t*)a.vc + head * D;
  const int j0 = c * CH;

  // every key and value row of the chunk is requested at once (positions past pos
  // reread the new token's row and are masked below); position pos comes from qkv
  uint4 kr[ROUNDS], vr[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int j = j0 + r * PPR + wave * PPW + grp;
    kr[r] = j >= a.pos ? load16<false>(knew + sub * 8) : load16<true>(Kc + (size_t)j * D + sub * 8);
    vr[r] = j >= a.pos ? load16<false>(vnew + sub * 8) : load16<true>(Vc + (size_t)j * D + sub * 8);
  }
  float q[8];
  unpack8<T>(load16<false>(qkv + h * D + sub * 8), q);
#pragma unroll
  for (int e = 0; e < 8; ++e) q[e] *= a.scale;

  // the chunk holding pos appends the new key and value to the cache
  if (c == a.nchunk - 1 && threadIdx.x < 2 * LP) {
    const int s = threadIdx.x % LP;
    if (threadIdx.x < LP) *(uint4*)(Kc + (size_t)a.pos * D + s * 8) = load16<false>(knew + s * 8);
    else *(uint4*)(Vc + (size_t)a.pos * D + s * 8) = load16<false>(vnew + s * 8);
  }

  // scores of the chunk's positions
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int jl = r * PPR + wave * PPW + grp;
    float k[8];
    unpack8<T>(kr[r], k);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf(q[e], k[e], s);
#pragma unroll
    for (int off = LP / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off);  // the LP lanes of one row
    if (sub == 0) sp[jl] = j0 + jl <= a.pos ? s : -INFINITY;
  }
  __syncthreads();
  if (wave == 0) {  // scores lane + 64 i of the chunk
    float sv[SPL], mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      sv[i] = sp[lane + 64 * i];
      mx = fmaxf(mx, sv[i]);
    }
    const float m = wave_max(mx);
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < SPL; ++i) {
      const float p = sv[i] == -INFINITY ? 0.f : expf(sv[i] - m);
      sp[lane + 64 * i] = p;
      ps += p;
    }
    const float l = wave_add(ps);
    if (lane == 0) {
      sml[0] = m;
      sml[1] = l;
    }
  }
  __syncthreads();

  // weighted sum of the chunk's value rows (masked positions have weight 0)
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const float p = sp[r * PPR + wave * PPW + grp];
    float v[8];
    unpack8<T>(vr[r], v);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(p, v[e], acc[e]);
  }
#pragma unroll
  for (int off = LP; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], off);
  if (grp == 0)
#pragma unroll
    for (int e = 0; e < 8; ++e) sacc[wave][sub * 8 + e] = acc[e];
  __syncthreads();

  const int t = threadIdx.x;
  float o = 0.f;
  if (t < D) o = (sacc[0][t] + sacc[1][t]) + (sacc[2][t] + sacc[3][t]);
  uint16_t* out = (uint16_t*)a.out + (size_t)b * a.ldo + h * D;
  if (a.nchunk == 1) {
    if (t < D) out[t] = T::from_f32(o / sml[1]);
    return;
  }

  // partial of this chunk, [m, l, o[0..D)], stored to memory
  const float* part = a.part + ((size_t)(b * a.heads + h) * a.max_chunks) * (D + 2);
  const uint32_t pbytes = (uint32_t)(a.max_chunks * (D + 2) * sizeof(float));
  const auto rs = rsrc(part, pbytes);
  const int mine = c * (D + 2);
  if (t < D) __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, o), rs, (mine + 2 + t) * 4, 0,
                                                   kCoherent);
  if (t == 0) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, sml[0]), rs, mine * 4, 0, kCoherent);
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, sml[1]), rs, (mine + 1) * 4, 0, kCoherent);
  }
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores have completed
  __syncthreads();
  if (t == 0) {
    uint32_t* cnt = a.cnt + (size_t)b * a.heads + h;
    const uint32_t prev = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == (uint32_t)(a.nchunk - 1);
    if (s_last) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // ready for the next call
  }
  __syncthreads();
  if (!s_last) return;
  // merge, in chunk order: the partials are requested kMergeRegs chunks at a time (one
  // memory round trip per kMergeRegs chunks), m and l through LDS
  auto ld = [&](int i) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, i * 4, 0, kCoherent));
  };
  float ov[kMergeRegs];
  if (t < D) {
#pragma unroll
    for (int u = 0; u < kMergeRegs; ++u) ov[u] = u < a.nchunk ? ld(u * (D + 2) + 2 + t) : 0.f;
  }
  for (int k = t; k < a.nchunk; k += kThreads) {
    s_m[k] = ld(k * (D + 2));
    s_l[k] = ld(k * (D + 2) + 1);
  }
  __syncthreads();
  if (t < D) {
    float M = -INFINITY;
    for (int k = 0; k < a.nchunk; ++k) M = fmaxf(M, s_m[k]);
    float L = 0.f, O = 0.f;
    for (int k0 = 0; k0 < a.nchunk; k0 += kMergeRegs) {
      if (k0 > 0) {
#pragma unroll
        for (int u = 0; u < kMergeRegs; ++u) ov[u] = k0 + u < a.nchunk ? ld((k0 + u) * (D + 2) + 2 + t) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kMergeRegs; ++u) {
        if (k0 + u < a.nchunk) {
          const float w = expf(s_m[k0 + u] - M);
          L = fmaf(s_l[k0 + u], w, L);
          O = fmaf(ov[u], w, O);
        }
      }
    }
    out[t] = T::from_f32(O / L);
  }
}

template <class T, int CH>
hipError_t launch_t(const AttnParams& a, int B, hipStream_t s) {
  const dim3 grid(a.nchunk, a.heads, B);
  if (a.head_dim == 128) hipLaunchKernelGGL((attn_kernel<T, 128, CH>), grid, dim3(kThreads), 0, s, a);
  else hipLaunchKernelGGL((attn_kernel<T, 64, CH>), grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

int attn_chunk() { return kChunk; }

int attn_max_positions() { return kChunk * kMaxChunks; }

hipError_t launch_attention(AttnParams a, int dtype, int B, hipStream_t stream) {
  if (B < 1 || a.pos < 0 || a.pos >= a.max_seq || (a.head_dim != 64 && a.head_dim != 128) || a.heads < 1)
    return hipErrorInvalidValue;
  const bool lng = a.pos + 1 >= kLongFrom;
  const int ch = lng ? kLongChunk : kChunk;
  a.nchunk = (a.pos + ch) / ch;  // chunks covering positions [0, pos]
  if (a.nchunk > a.max_chunks || a.nchunk > kMaxChunks) return hipErrorInvalidValue;
  a.scale = 1.0f / sqrtf((float)a.head_dim);
  if (lng) return dtype == 1 ? launch_t<BF16, kLongChunk>(a, B, stream) : launch_t<F16, kLongChunk>(a, B, stream);
  return dtype == 1 ? launch_t<BF16, kChunk>(a, B, stream) : launch_t<F16, kChunk>(a, B, stream);
}

}  // namespace hg
