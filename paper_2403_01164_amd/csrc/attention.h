// Internal launch interface of the decode-attention kernel (not part of the C ABI).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace hg {

// One decode step's attention for B sequences at position pos (HeteGen Sec. 2.1,
// Eq. 1).  qkv [B, 3H] in the activation type (row stride ldq elements) holds the
// new token's q | k | v; the cache holds keys and values of positions [0, pos) as
// kc / vc [max_batch][heads][max_seq][head_dim]; k and v of the new token are
// written at position pos.  out [B, H] (row stride ldo) receives the attention
// output rounded to the activation type.  part / cnt: scratch of the chunk merge,
// part >= max_batch * heads * max_chunks * (head_dim + 2) floats, cnt >=
// max_batch * heads words, zero before the first launch (the kernel leaves them
// zero).
struct AttnParams {
  const void* qkv;
  long long ldq;
  void* kc;
  void* vc;
  void* out;
  long long ldo;
  float* part;
  uint32_t* cnt;
  int heads, head_dim, max_seq, max_chunks, pos;
  int nchunk;   // set by the launcher
  float scale;  // set by the launcher: 1 / sqrt(head_dim)
};

// Positions per workgroup of the attention kernel for short caches (the smallest chunk:
// a partial buffer of ceil(max_seq / attn_chunk()) chunks per (batch, head) holds any
// position's chunks).
int attn_chunk();

// Largest cache (positions) the attention kernel supports.
int attn_max_positions();

// dtype: 0 = fp16, 1 = bf16; head_dim 64 or 128.
hipError_t launch_attention(AttnParams a, int dtype, int B, hipStream_t stream);

}  // namespace hg
