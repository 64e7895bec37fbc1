// CPU share of a heterogeneous linear (host threads).
#pragma once
#include <stdint.h>

namespace hg {

// y[b * ldy + (r - r0)] = sum_k x[b * K + k] * W[r * K + k] + bias[r]   for r in [r0, r1), b < B.
// x: binary32 [B][K]; W: 16-bit rows (dtype 0 = fp16, 1 = bf16) with row stride K;
// bias: 16-bit [N] or nullptr; y: binary32.  Runs on the calling thread and a worker team;
// nthreads <= 0 uses the OpenMP default thread count.
void cpu_share(const float* x, int B, int K, const uint16_t* W, int dtype, const uint16_t* bias, int r0, int r1,
               float* y, int ldy, int nthreads);

// fn(arg, g) for g in [0, ngrains) on the CPU share's worker team (`threads` threads
// including the caller; <= 0: the OpenMP default count), grains handed out in
// increasing order.  For other host-side work that must not leave a second team of
// threads spinning beside the CPU share's.
void team_for(int threads, int ngrains, void (*fn)(void*, int), void* arg);

// Streamed chunks queued by the library's contexts (+n when planned, -1 when consumed or
// dropped): while none is queued, the worker team spins longer between jobs.
void team_streamed_chunks(long long delta);

// Instruction set the CPU share dispatches to on this host ("avx512", "avx2", "scalar").
const char* cpu_share_isa();

}  // namespace hg
