// CPU share of the heterogeneous Linear (HeteGen Sec. 3.2: the CPU computes the
// part of the module whose parameters stay in host memory, concurrently with the
// transfer and GPU compute of the other part; Sec. 5 runs it on host cores).
//
// Threads take runs of 32 consecutive output rows from a shared queue, so each
// streams whole weight rows sequentially from DRAM.  A row block of R rows is
// processed together so that each binary32 x vector loaded from cache is used R
// times; 16-bit weights are widened to binary32 in registers (vcvtph2ps for fp16,
// a 16-bit shift for bf16) and accumulated with FMA; on hosts with AVX512-BF16, bf16
// weights instead go through vdpbf16ps (two bf16 products per binary32 lane, so one
// instruction per 32 weights and batch row, against a widening and two FMAs).  The
// instruction set is chosen at run time (AVX-512, else AVX2+F16C+FMA, else portable
// C), so one build runs on any x86-64 host.
#include "cpu_share.h"

#include <immintrin.h>
#include <linux/futex.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <atomic>
#include <chrono>
#include <climits>
#include <mutex>
#include <sched.h>
#include <thread>
#include <vector>

namespace hg {
namespace {

// ---------------- worker team ----------------
// The CPU shares of a decode step come ~1 ms apart, with the calling thread's kernel
// and copy enqueues (and the parameter manager thread) in between.  An OpenMP team
// keeps its workers spinning through such gaps (libgomp's default spin count), on
// every core, and the calling thread's and the manager's work then waits for the
// scheduler.  This team spins only briefly (kSpinUs) and then sleeps on a futex; the
// caller takes part in every job.  One job runs at a time (jobs from several host
// threads are serialised).  While no streamed chunk is queued anywhere in the process
// (no manager work), the workers spin longer (kIdleSpinUs), yielding the core each
// round, so back-to-back CPU shares of resident linears skip the futex wake-up
// (single linear [4096,1024] at CPU fraction 0.25: 57 -> 45 us per call).  Spinning
// that long while chunks stream slowed the OPT-30B all-host step by 15 %.
std::atomic<long long> g_streamed_chunks{0};
class Team {
 public:
  static Team& get() {
    static Team* t = new Team();  // never destroyed: its workers sleep until the process ends
    return *t;
  }
  // fn(arg, g) for every g in [0, ngrains), on `threads` threads including the caller;
  // grains are handed out in increasing order from a shared counter.
  void run(int threads, int ngrains, void (*fn)(void*, int), void* arg) {
    if (ngrains <= 0) return;
    const int nw = std::min(threads, ngrains) - 1;
    if (nw <= 0) {
      for (int g = 0; g < ngrains; ++g) fn(arg, g);
      return;
    }
    std::lock_guard<std::mutex> lk(run_mu_);
    grow(nw);
    fn_ = fn;
    arg_ = arg;
    ngrains_ = ngrains;
    nw_ = std::min(nw, nworkers_);  // fewer if threads could not be created
    next_.store(0, std::memory_order_relaxed);
    left_.store(nworkers_, std::memory_order_relaxed);  // every worker acknowledges the job
    gen_.fetch_add(1, std::memory_order_seq_cst);
    if (sleepers_.load(std::memory_order_seq_cst) > 0) syscall(SYS_futex, &gen_, FUTEX_WAKE_PRIVATE, INT_MAX, nullptr, nullptr, 0);
    grains();
    while (left_.load(std::memory_order_acquire) > 0) _mm_pause();
  }

 private:
  Team() {
    const char* e = getenv("HETEGEN_SPIN_US");
    spin_us_ = e ? atoi(e) : kSpinUs;
    const char* f = getenv("HETEGEN_IDLE_SPIN_US");
    idle_spin_us_ = f ? atoi(f) : kIdleSpinUs;
  }
  static constexpr int kSpinUs = 20, kIdleSpinUs = 300;
  void grains() {
    for (int g; (g = next_.fetch_add(1, std::memory_order_relaxed)) < ngrains_;) fn_(arg_, g);
  }
  void grow(int n) {
    while (nworkers_ < n) {
      const int i = nworkers_;
      const uint32_t g0 = gen_.load(std::memory_order_relaxed);
      try {
        std::thread t([this, i, g0] { work(i, g0); });
        t.detach();
      } catch (...) {
        return;  // no more threads: the job runs on those there are
      }
      ++nworkers_;
    }
  }
  void work(int i, uint32_t seen) {
    for (;;) {
      uint32_t g = gen_.load(std::memory_order_acquire);
      if (g == seen) {
        const auto t0 = std::chrono::steady_clock::now();
        for (;;) {
          const bool idle = g_streamed_chunks.load(std::memory_order_relaxed) <= 0;
          if (std::chrono::steady_clock::now() - t0 >= std::chrono::microseconds(idle ? idle_spin_us_ : spin_us_))
            break;
          for (int k = 0; k < 32; ++k) _mm_pause();
          if (idle) sched_yield();
          g = gen_.load(std::memory_order_acquire);
          if (g != seen) break;
        }
      }
      while (g == seen) {
        sleepers_.fetch_add(1, std::memory_order_seq_cst);
        if (gen_.load(std::memory_order_seq_cst) == seen)
          syscall(SYS_futex, &gen_, FUTEX_WAIT_PRIVATE, seen, nullptr, nullptr, 0);
        sleepers_.fetch_sub(1, std::memory_order_seq_cst);
        g = gen_.load(std::memory_order_acquire);
      }
      seen = g;  // the next job: every worker acknowledged the previous one before it was published
      if (i < nw_) grains();
      left_.fetch_sub(1, std::memory_order_release);
    }
  }
  std::mutex run_mu_;
  int nworkers_ = 0;  // detached worker threads
  std::atomic<uint32_t> gen_{0};
  std::atomic<int> sleepers_{0}, next_{0}, left_{0};
  void (*fn_)(void*, int) = nullptr;
  void* arg_ = nullptr;
  int ngrains_ = 0, nw_ = 0, spin_us_ = kSpinUs, idle_spin_us_ = kIdleSpinUs;
};

// ---------------- portable fallback ----------------
float f16_to_f32(uint16_t h) {
  uint32_t sign = (uint32_t)(h & 0x8000u) << 16, e = (h >> 10) & 0x1Fu, m = h & 0x3FFu, bits;
  if (e == 0x1Fu) {
    bits = sign | 0x7F800000u | (m << 13);
  } else if (e) {
    bits = sign | ((e + 112u) << 23) | (m << 13);
  } else if (!m) {
    bits = sign;
  } else {
    int sh = 0;
    while (!(m & 0x400u)) { m <<= 1; ++sh; }
    bits = sign | ((uint32_t)(113 - sh) << 23) | ((m & 0x3FFu) << 13);
  }
  float f;
  memcpy(&f, &bits, 4);
  return f;
}

float bf16_to_f32(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float f;
  memcpy(&f, &bits, 4);
  return f;
}

inline float wval(const uint16_t* p, int dtype) { return dtype == 1 ? bf16_to_f32(*p) : f16_to_f32(*p); }

void rows_scalar(const float* x, int B, int K, const uint16_t* W, int dtype, const uint16_t* bias, int r0, int ra,
                 int rb, float* y, int ldy) {
  for (int r = ra; r < rb; ++r) {
    const uint16_t* w = W + (int64_t)r * K;
    for (int b = 0; b < B; ++b) {
      float acc = 0.f;
      for (int k = 0; k < K; ++k) acc += x[(int64_t)b * K + k] * wval(w + k, dtype);
      if (bias) acc += wval(bias + r, dtype);
      y[(int64_t)b * ldy + (r - r0)] = acc;
    }
  }
}

// ---------------- AVX-512 ----------------
template <bool BF>
__attribute__((target("avx512f,avx512bw,avx512vl,f16c,fma"))) inline __m512 load16(const uint16_t* p) {
  __m256i v = _mm256_loadu_si256((const __m256i*)p);
  if (BF) return _mm512_castsi512_ps(_mm512_slli_epi32(_mm512_cvtepu16_epi32(v), 16));
  return _mm512_cvtph_ps(v);
}

template <bool BF>
__attribute__((target("avx512f,avx512bw,avx512vl,f16c,fma"))) inline __m512 load8(const uint16_t* p) {
  __m256i v = _mm256_maskz_loadu_epi16((__mmask16)0xFF, p);
  if (BF) return _mm512_castsi512_ps(_mm512_slli_epi32(_mm512_cvtepu16_epi32(v), 16));
  return _mm512_cvtph_ps(v);
}

// Software prefetch distance along each weight row: the hardware prefetcher alone
// leaves a core's memory pipe partly idle (measured on the 16-core Zen 5 host:
// +10-40 % at batch 1-4); at batch 4 twice as far (+2 % on both paths, interleaved A/B).
constexpr int kPrefetchBytes = 1024;
template <int B>
constexpr int prefetch_bytes() {
  return B == 4 ? 2 * kPrefetchBytes : kPrefetchBytes;
}

template <bool BF, int B, int R, int UN>
__attribute__((target("avx512f,avx512bw,avx512vl,f16c,fma"))) void block512(const float* x, int K, const uint16_t* W,
                                                                           const uint16_t* bias, int r0, int r,
                                                                           float* y, int ldy) {
  __m512 acc[R][B];
  for (int i = 0; i < R; ++i)
    for (int b = 0; b < B; ++b) acc[i][b] = _mm512_setzero_ps();
  const uint16_t* w[R];
  for (int i = 0; i < R; ++i) w[i] = W + (int64_t)(r + i) * K;
  int k = 0;
  for (; k + 16 * UN <= K; k += 16 * UN) {
    if ((k & 31) == 0)  // one prefetch per 64-byte line of every row (past the end: harmless)
      for (int i = 0; i < R; ++i) _mm_prefetch((const char*)(w[i] + k) + prefetch_bytes<B>(), _MM_HINT_T0);
    for (int u = 0; u < UN; ++u) {
      __m512 wv[R];
      for (int i = 0; i < R; ++i) wv[i] = load16<BF>(w[i] + k + 16 * u);
      for (int b = 0; b < B; ++b) {
        __m512 xv = _mm512_loadu_ps(x + (int64_t)b * K + k + 16 * u);
        for (int i = 0; i < R; ++i) acc[i][b] = _mm512_fmadd_ps(wv[i], xv, acc[i][b]);
      }
    }
  }
  for (; k + 16 <= K; k += 16) {
    __m512 wv[R];
    for (int i = 0; i < R; ++i) wv[i] = load16<BF>(w[i] + k);
    for (int b = 0; b < B; ++b) {
      __m512 xv = _mm512_loadu_ps(x + (int64_t)b * K + k);
      for (int i = 0; i < R; ++i) acc[i][b] = _mm512_fmadd_ps(wv[i], xv, acc[i][b]);
    }
  }
  if (k < K) {  // K % 8 == 0: one half vector left
    __m512 wv[R];
    for (int i = 0; i < R; ++i) wv[i] = load8<BF>(w[i] + k);
    for (int b = 0; b < B; ++b) {
      __m512 xv = _mm512_maskz_loadu_ps((__mmask16)0xFF, x + (int64_t)b * K + k);
      for (int i = 0; i < R; ++i) acc[i][b] = _mm512_fmadd_ps(wv[i], xv, acc[i][b]);
    }
  }
  for (int i = 0; i < R; ++i) {
    const float bv = bias ? wval(bias + r + i, BF ? 1 : 0) : 0.f;
    for (int b = 0; b < B; ++b) y[(int64_t)b * ldy + (r + i - r0)] = _mm512_reduce_add_ps(acc[i][b]) + bv;
  }
}

// Batch 5-8: R rows x B batch accumulators no longer fit the 32 vector registers, so
// the batch runs in two groups over chunks of KC elements: the first group streams a
// chunk of the R rows from memory, the second reuses it from L1.  Every (row, batch)
// accumulator still adds the same products in the same order as block512 (16 lanes,
// increasing k, the half-vector tail last), so the results are the same bits.
// (Measured on the 16-core Zen 5 host at batch 8, OPT-66B fc1 shape: 157 -> 282 GB/s.)
template <bool BF, int R, int LO, int NB>
__attribute__((target("avx512f,avx512bw,avx512vl,f16c,fma"), always_inline)) inline void group512(
    const float* x, int K, const uint16_t* const* w, int k0, int k1, bool tail, __m512 (*acc)[R]) {
  __m512 a[NB][R];
  for (int bb = 0; bb < NB; ++bb)
    for (int i = 0; i < R; ++i) a[bb][i] = acc[LO + bb][i];
  for (int k = k0; k < k1; k += 16) {
    if (LO == 0 && (k & 31) == 0)
      for (int i = 0; i < R; ++i) _mm_prefetch((const char*)(w[i] + k) + kPrefetchBytes, _MM_HINT_T0);
    __m512 wv[R];
    for (int i = 0; i < R; ++i) wv[i] = load16<BF>(w[i] + k);
    for (int bb = 0; bb < NB; ++bb) {
      __m512 xv = _mm512_loadu_ps(x + (int64_t)(LO + bb) * K + k);
      for (int i = 0; i < R; ++i) a[bb][i] = _mm512_fmadd_ps(wv[i], xv, a[bb][i]);
    }
  }
  if (tail) {  // K % 8 == 0: one half vector left at k1
    __m512 wv[R];
    for (int i = 0; i < R; ++i) wv[i] = load8<BF>(w[i] + k1);
    for (int bb = 0; bb < NB; ++bb) {
      __m512 xv = _mm512_maskz_loadu_ps((__mmask16)0xFF, x + (int64_t)(LO + bb) * K + k1);
      for (int i = 0; i < R; ++i) a[bb][i] = _mm512_fmadd_ps(wv[i], xv, a[bb][i]);
    }
  }
  for (int bb = 0; bb < NB; ++bb)
    for (int i = 0; i < R; ++i) acc[LO + bb][i] = a[bb][i];
}

template <bool BF, int B, int R>
__attribute__((target("avx512f,avx512bw,avx512vl,f16c,fma"))) void block512_split(const float* x, int K,
                                                                                 const uint16_t* W,
                                                                                 const uint16_t* bias, int r0, int r,
                                                                                 float* y, int ldy) {
  // 128-element chunks (the box's Zen 5 host, OPT-66B fc1 shape, interleaved A/B: 323.5 ->
  // 332.8 GB/s at B = 8, 349.5 -> 360.4 at B = 5 against 256; 64 slower at B = 8)
  constexpr int KC = 128, H0 = (B + 1) / 2;
  __m512 acc[B][R];
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < R; ++i) acc[b][i] = _mm512_setzero_ps();
  const uint16_t* w[R];
  for (int i = 0; i < R; ++i) w[i] = W + (int64_t)(r + i) * K;
  const int K16 = K & ~15;
  for (int k0 = 0; k0 < K; k0 += KC) {
    const int k1 = k0 + KC < K16 ? k0 + KC : K16;  // full vectors of this chunk
    const bool tail = k0 + KC >= K && K16 < K;
    group512<BF, R, 0, H0>(x, K, w, k0, k1, tail, acc);
    group512<BF, R, H0, B - H0>(x, K, w, k0, k1, tail, acc);
  }
  for (int i = 0; i < R; ++i) {
    const float bv = bias ? wval(bias + r + i, BF ? 1 : 0) : 0.f;
    for (int b = 0; b < B; ++b) y[(int64_t)b * ldy + (r + i - r0)] = _mm512_reduce_add_ps(acc[b][i]) + bv;
  }
}

// ---------------- AVX512-BF16 (bf16 weights) ----------------
// x [B, K] arrives as binary32 values that are bf16 values (the activation type), so it
// is narrowed to bf16 exactly, once per call; x with any value that bf16 cannot hold
// (low 16 bits set: possible through hetegen_cpu_linear) takes the widening path.  vdpbf16ps multiplies bf16 pairs exactly
// and adds them to binary32 lanes (lane j of a 32-element chunk takes elements 2j and
// 2j + 1); like every bf16 instruction of this extension it treats bf16 subnormal
// inputs as zero and flushes binary32 subnormal results (|v| < 2^-126), far below the
// oracle's tolerance for any row with a normal output.  Every (row, batch row)
// accumulator adds the chunks in increasing k, the masked tail last, in both kernels
// below, so a row's bits do not depend on the batch size.
#define HG_BF16_TARGET __attribute__((target("avx512f,avx512bw,avx512vl,avx512bf16,fma")))

HG_BF16_TARGET inline __m512bh ld_bh(const uint16_t* p) { return (__m512bh)_mm512_loadu_si512((const void*)p); }
HG_BF16_TARGET inline __m512bh ld_bh_tail(const uint16_t* p, int n) {  // n < 32 elements, the rest zero
  return (__m512bh)_mm512_maskz_loadu_epi16((__mmask32)((1u << n) - 1u), p);
}

// x (binary32) -> bf16 [B, K]: the upper halves of the binary32 patterns; returns whether
// every value was a bf16 value (lower half zero), i.e. the narrowing was exact
HG_BF16_TARGET bool narrow_bf16(const float* x, int n, uint16_t* out) {
  const __m512i low = _mm512_set1_epi32(0xFFFF);
  __mmask16 inexact = 0;
  int i = 0;
  for (; i + 32 <= n; i += 32) {
    const __m512i lo = _mm512_loadu_si512((const void*)(x + i)), hi = _mm512_loadu_si512((const void*)(x + i + 16));
    inexact |= _mm512_test_epi32_mask(lo, low) | _mm512_test_epi32_mask(hi, low);
    // the upper 16 bits of each lane, in lane order: 32 bf16 values
    const __m512i idx = _mm512_set_epi16(63, 61, 59, 57, 55, 53, 51, 49, 47, 45, 43, 41, 39, 37, 35, 33, 31, 29, 27, 25,
                                         23, 21, 19, 17, 15, 13, 11, 9, 7, 5, 3, 1);
    _mm512_storeu_si512((void*)(out + i), _mm512_permutex2var_epi16(lo, idx, hi));
  }
  bool exact = inexact == 0;
  for (; i < n; ++i) {
    uint32_t b;
    memcpy(&b, x + i, 4);
    exact = exact && (b & 0xFFFFu) == 0;
    out[i] = (uint16_t)(b >> 16);
  }
  return exact;
}

template <int B, int R>
HG_BF16_TARGET void block_bf16(const uint16_t* xb, int K, const uint16_t* W, const uint16_t* bias, int r0, int r,
                               float* y, int ldy) {
  __m512 acc[R][B];
  for (int i = 0; i < R; ++i)
    for (int b = 0; b < B; ++b) acc[i][b] = _mm512_setzero_ps();
  const uint16_t* w[R];
  for (int i = 0; i < R; ++i) w[i] = W + (int64_t)(r + i) * K;
  const int K32 = K & ~31;
  for (int k = 0; k < K32; k += 32) {
    for (int i = 0; i < R; ++i) _mm_prefetch((const char*)(w[i] + k) + prefetch_bytes<B>(), _MM_HINT_T0);
    __m512bh wv[R];
    for (int i = 0; i < R; ++i) wv[i] = ld_bh(w[i] + k);
    for (int b = 0; b < B; ++b) {
      const __m512bh xv = ld_bh(xb + (int64_t)b * K + k);
      for (int i = 0; i < R; ++i) acc[i][b] = _mm512_dpbf16_ps(acc[i][b], wv[i], xv);
    }
  }
  if (K32 < K) {
    __m512bh wv[R];
    for (int i = 0; i < R; ++i) wv[i] = ld_bh_tail(w[i] + K32, K - K32);
    for (int b = 0; b < B; ++b) {
      const __m512bh xv = ld_bh_tail(xb + (int64_t)b * K + K32, K - K32);
      for (int i = 0; i < R; ++i) acc[i][b] = _mm512_dpbf16_ps(acc[i][b], wv[i], xv);
    }
  }
  for (int i = 0; i < R; ++i) {
    const float bv = bias ? bf16_to_f32(bias[r + i]) : 0.f;
    for (int b = 0; b < B; ++b) y[(int64_t)b * ldy + (r + i - r0)] = _mm512_reduce_add_ps(acc[i][b]) + bv;
  }
}

// Batch 7-8: the R x B accumulators do not fit the registers; as in block512_split, the
// batch runs in two groups over chunks of KC elements, the second reusing the chunk
// of the R rows from L1.  (Up to B = 6 the 4 x B accumulators, four weight vectors and
// one x vector fit the 32 registers, and block_bf16 keeps them there.)
template <int R, int LO, int NB>
HG_BF16_TARGET __attribute__((always_inline)) inline void group_bf16(const uint16_t* xb, int K, const uint16_t* const* w,
                                                                     int k0, int k1, int tail, __m512 (*acc)[R]) {
  __m512 a[NB][R];
  for (int bb = 0; bb < NB; ++bb)
    for (int i = 0; i < R; ++i) a[bb][i] = acc[LO + bb][i];
  for (int k = k0; k < k1; k += 32) {
    if (LO == 0)
      for (int i = 0; i < R; ++i) _mm_prefetch((const char*)(w[i] + k) + kPrefetchBytes, _MM_HINT_T0);
    __m512bh wv[R];
    for (int i = 0; i < R; ++i) wv[i] = ld_bh(w[i] + k);
    for (int bb = 0; bb < NB; ++bb) {
      const __m512bh xv = ld_bh(xb + (int64_t)(LO + bb) * K + k);
      for (int i = 0; i < R; ++i) a[bb][i] = _mm512_dpbf16_ps(a[bb][i], wv[i], xv);
    }
  }
  if (tail) {  // tail < 32 elements at k1
    __m512bh wv[R];
    for (int i = 0; i < R; ++i) wv[i] = ld_bh_tail(w[i] + k1, tail);
    for (int bb = 0; bb < NB; ++bb) {
      const __m512bh xv = ld_bh_tail(xb + (int64_t)(LO + bb) * K + k1, tail);
      for (int i = 0; i < R; ++i) a[bb][i] = _mm512_dpbf16_ps(a[bb][i], wv[i], xv);
    }
  }
  for (int bb = 0; bb < NB; ++bb)
    for (int i = 0; i < R; ++i) acc[LO + bb][i] = a[bb][i];
}

template <int B, int R>
HG_BF16_TARGET void block_bf16_split(const uint16_t* xb, int K, const uint16_t* W, const uint16_t* bias, int r0, int r,
                                     float* y, int ldy) {
  // 64-element chunks (the box's Zen 5 host, OPT-66B fc1 shape, interleaved A/B: 321.6 ->
  // 360.9 GB/s at B = 8, 333.8 -> 370.8 at B = 7 against 256)
  constexpr int KC = 64, H0 = (B + 1) / 2;
  __m512 acc[B][R];
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < R; ++i) acc[b][i] = _mm512_setzero_ps();
  const uint16_t* w[R];
  for (int i = 0; i < R; ++i) w[i] = W + (int64_t)(r + i) * K;
  const int K32 = K & ~31;
  for (int k0 = 0; k0 < K; k0 += KC) {
    const int k1 = k0 + KC < K32 ? k0 + KC : K32;  // full 32-element chunks of this block
    const int tail = k0 + KC >= K ? K - K32 : 0;
    group_bf16<R, 0, H0>(xb, K, w, k0, k1, tail, acc);
    group_bf16<R, H0, B - H0>(xb, K, w, k0, k1, tail, acc);
  }
  for (int i = 0; i < R; ++i) {
    const float bv = bias ? bf16_to_f32(bias[r + i]) : 0.f;
    for (int b = 0; b < B; ++b) y[(int64_t)b * ldy + (r + i - r0)] = _mm512_reduce_add_ps(acc[b][i]) + bv;
  }
}

typedef void (*BlockBf16Fn)(const uint16_t*, int, const uint16_t*, const uint16_t*, int, int, float*, int);

template <int B>
void run_blocks_bf16(const uint16_t* xb, int K, const uint16_t* W, const uint16_t* bias, int r0, int r1, int ba,
                     int bb, float* y, int ldy) {
  // one group up to B = 6 (B = 5 / 6: 357.7 -> 377.6 / 358.1 -> 370.3 GB/s against two groups);
  // eight rows per block at B <= 2 (B = 2: 341.4 -> 353.3 GB/s; the same at B = 1)
  constexpr int R = 4;
  const BlockBf16Fn blk = B >= 7 ? block_bf16_split<B, R> : block_bf16<B, R>;
  const BlockBf16Fn blk8 = B <= 2 ? block_bf16<B, 8> : nullptr;
  for (int i = ba; i < bb;) {
    const int r = r0 + R * i;
    if (blk8 && i + 1 < bb && r + 2 * R <= r1) {
      blk8(xb, K, W, bias, r0, r, y, ldy);
      i += 2;
      continue;
    }
    if (r + R <= r1) blk(xb, K, W, bias, r0, r, y, ldy);
    else
      for (int q = r; q < r1; ++q) block_bf16<B, 1>(xb, K, W, bias, r0, q, y, ldy);
    ++i;
  }
}

void run_blocks_bf16_b(const uint16_t* xb, int B, int K, const uint16_t* W, const uint16_t* bias, int r0, int r1,
                       int ba, int bb, float* y, int ldy) {
  switch (B) {
    case 1: run_blocks_bf16<1>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 2: run_blocks_bf16<2>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 3: run_blocks_bf16<3>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 4: run_blocks_bf16<4>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 5: run_blocks_bf16<5>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 6: run_blocks_bf16<6>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 7: run_blocks_bf16<7>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    default: run_blocks_bf16<8>(xb, K, W, bias, r0, r1, ba, bb, y, ldy); break;
  }
}

// ---------------- AVX2 + F16C + FMA ----------------
template <bool BF>
__attribute__((target("avx2,f16c,fma"))) inline __m256 load8_avx2(const uint16_t* p) {
  __m128i v = _mm_loadu_si128((const __m128i*)p);
  if (BF) return _mm256_castsi256_ps(_mm256_slli_epi32(_mm256_cvtepu16_epi32(v), 16));
  return _mm256_cvtph_ps(v);
}

__attribute__((target("avx2,f16c,fma"))) inline float hsum256(__m256 v) {
  __m128 s = _mm_add_ps(_mm256_castps256_ps128(v), _mm256_extractf128_ps(v, 1));
  s = _mm_add_ps(s, _mm_movehl_ps(s, s));
  s = _mm_add_ss(s, _mm_shuffle_ps(s, s, 1));
  return _mm_cvtss_f32(s);
}

template <bool BF, int B, int R>
__attribute__((target("avx2,f16c,fma"))) void block256(const float* x, int K, const uint16_t* W, const uint16_t* bias,
                                                       int r0, int r, float* y, int ldy) {
  __m256 acc[R][B];
  for (int i = 0; i < R; ++i)
    for (int b = 0; b < B; ++b) acc[i][b] = _mm256_setzero_ps();
  const uint16_t* w[R];
  for (int i = 0; i < R; ++i) w[i] = W + (int64_t)(r + i) * K;
  for (int k = 0; k < K; k += 8) {
    if ((k & 31) == 0)
      for (int i = 0; i < R; ++i) _mm_prefetch((const char*)(w[i] + k) + kPrefetchBytes, _MM_HINT_T0);
    __m256 wv[R];
    for (int i = 0; i < R; ++i) wv[i] = load8_avx2<BF>(w[i] + k);
    for (int b = 0; b < B; ++b) {
      __m256 xv = _mm256_loadu_ps(x + (int64_t)b * K + k);
      for (int i = 0; i < R; ++i) acc[i][b] = _mm256_fmadd_ps(wv[i], xv, acc[i][b]);
    }
  }
  for (int i = 0; i < R; ++i) {
    const float bv = bias ? wval(bias + r + i, BF ? 1 : 0) : 0.f;
    for (int b = 0; b < B; ++b) y[(int64_t)b * ldy + (r + i - r0)] = hsum256(acc[i][b]) + bv;
  }
}

enum Isa { ISA_SCALAR = 0, ISA_AVX2 = 1, ISA_AVX512 = 2 };

Isa detect() {
  __builtin_cpu_init();
  if (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") && __builtin_cpu_supports("avx512vl"))
    return ISA_AVX512;
  if (__builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma") && __builtin_cpu_supports("f16c"))
    return ISA_AVX2;
  return ISA_SCALAR;
}

const Isa g_isa = detect();

bool detect_bf16() {
  __builtin_cpu_init();
  const char* e = getenv("HETEGEN_CPU_BF16");  // "0": keep the widening FMA path
  return g_isa == ISA_AVX512 && __builtin_cpu_supports("avx512bf16") && !(e && strcmp(e, "0") == 0);
}

const bool g_bf16 = detect_bf16();

typedef void (*BlockFn)(const float*, int, const uint16_t*, const uint16_t*, int, int, float*, int);

// Four rows per block (four weight streams per core), eight at B <= 3 on AVX-512 (the
// accumulators still fit the registers; interleaved A/B on the 16-core Zen 5 host,
// OPT-30B fc1 shape: +3-5 % at B = 1-3); the AVX-512 loop is unrolled twice at B <= 4
// (at B = 4, OPT-30B shapes: 327 -> 372 GB/s) and once with eight rows at B = 3, and
// from B = 5 on the batch runs in two groups per chunk (block512_split).  Blocks [ba, bb)
// of 4 rows from r0 (a grain starts at a multiple of 8 of them); the last block of the
// share may be partial.  A row's sums do not depend on the block it is computed in.
template <bool BF, int B>
void run_blocks(Isa isa, const float* x, int K, const uint16_t* W, const uint16_t* bias, int r0, int r1, int ba,
                int bb, float* y, int ldy) {
  constexpr int R = 4, UN = B <= 4 ? 2 : 1;
  constexpr bool R8 = B <= 3;
  BlockFn blk = isa != ISA_AVX512 ? block256<BF, B, R>
                : B >= 5         ? block512_split<BF, B, R>
                                 : block512<BF, B, R, UN>;
  BlockFn blk8 = isa == ISA_AVX512 && R8 ? block512<BF, B, 8, B <= 2 ? 2 : 1> : nullptr;
  BlockFn one = isa == ISA_AVX512 ? block512<BF, B, 1, 1> : block256<BF, B, 1>;
  for (int i = ba; i < bb;) {
    const int r = r0 + R * i;
    if (blk8 && i + 1 < bb && r + 2 * R <= r1) {
      blk8(x, K, W, bias, r0, r, y, ldy);
      i += 2;
      continue;
    }
    if (r + R <= r1) blk(x, K, W, bias, r0, r, y, ldy);
    else
      for (int q = r; q < r1; ++q) one(x, K, W, bias, r0, q, y, ldy);
    ++i;
  }
}

template <bool BF>
void run_blocks_b(Isa isa, const float* x, int B, int K, const uint16_t* W, const uint16_t* bias, int r0, int r1,
                  int ba, int bb, float* y, int ldy) {
  switch (B) {
    case 1: run_blocks<BF, 1>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 2: run_blocks<BF, 2>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 3: run_blocks<BF, 3>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 4: run_blocks<BF, 4>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 5: run_blocks<BF, 5>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 6: run_blocks<BF, 6>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    case 7: run_blocks<BF, 7>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
    default: run_blocks<BF, 8>(isa, x, K, W, bias, r0, r1, ba, bb, y, ldy); break;
  }
}

}  // namespace

const char* cpu_share_isa() {
  return g_isa == ISA_AVX512 ? (g_bf16 ? "avx512+bf16" : "avx512") : g_isa == ISA_AVX2 ? "avx2" : "scalar";
}

void team_streamed_chunks(long long delta) { g_streamed_chunks.fetch_add(delta, std::memory_order_relaxed); }

void team_for(int threads, int ngrains, void (*fn)(void*, int), void* arg) {
  Team::get().run(threads > 0 ? threads : omp_get_max_threads(), ngrains, fn, arg);
}

void cpu_share(const float* x, int B, int K, const uint16_t* W, int dtype, const uint16_t* bias, int r0, int r1,
               float* y, int ldy, int nthreads) {
  const int n = r1 - r0;
  if (n <= 0) return;
  const int nt_max = nthreads > 0 ? nthreads : omp_get_max_threads();
  // at least 8 rows per thread so short shares are not spread too thin
  int nt = (n + 7) / 8;
  if (nt > nt_max) nt = nt_max;
  if (nt < 1) nt = 1;
  struct Job {
    const float* x;
    int B, K;
    const uint16_t* W;
    int dtype;
    const uint16_t* bias;
    int r0, r1, blocks;
    float* y;
    int ldy;
    const uint16_t* xb;  // x narrowed to bf16 (bf16 weights on AVX512-BF16 hosts)
  } job{x, B, K, W, dtype, bias, r0, r1, (n + 3) / 4, y, ldy, nullptr};
  if (dtype == 1 && g_bf16) {
    // the calling thread's buffer: it stays valid while the job runs (the caller takes part)
    thread_local std::vector<uint16_t> xb;
    if (xb.size() < (size_t)B * K) xb.resize((size_t)B * K);
    if (narrow_bf16(x, B * K, xb.data())) job.xb = xb.data();
  }
  if (g_isa == ISA_SCALAR) {
    Team::get().run(nt, n, [](void* a, int g) {
      const Job& j = *(const Job*)a;
      rows_scalar(j.x, j.B, j.K, j.W, j.dtype, j.bias, j.r0, j.r0 + g, j.r0 + g + 1, j.y, j.ldy);
    }, &job);
    return;
  }
  // blocks of 4 rows handed out 8 at a time (32 rows, long sequential streams): a
  // core slowed by other work hands its remaining blocks to the others, which a
  // static split cannot (measured +5-38 % at batch 1 on the 16-core host).  Every
  // row is computed by one thread in the same order whatever the schedule.
  constexpr int kGrain = 8;
  const int grains = (job.blocks + kGrain - 1) / kGrain;
  Team::get().run(nt, grains, [](void* a, int g) {
    const Job& j = *(const Job*)a;
    const int ba = g * kGrain, bb = ba + kGrain < j.blocks ? ba + kGrain : j.blocks;
    if (j.xb) run_blocks_bf16_b(j.xb, j.B, j.K, j.W, j.bias, j.r0, j.r1, ba, bb, j.y, j.ldy);
    else if (j.dtype == 1) run_blocks_b<true>(g_isa, j.x, j.B, j.K, j.W, j.bias, j.r0, j.r1, ba, bb, j.y, j.ldy);
    else run_blocks_b<false>(g_isa, j.x, j.B, j.K, j.W, j.bias, j.r0, j.r1, ba, bb, j.y, j.ldy);
  }, &job);
}

}  // namespace hg
