// Host runtime of the heterogeneous-parallel Linear: context, pinned memory,
// the chunked host-to-device weight pipeline, the CPU/GPU split of one linear,
// the distribution-law planner and the decode step over a stack of linears.
//
// Dataflow of one linear with n_cpu CPU rows and n_gpu GPU rows (HeteGen Sec. 4.2,
// Fig. 5a, with the weights pinned once at load time so no per-call pinning):
//   1. the activation goes to the host: a kernel writes it as binary32 straight into
//      pinned host memory (no copy-engine queue in the way) and an event marks it;
//   2. the GPU rows are computed on the caller's stream: resident rows by one GEMV
//      launch, streamed rows chunk by chunk as the copy stream lands them in a ring
//      of device staging slots (ring slots are recycled through events);
//   3. the calling thread waits for the activation and computes the CPU rows on the
//      host cores while 2 proceeds;
//   4. a kernel reads the CPU rows from pinned memory, finishes them like the GPU
//      rows (ReLU / residual / rounding) and writes them into the output.
// Weights for later chunks are copied as soon as a ring slot is free, across
// linear and layer boundaries (Sec. 3.1: idle time is hidden by prefetching), by
// the context's parameter manager thread (Sec. 4.3), which owns the copy stream.
// Pageable weights take one more stage: the pin team copies each chunk into a
// pinned staging buffer while earlier chunks cross PCIe (Sec. 4.2, Fig. 5c).
#include <hip/hip_runtime_api.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <deque>
#include <exception>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/hetegen.h"
#include "attention.h"
#include "cpu_share.h"
#include "hbm_probe.h"
#include "kernels.h"
#include "pin_team.h"

namespace {

using Clock = std::chrono::steady_clock;

double ms_since(Clock::time_point t0) {
  return std::chrono::duration<double, std::milli>(Clock::now() - t0).count();
}

thread_local std::string g_create_error;

constexpr size_t kDefaultChunk = 32ull << 20;
constexpr uint32_t kDefaultSpinLimit = 1u << 22;  // polls of one grid-barrier wait (seconds)
constexpr int kBarrierGroups = 16;
constexpr size_t kCounterBytes = 256;
constexpr int kDefaultRing = 8;
constexpr int kMaxBatch = 8;
// Models created for batches of kTiledMinBatch or more keep their resident rows in the
// matrix-core tile order and run every batch of kTiledMinBatch or more on the matrix-core GEMV:
// the vector GEMV's dot products and reads of x grow with the batch (OPT-6.7B-shaped
// steps: 2.44 / 2.74 / 3.95 ms at batch 2 / 3 / 8 against 2.32 / 2.33 / 2.42 ms on the
// matrix cores), while at batch 1 the vector kernels with their fused LayerNorm are
// faster (2.19 against 2.30 ms); with both copies, batch 1 runs the row-major one.
constexpr int kTiledMinBatch = 2;
// Largest hidden size at which the matrix-core qkv and fc1 normalise their input from the
// LayerNorm partials of the linear before them: their prologue combines H / 16 partials per
// batch row before the first product, and above this a LayerNorm launch is cheaper (16-layer
// steps at batch 8 / 3: OPT-13B, H = 5120, 1.961 / 1.763 ms with partials against 2.029 /
// 1.820 with launches; OPT-30B, 7168, 3.557 / 3.137 against 3.529 / 3.174; OPT-66B, 9216,
// 5.727 / 5.113 against 5.584 / 5.115).  The choice depends on H alone, so that a batch row's
// bits do not depend on the batch size.
constexpr int kMaxPartialsH = 6144;
// Largest hidden size at which a model created for batches of 2 or more keeps a row-major
// copy beside its tiles for batch 1: above it batch 1 is faster on the tiles (all linears
// resident, created for batch 8, batch 1 per step: OPT-13B, H = 5120, 4.245 / 4.247 ms on
// the row-major copy against 4.302 / 4.304 on the tiles; OPT-30B, 7168, 9.450 / 9.452 against
// 9.293 / 9.294; OPT-66B, 9216, whose copies would not both fit, 20.18 ms on the tiles against
// 20.36-20.44 for a row-major model), and the tiles alone take half the memory.
constexpr int kMaxDualH = 6144;
// Resident row-major copies (batch 1) of GPU-only linears with K >= kMinSegmajorK (and K a
// multiple of hg::kSegElems) are stored segment-major: the batch-1 GEMV walks each row in
// 2048-element segments, every wavefront its own row, so in row-major order the wavefronts'
// loads fall on the same offsets of rows K * 2 bytes apart; segment-major, they read one
// contiguous window.  OPT-6.7B fc2 [4096, 16384]: 21.7 us against 22.1-22.8 us over weight
// placements (probe), the whole batch-1 step 2.168 against 2.203 ms (three runs each,
// alternating); out [4096, 4096] (two segments per row) gained nothing.
constexpr int kMinSegmajorK = 8192;
constexpr int kDefaultPinThreads = 4;
constexpr int kDefaultPinRing = 4;

}  // namespace

struct hetegen_ctx {
  int device = 0;
  int cpu_threads = 0;
  size_t chunk_bytes = kDefaultChunk;
  int ring = kDefaultRing;
  hipStream_t copy_stream = nullptr;
  hipStream_t capture_stream = nullptr;
  std::vector<void*> slot;
  std::vector<hipEvent_t> ev_ready, ev_free;
  hipEvent_t ev_x = nullptr, ev_y = nullptr;
  // pinned hand-off buffers (binary32), grown on demand
  float* x_host = nullptr;
  size_t x_host_bytes = 0;
  float* y_host = nullptr;
  size_t y_host_bytes = 0;
  bool y_pending = false;  // ev_y recorded after the last read of y_host
  // streamed-chunk pipeline, shared with the parameter manager thread under `mu`.
  // Chunk number s goes to ring slot s % ring; its copy may be enqueued once the
  // GEMV of chunk s - ring has been enqueued (head > s - ring).
  struct Chunk {
    const char* src;
    size_t bytes;
    bool pageable;
    bool host_wait;  // the slot wait may block the manager (the linear has no CPU rows)
  };
  std::mutex mu;
  std::condition_variable cv;
  std::deque<Chunk> jobs;  // planned chunks whose GEMV is not enqueued; front() is number `head`
  long long head = 0;
  long long copy_enq = 0;  // copies of chunks numbered below copy_enq are enqueued
  bool busy = false, stop = false, failed = false;
  std::string mgr_err;
  std::thread mgr;
  // pageable weights: pinned staging buffers and the team that fills them
  int pin_threads = kDefaultPinThreads;  // < 0: pageable weights refused
  int pin_ring = kDefaultPinRing;
  int numa_node = -1;                     // node of pinned allocations; < 0: thread policy
  std::vector<void*> bounce;
  std::vector<hipEvent_t> ev_bounce;
  long long bounce_seq = 0;  // manager thread only
  hg::PinTeam team;
  // profiling (the manager records copy events too: `prof_mu`)
  std::mutex prof_mu;
  bool profiling = false;
  struct Timed {
    hipEvent_t a, b;
    int kind;  // 0 = copy, 1 = gemv
    double bytes;
  };
  std::vector<Timed> timed;
  std::vector<hipEvent_t> ev_pool;
  hetegen_profile prof{};
  std::string err;
  // HETEGEN_POISON at creation: staging slots, pinned staging buffers and hand-off buffers
  // are filled with all-ones bits (NaN in fp16, bf16 and binary32) before every reuse
  bool poison = false;
  // split-K workspace of hetegen_linear_tiled (grown on demand; counters zero between launches)
  float* ws = nullptr;
  size_t ws_floats = 0;
  uint32_t* ws_cnt = nullptr;
  size_t ws_words = 0;
};

struct hetegen_model {
  struct Lin {
    int N = 0, K = 0;
    const void* W_host = nullptr;
    const void* bias_host = nullptr;
    double alpha = 0;
    int resident = 0;
    int n_gpu = 0, n_cpu = 0;
    bool pageable = false;     // W_host is plain host memory (staged when streamed)
    void* W_dev = nullptr;     // rows [0, n_gpu) when resident, row-major (batch 1 and row-major models)
    void* W_tile = nullptr;    // the same rows in matrix-core tile order (tiled models)
    int korder = 0;            // W_tile's order: 0 row-tile order, 1 k-major (hg::mfma_kmajor)
    int segmajor = 0;          // W_dev segment-major (hg::launch_segmajor; see kMinSegmajorK)
    void* bias_dev = nullptr;  // all N biases
  };
  int L = 0, H = 0, F = 0, dtype = 0, max_batch = 1;
  bool tiled = false;          // resident rows in matrix-core tile order (max_batch >= kTiledMinBatch)
  bool rowmajor = true;        // resident rows row-major (all models below kTiledMinBatch; tiled ones when
                               // both copies fit, see hetegen_model_create)
  float* ws = nullptr;         // split-K partials of the matrix-core GEMV
  uint32_t* ws_cnt = nullptr;  // its arrival counters, zero between launches
  size_t ws_floats = 0, ws_words = 0;
  float* ln_part = nullptr;    // LayerNorm partials of x after out / fc2 (two buffers of
                               // ln_partials_floats(H)), for the tiled GEMVs of fc1 / qkv
  bool ln_partials = true;     // use them (H <= kMaxPartialsH; HETEGEN_LN_PARTIALS=0 / 1 at creation forces)
  std::vector<Lin> lin;
  std::vector<double> lin_ms;  // host time of each linear in the last eager step
  void* arena = nullptr;  // device memory for resident weights and biases
  void* act = nullptr;    // device activations: x, qkv, f, ln
  void *xbuf = nullptr, *qkv = nullptr, *fbuf = nullptr, *lnbuf = nullptr;
  void* trace = nullptr;
  size_t trace_bytes = 0;
  // graph replay of an all-resident, GPU-only step
  bool graphable = false;
  hipGraphExec_t gexec = nullptr;
  int g_B = 0;
  const void* g_x = nullptr;
  void* g_out = nullptr;
  // persistent step (one cooperative launch per step), per batch size
  struct StepPlan {
    bool built = false, ok = false;
    void* table = nullptr;  // device StepLinear[4L]
    int grid = 0;
    size_t lds = 0;
  };
  StepPlan plan[kMaxBatch + 1];
  uint32_t* counters = nullptr;  // device barrier counters
  int ngroups = 0;
  int* err_host = nullptr;       // pinned: set by a barrier wait that gave up
  uint32_t barrier_base = 0;
  uint32_t spin_limit = 0;       // 0: the kernel's default
  int exec_mode = HETEGEN_EXEC_AUTO;
  int last_exec = 0;
  // KV cache of attention steps (Sec. 2.1, Eq. 1): K then V of every layer, each
  // [max_batch][heads][kv_seq][head_dim] in the model dtype
  int kv_seq = 0, head_dim = 0, heads = 0, kv_chunks = 0;
  void* kv = nullptr;
  float* kv_part = nullptr;    // chunk partials of the attention merge
  uint32_t* kv_cnt = nullptr;  // arrival counters of the merge, zero between launches
  void* abuf = nullptr;        // attention output [max_batch, H]
};

namespace {

hetegen_status fail(hetegen_ctx* ctx, hetegen_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx) ctx->err = buf;
  else g_create_error = buf;
  return code;
}

// Every exported call returns a status and lets no exception cross the C ABI: host
// allocation failures (vectors, queues, messages) become HETEGEN_ERR_OOM, anything else
// HETEGEN_ERR_INTERNAL; building the message may itself fail, so it is best-effort.
template <class F>
hetegen_status api_guard(hetegen_ctx* ctx, F&& f) noexcept {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    try {
      fail(ctx, HETEGEN_ERR_OOM, "host memory exhausted");
    } catch (...) {
    }
    return HETEGEN_ERR_OOM;
  } catch (const std::exception& e) {
    try {
      fail(ctx, HETEGEN_ERR_INTERNAL, "internal error: %s", e.what());
    } catch (...) {
    }
    return HETEGEN_ERR_INTERNAL;
  } catch (...) {
    try {
      fail(ctx, HETEGEN_ERR_INTERNAL, "internal error");
    } catch (...) {
    }
    return HETEGEN_ERR_INTERNAL;
  }
}

#define HIPCHK(ctx, expr)                                                                           \
  do {                                                                                              \
    hipError_t e_ = (expr);                                                                         \
    if (e_ != hipSuccess)                                                                           \
      return fail((ctx), HETEGEN_ERR_HIP, "%s failed: %s (%d)", #expr, hipGetErrorString(e_), (int)e_); \
  } while (0)

#define TRY(expr)                        \
  do {                                   \
    hetegen_status s_ = (expr);          \
    if (s_ != HETEGEN_OK) return s_;     \
  } while (0)

inline size_t elem_size(int dtype) { return dtype == HETEGEN_F32 ? 4 : 2; }

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int split_cpu_rows(int N, double alpha) {
  double c = floor(alpha * (double)N + 0.5);
  if (c < 0) c = 0;
  if (c > N) c = N;
  return (int)c;
}

// hipHostMalloc on the context's NUMA node: the calling thread's memory policy is set
// to bind to that node around the allocation (which then follows it) and restored.
hipError_t host_malloc(const hetegen_ctx* ctx, void** p, size_t bytes, unsigned flags) {
  if (ctx->numa_node < 0) return hipHostMalloc(p, bytes, flags);
  constexpr int kMpolBind = 2;
  int old_mode = 0;
  unsigned long old_mask[16] = {0};
  const bool saved = syscall(SYS_get_mempolicy, &old_mode, old_mask, 16 * 8 * sizeof(unsigned long), nullptr, 0) == 0;
  unsigned long mask[16] = {0};
  mask[ctx->numa_node / 64] = 1ul << (ctx->numa_node % 64);
  if (syscall(SYS_set_mempolicy, kMpolBind, mask, 16 * 8 * sizeof(unsigned long)) != 0) return hipErrorInvalidValue;
  const hipError_t e = hipHostMalloc(p, bytes, flags | hipHostMallocNumaUser);
  if (saved) (void)syscall(SYS_set_mempolicy, old_mode, old_mask, 16 * 8 * sizeof(unsigned long));
  else (void)syscall(SYS_set_mempolicy, 0, nullptr, 0);
  return e;
}

hetegen_status ensure_host(hetegen_ctx* ctx, float** buf, size_t* have, size_t need) {
  if (*have >= need) return HETEGEN_OK;
  if (*buf) {
    hipError_t e = hipHostFree(*buf);
    *buf = nullptr;
    *have = 0;
    if (e != hipSuccess) return fail(ctx, HETEGEN_ERR_HIP, "hipHostFree: %s", hipGetErrorString(e));
  }
  size_t bytes = std::max(need, (size_t)1 << 20);
  // coherent: written by kernels and read by the host (and the reverse) around events
  if (host_malloc(ctx, (void**)buf, bytes, hipHostMallocCoherent) != hipSuccess) {
    (void)hipGetLastError();
    *buf = nullptr;
    return fail(ctx, HETEGEN_ERR_OOM, "pinned hand-off buffer of %zu bytes", bytes);
  }
  *have = bytes;
  return HETEGEN_OK;
}

hetegen_status check_pinned(hetegen_ctx* ctx, const void* p, size_t bytes);

// Pinned weights are copied straight from W_host; pageable ones (plain host memory
// that HIP does not know) are staged through the pinned buffers unless the context
// refuses them.
hetegen_status check_weight(hetegen_ctx* ctx, const void* p, size_t bytes, bool* pageable) {
  *pageable = false;
  hipPointerAttribute_t a;
  hipError_t e = hipPointerGetAttributes(&a, p);
  if (e != hipSuccess) (void)hipGetLastError();
  if (e != hipSuccess || a.type == hipMemoryTypeUnregistered) {
    if (ctx->pin_threads < 0)
      return fail(ctx, HETEGEN_ERR_NOT_PINNED, "host weight %p is not page-locked memory", p);
    *pageable = true;
    return HETEGEN_OK;
  }
  return check_pinned(ctx, p, bytes);
}

hetegen_status check_pinned(hetegen_ctx* ctx, const void* p, size_t bytes) {
  const char* ends[2] = {(const char*)p, (const char*)p + bytes - 1};
  for (const char* q : ends) {
    hipPointerAttribute_t a;
    hipError_t e = hipPointerGetAttributes(&a, q);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(ctx, HETEGEN_ERR_NOT_PINNED, "host weight %p is not page-locked memory", (const void*)q);
    }
    if (a.type != hipMemoryTypeHost)
      return fail(ctx, HETEGEN_ERR_NOT_PINNED, "weight %p is not pinned host memory (type %d)", (const void*)q,
                  (int)a.type);
  }
  return HETEGEN_OK;
}

// ---- profiling helpers ----
hipEvent_t pool_event(hetegen_ctx* ctx) {
  std::lock_guard<std::mutex> lk(ctx->prof_mu);
  if (!ctx->ev_pool.empty()) {
    hipEvent_t e = ctx->ev_pool.back();
    ctx->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return e;
}

hetegen_status flush_profile(hetegen_ctx* ctx) {
  std::lock_guard<std::mutex> lk(ctx->prof_mu);
  for (auto& t : ctx->timed) {
    HIPCHK(ctx, hipEventSynchronize(t.b));
    float ms = 0;
    HIPCHK(ctx, hipEventElapsedTime(&ms, t.a, t.b));
    if (t.kind == 0) {
      ctx->prof.h2d_ms += ms;
      ctx->prof.h2d_bytes += t.bytes;
    } else {  // 1: a GEMV of streamed chunk rows, 2: of resident rows
      ctx->prof.gpu_ms += ms;
      ctx->prof.gpu_bytes += t.bytes;
      ctx->prof.gemv_launches++;
      if (t.kind == 2) {
        ctx->prof.res_gpu_ms += ms;
        ctx->prof.res_gpu_bytes += t.bytes;
      }
    }
    ctx->ev_pool.push_back(t.a);
    ctx->ev_pool.push_back(t.b);
  }
  ctx->timed.clear();
  return HETEGEN_OK;
}

struct TimedScope {
  hetegen_ctx* ctx;
  hipStream_t s;
  hipEvent_t a = nullptr;
  int kind;
  double bytes;
  TimedScope(hetegen_ctx* c, hipStream_t st, int k, double by) : ctx(c), s(st), kind(k), bytes(by) {
    if (ctx->profiling) {
      a = pool_event(ctx);
      if (a) (void)hipEventRecord(a, s);
    }
  }
  void end() {
    if (!a) return;
    hipEvent_t b = pool_event(ctx);
    if (!b) return;
    (void)hipEventRecord(b, s);
    std::lock_guard<std::mutex> lk(ctx->prof_mu);
    ctx->timed.push_back({a, b, kind, bytes});
    a = nullptr;
  }
};

// ---- streamed-chunk pipeline: the parameter manager ----
// Copy chunk number s into its ring slot after the GEMV that last read the slot; a
// pageable chunk is first staged into a pinned buffer whose previous copy has
// completed.  Runs on the manager thread.  A wait of the copy stream on the compute
// stream queued in front of a copy leaves the copy engine idle for tens of
// microseconds (pinned 32 MiB chunks: 51.4 against 55.4 GB/s), so the slot wait is
// skipped when that GEMV has already completed, and otherwise taken on the host when
// nothing else depends on how far ahead the manager runs (the chunk's linear has no
// CPU rows, so the calling thread only waits for the copies in order; the copies
// already queued keep the engine busy).  For a linear with CPU rows the calling
// thread enqueues the GEMVs of its chunks before the CPU share, which needs their
// copies enqueued without waiting for the GPU: there the wait stays on the stream.
bool copy_chunk(hetegen_ctx* ctx, long long s, const hetegen_ctx::Chunk& c, std::string* err) {
  const int slot = (int)(s % ctx->ring);
  hipError_t e;
#define MGR_HIP(expr)                                                           \
  do {                                                                        \
    if ((e = (expr)) != hipSuccess) {                                         \
      *err = std::string(#expr) + " failed: " + hipGetErrorString(e);         \
      return false;                                                           \
    }                                                                         \
  } while (0)
  const void* src = c.src;
  int b = -1;
  if (c.pageable) {
    b = (int)(ctx->bounce_seq++ % ctx->pin_ring);
    MGR_HIP(hipEventSynchronize(ctx->ev_bounce[b]));  // its previous copy has read it
    if (ctx->poison) memset(ctx->bounce[b], 0xFF, ctx->chunk_bytes);
    const auto t0 = Clock::now();
    ctx->team.copy((char*)ctx->bounce[b], c.src, c.bytes);
    {
      std::lock_guard<std::mutex> lk(ctx->prof_mu);
      ctx->prof.pin_ms += ms_since(t0);
      ctx->prof.pin_bytes += (double)c.bytes;
    }
    src = ctx->bounce[b];
  }
  const hipError_t q = hipEventQuery(ctx->ev_free[slot]);
  if (q != hipSuccess) {
    if (q != hipErrorNotReady) MGR_HIP(q);
    (void)hipGetLastError();  // not an error
    if (c.host_wait) MGR_HIP(hipEventSynchronize(ctx->ev_free[slot]));
    else MGR_HIP(hipStreamWaitEvent(ctx->copy_stream, ctx->ev_free[slot], 0));
  }
  // poisoned slot: a GEMV that read it before this copy landed, or past the chunk, sees NaN
  if (ctx->poison) MGR_HIP(hipMemsetAsync(ctx->slot[slot], 0xFF, ctx->chunk_bytes, ctx->copy_stream));
  TimedScope ts(ctx, ctx->copy_stream, 0, (double)c.bytes);
  MGR_HIP(hipMemcpyAsync(ctx->slot[slot], src, c.bytes, hipMemcpyHostToDevice, ctx->copy_stream));
  ts.end();
  MGR_HIP(hipEventRecord(ctx->ev_ready[slot], ctx->copy_stream));
  if (b >= 0) MGR_HIP(hipEventRecord(ctx->ev_bounce[b], ctx->copy_stream));
#undef MGR_HIP
  return true;
}

void manager_main(hetegen_ctx* ctx) {
  (void)hipSetDevice(ctx->device);
  std::unique_lock<std::mutex> lk(ctx->mu);
  for (;;) {
    ctx->cv.wait(lk, [&] {
      return ctx->stop || (!ctx->failed && ctx->copy_enq < ctx->head + (long long)ctx->jobs.size() &&
                           ctx->copy_enq - ctx->head < ctx->ring);
    });
    if (ctx->stop) return;
    const long long s = ctx->copy_enq;
    const hetegen_ctx::Chunk c = ctx->jobs[(size_t)(s - ctx->head)];
    ctx->busy = true;
    lk.unlock();
    std::string err;
    const bool ok = copy_chunk(ctx, s, c, &err);
    lk.lock();
    ctx->busy = false;
    if (ok) ctx->copy_enq = s + 1;
    else {
      ctx->failed = true;
      ctx->mgr_err = err;
    }
    ctx->cv.notify_all();
  }
}

int chunk_rows_for(const hetegen_ctx* ctx, int K, int dtype) {
  size_t row = (size_t)K * elem_size(dtype);
  size_t r = ctx->chunk_bytes / row;
  return r < 1 ? 1 : (int)std::min<size_t>(r, (size_t)1 << 30);
}

bool pipeline_idle(hetegen_ctx* ctx) {
  std::lock_guard<std::mutex> lk(ctx->mu);
  return ctx->jobs.empty();
}

// Pinned staging buffers and the pin team, at the first pageable chunk.
// Called with the pipeline idle (no copy in flight on the manager thread).
hetegen_status ensure_pin_resources(hetegen_ctx* ctx) {
  if (ctx->team.started()) return HETEGEN_OK;
  ctx->bounce.resize(ctx->pin_ring, nullptr);
  ctx->ev_bounce.resize(ctx->pin_ring, nullptr);
  for (int i = 0; i < ctx->pin_ring; ++i) {
    if (!ctx->bounce[i] && host_malloc(ctx, &ctx->bounce[i], ctx->chunk_bytes, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      ctx->bounce[i] = nullptr;
      return fail(ctx, HETEGEN_ERR_OOM, "pinned staging buffer of %zu bytes", ctx->chunk_bytes);
    }
    if (!ctx->ev_bounce[i]) {
      HIPCHK(ctx, hipEventCreateWithFlags(&ctx->ev_bounce[i], hipEventDisableTiming));
      HIPCHK(ctx, hipEventRecord(ctx->ev_bounce[i], ctx->copy_stream));
    }
  }
  if (!ctx->team.start(ctx->pin_threads)) return fail(ctx, HETEGEN_ERR_OOM, "pin team threads");
  return HETEGEN_OK;
}

// Queue the chunks of rows [0, n_gpu) of one streamed weight; the manager starts
// copying at once.
void plan_chunks(hetegen_ctx* ctx, const void* W_host, int n_gpu, int K, int dtype, bool pageable, bool host_wait) {
  const size_t row = (size_t)K * elem_size(dtype);
  const int cr = chunk_rows_for(ctx, K, dtype);
  {
    std::lock_guard<std::mutex> lk(ctx->mu);
    long long n = 0;
    for (int r0 = 0; r0 < n_gpu; r0 += cr, ++n) {
      int nr = std::min(cr, n_gpu - r0);
      ctx->jobs.push_back({(const char*)W_host + (size_t)r0 * row, (size_t)nr * row, pageable, host_wait});
    }
    hg::team_streamed_chunks(n);
  }
  ctx->cv.notify_all();
}

// The oldest planned chunk: whether its copy is enqueued (waiting for it when
// `block`, or when `block_pinned` and the chunk is pinned), its number and size.
hetegen_status front_chunk(hetegen_ctx* ctx, bool block, bool block_pinned, bool* ready, long long* seq,
                           size_t* bytes) {
  std::unique_lock<std::mutex> lk(ctx->mu);
  if (ctx->jobs.empty()) {
    lk.unlock();
    return fail(ctx, HETEGEN_ERR_INVALID_ARG, "internal: chunk pipeline is empty");
  }
  if (block || (block_pinned && !ctx->jobs.front().pageable))
    ctx->cv.wait(lk, [&] { return ctx->failed || ctx->copy_enq > ctx->head; });
  if (ctx->failed) {
    const std::string m = ctx->mgr_err;
    lk.unlock();
    return fail(ctx, HETEGEN_ERR_HIP, "parameter manager: %s", m.c_str());
  }
  *ready = ctx->copy_enq > ctx->head;
  *seq = ctx->head;
  *bytes = ctx->jobs.front().bytes;
  return HETEGEN_OK;
}

void pop_chunk(hetegen_ctx* ctx) {
  {
    std::lock_guard<std::mutex> lk(ctx->mu);
    ctx->jobs.pop_front();
    ctx->head++;
    hg::team_streamed_chunks(-1);
  }
  ctx->cv.notify_all();
}

// Drop the planned chunks after a failed call (copies already enqueued complete on
// the copy stream; nothing reads them).
void reset_pipeline(hetegen_ctx* ctx) {
  std::unique_lock<std::mutex> lk(ctx->mu);
  ctx->cv.wait(lk, [&] { return !ctx->busy; });
  hg::team_streamed_chunks(-(long long)ctx->jobs.size());
  ctx->jobs.clear();
  ctx->head = ctx->copy_enq;
  ctx->failed = false;
  ctx->mgr_err.clear();
}

// ---- one linear ----
struct Job {
  const void* x;
  long long ldx;
  int B, K, N, dtype;
  const void* W_host;
  const void* W_dev;  // rows [0, n_gpu) resident, or nullptr (streamed)
  const void* bias_host;
  const void* bias_dev;
  int n_gpu, n_cpu;
  void* y;
  long long ldy;
  int y_f32;
  int epi;
  const void* resid;
  long long ldr;
  int ln;
  void* ln_buf;     // device [B, K] for the normalised input when it must be materialised
  void* trace_in;   // optional copy of the linear's input [B, K]
  void* trace_out;  // optional copy of the output [B, N]
  bool tiled;       // W_dev is in matrix-core tile order (matrix-core GEMV)
  float* ws;        // its split-K workspace
  uint32_t* cnt;
  size_t ws_floats, cnt_words;
  int korder;       // tiled: W_dev's tile order
  int segmajor;     // W_dev segment-major (resident row-major copy, batch 1)
  const float* ln_in;  // tiled, ln, all rows resident: LayerNorm from these partials of x
  float* ln_out;       // tiled, all rows resident: also write the partials of y here
};

hetegen_status run_gemv(hetegen_ctx* ctx, const Job& j, const void* x, long long ldx, int ln, const void* W, int row0,
                        int rows, hipStream_t st, void* h_out, bool tiled = false, bool resident = false) {
  hg::GemvParams p{};
  const size_t ys = j.y_f32 ? 4 : 2;
  p.x = x;
  p.ldx = ldx;
  p.W = W;
  p.bias = j.bias_dev ? (const char*)j.bias_dev + (size_t)row0 * 2 : nullptr;
  p.y = (char*)j.y + (size_t)row0 * ys;
  p.ldy = j.ldy;
  p.resid = j.resid ? (const char*)j.resid + (size_t)row0 * 2 : nullptr;
  p.ldr = j.ldr;
  p.h_out = h_out;
  p.ldh = j.K;
  p.rows = rows;
  p.K = j.K;
  p.epi = j.epi;
  p.y_f32 = j.y_f32;
  p.ln = ln;
  p.segmajor = resident && !tiled ? j.segmajor : 0;
  TimedScope ts(ctx, st, resident ? 2 : 1, (double)rows * j.K * 2);
  if (tiled) {
    p.ws = j.ws;
    p.cnt = j.cnt;
    p.ws_floats = j.ws_floats;
    p.cnt_words = j.cnt_words;
    p.korder = j.korder;
    p.ln_in = ln ? j.ln_in : nullptr;
    p.ln_out = j.ln_out;
    HIPCHK(ctx, hg::launch_gemv_mfma(p, j.dtype, j.B, st));
  } else {
    HIPCHK(ctx, hg::launch_gemv(p, j.dtype, j.B, st, 0));
  }
  ts.end();
  return HETEGEN_OK;
}

hetegen_status run_linear(hetegen_ctx* ctx, const Job& j, hipStream_t st) {
  const auto tl = Clock::now();
  const size_t s = 2;
  // the LayerNorm inside the one resident GEMV: the vector kernels normalise x themselves,
  // the matrix-core kernel from the partials its producer wrote
  const bool fused_ln = j.ln && j.n_cpu == 0 && j.W_dev != nullptr &&
                        (j.tiled ? j.ln_in != nullptr : hg::gemv_fuses_ln(j.B));
  const void* xin = j.x;
  long long ldin = j.ldx;
  // 1. input: materialise LayerNorm(x) unless it is fused into one resident GEMV,
  //    and hand the input to the host when there are CPU rows.
  if (j.ln && !fused_ln) {
    if (j.n_cpu > 0) TRY(ensure_host(ctx, &ctx->x_host, &ctx->x_host_bytes, (size_t)j.B * j.K * 4));
    HIPCHK(ctx, hg::launch_layernorm(j.x, j.ldx, j.B, j.K, j.dtype, j.ln_buf, j.K, j.n_cpu > 0 ? ctx->x_host : nullptr,
                                     st));
    xin = j.ln_buf;
    ldin = j.K;
  } else if (j.n_cpu > 0) {
    TRY(ensure_host(ctx, &ctx->x_host, &ctx->x_host_bytes, (size_t)j.B * j.K * 4));
    HIPCHK(ctx, hg::launch_export_f32(j.x, j.ldx, j.B, j.K, j.dtype, ctx->x_host, st));
  }
  if (j.n_cpu > 0) HIPCHK(ctx, hipEventRecord(ctx->ev_x, st));
  if (j.trace_in && !fused_ln)
    HIPCHK(ctx, hipMemcpy2DAsync(j.trace_in, (size_t)j.K * s, xin, (size_t)ldin * s, (size_t)j.K * s, j.B,
                                 hipMemcpyDeviceToDevice, st));
  // 2. GPU rows: one GEMV when resident; otherwise one GEMV per streamed chunk, each
  //    waiting on the copy stream for its slot.  Before the CPU share only chunks
  //    whose copy is already enqueued, or will be at once (pinned chunks wait only
  //    for slots that these GEMVs free), so that staging pageable weights does not
  //    hold up the CPU share; the rest after it.
  const bool streamed = j.n_gpu > 0 && !j.W_dev;
  int r0 = 0;
  const int cr = chunk_rows_for(ctx, j.K, j.dtype);
  auto next_chunk = [&](bool block, bool* did) -> hetegen_status {
    *did = false;
    bool ready = false;
    long long seq = 0;
    size_t bytes = 0;
    TRY(front_chunk(ctx, block, true, &ready, &seq, &bytes));
    if (!ready) return HETEGEN_OK;
    const int nr = std::min(cr, j.n_gpu - r0);
    if (bytes != (size_t)nr * j.K * s) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "internal: chunk plan out of step");
    const int slot = (int)(seq % ctx->ring);
    // a copy that has already completed needs no wait; queuing a wait on the copy
    // stream costs the calling thread ~20 us per chunk, on the path between two CPU
    // shares (the event's last record is this chunk's copy: front_chunk saw it issued)
    const hipError_t q = hipEventQuery(ctx->ev_ready[slot]);
    if (q == hipErrorNotReady) {
      (void)hipGetLastError();  // not an error: keep it from surfacing at the next launch check
      HIPCHK(ctx, hipStreamWaitEvent(st, ctx->ev_ready[slot], 0));
    } else {
      HIPCHK(ctx, q);
    }
    TRY(run_gemv(ctx, j, xin, ldin, 0, ctx->slot[slot], r0, nr, st, nullptr));
    HIPCHK(ctx, hipEventRecord(ctx->ev_free[slot], st));
    pop_chunk(ctx);
    r0 += nr;
    *did = true;
    return HETEGEN_OK;
  };
  if (j.n_gpu > 0 && j.W_dev)
    TRY(run_gemv(ctx, j, xin, ldin, fused_ln ? 1 : 0, j.W_dev, 0, j.n_gpu, st, fused_ln ? j.trace_in : nullptr,
                 j.tiled, true));
  while (streamed && r0 < j.n_gpu) {
    bool did = false;
    TRY(next_chunk(j.n_cpu == 0, &did));
    if (!did) break;
  }
  // 3. CPU rows on the calling thread and the CPU share's worker team
  if (j.n_cpu > 0) {
    // the previous import kernel may still read y_host (it precedes ev_x in stream
    // order, so this wait is part of the wait for the input)
    const auto tw = Clock::now();
    if (ctx->y_pending) HIPCHK(ctx, hipEventSynchronize(ctx->ev_y));
    ctx->y_pending = false;
    TRY(ensure_host(ctx, &ctx->y_host, &ctx->y_host_bytes, (size_t)j.B * j.n_cpu * 4));
    if (ctx->poison) memset(ctx->y_host, 0xFF, (size_t)j.B * j.n_cpu * 4);  // rows the CPU share leaves unwritten
    HIPCHK(ctx, hipEventSynchronize(ctx->ev_x));
    ctx->prof.xwait_ms += ms_since(tw);
    ctx->prof.cpu_shares++;
    auto t0 = Clock::now();
    hg::cpu_share(ctx->x_host, j.B, j.K, (const uint16_t*)j.W_host, j.dtype, (const uint16_t*)j.bias_host, j.n_gpu, j.N,
                  ctx->y_host, j.n_cpu, ctx->cpu_threads);
    ctx->prof.cpu_ms += ms_since(t0);
    ctx->prof.cpu_bytes += (double)j.n_cpu * j.K * s;
    // the next CPU share must wait for its own hand-off: poisoned, a read before it lands is NaN
    if (ctx->poison) memset(ctx->x_host, 0xFF, (size_t)j.B * j.K * 4);
    // 4. finish and place the CPU rows
    const size_t ys = j.y_f32 ? 4 : 2;
    HIPCHK(ctx, hg::launch_import_rows(ctx->y_host, j.B, j.n_cpu, j.dtype, j.epi, (char*)j.y + (size_t)j.n_gpu * ys,
                                       j.ldy, j.y_f32, j.resid ? (const char*)j.resid + (size_t)j.n_gpu * 2 : nullptr,
                                       j.ldr, st));
    HIPCHK(ctx, hipEventRecord(ctx->ev_y, st));
    ctx->y_pending = true;
  }
  const auto tt = Clock::now();
  while (streamed && r0 < j.n_gpu) {
    bool did = false;
    TRY(next_chunk(true, &did));
  }
  if (j.n_cpu > 0) ctx->prof.tailwait_ms += ms_since(tt);
  if (j.trace_out)
    HIPCHK(ctx, hipMemcpy2DAsync(j.trace_out, (size_t)j.N * s, j.y, (size_t)j.ldy * s, (size_t)j.N * s, j.B,
                                 hipMemcpyDeviceToDevice, st));
  if (j.n_cpu > 0) ctx->prof.hetlin_ms += ms_since(tl);
  return HETEGEN_OK;
}

hetegen_status finish_call(hetegen_ctx* ctx, Clock::time_point t0) {
  if (ctx->profiling) TRY(flush_profile(ctx));
  ctx->prof.wall_ms += ms_since(t0);
  return HETEGEN_OK;
}

}  // namespace

extern "C" {

hetegen_status hetegen_create(const hetegen_config* cfg, hetegen_ctx** out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!out) return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    hetegen_config c{};
    if (cfg) c = *cfg;
    if (c.ring_depth == 0) c.ring_depth = kDefaultRing;
    if (c.chunk_bytes == 0) c.chunk_bytes = kDefaultChunk;
    if (c.ring_depth < 2 || c.ring_depth > 64)
      return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "ring_depth %d outside [2, 64]", c.ring_depth);
    if (c.chunk_bytes < 4096 || (c.chunk_bytes & 15u))
      return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "chunk_bytes %zu must be >= 4096 and a multiple of 16",
                  c.chunk_bytes);
    if (c.pin_threads == 0) c.pin_threads = kDefaultPinThreads;
    if (c.pin_ring == 0) c.pin_ring = kDefaultPinRing;
    if (c.pin_threads > 64 || c.pin_ring < 2 || c.pin_ring > 64)
      return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "pin_threads %d must be <= 64 and pin_ring %d in [2, 64]",
                  c.pin_threads, c.pin_ring);
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess || ndev <= 0) {
      (void)hipGetLastError();
      return fail(nullptr, HETEGEN_ERR_HIP, "no HIP device (%s)", hipGetErrorString(e));
    }
    if (c.device < 0 || c.device >= ndev)
      return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "device %d outside [0, %d)", c.device, ndev);
    if (c.numa_node < 0 || c.numa_node > 1024)
      return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "numa_node %d outside [0, 1024]", c.numa_node);
    if (c.numa_node > 0) {
      char path[64];
      snprintf(path, sizeof path, "/sys/devices/system/node/node%d", c.numa_node - 1);
      if (access(path, F_OK) != 0)
        return fail(nullptr, HETEGEN_ERR_INVALID_ARG, "NUMA node %d does not exist", c.numa_node - 1);
    }
    hetegen_ctx* ctx = new hetegen_ctx();
    ctx->device = c.device;
    ctx->cpu_threads = c.cpu_threads;
    ctx->chunk_bytes = c.chunk_bytes;
    ctx->ring = c.ring_depth;
    ctx->pin_threads = c.pin_threads < 0 ? -1 : c.pin_threads;
    ctx->pin_ring = c.pin_ring;
    ctx->numa_node = c.numa_node - 1;
    {
      const char* pe = getenv("HETEGEN_POISON");
      ctx->poison = pe && *pe && strcmp(pe, "0") != 0;
    }
    auto bail = [&](hetegen_status st) {
      g_create_error = ctx->err;
      hetegen_destroy(ctx);
      return st;
    };
    if (hipSetDevice(c.device) != hipSuccess) return bail(fail(ctx, HETEGEN_ERR_HIP, "hipSetDevice(%d)", c.device));
    // address of this device's fixed split-K scratch (hetegen_linear_tiled_noalloc), once per device
    {
      const hipError_t se = hg::scratch_init(c.device);
      if (se != hipSuccess) return bail(fail(ctx, HETEGEN_ERR_HIP, "scratch set-up: %s", hipGetErrorString(se)));
    }
    if (hipStreamCreateWithFlags(&ctx->copy_stream, hipStreamNonBlocking) != hipSuccess ||
        hipStreamCreateWithFlags(&ctx->capture_stream, hipStreamNonBlocking) != hipSuccess)
      return bail(fail(ctx, HETEGEN_ERR_HIP, "stream creation failed"));
    if (hipEventCreateWithFlags(&ctx->ev_x, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ctx->ev_y, hipEventDisableTiming) != hipSuccess)
      return bail(fail(ctx, HETEGEN_ERR_HIP, "event creation failed"));
    ctx->slot.assign(c.ring_depth, nullptr);
    ctx->ev_ready.assign(c.ring_depth, nullptr);
    ctx->ev_free.assign(c.ring_depth, nullptr);
    for (int i = 0; i < c.ring_depth; ++i) {
      if (hipMalloc(&ctx->slot[i], c.chunk_bytes) != hipSuccess) {
        (void)hipGetLastError();
        ctx->slot[i] = nullptr;
        return bail(fail(ctx, HETEGEN_ERR_OOM, "staging slot of %zu bytes", c.chunk_bytes));
      }
      if (hipEventCreateWithFlags(&ctx->ev_ready[i], hipEventDisableTiming) != hipSuccess ||
          hipEventCreateWithFlags(&ctx->ev_free[i], hipEventDisableTiming | hipEventBlockingSync) != hipSuccess)
        return bail(fail(ctx, HETEGEN_ERR_HIP, "event creation failed"));
      if (ctx->poison && hipMemset(ctx->slot[i], 0xFF, c.chunk_bytes) != hipSuccess)
        return bail(fail(ctx, HETEGEN_ERR_HIP, "staging slot poisoning failed"));
      // every slot starts free
      if (hipEventRecord(ctx->ev_free[i], ctx->copy_stream) != hipSuccess)
        return bail(fail(ctx, HETEGEN_ERR_HIP, "hipEventRecord failed"));
    }
    try {
      ctx->mgr = std::thread(manager_main, ctx);
    } catch (...) {
      return bail(fail(ctx, HETEGEN_ERR_OOM, "parameter manager thread"));
    }
    *out = ctx;
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_destroy(hetegen_ctx* ctx) {
  return api_guard(nullptr, [&]() -> hetegen_status {  // ctx is gone by the end
    if (!ctx) return HETEGEN_OK;
    if (ctx->mgr.joinable()) {
      {
        std::lock_guard<std::mutex> lk(ctx->mu);
        ctx->stop = true;
      }
      ctx->cv.notify_all();
      ctx->mgr.join();
    }
    hg::team_streamed_chunks(-(long long)ctx->jobs.size());  // chunks a failed call left queued
    ctx->jobs.clear();
    ctx->team.shutdown();
    (void)hipSetDevice(ctx->device);
    (void)hipDeviceSynchronize();
    for (size_t i = 0; i < ctx->bounce.size(); ++i) {
      if (ctx->bounce[i]) (void)hipHostFree(ctx->bounce[i]);
      if (ctx->ev_bounce[i]) (void)hipEventDestroy(ctx->ev_bounce[i]);
    }
    for (auto& t : ctx->timed) {
      (void)hipEventDestroy(t.a);
      (void)hipEventDestroy(t.b);
    }
    for (auto e : ctx->ev_pool) (void)hipEventDestroy(e);
    for (size_t i = 0; i < ctx->slot.size(); ++i) {
      if (ctx->slot[i]) (void)hipFree(ctx->slot[i]);
      if (ctx->ev_ready[i]) (void)hipEventDestroy(ctx->ev_ready[i]);
      if (ctx->ev_free[i]) (void)hipEventDestroy(ctx->ev_free[i]);
    }
    if (ctx->ev_x) (void)hipEventDestroy(ctx->ev_x);
    if (ctx->ev_y) (void)hipEventDestroy(ctx->ev_y);
    if (ctx->x_host) (void)hipHostFree(ctx->x_host);
    if (ctx->y_host) (void)hipHostFree(ctx->y_host);
    if (ctx->ws) (void)hipFree(ctx->ws);
    if (ctx->ws_cnt) (void)hipFree(ctx->ws_cnt);
    if (ctx->copy_stream) (void)hipStreamDestroy(ctx->copy_stream);
    if (ctx->capture_stream) (void)hipStreamDestroy(ctx->capture_stream);
    (void)hipGetLastError();
    delete ctx;
    return HETEGEN_OK;
  });
}

const char* hetegen_last_error(const hetegen_ctx* ctx) { return ctx ? ctx->err.c_str() : g_create_error.c_str(); }

const char* hetegen_cpu_share_isa(void) { return hg::cpu_share_isa(); }

hetegen_status hetegen_host_alloc(hetegen_ctx* ctx, size_t bytes, void** p) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx || !p || bytes == 0) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_host_alloc: bad arguments");
    *p = nullptr;
    HIPCHK(ctx, hipSetDevice(ctx->device));
    if (host_malloc(ctx, p, bytes, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      *p = nullptr;
      return fail(ctx, HETEGEN_ERR_OOM, "pinned allocation of %zu bytes failed", bytes);
    }
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_host_free(hetegen_ctx* ctx, void* p) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "ctx is NULL");
    if (!p) return HETEGEN_OK;
    HIPCHK(ctx, hipHostFree(p));
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_linear(hetegen_ctx* ctx, const void* x_dev, int B, int K, const void* W_host,
                              const void* W_dev_resident, int N, hetegen_dtype w_dtype, const void* bias_host,
                              const void* bias_dev, double alpha, void* y_dev, hetegen_dtype y_dtype, void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    auto t0 = Clock::now();
    ctx->err.clear();
    if (!x_dev || !W_host || !y_dev) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "x_dev, W_host and y_dev are required");
    if (!(alpha >= 0.0 && alpha <= 1.0)) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "alpha %g outside [0, 1]", alpha);
    if (N < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "N = %d", N);
    if (B < 1 || B > kMaxBatch) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B = %d outside [1, %d]", B, kMaxBatch);
    if (K < 8 || K % 8) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "K = %d must be a positive multiple of 8", K);
    if (w_dtype != HETEGEN_F16 && w_dtype != HETEGEN_BF16)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "weight dtype %d: fp16 or bf16 only", (int)w_dtype);
    if (y_dtype != w_dtype && y_dtype != HETEGEN_F32)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "y dtype must be the weight dtype or fp32");
    if (!aligned16(x_dev) || !aligned16(W_host) || (W_dev_resident && !aligned16(W_dev_resident)))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "x, W and the resident copy must be 16-byte aligned");
    const int n_cpu = split_cpu_rows(N, alpha), n_gpu = N - n_cpu;
    if ((n_cpu > 0 && !bias_host && bias_dev) || (n_gpu > 0 && !bias_dev && bias_host))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "bias: pass bias_host and bias_dev, or neither");
    bool pageable = false;
    // W_host is read by the CPU share and by the streamed chunks; a call with every row
    // resident on the GPU does not touch it
    if (n_cpu > 0 || !W_dev_resident) TRY(check_weight(ctx, W_host, (size_t)N * K * 2, &pageable));
    const size_t row = (size_t)K * 2;
    if (!W_dev_resident && n_gpu > 0 && row > ctx->chunk_bytes)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "a weight row (%zu bytes) exceeds chunk_bytes", row);
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hipStream_t st = (hipStream_t)stream;
    Job j{};
    j.x = x_dev;
    j.ldx = K;
    j.B = B;
    j.K = K;
    j.N = N;
    j.dtype = w_dtype;
    j.W_host = W_host;
    j.W_dev = W_dev_resident;
    j.bias_host = bias_host;
    j.bias_dev = bias_dev;
    j.n_gpu = n_gpu;
    j.n_cpu = n_cpu;
    j.y = y_dev;
    j.ldy = N;
    j.y_f32 = y_dtype == HETEGEN_F32;
    j.epi = hg::EPI_NONE;
    if (!W_dev_resident && n_gpu > 0) {
      if (!pipeline_idle(ctx)) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "internal: stale chunk plan");
      if (pageable) TRY(ensure_pin_resources(ctx));
      plan_chunks(ctx, W_host, n_gpu, K, w_dtype, pageable, n_cpu == 0);
    }
    hetegen_status stt = run_linear(ctx, j, st);
    if (stt != HETEGEN_OK) {
      reset_pipeline(ctx);
      return stt;
    }
    return finish_call(ctx, t0);
  });
}

// ---- resident weights in matrix-core tile order ----
size_t hetegen_tiled_bytes(int rows, int K) {
  if (rows < 1 || K < 8 || K % 8) return 0;
  return hg::tiled_bytes(rows, K);
}

hetegen_status hetegen_tile_weights(hetegen_ctx* ctx, const void* W_dev, int rows, int K, void* W_tiled_dev,
                                    void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!W_dev || !W_tiled_dev || rows < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_tile_weights: bad arguments");
    if (K < 8 || K % 8) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "K = %d must be a positive multiple of 8", K);
    if (!aligned16(W_dev) || !aligned16(W_tiled_dev))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "W and its tiled copy must be 16-byte aligned");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    HIPCHK(ctx, hg::launch_tile(W_dev, K, rows, K, W_tiled_dev, (hipStream_t)stream));
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_linear_tiled(hetegen_ctx* ctx, const void* x_dev, int B, int K, const void* W_tiled_dev, int N,
                                    hetegen_dtype w_dtype, const void* bias_dev, void* y_dev, hetegen_dtype y_dtype,
                                    void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    auto t0 = Clock::now();
    ctx->err.clear();
    if (!x_dev || !W_tiled_dev || !y_dev) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "x_dev, W_tiled_dev and y_dev are required");
    if (N < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "N = %d", N);
    if (B < 1 || B > kMaxBatch) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B = %d outside [1, %d]", B, kMaxBatch);
    if (K < 8 || K % 8) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "K = %d must be a positive multiple of 8", K);
    if ((long long)B * K >= (1LL << 30))  // x is read through a buffer descriptor (32-bit offsets)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B * K = %lld: x must hold fewer than 2^30 elements", (long long)B * K);
    if (w_dtype != HETEGEN_F16 && w_dtype != HETEGEN_BF16)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "weight dtype %d: fp16 or bf16 only", (int)w_dtype);
    if (y_dtype != w_dtype && y_dtype != HETEGEN_F32)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "y dtype must be the weight dtype or fp32");
    if (!aligned16(x_dev) || !aligned16(W_tiled_dev))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "x and the tiled weight must be 16-byte aligned");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hipStream_t st = (hipStream_t)stream;
    // split-K workspace, sized for the largest batch so that batch changes do not regrow it
    const size_t need = hg::mfma_ws_floats(N, K, kMaxBatch), words = hg::mfma_cnt_words(N, K);
    if (need > ctx->ws_floats || words > ctx->ws_words) {
      HIPCHK(ctx, hipDeviceSynchronize());  // earlier launches may still use the old buffers
      if (ctx->ws) (void)hipFree(ctx->ws);
      if (ctx->ws_cnt) (void)hipFree(ctx->ws_cnt);
      ctx->ws = nullptr;
      ctx->ws_cnt = nullptr;
      ctx->ws_floats = ctx->ws_words = 0;
      const size_t nf = std::max(need, (size_t)1), nw = std::max(words, (size_t)1);
      if (hipMalloc((void**)&ctx->ws, nf * 4) != hipSuccess || hipMalloc((void**)&ctx->ws_cnt, nw * 4) != hipSuccess) {
        (void)hipGetLastError();
        return fail(ctx, HETEGEN_ERR_OOM, "split-K workspace of %zu floats", nf);
      }
      HIPCHK(ctx, hipMemset(ctx->ws_cnt, 0, nw * 4));
      ctx->ws_floats = nf;
      ctx->ws_words = nw;
    }
    hg::GemvParams p{};
    p.x = x_dev;
    p.ldx = K;
    p.W = W_tiled_dev;
    p.bias = bias_dev;
    p.y = y_dev;
    p.ldy = N;
    p.rows = N;
    p.K = K;
    p.epi = hg::EPI_NONE;
    p.y_f32 = y_dtype == HETEGEN_F32;
    p.ws = ctx->ws;
    p.cnt = ctx->ws_cnt;
    p.ws_floats = ctx->ws_floats;
    p.cnt_words = ctx->ws_words;
    TimedScope ts(ctx, st, 1, (double)N * K * 2);
    HIPCHK(ctx, hg::launch_gemv_mfma(p, w_dtype, B, st));
    ts.end();
    return finish_call(ctx, t0);
  });
}

hetegen_status hetegen_linear_tiled_noalloc(hetegen_ctx* ctx, const void* x_dev, int B, int K,
                                            const void* W_tiled_dev, int N, hetegen_dtype w_dtype,
                                            const void* bias_dev, void* y_dev, hetegen_dtype y_dtype, void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!x_dev || !W_tiled_dev || !y_dev) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "x_dev, W_tiled_dev and y_dev are required");
    if (N < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "N = %d", N);
    if (B < 1 || B > kMaxBatch) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B = %d outside [1, %d]", B, kMaxBatch);
    if (K < 8 || K % 8) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "K = %d must be a positive multiple of 8", K);
    if ((long long)B * K >= (1LL << 30))  // x is read through a buffer descriptor (32-bit offsets)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B * K = %lld: x must hold fewer than 2^30 elements", (long long)B * K);
    if (w_dtype != HETEGEN_F16 && w_dtype != HETEGEN_BF16)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "weight dtype %d: fp16 or bf16 only", (int)w_dtype);
    if (y_dtype != w_dtype && y_dtype != HETEGEN_F32)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "y dtype must be the weight dtype or fp32");
    if (!aligned16(x_dev) || !aligned16(W_tiled_dev))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "x and the tiled weight must be 16-byte aligned");
    const size_t need = hg::mfma_ws_floats(N, K, B), words = hg::mfma_cnt_words(N, K);
    if (need > hg::kScratchFloats || words > hg::kScratchCounterWords)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED,
                  "[%d, %d] at batch %d needs %zu partial floats and %zu counters of split-K scratch; the fixed "
                  "scratch holds %zu and %zu (use hetegen_linear_tiled)",
                  N, K, B, need, words, hg::kScratchFloats, hg::kScratchCounterWords);
    HIPCHK(ctx, hipSetDevice(ctx->device));
    uint32_t* base = (uint32_t*)hg::scratch_ptr(ctx->device);
    if (!base) return fail(ctx, HETEGEN_ERR_HIP, "the fixed scratch of device %d is not set up", ctx->device);
    hg::GemvParams p{};
    p.x = x_dev;
    p.ldx = K;
    p.W = W_tiled_dev;
    p.bias = bias_dev;
    p.y = y_dev;
    p.ldy = N;
    p.rows = N;
    p.K = K;
    p.epi = hg::EPI_NONE;
    p.y_f32 = y_dtype == HETEGEN_F32;
    p.cnt = base;
    p.ws = (float*)(base + hg::kScratchCounterWords);
    p.cnt_words = hg::kScratchCounterWords;
    p.ws_floats = hg::kScratchFloats;
    HIPCHK(ctx, hg::launch_gemv_mfma(p, w_dtype, B, (hipStream_t)stream));
    return HETEGEN_OK;
  });
}

// ---- planner (pure host arithmetic) ----
hetegen_status hetegen_layer_plan(const hetegen_shape* shapes, int n, const hetegen_bw* bw, int n_bw, int flags,
                                  double* alpha_out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!shapes || !bw || !alpha_out || n < 0 || !(n_bw == 1 || n_bw == n)) return HETEGEN_ERR_INVALID_ARG;
    for (int i = 0; i < n; ++i) {
      const hetegen_bw& b = bw[n_bw == 1 ? 0 : i];
      if (shapes[i].N < 1 || shapes[i].K < 1) return HETEGEN_ERR_INVALID_ARG;
      if (shapes[i].resident) {
        alpha_out[i] = 0.0;
        continue;
      }
      const double vc = b.cpu_Bps, vg = b.hbm_gemv_Bps;
      double vm = b.h2d_Bps;
      if (!(vc > 0 && std::isfinite(vc) && vg > 0 && std::isfinite(vg) && vm > 0 && std::isfinite(vm)))
        return HETEGEN_ERR_INVALID_ARG;
      if (b.pin_Bps > 0) {
        if (!std::isfinite(b.pin_Bps)) return HETEGEN_ERR_INVALID_ARG;
        vm = std::min(vm, b.pin_Bps);  // T_COM = max(T_PIN, T_TRANS)
      }
      // CPU fraction = 1 - alpha_gpu; written as the balance of per-byte times so that
      // large speed ratios do not overflow: (1/Vcom + 1/Vgpu) / (1/Vcpu + 1/Vcom + 1/Vgpu).
      double c;
      if (flags & HETEGEN_PLAN_APPROX) c = (1.0 / vm) / (1.0 / vc + 1.0 / vm);
      else c = (1.0 / vm + 1.0 / vg) / (1.0 / vc + 1.0 / vm + 1.0 / vg);
      alpha_out[i] = std::min(1.0, std::max(0.0, c));
    }
    return HETEGEN_OK;
  });
}

}  // extern "C"

// ---- alpha benchmark: least-squares polynomial fit and crossing ----
namespace {

// Coefficients c[0..d] of sum_j c[j] s^j fitted to (s_i, t_i), normal equations with
// partial pivoting; s is the centred and scaled ratio, so the system stays well
// conditioned.
bool lsq_poly(const std::vector<double>& s, const double* t, int d, double* c) {
  double A[4][5] = {};
  for (size_t i = 0; i < s.size(); ++i) {
    double p[7];
    p[0] = 1.0;
    for (int j = 1; j <= 2 * d; ++j) p[j] = p[j - 1] * s[i];
    for (int r = 0; r <= d; ++r) {
      for (int q = 0; q <= d; ++q) A[r][q] += p[r + q];
      A[r][d + 1] += p[r] * t[i];
    }
  }
  for (int col = 0; col <= d; ++col) {
    int piv = col;
    for (int r = col + 1; r <= d; ++r)
      if (fabs(A[r][col]) > fabs(A[piv][col])) piv = r;
    if (fabs(A[piv][col]) < 1e-300) return false;
    if (piv != col)
      for (int q = 0; q <= d + 1; ++q) std::swap(A[piv][q], A[col][q]);
    for (int r = 0; r <= d; ++r) {
      if (r == col) continue;
      const double f = A[r][col] / A[col][col];
      for (int q = col; q <= d + 1; ++q) A[r][q] -= f * A[col][q];
    }
  }
  for (int r = 0; r <= d; ++r) c[r] = A[r][d + 1] / A[r][r];
  return true;
}

double poly(const double* c, int d, double s) {
  double v = c[d];
  for (int j = d - 1; j >= 0; --j) v = v * s + c[j];
  return v;
}

}  // namespace

extern "C" hetegen_status hetegen_alpha_fit(const double* alphas, const double* t_cpu, const double* t_com, int n,
                                            int degree, double lo, double hi, double* alpha_out, int* crossed) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!alphas || !t_cpu || !t_com || !alpha_out || degree < 1 || degree > 3 || n < degree + 1 || !(lo < hi))
      return HETEGEN_ERR_INVALID_ARG;
    double amin = alphas[0], amax = alphas[0];
    for (int i = 0; i < n; ++i) {
      if (!std::isfinite(alphas[i]) || !std::isfinite(t_cpu[i]) || !std::isfinite(t_com[i]))
        return HETEGEN_ERR_INVALID_ARG;
      amin = std::min(amin, alphas[i]);
      amax = std::max(amax, alphas[i]);
    }
    const double ctr = 0.5 * (amin + amax), half = amax > amin ? 0.5 * (amax - amin) : 1.0;
    std::vector<double> sv(n);
    for (int i = 0; i < n; ++i) sv[i] = (alphas[i] - ctr) / half;
    double cc[4], cg[4];
    if (!lsq_poly(sv, t_cpu, degree, cc) || !lsq_poly(sv, t_com, degree, cg)) return HETEGEN_ERR_INVALID_ARG;
    auto fc = [&](double a) { return poly(cc, degree, (a - ctr) / half); };
    auto fg = [&](double a) { return poly(cg, degree, (a - ctr) / half); };
    auto g = [&](double a) { return fc(a) - fg(a); };
    // sign changes of F_CPU - F_COM on a fine grid, each refined by bisection
    const int M = 2000;
    double best = 0, best_t = INFINITY;
    bool found = false;
    double a0 = lo, g0 = g(lo);
    for (int i = 1; i <= M; ++i) {
      const double a1 = lo + (hi - lo) * i / M, g1 = g(a1);
      if (g0 == 0 || (g0 < 0) != (g1 < 0)) {
        double l = a0, r = a1, gl = g0;
        if (g0 == 0) r = a0;
        for (int it = 0; it < 200 && r - l > 0; ++it) {
          const double mid = 0.5 * (l + r), gm = g(mid);
          if (mid <= l || mid >= r) break;
          if ((gm < 0) == (gl < 0)) {
            l = mid;
            gl = gm;
          } else {
            r = mid;
          }
        }
        const double root = 0.5 * (l + r);
        if (fc(root) < best_t) {
          best_t = fc(root);
          best = root;
          found = true;
        }
      }
      a0 = a1;
      g0 = g1;
    }
    if (!found) {  // no crossing: bracket point with the smallest max(F_CPU, F_COM)
      const int G = 10000;
      for (int i = 0; i <= G; ++i) {
        const double a = lo + (hi - lo) * i / G, m = std::max(fc(a), fg(a));
        if (m < best_t) {
          best_t = m;
          best = a;
        }
      }
    }
    *alpha_out = std::min(hi, std::max(lo, best));
    if (crossed) *crossed = found ? 1 : 0;
    return HETEGEN_OK;
  });
}

extern "C" hetegen_status hetegen_alpha_minimize(const double* alphas, const double* t, int n, int degree, double lo,
                                                 double hi, double* alpha_out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!alphas || !t || !alpha_out || degree < 1 || degree > 3 || n < degree + 1 || !(lo < hi))
      return HETEGEN_ERR_INVALID_ARG;
    double amin = alphas[0], amax = alphas[0];
    for (int i = 0; i < n; ++i) {
      if (!std::isfinite(alphas[i]) || !std::isfinite(t[i])) return HETEGEN_ERR_INVALID_ARG;
      amin = std::min(amin, alphas[i]);
      amax = std::max(amax, alphas[i]);
    }
    const double ctr = 0.5 * (amin + amax), half = amax > amin ? 0.5 * (amax - amin) : 1.0;
    std::vector<double> sv(n);
    for (int i = 0; i < n; ++i) sv[i] = (alphas[i] - ctr) / half;
    double c[4];
    if (!lsq_poly(sv, t, degree, c)) return HETEGEN_ERR_INVALID_ARG;
    const int G = 10000;
    double best = lo, best_t = INFINITY;
    for (int i = 0; i <= G; ++i) {
      const double a = lo + (hi - lo) * i / G, v = poly(c, degree, (a - ctr) / half);
      if (v < best_t) {
        best_t = v;
        best = a;
      }
    }
    *alpha_out = best;
    return HETEGEN_OK;
  });
}

extern "C" hetegen_status hetegen_alpha_benchmark(hetegen_ctx* ctx, const void* x_dev, int B, int K,
                                                  const void* W_host, int N, hetegen_dtype dtype,
                                                  const void* bias_host, const void* bias_dev, void* y_dev,
                                                  double alpha0, double gamma, double lambda, int degree, int reps,
                                                  void* stream, double* alpha_out, int* crossed) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    if (!alpha_out || !(gamma >= 0) || !(lambda > 0) || reps < 1 || !(alpha0 >= 0 && alpha0 <= 1) || degree < 1 ||
        degree > 3)
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_alpha_benchmark: bad arguments");
    const double lo = std::max(0.0, alpha0 - gamma), hi = std::min(1.0, alpha0 + gamma);
    std::vector<double> as, tc, tg;
    for (int i = 0;; ++i) {
      const double a = lo + i * lambda;
      if (a > hi + 1e-9) break;
      as.push_back(std::min(a, hi));
    }
    if ((int)as.size() < degree + 1 || !(lo < hi))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "bracket holds %zu points; degree %d needs %d", as.size(), degree,
                  degree + 1);
    const bool was = ctx->profiling;
    ctx->profiling = true;
    TRY(flush_profile(ctx));
    const hetegen_profile saved = ctx->prof;
    hetegen_status st = HETEGEN_OK;
    for (double a : as) {
      std::vector<double> c, g;
      for (int r = 0; r <= reps && st == HETEGEN_OK; ++r) {
        ctx->prof = hetegen_profile{};
        st = hetegen_linear(ctx, x_dev, B, K, W_host, nullptr, N, dtype, bias_host, bias_dev, a, y_dev, HETEGEN_F32,
                            stream);
        if (st == HETEGEN_OK && r > 0) {  // the first run of each point warms it up
          c.push_back(ctx->prof.cpu_ms);
          g.push_back(ctx->prof.h2d_ms + ctx->prof.gpu_ms);
        }
      }
      if (st != HETEGEN_OK) break;
      std::sort(c.begin(), c.end());
      std::sort(g.begin(), g.end());
      tc.push_back(c[c.size() / 2]);
      tg.push_back(g[g.size() / 2]);
    }
    ctx->prof = saved;
    ctx->profiling = was;
    if (st != HETEGEN_OK) return st;
    hetegen_status fs = hetegen_alpha_fit(as.data(), tc.data(), tg.data(), (int)as.size(), degree, lo, hi, alpha_out,
                                          crossed);
    if (fs != HETEGEN_OK) return fail(ctx, fs, "alpha fit failed");
    return HETEGEN_OK;
  });
}

extern "C" hetegen_status hetegen_cpu_linear(const float* x, int B, int K, const void* W_host, hetegen_dtype dtype,
                                             const void* bias_host, int r0, int r1, float* y, int ldy, int threads) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!x || !W_host || !y || B < 1 || B > kMaxBatch || K < 8 || K % 8 || r0 < 0 || r1 < r0 || ldy < r1 - r0 ||
        (dtype != HETEGEN_F16 && dtype != HETEGEN_BF16))
      return HETEGEN_ERR_INVALID_ARG;
    hg::cpu_share(x, B, K, (const uint16_t*)W_host, dtype, (const uint16_t*)bias_host, r0, r1, y, ldy, threads);
    return HETEGEN_OK;
  });
}

// ---- heterogeneous module scheduler (Sec. 4.5, Eq. 13) ----
extern "C" hetegen_status hetegen_module_schedule(const double* t_cpu, const double* mem, const int* layer, int n,
                                                  double budget_bytes, int* resident_out, double* used_out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (n < 0 || (n > 0 && (!t_cpu || !mem || !layer || !resident_out)) || !(budget_bytes >= 0))
      return HETEGEN_ERR_INVALID_ARG;
    std::vector<double> g(n);
    std::map<int, std::vector<int>> by_layer;  // layers in increasing order
    for (int i = 0; i < n; ++i) {
      if (!std::isfinite(t_cpu[i]) || t_cpu[i] < 0 || !std::isfinite(mem[i]) || !(mem[i] > 0) || layer[i] < 0)
        return HETEGEN_ERR_INVALID_ARG;
      g[i] = t_cpu[i] / mem[i];
      by_layer[layer[i]].push_back(i);
    }
    // modules of each layer by decreasing gain (stable: index order among equal gains)
    size_t depth = 0;
    for (auto& kv : by_layer) {
      std::stable_sort(kv.second.begin(), kv.second.end(), [&](int a, int b) { return g[a] > g[b]; });
      depth = std::max(depth, kv.second.size());
    }
    double used = 0.0;
    for (int i = 0; i < n; ++i) resident_out[i] = 0;
    for (size_t r = 0; r < depth; ++r) {
      for (const auto& kv : by_layer) {
        const auto& v = kv.second;
        if (r >= v.size()) continue;
        const int i = v[r];
        if (used + mem[i] <= budget_bytes) {
          resident_out[i] = 1;
          used += mem[i];
        }
      }
    }
    if (used_out) *used_out = used;
    return HETEGEN_OK;
  });
}

extern "C" {

hetegen_status hetegen_set_profiling(hetegen_ctx* ctx, int on) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->profiling = on != 0;
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_get_profile(hetegen_ctx* ctx, hetegen_profile* out, int reset) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx || !out) return HETEGEN_ERR_INVALID_ARG;
    TRY(flush_profile(ctx));
    *out = ctx->prof;
    if (reset) ctx->prof = hetegen_profile{};
    return HETEGEN_OK;
  });
}

}  // extern "C"

// ---- bandwidth probe ----
extern "C" hetegen_status hetegen_probe(hetegen_ctx* ctx, const void* W_host, int N, int K, hetegen_dtype dtype, int B,
                                        int reps, int flags, hetegen_bw* out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx || !W_host || !out || N < 1 || K < 8 || K % 8 || B < 1 || B > kMaxBatch || reps < 1 ||
        (dtype != HETEGEN_F16 && dtype != HETEGEN_BF16))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_probe: bad arguments");
    bool pageable = false;
    TRY(check_weight(ctx, W_host, (size_t)N * K * 2, &pageable));
    HIPCHK(ctx, hipSetDevice(ctx->device));
    if (!pipeline_idle(ctx)) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "internal: stale chunk plan");
    HIPCHK(ctx, hipDeviceSynchronize());  // earlier GEMVs may still read the staging slots
    if (pageable) TRY(ensure_pin_resources(ctx));
    const size_t wbytes = (size_t)N * K * 2;
    auto median = [](std::vector<double> v) {
      std::sort(v.begin(), v.end());
      return v[v.size() / 2];
    };
    // V_CPU: the CPU share over all rows
    if (ctx->y_pending) HIPCHK(ctx, hipEventSynchronize(ctx->ev_y));
    ctx->y_pending = false;
    TRY(ensure_host(ctx, &ctx->x_host, &ctx->x_host_bytes, (size_t)B * K * 4));
    TRY(ensure_host(ctx, &ctx->y_host, &ctx->y_host_bytes, (size_t)B * N * 4));
    memset(ctx->x_host, 0, (size_t)B * K * 4);
    // In a step every weight comes from DRAM (a step's weights dwarf the host caches);
    // a single linear re-read by the probe can sit in a large L3, so the caches are
    // flushed before every pass by reading a 1 GiB buffer (reading, not writing: dirty
    // lines written back during the timed pass would slow it).
    std::vector<uint64_t> flush;
    try {
      flush.assign(((size_t)1 << 30) / sizeof(uint64_t), 1);
    } catch (...) {
      return fail(ctx, HETEGEN_ERR_OOM, "probe cache-flush buffer");
    }
    uint64_t flush_sink = 0;
    // read on the CPU share's own worker team (a second team would still be spinning
    // when the timed pass starts)
    struct Flush {
      const uint64_t* p;
      long long n;
      uint64_t part[64];
    } fl{flush.data(), (long long)flush.size(), {}};
    enum { kFlushGrains = 64 };
    auto flush_caches = [&](int) {
      hg::team_for(ctx->cpu_threads, kFlushGrains, [](void* a, int g) {
        Flush& f = *(Flush*)a;
        const long long per = (f.n / kFlushGrains + 7) & ~7LL;
        const long long b = per * g, e = std::min(f.n, b + per);
        uint64_t acc = 0;
        for (long long i = b; i < e; i += 8) acc ^= f.p[i];  // one word per 64-byte line
        f.part[g] = acc;
      }, &fl);
      for (int g = 0; g < kFlushGrains; ++g) flush_sink ^= fl.part[g];
    };
    std::vector<double> tc;
    for (int r = -1; r < reps; ++r) {  // one untimed pass first: threads up, TLBs warm
      flush_caches(r & 0xff);
      auto t0 = Clock::now();
      hg::cpu_share(ctx->x_host, B, K, (const uint16_t*)W_host, dtype, nullptr, 0, N, ctx->y_host, N, ctx->cpu_threads);
      if (r >= 0) tc.push_back(ms_since(t0) * 1e-3);
    }
    // V_PIN (pageable weights): the pin team staging W_host chunk by chunk
    const size_t row = (size_t)K * 2;
    const size_t cbytes = (size_t)chunk_rows_for(ctx, K, dtype) * row;
    std::vector<double> tp;
    for (int r = 0; pageable && r < reps; ++r) {
      HIPCHK(ctx, hipStreamSynchronize(ctx->copy_stream));  // no copy reads the staging buffers
      flush_caches(r & 0xff);
      auto t0 = Clock::now();
      int i = 0;
      for (size_t off = 0; off < wbytes; off += cbytes, ++i)
        ctx->team.copy((char*)ctx->bounce[i % ctx->pin_ring], (const char*)W_host + off,
                       std::min(cbytes, wbytes - off));
      tp.push_back(ms_since(t0) * 1e-3);
    }
    // V_COM: chunked copies through the ring on the copy stream, from W_host or (pageable)
    // from the pinned staging buffers
    hipEvent_t a, b;
    HIPCHK(ctx, hipEventCreate(&a));
    HIPCHK(ctx, hipEventCreate(&b));
    std::vector<double> tm;
    for (int r = 0; r < reps; ++r) {
      HIPCHK(ctx, hipEventRecord(a, ctx->copy_stream));
      int i = 0;
      for (size_t off = 0; off < wbytes; off += cbytes, ++i) {
        const size_t nb = std::min(cbytes, wbytes - off);
        const void* src = pageable ? ctx->bounce[i % ctx->pin_ring] : (const char*)W_host + off;
        HIPCHK(ctx, hipMemcpyAsync(ctx->slot[i % ctx->ring], src, nb, hipMemcpyHostToDevice, ctx->copy_stream));
      }
      HIPCHK(ctx, hipEventRecord(b, ctx->copy_stream));
      HIPCHK(ctx, hipEventSynchronize(b));
      float ms = 0;
      HIPCHK(ctx, hipEventElapsedTime(&ms, a, b));
      tm.push_back(ms * 1e-3);
    }
    // concurrent rates: the copies of W once, the CPU share over W back to back until they end
    std::vector<double> cc, cm;
    for (int r = 0; (flags & HETEGEN_PROBE_CONCURRENT) && !pageable && r < reps; ++r) {
      flush_caches(r & 0xff);
      HIPCHK(ctx, hipEventRecord(a, ctx->copy_stream));
      for (size_t off = 0, i = 0; off < wbytes; off += cbytes, ++i)
        HIPCHK(ctx, hipMemcpyAsync(ctx->slot[i % ctx->ring], (const char*)W_host + off, std::min(cbytes, wbytes - off),
                                   hipMemcpyHostToDevice, ctx->copy_stream));
      HIPCHK(ctx, hipEventRecord(b, ctx->copy_stream));
      double t_sum = 0;  // CPU passes that ended before the copies did (each on cold caches)
      int n_done = 0;
      for (int pass = 0;; ++pass) {
        if (pass > 0) flush_caches((r + pass) & 0xff);
        const auto t0 = Clock::now();
        hg::cpu_share(ctx->x_host, B, K, (const uint16_t*)W_host, dtype, nullptr, 0, N, ctx->y_host, N,
                      ctx->cpu_threads);
        const double t = ms_since(t0) * 1e-3;
        const hipError_t q = hipEventQuery(b);
        if (q == hipErrorNotReady) {
          (void)hipGetLastError();
          t_sum += t;
          ++n_done;
          continue;
        }
        HIPCHK(ctx, q);
        if (n_done == 0) {  // the copies ended within the first pass: count that pass
          t_sum = t;
          n_done = 1;
        }
        break;
      }
      float ms = 0;
      HIPCHK(ctx, hipEventElapsedTime(&ms, a, b));
      cc.push_back(t_sum / n_done);
      cm.push_back(ms * 1e-3);
    }
    // V_GPU: the GEMV over a device copy of W
    void *Wd = nullptr, *xd = nullptr, *yd = nullptr;
    hetegen_status st = HETEGEN_OK;
    std::vector<double> tg;
    if (hipMalloc(&Wd, wbytes) != hipSuccess || hipMalloc(&xd, (size_t)B * K * 2) != hipSuccess ||
        hipMalloc(&yd, (size_t)B * N * 4) != hipSuccess) {
      (void)hipGetLastError();
      st = fail(ctx, HETEGEN_ERR_OOM, "probe buffers");
    }
    if (st == HETEGEN_OK && (hipMemcpy(Wd, W_host, wbytes, hipMemcpyHostToDevice) != hipSuccess ||
                             hipMemset(xd, 0, (size_t)B * K * 2) != hipSuccess))
      st = fail(ctx, HETEGEN_ERR_HIP, "probe upload failed");
    for (int r = 0; st == HETEGEN_OK && r < reps + 1; ++r) {
      hg::GemvParams p{};
      p.x = xd;
      p.ldx = K;
      p.W = Wd;
      p.y = yd;
      p.ldy = N;
      p.rows = N;
      p.K = K;
      p.y_f32 = 1;
      if (hipEventRecord(a, ctx->capture_stream) != hipSuccess ||
          hg::launch_gemv(p, dtype, B, ctx->capture_stream, 0) != hipSuccess ||
          hipEventRecord(b, ctx->capture_stream) != hipSuccess || hipEventSynchronize(b) != hipSuccess) {
        st = fail(ctx, HETEGEN_ERR_HIP, "probe GEMV failed");
        break;
      }
      float ms = 0;
      (void)hipEventElapsedTime(&ms, a, b);
      if (r > 0) tg.push_back(ms * 1e-3);
    }
    if (Wd) (void)hipFree(Wd);
    if (xd) (void)hipFree(xd);
    if (yd) (void)hipFree(yd);
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    (void)hipGetLastError();
    if (st != HETEGEN_OK) return st;
    if (flush_sink == 0x5a5a5a5a5a5a5a5aull) ctx->err = "";  // keeps the flush reads
    out->cpu_Bps = wbytes / median(cc.empty() ? tc : cc);
    out->h2d_Bps = wbytes / median(cm.empty() ? tm : cm);
    out->hbm_gemv_Bps = wbytes / median(tg);
    out->pin_Bps = pageable ? wbytes / median(tp) : 0;
    return HETEGEN_OK;
  });
}

// ---- launch round trip ----
extern "C" hetegen_status hetegen_probe_launch(hetegen_ctx* ctx, int reps, void* stream, double* us_out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!us_out || reps < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_probe_launch: bad arguments");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hipStream_t st = (hipStream_t)stream;
    HIPCHK(ctx, hipStreamSynchronize(st));
    std::vector<double> t;
    for (int r = 0; r < reps + 10; ++r) {
      const auto t0 = Clock::now();
      HIPCHK(ctx, hg::launch_empty(st));
      HIPCHK(ctx, hipStreamSynchronize(st));
      if (r >= 10) t.push_back(ms_since(t0) * 1e3);
    }
    std::sort(t.begin(), t.end());
    *us_out = t[t.size() / 2];
    return HETEGEN_OK;
  });
}

// ---- idle host-to-device link rate ----
extern "C" hetegen_status hetegen_probe_link(hetegen_ctx* ctx, size_t bytes, int reps, double* Bps_out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!Bps_out || reps < 1 || bytes < ((size_t)1 << 20) || (bytes & 15))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_probe_link: bad arguments");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    void* dev = nullptr;
    void* host = nullptr;
    if (host_malloc(ctx, &host, bytes, hipHostMallocDefault) != hipSuccess || hipMalloc(&dev, bytes) != hipSuccess) {
      (void)hipGetLastError();
      if (host) (void)hipHostFree(host);
      if (dev) (void)hipFree(dev);
      return fail(ctx, HETEGEN_ERR_OOM, "link probe buffers of %zu bytes", bytes);
    }
    memset(host, 0x11, bytes);  // touch every page before timing
    hipEvent_t a = nullptr, b = nullptr;
    hetegen_status st = HETEGEN_OK;
    std::vector<double> t;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess)
      st = fail(ctx, HETEGEN_ERR_HIP, "link probe events");
    for (int r = 0; st == HETEGEN_OK && r <= reps; ++r) {  // the first copy warms up
      float ms = 0;
      if (hipEventRecord(a, ctx->copy_stream) != hipSuccess ||
          hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, ctx->copy_stream) != hipSuccess ||
          hipEventRecord(b, ctx->copy_stream) != hipSuccess || hipEventSynchronize(b) != hipSuccess ||
          hipEventElapsedTime(&ms, a, b) != hipSuccess) {
        st = fail(ctx, HETEGEN_ERR_HIP, "link probe copy failed");
        break;
      }
      if (r > 0) t.push_back(ms * 1e-3);
    }
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    (void)hipHostFree(host);
    (void)hipFree(dev);
    (void)hipGetLastError();
    if (st != HETEGEN_OK) return st;
    std::sort(t.begin(), t.end());
    *Bps_out = (double)bytes / t[t.size() / 2];
    return HETEGEN_OK;
  });
}

// ---- achievable HBM read bandwidth ----
extern "C" hetegen_status hetegen_probe_hbm(hetegen_ctx* ctx, size_t bytes, int reps, double* Bps_out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!Bps_out || reps < 1 || bytes < ((size_t)1 << 20) || (bytes & 15))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_probe_hbm: bad arguments");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    void* buf = nullptr;
    uint32_t* sink = nullptr;
    if (hipMalloc(&buf, bytes) != hipSuccess || hipMalloc((void**)&sink, 256) != hipSuccess) {
      (void)hipGetLastError();
      if (buf) (void)hipFree(buf);
      return fail(ctx, HETEGEN_ERR_OOM, "probe buffer of %zu bytes", bytes);
    }
    hipEvent_t a = nullptr, b = nullptr;
    hetegen_status st = HETEGEN_OK;
    std::vector<double> t;
    int ncu = 0;
    if (hipMemset(buf, 0x11, bytes) != hipSuccess || hipEventCreate(&a) != hipSuccess ||
        hipEventCreate(&b) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, ctx->device) != hipSuccess)
      st = fail(ctx, HETEGEN_ERR_HIP, "probe setup failed");
    for (int r = 0; st == HETEGEN_OK && r <= reps; ++r) {  // the first run warms up
      float ms = 0;
      if (hipEventRecord(a, ctx->capture_stream) != hipSuccess ||
          hg::launch_read(buf, bytes, sink, 4 * std::max(ncu, 1), ctx->capture_stream) != hipSuccess ||
          hipEventRecord(b, ctx->capture_stream) != hipSuccess || hipEventSynchronize(b) != hipSuccess ||
          hipEventElapsedTime(&ms, a, b) != hipSuccess) {
        st = fail(ctx, HETEGEN_ERR_HIP, "probe read kernel failed");
        break;
      }
      if (r > 0) t.push_back(ms * 1e-3);
    }
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    (void)hipFree(buf);
    (void)hipFree(sink);
    (void)hipGetLastError();
    if (st != HETEGEN_OK) return st;
    std::sort(t.begin(), t.end());
    *Bps_out = (double)bytes / t[t.size() / 2];
    return HETEGEN_OK;
  });
}

// ---- decode step over decoder-layer linears ----
namespace {

void model_free(hetegen_model* m) {
  if (!m) return;
  if (m->gexec) (void)hipGraphExecDestroy(m->gexec);
  for (auto& pl : m->plan)
    if (pl.table) (void)hipFree(pl.table);
  if (m->counters) (void)hipFree(m->counters);
  if (m->err_host) (void)hipHostFree(m->err_host);
  if (m->arena) (void)hipFree(m->arena);
  if (m->act) (void)hipFree(m->act);
  if (m->kv) (void)hipFree(m->kv);
  if (m->kv_part) (void)hipFree(m->kv_part);
  if (m->kv_cnt) (void)hipFree(m->kv_cnt);
  if (m->abuf) (void)hipFree(m->abuf);
  if (m->ws) (void)hipFree(m->ws);
  if (m->ws_cnt) (void)hipFree(m->ws_cnt);
  if (m->ln_part) (void)hipFree(m->ln_part);
  (void)hipGetLastError();
  delete m;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

size_t kv_layer_elems(const hetegen_model* m) {
  return (size_t)m->max_batch * m->heads * m->kv_seq * m->head_dim;
}

// Attention of layer l at position pos over the cache: reads q | k | v from the
// qkv buffer, appends k and v at pos, writes the output to abuf.
hetegen_status run_attention(hetegen_ctx* ctx, hetegen_model* m, int l, int B, int pos, hipStream_t st) {
  hg::AttnParams a{};
  const size_t per = kv_layer_elems(m);
  a.qkv = m->qkv;
  a.ldq = 3LL * m->H;
  a.kc = (uint16_t*)m->kv + (size_t)(2 * l) * per;
  a.vc = (uint16_t*)m->kv + (size_t)(2 * l + 1) * per;
  a.out = m->abuf;
  a.ldo = m->H;
  a.part = m->kv_part;
  a.cnt = m->kv_cnt;
  a.heads = m->heads;
  a.head_dim = m->head_dim;
  a.max_seq = m->kv_seq;
  a.max_chunks = m->kv_chunks;
  a.pos = pos;
  HIPCHK(ctx, hg::launch_attention(a, m->dtype, B, st));
  return HETEGEN_OK;
}

// One step.  pos < 0: the attention of every layer is that of an empty cache (the
// value slice of qkv); pos >= 0: attention over the KV cache at position pos.
hetegen_status enqueue_step(hetegen_ctx* ctx, hetegen_model* m, const void* x_dev, void* out_dev, int B,
                            hipStream_t st, int pos = -1) {
  const int H = m->H, F = m->F;
  // plan every streamed chunk of the step up front so the copy stream can run
  // ahead across linears and layers, bounded by the ring
  if (!pipeline_idle(ctx)) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "internal: stale chunk plan");
  for (const auto& l : m->lin)
    if (!l.resident && l.n_gpu > 0 && l.pageable) TRY(ensure_pin_resources(ctx));
  for (const auto& l : m->lin)
    if (!l.resident && l.n_gpu > 0) plan_chunks(ctx, l.W_host, l.n_gpu, l.K, m->dtype, l.pageable, l.n_cpu == 0);
  char* tr = (char*)m->trace;
  auto take = [&](size_t elems) -> void* {
    if (!tr) return nullptr;
    void* p = tr;
    tr += elems * 2;
    return p;
  };
  // every row of linear i on the matrix-core GEMV (resident, tile order, no CPU rows):
  // then out and fc2 leave LayerNorm partials of x for a following fc1 / qkv of that
  // kind, which normalises its input itself instead of after a LayerNorm launch
  auto all_tiled = [&](int i) {
    const auto& lin = m->lin[i];
    return m->ln_partials && lin.W_tile && lin.n_cpu == 0 && lin.n_gpu == lin.N &&
           (B >= kTiledMinBatch || !lin.W_dev);
  };
  const size_t part = hg::ln_partials_floats(H);
  for (int l = 0; l < m->L; ++l) {
    const void* xl = l == 0 ? x_dev : m->xbuf;
    for (int which = 0; which < 4; ++which) {
      const auto& lin = m->lin[4 * l + which];
      Job j{};
      j.B = B;
      j.K = lin.K;
      j.N = lin.N;
      j.dtype = m->dtype;
      j.W_host = lin.W_host;
      // resident rows: the tile-ordered copy from kTiledMinBatch on (or when it is the only one)
      const bool use_tile = lin.W_tile && (B >= kTiledMinBatch || !lin.W_dev);
      j.W_dev = use_tile ? lin.W_tile : lin.W_dev;
      j.bias_host = lin.bias_host;
      j.bias_dev = lin.bias_dev;
      j.n_gpu = lin.n_gpu;
      j.n_cpu = lin.n_cpu;
      j.tiled = use_tile;
      j.ws = m->ws;
      j.cnt = m->ws_cnt;
      j.ws_floats = m->ws_floats;
      j.cnt_words = m->ws_words;
      j.korder = use_tile ? lin.korder : 0;
      j.segmajor = use_tile ? 0 : lin.segmajor;  // the row-major copy runs batch 1 only
      j.ln_buf = m->lnbuf;
      const int i = 4 * l + which;
      if (which == 0 && l > 0 && all_tiled(i - 1) && all_tiled(i)) j.ln_in = m->ln_part;
      if (which == 1 && all_tiled(i) && all_tiled(i + 1)) j.ln_out = m->ln_part + part;
      if (which == 2 && all_tiled(i - 1) && all_tiled(i)) j.ln_in = m->ln_part + part;
      if (which == 3 && l + 1 < m->L && all_tiled(i) && all_tiled(i + 1)) j.ln_out = m->ln_part;
      j.y_f32 = 0;
      switch (which) {
        case 0:  // qkv = LN(x) Wqkv^T + b
          j.x = xl; j.ldx = H; j.ln = 1;
          j.y = m->qkv; j.ldy = 3 * H; j.epi = hg::EPI_NONE;
          break;
        case 1:  // x = x + (A Wout^T + b): A = attention over the cache, or V = qkv[:, 2H:3H]
          if (pos >= 0) {
            TRY(run_attention(ctx, m, l, B, pos, st));
            j.x = m->abuf; j.ldx = H;
          } else {
            j.x = (const char*)m->qkv + (size_t)2 * H * 2; j.ldx = 3 * H;
          }
          j.ln = 0;
          j.y = m->xbuf; j.ldy = H; j.epi = hg::EPI_RESID; j.resid = xl; j.ldr = H;
          break;
        case 2:  // f = ReLU(LN(x) Wfc1^T + b)
          j.x = m->xbuf; j.ldx = H; j.ln = 1;
          j.y = m->fbuf; j.ldy = F; j.epi = hg::EPI_RELU;
          break;
        default:  // x = x + (f Wfc2^T + b)
          j.x = m->fbuf; j.ldx = F; j.ln = 0;
          j.y = l == m->L - 1 ? out_dev : m->xbuf; j.ldy = H; j.epi = hg::EPI_RESID; j.resid = m->xbuf; j.ldr = H;
          break;
      }
      j.trace_in = take((size_t)B * j.K);
      j.trace_out = take((size_t)B * j.N);
      const auto t0 = Clock::now();
      TRY(run_linear(ctx, j, st));
      m->lin_ms[4 * l + which] = ms_since(t0);
    }
  }
  return HETEGEN_OK;
}

// Launch plan of the persistent step for batch B: grid of co-resident workgroups
// (up to 4 per CU), each linear's rows cut into equal contiguous blocks, and the
// device table of the linears.  Leaves plan.ok false when the step cannot run
// persistently (x too large for LDS, no cooperative launch, too little occupancy).
hetegen_status build_plan(hetegen_ctx* ctx, hetegen_model* m, int B) {
  auto& pl = m->plan[B];
  pl.built = true;
  pl.ok = false;
  if (!m->graphable || !m->rowmajor || B >= kTiledMinBatch) return HETEGEN_OK;  // reads row-major weights
  int ncu = 0, coop = 0;
  HIPCHK(ctx, hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, ctx->device));
  HIPCHK(ctx, hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, ctx->device));
  if (!coop || ncu < 1) return HETEGEN_OK;
  const int unit = hg::gemv_rows_unit(B) * 4;
  const int n = (int)m->lin.size();
  for (int per_cu = 4; per_cu >= 1; --per_cu) {
    const long long G = (long long)ncu * per_cu;
    std::vector<int> rpw(n);
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
      const long long units = (m->lin[i].n_gpu + unit - 1) / unit;
      rpw[i] = (int)(((units + G - 1) / G) * unit);
      lds = std::max(lds, hg::gemv_lds_bytes(B, m->lin[i].K, rpw[i]));
    }
    if (lds > hg::gemv_lds_limit()) return HETEGEN_OK;
    if (hg::step_blocks_per_cu(m->dtype, B, lds) < per_cu) continue;
    std::vector<hg::StepLinear> tab(n);
    const int H = m->H, F = m->F;
    for (int l = 0; l < m->L; ++l) {
      for (int which = 0; which < 4; ++which) {
        const int i = 4 * l + which;
        const auto& lin = m->lin[i];
        hg::StepLinear& d = tab[i];
        d.W = lin.W_dev;
        d.bias = lin.bias_dev;
        d.rows = lin.n_gpu;
        d.K = lin.K;
        d.rpw = rpw[i];
        d.segmajor = lin.segmajor;
        switch (which) {
          case 0:
            d.x = m->xbuf; d.x_in = l == 0; d.ldx = H; d.ln = 1;
            d.y = m->qkv; d.ldy = 3 * H; d.epi = hg::EPI_NONE;
            break;
          case 1:
            d.x = (const char*)m->qkv + (size_t)2 * H * 2; d.ldx = 3 * H;
            d.y = m->xbuf; d.ldy = H; d.epi = hg::EPI_RESID; d.resid = m->xbuf; d.resid_in = l == 0; d.ldr = H;
            break;
          case 2:
            d.x = m->xbuf; d.ldx = H; d.ln = 1;
            d.y = m->fbuf; d.ldy = F; d.epi = hg::EPI_RELU;
            break;
          default:
            d.x = m->fbuf; d.ldx = F;
            d.y = m->xbuf; d.y_out = l == m->L - 1; d.ldy = H; d.epi = hg::EPI_RESID; d.resid = m->xbuf; d.ldr = H;
            break;
        }
      }
    }
    if (hipMalloc(&pl.table, sizeof(hg::StepLinear) * n) != hipSuccess) {
      (void)hipGetLastError();
      pl.table = nullptr;
      return fail(ctx, HETEGEN_ERR_OOM, "persistent step table");
    }
    HIPCHK(ctx, hipMemcpy(pl.table, tab.data(), sizeof(hg::StepLinear) * n, hipMemcpyHostToDevice));
    pl.grid = (int)G;
    pl.lds = lds;
    pl.ok = true;
    return HETEGEN_OK;
  }
  return HETEGEN_OK;
}

// One persistent step; *launched is false when the launch was refused (the caller
// falls back to another mode).
hetegen_status run_persistent(hetegen_ctx* ctx, hetegen_model* m, const void* x_dev, void* out_dev, int B,
                              hipStream_t st, bool* launched) {
  *launched = false;
  auto& pl = m->plan[B];
  if (!pl.built) TRY(build_plan(ctx, m, B));
  if (!pl.ok) return HETEGEN_OK;
  hg::StepArgs a{};
  a.lin = (const hg::StepLinear*)pl.table;
  a.nlin = (int)m->lin.size();
  a.x_in = x_dev;
  a.out = out_dev;
  a.counters = m->counters;
  a.barrier_base = m->barrier_base;
  a.ngroups = m->ngroups;
  a.err = m->err_host;
  a.spin_limit = m->spin_limit ? m->spin_limit : kDefaultSpinLimit;
  hipError_t e = hg::launch_step(a, m->dtype, B, pl.grid, pl.lds, st);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    pl.ok = false;  // do not try again for this batch size
    return HETEGEN_OK;
  }
  m->barrier_base += (uint32_t)a.nlin;
  *launched = true;
  return HETEGEN_OK;
}

}  // namespace

extern "C" {

hetegen_status hetegen_model_create(hetegen_ctx* ctx, int L, int H, int F, hetegen_dtype dtype, void* const* W_host,
                                    void* const* bias_host, const double* alpha, const int* resident, int max_batch,
                                    hetegen_model** out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!out || !W_host || !alpha || L < 1 || H < 8 || F < 8 || H % 8 || F % 8 || max_batch < 1 ||
        max_batch > kMaxBatch)
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_model_create: bad arguments");
    if (dtype != HETEGEN_F16 && dtype != HETEGEN_BF16)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "model dtype: fp16 or bf16");
    if (H > hg::kMaxLnK) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "hidden size %d above %d", H, hg::kMaxLnK);
    *out = nullptr;
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hetegen_model* m = new hetegen_model();
    m->L = L;
    m->H = H;
    m->F = F;
    m->dtype = dtype;
    m->max_batch = max_batch;
    m->tiled = max_batch >= kTiledMinBatch;
    m->rowmajor = !m->tiled;
    m->lin.resize((size_t)4 * L);
    m->lin_ms.assign((size_t)4 * L, 0.0);
    size_t dev_bytes = 0, rm_bytes = 0, tile_bytes = 0;
    for (int i = 0; i < 4 * L; ++i) {
      auto& l = m->lin[i];
      const int which = i % 4;
      l.N = which == 0 ? 3 * H : which == 2 ? F : H;
      l.K = which == 3 ? F : H;
      l.W_host = W_host[i];
      l.bias_host = bias_host ? bias_host[i] : nullptr;
      l.alpha = alpha[i];
      l.resident = resident ? resident[i] != 0 : 0;
      if (!l.W_host || !(l.alpha >= 0 && l.alpha <= 1) || !aligned16(l.W_host)) {
        model_free(m);
        return fail(ctx, HETEGEN_ERR_INVALID_ARG, "linear %d: weight pointer or alpha invalid", i);
      }
      hetegen_status st = check_weight(ctx, l.W_host, (size_t)l.N * l.K * 2, &l.pageable);
      if (st != HETEGEN_OK) {
        model_free(m);
        return st;
      }
      if ((size_t)l.K * 2 > ctx->chunk_bytes && !l.resident) {
        model_free(m);
        return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "linear %d: a row exceeds chunk_bytes", i);
      }
      l.n_cpu = split_cpu_rows(l.N, l.alpha);
      l.n_gpu = l.N - l.n_cpu;
      if (l.resident) {
        rm_bytes += align256((size_t)l.n_gpu * l.K * 2);
        tile_bytes += align256(hg::tiled_bytes(l.n_gpu, l.K));
      }
      if (l.bias_host) dev_bytes += align256((size_t)l.N * 2);
    }
    if (m->tiled) {
      const char* lp = getenv("HETEGEN_LN_PARTIALS");
      m->ln_partials = lp && strcmp(lp, "0") == 0 ? false : lp && strcmp(lp, "1") == 0 ? true : H <= kMaxPartialsH;
    }
    // A tiled model with H <= kMaxDualH also keeps the row-major copy, for batch 1 on the
    // vector GEMV, when both copies take at most half of the device memory free now
    // (HETEGEN_DUAL_LAYOUT=0 / 1 at creation: tile order only / the row-major copy at any H)
    if (m->tiled && rm_bytes) {
      size_t free_b = 0, total_b = 0;
      const char* de = getenv("HETEGEN_DUAL_LAYOUT");
      const bool allow = de && strcmp(de, "0") == 0 ? false : de && strcmp(de, "1") == 0 ? true : H <= kMaxDualH;
      if (allow && hipMemGetInfo(&free_b, &total_b) == hipSuccess && rm_bytes + tile_bytes <= free_b / 2)
        m->rowmajor = true;
      (void)hipGetLastError();
    }
    dev_bytes += (m->rowmajor ? rm_bytes : 0) + (m->tiled ? tile_bytes : 0);
    if (dev_bytes && hipMalloc(&m->arena, dev_bytes) != hipSuccess) {
      (void)hipGetLastError();
      model_free(m);
      return fail(ctx, HETEGEN_ERR_OOM, "%zu bytes of HBM for resident weights", dev_bytes);
    }
    // tile order: each resident block goes through a device staging buffer and is
    // reordered into the arena; the split-K workspace is sized for the largest need
    void* stage = nullptr;
    size_t ws_floats = 0, ws_words = 0;
    if (m->tiled) {
      size_t most = 0;
      for (const auto& l : m->lin)
        if (l.resident) {
          most = std::max(most, (size_t)l.n_gpu * l.K * 2);
          ws_floats = std::max(ws_floats, hg::mfma_ws_floats(l.n_gpu, l.K, max_batch));
          ws_words = std::max(ws_words, hg::mfma_cnt_words(l.n_gpu, l.K));
        }
      if ((most && !m->rowmajor && hipMalloc(&stage, most) != hipSuccess) ||
          (ws_floats && hipMalloc((void**)&m->ws, ws_floats * 4) != hipSuccess) ||
          (ws_words && hipMalloc((void**)&m->ws_cnt, ws_words * 4) != hipSuccess) ||
          hipMalloc((void**)&m->ln_part, 2 * hg::ln_partials_floats(H) * 4) != hipSuccess) {
        (void)hipGetLastError();
        if (stage) (void)hipFree(stage);
        model_free(m);
        return fail(ctx, HETEGEN_ERR_OOM, "tile staging buffer, split-K workspace or LayerNorm partials");
      }
      if (ws_words && hipMemset(m->ws_cnt, 0, ws_words * 4) != hipSuccess) {
        (void)hipFree(stage);
        model_free(m);
        return fail(ctx, HETEGEN_ERR_HIP, "split-K counter initialisation failed");
      }
      m->ws_floats = ws_floats;
      m->ws_words = ws_words;
    }
    // tile order per linear (HETEGEN_TILE_KORDER=0 / 1 at creation: row-tile order / k-major
    // for every linear)
    const char* ko = getenv("HETEGEN_TILE_KORDER");
    const int korder_env = ko && (strcmp(ko, "0") == 0 || strcmp(ko, "1") == 0) ? atoi(ko) : -1;
    // segment-major row-major copies (HETEGEN_SEGMAJOR=0 at creation: plain row-major)
    const char* sm = getenv("HETEGEN_SEGMAJOR");
    const bool seg_on = !(sm && strcmp(sm, "0") == 0);
    char* p = (char*)m->arena;
    for (auto& l : m->lin) {
      if (l.resident) {
        // the row-major copy (when kept) is uploaded first and is also the tiling's source;
        // otherwise the rows pass through the staging buffer
        const size_t rb = (size_t)l.n_gpu * l.K * 2;
        bool ok = true;
        void* src = stage;
        void* rm_stage = nullptr;  // row-major rows of a segment-major copy (also the tiling's source)
        if (m->rowmajor) {
          l.W_dev = p;
          src = p;
          p += align256(rb);
          if (seg_on && l.n_gpu > 0 && l.n_cpu == 0 && l.K % hg::kSegElems == 0 && l.K >= kMinSegmajorK) {
            if (hipMalloc(&rm_stage, rb) == hipSuccess) {
              l.segmajor = 1;
            } else {  // no room for the staging copy: this linear stays row-major
              (void)hipGetLastError();
              rm_stage = nullptr;
            }
          }
          if (l.segmajor) {
            ok = hipMemcpy(rm_stage, l.W_host, rb, hipMemcpyHostToDevice) == hipSuccess &&
                 hg::launch_segmajor(rm_stage, l.n_gpu, l.K, l.W_dev, nullptr) == hipSuccess;
            src = rm_stage;
          } else if (l.n_gpu > 0) {
            ok = hipMemcpy(l.W_dev, l.W_host, rb, hipMemcpyHostToDevice) == hipSuccess;
          }
        }
        if (m->tiled) {
          l.W_tile = p;
          l.korder = korder_env >= 0 ? korder_env : hg::mfma_kmajor(l.n_gpu, l.K);
          p += align256(hg::tiled_bytes(l.n_gpu, l.K));
          if (ok && l.n_gpu > 0)
            ok = (m->rowmajor || hipMemcpy(stage, l.W_host, rb, hipMemcpyHostToDevice) == hipSuccess) &&
                 hg::launch_tile(src, l.K, l.n_gpu, l.K, l.W_tile, nullptr, l.korder) == hipSuccess &&
                 hipDeviceSynchronize() == hipSuccess;
        }
        if (rm_stage) {
          ok = hipDeviceSynchronize() == hipSuccess && ok;
          (void)hipFree(rm_stage);
        }
        if (!ok) {
          (void)hipGetLastError();
          if (stage) (void)hipFree(stage);
          model_free(m);
          return fail(ctx, HETEGEN_ERR_HIP, "resident upload failed");
        }
      }
      if (l.bias_host) {
        l.bias_dev = p;
        if (hipMemcpy(p, l.bias_host, (size_t)l.N * 2, hipMemcpyHostToDevice) != hipSuccess) {
          if (stage) (void)hipFree(stage);
          model_free(m);
          return fail(ctx, HETEGEN_ERR_HIP, "bias upload failed");
        }
        p += align256((size_t)l.N * 2);
      }
    }
    if (stage) (void)hipFree(stage);
    const size_t B = max_batch;
    const size_t xb = align256(B * H * 2), qb = align256(B * 3 * H * 2), fb = align256(B * F * 2),
                 lb = align256(B * std::max(H, F) * 2);
    if (hipMalloc(&m->act, xb + qb + fb + lb) != hipSuccess) {
      (void)hipGetLastError();
      model_free(m);
      return fail(ctx, HETEGEN_ERR_OOM, "activation buffers");
    }
    m->xbuf = m->act;
    m->qkv = (char*)m->act + xb;
    m->fbuf = (char*)m->act + xb + qb;
    m->lnbuf = (char*)m->act + xb + qb + fb;
    // size the pinned hand-off buffers once, so no step reallocates them
    if (ctx->y_pending) HIPCHK(ctx, hipEventSynchronize(ctx->ev_y));
    ctx->y_pending = false;
    {
      hetegen_status hs = ensure_host(ctx, &ctx->x_host, &ctx->x_host_bytes, B * std::max(H, F) * 4);
      if (hs == HETEGEN_OK) hs = ensure_host(ctx, &ctx->y_host, &ctx->y_host_bytes, B * std::max(3 * H, F) * 4);
      if (hs != HETEGEN_OK) {
        model_free(m);
        return hs;
      }
    }
    m->graphable = true;
    for (const auto& l : m->lin)
      if (l.n_cpu > 0 || !l.resident) m->graphable = false;
    if (m->graphable) {
      m->ngroups = kBarrierGroups;
      const size_t cb = (size_t)(m->ngroups + 1) * kCounterBytes;
      if (hipMalloc((void**)&m->counters, cb) != hipSuccess ||
          hipHostMalloc((void**)&m->err_host, sizeof(int), hipHostMallocCoherent) != hipSuccess) {
        (void)hipGetLastError();
        model_free(m);
        return fail(ctx, HETEGEN_ERR_OOM, "barrier counters");
      }
      *m->err_host = 0;
      if (hipMemset(m->counters, 0, cb) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
        model_free(m);
        return fail(ctx, HETEGEN_ERR_HIP, "barrier counter initialisation failed");
      }
    }
    *out = m;
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_set_exec(hetegen_model* m, int mode, uint32_t barrier_spin_limit) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!m || mode < HETEGEN_EXEC_AUTO || mode > HETEGEN_EXEC_EAGER) return HETEGEN_ERR_INVALID_ARG;
    if ((mode == HETEGEN_EXEC_PERSISTENT || mode == HETEGEN_EXEC_GRAPH) && !m->graphable)
      return HETEGEN_ERR_UNSUPPORTED;
    if (mode == HETEGEN_EXEC_PERSISTENT && !m->rowmajor) return HETEGEN_ERR_UNSUPPORTED;
    m->exec_mode = mode;
    m->spin_limit = barrier_spin_limit;
    return HETEGEN_OK;
  });
}

int hetegen_model_last_exec(const hetegen_model* m) { return m ? m->last_exec : -1; }

int hetegen_model_layouts(const hetegen_model* m) {
  if (!m) return 0;
  int kmajor = 0, segmajor = 0;
  for (const auto& l : m->lin) {
    kmajor |= l.W_tile && l.korder == 1;
    segmajor |= l.W_dev && l.segmajor;
  }
  return (m->rowmajor ? HETEGEN_LAYOUT_ROWMAJOR : 0) | (m->tiled ? HETEGEN_LAYOUT_TILED : 0) |
         (kmajor ? HETEGEN_LAYOUT_KMAJOR : 0) | (segmajor ? HETEGEN_LAYOUT_SEGMAJOR : 0);
}

hetegen_status hetegen_model_set_alpha(hetegen_model* m, const double* alpha) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!m || !alpha) return HETEGEN_ERR_INVALID_ARG;
    for (size_t i = 0; i < m->lin.size(); ++i)
      if (!m->lin[i].resident && !(alpha[i] >= 0 && alpha[i] <= 1)) return HETEGEN_ERR_INVALID_ARG;
    for (size_t i = 0; i < m->lin.size(); ++i) {
      auto& l = m->lin[i];
      if (l.resident) continue;
      l.alpha = alpha[i];
      l.n_cpu = split_cpu_rows(l.N, l.alpha);
      l.n_gpu = l.N - l.n_cpu;
    }
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_get_alpha(const hetegen_model* m, double* alpha_out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!m || !alpha_out) return HETEGEN_ERR_INVALID_ARG;
    for (size_t i = 0; i < m->lin.size(); ++i) alpha_out[i] = m->lin[i].alpha;
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_read_ms(hetegen_ctx* ctx, const hetegen_model* m, int reps, void* stream,
                                     double* ms_out) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!m || !ms_out || reps < 1) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_model_read_ms: bad arguments");
    std::vector<std::pair<const void*, size_t>> bufs;
    for (const auto& l : m->lin)
      if (l.resident && l.n_gpu > 0) bufs.emplace_back(l.W_dev ? l.W_dev : l.W_tile, (size_t)l.n_gpu * l.K * 2);
    if (bufs.empty()) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_model_read_ms: no resident GPU rows");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hipStream_t st = stream ? (hipStream_t)stream : ctx->capture_stream;
    int ncu = 0;
    HIPCHK(ctx, hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, ctx->device));
    uint32_t* sink = nullptr;
    if (hipMalloc((void**)&sink, 256) != hipSuccess) {
      (void)hipGetLastError();
      return fail(ctx, HETEGEN_ERR_OOM, "hetegen_model_read_ms: sink");
    }
    hipEvent_t a = nullptr, b = nullptr;
    hetegen_status rs = HETEGEN_OK;
    std::vector<double> t;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess)
      rs = fail(ctx, HETEGEN_ERR_HIP, "hetegen_model_read_ms: events");
    for (int r = 0; rs == HETEGEN_OK && r <= reps; ++r) {  // the first pass warms up
      bool ok = hipEventRecord(a, st) == hipSuccess;
      for (size_t i = 0; ok && i < bufs.size(); ++i)
        ok = hg::launch_read(bufs[i].first, bufs[i].second, sink, 4 * std::max(ncu, 1), st) == hipSuccess;
      float ms = 0;
      ok = ok && hipEventRecord(b, st) == hipSuccess && hipEventSynchronize(b) == hipSuccess &&
           hipEventElapsedTime(&ms, a, b) == hipSuccess;
      if (!ok) rs = fail(ctx, HETEGEN_ERR_HIP, "hetegen_model_read_ms: read pass failed");
      else if (r > 0) t.push_back(ms);
    }
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
    (void)hipFree(sink);
    (void)hipGetLastError();
    if (rs != HETEGEN_OK) return rs;
    std::sort(t.begin(), t.end());
    *ms_out = t[t.size() / 2];
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_linear_ms(const hetegen_model* m, double* ms_out) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!m || !ms_out) return HETEGEN_ERR_INVALID_ARG;
    for (size_t i = 0; i < m->lin.size(); ++i) ms_out[i] = m->lin_ms[i];
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_alpha_benchmark(hetegen_ctx* ctx, hetegen_model* m, const void* x_dev, void* out_dev,
                                             int B, double gamma, double lambda, int degree, int reps, int objective,
                                             void* stream, double* delta_out, int* crossed) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    if (!m || !delta_out || !(gamma > 0) || !(lambda > 0) || reps < 1 || degree < 1 || degree > 3 ||
        (objective != HETEGEN_BENCH_CROSSING && objective != HETEGEN_BENCH_WALL))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "hetegen_model_alpha_benchmark: bad arguments");
    std::vector<double> base(m->lin.size());
    bool any = false;
    for (size_t i = 0; i < m->lin.size(); ++i) {
      base[i] = m->lin[i].alpha;
      any = any || !m->lin[i].resident;
    }
    if (!any) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "no streamed linear to balance");
    auto apply = [&](double d) {
      std::vector<double> a(base);
      for (size_t i = 0; i < a.size(); ++i)
        if (!m->lin[i].resident) a[i] = std::min(1.0, std::max(0.0, base[i] + d));
      return hetegen_model_set_alpha(m, a.data());
    };
    const bool was = ctx->profiling;
    TRY(flush_profile(ctx));
    const hetegen_profile saved = ctx->prof;
    auto med = [](std::vector<double> v) {
      std::sort(v.begin(), v.end());
      return v[v.size() / 2];
    };
    // One pass measures the bracket [center - gamma, center + gamma]; when its solution
    // is a bracket end (the curves do not meet inside, or the time still falls there),
    // the bracket is re-centred on that end and measured again, up to kPasses in all.
    constexpr int kPasses = 3;
    double center = 0.0, d_best = 0.0;
    int cr = 0;
    hetegen_status st = HETEGEN_OK;
    for (int pass = 0; pass < kPasses && st == HETEGEN_OK; ++pass) {
      std::vector<double> ds, tc, tg, tw;
      for (int i = 0;; ++i) {
        const double d = -gamma + i * lambda;
        if (d > gamma + 1e-9) break;
        ds.push_back(center + std::min(d, gamma));
      }
      if ((int)ds.size() < degree + 1) {
        st = fail(ctx, HETEGEN_ERR_INVALID_ARG, "too few points in the bracket");
        break;
      }
      ctx->profiling = objective == HETEGEN_BENCH_CROSSING;
      for (double d : ds) {
        st = apply(d);
        std::vector<double> c, g, w;
        for (int r = 0; r <= reps && st == HETEGEN_OK; ++r) {
          ctx->prof = hetegen_profile{};
          auto t0 = Clock::now();
          st = hetegen_decode_step(ctx, m, x_dev, out_dev, B, stream);
          if (st == HETEGEN_OK && hipStreamSynchronize((hipStream_t)stream) != hipSuccess)
            st = fail(ctx, HETEGEN_ERR_HIP, "hipStreamSynchronize failed");
          const double wall = ms_since(t0);
          if (st == HETEGEN_OK) st = flush_profile(ctx);
          if (st == HETEGEN_OK && r > 0) {
            c.push_back(ctx->prof.cpu_ms);
            g.push_back(ctx->prof.h2d_ms + ctx->prof.gpu_ms);
            w.push_back(wall);
          }
        }
        if (st != HETEGEN_OK) break;
        tc.push_back(med(c));
        tg.push_back(med(g));
        tw.push_back(med(w));
      }
      ctx->profiling = was;
      if (st != HETEGEN_OK) break;
      const double lo = center - gamma, hi = center + gamma;
      hetegen_status fs = objective == HETEGEN_BENCH_CROSSING
                              ? hetegen_alpha_fit(ds.data(), tc.data(), tg.data(), (int)ds.size(), degree, lo, hi,
                                                  &d_best, &cr)
                              : hetegen_alpha_minimize(ds.data(), tw.data(), (int)ds.size(), degree, lo, hi, &d_best);
      if (fs != HETEGEN_OK) {
        st = fail(ctx, fs, "alpha fit failed");
        break;
      }
      const bool at_end = (d_best <= lo || d_best >= hi) && !(objective == HETEGEN_BENCH_CROSSING && cr);
      if (!at_end) break;
      center = d_best;
    }
    ctx->prof = saved;
    ctx->profiling = was;
    if (st != HETEGEN_OK) {
      (void)hetegen_model_set_alpha(m, base.data());
      return st;
    }
    TRY(apply(d_best));
    *delta_out = d_best;
    if (crossed) *crossed = cr;
    return HETEGEN_OK;
  });
}

size_t hetegen_model_trace_bytes(const hetegen_model* m, int B) {
  if (!m || B < 1) return 0;
  size_t e = 0;
  for (const auto& l : m->lin) e += (size_t)B * (l.K + l.N);
  return e * 2;
}

hetegen_status hetegen_model_set_trace(hetegen_model* m, void* trace_dev, size_t bytes) {
  return api_guard(nullptr, [&]() -> hetegen_status {
    if (!m) return HETEGEN_ERR_INVALID_ARG;
    if (trace_dev && !aligned16(trace_dev)) return HETEGEN_ERR_INVALID_ARG;
    m->trace = trace_dev;
    m->trace_bytes = trace_dev ? bytes : 0;
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_model_destroy(hetegen_ctx* ctx, hetegen_model* m) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    if (!m) return HETEGEN_OK;
    (void)hipSetDevice(ctx->device);
    (void)hipDeviceSynchronize();
    model_free(m);
    return HETEGEN_OK;
  });
}

hetegen_status hetegen_decode_step(hetegen_ctx* ctx, hetegen_model* m, const void* x_dev, void* out_dev, int B,
                                   void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    auto t0 = Clock::now();
    ctx->err.clear();
    if (!m || !x_dev || !out_dev || x_dev == out_dev)
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "decode_step: bad pointers");
    if (B < 1 || B > m->max_batch) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B = %d outside [1, %d]", B, m->max_batch);
    if (!aligned16(x_dev) || !aligned16(out_dev))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "x/out must be 16-byte aligned");
    if (m->trace && m->trace_bytes < hetegen_model_trace_bytes(m, B))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "trace buffer too small");
    if (m->err_host && *(volatile int*)m->err_host)
      return fail(ctx, HETEGEN_ERR_HIP, "a grid-barrier wait of an earlier persistent step gave up; that step's "
                                        "output is undefined");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    hipStream_t st = (hipStream_t)stream;
    // AUTO runs per-linear launches directly: on this device back-to-back GEMV launches
    // leave no gap, and the grid barrier of the persistent step costs more than a launch
    const bool fast = m->graphable && !m->trace && !ctx->profiling && m->exec_mode != HETEGEN_EXEC_EAGER &&
                      m->exec_mode != HETEGEN_EXEC_AUTO;
    if (fast && m->exec_mode == HETEGEN_EXEC_PERSISTENT) {
      bool launched = false;
      TRY(run_persistent(ctx, m, x_dev, out_dev, B, st, &launched));
      if (launched) {
        m->last_exec = HETEGEN_EXEC_PERSISTENT;
        return finish_call(ctx, t0);
      }
      if (m->exec_mode == HETEGEN_EXEC_PERSISTENT)
        return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "the persistent step cannot run for batch %d on this device", B);
    }
    const bool use_graph = fast;
    if (use_graph) {
      if (!m->gexec || m->g_B != B || m->g_x != x_dev || m->g_out != out_dev) {
        if (m->gexec) {
          HIPCHK(ctx, hipGraphExecDestroy(m->gexec));
          m->gexec = nullptr;
        }
        hipGraph_t g = nullptr;
        HIPCHK(ctx, hipStreamBeginCapture(ctx->capture_stream, hipStreamCaptureModeThreadLocal));
        hetegen_status cs = enqueue_step(ctx, m, x_dev, out_dev, B, ctx->capture_stream);
        hipError_t ce = hipStreamEndCapture(ctx->capture_stream, &g);
        if (cs != HETEGEN_OK) {
          if (g) (void)hipGraphDestroy(g);
          return cs;
        }
        if (ce != hipSuccess) return fail(ctx, HETEGEN_ERR_HIP, "hipStreamEndCapture: %s", hipGetErrorString(ce));
        hipError_t ie = hipGraphInstantiate(&m->gexec, g, nullptr, nullptr, 0);
        (void)hipGraphDestroy(g);
        if (ie != hipSuccess) {
          m->gexec = nullptr;
          return fail(ctx, HETEGEN_ERR_HIP, "hipGraphInstantiate: %s", hipGetErrorString(ie));
        }
        m->g_B = B;
        m->g_x = x_dev;
        m->g_out = out_dev;
      }
      HIPCHK(ctx, hipGraphLaunch(m->gexec, st));
      m->last_exec = HETEGEN_EXEC_GRAPH;
      return finish_call(ctx, t0);
    }
    m->last_exec = HETEGEN_EXEC_EAGER;
    hetegen_status s = enqueue_step(ctx, m, x_dev, out_dev, B, st);
    if (s != HETEGEN_OK) {
      reset_pipeline(ctx);
      return s;
    }
    return finish_call(ctx, t0);
  });
}

// ---- KV cache and attention steps (Sec. 2.1, Eq. 1) ----
hetegen_status hetegen_model_kv_create(hetegen_ctx* ctx, hetegen_model* m, int max_seq, int head_dim) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    if (!m || max_seq < 1 || max_seq > hg::attn_max_positions())
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "kv_create: max_seq %d outside [1, %d]", max_seq,
                  hg::attn_max_positions());
    if ((head_dim != 64 && head_dim != 128) || m->H % head_dim)
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "head_dim %d: 64 or 128, dividing H = %d", head_dim, m->H);
    if (m->kv) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "kv_create: the model already has a KV cache");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    const int chunk = hg::attn_chunk();
    m->heads = m->H / head_dim;
    m->head_dim = head_dim;
    m->kv_seq = max_seq;
    m->kv_chunks = (max_seq + chunk - 1) / chunk;
    const size_t kv_bytes = 2 * (size_t)m->L * kv_layer_elems(m) * 2;
    const size_t part_bytes = (size_t)m->max_batch * m->heads * m->kv_chunks * (head_dim + 2) * sizeof(float);
    const size_t cnt_bytes = (size_t)m->max_batch * m->heads * sizeof(uint32_t);
    if (hipMalloc(&m->kv, kv_bytes) != hipSuccess || hipMalloc((void**)&m->kv_part, part_bytes) != hipSuccess ||
        hipMalloc((void**)&m->kv_cnt, cnt_bytes) != hipSuccess ||
        hipMalloc(&m->abuf, (size_t)m->max_batch * m->H * 2) != hipSuccess) {
      (void)hipGetLastError();
      if (m->kv) (void)hipFree(m->kv);
      if (m->kv_part) (void)hipFree(m->kv_part);
      if (m->kv_cnt) (void)hipFree(m->kv_cnt);
      if (m->abuf) (void)hipFree(m->abuf);
      m->kv = nullptr;
      m->kv_part = nullptr;
      m->kv_cnt = nullptr;
      m->abuf = nullptr;
      m->kv_seq = 0;
      return fail(ctx, HETEGEN_ERR_OOM, "KV cache of %zu bytes", kv_bytes);
    }
    HIPCHK(ctx, hipMemset(m->kv_cnt, 0, cnt_bytes));
    HIPCHK(ctx, hipMemset(m->kv, 0, kv_bytes));
    return HETEGEN_OK;
  });
}

}  // extern "C"

namespace {

// Copy positions [pos0, pos0 + n) of layer l between the cache and token-major
// device buffers [B, n, H] (to_cache: buffers -> cache).
hetegen_status kv_copy(hetegen_ctx* ctx, hetegen_model* m, int l, int B, int pos0, int n, void* k, void* v,
                       hipStream_t st, bool to_cache) {
  if (!m || !m->kv) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "the model has no KV cache");
  if (!k || !v || l < 0 || l >= m->L || B < 1 || B > m->max_batch || pos0 < 0 || n < 1 || pos0 + n > m->kv_seq)
    return fail(ctx, HETEGEN_ERR_INVALID_ARG, "kv copy: bad arguments");
  HIPCHK(ctx, hipSetDevice(ctx->device));
  const size_t per = kv_layer_elems(m), D = m->head_dim, row = D * 2, tok = (size_t)m->H * 2;
  for (int which = 0; which < 2; ++which) {
    char* cache = (char*)m->kv + (size_t)(2 * l + which) * per * 2;
    char* buf = (char*)(which ? v : k);
    for (int b = 0; b < B; ++b) {
      for (int h = 0; h < m->heads; ++h) {
        char* c = cache + (((size_t)b * m->heads + h) * m->kv_seq + pos0) * row;
        char* t = buf + (size_t)b * n * tok + (size_t)h * row;
        if (to_cache) HIPCHK(ctx, hipMemcpy2DAsync(c, row, t, tok, row, n, hipMemcpyDeviceToDevice, st));
        else HIPCHK(ctx, hipMemcpy2DAsync(t, tok, c, row, row, n, hipMemcpyDeviceToDevice, st));
      }
    }
  }
  return HETEGEN_OK;
}

}  // namespace

extern "C" {

hetegen_status hetegen_model_kv_write(hetegen_ctx* ctx, hetegen_model* m, int layer, int B, int pos0, int n,
                                      const void* k_dev, const void* v_dev, void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    return kv_copy(ctx, m, layer, B, pos0, n, const_cast<void*>(k_dev), const_cast<void*>(v_dev),
                   (hipStream_t)stream, true);
  });
}

hetegen_status hetegen_model_kv_read(hetegen_ctx* ctx, hetegen_model* m, int layer, int B, int pos0, int n,
                                     void* k_dev, void* v_dev, void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    ctx->err.clear();
    return kv_copy(ctx, m, layer, B, pos0, n, k_dev, v_dev, (hipStream_t)stream, false);
  });
}

hetegen_status hetegen_decode_step_kv(hetegen_ctx* ctx, hetegen_model* m, const void* x_dev, void* out_dev, int B,
                                      int pos, void* stream) {
  return api_guard(ctx, [&]() -> hetegen_status {
    if (!ctx) return HETEGEN_ERR_INVALID_ARG;
    auto t0 = Clock::now();
    ctx->err.clear();
    if (!m || !x_dev || !out_dev || x_dev == out_dev)
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "decode_step: bad pointers");
    if (!m->kv) return fail(ctx, HETEGEN_ERR_INVALID_ARG, "the model has no KV cache (hetegen_model_kv_create)");
    if (pos < 0 || pos >= m->kv_seq)
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "position %d outside the cache [0, %d)", pos, m->kv_seq);
    if (B < 1 || B > m->max_batch) return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "B = %d outside [1, %d]", B, m->max_batch);
    if (!aligned16(x_dev) || !aligned16(out_dev))
      return fail(ctx, HETEGEN_ERR_UNSUPPORTED, "x/out must be 16-byte aligned");
    if (m->trace && m->trace_bytes < hetegen_model_trace_bytes(m, B))
      return fail(ctx, HETEGEN_ERR_INVALID_ARG, "trace buffer too small");
    HIPCHK(ctx, hipSetDevice(ctx->device));
    m->last_exec = HETEGEN_EXEC_EAGER;
    hetegen_status s = enqueue_step(ctx, m, x_dev, out_dev, B, (hipStream_t)stream, pos);
    if (s != HETEGEN_OK) {
      reset_pipeline(ctx);
      return s;
    }
    return finish_call(ctx, t0);
  });
}

}  // extern "C"
