/*
 * hetegen.h - C ABI of the MI355X heterogeneous-parallel Linear (HeteGen,
 * arXiv 2403.01164) for batch-1..8 decoding.
 *
 * A linear module y = x W^T + b with its weight W [N, K] in pinned host memory
 * is split by output feature: the leading rows [0, n_gpu) are computed on the
 * GPU (resident in HBM, or streamed host-to-device in chunks), the trailing rows
 * [n_gpu, N) on host cores, and both parts land in one device output
 * (Sec. 3.1 "Parallelism Strategy", Fig. 3a, Eq. 2: heterogeneous tensor
 * parallelism partitions the weight; Sec. 4.2, Fig. 5a: activation to the CPU,
 * CPU compute concurrent with weight transfer, CPU outputs back to the GPU).
 *
 * Conventions used by every call:
 *  - alpha is the CPU fraction of the output features:
 *        n_cpu = min(N, floor(alpha * N + 0.5)),  n_gpu = N - n_cpu.
 *    The paper's alpha (Sec. 3.2) is the GPU fraction, i.e. 1 - alpha here.
 *  - Matrices are row-major.  W has N rows of K elements (nn.Linear layout).
 *    x is [B, K], y is [B, N]; row strides are given in elements.
 *  - Element types: HETEGEN_F16 (IEEE binary16), HETEGEN_BF16, HETEGEN_F32.
 *    Weights, activations and biases of one call share one 16-bit type;
 *    accumulation is binary32.
 *  - Streams are hipStream_t values passed as void*; NULL is the null stream.
 *  - Every call returns a status and never throws or aborts across the ABI.
 *    On failure hetegen_last_error() describes the error; outputs are undefined.
 *  - A context is not thread-safe: one in-flight call per context.
 */
#ifndef HETEGEN_H
#define HETEGEN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HETEGEN_API __attribute__((visibility("default")))

typedef enum {
  HETEGEN_OK = 0,
  HETEGEN_ERR_INVALID_ARG = 1, /* null pointer, bad size, alpha outside [0,1] or not finite */
  HETEGEN_ERR_NOT_PINNED = 2,  /* a host weight buffer is not page-locked host memory */
  HETEGEN_ERR_UNSUPPORTED = 3, /* K % 8 != 0, B outside [1, 8], misaligned pointer, dtype mix */
  HETEGEN_ERR_OOM = 4,         /* device, pinned or host allocation failed */
  HETEGEN_ERR_HIP = 5,         /* a HIP runtime call failed (code in the message) */
  HETEGEN_ERR_INTERNAL = 6     /* any other host-side failure (message says what); no call
                                  lets an exception cross this interface */
} hetegen_status;

typedef enum { HETEGEN_F16 = 0, HETEGEN_BF16 = 1, HETEGEN_F32 = 2 } hetegen_dtype;

typedef struct hetegen_ctx hetegen_ctx;
typedef struct hetegen_model hetegen_model;

typedef struct {
  int device;         /* HIP device ordinal */
  int cpu_threads;    /* host threads for the CPU share (the calling thread and a worker team);
                         <= 0: the OpenMP default thread count (OMP_NUM_THREADS) */
  size_t chunk_bytes; /* weight bytes per streamed chunk; 0: 32 MiB */
  int ring_depth;     /* device staging slots for streamed chunks, in [2, 64]; 0: 8 */
  int pin_threads;    /* host threads that stage pageable weights into pinned memory
                         (Sec. 4.2 hybrid pin || transfer), in [1, 64]; 0: 4;
                         < 0: pageable weights are refused with HETEGEN_ERR_NOT_PINNED */
  int pin_ring;       /* pinned staging buffers of chunk_bytes each, in [2, 64]; 0: 4 */
  int numa_node;      /* NUMA placement of the pinned host memory the context allocates
                         (hetegen_host_alloc, hand-off and staging buffers): n > 0 binds it to
                         node n - 1 (INVALID_ARG if that node does not exist); 0: the
                         allocating thread's own memory policy */
} hetegen_config;

/* Create a context on cfg->device: a copy stream, the staging ring
 * (ring_depth x chunk_bytes of HBM), pinned hand-off buffers, events and the
 * parameter manager thread (Sec. 4.3), which owns the copy stream: it walks the
 * streamed chunks of a call in order and copies each into the staging ring as soon
 * as the slot is free, running ahead of the GEMVs across linears and layers.  A
 * chunk of pageable weights is first copied into a pinned staging buffer by the
 * pin team (pin_threads threads, the manager included) while earlier chunks are in
 * flight over PCIe, so pinning and transfer overlap (Eq. 8: T_COM = max(T_PIN,
 * T_TRANS)); pinned memory stays bounded by pin_ring x chunk_bytes, allocated at
 * the first pageable chunk.  For full overlap with the CPU share, ring_depth x
 * chunk_bytes should hold the largest GPU share of a streamed linear: the GEMVs of
 * chunks that were not yet staged when the CPU share starts are enqueued after it.
 * cfg may be NULL (device 0, defaults).  *out receives the context.
 * Testing aid: with the environment variable HETEGEN_POISON set (and not "0") when the
 * context is created, every staging slot, pinned staging buffer and host hand-off
 * buffer is filled with all-ones bits (NaN in fp16, bf16 and binary32) before each
 * reuse, so a read that is not ordered after the data it needs shows up as NaN; it
 * costs one device fill per streamed chunk. */
HETEGEN_API hetegen_status hetegen_create(const hetegen_config* cfg, hetegen_ctx** out);

/* Wait for the context's work and free everything it owns.  NULL is a no-op. */
HETEGEN_API hetegen_status hetegen_destroy(hetegen_ctx* ctx);

/* Message of the last failing call on ctx ("" if none).  With ctx == NULL, the
 * message of the last failing hetegen_create on this thread.  The string stays
 * valid until the next call on ctx. */
HETEGEN_API const char* hetegen_last_error(const hetegen_ctx* ctx);

/* Instruction set the CPU share uses on this host, chosen at load time: "avx512+bf16"
 * (bf16 weights through the AVX512-BF16 dot product, fp16 widened to binary32 and
 * FMA; the environment variable HETEGEN_CPU_BF16=0 at load keeps bf16 on the widening
 * path too), "avx512", "avx2" or "scalar".  A static string. */
HETEGEN_API const char* hetegen_cpu_share_isa(void);

/* Page-locked host memory for weights: *p receives `bytes` bytes that the CPU
 * share reads directly and the copy engines read over PCIe (not write-combined).
 * Free with hetegen_host_free.  OOM if the allocation fails. */
HETEGEN_API hetegen_status hetegen_host_alloc(hetegen_ctx* ctx, size_t bytes, void** p);
HETEGEN_API hetegen_status hetegen_host_free(hetegen_ctx* ctx, void* p);

/* One heterogeneous linear module (Sec. 3.1, Eq. 2; Sec. 4.2, Fig. 5a):
 *
 *   y[b, j] = sum_k x[b, k] * W[j, k] + bias[j],   b < B, j < N,
 *
 * rows j < n_gpu on the GPU, rows j >= n_gpu on host threads (see alpha above).
 *   x_dev          device, [B, K] in w_dtype, row stride K, 16-byte aligned.
 *   W_host         host [N, K] w_dtype: pinned (hetegen_host_alloc or hipHostMalloc),
 *                  or pageable (staged through pinned buffers, see hetegen_create).
 *   W_dev_resident optional device copy of rows [0, n_gpu) (row stride K); when
 *                  NULL the GPU rows are streamed from W_host through the staging
 *                  ring in chunks, overlapped with the CPU share.
 *   bias_host      optional host [N] w_dtype, read for the CPU rows;
 *   bias_dev       optional device [N] w_dtype, read for the GPU rows.  Pass both
 *                  or neither (a side with rows needs its pointer).
 *   y_dev          device [B, N] of y_dtype (w_dtype or HETEGEN_F32), row stride N.
 * GPU work is enqueued on `stream`.  The call returns after the CPU share is
 * computed and its upload is enqueued; y is complete in `stream` order.
 * B in [1, 8], K % 8 == 0, K >= 8, N >= 1.  NOT_PINNED if W_host is pageable and
 * the context refuses pageable weights (pin_threads < 0). */
HETEGEN_API hetegen_status hetegen_linear(hetegen_ctx* ctx, const void* x_dev, int B, int K, const void* W_host,
                              const void* W_dev_resident, int N, hetegen_dtype w_dtype,
                              const void* bias_host, const void* bias_dev, double alpha, void* y_dev,
                              hetegen_dtype y_dtype, void* stream);

/* ---- GPU rows of a resident weight in matrix-core tile order ----
 * The GPU's share of a module (Sec. 3.1, Eq. 2; Sec. 4.2: the GPU computes its part
 * of the output from weights in device memory), all rows resident.  The weight
 * [N, K] is stored as 1 KiB tiles of 16 rows x 32 columns, row tile after row tile
 * (the k-tiles of rows [16 t, 16 t + 16) are contiguous); within a tile the 16 bytes
 * at offset 16 l hold W[16 t + l % 16][32 k + 8 (l / 16) + e], e < 8.  Rows past N
 * and columns past K are zero.  One tile is the 16-row operand of one 16x16x32
 * matrix-core product, so the GEMV reads every tile with one coalesced 1 KiB load
 * and runs on the matrix cores at every batch size (decode steps of models created
 * for batches of 2 or more keep their resident rows in this order). */

/* Bytes of the tile-ordered copy of a [rows, K] weight (0 for rows < 1 or K not a
 * positive multiple of 8). */
HETEGEN_API size_t hetegen_tiled_bytes(int rows, int K);

/* W_tiled_dev = tile order of W_dev [rows, K] (device, row-major, row stride K);
 * both device pointers, 16-byte aligned, caller-owned; W_tiled_dev holds
 * hetegen_tiled_bytes(rows, K) bytes and may not overlap W_dev.  Enqueued on
 * `stream`.  K % 8 == 0. */
HETEGEN_API hetegen_status hetegen_tile_weights(hetegen_ctx* ctx, const void* W_dev, int rows, int K,
                                                void* W_tiled_dev, void* stream);

/* y[b, j] = sum_k x[b, k] * W[j, k] + bias[j] for all N rows on the GPU, W given in
 * tile order (hetegen_tile_weights).  x_dev [B, K] and y_dev [B, N] (row strides K
 * and N) as in hetegen_linear; bias_dev optional device [N].  Binary32 sums (the
 * matrix core's products of 16-bit values are exact).  When one workgroup per 16-row
 * tile would load the device's compute units unevenly (the busiest more than 1.15x
 * the mean), the sum over K is split over up to 8 workgroups (each at least 32
 * 32-column tiles long) whose partial sums are added in a fixed order: the split
 * depends on N, K and the device's compute-unit count, not on B or timing, so a
 * batch row's bits do not depend on the batch size.  Uses the context's split-K
 * workspace, which the first call with a larger need allocates (device memory,
 * after waiting for the device); calls on one context must not overlap.  Enqueued
 * on `stream`.  B in [1, 8], K % 8 == 0, N >= 1, B * K < 2^30 (x is read through
 * a buffer descriptor, whose offsets are 32-bit). */
HETEGEN_API hetegen_status hetegen_linear_tiled(hetegen_ctx* ctx, const void* x_dev, int B, int K,
                                                const void* W_tiled_dev, int N, hetegen_dtype w_dtype,
                                                const void* bias_dev, void* y_dev, hetegen_dtype y_dtype,
                                                void* stream);

/* hetegen_linear_tiled for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation): same
 * arguments and results, but the split-K partials and arrival counters live in a
 * fixed scratch array compiled into the library, one per GPU, set up by
 * hetegen_create and held until the process ends (262144 floats of partials and
 * 65536 counters, 1.25 MiB per GPU).  The call allocates nothing; it returns
 * UNSUPPORTED, without launching, for a shape whose split (see hetegen_linear_tiled)
 * needs more than that, i.e. ceil(N / 16) * splits * 16 * B floats.  On a 256-CU
 * device every linear of OPT-6.7B to OPT-175B fits at batch 8 (the largest need,
 * OPT-13B's [5120, 5120] and [5120, 20480] in 4 splits, is 163840 floats); a split
 * linear of more than 1024 row tiles at batch 8, such as [16400, 36864], does not.  Every
 * call on one GPU shares that GPU's scratch: calls that overlap on one GPU (from
 * several streams, contexts or threads) race and give undefined results.  A launch
 * returns the counters it used to zero, so calls in stream order need no clearing. */
HETEGEN_API hetegen_status hetegen_linear_tiled_noalloc(hetegen_ctx* ctx, const void* x_dev, int B, int K,
                                                        const void* W_tiled_dev, int N, hetegen_dtype w_dtype,
                                                        const void* bias_dev, void* y_dev, hetegen_dtype y_dtype,
                                                        void* stream);

/* ---- Alpha planner: computation distribution law (Sec. 3.2, Eq. 4-7; Eq. 8-9) ---- */

typedef struct {
  int N, K;            /* weight shape */
  hetegen_dtype dtype; /* element type of W */
  int resident;        /* 1: the whole module stays on the GPU (alpha = 0) */
} hetegen_shape;

/* Speeds in weight bytes per second (the paper's "parameter size divided by
 * processing time", Fig. 1 caption). */
typedef struct {
  double cpu_Bps;      /* V_CPU: CPU share GEMV */
  double h2d_Bps;      /* V_COM transfer part: pinned host-to-device copy */
  double hbm_gemv_Bps; /* V_GPU: GPU GEMV */
  double pin_Bps;      /* pinning speed for pageable weights; <= 0: weights pre-pinned */
} hetegen_bw;

#define HETEGEN_PLAN_APPROX 1 /* use Eq. 6/7 (GPU time neglected) instead of Eq. 5 */

/* alpha_out[i] = CPU fraction for shapes[i]:
 *   resident -> 0, otherwise clamp(1 - alpha_gpu, 0, 1) with
 *   alpha_gpu = V_GPU V_COM / (V_CPU V_GPU + V_CPU V_COM + V_COM V_GPU)   (Eq. 5)
 *   or V_COM / (V_COM + V_CPU) with HETEGEN_PLAN_APPROX                    (Eq. 6)
 *   where V_COM = min(h2d_Bps, pin_Bps) when pin_Bps > 0 (Eq. 8: T_COM = max(T_PIN, T_TRANS)).
 * bw holds n_bw == n entries (one per shape) or n_bw == 1 (shared).  Speeds must
 * be finite and > 0.  Pure host arithmetic; no device is touched. */
HETEGEN_API hetegen_status hetegen_layer_plan(const hetegen_shape* shapes, int n, const hetegen_bw* bw, int n_bw,
                                  int flags, double* alpha_out);

/* Measure V_CPU, V_COM and V_GPU for one shape on this context (the inputs of the
 * distribution law): the CPU share GEMV over all N rows of W_host (alpha = 1), the
 * chunked host-to-device copy of W_host through the staging ring, and the GPU
 * GEMV over the staged chunks; each is the median of `reps` runs in weight bytes
 * per second (the CPU share after one untimed pass; host caches are flushed
 * before every CPU pass, as a step's weights always come from DRAM).  W_host is
 * [N, K]; batch B.
 * Pinned W_host: pin_Bps is set to 0 (no pinning).  Pageable W_host: pin_Bps is the
 * pin team's rate staging W_host into the pinned buffers, h2d_Bps the copy rate
 * from those buffers, each measured alone (the planner takes the smaller, Eq. 8).
 * flags & HETEGEN_PROBE_CONCURRENT (pinned W_host): cpu_Bps and h2d_Bps are instead
 * measured with the CPU share and the copies running at the same time, as they do
 * in a heterogeneous linear (both read host memory; Sec. 4.4 notes that measured
 * speeds depend on such system conditions): the copies of W_host run once while
 * the CPU share repeats over W_host, on flushed caches each time; the CPU rate
 * counts the passes that ended before the copies did. */
#define HETEGEN_PROBE_CONCURRENT 1
HETEGEN_API hetegen_status hetegen_probe(hetegen_ctx* ctx, const void* W_host, int N, int K, hetegen_dtype dtype,
                                         int B, int reps, int flags, hetegen_bw* out);

/* Achievable HBM read bandwidth: a streaming read of `bytes` (>= 1 MiB, a multiple
 * of 16) of device memory with 16-byte non-temporal loads (those of the GEMV), four
 * workgroups per CU; *Bps_out = bytes / median time of `reps` runs.  The
 * denominator the resident GEMV is compared with next to the nominal HBM peak. */
HETEGEN_API hetegen_status hetegen_probe_hbm(hetegen_ctx* ctx, size_t bytes, int reps, double* Bps_out);

/* Idle host-to-device link rate: one hipMemcpyAsync of `bytes` (>= 1 MiB, a multiple
 * of 16) from a pinned host buffer (allocated like hetegen_host_alloc, touched first)
 * to device memory on the context's copy stream, nothing else running in the call;
 * *Bps_out = bytes / median time of `reps` copies after one warm-up copy.  The link
 * figure the streamed path is compared with (Sec. 5, Table 1 lists the platform's
 * CPU-GPU link bandwidth); the planner's V_COM comes from hetegen_probe. */
HETEGEN_API hetegen_status hetegen_probe_link(hetegen_ctx* ctx, size_t bytes, int reps, double* Bps_out);

/* Launch round trip: host time from the launch of an empty kernel (one wavefront) on
 * `stream` to the return of hipStreamSynchronize(stream), median of `reps` >= 1 after
 * ten warm-ups, in microseconds (*us_out).  The fixed cost of a synchronous call on
 * top of the duration of its kernels: the floor of a single small linear's latency,
 * which no kernel work reaches below (hetegen_linear hands x to the host and y back,
 * i.e. one such round trip per direction when it has CPU rows). */
HETEGEN_API hetegen_status hetegen_probe_launch(hetegen_ctx* ctx, int reps, void* stream, double* us_out);

/* The CPU share alone (Sec. 3.2: the host cores compute the rows whose parameters
 * stay in host memory), on the calling thread and the library's CPU worker team (one
 * job at a time; calls from several threads are serialised), no device involved:
 *   y[b * ldy + (j - r0)] = sum_k x[b * K + k] * W[j * K + k] + bias[j],
 *   j in [r0, r1), b < B,
 * x binary32 [B, K] host, W [N, K] host (pinned or pageable), bias host [N] or NULL,
 * y binary32 host.  Binary32 accumulation, 16-bit weights widened exactly (with bf16
 * weights and every x value a bf16 value, on AVX512-BF16 hosts: bf16 pair products, exact,
 * added to binary32 lanes; bf16 subnormals count as zero there).
 * threads <= 0: the OpenMP default thread count.  B in [1, 8], K % 8 == 0, 0 <= r0 <= r1. */
HETEGEN_API hetegen_status hetegen_cpu_linear(const float* x, int B, int K, const void* W_host, hetegen_dtype dtype,
                                              const void* bias_host, int r0, int r1, float* y, int ldy, int threads);

/* ---- Alpha benchmark (Sec. 4.4, Eq. 10-12) ----
 * The closed form assumes speeds proportional to bytes; measured CPU and transfer
 * times are not (contention for host memory, per-call overheads).  The alpha
 * benchmark varies the CPU fraction over [alpha0 - gamma, alpha0 + gamma] in steps
 * of lambda, measures at each point the CPU-share time and the GPU-side time
 * (chunk transfers plus GEMV launches, Eq. 2's T_COM + T_GPU) of one heterogeneous
 * linear, fits least-squares polynomials F_CPU and F_COM of the given degree and
 * returns the CPU fraction where they meet.  When the fitted curves do not cross
 * inside the bracket, the bracket point with the smallest max(F_CPU, F_COM) is
 * returned and *crossed is 0. */

/* Fit-and-solve on given samples (pure host arithmetic): alphas[n], t_cpu[n],
 * t_com[n]; n >= degree + 1, degree in [1, 3], lo < hi. */
HETEGEN_API hetegen_status hetegen_alpha_fit(const double* alphas, const double* t_cpu, const double* t_com, int n,
                                             int degree, double lo, double hi, double* alpha_out, int* crossed);

/* The CPU fraction in [lo, hi] minimising a least-squares polynomial of the given
 * degree fitted to measured times (alphas[n], t[n]); a grid of 10^4 intervals.  Used
 * by the step-level benchmark's wall-time objective. */
HETEGEN_API hetegen_status hetegen_alpha_minimize(const double* alphas, const double* t, int n, int degree, double lo,
                                                  double hi, double* alpha_out);

/* Measure and solve for one linear (arguments as in hetegen_linear, GPU rows always
 * streamed from W_host; y_dev receives the last run's output).  reps runs per point,
 * medians are fitted.  Bracket ends are clamped to [0, 1]. */
HETEGEN_API hetegen_status hetegen_alpha_benchmark(hetegen_ctx* ctx, const void* x_dev, int B, int K, const void* W_host,
                                                   int N, hetegen_dtype dtype, const void* bias_host,
                                                   const void* bias_dev, void* y_dev, double alpha0, double gamma,
                                                   double lambda, int degree, int reps, void* stream,
                                                   double* alpha_out, int* crossed);

/* ---- Heterogeneous module scheduler (Sec. 4.5, Eq. 13) ----
 * Decides which whole modules become GPU-resident when HBM is left over.  Moving
 * module i onto the GPU saves its heterogeneous time t_cpu[i] (seconds, the
 * benchmarked balanced time of Eq. 11) and takes mem[i] bytes of HBM; its gain is
 * g = t_cpu[i] / mem[i].  Modules are visited round robin over the layers
 * (layer[i] >= 0, layers in increasing order): every layer's highest-g module,
 * then every layer's second-highest, and so on, equal gains in index order.  A
 * visited module becomes resident when it fits in what is left of budget_bytes
 * (a sum of doubles in visit order, compared with <=); one that does not fit is
 * skipped and the walk continues.  resident_out[n] receives 1/0; *used_out (may be
 * NULL) the bytes taken.  t_cpu[i] must be finite and >= 0, mem[i] finite and > 0,
 * budget_bytes >= 0 (+inf: no limit).  Pure host arithmetic. */
HETEGEN_API hetegen_status hetegen_module_schedule(const double* t_cpu, const double* mem, const int* layer, int n,
                                                   double budget_bytes, int* resident_out, double* used_out);

/* ---- Decode step over a stack of decoder layers (Sec. 4.2: heterogeneous
 * linears, every other module on the GPU) ----
 *
 * Layer l owns four linears in the order qkv [3H, H], out [H, H], fc1 [F, H],
 * fc2 [H, F]; linear i = 4 l + m.  One step maps x [B, H] to out [B, H]:
 *   h = LN(x); q = qkv(h); a = q[:, 2H:3H]; x = x + out(a);
 *   h = LN(x); f = ReLU(fc1(h)); x = x + fc2(f)
 * with LN a LayerNorm over H without affine terms (eps 1e-5), every
 * intermediate stored in the model's 16-bit type (round to nearest even) and
 * a value-only attention (one position, empty KV cache: the result is V). */

/* W_host[i], bias_host[i]: host weights (pinned, or pageable as for
 * hetegen_linear) and host biases of linear i (caller-owned, must outlive the
 * model).  alpha[i]: CPU fraction of linear i.
 * resident[i] != 0: rows [0, n_gpu) of linear i are copied to HBM at creation;
 * otherwise they are streamed every step.  max_batch in [1, 8]; H, F multiples
 * of 8, H <= 16384 (UNSUPPORTED above: the LayerNorm keeps a row in registers; the
 * largest OPT hidden size is 12288).  Layout of the resident rows: with max_batch
 * 1 they are row-major and run on the vector GEMV (fused LayerNorm, the faster
 * kernels at batch 1); with max_batch >= 2 they are stored in matrix-core tile
 * order and batches of 2 and more run on the matrix-core GEMV (see
 * hetegen_linear_tiled; the model also owns its split-K workspace).  Up to a
 * hidden size of 6144 such a model also keeps the row-major copy, and runs batch 1
 * from it, when both copies take at most half of the device memory free at creation;
 * above 6144 batch 1 runs on the tiles too, which is faster there (the environment
 * variable HETEGEN_DUAL_LAYOUT=0 / 1 at creation: tile order only / the row-major copy
 * too at any hidden size, memory allowing);
 * hetegen_model_layouts tells which copies a model holds.  On the matrix-core path,
 * when out (fc2) and the fc1 (next qkv) after it run every row on the GPU, out / fc2
 * also leave per-16-element LayerNorm partials of their output (sum, sum of squared
 * deviations), and fc1 / qkv normalise their input from them instead of after a
 * LayerNorm launch (Chan-Golub-LeVeque combination in a fixed order), when H <= 6144:
 * for larger hidden sizes combining the H / 16 partials costs more than the launch (the
 * variable HETEGEN_LN_PARTIALS=0 or 1 at creation forces the launches or the partials).
 * A tiled linear whose matrix-core grid puts the same number of workgroups, 1 to 4, on
 * every compute unit keeps its tiles k-major (k-tile kt of row tile rt at tile kt *
 * ceil(n_gpu / 16) + rt), so that workgroups walking K side by side read one contiguous
 * window; the others keep hetegen_tile_weights' order (HETEGEN_TILE_KORDER=0 or 1 at
 * creation: one order for every linear).  The row-major copy of a GPU-only linear with
 * K >= 8192 and K a multiple of 2048 is stored segment-major (2048-element segment s of
 * row r at (s * n_gpu + r) * 2048 elements), which batch-1 wavefronts walking rows side
 * by side read as one window (HETEGEN_SEGMAJOR=0 at creation: plain row-major).  Neither
 * order changes the bits.  Results do not depend on the layout or the LayerNorm path
 * beyond rounding (all pass the oracle's tolerance). */
HETEGEN_API hetegen_status hetegen_model_create(hetegen_ctx* ctx, int L, int H, int F, hetegen_dtype dtype,
                                    void* const* W_host, void* const* bias_host, const double* alpha,
                                    const int* resident, int max_batch, hetegen_model** out);

/* Replace the CPU fractions of the non-resident linears (alpha[i] ignored for a
 * resident linear; its split is fixed at creation). */
HETEGEN_API hetegen_status hetegen_model_set_alpha(hetegen_model* model, const double* alpha);

/* One decode step: out_dev [B, H] = step(x_dev [B, H]); both device, model dtype,
 * 16-byte aligned; out_dev may not alias x_dev.  GPU work is enqueued on `stream`;
 * the call returns after the last CPU share.  When every linear is GPU-only and
 * resident, the step can instead be replayed from a HIP graph captured once per
 * (B, x_dev, out_dev, stream) or run as one persistent kernel (HETEGEN_EXEC_*). */
HETEGEN_API hetegen_status hetegen_decode_step(hetegen_ctx* ctx, hetegen_model* model, const void* x_dev,
                                   void* out_dev, int B, void* stream);

/* How hetegen_decode_step runs a step whose linears are all GPU-only and resident:
 *   AUTO        per-linear launches (as EAGER), the fastest mode measured on MI355X
 *   PERSISTENT  one cooperative launch per step: every workgroup takes the same
 *               row block of every linear, grid barriers between linears, the
 *               next linear's weights requested before each barrier
 *   GRAPH       one GEMV launch per linear, captured once into a HIP graph
 *   EAGER       one GEMV launch per linear, launched directly
 * Steps with CPU rows or streamed linears always run eagerly.  All modes give
 * bit-identical results. */
#define HETEGEN_EXEC_AUTO 0
#define HETEGEN_EXEC_PERSISTENT 1
#define HETEGEN_EXEC_GRAPH 2
#define HETEGEN_EXEC_EAGER 3

/* Select the execution mode (UNSUPPORTED when a forced mode cannot run this
 * model; PERSISTENT needs the row-major copy of the resident rows and runs batch
 * 1 only).  barrier_spin_limit bounds the polls of one grid-barrier wait in the
 * persistent mode (0: the default, seconds of waiting); a wait that gives up lets
 * the step finish with undefined outputs and makes the next hetegen_decode_step
 * on the model fail with HETEGEN_ERR_HIP.  A small limit exists to test that path. */
HETEGEN_API hetegen_status hetegen_model_set_exec(hetegen_model* model, int mode, uint32_t barrier_spin_limit);

/* Mode the last hetegen_decode_step on the model used (HETEGEN_EXEC_*), or -1. */
HETEGEN_API int hetegen_model_last_exec(const hetegen_model* model);

/* Layouts of the model's resident rows (see hetegen_model_create): a bitwise OR of
 * HETEGEN_LAYOUT_ROWMAJOR, HETEGEN_LAYOUT_TILED, HETEGEN_LAYOUT_KMAJOR (some tiled linear
 * keeps its tiles k-major) and HETEGEN_LAYOUT_SEGMAJOR (some row-major copy is stored
 * segment-major), 0 for NULL or no resident rows kept in either. */
#define HETEGEN_LAYOUT_ROWMAJOR 1
#define HETEGEN_LAYOUT_TILED 2
#define HETEGEN_LAYOUT_KMAJOR 4
#define HETEGEN_LAYOUT_SEGMAJOR 8
HETEGEN_API int hetegen_model_layouts(const hetegen_model* model);

/* Alpha benchmark at the granularity of the decode step (Sec. 4.4 applied to the
 * chain of modules).  The call shifts the CPU fraction of every streamed linear by
 * a common offset delta in [-gamma, gamma] (steps of lambda; each fraction clamped
 * to [0, 1]) and times steps on x_dev -> out_dev at every point.
 *   HETEGEN_BENCH_CROSSING: the paper's objective on step totals: fits F_CPU(delta)
 *     (CPU-share time) and F_COM(delta) (transfers plus GEMVs) from profiled steps
 *     and solves for their crossing (as hetegen_alpha_fit);
 *   HETEGEN_BENCH_WALL: fits the steps' wall time and takes its minimiser (as
 *     hetegen_alpha_minimize).  Within a step the ring lets transfers run ahead
 *     across linears and the hand-offs and host-memory contention are not in either
 *     summed time, so the wall-time objective is the one that tracks latency.
 * When the solution is a bracket end (no crossing inside, or the time still falls
 * at the end), the bracket is re-centred on it and measured again: at most three
 * brackets in all.  reps timed steps per point (plus one warm-up).  The model keeps
 * the refined fractions; *delta_out receives the total offset; *crossed is set for
 * the crossing objective.  Resident linears are unchanged. */
#define HETEGEN_BENCH_CROSSING 0
#define HETEGEN_BENCH_WALL 1
HETEGEN_API hetegen_status hetegen_model_alpha_benchmark(hetegen_ctx* ctx, hetegen_model* model, const void* x_dev,
                                                         void* out_dev, int B, double gamma, double lambda,
                                                         int degree, int reps, int objective, void* stream,
                                                         double* delta_out, int* crossed);

/* Read ceiling of the model's resident GPU rows: the rows [0, n_gpu) of every
 * resident linear (its device copy, n_gpu * K elements) read in step order by the
 * streaming read kernel of hetegen_probe_hbm, one launch per linear, on `stream`
 * (a hipStream_t; NULL = the context's own stream).  *ms_out = median wall time of
 * `reps` (>= 1) such passes after one warm-up pass.  A decode step over the same
 * resident linears reads at least these bytes in at least these launches, so this
 * bounds its time from below (launch ramp and drain included).  INVALID_ARG when
 * the model has no resident GPU rows. */
HETEGEN_API hetegen_status hetegen_model_read_ms(hetegen_ctx* ctx, const hetegen_model* model, int reps,
                                                 void* stream, double* ms_out);

/* Current CPU fraction of every linear (4L entries). */
HETEGEN_API hetegen_status hetegen_model_get_alpha(const hetegen_model* model, double* alpha_out);

/* Host milliseconds each linear (4L entries) took in the last step that ran linear
 * by linear (HETEGEN_EXEC_EAGER, or any step with CPU rows or streamed rows): from
 * the start of its enqueue to the end of its CPU share and the enqueue of its
 * return, i.e. its share of the calling thread's critical path.  The module
 * scheduler's benchmarked heterogeneous time (Sec. 4.5) when every linear is
 * heterogeneous.  Zeros before such a step. */
HETEGEN_API hetegen_status hetegen_model_linear_ms(const hetegen_model* model, double* ms_out);

/* ---- KV cache and attention over it (Sec. 2.1, Eq. 1) ----
 * hetegen_decode_step uses the attention of an empty cache (the value slice).
 * With a KV cache the model runs full decode steps: at position pos each layer's
 * attention appends the new token's key and value (qkv[:, H:2H], qkv[:, 2H:3H])
 * to the cache at pos and attends its query qkv[:, 0:H] to positions [0, pos]:
 *   per head h (head_dim D, H / D heads): s_j = q_h . K_j,h / sqrt(D),
 *   a_h = sum_j softmax(s)_j V_j,h, rounded to the model dtype (RNE);
 * a [B, H] then feeds the out linear.  Softmax in binary32 with exact max
 * subtraction; every sequence of the batch is at the same position. */

/* Give the model a cache of max_seq positions, 1 <= max_seq <= 16384 (device
 * memory: 2 * L * max_batch * max_seq * H * 2 bytes, zeroed) and the attention's
 * scratch.  head_dim: 64 or 128, dividing H.  Once per model. */
HETEGEN_API hetegen_status hetegen_model_kv_create(hetegen_ctx* ctx, hetegen_model* model, int max_seq, int head_dim);

/* Copy positions [pos0, pos0 + n) of layer `layer` for sequences [0, B) between the
 * cache and device buffers k_dev, v_dev of layout [B, n, H] (model dtype, one row per
 * token, heads concatenated as in the qkv output); enqueued on `stream`.  Writing
 * stands in for a prefill; reading is for inspection. */
HETEGEN_API hetegen_status hetegen_model_kv_write(hetegen_ctx* ctx, hetegen_model* model, int layer, int B, int pos0,
                                                  int n, const void* k_dev, const void* v_dev, void* stream);
HETEGEN_API hetegen_status hetegen_model_kv_read(hetegen_ctx* ctx, hetegen_model* model, int layer, int B, int pos0,
                                                 int n, void* k_dev, void* v_dev, void* stream);

/* One full decode step of the token at position pos (0 <= pos < max_seq; the cache
 * holds positions [0, pos) of every layer): as hetegen_decode_step with the
 * attention above; runs linear by linear (HETEGEN_EXEC_EAGER).  Heterogeneous and
 * streamed linears work as in hetegen_decode_step. */
HETEGEN_API hetegen_status hetegen_decode_step_kv(hetegen_ctx* ctx, hetegen_model* model, const void* x_dev,
                                                  void* out_dev, int B, int pos, void* stream);

/* Optional trace of every linear's input and output (model dtype), for
 * teacher-forced checks.  Linear i writes its input [B, K_i] and then its output
 * [B, N_i] (after the fused ReLU or residual sum), packed in order of i; the
 * required size for batch B is hetegen_model_trace_bytes().  trace_dev == NULL
 * turns tracing off.  Tracing disables the graph replay. */
HETEGEN_API size_t hetegen_model_trace_bytes(const hetegen_model* model, int B);
HETEGEN_API hetegen_status hetegen_model_set_trace(hetegen_model* model, void* trace_dev, size_t bytes);

HETEGEN_API hetegen_status hetegen_model_destroy(hetegen_ctx* ctx, hetegen_model* model);

/* ---- Per-resource busy times (the Table 2 breakdown) ---- */

typedef struct {
  double wall_ms;      /* host wall time inside hetegen_linear / hetegen_decode_step */
  double cpu_ms;       /* host time computing CPU shares */
  double h2d_ms;       /* copy-stream time moving streamed weight chunks */
  double gpu_ms;       /* GPU GEMV kernel time (events around each launch) */
  double h2d_bytes;    /* weight bytes streamed */
  double gpu_bytes;    /* weight bytes read by GPU GEMV launches */
  double cpu_bytes;    /* weight bytes read by CPU shares */
  int64_t gemv_launches;
  double pin_ms;       /* host time the pin team spent staging pageable chunks */
  double pin_bytes;    /* bytes staged */
  double xwait_ms;     /* host time waiting, before a CPU share, for its input to reach host memory
                          (the GPU work ahead of it in stream order, then the hand-off) */
  double tailwait_ms;  /* host time waiting, after a CPU share, to enqueue the GEMVs of the linear's
                          remaining chunks (their copies not yet issued: the link is behind) */
  int64_t cpu_shares;  /* linears computed with CPU rows */
  double hetlin_ms;    /* host time inside those linears (CPU share, the waits above, and enqueueing
                          their kernels and chunk GEMVs) */
  double res_gpu_ms;   /* the part of gpu_ms spent on HBM-resident rows (not streamed chunks) */
  double res_gpu_bytes; /* the weight bytes of those launches */
} hetegen_profile;

/* on != 0: bracket every chunk copy and GEMV launch with events and synchronise at
 * the end of each call to accumulate the times (adds overhead; for measurement). */
HETEGEN_API hetegen_status hetegen_set_profiling(hetegen_ctx* ctx, int on);
HETEGEN_API hetegen_status hetegen_get_profile(hetegen_ctx* ctx, hetegen_profile* out, int reset);

#ifdef __cplusplus
}
#endif

#endif /* HETEGEN_H */
