// Internal launch interface of the gfx950 kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace hg {

enum Epi : int { EPI_NONE = 0, EPI_RELU = 1, EPI_RESID = 2 };

// y[b, r] = epi(sum_k xn[b, k] * W[r, k] + bias[r]) for b < B, r < rows, where xn is
// x, or LayerNorm(x) rounded to the activation type when ln != 0.
struct GemvParams {
  const void* x;       // [B, K] activation type, row stride ldx elements, 16-byte aligned
  long long ldx;
  const void* W;       // [rows, K] row-major, 16-byte aligned
  const void* bias;    // [rows] activation type, or nullptr
  void* y;             // element (b, r) at y[b * ldy + r]
  long long ldy;
  const void* resid;   // EPI_RESID: element (b, r) at resid[b * ldr + r]
  long long ldr;
  void* h_out;         // ln != 0 and non-null: block 0 also writes LayerNorm(x) here
  long long ldh;
  int rows;
  int K;
  int epi;
  int y_f32;           // 1: y is float32, 0: y is the activation type
  int ln;
  int ktile;           // set by the launcher: K elements staged in LDS per pass (tiled kernel)
  int rpw;             // set by the launcher: rows per workgroup (contiguous block)
  // matrix-core GEMV on tile-ordered weights (launch_gemv_mfma) only:
  float* ws;           // split-K partials: at least mfma_ws_floats(rows, K, B) floats
  uint32_t* cnt;       // split-K arrival counters: at least mfma_cnt_words(rows, K) words, zero between launches
  size_t ws_floats;    // floats at ws and words at cnt (checked by the launcher)
  size_t cnt_words;
  int korder;          // W's tile order (launch_tile's korder: 0 row-tile order, 1 k-major)
  int segmajor;        // W segment-major (launch_segmajor): gemv_x1_kernel and the persistent step only
  const float* ln_in;  // ln != 0: LayerNorm partials of x (ln_partials_floats(K)), written by the
                       // launch that produced x through ln_out
  float* ln_out;       // or nullptr: LayerNorm partials of y (y in the activation type)
};

// One linear of the persistent decode step (a device-resident table entry).
// x_in / resid_in / y_out select the step's input or output pointer instead of
// the buffer stored here.
struct StepLinear {
  const void* W;
  const void* bias;
  const void* x;
  long long ldx;
  void* y;
  long long ldy;
  const void* resid;
  long long ldr;
  int rows, K, epi, ln, rpw;
  int x_in, resid_in, y_out;
  int segmajor;  // W segment-major (launch_segmajor)
};

struct StepArgs {
  const StepLinear* lin;  // device table of nlin entries
  int nlin;
  const void* x_in;
  void* out;
  uint32_t* counters;     // barrier counters: ngroups + 1 words, 256 bytes apart, zeroed at creation
  uint32_t barrier_base;  // barriers completed by earlier steps on these counters
  int ngroups;
  int* err;               // set to 1 (system scope) if a barrier wait gave up
  uint32_t spin_limit;    // polls before a barrier wait gives up
};

// Rows handed to one wavefront at a time by the GEMV for batch B; a workgroup's
// row block is a multiple of 4x this.
int gemv_rows_unit(int B);

// Dynamic LDS of the main GEMV for batch B, reduction K and rows_per_block rows.
size_t gemv_lds_bytes(int B, int K, int rows_per_block);

// Largest LDS the persistent step accepts per workgroup (the per-linear main GEMV may
// use up to the device's LDS per workgroup, less 1 KiB, before it switches to the
// K-tiled kernel).
size_t gemv_lds_limit();

// Whether a resident eager GEMV at batch B normalises its input itself (GemvParams.ln)
// rather than after a separate LayerNorm launch; both give the same bits.
bool gemv_fuses_ln(int B);

// Co-resident workgroups of the persistent step kernel per CU (0 if unsupported).
int step_blocks_per_cu(int dtype, int B, size_t lds);

// Cooperative launch of the persistent step (grid must be co-resident).
hipError_t launch_step(const StepArgs& a, int dtype, int B, int grid, size_t lds, hipStream_t stream);

// dtype: 0 = fp16, 1 = bf16.  grid_cap bounds the number of workgroups
// (0 = default).  Returns the launch status.
hipError_t launch_gemv(GemvParams p, int dtype, int B, hipStream_t stream, int grid_cap);

// Segment-major layout of a row-major weight [rows, K] (K a multiple of kSegElems): the
// kSegElems-element segment s of row r is stored at (s * rows + r) * kSegElems elements, so
// that wavefronts walking rows side by side read one contiguous window.
constexpr int kSegElems = 2048;
// dst = segment-major copy of row-major W [rows, K] (16-byte aligned, not overlapping).
hipError_t launch_segmajor(const void* W, int rows, int K, void* dst, hipStream_t stream);

// Largest LayerNorm width (hidden size) the kernels support.
constexpr int kMaxLnK = 16384;

// h[b, :] = act(LayerNorm(x[b, :])) for b < B (device), and optionally
// h_host_f32[b * K + k] = float(h[b, k]) (pinned host memory).  K <= kMaxLnK.
hipError_t launch_layernorm(const void* x, long long ldx, int B, int K, int dtype, void* h, long long ldh,
                            float* h_host_f32, hipStream_t stream);

// dst_host_f32[b * K + k] = float(x[b * ldx + k])  (device -> pinned host, in a kernel).
hipError_t launch_export_f32(const void* x, long long ldx, int B, int K, int dtype, float* dst_host_f32,
                             hipStream_t stream);

// y[b * ldy + c] = epi(src_host_f32[b * n + c]) for c < n, b < B: the CPU rows' sums
// (bias included) read from pinned host memory, finished like the GPU rows.
hipError_t launch_import_rows(const float* src_host_f32, int B, int n, int dtype, int epi, void* y,
                              long long ldy, int y_f32, const void* resid, long long ldr, hipStream_t stream);

// ---- matrix-core GEMV on tile-ordered weights ----
// A weight block [rows, K] in tile order is a sequence of 1 KiB tiles of 16 rows x 32
// columns, row tile by row tile (all k-tiles of rows [16 rt, 16 rt + 16) are contiguous);
// within a tile, the 16 bytes at 16 * l hold W[16 rt + l % 16][32 kt + 8 (l / 16) + e],
// e < 8: the operand layout of one 16x16x32 matrix-core instruction, so one load per
// lane reads the whole tile.  Rows past `rows` and columns past K are zero.
size_t tiled_bytes(int rows, int K);

// dst = tile order of W [rows, K] (row stride ldw elements, 16-byte aligned rows).
// korder 1: k-major tile order instead, k-tile kt of row tile rt at tile kt * ceil(rows / 16) + rt.
hipError_t launch_tile(const void* W, long long ldw, int rows, int K, void* dst, hipStream_t stream, int korder = 0);

// K-splits of the matrix-core GEMV for `rows` rows and reduction length K on the current
// device (1 = no split; it depends on the device's compute-unit count, not on the batch),
// and the workspace a launch at batch B needs (0 when not split).
int mfma_splits(int rows, int K);
// Tile order for a model's copy of W [rows, K] on the current device: 1 k-major, 0 row-tile
// order (1 when the launch grid puts the same number of workgroups, at most 4, on every CU).
int mfma_kmajor(int rows, int K);
size_t mfma_ws_floats(int rows, int K, int B);
size_t mfma_cnt_words(int rows, int K);

// LayerNorm partials of a [B, n] activation: for every 16-element group q of a row and
// batch row b < 8, the pair (sum of the group's values, sum of their squared deviations
// from the group's mean) at floats 2 (8 q + b) and 2 (8 q + b) + 1 (the last group may
// hold 8 elements).  A LayerNorm of the row combines them in a fixed order.
size_t ln_partials_floats(int n);

// y = epi(xn W^T + bias) with W in tile order (p.W), every row on the GPU, where xn is x,
// or, when p.ln != 0, LayerNorm(x) from the partials p.ln_in (h_out, if set, receives xn
// from workgroup 0).  With p.ln_out set the launch also writes the partials of y (p.y_f32
// must be 0).  Split launches need p.ws and p.cnt with their sizes in p.ws_floats and
// p.cnt_words (hipErrorInvalidValue if too small).
hipError_t launch_gemv_mfma(GemvParams p, int dtype, int B, hipStream_t stream);

// Fixed split-K scratch of the matrix-core GEMV, one per GPU, for callers that cannot
// allocate: kScratchCounterWords counters, then kScratchFloats floats of partials.
constexpr size_t kScratchCounterWords = 65536;
constexpr size_t kScratchFloats = (size_t)1 << 18;
// Takes the scratch's address on `device` (which must be current) and zeroes its counters,
// once per device; later calls return at once.
hipError_t scratch_init(int device);
// The scratch's device address on `device` (nullptr before scratch_init).
void* scratch_ptr(int device);

}  // namespace hg
