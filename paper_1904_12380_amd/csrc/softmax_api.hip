// C ABI of the row-softmax library: argument checks, the dispatch on cols,
// and the launches.  Declarations and the contract are in
// include/softmax_mi355x.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>
#include <utility>
#include <vector>

#include "../../include/softmax_mi355x.h"
#include "sm_host.hpp"
#include "sm_kernels.hpp"

namespace {

using namespace smx;
using namespace smx_host;

// Bucket limits on cols.
constexpr int64_t kPackedMaxCols = 64;

// The packed kernel's persistent grid: six 256-thread workgroups per CU on
// MI355X's 256 CUs.  Measured on 115200 x 50: up to six per CU the
// prefetched next tile overlaps the current tile's compute (8.6 us); seven
// or more per CU, or one tile per workgroup, take 10.4-11.2 us.
constexpr int64_t kPackedBlocksPerCU = 6;
constexpr int64_t kDeviceCUs = 256;
constexpr int64_t kWaveRowMaxCols = 4096;
// With 32-bit access, 64 values per lane need more registers than a
// wavefront has (the kernel would spill): such rows go to k_block_row.
constexpr int64_t kWaveRowMaxColsScalar = 2048;
constexpr int64_t kBlockRowMaxCols = 32768;

// Split rows, one-pass kernel: 512-thread workgroups holding 32 columns per
// lane (chunks of 16384 columns, eight waves per SIMD) for rows of up to
// 64 chunks, or 64 columns per lane (chunks of 32768, four waves per SIMD)
// for rows of up to 64 of those.  On 64 x 262144 the 16384-column chunks
// take 22.8 us against 24.6 us for 32768-column ones.
constexpr int kOnePassThreads = 512;
constexpr int kOnePassVSmall = 8;
constexpr int kOnePassVLarge = 16;
constexpr int64_t kOnePassChunkSmall = int64_t(4) * kOnePassVSmall * kOnePassThreads;
constexpr int64_t kOnePassChunkLarge = int64_t(4) * kOnePassVLarge * kOnePassThreads;
// A row may span at most this many workgroups on the one-pass path (the
// exchange is read by one wavefront, one slot per lane).
constexpr int64_t kOnePassMaxChunks = 64;
// Rows per launch keep a launch within the workgroups MI355X's 256 CUs hold
// at once: four per CU with the small chunks, two with the large ones.
constexpr int64_t kOnePassMaxBlocksSmall = 1024;
constexpr int64_t kOnePassMaxBlocksLarge = 512;
constexpr int64_t kOnePassMaxBlocks = kOnePassMaxBlocksSmall;
// NLL outputs on the one-pass path: 1024-thread workgroups, two per CU.
constexpr int kNllThreads = 1024;
constexpr int64_t kNllChunk = int64_t(4) * kOnePassVSmall * kNllThreads;
constexpr int64_t kNllMaxBlocks = 512;
static_assert(kNllMaxBlocks <= kOnePassMaxBlocks, "NLL launches fit the exchange slots");

// Split rows, two-pass fallback for rows longer than kOnePassMaxChunks
// chunks: 512-thread workgroups holding 32 columns per lane (chunks of
// 16384 columns).
constexpr int kSplitThreads = 512;
constexpr int kSplitV = 8;
constexpr int64_t kSplitChunk = int64_t(4) * kSplitV * kSplitThreads;

// Library-owned workspace for split rows, one per (device, stream) for
// eager calls (launches that may overlap in time never share one) and one
// per device shared by captured graphs:
//   [0, 128 KiB)          two-pass partials, float2
//   [128 KiB, +8 KiB)     one-pass exchange slots, 64-bit, kSlotEmpty at rest
//   [136 KiB, +4 KiB)     one-pass departure counters, zero at rest
constexpr int64_t kWorkspaceBytes = int64_t(140) << 10;
constexpr int64_t kWorkspacePairs = (int64_t(128) << 10) / int64_t(sizeof(float2));
constexpr int64_t kSlotsOffset = int64_t(128) << 10;
constexpr int64_t kSlotsBytes = kOnePassMaxBlocks * 8;
constexpr int64_t kDepartOffset = kSlotsOffset + kSlotsBytes;
constexpr int64_t kDepartBytes = kOnePassMaxBlocks * 4;
static_assert(kDepartOffset + kDepartBytes <= kWorkspaceBytes, "workspace layout fits");
constexpr int kMaxDevices = 64;
constexpr int kMaxStreamWorkspaces = 64;  // per device

struct StreamWorkspace {
  hipStream_t stream;
  char* mem;
  uint64_t last_use;
};
struct DeviceState {
  std::vector<StreamWorkspace> per_stream;
  char* capture_ws = nullptr;
  uint64_t clock = 0;
};
std::mutex g_mu;
DeviceState g_dev[kMaxDevices];

inline int64_t pow2_at_least(int64_t v) {
  int64_t p = 1;
  while (p < v) p <<= 1;
  return p;
}

// rows*cols*4 must fit in int64 and both counts must be non-negative.
int check_sizes(int64_t rows, int64_t cols) {
  if (rows < 0 || cols < 0) return SOFTMAX_ERR_INVALID_ARG;
  if (rows == 0 || cols == 0) return SOFTMAX_OK;
  if (rows > INT64_MAX / 4 / cols) return SOFTMAX_ERR_INVALID_ARG;
  return SOFTMAX_OK;
}

softmax_plan_t make_plan(const float* x, const float* y, int64_t rows, int64_t cols) {
  softmax_plan_t p{};
  p.chunks_per_row = 1;
  if (rows == 0 || cols == 0) {
    p.kernel = SOFTMAX_KERNEL_NONE;
    return p;
  }
  const bool a16 = aligned16(x) && aligned16(y);
  const bool vec_rows = a16 && (cols % 4 == 0);
  if (cols <= kPackedMaxCols) {
    // G lanes per row with at most 16 columns per lane; a persistent grid of
    // kPackedBlocksPerCU workgroups per CU loops over tiles of 256/G rows.
    const int64_t g = cols <= 16 ? 1 : cols <= 32 ? 2 : 4;
    p.kernel = SOFTMAX_KERNEL_PACKED;
    p.vec_width = a16 ? 4 : 1;
    p.lanes_per_row = static_cast<int32_t>(g);
    p.elems_per_lane = static_cast<int32_t>(ceil_div(cols, g));
    p.block_threads = 256;
    const int64_t tile = 256 / g;
    p.grid = std::min(ceil_div(rows, tile), kPackedBlocksPerCU * kDeviceCUs);
    p.launches = 1;
  } else if (cols <= (vec_rows ? kWaveRowMaxCols : kWaveRowMaxColsScalar)) {
    const int64_t v = pow2_at_least(ceil_div(cols, 256));
    p.kernel = SOFTMAX_KERNEL_WAVE_ROW;
    p.vec_width = vec_rows ? 4 : 1;
    p.lanes_per_row = 64;
    p.elems_per_lane = static_cast<int32_t>(4 * v);
    p.block_threads = 256;
    p.grid = std::min(ceil_div(rows, 4), kMaxGrid);
    p.launches = 1;
  } else if (cols <= kBlockRowMaxCols) {
    const int64_t v = std::max<int64_t>(2, pow2_at_least(ceil_div(cols, 4096)));
    p.kernel = SOFTMAX_KERNEL_BLOCK_ROW;
    p.vec_width = vec_rows ? 4 : 1;
    p.lanes_per_row = 1024;
    p.elems_per_lane = static_cast<int32_t>(4 * v);
    p.block_threads = 1024;
    p.grid = std::min(rows, kMaxGrid);
    p.launches = 1;
  } else {
    p.kernel = SOFTMAX_KERNEL_SPLIT_ROW;
    p.vec_width = vec_rows ? 4 : 1;
    p.workspace_bytes = kWorkspaceBytes;
    const int64_t gs = ceil_div(cols, kOnePassChunkSmall);
    const int64_t gl = ceil_div(cols, kOnePassChunkLarge);
    // The large chunks (64 values per lane) are taken with 128-bit access
    // only: with 32-bit access they would spill, and such rows take the
    // two-pass path instead.
    if (gs <= kOnePassMaxChunks || (vec_rows && gl <= kOnePassMaxChunks)) {
      // One pass: whole rows per launch, all workgroups resident together.
      const bool small = gs <= kOnePassMaxChunks;
      const int64_t g1 = small ? gs : gl;
      const int64_t rows_per_launch =
          (small ? kOnePassMaxBlocksSmall : kOnePassMaxBlocksLarge) / g1;
      p.lanes_per_row = kOnePassThreads;
      p.elems_per_lane = 4 * (small ? kOnePassVSmall : kOnePassVLarge);
      p.block_threads = kOnePassThreads;
      p.chunks_per_row = g1;
      p.grid = std::min(rows, rows_per_launch) * g1;
      p.launches = static_cast<int32_t>(ceil_div(rows, rows_per_launch));
    } else {
      // Two passes: partials, then merge and write, in batches of rows.
      const int64_t g2 = ceil_div(cols, kSplitChunk);
      const int64_t rows_per_batch = std::max<int64_t>(1, kWorkspacePairs / g2);
      p.lanes_per_row = kSplitThreads;
      p.elems_per_lane = 4 * kSplitV;
      p.block_threads = kSplitThreads;
      p.chunks_per_row = g2;
      p.grid = std::min(std::min(rows, rows_per_batch) * g2, kMaxGrid);
      p.launches = static_cast<int32_t>(2 * ceil_div(rows, rows_per_batch));
    }
  }
  return p;
}

// k_packed instances: G = 1 with EPL = 1..16, G = 2 and G = 4 with
// EPL = 9..16 (a plan never asks for fewer columns per lane at G > 1).
template <int G, bool VEC4, int EM, int... E>
const void* packed_fn(int epl, std::integer_sequence<int, E...>) {
  static const void* const table[] = {
      reinterpret_cast<const void*>(&k_packed<G, (G == 1 ? 1 : 9) + E, VEC4, EM>)...};
  const int idx = epl - (G == 1 ? 1 : 9);
  return (idx >= 0 && idx < static_cast<int>(sizeof...(E))) ? table[idx] : nullptr;
}

template <bool VEC4, int EM>
hipError_t dispatch_packed(const softmax_plan_t& p, const float* x, float* y,
                           const int64_t* labels, int64_t rows, int64_t cols, Clip c,
                           hipStream_t s) {
  const void* fn = nullptr;
  switch (p.lanes_per_row) {
    case 1:
      fn = packed_fn<1, VEC4, EM>(p.elems_per_lane, std::make_integer_sequence<int, 16>{});
      break;
    case 2:
      fn = packed_fn<2, VEC4, EM>(p.elems_per_lane, std::make_integer_sequence<int, 8>{});
      break;
    default:
      fn = packed_fn<4, VEC4, EM>(p.elems_per_lane, std::make_integer_sequence<int, 8>{});
      break;
  }
  if (fn == nullptr) return hipErrorInvalidValue;
  void* args[] = {&x, &y, &labels, &rows, &cols, &c};
  return launch(fn, p.grid, 256, args, s);
}

template <int V, bool VEC4, int EM>
hipError_t run_wave(const float* x, float* y, const int64_t* labels, int64_t rows,
                    int64_t cols, Clip c, int64_t grid, hipStream_t s) {
  void* args[] = {&x, &y, &labels, &rows, &cols, &c};
  return launch(reinterpret_cast<const void*>(&k_wave_row<V, VEC4, EM>), grid, 256, args,
                s);
}

template <bool VEC4, int EM>
hipError_t dispatch_wave(const softmax_plan_t& p, const float* x, float* y,
                         const int64_t* labels, int64_t rows, int64_t cols, Clip c,
                         hipStream_t s) {
  switch (p.elems_per_lane / 4) {
    case 1: return run_wave<1, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    case 2: return run_wave<2, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    case 4: return run_wave<4, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    case 8: return run_wave<8, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    default:
      // 64 values per lane only with 128-bit access (see make_plan).
      if constexpr (VEC4) return run_wave<16, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
      return hipErrorInvalidValue;
  }
}

template <int V, bool VEC4, int EM>
hipError_t run_block(const float* x, float* y, const int64_t* labels, int64_t rows,
                     int64_t cols, Clip c, int64_t grid, hipStream_t s) {
  void* args[] = {&x, &y, &labels, &rows, &cols, &c};
  return launch(reinterpret_cast<const void*>(&k_block_row<1024, V, VEC4, EM>), grid, 1024,
                args, s);
}

template <bool VEC4, int EM>
hipError_t dispatch_block(const softmax_plan_t& p, const float* x, float* y,
                          const int64_t* labels, int64_t rows, int64_t cols, Clip c,
                          hipStream_t s) {
  switch (p.elems_per_lane / 4) {
    case 2: return run_block<2, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    case 4: return run_block<4, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
    default: return run_block<8, VEC4, EM>(x, y, labels, rows, cols, c, p.grid, s);
  }
}

// The output and labels of rows r0.. of a call: y advances by a row of
// outputs, or by one loss per row for NLL outputs (whose labels advance
// with it).
template <int EM>
float* out_rows(float* y, int64_t r0, int64_t cols) {
  return EM == kNllOut ? y + r0 : y + r0 * cols;
}
template <int EM>
const int64_t* label_rows(const int64_t* labels, int64_t r0) {
  return EM == kNllOut ? labels + r0 : labels;
}

template <bool VEC4, int EM>
hipError_t run_split(const float* x, float* y, const int64_t* labels, float2* ws,
                     int64_t rows, int64_t cols, int64_t chunks, Clip c, hipStream_t s) {
  const int64_t rows_per_batch = std::max<int64_t>(1, kWorkspacePairs / chunks);
  for (int64_t r0 = 0; r0 < rows; r0 += rows_per_batch) {
    int64_t nb = std::min(rows_per_batch, rows - r0);
    const float* xb = x + r0 * cols;
    float* yb = out_rows<EM>(y, r0, cols);
    const int64_t* lb = label_rows<EM>(labels, r0);
    const int64_t grid = std::min(nb * chunks, kMaxGrid);
    void* a1[] = {&xb, &ws, &nb, &cols, &chunks, &c};
    hipError_t e = launch(
        reinterpret_cast<const void*>(&k_split_stats<kSplitThreads, kSplitV, VEC4, EM>),
        grid, kSplitThreads, a1, s);
    if (e != hipSuccess) return e;
    const float2* wsc = ws;
    void* a2[] = {&xb, &yb, &lb, &wsc, &nb, &cols, &chunks, &c};
    e = launch(
        reinterpret_cast<const void*>(&k_split_apply<kSplitThreads, kSplitV, VEC4, EM>),
        grid, kSplitThreads, a2, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int V, bool VEC4, int EM, int NT = kOnePassThreads>
hipError_t run_onepass(const float* x, float* y, const int64_t* labels, char* ws,
                       int64_t rows, int64_t cols, int64_t chunks, int64_t max_blocks, Clip c,
                       hipStream_t s) {
  unsigned long long* part = reinterpret_cast<unsigned long long*>(ws + kSlotsOffset);
  unsigned* depart = reinterpret_cast<unsigned*>(ws + kDepartOffset);
  const int64_t rows_per_launch = max_blocks / chunks;
  int ichunks = static_cast<int>(chunks);
  for (int64_t r0 = 0; r0 < rows; r0 += rows_per_launch) {
    const int64_t nb = std::min(rows_per_launch, rows - r0);
    const float* xb = x + r0 * cols;
    float* yb = out_rows<EM>(y, r0, cols);
    const int64_t* lb = label_rows<EM>(labels, r0);
    void* args[] = {&xb, &yb, &lb, &part, &depart, &cols, &ichunks, &c};
    hipError_t e = launch(
        reinterpret_cast<const void*>(&k_split_onepass<NT, V, VEC4, EM>), nb * chunks, NT,
        args, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// A workspace in its resting state: exchange slots empty, counters zero.
hipError_t new_workspace(char** out) {
  void* mem = nullptr;
  hipError_t e = hipMalloc(&mem, kWorkspaceBytes);
  if (e != hipSuccess) return e;
  char* ws = static_cast<char*>(mem);
  e = hipMemset(ws, 0, kWorkspaceBytes);
  if (e == hipSuccess) e = hipMemset(ws + kSlotsOffset, 0xFF, kSlotsBytes);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return e;
  }
  *out = ws;
  return hipSuccess;
}

// Workspace for a split-row call on (dev, s).  Eager calls get one per
// stream (allocated on first use); under stream capture the device's shared
// capture workspace is used, which an earlier eager split-row call on the
// device must have created.
int workspace_for(int dev, hipStream_t s, bool capturing, char** out) {
  DeviceState& st = g_dev[dev];
  hipError_t e;
  if (capturing) {
    if (st.capture_ws == nullptr) return SOFTMAX_ERR_INVALID_ARG;
    *out = st.capture_ws;
    return SOFTMAX_OK;
  }
  ++st.clock;
  for (StreamWorkspace& w : st.per_stream) {
    if (w.stream == s) {
      w.last_use = st.clock;
      *out = w.mem;
      return SOFTMAX_OK;
    }
  }
  if (st.capture_ws == nullptr) {
    e = new_workspace(&st.capture_ws);
    if (e != hipSuccess) return fail_hip(e);
  }
  if (static_cast<int>(st.per_stream.size()) >= kMaxStreamWorkspaces) {
    // Recycle the least recently used stream's workspace once the device
    // is idle, so none of that stream's work can still be using it.
    e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail_hip(e);
    StreamWorkspace* lru = &st.per_stream[0];
    for (StreamWorkspace& w : st.per_stream)
      if (w.last_use < lru->last_use) lru = &w;
    lru->stream = s;
    lru->last_use = st.clock;
    *out = lru->mem;
    return SOFTMAX_OK;
  }
  char* mem = nullptr;
  e = new_workspace(&mem);
  if (e != hipSuccess) return fail_hip(e);
  st.per_stream.push_back(StreamWorkspace{s, mem, st.clock});
  *out = mem;
  return SOFTMAX_OK;
}

template <bool VEC4, int EM>
hipError_t split_launch(const softmax_plan_t& p, const float* x, float* y,
                        const int64_t* labels, int64_t rows, int64_t cols, char* ws, Clip c,
                        hipStream_t s) {
  // NLL outputs with 128-bit access take 1024-thread workgroups (chunks of
  // 32768 columns, two per CU): their workgroups never wait for each other,
  // and keep no values, so the wider chunk only saves workgroups (long rows
  // 16.1 -> 14.6 us).  The other modes hold their chunk in registers through
  // the exchange and would spill at that width.
  if constexpr (EM == kNllOut && VEC4) {
    const int64_t gn = ceil_div(cols, kNllChunk);
    if (gn <= kOnePassMaxChunks)
      return run_onepass<kOnePassVSmall, VEC4, EM, kNllThreads>(x, y, labels, ws, rows, cols,
                                                                  gn, kNllMaxBlocks, c, s);
  }
  // Plans with at most kOnePassMaxChunks chunks per row are one-pass (their
  // chunk size is told by elems_per_lane); longer rows are two-pass.
  const int64_t g = p.chunks_per_row;
  if (g <= kOnePassMaxChunks && p.elems_per_lane == 4 * kOnePassVSmall)
    return run_onepass<kOnePassVSmall, VEC4, EM>(x, y, labels, ws, rows, cols, g,
                                                   kOnePassMaxBlocksSmall, c, s);
  if constexpr (VEC4) {
    if (g <= kOnePassMaxChunks)
      return run_onepass<kOnePassVLarge, VEC4, EM>(x, y, labels, ws, rows, cols, g,
                                                     kOnePassMaxBlocksLarge, c, s);
  }
  return run_split<VEC4, EM>(x, y, labels, reinterpret_cast<float2*>(ws), rows, cols, g, c,
                             s);
}

template <int EM>
hipError_t split_mode(const softmax_plan_t& p, const float* x, float* y,
                      const int64_t* labels, int64_t rows, int64_t cols, char* ws, Clip c,
                      hipStream_t s) {
  return p.vec_width == 4 ? split_launch<true, EM>(p, x, y, labels, rows, cols, ws, c, s)
                          : split_launch<false, EM>(p, x, y, labels, rows, cols, ws, c, s);
}

int split_call(const softmax_plan_t& p, const float* x, float* y, const int64_t* labels,
               int64_t rows, int64_t cols, int dev, Clip c, int em, hipStream_t s) {
  if (dev < 0 || dev >= kMaxDevices) return SOFTMAX_ERR_INVALID_ARG;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(s, &cap);
  if (e != hipSuccess) return fail_hip(e);
  char* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    const int rc = workspace_for(dev, s, cap != hipStreamCaptureStatusNone, &ws);
    if (rc != SOFTMAX_OK) return rc;
  }
  switch (em) {
    case kExpWide: e = split_mode<kExpWide>(p, x, y, labels, rows, cols, ws, c, s); break;
    case kExpFast: e = split_mode<kExpFast>(p, x, y, labels, rows, cols, ws, c, s); break;
    case kLogOut: e = split_mode<kLogOut>(p, x, y, labels, rows, cols, ws, c, s); break;
    case kNllOut: e = split_mode<kNllOut>(p, x, y, labels, rows, cols, ws, c, s); break;
    default: e = split_mode<kExpAccurate>(p, x, y, labels, rows, cols, ws, c, s); break;
  }
  return e == hipSuccess ? SOFTMAX_OK : fail_hip(e);
}

template <int EM>
hipError_t launch_rows(const softmax_plan_t& p, const float* x, float* y,
                       const int64_t* labels, int64_t rows, int64_t cols, Clip c,
                       hipStream_t s) {
  switch (p.kernel) {
    case SOFTMAX_KERNEL_PACKED:
      return p.vec_width == 4 ? dispatch_packed<true, EM>(p, x, y, labels, rows, cols, c, s)
                              : dispatch_packed<false, EM>(p, x, y, labels, rows, cols, c, s);
    case SOFTMAX_KERNEL_WAVE_ROW:
      return p.vec_width == 4 ? dispatch_wave<true, EM>(p, x, y, labels, rows, cols, c, s)
                              : dispatch_wave<false, EM>(p, x, y, labels, rows, cols, c, s);
    case SOFTMAX_KERNEL_BLOCK_ROW:
      return p.vec_width == 4 ? dispatch_block<true, EM>(p, x, y, labels, rows, cols, c, s)
                              : dispatch_block<false, EM>(p, x, y, labels, rows, cols, c, s);
    default:
      return hipSuccess;
  }
}

// Every launch of one call in mode em, on a plan made for it.
int launch_mode(const softmax_plan_t& p, const float* x, float* y, const int64_t* labels,
                int64_t rows, int64_t cols, int dev, Clip c, int em, hipStream_t stream) {
  if (p.kernel == SOFTMAX_KERNEL_SPLIT_ROW)
    return split_call(p, x, y, labels, rows, cols, dev, c, em, stream);
  hipError_t e;
  switch (em) {
    case kExpWide: e = launch_rows<kExpWide>(p, x, y, labels, rows, cols, c, stream); break;
    case kExpFast: e = launch_rows<kExpFast>(p, x, y, labels, rows, cols, c, stream); break;
    case kLogOut: e = launch_rows<kLogOut>(p, x, y, labels, rows, cols, c, stream); break;
    case kNllOut: e = launch_rows<kNllOut>(p, x, y, labels, rows, cols, c, stream); break;
    default: e = launch_rows<kExpAccurate>(p, x, y, labels, rows, cols, c, stream); break;
  }
  return e == hipSuccess ? SOFTMAX_OK : fail_hip(e);
}

int check_pointers(const float* x, const float* y, int64_t n_elems, int* dev) {
  const int64_t bytes = n_elems * 4;
  if (x == nullptr || y == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (partial_overlap(x, y, bytes)) return SOFTMAX_ERR_INVALID_ARG;
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return fail_hip(e);
  int rc = check_device_range(x, bytes, *dev);
  if (rc != SOFTMAX_OK) return rc;
  if (y != x) rc = check_device_range(y, bytes, *dev);
  return rc;
}

// The row softmax with kernel mode em (kExpAccurate, kExpWide, kExpFast,
// or kLogOut for log outputs) after the clip and size checks.
int softmax_rows(const float* x, float* y, int64_t rows, int64_t cols, Clip c, int em,
                 hipStream_t stream) {
  int rc = check_sizes(rows, cols);
  if (rc != SOFTMAX_OK) return rc;
  if (rows == 0 || cols == 0) return SOFTMAX_OK;
  int dev = 0;
  rc = check_pointers(x, y, rows * cols, &dev);
  if (rc != SOFTMAX_OK) return rc;
  return launch_mode(make_plan(x, y, rows, cols), x, y, nullptr, rows, cols, dev, c, em,
                     stream);
}

}  // namespace

extern "C" {

SOFTMAX_API int softmax_plan(const float* x, const float* y, int64_t rows, int64_t cols,
                             softmax_plan_t* plan) {
  if (plan == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  const int rc = check_sizes(rows, cols);
  if (rc != SOFTMAX_OK) return rc;
  if (rows > 0 && cols > 0) {
    if (x == nullptr || y == nullptr) return SOFTMAX_ERR_INVALID_ARG;
    if (partial_overlap(x, y, rows * cols * 4)) return SOFTMAX_ERR_INVALID_ARG;
  }
  *plan = make_plan(x, y, rows, cols);
  return SOFTMAX_OK;
}

SOFTMAX_API int softmax_fwd_clip(const float* x, float* y, int64_t rows, int64_t cols,
                                 float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, wide ? kExpWide : kExpAccurate, stream);
}

SOFTMAX_API int softmax_fwd_approx(const float* x, float* y, int64_t rows, int64_t cols,
                                   float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, kExpFast, stream);
}

SOFTMAX_API int softmax_log_fwd(const float* x, float* y, int64_t rows, int64_t cols,
                                float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, kLogOut, stream);
}

SOFTMAX_API int softmax_nll_fwd(const float* x, const int64_t* labels, float* loss,
                                int64_t rows, int64_t cols, float clip_lo,
                                hipStream_t stream) {
  Clip c;
  bool wide = false;
  int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  rc = check_sizes(rows, cols);
  if (rc != SOFTMAX_OK) return rc;
  if (rows == 0) return SOFTMAX_OK;
  if (cols == 0) return SOFTMAX_ERR_INVALID_ARG;  // no row has a valid label
  if (x == nullptr || labels == nullptr || loss == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (rows > INT64_MAX / 8) return SOFTMAX_ERR_INVALID_ARG;
  const int64_t xbytes = rows * cols * 4;
  const int64_t lbytes = rows * 8;
  const int64_t obytes = rows * 4;
  if (ranges_overlap(loss, obytes, x, xbytes) || ranges_overlap(loss, obytes, labels, lbytes))
    return SOFTMAX_ERR_INVALID_ARG;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e);
  if ((rc = check_device_range(x, xbytes, dev)) != SOFTMAX_OK) return rc;
  if ((rc = check_device_range(labels, lbytes, dev)) != SOFTMAX_OK) return rc;
  if ((rc = check_device_range(loss, obytes, dev)) != SOFTMAX_OK) return rc;
  // The plan's access width follows x alone: the losses are 32-bit stores.
  return launch_mode(make_plan(x, x, rows, cols), x, loss, labels, rows, cols, dev, c, kNllOut,
                     stream);
}

SOFTMAX_API int softmax_fwd(const float* x, float* y, int64_t rows, int64_t cols,
                            hipStream_t stream) {
  return softmax_fwd_clip(x, y, rows, cols, SOFTMAX_CLIP_LO, stream);
}

SOFTMAX_API const char* softmax_strerror(int code) {
  switch (code) {
    case SOFTMAX_OK: return "success";
    case SOFTMAX_ERR_INVALID_ARG:
      return "invalid argument (negative or overflowing size, null pointer, "
             "partially overlapping x and y, or a clip bound that is NaN or above "
             "SOFTMAX_CLIP_MAX)";
    case SOFTMAX_ERR_HIP: return "HIP call or kernel launch failed";
    case SOFTMAX_ERR_NOT_DEVICE:
      return "pointer is not memory the current device can use, or the range "
             "runs past its allocation";
    default: return "unknown softmax error code";
  }
}

SOFTMAX_API int softmax_last_hip_error(void) { return smx_host::tl_last_hip_error; }

SOFTMAX_API int softmax_exp_probe(const float* x, const float* m, float* e, int64_t n,
                                  float clip_lo, int approx, hipStream_t stream) {
  Clip c;
  bool wide = false;
  if (make_clip(clip_lo, &c, &wide) != SOFTMAX_OK) return SOFTMAX_ERR_INVALID_ARG;
  if (n < 0 || n > INT64_MAX / 4) return SOFTMAX_ERR_INVALID_ARG;
  if (n == 0) return SOFTMAX_OK;
  if (x == nullptr || m == nullptr || e == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (any_overlap(e, x, n * 4) || any_overlap(e, m, n * 4)) return SOFTMAX_ERR_INVALID_ARG;
  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return fail_hip(he);
  int rc = check_device_range(x, n * 4, dev);
  if (rc == SOFTMAX_OK) rc = check_device_range(m, n * 4, dev);
  if (rc == SOFTMAX_OK) rc = check_device_range(e, n * 4, dev);
  if (rc != SOFTMAX_OK) return rc;
  const int64_t grid = std::min(ceil_div(n, 256), kMaxGrid);
  void* args[] = {&x, &m, &e, &n, &c};
  const void* fn = approx ? reinterpret_cast<const void*>(&k_exp_probe<kExpFast>)
                  : wide  ? reinterpret_cast<const void*>(&k_exp_probe<kExpWide>)
                          : reinterpret_cast<const void*>(&k_exp_probe<kExpAccurate>);
  he = launch(fn, grid, 256, args, stream);
  return he == hipSuccess ? SOFTMAX_OK : fail_hip(he);
}

SOFTMAX_API int softmax_copy_probe(const float* x, float* y, int64_t n, hipStream_t stream) {
  if (n < 0 || n > INT64_MAX / 4) return SOFTMAX_ERR_INVALID_ARG;
  if (n == 0) return SOFTMAX_OK;
  if (x == nullptr || y == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (any_overlap(x, y, n * 4)) return SOFTMAX_ERR_INVALID_ARG;
  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return fail_hip(he);
  int rc = check_device_range(x, n * 4, dev);
  if (rc == SOFTMAX_OK) rc = check_device_range(y, n * 4, dev);
  if (rc != SOFTMAX_OK) return rc;
  if (aligned16(x) && aligned16(y) && n % 4 == 0) {
    int64_t n4 = n / 4;
    const int64_t grid = std::min(ceil_div(n4, 256 * kCopyUnroll), kMaxGrid);
    void* args[] = {&x, &y, &n4};
    he = launch(reinterpret_cast<const void*>(&k_copy4), grid, 256, args, stream);
  } else {
    const int64_t grid = std::min(ceil_div(n, 256), kMaxGrid);
    void* args[] = {&x, &y, &n};
    he = launch(reinterpret_cast<const void*>(&k_copy1), grid, 256, args, stream);
  }
  return he == hipSuccess ? SOFTMAX_OK : fail_hip(he);
}

}  // extern "C"
