// C ABI of the row-softmax library: argument checks, the dispatch on cols,
// the exchange table of split rows, the store schedule, and the launches.
// Declarations and the contract are in include/softmax_mi355x.h.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <mutex>
#include <utility>
#include <vector>

#include "../../include/softmax_mi355x.h"
#include "sm_host.hpp"
#include "sm_kernels.hpp"

// The exchange table of rows split over several workgroups (layout in
// sm_exchange.hpp).  The kernels claim and free its row entries themselves,
// and it is all zero at rest, as it starts.  Every device the library runs
// on holds its own copy until the process ends.  Host code never uses this
// name as an address: it passes the kernels the device address that
// hipGetSymbolAddress gives for the current device (device_facts below).
static __device__ __align__(256) uint64_t scratch[smx::xch::kScratchWords];

namespace {

using namespace smx;
using namespace smx_host;

// Bucket limits on cols.
constexpr int64_t kPackedMaxCols = 64;
// Probability rows of up to this many columns that are not whole 16-byte
// strips (or whose x or y is not 16-byte aligned) also take the packed
// kernel, with 8 or 16 lanes per row: per 64 MiB of logits, 65 columns
// took 64 us with one wavefront per row and 32-bit access (65 of 256
// register slots of a wavefront in use).
constexpr int64_t kPackedProbMaxCols = 256;
// The packed kernel's persistent grid: six 256-thread workgroups per CU.
// Measured on 115200 x 50: up to six per CU the prefetched next tile
// overlaps the current tile's compute; seven or more per CU, or one tile per
// workgroup, are slower.
constexpr int64_t kPackedBlocksPerCU = 6;
constexpr int64_t kWaveRowMaxCols = 4096;
// With 32-bit access, 64 values per lane need more registers than a
// wavefront has (the kernel would spill): such rows go to k_block_row.
constexpr int64_t kWaveRowMaxColsScalar = 2048;
constexpr int64_t kBlockRowMaxCols = 32768;
constexpr int kBlockThreads = 1024;
// Probability and log rows longer than this take the one-pass split kernel
// rather than one workgroup per row (measured with the dispatch sweep,
// paper_1904_12380_amd/sweep.py).  Per 64 MiB of logits, 16384 columns ran
// 21.8 us split against 25.8 us and 32768 columns 21.7 against 22.2.  Rows
// of 8193 to 16380 columns make two chunks, the second partly empty, and
// more rows than one launch of resident workgroups takes (1024 rows), so the
// last launch is ragged.  There one workgroup per row was 11-28% faster at
// 64 MiB, 10-35% at 128 MiB and 16-33% at 4 and 16 MiB.  At 16380 columns
// the split kernel was 7% faster at 64 MiB and level at 128 MiB.  Log rows
// of 16384 to 32768 columns ran 22.3-22.5 us split against 24.2-26.7 us in
// one workgroup.  Rows of 16381 to 16383 columns that are not whole strips
// keep the split kernel (16383: 28.0 us split with 32-bit access against
// 30.6 in one workgroup).  NLL rows keep k_block_row up to
// kBlockRowMaxCols.
constexpr int64_t kSplitMinColsProb = 16380;
// k_group_rows: when one workgroup per row block would take more than one
// but at most this many rounds of the resident workgroups, the grid is
// capped at the resident ones (each loops over row blocks, loading the next
// block before reducing the current one): a last round that leaves most of
// the chip idle costs more than the loop.  Above it, one workgroup per row
// block keeps more loads in flight.
constexpr int64_t kGroupRowsPersistentRounds = 2;
// Rows of at most 256 columns in whole strips: the grouped-rows kernel or
// the LDS-staged packed kernel (library_shape), by the rounds of resident
// workgroups one grouped-rows workgroup per row block would take and by the
// fill, the share of a row's G lanes that hold a strip.  Measured on 4 to
// 256 columns at 2 to 64 MiB:
//  * at most kGroupRowsOneStep rounds at U = 1 (a small launch): grouped
//    rows with U = 1 at any fill; at 2 to 8 MiB U = 1 ran 3-12% faster than
//    U = 2, and at 3 MiB 3-21% faster than the packed kernel on rows of
//    fill 0.52-0.69;
//  * beyond that, fill below 3/4 (36-44, 68-92 and 132-188 columns): the
//    packed kernel, faster by up to 35% at every size from 8 MiB on, except
//    on some rows at 40 MiB and above, where it was up to 4% slower;
//  * fill below 1, or G >= 32 (rows of more than 64 columns), at more than
//    one and at most kGroupRowsPackedRounds = 2.5 rounds at U = 2: the
//    packed kernel, level to 18% faster on rows of fill 3/4 to 1 (12 to
//    244 columns) at 1.0-2.5 rounds, and on 128 and 256 columns from 1%
//    slower to 6% faster; from about 2.75 rounds (40 and 48 MiB) it ranged
//    from 5% faster to 8% slower, and at 4-5 rounds (64 MiB) it was 1-6%
//    slower.
//    Full rows of at most 64 columns keep grouped rows (at 22 MiB 17-44%
//    faster than packed, whose LDS tiles of 16 and 32 columns take bank
//    conflicts).
constexpr int64_t kGroupRowsMinFillNum = 3;
constexpr int64_t kGroupRowsMinFillDen = 4;
constexpr int64_t kGroupRowsPackedRoundsNum = 5;  // kGroupRowsPackedRounds = 2.5
constexpr int64_t kGroupRowsPackedRoundsDen = 2;
constexpr int64_t kGroupRowsOneStepNum = 13;  // kGroupRowsOneStep = 1.3 rounds
constexpr int64_t kGroupRowsOneStepDen = 10;

// Split rows, one pass: a row spans at most this many workgroups (the
// exchange is read by one wavefront, one slot per lane).  Chunk shapes,
// threads x 4-element strips per lane: probability and log rows take 256 x 8
// (8192 columns) up to kSmallChunkMaxChunks chunks; then every mode takes
// 512 x 8 (16384 columns) up to 64 chunks, then 512 x 16 (32768, 128-bit
// access only: with 32-bit access it would spill).  Measured per 64 MiB:
// 256 x 8 ran 21.6-21.8 us on rows of 16384 to 65536 columns against
// 21.8-22.7 for 512 x 8, but 22.5 against 21.7 on 131072 columns and 24.2
// against 22.0 on 262144 (the row's wait for 16 or 32 partials costs more
// than the smaller workgroups gain).  NLL outputs take 512 x 8 from the
// first chunk: their workgroups never wait for each other and keep no
// values; 1024 x 8 (32768 columns) measured 3-4% slower on 131072 to 524288
// columns (64 x 262144: 15.9 against 15.3 us).
constexpr int64_t kOnePassMaxChunks = 64;
constexpr int64_t kSmallChunkMaxChunks = 8;
// Probability rows past kSmallChunkMaxChunks 8192-column chunks take
// 8192-column chunks anyway (library_shape) when
//  * that needs fewer launches (each launch holds the rows whose workgroups
//    are resident at once): 300000 columns x 55 rows made 53 + 2 rows in
//    16384-column chunks and one launch in 8192-column ones, 24.8 against
//    29.7 us;
//  * or the 16384-column grid would hold fewer than 5/8 of a workgroup per
//    CU and a row at most 40 8192-column chunks: at 8 MiB (114-140
//    workgroups) on 100000-300000 columns 8.3-8.9 against 8.9-9.3 us, but
//    524288 columns (64 chunks) 10.0 against 9.8;
//  * or that grid would hold fewer than 2 per CU, a row at most 32 chunks,
//    and 16384-column chunks would pad the row by at least 1/32 more: at
//    16 MiB (247-287 workgroups) 100000 and 200000 columns ran 10.9 and
//    10.7 against 11.8 and 12.0 us, while 131072, 262144 and 300000 columns
//    (no or 2.7% more padding) ran 1-7% faster in 16384-column chunks;
//  * or that grid would hold fewer than 3 per CU and 16384-column chunks
//    would pad the row by at least 1/16 more: at 32 MiB 100000 columns (581
//    workgroups, 8.2% more padding) 14.3 against 15.0 us, while 200000
//    columns (4.1%) ran 0.9% faster in 16384-column chunks.
// Where the 16384-column grid fills the chip (64 MiB), only fewer launches
// changed the choice.
constexpr int64_t kSplitSparseNum = 5;  // workgroups per CU, 5/8
constexpr int64_t kSplitSparseDen = 8;
constexpr int64_t kSplitSparseMaxChunks = 40;
constexpr int64_t kSplitThinPerCU = 2;
constexpr int64_t kSplitThinMaxChunks = 32;
constexpr int64_t kSplitThinPadDen = 32;  // extra padding of at least cols / 32
constexpr int64_t kSplitWidePerCU = 3;
constexpr int64_t kSplitWidePadDen = 16;  // extra padding of at least cols / 16
// Probability rows of three 8192-column chunks whose last one is partly
// empty (16384 < cols < 24576, whole strips) take one workgroup per row
// (library_shape) when there are at least 1/3 and at most 15/16 as many rows
// as compute units: then every row has a CU to itself and the split grid
// would spend a third of its workgroups on the part-empty chunk.  Measured
// at 8 and 16 MiB (85-240 rows): 17408 to 22528 columns ran 8.1-8.4 us
// against 8.7-8.9 and 9.8-10.0 against 10.5-10.9 (5-9% faster); 24576
// columns (no empty part) 1-9% slower in one workgroup, and 16388 columns x
// 255 rows 1.3% slower.  At the bounds: 46-81 rows ran 3-6% faster split,
// 89-105 rows 5-7% faster in one workgroup; 243 and 256 rows of 20480
// columns 1.5-2.5% faster split.  With more rows than CUs the split kernel
// was level or faster except at 17408 and 18432 columns x 455-481 rows
// (4.5% slower).
constexpr int64_t kBlockOverSplitMinRowsDen = 3;   // rows >= CUs / 3
constexpr int64_t kBlockOverSplitMaxRowsNum = 15;  // rows <= CUs * 15/16
constexpr int64_t kBlockOverSplitMaxRowsDen = 16;

// Split rows, two passes (rows too long for the one-pass shapes): 512 x 8
// chunks, at most 64 workgroups per row (one exchange slot each, every
// workgroup taking a stride of the row's chunks) and about 2048 per launch.
constexpr int kSplitThreads = 512;
constexpr int kSplitV = 8;
constexpr int64_t kTwoPassWorkgroups = 2048;

// Store schedule of the one-pass split-row launches, in which every
// workgroup is resident at once and takes one chunk: the stores wait until
// the launch's loads are expected to be over, read_bytes / rate + base, so
// that HBM serves the launch's reads and writes as two phases instead of
// interleaving them.  The rate is MI355X's measured streaming read rate of
// such launches; a launch whose reads take longer simply starts its stores
// while the last reads are still arriving.  Small launches are left alone
// (their phases are short next to the launch latency).  The row kernels
// (k_wave_row, k_block_row) take the same delay only through
// softmax_fwd_planned: measured on 4096 x 1000 and 512 x 32768 it gained
// nothing there (their stores already spread out behind the exponentials),
// while on 64 x 262144 and on 512 x 32768 in 16384-column chunks the split
// kernel gained 0.05-0.3 us.
constexpr double kStoreReadBytesPerNs = 7600.0;
constexpr int64_t kStoreBaseNs = 300;
constexpr int64_t kStoreMinBytes = int64_t(8) << 20;
constexpr int64_t kStoreMaxNs = 200000;

// ---------------------------------------------------------------------------
// Per-device facts: compute units, the wall clock's rate, and the device
// address of `scratch`, taken once per device with that device current.
struct DeviceFacts {
  int dev = 0;
  int cus = 0;
  int64_t wall_khz = 0;
  uint64_t* scratch = nullptr;
};
std::mutex g_facts_mu;
bool g_facts_ready[kMaxDevices] = {};
DeviceFacts g_facts[kMaxDevices];

int device_facts(int dev, DeviceFacts* out) {
  if (dev < 0 || dev >= kMaxDevices) return SOFTMAX_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_facts_mu);
  if (!g_facts_ready[dev]) {
    DeviceFacts f;
    f.dev = dev;
    int rc = device_cus(dev, &f.cus);
    if (rc != SOFTMAX_OK) return rc;
    int khz = 0;
    hipError_t e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return fail_hip(e);
    if (khz <= 0) return SOFTMAX_ERR_INVALID_ARG;
    f.wall_khz = khz;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail_hip(e);
    if (p == nullptr) return SOFTMAX_ERR_HIP;
    f.scratch = static_cast<uint64_t*>(p);
    g_facts[dev] = f;
    g_facts_ready[dev] = true;
  }
  *out = g_facts[dev];
  return SOFTMAX_OK;
}

// Workgroups of `fn` (at `block` threads) that one CU holds at once, from
// the runtime's occupancy calculator; cached per (device, kernel).
struct OccEntry {
  int dev;
  const void* fn;
  int per_cu;
};
std::mutex g_occ_mu;
std::vector<OccEntry> g_occ;

int blocks_per_cu(int dev, const void* fn, int block, int* out) {
  std::lock_guard<std::mutex> lock(g_occ_mu);
  for (const OccEntry& o : g_occ) {
    if (o.dev == dev && o.fn == fn) {
      *out = o.per_cu;
      return SOFTMAX_OK;
    }
  }
  int n = 0;
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, 0);
  if (e != hipSuccess) return fail_hip(e);
  if (n <= 0) return SOFTMAX_ERR_HIP;
  g_occ.push_back(OccEntry{dev, fn, n});
  *out = n;
  return SOFTMAX_OK;
}

// Per-call part of the exchange key (the launch's output address fills the
// high bits): calls made at the same time never share a key unless they
// write the same output, and an entry left claimed after a give-up is not
// picked up by later calls.
std::atomic<uint32_t> g_nonce{1};

// Per device: the exchange entry the next split-row launch starts at.
// Every launch takes as many consecutive entries as it has rows (mod
// xch::kEntries), so launches in flight together never meet at an entry
// while they hold fewer than xch::kEntries rows between them.
std::atomic<uint32_t> g_entry_cursor[kMaxDevices];

inline uint32_t entry_base(const DeviceFacts& f, int64_t rows_in_launch) {
  return g_entry_cursor[f.dev].fetch_add(static_cast<uint32_t>(rows_in_launch),
                                        std::memory_order_relaxed);
}

inline uint64_t exchange_key(const void* out_first_row, uint32_t nonce) {
  return (static_cast<uint64_t>(reinterpret_cast<uintptr_t>(out_first_row)) << 16) |
         (nonce & 0xFFFFu);
}

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

// ---------------------------------------------------------------------------
// Kernel instances.  A shape names one compiled kernel: its family, access
// width, threads per workgroup and strips per lane (packed rows: lanes per
// row and columns per lane).
struct Shape {
  int kernel = SOFTMAX_KERNEL_NONE;
  bool vec4 = false;
  int threads = 0;
  int v = 0;        // 128-bit strips (or groups of four scalars) per lane
  int g = 0;        // packed rows: lanes per row
  int epl = 0;      // packed rows: columns per lane
  bool two_pass = false;
  bool ph = false;  // 128-bit access to rows that are not 16-byte aligned (row phase)
};

// k_packed instances: G = 1 with EPL = 1..16, G = 2, 4, 8 and 16 with
// EPL = 9..16 (a plan never asks for fewer columns per lane at G > 1); G = 8
// and 16 (rows of 65 to 256 columns) for probability outputs only.
template <int G, bool VEC4, int EM, int... E>
const void* packed_fn(int epl, std::integer_sequence<int, E...>) {
  static const void* const table[] = {
      reinterpret_cast<const void*>(&k_packed<G, (G == 1 ? 1 : 9) + E, VEC4, EM>)...};
  const int idx = epl - (G == 1 ? 1 : 9);
  return (idx >= 0 && idx < static_cast<int>(sizeof...(E))) ? table[idx] : nullptr;
}

// k_group_rows instances: G = 1, 2, ..., 64 lanes per row, U = 1 or 2 row
// groups per wavefront step.
template <int U, int EM>
const void* group_rows_fn(int g) {
  auto cast = [](auto f) { return reinterpret_cast<const void*>(f); };
  switch (g) {
    case 1: return cast(&k_group_rows<1, U, EM>);
    case 2: return cast(&k_group_rows<2, U, EM>);
    case 4: return cast(&k_group_rows<4, U, EM>);
    case 8: return cast(&k_group_rows<8, U, EM>);
    case 16: return cast(&k_group_rows<16, U, EM>);
    case 32: return cast(&k_group_rows<32, U, EM>);
    case 64: return cast(&k_group_rows<64, U, EM>);
    default: return nullptr;
  }
}

template <int EM, bool VEC4>
const void* shape_fn(const Shape& s, bool stats_pass) {
  auto cast = [](auto f) { return reinterpret_cast<const void*>(f); };
  switch (s.kernel) {
    case SOFTMAX_KERNEL_GROUP_ROWS:
      if constexpr (VEC4 && (EM == kExpAccurate || EM == kExpWide || EM == kExpFast)) {
        if (s.v == 1) return group_rows_fn<1, EM>(s.g);
        if (s.v == 2) return group_rows_fn<2, EM>(s.g);
      }
      return nullptr;
    case SOFTMAX_KERNEL_PACKED:
      if (s.g == 1) return packed_fn<1, VEC4, EM>(s.epl, std::make_integer_sequence<int, 16>{});
      if (s.g == 2) return packed_fn<2, VEC4, EM>(s.epl, std::make_integer_sequence<int, 8>{});
      if (s.g == 4) return packed_fn<4, VEC4, EM>(s.epl, std::make_integer_sequence<int, 8>{});
      if constexpr (EM == kExpAccurate || EM == kExpWide || EM == kExpFast) {
        if (s.g == 8) return packed_fn<8, VEC4, EM>(s.epl, std::make_integer_sequence<int, 8>{});
        if (s.g == 16)
          return packed_fn<16, VEC4, EM>(s.epl, std::make_integer_sequence<int, 8>{});
      }
      return nullptr;
    case SOFTMAX_KERNEL_WAVE_ROW:
      if (s.ph) {
        if constexpr (VEC4 && (EM == kExpAccurate || EM == kExpWide || EM == kExpFast)) {
          switch (s.v) {
            case 1: return cast(&k_wave_row<1, true, EM, true>);
            case 2: return cast(&k_wave_row<2, true, EM, true>);
            case 4: return cast(&k_wave_row<4, true, EM, true>);
            case 8: return cast(&k_wave_row<8, true, EM, true>);
            case 16: return cast(&k_wave_row<16, true, EM, true>);
            default: return nullptr;
          }
        }
        return nullptr;
      }
      switch (s.v) {
        case 1: return cast(&k_wave_row<1, VEC4, EM>);
        case 2: return cast(&k_wave_row<2, VEC4, EM>);
        case 4: return cast(&k_wave_row<4, VEC4, EM>);
        case 8: return cast(&k_wave_row<8, VEC4, EM>);
        case 16:
          if constexpr (VEC4) return cast(&k_wave_row<16, VEC4, EM>);
          return nullptr;
        default: return nullptr;
      }
    case SOFTMAX_KERNEL_BLOCK_ROW:
      if (s.ph) {
        if constexpr (VEC4 && (EM == kExpAccurate || EM == kExpWide || EM == kExpFast)) {
          switch (s.v) {
            case 2: return cast(&k_block_row<kBlockThreads, 2, true, EM, true>);
            case 4: return cast(&k_block_row<kBlockThreads, 4, true, EM, true>);
            default: return nullptr;
          }
        }
        return nullptr;
      }
      switch (s.v) {
        case 2: return cast(&k_block_row<kBlockThreads, 2, VEC4, EM>);
        case 4: return cast(&k_block_row<kBlockThreads, 4, VEC4, EM>);
        case 8: return cast(&k_block_row<kBlockThreads, 8, VEC4, EM>);
        default: return nullptr;
      }
    case SOFTMAX_KERNEL_SPLIT_ROW:
      if (s.two_pass) {
        if (s.threads != kSplitThreads || s.v != kSplitV) return nullptr;
        return stats_pass ? cast(&k_split_stats<kSplitThreads, kSplitV, VEC4, EM>)
                          : cast(&k_split_apply<kSplitThreads, kSplitV, VEC4, EM>);
      }
      if (s.ph) {
        if constexpr (VEC4 && (EM == kExpAccurate || EM == kExpWide || EM == kExpFast)) {
          if (s.threads == 256 && s.v == 8) return cast(&k_split_onepass<256, 8, true, EM, true>);
          if (s.threads == 512 && s.v == 8) return cast(&k_split_onepass<512, 8, true, EM, true>);
        }
        return nullptr;
      }
      if (s.threads == 256 && s.v == 8) return cast(&k_split_onepass<256, 8, VEC4, EM>);
      if (s.threads == 512 && s.v == 8) return cast(&k_split_onepass<512, 8, VEC4, EM>);
      if constexpr (VEC4) {
        if (s.threads == 512 && s.v == 16) return cast(&k_split_onepass<512, 16, VEC4, EM>);
      }
      return nullptr;
    default:
      return nullptr;
  }
}

template <int EM>
const void* shape_fn_mode(const Shape& s, bool stats_pass) {
  return s.vec4 ? shape_fn<EM, true>(s, stats_pass) : shape_fn<EM, false>(s, stats_pass);
}

const void* kernel_fn(const Shape& s, int em, bool stats_pass = false) {
  switch (em) {
    case kExpWide: return shape_fn_mode<kExpWide>(s, stats_pass);
    case kExpFast: return shape_fn_mode<kExpFast>(s, stats_pass);
    case kLogOut: return shape_fn_mode<kLogOut>(s, stats_pass);
    case kNllOut: return shape_fn_mode<kNllOut>(s, stats_pass);
    default: return shape_fn_mode<kExpAccurate>(s, stats_pass);
  }
}

inline int64_t chunk_cols(const Shape& s) { return int64_t(4) * s.v * s.threads; }

// Chunks per row of a split shape: with the row phase (s.ph) the chunks
// must cover cols + 3 columns (a row may start up to 3 floats past a
// 16-byte boundary, and every chunk but the first is aligned).
inline int64_t row_chunks(const Shape& s, int64_t cols) {
  return ceil_div(cols + (s.ph ? 3 : 0), chunk_cols(s));
}

// Lanes per row of the packed kernel: at most 16 columns per lane.
inline int packed_lanes(int64_t cols) {
  return cols <= 16 ? 1 : cols <= 32 ? 2 : cols <= 64 ? 4 : cols <= 128 ? 8 : 16;
}

// Lanes per row of the grouped-rows kernel: one 16-byte strip per lane, a
// power of two.
inline int group_rows_lanes(int64_t cols) {
  return static_cast<int>(pow2_at_least(ceil_div(cols, 4)));
}

// Whether kernel family `kernel` may use 128-bit access: both pointers
// 16-byte aligned and, except for packed rows (which move whole tiles of a
// multiple of four rows), rows made of whole float4s.
inline bool can_vec4(int kernel, const float* x, const float* y, int64_t cols) {
  const bool a16 = aligned16(x) && aligned16(y);
  return kernel == SOFTMAX_KERNEL_PACKED ? a16 : (a16 && cols % 4 == 0);
}

// Rows taken with 128-bit access in the aligned strips around each row
// (k_wave_row / k_block_row with PH): cols not a multiple of 4, x and y
// 16-byte aligned, and 2048 < cols <= 16377.  Measured per 64 MiB: 4093
// columns 29.3 us against 37.7 us with 32-bit access, 8189 columns 28.1;
// but 65, 250 and 2047 columns ran slower than with 32-bit access (84
// against 64, 28.5 against 25.0, 31.9 against 28.6 us): the straddling
// strips are element by element, and the strips must cover cols + 3.
inline bool phase_rows(const float* x, const float* y, int64_t cols) {
  return cols % 4 != 0 && cols > kWaveRowMaxColsScalar && cols + 3 <= kSplitMinColsProb &&
         aligned16(x) && aligned16(y);
}

// Split rows taken with the row phase (k_split_onepass with PH): threads
// per workgroup (8192-column chunks while a row needs at most 8, else
// 16384), and whether a row qualifies: cols not a multiple of 4, x and y
// 16-byte aligned, more than one 8192-column chunk, one pass, and the phase
// adds no chunk (the library takes it only past phase_rows' range; a
// caller's plan may ask for it from 8190 columns) (the chunks cover cols + 3 columns; where that
// takes one more chunk than cols, the extra, nearly empty workgroups per
// row cost more than 128-bit access gains: 16383 columns ran 33.5 us with
// the phase and 28.2 us with 32-bit access, 131071 columns 33.2 against
// 28.6).  Measured per 64 MiB: 32765 and 65533 columns ran 23.9 us with the
// phase against about 28.3 with 32-bit access.
inline int split_phase_threads(int64_t cols) {
  return ceil_div(cols + 3, int64_t(4) * 8 * 256) <= kSmallChunkMaxChunks ? 256 : 512;
}
inline bool split_phase_rows(const float* x, const float* y, int64_t cols) {
  if (cols % 4 == 0 || cols + 3 <= 8192 || !aligned16(x) || !aligned16(y)) return false;
  const int64_t ch = int64_t(4) * 8 * split_phase_threads(cols);
  return ceil_div(cols + 3, ch) == ceil_div(cols, ch) &&
         ceil_div(cols + 3, ch) <= kOnePassMaxChunks;
}

// Row kernel for rows accessed with their phase: the strips must cover
// cols + 3 columns (a row may start up to 3 floats past a 16-byte boundary).
void phase_row_shape(int64_t cols, Shape* s) {
  const int64_t span = cols + 3;
  if (span <= kWaveRowMaxCols) {
    s->kernel = SOFTMAX_KERNEL_WAVE_ROW;
    s->threads = 256;
    s->v = static_cast<int>(pow2_at_least(ceil_div(span, 256)));
  } else {
    s->kernel = SOFTMAX_KERNEL_BLOCK_ROW;
    s->threads = kBlockThreads;
    s->v = static_cast<int>(std::max<int64_t>(2, pow2_at_least(ceil_div(span, 4096))));
  }
}

// The library's shape for a call (mode em) from the arguments alone;
// library_shape refines it for short rows by the row count and the device.
Shape default_shape(const float* x, const float* y, int64_t cols, int em) {
  Shape s;
  const bool prob = em != kLogOut && em != kNllOut;
  s.vec4 = can_vec4(cols <= kPackedMaxCols ? SOFTMAX_KERNEL_PACKED : SOFTMAX_KERNEL_SPLIT_ROW,
                    x, y, cols);
  if (prob && cols <= kGroupRowsMaxCols && can_vec4(SOFTMAX_KERNEL_GROUP_ROWS, x, y, cols)) {
    s.kernel = SOFTMAX_KERNEL_GROUP_ROWS;
    s.vec4 = true;
    s.threads = 256;
    s.g = group_rows_lanes(cols);
    s.v = 2;
  } else if (cols <= (prob ? kPackedProbMaxCols : kPackedMaxCols)) {
    // G lanes per row with at most 16 columns per lane.
    s.kernel = SOFTMAX_KERNEL_PACKED;
    s.vec4 = can_vec4(SOFTMAX_KERNEL_PACKED, x, y, cols);
    s.threads = 256;
    s.g = packed_lanes(cols);
    s.epl = static_cast<int>(ceil_div(cols, s.g));
  } else if (prob && phase_rows(x, y, cols)) {
    // Rows that are not whole 16-byte strips, in aligned x and y: 128-bit
    // access in the aligned strips around each row.
    s.vec4 = true;
    s.ph = true;
    phase_row_shape(cols, &s);
  } else if (prob && split_phase_rows(x, y, cols)) {
    // Long rows that are not whole 16-byte strips, in aligned x and y: the
    // one-pass split kernel with the row phase.
    s.kernel = SOFTMAX_KERNEL_SPLIT_ROW;
    s.vec4 = true;
    s.ph = true;
    s.v = 8;
    s.threads = split_phase_threads(cols);
  } else if (cols <= (s.vec4 ? kWaveRowMaxCols : kWaveRowMaxColsScalar)) {
    s.kernel = SOFTMAX_KERNEL_WAVE_ROW;
    s.threads = 256;
    s.v = static_cast<int>(pow2_at_least(ceil_div(cols, 256)));
  } else if (cols <= (em != kNllOut ? kSplitMinColsProb : kBlockRowMaxCols)) {
    s.kernel = SOFTMAX_KERNEL_BLOCK_ROW;
    s.threads = kBlockThreads;
    s.v = static_cast<int>(std::max<int64_t>(2, pow2_at_least(ceil_div(cols, 4096))));
  } else {
    s.kernel = SOFTMAX_KERNEL_SPLIT_ROW;
    if (em != kNllOut && ceil_div(cols, int64_t(4) * 8 * 256) <= kSmallChunkMaxChunks) {
      s.threads = 256;
      s.v = 8;
    } else if (ceil_div(cols, int64_t(4) * 8 * 512) <= kOnePassMaxChunks) {
      s.threads = 512;
      s.v = 8;
    } else if (s.vec4 && ceil_div(cols, int64_t(4) * 16 * 512) <= kOnePassMaxChunks) {
      s.threads = 512;
      s.v = 16;
    } else {
      s.threads = kSplitThreads;
      s.v = kSplitV;
      s.two_pass = true;
    }
  }
  return s;
}

// A caller's shape (softmax_fwd_planned): the family, access width and, for
// split rows, the chunk shape; everything else is derived.  Returns false
// when the shape is not one the library has or cannot take these rows.
bool requested_shape(const softmax_plan_t& want, const float* x, const float* y, int64_t cols,
                     int em, Shape* out) {
  Shape s;
  s.kernel = want.kernel;
  if (want.vec_width != 1 && want.vec_width != 4) return false;
  s.vec4 = want.vec_width == 4;
  // 128-bit access to rows that are not whole 16-byte strips: the row
  // kernels with the row phase (probability outputs, aligned x and y).
  const bool row_kernel =
      s.kernel == SOFTMAX_KERNEL_WAVE_ROW || s.kernel == SOFTMAX_KERNEL_BLOCK_ROW;
  // The same for split rows (one pass, 8192- or 16384-column chunks).
  if (s.vec4 && s.kernel == SOFTMAX_KERNEL_SPLIT_ROW && split_phase_rows(x, y, cols) &&
      em != kLogOut && em != kNllOut) {
    s.ph = true;
    s.threads = want.block_threads;
    s.v = want.elems_per_lane / 4;
    if (want.elems_per_lane % 4 != 0 || s.v != 8) return false;
    if (row_chunks(s, cols) > kOnePassMaxChunks) return false;
    if (kernel_fn(s, em) == nullptr) return false;
    *out = s;
    return true;
  }
  if (s.vec4 && row_kernel && phase_rows(x, y, cols) && em != kLogOut && em != kNllOut) {
    const int64_t span = cols + 3;
    if (span > (s.kernel == SOFTMAX_KERNEL_WAVE_ROW ? kWaveRowMaxCols : kSplitMinColsProb))
      return false;
    s.ph = true;
    s.threads = s.kernel == SOFTMAX_KERNEL_WAVE_ROW ? 256 : kBlockThreads;
    s.v = static_cast<int>(s.kernel == SOFTMAX_KERNEL_WAVE_ROW
                               ? pow2_at_least(ceil_div(span, 256))
                               : std::max<int64_t>(2, pow2_at_least(ceil_div(span, 4096))));
    if (kernel_fn(s, em) == nullptr) return false;
    *out = s;
    return true;
  }
  if (s.vec4 && !can_vec4(s.kernel, x, y, cols)) return false;
  switch (s.kernel) {
    case SOFTMAX_KERNEL_GROUP_ROWS:
      if (cols > kGroupRowsMaxCols || !s.vec4) return false;
      s.threads = 256;
      s.g = group_rows_lanes(cols);
      s.v = 2;
      break;
    case SOFTMAX_KERNEL_PACKED:
      if (cols > ((em == kLogOut || em == kNllOut) ? kPackedMaxCols : kPackedProbMaxCols))
        return false;
      s.threads = 256;
      s.g = packed_lanes(cols);
      s.epl = static_cast<int>(ceil_div(cols, s.g));
      break;
    case SOFTMAX_KERNEL_WAVE_ROW:
      if (cols > (s.vec4 ? kWaveRowMaxCols : kWaveRowMaxColsScalar)) return false;
      s.threads = 256;
      s.v = static_cast<int>(pow2_at_least(ceil_div(cols, 256)));
      break;
    case SOFTMAX_KERNEL_BLOCK_ROW:
      if (cols > kBlockRowMaxCols) return false;
      s.threads = kBlockThreads;
      s.v = static_cast<int>(std::max<int64_t>(2, pow2_at_least(ceil_div(cols, 4096))));
      break;
    case SOFTMAX_KERNEL_SPLIT_ROW: {
      s.threads = want.block_threads;
      s.v = want.elems_per_lane / 4;
      if (want.elems_per_lane % 4 != 0) return false;
      const int64_t chunks = row_chunks(s, cols);
      s.two_pass = chunks > kOnePassMaxChunks;
      break;
    }
    default:
      return false;
  }
  if (kernel_fn(s, em) == nullptr) return false;
  *out = s;
  return true;
}

// Everything a call launches: the shape, its grid, rows per launch, chunks,
// the store delay in ns and in wall-clock ticks, and the exchange wait limit.
struct Plan {
  Shape shape;
  int64_t grid = 0;
  int64_t rows_per_launch = 0;
  int64_t launches = 0;
  int64_t chunks = 1;
  int64_t wpr = 1;  // two-pass: workgroups per row
  int64_t delay_ns = 0;       // the first launch's
  uint32_t delay_ticks = 0;
  bool delay_per_launch = false;  // the library's schedule: each launch by its own reads
  uint32_t limit_ticks = 0;
};

uint32_t ns_to_ticks(int64_t ns, const DeviceFacts& f) {
  const int64_t t = (ns * f.wall_khz + 999999) / 1000000;
  return static_cast<uint32_t>(std::min<int64_t>(t, UINT32_MAX));
}

// The library's store delay for a launch that reads `bytes` (0: none).
int64_t store_delay_ns(int64_t bytes) {
  if (bytes < kStoreMinBytes) return 0;
  return std::min(static_cast<int64_t>(bytes / kStoreReadBytesPerNs) + kStoreBaseNs, kStoreMaxNs);
}

// Rows per k_group_rows workgroup and step: four wavefronts, each U row
// groups of 64 / G rows.
inline int64_t group_rows_block(const Shape& s) { return int64_t(4) * s.v * (64 / s.g); }

// Resident workgroups of the kernel for shape s on device dev.
int resident_workgroups(const Shape& s, int em, int dev, const DeviceFacts& f, int64_t* out) {
  const void* fn = kernel_fn(s, em);
  if (fn == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  int per_cu = 0;
  const int rc = blocks_per_cu(dev, fn, s.threads, &per_cu);
  *out = int64_t(per_cu) * f.cus;
  return rc;
}

// Row groups per wavefront step (s->v) of a grouped-rows shape: 1 when one
// workgroup per row block at U = 1 takes at most kGroupRowsOneStep rounds
// of the resident workgroups, else 2.
int group_rows_steps(int64_t rows, int em, int dev, const DeviceFacts& f, Shape* s) {
  Shape one = *s;
  one.v = 1;
  int64_t resident = 0;
  const int rc = resident_workgroups(one, em, dev, f, &resident);
  if (rc != SOFTMAX_OK) return rc;
  s->v = ceil_div(rows, group_rows_block(one)) * kGroupRowsOneStepDen <=
                 resident * kGroupRowsOneStepNum
             ? 1
             : 2;
  return SOFTMAX_OK;
}

// The library's shape once rows and the device are known: rows of at most
// 256 columns in whole strips take the grouped-rows kernel or the packed
// kernel by the rules measured above (kGroupRowsMinFill, kGroupRowsOneStep
// and kGroupRowsPackedRounds); long probability rows choose their chunk
// size by launches and fill (kSplitFillMinPerCU).
int library_shape(const float* x, const float* y, int64_t rows, int64_t cols, int em, int dev,
                  const DeviceFacts& f, Shape* out) {
  Shape s = default_shape(x, y, cols, em);
  if (s.kernel == SOFTMAX_KERNEL_GROUP_ROWS) {
    Shape steps = s;
    int rc = group_rows_steps(rows, em, dev, f, &steps);  // steps.v == 1: a small launch
    int64_t resident = 0;                                // at U = 2
    if (rc == SOFTMAX_OK) rc = resident_workgroups(s, em, dev, f, &resident);
    if (rc != SOFTMAX_OK) return rc;
    const int64_t strips = ceil_div(cols, 4);
    const int64_t blocks = ceil_div(rows, group_rows_block(s));
    const bool sparse = strips * kGroupRowsMinFillDen < s.g * kGroupRowsMinFillNum;
    const bool mid = (strips < s.g || s.g >= 32) && blocks > resident &&
                     blocks * kGroupRowsPackedRoundsDen <= kGroupRowsPackedRoundsNum * resident;
    if (steps.v == 2 && (sparse || mid)) {
      s.kernel = SOFTMAX_KERNEL_PACKED;
      s.vec4 = can_vec4(SOFTMAX_KERNEL_PACKED, x, y, cols);
      s.threads = 256;
      s.v = 0;
      s.g = packed_lanes(cols);
      s.epl = static_cast<int>(ceil_div(cols, s.g));
    }
  } else if (s.kernel == SOFTMAX_KERNEL_SPLIT_ROW && !s.two_pass && s.threads == 512 &&
             s.v == 8 && em != kLogOut && em != kNllOut) {
    // Probability rows in 16384-column chunks: 8192-column chunks instead
    // by launches and grid fill (kSplitSparseNum, kSplitThinPerCU).
    Shape small = s;
    small.threads = 256;
    const int64_t c512 = row_chunks(s, cols);
    const int64_t c256 = row_chunks(small, cols);
    if (c256 <= kOnePassMaxChunks) {
      int64_t r512 = 0;
      int64_t r256 = 0;
      int rc = resident_workgroups(s, em, dev, f, &r512);
      if (rc == SOFTMAX_OK) rc = resident_workgroups(small, em, dev, f, &r256);
      if (rc != SOFTMAX_OK) return rc;
      const int64_t per512 = std::min(r512 / c512, int64_t(xch::kMaxRowsPerLaunch));
      const int64_t per256 = std::min(r256 / c256, int64_t(xch::kMaxRowsPerLaunch));
      if (per512 > 0 && per256 > 0) {
        const int64_t grid512 = std::min(rows, per512) * c512;
        const int64_t pad_more = c512 * chunk_cols(s) - c256 * chunk_cols(small);
        const bool fewer_launches = ceil_div(rows, per256) < ceil_div(rows, per512);
        const bool sparse = grid512 * kSplitSparseDen < kSplitSparseNum * f.cus &&
                            c256 <= kSplitSparseMaxChunks;
        const bool thin = grid512 < kSplitThinPerCU * f.cus && c256 <= kSplitThinMaxChunks &&
                          pad_more * kSplitThinPadDen >= cols;
        const bool padded = grid512 < kSplitWidePerCU * f.cus && c256 <= kSplitThinMaxChunks &&
                            pad_more * kSplitWidePadDen >= cols;
        if (fewer_launches || sparse || thin || padded) s = small;
      }
    }
  } else if (s.kernel == SOFTMAX_KERNEL_SPLIT_ROW && !s.two_pass && !s.ph && s.vec4 &&
             s.threads == 256 && s.v == 8 && em != kLogOut && em != kNllOut &&
             cols > 2 * chunk_cols(s) && cols < 3 * chunk_cols(s) &&
             rows * kBlockOverSplitMinRowsDen >= f.cus &&
             rows * kBlockOverSplitMaxRowsDen <= kBlockOverSplitMaxRowsNum * f.cus) {
    // Three 8192-column chunks, the last partly empty, and a CU per row:
    // one workgroup per row (kBlockOverSplitMinRowsDen).
    s.kernel = SOFTMAX_KERNEL_BLOCK_ROW;
    s.threads = kBlockThreads;
    s.v = static_cast<int>(std::max<int64_t>(2, pow2_at_least(ceil_div(cols, 4096))));
  }
  *out = s;
  return SOFTMAX_OK;
}

// delay_req: -1 for the library's schedule, else the delay itself in ns.
int make_plan(const Shape& s, int64_t rows, int64_t cols, int em, int dev,
              const DeviceFacts& f, int64_t delay_req, Plan* out) {
  Plan p;
  p.shape = s;
  if (s.kernel == SOFTMAX_KERNEL_GROUP_ROWS) {
    const int rc = group_rows_steps(rows, em, dev, f, &p.shape);
    if (rc != SOFTMAX_OK) return rc;
  }
  const void* fn = kernel_fn(p.shape, em);
  if (fn == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  int per_cu = 0;
  int rc = blocks_per_cu(dev, fn, s.threads, &per_cu);
  if (rc != SOFTMAX_OK) return rc;
  const int64_t resident = int64_t(per_cu) * f.cus;
  bool one_wave = false;
  int64_t launch_read_bytes = 0;
  switch (s.kernel) {
    case SOFTMAX_KERNEL_GROUP_ROWS:
      p.grid = ceil_div(rows, group_rows_block(p.shape));
      if (p.grid <= kGroupRowsPersistentRounds * resident) p.grid = std::min(p.grid, resident);
      p.grid = std::min(p.grid, kMaxGrid);
      p.rows_per_launch = rows;
      p.launches = 1;
      break;
    case SOFTMAX_KERNEL_PACKED: {
      const int64_t tile = 256 / s.g;
      p.grid = std::min(ceil_div(rows, tile), kPackedBlocksPerCU * f.cus);
      p.rows_per_launch = rows;
      p.launches = 1;
      break;
    }
    case SOFTMAX_KERNEL_WAVE_ROW:
      p.grid = std::min(ceil_div(rows, 4), kMaxGrid);
      p.rows_per_launch = rows;
      p.launches = 1;
      break;
    case SOFTMAX_KERNEL_BLOCK_ROW:
      p.grid = std::min(rows, kMaxGrid);
      p.rows_per_launch = rows;
      p.launches = 1;
      break;
    default: {  // split rows
      p.chunks = row_chunks(s, cols);
      if (!s.two_pass) {
        // Whole rows per launch, every workgroup of a launch resident at
        // once.
        if (p.chunks > resident || p.chunks > kOnePassMaxChunks) return SOFTMAX_ERR_INVALID_ARG;
        p.rows_per_launch = std::min(resident / p.chunks, int64_t(xch::kMaxRowsPerLaunch));
        p.grid = std::min(rows, p.rows_per_launch) * p.chunks;
        p.launches = ceil_div(rows, p.rows_per_launch);
        // The store schedule pays with 128-bit access; with 32-bit access
        // (rows of 16383 and 32765 columns) it measured 0.1-0.4 us slower.
        one_wave = em != kNllOut && s.vec4;
        launch_read_bytes = std::min(rows, p.rows_per_launch) * cols * 4;
      } else {
        // Workgroup w of a row takes chunks w, w + wpr, ...
        p.wpr = std::min<int64_t>(p.chunks, xch::kEntrySlots);
        p.rows_per_launch = std::min<int64_t>(std::max<int64_t>(1, kTwoPassWorkgroups / p.wpr),
                                              xch::kMaxRowsPerLaunch);
        p.grid = std::min(rows, p.rows_per_launch) * p.wpr;
        p.launches = 2 * ceil_div(rows, p.rows_per_launch);
      }
      break;
    }
  }
  if (delay_req < 0) {
    p.delay_ns = one_wave ? store_delay_ns(launch_read_bytes) : 0;
    p.delay_per_launch = one_wave;
  } else {
    p.delay_ns = delay_req;
  }
  p.delay_ns = std::min(p.delay_ns, kStoreMaxNs);
  p.delay_ticks = p.delay_ns > 0 ? ns_to_ticks(p.delay_ns, f) : 0;
  p.limit_ticks = ns_to_ticks(int64_t(xch::kWaitLimitUs) * 1000, f);
  *out = p;
  return SOFTMAX_OK;
}

softmax_plan_t public_plan(const Plan& p, int64_t rows) {
  softmax_plan_t o{};
  const Shape& s = p.shape;
  o.kernel = s.kernel;
  o.vec_width = s.vec4 ? 4 : 1;
  o.block_threads = s.threads;
  o.chunks_per_row = p.chunks;
  o.grid = p.grid;
  o.launches = static_cast<int32_t>(p.launches);
  o.store_delay_ns = p.delay_ns;
  switch (s.kernel) {
    case SOFTMAX_KERNEL_GROUP_ROWS:
      o.lanes_per_row = s.g;
      o.elems_per_lane = 4;
      break;
    case SOFTMAX_KERNEL_PACKED:
      o.lanes_per_row = s.g;
      o.elems_per_lane = s.epl;
      break;
    case SOFTMAX_KERNEL_WAVE_ROW:
      o.lanes_per_row = 64;
      o.elems_per_lane = 4 * s.v;
      break;
    default:
      o.lanes_per_row = s.threads;
      o.elems_per_lane = 4 * s.v;
      break;
  }
  o.workspace_bytes = s.kernel == SOFTMAX_KERNEL_SPLIT_ROW ? xch::kScratchBytes : 0;
  (void)rows;
  return o;
}

// ---------------------------------------------------------------------------
// Launches.

// The output and labels of rows r0.. of a call: y advances by a row of
// outputs, or by one loss per row for NLL outputs (whose labels advance
// with it).
inline float* out_rows(float* y, int64_t r0, int64_t cols, int em) {
  return em == kNllOut ? y + r0 : y + r0 * cols;
}
inline const int64_t* label_rows(const int64_t* labels, int64_t r0, int em) {
  return em == kNllOut ? labels + r0 : labels;
}

hipError_t run_plan(const Plan& p, const float* x, float* y, const int64_t* labels,
                    int64_t rows, int64_t cols, Clip c, int em, const DeviceFacts& f,
                    hipStream_t st) {
  const Shape& s = p.shape;
  const void* fn = kernel_fn(s, em);
  uint32_t delay = p.delay_ticks;
  switch (s.kernel) {
    case SOFTMAX_KERNEL_GROUP_ROWS: {
      void* args[] = {&x, &y, &rows, &cols, &c};
      return launch(fn, p.grid, 256, args, st);
    }
    case SOFTMAX_KERNEL_PACKED: {
      void* args[] = {&x, &y, &labels, &rows, &cols, &c};
      return launch(fn, p.grid, 256, args, st);
    }
    case SOFTMAX_KERNEL_WAVE_ROW:
    case SOFTMAX_KERNEL_BLOCK_ROW: {
      void* args[] = {&x, &y, &labels, &rows, &cols, &c, &delay};
      return launch(fn, p.grid, s.threads, args, st);
    }
    default:
      break;
  }
  const uint32_t nonce = g_nonce.fetch_add(1, std::memory_order_relaxed);
  if (!s.two_pass) {
    int ichunks = static_cast<int>(p.chunks);
    for (int64_t r0 = 0; r0 < rows; r0 += p.rows_per_launch) {
      const int64_t nb = std::min(p.rows_per_launch, rows - r0);
      const float* xb = x + r0 * cols;
      float* yb = out_rows(y, r0, cols, em);
      const int64_t* lb = label_rows(labels, r0, em);
      // A short last launch waits only as long as its own reads take: with
      // the first launch's delay, 10 rows of 40000 columns after 409 waited
      // 8.9 us before storing.
      if (p.delay_per_launch) {
        const int64_t ns = store_delay_ns(nb * cols * 4);
        delay = ns > 0 ? ns_to_ticks(ns, f) : 0;
      }
      XchArgs xa{f.scratch, exchange_key(yb, nonce), p.limit_ticks, 1u,  // join
                 entry_base(f, nb), 0u};
      void* args[] = {&xb, &yb, &lb, &xa, &cols, &ichunks, &delay, &c};
      const hipError_t e = launch(fn, nb * p.chunks, s.threads, args, st);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const void* fn_stats = kernel_fn(s, em, true);
  int iwpr = static_cast<int>(p.wpr);
  int64_t chunks = p.chunks;
  for (int64_t r0 = 0; r0 < rows; r0 += p.rows_per_launch) {
    const int64_t nb = std::min(p.rows_per_launch, rows - r0);
    const float* xb = x + r0 * cols;
    float* yb = out_rows(y, r0, cols, em);
    const int64_t* lb = label_rows(labels, r0, em);
    XchArgs xa{f.scratch, exchange_key(yb, nonce), p.limit_ticks, 1u, entry_base(f, nb), 0u};
    void* a1[] = {&xb, &xa, &cols, &iwpr, &chunks, &c};
    hipError_t e = launch(fn_stats, nb * p.wpr, s.threads, a1, st);
    if (e != hipSuccess) return e;
    XchArgs xb2{f.scratch, xa.key, p.limit_ticks, 0u, xa.base, 0u};  // find only
    void* a2[] = {&xb, &yb, &lb, &xb2, &cols, &iwpr, &chunks, &c};
    e = launch(fn, nb * p.wpr, s.threads, a2, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
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
// or kLogOut for log outputs) after the clip and size checks; `want` is a
// caller's shape (softmax_fwd_planned) or null for the library's.
int softmax_rows(const float* x, float* y, int64_t rows, int64_t cols, Clip c, int em,
                 const softmax_plan_t* want, hipStream_t stream) {
  int rc = check_sizes(rows, cols);
  if (rc != SOFTMAX_OK) return rc;
  Shape s;
  if (want != nullptr) {
    if (want->store_delay_ns < -1 || want->store_delay_ns > kStoreMaxNs)
      return SOFTMAX_ERR_INVALID_ARG;
    if (rows > 0 && cols > 0 && !requested_shape(*want, x, y, cols, em, &s))
      return SOFTMAX_ERR_INVALID_ARG;
  }
  if (rows == 0 || cols == 0) return SOFTMAX_OK;
  int dev = 0;
  rc = check_pointers(x, y, rows * cols, &dev);
  if (rc != SOFTMAX_OK) return rc;
  DeviceFacts f;
  if ((rc = device_facts(dev, &f)) != SOFTMAX_OK) return rc;
  if (want == nullptr && (rc = library_shape(x, y, rows, cols, em, dev, f, &s)) != SOFTMAX_OK)
    return rc;
  Plan p;
  rc = make_plan(s, rows, cols, em, dev, f, want ? want->store_delay_ns : -1, &p);
  if (rc != SOFTMAX_OK) return rc;
  const hipError_t e = run_plan(p, x, y, nullptr, rows, cols, c, em, f, stream);
  return e == hipSuccess ? SOFTMAX_OK : fail_hip(e);
}

}  // namespace

extern "C" {

SOFTMAX_API int softmax_plan(const float* x, const float* y, int64_t rows, int64_t cols,
                             softmax_plan_t* plan) {
  if (plan == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  int rc = check_sizes(rows, cols);
  if (rc != SOFTMAX_OK) return rc;
  if (rows == 0 || cols == 0) {
    *plan = softmax_plan_t{};
    plan->chunks_per_row = 1;
    return SOFTMAX_OK;
  }
  if (x == nullptr || y == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (partial_overlap(x, y, rows * cols * 4)) return SOFTMAX_ERR_INVALID_ARG;
  // The launch geometry needs the current device; without one only the
  // device-independent fields are filled in.
  int ndev = 0;
  int dev = 0;
  DeviceFacts f;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0 || hipGetDevice(&dev) != hipSuccess ||
      device_facts(dev, &f) != SOFTMAX_OK) {
    (void)hipGetLastError();
    const Shape s = default_shape(x, y, cols, kExpAccurate);
    Plan p;
    p.shape = s;
    if (s.kernel == SOFTMAX_KERNEL_SPLIT_ROW) p.chunks = row_chunks(s, cols);
    *plan = public_plan(p, rows);
    return SOFTMAX_OK;
  }
  Shape s;
  rc = library_shape(x, y, rows, cols, kExpAccurate, dev, f, &s);
  if (rc != SOFTMAX_OK) return rc;
  Plan p;
  rc = make_plan(s, rows, cols, kExpAccurate, dev, f, -1, &p);
  if (rc != SOFTMAX_OK) return rc;
  *plan = public_plan(p, rows);
  return SOFTMAX_OK;
}

SOFTMAX_API int softmax_fwd_clip(const float* x, float* y, int64_t rows, int64_t cols,
                                 float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, wide ? kExpWide : kExpAccurate, nullptr, stream);
}

SOFTMAX_API int softmax_fwd_planned(const float* x, float* y, int64_t rows, int64_t cols,
                                    const softmax_plan_t* plan, hipStream_t stream) {
  if (plan == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  Clip c;
  bool wide = false;
  const int rc = make_clip(SOFTMAX_CLIP_LO, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, kExpAccurate, plan, stream);
}

SOFTMAX_API int softmax_fwd_approx(const float* x, float* y, int64_t rows, int64_t cols,
                                   float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, kExpFast, nullptr, stream);
}

SOFTMAX_API int softmax_log_fwd(const float* x, float* y, int64_t rows, int64_t cols,
                                float clip_lo, hipStream_t stream) {
  Clip c;
  bool wide = false;
  const int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  return softmax_rows(x, y, rows, cols, c, kLogOut, nullptr, stream);
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
  DeviceFacts f;
  if ((rc = device_facts(dev, &f)) != SOFTMAX_OK) return rc;
  // The access width follows x alone: the losses are 32-bit stores.
  Plan p;
  rc = make_plan(default_shape(x, x, cols, kNllOut), rows, cols, kNllOut, dev, f, -1, &p);
  if (rc != SOFTMAX_OK) return rc;
  e = run_plan(p, x, loss, labels, rows, cols, c, kNllOut, f, stream);
  return e == hipSuccess ? SOFTMAX_OK : fail_hip(e);
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
             "partially overlapping x and y, a clip bound that is NaN or above "
             "SOFTMAX_CLIP_MAX, or a plan the library cannot run)";
    case SOFTMAX_ERR_HIP: return "HIP call or kernel launch failed";
    case SOFTMAX_ERR_NOT_DEVICE:
      return "pointer is not memory the current device can use, or the range "
             "runs past its allocation";
    default: return "unknown softmax error code";
  }
}

SOFTMAX_API int softmax_last_hip_error(void) { return smx_host::tl_last_hip_error; }

SOFTMAX_API int softmax_exchange_status(uint64_t* join_give_ups, uint64_t* wait_give_ups,
                                        int32_t* entries_in_use) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e);
  DeviceFacts f;
  int rc = device_facts(dev, &f);
  if (rc != SOFTMAX_OK) return rc;
  uint64_t diag[2] = {0, 0};
  e = hipMemcpy(diag, f.scratch + xch::kDiagWord, sizeof(diag), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail_hip(e);
  // the owner word of every entry
  std::vector<uint64_t> owners(xch::kEntries);
  e = hipMemcpy2D(owners.data(), sizeof(uint64_t), f.scratch, xch::kEntryWords * sizeof(uint64_t),
                  sizeof(uint64_t), xch::kEntries, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail_hip(e);
  int32_t busy = 0;
  for (uint64_t o : owners) busy += o != 0 ? 1 : 0;
  if (join_give_ups != nullptr) *join_give_ups = diag[xch::kDiagJoinGiveUps];
  if (wait_give_ups != nullptr) *wait_give_ups = diag[xch::kDiagWaitGiveUps];
  if (entries_in_use != nullptr) *entries_in_use = busy;
  return SOFTMAX_OK;
}

SOFTMAX_API int softmax_exp_probe(const float* x, const float* m, float* e, int64_t n,
                                  float clip_lo, int approx, hipStream_t stream) {
  Clip c;
  bool wide = false;
  if (make_clip(clip_lo, &c, &wide) != SOFTMAX_OK) return SOFTMAX_ERR_INVALID_ARG;
  if (approx < 0 || approx > 2) return SOFTMAX_ERR_INVALID_ARG;
  if (n < 0 || n > INT64_MAX / 4) return SOFTMAX_ERR_INVALID_ARG;
  if (n == 0) return SOFTMAX_OK;
  if (x == nullptr || e == nullptr || (m == nullptr && approx != 2))
    return SOFTMAX_ERR_INVALID_ARG;
  if (any_overlap(e, x, n * 4) || (m != nullptr && any_overlap(e, m, n * 4)))
    return SOFTMAX_ERR_INVALID_ARG;
  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return fail_hip(he);
  int rc = check_device_range(x, n * 4, dev);
  if (rc == SOFTMAX_OK && m != nullptr) rc = check_device_range(m, n * 4, dev);
  if (rc == SOFTMAX_OK) rc = check_device_range(e, n * 4, dev);
  if (rc != SOFTMAX_OK) return rc;
  const int64_t grid = std::min(ceil_div(n, 256), kMaxGrid);
  void* args[] = {&x, &m, &e, &n, &c};
  const void* fn = approx == 2 ? reinterpret_cast<const void*>(&k_exp_probe<kExpRaw>)
                   : approx    ? reinterpret_cast<const void*>(&k_exp_probe<kExpFast>)
                   : wide      ? reinterpret_cast<const void*>(&k_exp_probe<kExpWide>)
                               : reinterpret_cast<const void*>(&k_exp_probe<kExpAccurate>);
  he = launch(fn, grid, 256, args, stream);
  return he == hipSuccess ? SOFTMAX_OK : fail_hip(he);
}

SOFTMAX_API int softmax_copy_probe(const float* x, float* y, int64_t n, hipStream_t stream) {
  if (n < 0 || n > INT64_MAX / 4) return SOFTMAX_ERR_INVALID_ARG;
  if (n == 0) return SOFTMAX_OK;
  if (x == nullptr || y == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (partial_overlap(x, y, n * 4)) return SOFTMAX_ERR_INVALID_ARG;
  int dev = 0;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return fail_hip(he);
  int rc = check_device_range(x, n * 4, dev);
  if (rc == SOFTMAX_OK && y != x) rc = check_device_range(y, n * 4, dev);
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
