// Cross-workgroup exchange for rows split over several workgroups, and the
// wall-clock store schedule of the one-wave row kernels.
//
// The exchange lives in a fixed table of row entries in a static device
// array (the library allocates no memory).  The workgroups of one row meet
// at one entry: entry (base + row) mod kEntries, where the host gives every
// launch a base from a per-device cursor that advances by the launch's row
// count, so the rows of a launch take consecutive entries and launches in
// flight together take disjoint ones while they hold fewer than kEntries
// rows between them.  The first workgroup of the row to arrive claims the
// entry with a compare-and-swap of its owner word from 0 to the row's tag
// (a hash of the launch's key and the row; the key mixes the output
// address with a per-call nonce); the others find the tag there and join.
// Each publishes a partial pair in its slot, and the last to leave puts the
// entry back to rest (slots, counter and owner zero).  A row whose entry is
// still held (by a launch kEntries rows of split-row work earlier, or by a
// second replay of the same graph) waits for it.  So calls on any number
// of streams, graphs replayed at the same time, and a first call made under
// stream capture all work without host-side synchronisation, and every
// atomic is shared only by the workgroups of one row.
//
// Rows that waited for an entry held by another launch could deadlock: the
// waiting workgroups hold compute-unit slots that the holder's remaining
// workgroups need.  Disjoint bases keep concurrent launches from ever
// waiting on each other; the bounded wait turns what is left into a NaN
// row (counted) rather than a hang.
//
// Every wait is bounded by the wall clock.  A workgroup that gives up
// counts itself in a give-up counter (readable from the host), writes NaN
// for its outputs, and leaves the entry alone.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace smx {
namespace xch {

constexpr int kEntries = 4096;        // row entries per device
constexpr int kEntrySlots = 64;       // 64-bit slots per entry: one per workgroup of the row
constexpr int kHeaderWords = 8;       // owner, departures: one 64-byte line
constexpr int kEntryWords = kHeaderWords + kEntrySlots;   // 576 bytes
constexpr int kDiagWord = kEntries * kEntryWords;          // give-up counters
constexpr int kDiagWords = 32;
constexpr int64_t kScratchWords = int64_t(kDiagWord) + kDiagWords;
constexpr int64_t kScratchBytes = kScratchWords * 8;       // 2,359,552 bytes
// Rows per launch: a launch's rows take distinct entries.
constexpr int kMaxRowsPerLaunch = 1024;

// Diagnostic counters (64-bit words after the entries).
constexpr int kDiagJoinGiveUps = 0;   // the row's entry stayed in use by another row
constexpr int kDiagWaitGiveUps = 1;   // a row's partials did not all arrive in time

// Bound of every wait, in microseconds of wall clock.
constexpr uint32_t kWaitLimitUs = 20000;

static_assert((kEntries & (kEntries - 1)) == 0, "entry index is a mask");
static_assert(kMaxRowsPerLaunch <= kEntries, "a launch's rows never share an entry");

__device__ __forceinline__ uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_agent32(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t add_agent(uint64_t* p, uint64_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A 64-bit mix (the finaliser of SplitMix64).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace xch

// The constant-rate wall clock (s_memrealtime; its rate is the device's
// wall-clock attribute, read by the host).
__device__ __forceinline__ uint64_t wall_clock() { return __builtin_amdgcn_s_memrealtime(); }

// Holds the calling wavefront until the wall clock reaches t.
__device__ __forceinline__ void wait_until(uint64_t t) {
  while (static_cast<int64_t>(wall_clock() - t) < 0) __builtin_amdgcn_s_sleep(2);
}

// wait_until, once `v` has been computed: the row sum is then final and its
// partial terms are dead, so the wait keeps no more registers live than the
// stores need.
__device__ __forceinline__ void wait_until_after(uint64_t t, float v) {
  asm volatile("" : : "v"(v));
  wait_until(t);
}

// A launch's exchange context: the scratch table, the call's key, the wait
// limit in wall-clock ticks, and whether the launch's workgroups may claim
// a free entry (join) or only find the one their row already holds (the
// second pass of the two-pass kernels).
struct XchArgs {
  uint64_t* scratch;
  uint64_t key;
  uint32_t limit_ticks;
  uint32_t join;
  uint32_t base;  // entry of the launch's row 0 (mod kEntries)
  uint32_t unused;
};

// Entry of row `lrow` of the launch, joined (or, with a.join == 0, found)
// by the calling lane; null once `deadline` has passed.
__device__ __forceinline__ uint64_t* row_entry(const XchArgs& a, int lrow, uint64_t deadline) {
  using namespace xch;
  const uint64_t h = mix64(a.key);
  const int e = static_cast<int>((a.base + static_cast<uint32_t>(lrow)) & (kEntries - 1));
  uint64_t tag = mix64(h ^ (static_cast<uint64_t>(lrow) * 0x9E3779B97F4A7C15ull));
  if (tag == 0) tag = 1;
  uint64_t* entry = a.scratch + int64_t(e) * kEntryWords;
  while (true) {
    uint64_t seen;
    if (a.join) {
      uint64_t expected = 0;
      __hip_atomic_compare_exchange_strong(&entry[0], &expected, tag, __ATOMIC_RELAXED,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      seen = expected;  // 0 if this call claimed it, else the owner it found
      if (seen == 0 || seen == tag) return entry;
    } else {
      seen = ld_agent(&entry[0]);
      if (seen == tag) return entry;
    }
    if (static_cast<int64_t>(wall_clock() - deadline) > 0) return nullptr;
    __builtin_amdgcn_s_sleep(2);
  }
}

// Counts a give-up of kind `which` (one lane calls it).
__device__ __forceinline__ void count_give_up(const XchArgs& a, int which) {
  xch::add_agent(&a.scratch[xch::kDiagWord + which], 1ull);
}

// Slots hold ~pack(m, s), so that 0 means empty; a pair whose packing is
// all ones (a NaN pattern) is published as the canonical NaN pair instead.
__device__ __forceinline__ uint64_t encode_pair(float m, float s) {
  uint64_t v = static_cast<uint64_t>(__builtin_bit_cast(uint32_t, m)) |
               (static_cast<uint64_t>(__builtin_bit_cast(uint32_t, s)) << 32);
  if (v == ~0ull) {
    const uint64_t qnan = __builtin_bit_cast(uint32_t, __builtin_nanf(""));
    v = qnan | (qnan << 32);
  }
  return ~v;
}
__device__ __forceinline__ float decode_m(uint64_t e) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(~e));
}
__device__ __forceinline__ float decode_s(uint64_t e) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(~e >> 32));
}

__device__ __forceinline__ uint64_t* entry_slots(uint64_t* entry) {
  return entry + xch::kHeaderWords;
}

// Called by one lane once its workgroup is finished with its row's entry
// (every read of the row's slots by this workgroup has returned): counts the
// workgroup out (inc is 1; callers pass it through a register that depends
// on their last slot read, so that the count cannot be issued before that
// read has returned), and returns true for the last of the row's `g`
// workgroups, which then releases the entry (release_entry).
__device__ __forceinline__ bool depart_entry(uint64_t* entry, int g, uint32_t inc) {
  uint32_t* depart = reinterpret_cast<uint32_t*>(entry + 1);
  const uint32_t old = xch::add_agent32(depart, inc);
  return old == static_cast<uint32_t>(g) - 1u;
}

// Last step of the last workgroup of a row, by one lane of the wavefront
// that stored zero into the row's slots (the wait below covers those
// stores): resets the departure count, then frees the entry.
__device__ __forceinline__ void release_entry(uint64_t* entry) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(entry + 1), 0u, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_s_waitcnt(0);
  xch::st_agent(&entry[0], 0ull);
}

}  // namespace smx
