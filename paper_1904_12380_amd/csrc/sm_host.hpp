// Host-side helpers shared by the library's C entry points: argument and
// pointer checks, the clip argument, error recording and launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>
#include <mutex>

#include "../../include/softmax_mi355x.h"
#include "sm_device.hpp"

namespace smx_host {

using smx::Clip;
using smx::kClipFloor;
using smx::kClipLo;
using smx::kClipWide;
using smx::kExpClipLo;

// hipError_t of the last SOFTMAX_ERR_HIP returned on this thread, shared by
// every entry point of the library.
inline thread_local int tl_last_hip_error = 0;

// Largest grid any launch uses; the kernels loop over the rest.
constexpr int64_t kMaxGrid = int64_t(1) << 20;

inline bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline int fail_hip(hipError_t e) {
  tl_last_hip_error = static_cast<int>(e);
  return SOFTMAX_ERR_HIP;
}

// Byte ranges [a, a+n) and [b, b+n) overlap without being identical.
inline bool partial_overlap(const void* a, const void* b, int64_t n) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a);
  const uintptr_t pb = reinterpret_cast<uintptr_t>(b);
  if (pa == pb) return false;
  return pa < pb + static_cast<uintptr_t>(n) && pb < pa + static_cast<uintptr_t>(n);
}

// Byte ranges [a, a+na) and [b, b+nb) share a byte (empty ranges never do).
inline bool ranges_overlap(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a);
  const uintptr_t pb = reinterpret_cast<uintptr_t>(b);
  return na > 0 && nb > 0 && pa < pb + static_cast<uintptr_t>(nb) &&
         pb < pa + static_cast<uintptr_t>(na);
}

inline bool any_overlap(const void* a, const void* b, int64_t n) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a);
  const uintptr_t pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + static_cast<uintptr_t>(n) && pb < pa + static_cast<uintptr_t>(n);
}

// The device can use [p, p+bytes): memory registered with HIP, on the
// current device when it is device memory, and inside one allocation.
inline int check_device_range(const void* p, int64_t bytes, int dev) {
  hipPointerAttribute_t a;
  hipError_t e = hipPointerGetAttributes(&a, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return SOFTMAX_ERR_NOT_DEVICE;
  }
  if (a.type == hipMemoryTypeDevice) {
    if (a.device != dev) return SOFTMAX_ERR_NOT_DEVICE;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void*>(p));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return SOFTMAX_ERR_NOT_DEVICE;
    }
    const uintptr_t lo = reinterpret_cast<uintptr_t>(base);
    const uintptr_t pp = reinterpret_cast<uintptr_t>(p);
    if (pp < lo || pp + static_cast<uintptr_t>(bytes) > lo + size)
      return SOFTMAX_ERR_NOT_DEVICE;
    return SOFTMAX_OK;
  }
  // Pinned (registered) host memory and managed memory are usable by the
  // device; unregistered pageable memory is not.
  if (a.type == hipMemoryTypeHost || a.type == hipMemoryTypeManaged) return SOFTMAX_OK;
  return SOFTMAX_ERR_NOT_DEVICE;
}

// Compute units of device `dev` (hipDeviceAttributeMultiprocessorCount),
// queried once per device: persistent grids and the one-pass launches are
// sized from it rather than from MI355X's 256.
constexpr int kMaxDevices = 64;
inline std::mutex g_cu_mu;
inline int g_cu_count[kMaxDevices] = {};

inline int device_cus(int dev, int* cus) {
  if (dev < 0 || dev >= kMaxDevices) return SOFTMAX_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_cu_mu);
  if (g_cu_count[dev] == 0) {
    int n = 0;
    const hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return fail_hip(e);
    if (n <= 0) return SOFTMAX_ERR_INVALID_ARG;
    g_cu_count[dev] = n;
  }
  *cus = g_cu_count[dev];
  return SOFTMAX_OK;
}

inline hipError_t launch(const void* fn, int64_t grid, int block, void** args, hipStream_t s) {
  return hipLaunchKernel(fn, dim3(static_cast<uint32_t>(grid)), dim3(block), args, 0, s);
}

// The clip as the kernels take it, from the caller's bound: NaN and bounds
// above SOFTMAX_CLIP_MAX are rejected; bounds below kClipFloor (and -inf)
// run at kClipFloor with clipped value RN(e^bound) = 0.
inline int make_clip(float clip_lo, Clip* c, bool* wide) {
  if (!(clip_lo <= SOFTMAX_CLIP_MAX)) return SOFTMAX_ERR_INVALID_ARG;  // NaN too
  c->lo = clip_lo < kClipFloor ? kClipFloor : clip_lo;
  c->e_lo = clip_lo == kClipLo ? kExpClipLo
                               : static_cast<float>(std::exp(static_cast<double>(clip_lo)));
  c->lo_out = clip_lo;
  *wide = c->lo < kClipWide;
  return SOFTMAX_OK;
}

}  // namespace smx_host
