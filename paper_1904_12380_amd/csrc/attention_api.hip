// C ABI of the fused softmax attention: argument checks and the launch.
// Declaration and contract: include/softmax_mi355x.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "../../include/softmax_mi355x.h"
#include "sm_attention.hpp"
#include "sm_host.hpp"

namespace {

using namespace smx;
using namespace smx_host;

// Workgroups per CU for the persistent grid (each holds 4 wavefronts of one
// batch element's 64-query block at a time).
constexpr int64_t kAttnBlocksPerCU = 8;

// sizes: all >= 0, lk in [1, 64] when there is work, d and dv at most
// SOFTMAX_ATTN_MAX_DIM, and every tensor's byte count fits in int64.
int check_attention_sizes(int64_t batch, int64_t lq, int64_t lk, int64_t d, int64_t dv) {
  if (batch < 0 || lq < 0 || lk < 0 || d < 0 || dv < 0) return SOFTMAX_ERR_INVALID_ARG;
  if (lq > INT32_MAX / 2 || d > SOFTMAX_ATTN_MAX_DIM || dv > SOFTMAX_ATTN_MAX_DIM)
    return SOFTMAX_ERR_INVALID_ARG;
  if (lk > SOFTMAX_ATTN_MAX_KEYS) return SOFTMAX_ERR_INVALID_ARG;
  if (batch == 0 || lq == 0 || dv == 0) return SOFTMAX_OK;
  if (lk == 0) return SOFTMAX_ERR_INVALID_ARG;
  const int64_t per_q = lq * std::max<int64_t>(d, dv);
  const int64_t per_k = lk * std::max<int64_t>(d, dv);
  if (batch > INT64_MAX / 4 / std::max(per_q, per_k)) return SOFTMAX_ERR_INVALID_ARG;
  return SOFTMAX_OK;
}

template <int NKT, bool VEC4, bool WIDE>
hipError_t run_attention(const float* q, const float* k, const float* v, float* o,
                         int64_t batch, int lq, int lk, int d, int dv, float scale, Clip c,
                         int64_t cus, hipStream_t s) {
  const int64_t items = batch * ((lq + 63) / 64);
  const int64_t grid = std::min(items, kAttnBlocksPerCU * cus);
  void* args[] = {&q, &k, &v, &o, &batch, &lq, &lk, &d, &dv, &scale, &c};
  return launch(reinterpret_cast<const void*>(&k_attention<NKT, VEC4, WIDE>), grid, 256, args,
                s);
}

// LDS-staged kernel: two workgroups per CU (80 KiB of LDS each).
constexpr int64_t kAttnLdsBlocksPerCU = 2;

template <int NKT, bool WIDE>
hipError_t run_attention_lds(const float* q, const float* k, const float* v, float* o,
                             int64_t batch, int lq, int lk, int d, int dv, float scale, Clip c,
                             int64_t cus, hipStream_t s) {
  const int64_t items = batch * ((lq + 63) / 64);
  const int64_t grid = std::min(items, kAttnLdsBlocksPerCU * cus);
  void* args[] = {&q, &k, &v, &o, &batch, &lq, &lk, &d, &dv, &scale, &c};
  return launch(reinterpret_cast<const void*>(&k_attention_lds<NKT, WIDE>), grid, 256, args, s);
}

// The DAM tile (d = dv = 200, 49 or 50 keys) with d known at compile time,
// on the ping-pong schedule: one workgroup of 8 wavefronts per CU, 160 KiB
// of LDS (two buffers of K_b, V_b and a zero row).  The kernel scores the
// last key tile on the VALU and needs at most 2 keys there.
constexpr int kAttnDamDim = 200;

bool dam_tile(int lk, int d, int dv) {
  return d == kAttnDamDim && dv == kAttnDamDim && lk > 48 && lk <= 50 &&
         (lk * (d + dv) + dv + 16) * 4 <= kAttnLdsBytes;
}

template <bool WIDE>
hipError_t run_attention_dam(const float* q, const float* k, const float* v, float* o,
                             int64_t batch, int lq, int lk, int d, int dv, float scale, Clip c,
                             int64_t cus, hipStream_t s) {
  const int64_t items = batch * ((lq + 63) / 64);
  const int64_t grid = std::min(items, cus);
  void* args[] = {&q, &k, &v, &o, &batch, &lq, &lk, &d, &dv, &scale, &c};
  return launch(reinterpret_cast<const void*>(&k_attention_pp<4, WIDE, kAttnDamDim>), grid, 512,
                args, s);
}

template <bool WIDE>
hipError_t dispatch_attention_lds(const float* q, const float* k, const float* v, float* o,
                                  int64_t batch, int lq, int lk, int d, int dv, float scale,
                                  Clip c, int64_t cus, hipStream_t s) {
  switch ((lk + 15) / 16) {
    case 1: return run_attention_lds<1, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    case 2: return run_attention_lds<2, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    case 3: return run_attention_lds<3, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    default: return run_attention_lds<4, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
  }
}

template <bool VEC4, bool WIDE>
hipError_t dispatch_attention(const float* q, const float* k, const float* v, float* o,
                              int64_t batch, int lq, int lk, int d, int dv, float scale,
                              Clip c, int64_t cus, hipStream_t s) {
  switch ((lk + 15) / 16) {
    case 1: return run_attention<1, VEC4, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    case 2: return run_attention<2, VEC4, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    case 3: return run_attention<3, VEC4, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
    default: return run_attention<4, VEC4, WIDE>(q, k, v, o, batch, lq, lk, d, dv, scale, c, cus, s);
  }
}

}  // namespace

extern "C" {

SOFTMAX_API int softmax_attention_fwd(const float* q, const float* k, const float* v,
                                      float* o, int64_t batch, int64_t lq, int64_t lk,
                                      int64_t d, int64_t dv, float scale, float clip_lo,
                                      hipStream_t stream) {
  Clip c;
  bool wide = false;
  int rc = make_clip(clip_lo, &c, &wide);
  if (rc != SOFTMAX_OK) return rc;
  if (!std::isfinite(scale)) return SOFTMAX_ERR_INVALID_ARG;
  rc = check_attention_sizes(batch, lq, lk, d, dv);
  if (rc != SOFTMAX_OK) return rc;
  if (batch == 0 || lq == 0 || dv == 0) return SOFTMAX_OK;

  const int64_t qbytes = batch * lq * d * 4;
  const int64_t kbytes = batch * lk * d * 4;
  const int64_t vbytes = batch * lk * dv * 4;
  const int64_t obytes = batch * lq * dv * 4;
  if (o == nullptr || v == nullptr) return SOFTMAX_ERR_INVALID_ARG;
  if (d > 0 && (q == nullptr || k == nullptr)) return SOFTMAX_ERR_INVALID_ARG;
  // The output may not overlap any input.
  const uintptr_t po = reinterpret_cast<uintptr_t>(o);
  auto overlaps = [&](const float* p, int64_t n) {
    const uintptr_t pp = reinterpret_cast<uintptr_t>(p);
    return n > 0 && pp < po + static_cast<uintptr_t>(obytes) &&
           po < pp + static_cast<uintptr_t>(n);
  };
  if (overlaps(q, qbytes) || overlaps(k, kbytes) || overlaps(v, vbytes))
    return SOFTMAX_ERR_INVALID_ARG;

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e);
  if (qbytes > 0 && (rc = check_device_range(q, qbytes, dev)) != SOFTMAX_OK) return rc;
  if (kbytes > 0 && (rc = check_device_range(k, kbytes, dev)) != SOFTMAX_OK) return rc;
  if ((rc = check_device_range(v, vbytes, dev)) != SOFTMAX_OK) return rc;
  if ((rc = check_device_range(o, obytes, dev)) != SOFTMAX_OK) return rc;

  int cus = 0;
  if ((rc = device_cus(dev, &cus)) != SOFTMAX_OK) return rc;
  // 128-bit accesses for every operand, or 32-bit ones for all of them.
  const bool vec4 = d % 4 == 0 && dv % 4 == 0 && aligned16(q) && aligned16(k) &&
                    aligned16(v) && aligned16(o);
  const int ilq = static_cast<int>(lq), ilk = static_cast<int>(lk);
  const int id = static_cast<int>(d), idv = static_cast<int>(dv);
  // K_b and V_b staged in LDS when they fit and every access is 128-bit.
  const bool lds = vec4 && d <= kAttnMaxDQ && lk * (d + dv) * 4 <= kAttnLdsBytes;
  if (lds && dam_tile(ilk, id, idv))
    e = wide ? run_attention_dam<true>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c, cus, stream)
             : run_attention_dam<false>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c, cus,
                                        stream);
  else if (lds)
    e = wide ? dispatch_attention_lds<true>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                            cus, stream)
             : dispatch_attention_lds<false>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                             cus, stream);
  else if (vec4)
    e = wide ? dispatch_attention<true, true>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                              cus, stream)
             : dispatch_attention<true, false>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                               cus, stream);
  else
    e = wide ? dispatch_attention<false, true>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                               cus, stream)
             : dispatch_attention<false, false>(q, k, v, o, batch, ilq, ilk, id, idv, scale, c,
                                                cus, stream);
  return e == hipSuccess ? SOFTMAX_OK : fail_hip(e);
}

}  // extern "C"
