// Device primitives for the clipped row softmax on CDNA4 (gfx950, wave64).
//
//   * exp_shift_clip(): e = exp(max(x - M, -64)) with the shift carried as an
//     exact double-float and the exp argument in extended precision, so the
//     result is within about 1.5 ulp of the true value over the whole clipped
//     range (the clip is the ValueClip of the paper's reference functor,
//     Sec. 1.2 Fig. 1; the bound -64 is this library's documented choice).
//   * seg_max / seg_sum: reductions over aligned groups of W lanes using DPP
//     (quad_perm, row_half_mirror, row_mirror) inside a 16-lane row and the
//     gfx950 permlane16/permlane32 swaps across rows.  These play the part of
//     the paper's SIMD horizontal reductions (Sec. 2.4.2 sum, Sec. 2.5 max)
//     on a 64-lane wavefront.  Every lane of a group ends with the same bits.
//
// Floating-point contraction is off for this whole library (-ffp-contract=off
// on the command line and the pragma below): the two-sum below is only exact
// if the compiler keeps every rounding step as written.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace smx {

// Lower bound applied to the shifted logit x - max before exp.
constexpr float kClipLo = -64.0f;

// log2(e) split into fp32 parts: hi = RN(log2 e), lo = RN(log2 e - hi).
constexpr float kLog2eHi = 0x1.715476p+0f;   // 1.44269502162933349609375
constexpr float kLog2eLo = 0x1.4ae0c0p-26f;  // 1.925963033500011e-08
// RN(ln 2): only scales the tiny low-order part of the exponent.
constexpr float kLn2 = 0x1.62e430p-1f;

__device__ __forceinline__ float fma_(float a, float b, float c) {
  return __builtin_fmaf(a, b, c);
}

// exp(max(x + neg_m, kClipLo)) where neg_m = -(row max).
//
// 1. Knuth's two-sum gives d = x + neg_m exactly as dh + dl (|dl| <= ulp/2).
// 2. The clip is decided on the exact d: d < L  <=>  dh < L or (dh == L and
//    dl < 0), because L = -64 is an fp32 value and rounding is monotonic.
//    A compare-select (not an IEEE max) keeps NaN as NaN; d = -inf clips.
// 3. t = c * log2(e) as th + tl: th = RN(ch * hi); tl gathers the product's
//    rounding error (one fma, exact), ch * lo and cl * hi.
// 4. e = 2^th * 2^tl ~= v_exp_f32(th) * (1 + tl * ln2); |tl| <= 4e-6, so the
//    dropped quadratic term is below 1e-11 relative.
// Domain after the clip: th in [-92.33, 0], so 2^th is a normal fp32 and
// v_exp_f32 needs no denormal scaling.
__device__ __forceinline__ float exp_shift_clip(float x, float neg_m) {
  const float dh = x + neg_m;
  const float xv = dh - neg_m;
  const float mv = dh - xv;
  const float dl = (x - xv) + (neg_m - mv);
  const bool clip = (dh < kClipLo) || ((dh == kClipLo) && (dl < 0.0f));
  const float ch = clip ? kClipLo : dh;
  const float cl = clip ? 0.0f : dl;
  const float th = ch * kLog2eHi;
  float tl = fma_(ch, kLog2eHi, -th);
  tl = fma_(ch, kLog2eLo, tl);
  tl = fma_(cl, kLog2eHi, tl);
  const float e0 = __builtin_amdgcn_exp2f(th);
  return fma_(e0, tl * kLn2, e0);
}

// ---------------------------------------------------------------------------
// Cross-lane moves.
// DPP control words (gfx9 encoding).
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm:[1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm:[2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror (8-lane reverse)
constexpr int kDppMirror = 0x140;     // row_mirror (16-lane reverse)

template <int Ctrl>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), Ctrl,
                                         0xF, 0xF, false));
}

// Value held by the partner 16-lane row (rows 0<->1, 2<->3).
__device__ __forceinline__ float row16_partner(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto p = __builtin_amdgcn_permlane16_swap(iv, iv, false, false);
  // p[0]: odd rows now hold the even rows' values; p[1]: even rows hold the
  // odd rows' values.  Each lane picks the one that is not its own row.
  return __builtin_bit_cast(float, ((__lane_id() >> 4) & 1) ? p[0] : p[1]);
}

// Value held by the partner 32-lane half (lanes 0-31 <-> 32-63).
__device__ __forceinline__ float half32_partner(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto p = __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
  return __builtin_bit_cast(float, (__lane_id() >> 5) ? p[0] : p[1]);
}

// Max over aligned groups of W lanes (W = 1, 2, 4, ..., 64); every lane of a
// group returns the group maximum.  NaN handling follows v_max_f32; callers
// never rely on the max to propagate NaN (the exp/sum stage does that).
template <int W>
__device__ __forceinline__ float seg_max(float v) {
  static_assert(W >= 1 && W <= 64 && (W & (W - 1)) == 0, "W: power of 2");
  if constexpr (W >= 2) v = fmaxf(v, dpp_mov<kDppQuadSwap1>(v));
  if constexpr (W >= 4) v = fmaxf(v, dpp_mov<kDppQuadSwap2>(v));
  if constexpr (W >= 8) v = fmaxf(v, dpp_mov<kDppHalfMirror>(v));
  if constexpr (W >= 16) v = fmaxf(v, dpp_mov<kDppMirror>(v));
  if constexpr (W >= 32) v = fmaxf(v, row16_partner(v));
  if constexpr (W >= 64) v = fmaxf(v, half32_partner(v));
  return v;
}

// Sum over aligned groups of W lanes, as a butterfly: at each level a lane
// adds its partner's partial, so all lanes of a group compute the same
// additions (fp add is commutative) and hold bit-identical totals.
template <int W>
__device__ __forceinline__ float seg_sum(float v) {
  static_assert(W >= 1 && W <= 64 && (W & (W - 1)) == 0, "W: power of 2");
  if constexpr (W >= 2) v = v + dpp_mov<kDppQuadSwap1>(v);
  if constexpr (W >= 4) v = v + dpp_mov<kDppQuadSwap2>(v);
  if constexpr (W >= 8) v = v + dpp_mov<kDppHalfMirror>(v);
  if constexpr (W >= 16) v = v + dpp_mov<kDppMirror>(v);
  if constexpr (W >= 32) v = v + row16_partner(v);
  if constexpr (W >= 64) v = v + half32_partner(v);
  return v;
}

// Pairwise (tree) sum of a register array, depth ceil(log2 N): keeps the
// per-lane rounding chain short on long rows.
template <int N>
__device__ __forceinline__ float tree_sum(const float (&a)[N]) {
  float t[N];
#pragma unroll
  for (int i = 0; i < N; ++i) t[i] = a[i];
#pragma unroll
  for (int stride = 1; stride < N; stride *= 2) {
#pragma unroll
    for (int i = 0; i + stride < N; i += 2 * stride) t[i] = t[i] + t[i + stride];
  }
  return t[0];
}

template <int N>
__device__ __forceinline__ float array_max(const float (&a)[N]) {
  float m = a[0];
#pragma unroll
  for (int i = 1; i < N; ++i) m = fmaxf(m, a[i]);
  return m;
}

}  // namespace smx
