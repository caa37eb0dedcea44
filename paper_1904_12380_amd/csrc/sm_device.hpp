// Device primitives for the clipped row softmax on CDNA4 (gfx950, wave64).
//
//   * exp_shift_clip(): e = exp(max(x - M, lo)) with the shift and the exp
//     argument in binary64 (full rate on gfx950) and v_exp_f32 on the fp32
//     part, so the result is within 1.5 ulp of the exact value over the
//     whole clipped range (the clip is the ValueClip of the paper's
//     reference functor, Sec. 1.2 Fig. 1; the default bound -64 is this
//     library's documented choice, and lo = -inf, no clip, is the optimised
//     functor of Sec. 2.3 Fig. 4).
//   * seg_max / seg_sum: reductions over aligned groups of W lanes using DPP
//     (quad_perm, row_half_mirror, row_mirror) inside a 16-lane row and the
//     gfx950 permlane16/permlane32 swaps across rows.  These play the part of
//     the paper's SIMD horizontal reductions (Sec. 2.4.2 sum, Sec. 2.5 max)
//     on a 64-lane wavefront.  Every lane of a group ends with the same bits.
//
// Floating-point contraction is off for this whole library (-ffp-contract=off
// on the command line and the pragma below), so every rounding step of the
// exp argument happens exactly as written.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace smx {

// Default lower bound applied to the shifted logit x - max before exp, and
// RN(e^-64), the value of every exponential it clips.
constexpr float kClipLo = -64.0f;
constexpr float kExpClipLo = 0x1.969d48p-93f;  // 1.6038109e-28

// Other bounds.  Bounds below kClipFloor, and no clip at all, run as
// kClipFloor with a clipped value of 0: every fp32 exponential below
// e^-103.98 rounds to 0, so the outputs are the same.  Bounds below
// kClipWide let unclipped exponentials fall under 2^-126 (denormal or 0),
// which needs the wide form of exp_shift_clip.
constexpr float kClipFloor = -128.0f;
constexpr float kClipWide = -87.0f;

// How a kernel evaluates the clipped exponential (a template argument):
//   kExpAccurate  binary64 argument, v_exp_f32 on the fp32 part (results
//                 normal: bounds >= kClipWide);
//   kExpWide      the same, plus the range below 2^-126 (bounds < kClipWide);
//   kExpFast      the single-instruction exponential on an fp32 argument,
//                 v_exp_f32(RN(RN(x - M) * RN(log2 e))): the cheaper
//                 approximation the paper suggests as further work (Sec. 4).
//                 Its relative error grows with |x - M|: below
//                 1.5e-7 |x - M| + 1.2e-7 where the result is normal; results
//                 under 2^-126 are flushed to 0.
constexpr int kExpAccurate = 0;
constexpr int kExpWide = 1;
constexpr int kExpFast = 2;
// A fourth kernel mode: the output is the log of the clipped softmax,
// y = c - ln S with c = max(x - M, lo), instead of e / S.  Its row sums
// take the cheap exponential term by term (the bound that allows it is at
// kSumExp; terms under 2^-126 do not matter next to S >= 1) and the
// accurate one to merge partial sums.
constexpr int kLogOut = 3;
// A fifth: one value per row, the negative log-likelihood of the row's
// label, ln S - c_label (minus the label's log output); sums as kLogOut.
constexpr int kNllOut = 4;
// Modes whose output step needs the logits rather than the exponentials.
template <int MODE>
constexpr bool keeps_logits() { return MODE == kLogOut || MODE == kNllOut; }
template <int MODE>
constexpr int exp_mode() { return keeps_logits<MODE>() ? kExpAccurate : MODE; }

// The clip as a kernel argument: lo in [kClipFloor, 0] and e_lo = RN(e^lo')
// for the caller's bound lo' (0 when lo' < -103.98 or lo' = -inf).
struct Clip {
  float lo;
  float e_lo;
  float lo_out;  // the caller's bound itself (may be -inf), for log outputs
};

// RN(log2 e) and RN(ln 2) in binary64.
constexpr double kLog2e = 0x1.71547652b82fep+0;
constexpr double kLn2 = 0x1.62e42fefa39efp-1;

// Native 4 x fp32 vector: loads and stores of it are single 128-bit
// accesses (global_load_dwordx4 / global_store_dwordx4).
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming 128-bit load and store: x is read once and y written once, so
// both use the nontemporal cache policy.  Stores at device coherence scope
// (sc1) instead were measured in the same process against these: faster on
// a plain copy of 64 MiB each way (22.4 against 23.3 us) and by 0.3 us on
// one 1024-thread workgroup per row of 32768 columns, but slower on the
// one-pass split rows of 64 x 262144 (23.9 against 22.6 us), on
// 4096 x 1000 (7.7 against 6.8) and on 115200 x 50 (9.2 against 8.7).
__device__ __forceinline__ f32x4 ld_stream(const float* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
__device__ __forceinline__ void st_stream(float* p, f32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}

// Per-row constants of the shifted, clipped exponential.
//   neg_m: -M in binary64.
//   tc:    the smallest fp32 value >= M + lo (computed exactly), so that for
//          every fp32 x:  x < tc  <=>  x - M < lo.  The clip test is then one
//          fp32 compare per element.  M = NaN gives tc = NaN (no element is
//          clipped and NaN propagates); M = -inf gives tc = -inf.
//   e_lo:  the value of a clipped exponential.
struct RowShift {
  double neg_m;
  float m;
  float tc;
  float e_lo;
  float tc_out;  // as tc, for the caller's bound (log outputs)
  float lo_out;
};

// The smallest fp32 value >= s (s in binary64).
__device__ __forceinline__ float round_up_f32(double s) {
  float f = static_cast<float>(s);
  if (static_cast<double>(f) < s) {
    // next fp32 towards +inf (f < s <= f + ulp, f finite)
    const unsigned u = __builtin_bit_cast(unsigned, f);
    f = __builtin_bit_cast(float, f < 0.0f ? u - 1u : (f == 0.0f ? 1u : u + 1u));
  }
  return f;
}

__device__ __forceinline__ RowShift row_shift(float m, Clip clip) {
  RowShift r;
  r.neg_m = -static_cast<double>(m);
  r.m = m;
  // M + lo is exact in binary64 unless the exponents of M and lo differ by
  // more than 29 (|M| < 2^-23 |lo|), where the rounding is below 2^-47 |lo|
  // and only moves the boundary by that much.
  r.tc = round_up_f32(static_cast<double>(m) + static_cast<double>(clip.lo));
  r.e_lo = clip.e_lo;
  r.tc_out = round_up_f32(static_cast<double>(m) + static_cast<double>(clip.lo_out));
  r.lo_out = clip.lo_out;
  return r;
}

// ln S = RN(v_log_f32(S) * RN(ln 2)): log2 within 1 ulp, one product
// rounding; S >= 1 for every row with a finite max.
__device__ __forceinline__ float log_of_sum(float s) {
  return __builtin_amdgcn_logf(s) * 0x1.62e430p-1f;
}

// One log-softmax output: y = RN(c - ln S) with c = RN(x - M), or the
// caller's bound itself where x - M is below it; with no clip a -inf entry
// gives -inf.  Three fp32 roundings and ln S's error: within
// 1.2e-7 |y| + 2.4e-7 ln S of c - ln S, under the header's bound.
__device__ __forceinline__ float log_out(float x, RowShift rs, float log_s) {
  const float c = x < rs.tc_out ? rs.lo_out : x - rs.m;
  return c - log_s;
}

// exp(max(x - M, lo)) for fp32 x, within 1.5 ulp of the exact value where
// that is a normal fp32, and within 2^-150 plus 1.5 ulp-relative (the error
// carried into the final rounding onto the denormal grid) below it.
//
// 1. d = x - M in binary64: exact whenever the exponents of x and M differ by
//    at most 29; otherwise its relative error is below 2^-53.
// 2. t = d * log2(e) in binary64, th = RN32(t), and the remainder
//    r = d - th * ln2 from one binary64 fma (|r| <= 2^-18 * ln2 = 2.6e-6).
// 3. e = 2^th * e^r = v_exp_f32(th) * (1 + r), rounded once by an fp32 fma;
//    the dropped r^2/2 is below 4e-12.  With lo >= kClipWide, th stays in
//    [-125.6, 0], where 2^th is a normal fp32.
// 4. kExpWide (lo < kClipWide): v_exp_f32 returns no denormals, so for
//    th < -126 the fma works on 2^(th+64) (exact shift, th >= -185 since
//    lo >= kClipFloor) and one final multiplication by 2^-64 rounds the
//    result into the denormal range.
// 5. Clipped elements (x < tc) return e_lo; this also covers x = -inf.
//    NaN inputs, and rows whose max is +inf or -inf, give NaN.
template <int EM>
__device__ __forceinline__ float exp_shift_clip(float x, RowShift rs) {
  if constexpr (EM == kExpFast) {
    const float t = (x - rs.m) * 0x1.715476p+0f;     // RN(log2 e) in fp32
    const float e = __builtin_amdgcn_exp2f(t);
    return x < rs.tc ? rs.e_lo : e;
  }
  const double d = static_cast<double>(x) + rs.neg_m;
  const double t = d * kLog2e;
  const float th = static_cast<float>(t);
  const double r = __builtin_fma(static_cast<double>(th), -kLn2, d);
  float e;
  if constexpr (EM == kExpWide) {
    const bool tiny = th < -126.0f;
    const float e0 = __builtin_amdgcn_exp2f(tiny ? th + 64.0f : th);
    const float ew = __builtin_fmaf(e0, static_cast<float>(r), e0);
    e = tiny ? ew * 0x1p-64f : ew;
  } else {
    const float e0 = __builtin_amdgcn_exp2f(th);
    e = __builtin_fmaf(e0, static_cast<float>(r), e0);
  }
  return x < rs.tc ? rs.e_lo : e;
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
