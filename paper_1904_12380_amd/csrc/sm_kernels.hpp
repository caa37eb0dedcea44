// HIP kernels for the clipped row softmax on gfx950.
//
// Every kernel computes, per row of a row-major [rows, cols] fp32 matrix,
//   y = exp(max(x - rowmax, lo)) / sum(exp(max(x - rowmax, lo)))
// in the order of the paper's optimised functor (Sec. 2.3, Fig. 4: row max,
// subtract, exp, row sum, scale by the reciprocal of the sum) with the clip
// of the reference functor (Sec. 1.2, Fig. 1) at a bound lo given as a
// kernel argument (default -64; no clip runs as the floor bound with a
// clipped value of 0).  The MODE template argument says how the exponential
// is evaluated (accurate, accurate into the denormal range, or the fast
// approximation) or what is written instead of y: its logarithm, or one
// negative log-likelihood per row.  Unlike the CPU functor, no kernel uses
// y as scratch: x is read from HBM once (twice for rows over 2^21 columns)
// and y is written once.
//
//   k_group_rows  cols <= 256 in whole 16-byte strips, probability
//                 outputs: G lanes per row, each holding one 128-bit strip
//                 as the coalesced load leaves it; segmented DPP reductions.
//   k_packed      cols <= 64 otherwise: a persistent workgroup stages tiles
//                 of whole rows in LDS with 128-bit loads, groups of G lanes
//                 reduce one row each with DPP, and the tile goes back out
//                 with 128-bit stores; the next tile's loads are issued early.
//   k_wave_row    cols <= 4096: one wavefront per row, the row held in VGPRs.
//   k_block_row   cols <= 8192 (32768 for log and NLL outputs): one
//                 workgroup per row, the row held in VGPRs, per-wave
//                 partials combined through LDS.
//   k_split_onepass   rows of up to 64 chunks: one workgroup per chunk,
//                 partials exchanged between the row's workgroups in the
//                 middle of the kernel, x read once.
//   k_split_stats / k_split_apply   longer rows: G workgroups per row; the
//                 first pass writes a (max, sum) partial per chunk, the
//                 second merges them and writes the chunk's outputs.
//
// In-place calls (x == y) are safe in every kernel: each element is read
// into registers (or LDS) by the workgroup that later writes it, before any
// write to it, and no workgroup reads another's outputs.
#pragma once

#include "sm_device.hpp"
#include "sm_exchange.hpp"

namespace smx {

constexpr float kNegInf = -__builtin_inff();

// ---------------------------------------------------------------------------
// Block-wide reductions (NW wavefronts).  A wave reduces with DPP, lane 0
// publishes to LDS, and after the barrier every thread combines the NW
// values in the same fixed order, so all threads hold identical bits.
template <int NW>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = seg_max<64>(v);
  if constexpr (NW == 1) return v;
  if (__lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) m = fmaxf(m, red[w]);
  return m;
}

template <int NW>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = seg_sum<64>(v);
  if constexpr (NW == 1) return v;
  if (__lane_id() == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float t[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) t[w] = red[w];
  return tree_sum(t);
}

// x itself, as a value the compiler cannot see through: store addresses
// built from it are formed just before the stores instead of being kept in
// registers from the loads (which share them) across the reductions.
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Loads N = 4*V elements of a row segment p[0, lim) into registers: element
// i of this lane sits at p[lane_off + stride*i] (scalar) or, for 128-bit
// loads, at p[4*(lane_off + stride*j) + k] with i = 4j + k.  Offsets are
// 32-bit (a segment is at most 2^20 columns), so the address is one base
// register plus a 32-bit lane offset.  Columns at or past `lim` read as
// -inf: they take part in the max as a neutral value and their clipped
// exponential (e^lo with lo <= -48, or 0 with no clip) changes a row sum of
// at least 1 by under 4096 e^-48 < 1e-17 relative, so no per-element mask
// is needed later.  Strip j covers [4*stride*j, 4*stride*(j+1)); when all
// of it is inside the segment (a uniform test) no lane is masked.
template <int V, bool VEC4>
__device__ __forceinline__ void load_strip(float (&v)[4 * V], const float* p, int lane_off,
                                           int stride, int lim) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int c = 4 * (lane_off + stride * j);
      f32x4 q;
      if (4 * stride * (j + 1) <= lim) {
        q = ld_stream(p + c);
      } else {
        q = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
        if (c < lim) q = ld_stream(p + c);
      }
      v[4 * j + 0] = q.x;
      v[4 * j + 1] = q.y;
      v[4 * j + 2] = q.z;
      v[4 * j + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      const int c = lane_off + stride * i;
      if (stride * (i + 1) <= lim)
        v[i] = __builtin_nontemporal_load(p + c);
      else
        v[i] = (c < lim) ? __builtin_nontemporal_load(p + c) : kNegInf;
    }
  }
}

// The same loads with no control flow between them (a column past the
// segment loads column 0 and is then replaced by -inf), for the online
// reduction below: each use then waits only for its own loads, not for the
// whole strip.  It keeps one offset register per strip live, so it is used
// only where the registers allow.  With 128-bit access lim is a multiple of
// 4 (a segment's four columns are all inside it or all past it).
template <int V, bool VEC4>
__device__ __forceinline__ void load_strip_flat(float (&v)[4 * V], const float* p,
                                                int lane_off, int stride, int lim) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int c = 4 * (lane_off + stride * j);
      const bool in = c < lim;
      const f32x4 q = ld_stream(p + (in ? c : 0));
      v[4 * j + 0] = in ? q.x : kNegInf;
      v[4 * j + 1] = in ? q.y : kNegInf;
      v[4 * j + 2] = in ? q.z : kNegInf;
      v[4 * j + 3] = in ? q.w : kNegInf;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      const int c = lane_off + stride * i;
      const bool in = c < lim;
      const float q = __builtin_nontemporal_load(p + (in ? c : 0));
      v[i] = in ? q : kNegInf;
    }
  }
}

// The exponential of the row-sum terms for log and NLL outputs.  Those
// outputs need ln S, not the terms, and the cheap exponential keeps ln S
// within their bound: a term at x - M = d has relative error at most
// 1.5e-7 |d| + 1.2e-7, and averaged with the softmax weights p,
// E_p[-d] = H(p) - ln S <= ln C - ln S (H the entropy).  So S is off by at
// most 1.5e-7 (ln C - ln S) + 1.2e-7 relative; with ln S's own 1.8e-7 ln S
// (v_log_f32 and the product by ln 2) and the sum's rounding, ln S stays
// within 2.5e-7 ln C + 2e-6.  For a row in chunks the terms are taken
// against the chunk max m_g <= M, so |x - m_g| <= |d| and the same average
// applies; merges of partial sums keep the accurate exponential (exp_mode).
constexpr int kSumExp = kExpFast;

// This lane's pairwise partial sum of the clipped exponentials.  For
// probability outputs v is replaced by the exponentials; for log and NLL
// outputs (keeps_logits) v keeps the logits, which the output step needs.
// SE: the exponential of the sum terms for log and NLL outputs (kSumExp,
// or the accurate one where the cheap one costs registers).
template <int MODE, int N, int SE = kSumExp>
__device__ __forceinline__ float exp_strip(float (&v)[N], RowShift rs) {
  if constexpr (keeps_logits<MODE>()) {
    // Eight interleaved partial sums, then their tree: no second array of N
    // registers next to the logits.
    constexpr int P = N < 8 ? N : 8;
    float t[P];
#pragma unroll
    for (int i = 0; i < P; ++i) t[i] = exp_shift_clip<SE>(v[i], rs);
#pragma unroll
    for (int i = P; i < N; ++i) t[i % P] = t[i % P] + exp_shift_clip<SE>(v[i], rs);
    return tree_sum(t);
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = exp_shift_clip<MODE>(v[i], rs);
    return tree_sum(v);
  }
}

// Lane-local online reduction of the logits in v, for the modes that keep
// them (log and NLL outputs) in the one-pass split kernel, whose chunks
// hold 32 values per lane (on shorter strips the extra rescaling costs more
// than the overlap gains): v is taken in sub-strips of 8 elements (two
// 128-bit loads) in load order, each reduced against the running lane max
// as soon as its own loads have returned, so the exponentials of the first
// columns overlap the arrival of the last instead of waiting for the whole
// row.  Returns the lane max m (-inf when every element is) and
// s = sum exp(max(x - m, lo)) over the lane's elements (shift 0 while m is
// -inf, where every term is the clipped value).  When the max grows the
// running sum is rescaled by the clipped exponential of the step; like a
// clip taken against a partial max, that changes S by at most cols * e^lo
// relative (under 1e-10 for lo <= -48).
template <int N, int SUB_MAX = 8>
__device__ __forceinline__ float2 lane_online(const float (&v)[N], Clip clip) {
  constexpr int SUB = N < SUB_MAX ? N : SUB_MAX;
  static_assert(N % SUB == 0, "whole sub-strips");
  float m = kNegInf;
  float s = 0.0f;
#pragma unroll
  for (int k0 = 0; k0 < N; k0 += SUB) {
    float mk = v[k0];
#pragma unroll
    for (int i = 1; i < SUB; ++i) mk = fmaxf(mk, v[k0 + i]);
    const float m_new = fmaxf(m, mk);
    const RowShift rs = row_shift(m_new == kNegInf ? 0.0f : m_new, clip);
    // two interleaved partials keep few exponentials live at once
    float p0 = exp_shift_clip<kSumExp>(v[k0], rs);
    float p1 = SUB > 1 ? exp_shift_clip<kSumExp>(v[k0 + 1], rs) : 0.0f;
#pragma unroll
    for (int i = 2; i < SUB; i += 2) {
      p0 = p0 + exp_shift_clip<kSumExp>(v[k0 + i], rs);
      if (i + 1 < SUB) p1 = p1 + exp_shift_clip<kSumExp>(v[k0 + i + 1], rs);
    }
    const float sk = p0 + p1;
    if (k0 == 0) {
      s = sk;
    } else {
      const float f = m == kNegInf ? 1.0f : exp_shift_clip<kExpAccurate>(m, rs);
      s = s * f + sk;
    }
    m = m_new;
    // Materialise this sub-strip's running (m, s) here: otherwise the
    // compiler sinks its exponentials to the next sub-strip and takes every
    // max first, which waits for all of the row's loads.
    asm volatile("" : "+v"(s), "+v"(m));
  }
  return make_float2(m, s);
}

// This lane's share of the row sum against the row max M (rs), from its
// lane_online result: s * exp(max(m - M, lo)), or s itself for a lane with
// no finite element.
template <int EM = kExpAccurate>
__device__ __forceinline__ float lane_share(float2 ms, RowShift rs) {
  return ms.x == kNegInf ? ms.y : ms.y * exp_shift_clip<EM>(ms.x, rs);
}

// Loads as load_strip, for a segment whose strips are all whole
// (lim = 4*V*stride): no masks and no control flow, and issued in order
// (the scheduling barriers keep the compiler from reordering them), so each
// use of a value waits only for the loads up to its own.
template <int V, bool VEC4>
__device__ __forceinline__ void load_strip_whole(float (&v)[4 * V], const float* p,
                                                 int lane_off, int stride) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const f32x4 q = ld_stream(p + 4 * (lane_off + stride * j));
      __builtin_amdgcn_sched_barrier(0);
      v[4 * j + 0] = q.x;
      v[4 * j + 1] = q.y;
      v[4 * j + 2] = q.z;
      v[4 * j + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      v[i] = __builtin_nontemporal_load(p + lane_off + stride * i);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// 128-bit access to a row segment p[0, lim) that starts `a` floats (0..3)
// past a 16-byte boundary: rows whose length is not a multiple of 4 in a
// 16-byte aligned matrix.  Lane strip j is the aligned float4 at
// p - a + 4 * (lane_off + stride * j), holding segment columns c0 .. c0 + 3
// with c0 = 4 * (lane_off + stride * j) - a; element 4 j + k of v is column
// c0 + k.  The strips must cover lim + a columns.  Every strip that holds a
// column of the segment is one 128-bit load, and columns outside [0, lim)
// are replaced by -inf after the load.  A straddling strip therefore also
// reads up to 3 floats of the neighbouring row, or, at the end of the
// matrix, up to 12 bytes past it inside the same 16-byte block, which lies
// in the same memory page as the row's last column; those values are never
// used.  (Element-wise loads in the straddling strips measured 1.5-10%
// slower on rows of 2049 to 8189 columns, from the extra instructions and
// divergence, and cost the split kernels 5-13 spilled VGPRs.)
template <int V>
__device__ __forceinline__ void load_strip_ph(float (&v)[4 * V], const float* p, int a,
                                              int lane_off, int stride, int lim) {
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int c0 = 4 * (lane_off + stride * j) - a;
    f32x4 q = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
    if (c0 < lim) q = ld_stream(p + c0);
    v[4 * j + 0] = (c0 + 0 >= 0 && c0 + 0 < lim) ? q.x : kNegInf;
    v[4 * j + 1] = (c0 + 1 >= 0 && c0 + 1 < lim) ? q.y : kNegInf;
    v[4 * j + 2] = (c0 + 2 >= 0 && c0 + 2 < lim) ? q.z : kNegInf;
    v[4 * j + 3] = (c0 + 3 >= 0 && c0 + 3 < lim) ? q.w : kNegInf;
  }
}

// Stores out(v[i]) for the columns of the segment, strips as load_strip_ph.
// A strip wholly inside [0, lim) is one 128-bit store; a strip that
// straddles either end of the segment writes only its columns inside it,
// with 32-bit stores, so nothing of a neighbouring row is written (in-place
// calls and other rows' outputs stay intact).
template <int V, typename F>
__device__ __forceinline__ void store_strip_ph(const float (&v)[4 * V], F out, float* p, int a,
                                               int lane_off, int stride, int lim) {
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int c0 = 4 * (lane_off + stride * j) - a;
    if (c0 >= 0 && c0 + 4 <= lim) {
      f32x4 q;
      q.x = out(v[4 * j + 0]);
      q.y = out(v[4 * j + 1]);
      q.z = out(v[4 * j + 2]);
      q.w = out(v[4 * j + 3]);
      st_stream(p + c0, q);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int c = c0 + k;
        if (c >= 0 && c < lim) __builtin_nontemporal_store(out(v[4 * j + k]), p + c);
      }
    }
  }
}

// Sub-strip length of the online reduction of the probability modes.
constexpr int kOnlineSub = 8;
// Whether a lane's N values take that reduction (two sub-strips at least).
template <int N>
constexpr bool online_exp() { return N >= 2 * kOnlineSub; }

// The probability modes' online form of a lane's reduction (lanes holding
// N >= 16 values, in load order): v is taken in sub-strips of kOnlineSub
// elements, and each is replaced by its clipped exponentials against the
// lane's running max as soon as its own loads have returned, so the
// exponential work overlaps the arrival of the rest of the segment instead
// of starting after its last load.  mk[k] keeps the running max that
// sub-strip k was taken against, for the output step (store_online).
// Returns the lane max m (-inf when every element is) and
// s = sum exp(max(x - m, lo)) over the lane's elements, with the same
// rescaling rule as lane_online.
template <int MODE, int N>
__device__ __forceinline__ float2 lane_online_exp(float (&v)[N], float (&mk)[N / kOnlineSub],
                                                  Clip clip) {
  constexpr int SUB = kOnlineSub;
  static_assert(N % SUB == 0, "whole sub-strips");
  float m = kNegInf;
  float s = 0.0f;
#pragma unroll
  for (int k0 = 0; k0 < N; k0 += SUB) {
    float mx = v[k0];
#pragma unroll
    for (int i = 1; i < SUB; ++i) mx = fmaxf(mx, v[k0 + i]);
    const float m_new = fmaxf(m, mx);
    const RowShift rs = row_shift(m_new == kNegInf ? 0.0f : m_new, clip);
    float t[SUB];
#pragma unroll
    for (int i = 0; i < SUB; ++i) {
      v[k0 + i] = exp_shift_clip<MODE>(v[k0 + i], rs);
      t[i] = v[k0 + i];
    }
    const float sk = tree_sum(t);
    if (k0 == 0) {
      s = sk;
    } else {
      const float f = m == kNegInf ? 1.0f : exp_shift_clip<exp_mode<MODE>()>(m, rs);
      s = s * f + sk;
    }
    m = m_new;
    mk[k0 / SUB] = m_new;
    // Finish this sub-strip here: its exponentials are not sunk below the
    // next sub-strip's max, which waits for that sub-strip's loads.
    asm volatile("" : "+v"(s), "+v"(m));
    __builtin_amdgcn_sched_barrier(0);
  }
  return make_float2(m, s);
}

// A segment's (m, s) through lane_online_exp, over the workgroup's NW
// wavefronts: m the segment max, s its sum of exp(max(x - m, lo)) (for
// m = -inf, the lanes' sums of clipped values).  v holds the lane's
// exponentials afterwards (see lane_online_exp).
// With PH the segment starts `a` floats past a 16-byte boundary
// (load_strip_ph); a = 0 and a whole segment take the aligned loads.
template <int NW, int V, bool VEC4, int MODE, bool PH = false>
__device__ __forceinline__ float2 segment_online(float (&v)[4 * V],
                                                 float (&mk)[4 * V / kOnlineSub],
                                                 const float* p, int lane_off, int stride,
                                                 int lim, Clip clip, float* red_max,
                                                 float* red_sum, int a = 0) {
  // Each branch reduces its own loads: after a join the compiler would wait
  // for all of them before the first use.
  float2 ms;
  if (lim == 4 * V * stride && a == 0) {
    load_strip_whole<V, VEC4>(v, p, lane_off, stride);
    ms = lane_online_exp<MODE>(v, mk, clip);
  } else if constexpr (PH) {
    load_strip_ph<V>(v, p, a, opaque(lane_off), stride, lim);
    ms = lane_online_exp<MODE>(v, mk, clip);
  } else {
    load_strip<V, VEC4>(v, p, opaque(lane_off), stride, lim);
    ms = lane_online_exp<MODE>(v, mk, clip);
  }
  const float m = block_max<NW>(ms.x, red_max);
  const float s = block_sum<NW>(
      lane_share<exp_mode<MODE>()>(ms, row_shift(m == kNegInf ? 0.0f : m, clip)), red_sum);
  return make_float2(m, s);
}

// Stores out(v[i]) for the columns of the strip that are inside the row.
template <int V, bool VEC4, typename F>
__device__ __forceinline__ void store_strip(const float (&v)[4 * V], F out, float* p,
                                            int lane_off, int stride, int lim) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int c = 4 * (lane_off + stride * j);
      f32x4 q;
      q.x = out(v[4 * j + 0]);
      q.y = out(v[4 * j + 1]);
      q.z = out(v[4 * j + 2]);
      q.w = out(v[4 * j + 3]);
      if (4 * stride * (j + 1) <= lim || c < lim) st_stream(p + c, q);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      const int c = lane_off + stride * i;
      if (stride * (i + 1) <= lim || c < lim) __builtin_nontemporal_store(out(v[i]), p + c);
    }
  }
}

// The output step of a row whose shift is rs and whose sum of clipped
// exponentials is s: v holds e (probabilities, y = e / S) or x (log
// outputs, y = c - ln S).
template <int V, bool VEC4, int MODE>
__device__ __forceinline__ void store_row(const float (&v)[4 * V], RowShift rs, float s,
                                          float* p, int lane_off, int stride, int lim) {
  if constexpr (MODE == kLogOut) {
    const float ls = log_of_sum(s);
    store_strip<V, VEC4>(v, [&](float xv) { return log_out(xv, rs, ls); }, p, lane_off, stride,
                         lim);
  } else {
    const float rcp = 1.0f / s;
    store_strip<V, VEC4>(v, [&](float ev) { return ev * rcp; }, p, lane_off, stride, lim);
  }
}

// Stores the probabilities of a segment left by segment_online: with the
// row's shift rs (max M) and rcp = 1/S,
//     y = max(e * exp(max(mk - M, lo)) * rcp, e_lo * rcp)
// per sub-strip.  For x - M >= lo the rescaled e is exp(x - M) / S; below
// it, under e^lo / S, so the max gives the clipped value exactly.
// With PH the segment starts `a` floats past a 16-byte boundary, as in
// segment_online.
template <int V, bool VEC4, int MODE, bool PH = false>
__device__ __forceinline__ void store_online(float (&v)[4 * V],
                                             const float (&mk)[4 * V / kOnlineSub], RowShift rs,
                                             float rcp, float* p, int lane_off, int stride,
                                             int lim, int a = 0) {
  constexpr int SUB = kOnlineSub;
  const float floor_y = rs.e_lo * rcp;
#pragma unroll
  for (int k = 0; k < 4 * V / SUB; ++k) {
    const float sc = exp_shift_clip<exp_mode<MODE>()>(mk[k], rs) * rcp;
#pragma unroll
    for (int i = 0; i < SUB; ++i) v[k * SUB + i] = fmaxf(v[k * SUB + i] * sc, floor_y);
  }
  if constexpr (PH)
    store_strip_ph<V>(v, [](float ev) { return ev; }, p, a, lane_off, stride, lim);
  else
    store_strip<V, VEC4>(v, [](float ev) { return ev; }, p, lane_off, stride, lim);
}

// The row's label as a column of the segment [c0, c0 + lim), or -1 when it
// lies outside the segment (or outside the row).
__device__ __forceinline__ int seg_label(int64_t label, int64_t c0, int lim) {
  const int64_t l = label - c0;
  return (l >= 0 && l < lim) ? static_cast<int>(l) : -1;
}

// Index into this lane's v (laid out as in load_strip) of segment column
// lc, or -1 when this lane does not hold it (or lc < 0).
template <int V, bool VEC4>
__device__ __forceinline__ int held_index(int lc, int lane_off, int stride) {
  if (lc < 0) return -1;
  const int t = (VEC4 ? lc >> 2 : lc) - lane_off;
  if (t < 0 || t % stride != 0) return -1;
  const int i = t / stride;
  if constexpr (VEC4) {
    return i < V ? 4 * i + (lc & 3) : -1;
  } else {
    return i < 4 * V ? i : -1;
  }
}

// What a lane contributes to an NLL output: the label's logit, if this lane
// holds its column (`found`), and whether it must write NaN for a label
// outside the row (`bad`: one thread of the row's first segment).
struct LabelPick {
  float x;
  bool found;
  bool bad;
};

// Picks the label's logit out of this lane's v (laid out as in load_strip)
// for the segment [c0, c0 + lim).  Taken right after the loads, so that v
// need not stay live through the row reductions.  Other modes pick nothing.
template <int V, bool VEC4, int MODE>
__device__ __forceinline__ LabelPick pick_label(const float (&v)[4 * V], int64_t label,
                                                int64_t cols, int64_t c0, int lim, int lane_off,
                                                int stride, bool first) {
  LabelPick p{0.0f, false, false};
  if constexpr (MODE == kNllOut) {
    const int idx = held_index<V, VEC4>(seg_label(label, c0, lim), lane_off, stride);
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) p.x = idx == i ? v[i] : p.x;
    p.found = idx >= 0;
    p.bad = first && (label < 0 || label >= cols);
  }
  return p;
}

// The output step of the segment [c0, c0 + lim) of `row`: the row's
// outputs (probabilities or logs) into y + row * cols + c0, or for NLL
// outputs the one loss y[row] = ln S - c_label, written by the lane that
// picked the label's logit (NaN for a label outside [0, cols)).
template <int V, bool VEC4, int MODE>
__device__ __forceinline__ void finish_row(const float (&v)[4 * V], RowShift rs, float s,
                                           float* y, int64_t row, int64_t cols, int64_t c0,
                                           int lim, LabelPick pick, int lane_off, int stride) {
  if constexpr (MODE == kNllOut) {
    if (pick.found) y[row] = -log_out(pick.x, rs, log_of_sum(s));
    if (pick.bad) y[row] = __builtin_nanf("");
  } else {
    store_row<V, VEC4, MODE>(v, rs, s, y + row * cols + c0, lane_off, stride, lim);
  }
}

// The label of `row` for NLL outputs (0 in the other modes, where labels
// is null).
template <int MODE>
__device__ __forceinline__ int64_t row_label(const int64_t* labels, int64_t row) {
  if constexpr (MODE == kNllOut) {
    return labels[row];
  } else {
    return 0;
  }
}

// Columns of a row segment that starts at column c0: min(cols - c0, cap).
__device__ __forceinline__ int seg_len(int64_t cols, int64_t c0, int64_t cap) {
  const int64_t left = cols - c0;
  return static_cast<int>(left < cap ? left : cap);
}

// ---------------------------------------------------------------------------
// (a) Packed rows, cols <= G*EPL, with G lanes per row (G = 1, 2 or 4) and
// EPL <= 16 columns per lane, both compile-time.
//
// A 256-thread workgroup works on tiles of kRows = 256/G consecutive rows:
// one row per group of G lanes, so a tile is done in one pass.  kRows is a
// multiple of 4, so a tile starts on a 16-byte boundary whenever x and y do,
// whatever cols is (cols = 50 gives 200-byte rows).  Tiles move
// HBM -> registers -> LDS -> HBM with 128-bit accesses; lane j of a row group
// takes columns j, j+G, ..., j+(EPL-1)G.
//
// The grid is persistent (a few workgroups per CU, each looping over tiles)
// and every workgroup issues the loads of its next tile right after staging
// the current one, so they are in flight while the current tile computes.
template <int G, int EPL, int MODE>
__device__ __forceinline__ void packed_rows(float* tile, int nr, int ccols, int r, int j,
                                            Clip clip, int64_t label, float* yl) {
  const bool active = r < nr;
  float* tr = tile + r * ccols;
  float v[EPL];
#pragma unroll
  for (int k = 0; k < EPL; ++k) {
    const int c = j + G * k;
    v[k] = (active && c < ccols) ? tr[c] : kNegInf;
  }
  const RowShift rs = row_shift(seg_max<G>(array_max(v)), clip);
  const float s = seg_sum<G>(exp_strip<MODE>(v, rs));
  if constexpr (MODE == kNllOut) {
    // One loss per row into yl[r], by lane 0 of the row: the label's logit
    // is still in the tile; a label outside the row gives NaN.
    if (active && j == 0) {
      const bool ok = label >= 0 && label < ccols;
      yl[r] = ok ? -log_out(tr[ok ? label : 0], rs, log_of_sum(s)) : __builtin_nanf("");
    }
  } else if constexpr (MODE == kLogOut) {
    const float ls = log_of_sum(s);
#pragma unroll
    for (int k = 0; k < EPL; ++k) {
      const int c = j + G * k;
      if (active && c < ccols) tr[c] = log_out(v[k], rs, ls);
    }
  } else {
    const float rcp = 1.0f / s;
#pragma unroll
    for (int k = 0; k < EPL; ++k) {
      const int c = j + G * k;
      if (active && c < ccols) tr[c] = v[k] * rcp;
    }
  }
}

template <int G, int EPL, bool VEC4, int MODE>
__global__ __launch_bounds__(256) void k_packed(const float* x, float* y,
                                                const int64_t* labels, int64_t rows,
                                                int64_t cols, Clip clip) {
  constexpr int kRows = 256 / G;
  constexpr int kTileFloats = kRows * G * EPL;  // = 256 * EPL
  constexpr int kPer = VEC4 ? (kTileFloats / 4 + 255) / 256 : (kTileFloats + 255) / 256;
  __shared__ float tile[kTileFloats];

  const int tid = threadIdx.x;
  const int ccols = static_cast<int>(cols);
  const int64_t ntiles = (rows + kRows - 1) / kRows;
  const int r = tid / G;
  const int j = tid % G;

  // Registers for the next tile: kPer 128-bit (or 32-bit) values per thread,
  // and (NLL outputs) the label of this thread's row of it.
  f32x4 q4[VEC4 ? kPer : 1];
  float q1[VEC4 ? 1 : kPer];
  int64_t lab_next = -1;
  auto issue = [&](int64_t t) {
    const int64_t row0 = t * kRows;
    const int nr = static_cast<int>(rows - row0 < kRows ? rows - row0 : kRows);
    const int n = nr * ccols;
    const float* xs = x + row0 * cols;
    if constexpr (MODE == kNllOut) {
      if (r < nr) lab_next = labels[row0 + r];
    }
    if constexpr (VEC4) {
      const int n4 = n >> 2;
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        q4[u] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (i < n4) q4[u] = ld_stream(xs + 4 * i);
      }
    } else {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        q1[u] = 0.0f;
        if (i < n) q1[u] = __builtin_nontemporal_load(xs + i);
      }
    }
  };

  int64_t t = blockIdx.x;
  if (t < ntiles) issue(t);
  for (; t < ntiles; t += gridDim.x) {
    const int64_t row0 = t * kRows;
    const int nr = static_cast<int>(rows - row0 < kRows ? rows - row0 : kRows);
    const int n = nr * ccols;
    const float* xs = x + row0 * cols;

    if constexpr (VEC4) {
      const int n4 = n >> 2;
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        if (i < n4) *reinterpret_cast<f32x4*>(tile + 4 * i) = q4[u];
      }
      for (int i = (n4 << 2) + tid; i < n; i += 256) tile[i] = xs[i];
    } else {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        if (i < n) tile[i] = q1[u];
      }
    }
    __syncthreads();
    const int64_t label = lab_next;
    if (t + gridDim.x < ntiles) issue(t + gridDim.x);

    packed_rows<G, EPL, MODE>(tile, nr, ccols, r, j, clip, label, y + row0);
    __syncthreads();

    if constexpr (MODE != kNllOut) {
      float* ys = y + row0 * cols;
      if constexpr (VEC4) {
        const int n4 = n >> 2;
        for (int i = tid; i < n4; i += 256)
          st_stream(ys + 4 * i, *reinterpret_cast<const f32x4*>(tile + 4 * i));
        for (int i = (n4 << 2) + tid; i < n; i += 256) ys[i] = tile[i];
      } else {
        for (int i = tid; i < n; i += 256) __builtin_nontemporal_store(tile[i], ys + i);
      }
    }
    __syncthreads();
  }
}

// (a, aligned) Rows of at most 256 columns made of whole 16-byte strips
// (cols a multiple of 4, x and y 16-byte aligned), probability outputs.
// G lanes per row (G the power of two >= cols / 4), each lane one 128-bit
// strip of 4 columns, so a wavefront's load instruction covers 64 / G
// consecutive rows exactly as the coalesced load leaves them: no LDS and no
// relayout.  The row max and sum are segmented reductions over the row's G
// lanes (DPP within 16 lanes, permlane swaps beyond).  Each wavefront keeps
// U such row groups in flight (U * 1 KiB of loads).  Lanes past the row's
// strips read -inf (a clipped term, as in load_strip).
//
// U is 1 or 2, chosen per call by the host.  U = 2, one workgroup per
// block of rows: per 64 MiB of logits on 4 to 256 columns this ran
// 23.4-23.9 us, against 23.7-25.4 us with U = 4 and 25.4-26.8 us with U = 8
// (81 VGPRs, five wavefronts per SIMD).  U = 1 pays when the launch is small
// enough that U = 2 would leave resident workgroup slots empty: at 2 to
// 8 MiB on 16 to 256 columns it ran 3-12% faster than U = 2, and at 64 MiB
// up to 9% slower.  A workgroup may loop over several row blocks (grid
// stride), loading the next block before it reduces the current one; the
// host caps the grid at the resident workgroups only when one workgroup per
// block would take more than one and at most two rounds of them (22 MiB on
// 4 to 256 columns: 8.9-9.4 us against 10.0-10.3 us with a second, mostly
// empty round; at 64 and 128 MiB the capped grid was 3-15% slower than one
// workgroup per block).  The LDS-staged packed kernel took 24.2-24.5 us on
// 4 and 64 columns and 35.3 us on 16 (its lanes read LDS rows at a stride
// of 16 words: bank conflicts), and one wavefront per row 42.5 us on 100
// columns (25 of 64 lanes busy).  Rows that leave many of their G lanes
// idle go to the packed kernel instead (host dispatch).
constexpr int kGroupRowsMaxCols = 256;

template <int G, int U, int MODE>
__global__ __launch_bounds__(256) void k_group_rows(const float* x, float* y, int64_t rows,
                                                    int64_t cols, Clip clip) {
  static_assert(G >= 1 && G <= 64 && (G & (G - 1)) == 0, "G: power of 2 up to 64");
  constexpr int R = 64 / G;                       // rows per group
  constexpr int64_t kWaveRows = int64_t(U) * R;   // rows per wavefront step
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  const int rho = lane / G;
  const int j = lane % G;
  const bool col_ok = 4 * j < cols;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 4 * kWaveRows;
  auto load = [&](f32x4 (&q)[U], int64_t r0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = r0 + u * R + rho;
      q[u] = f32x4{kNegInf, kNegInf, kNegInf, kNegInf};
      if (col_ok && row < rows) q[u] = ld_stream(x + row * cols + 4 * j);
    }
  };
  int64_t r0 = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * kWaveRows;
  f32x4 q[U];
  load(q, r0);
  for (; r0 < rows; r0 += stride) {
    // The next step's loads are issued before this step's rows are reduced.
    f32x4 qn[U];
    load(qn, r0 + stride);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = r0 + u * R + rho;
      const float m = seg_max<G>(fmaxf(fmaxf(q[u].x, q[u].y), fmaxf(q[u].z, q[u].w)));
      const RowShift rs = row_shift(m, clip);
      float e[4] = {exp_shift_clip<MODE>(q[u].x, rs), exp_shift_clip<MODE>(q[u].y, rs),
                    exp_shift_clip<MODE>(q[u].z, rs), exp_shift_clip<MODE>(q[u].w, rs)};
      const float rcp = 1.0f / seg_sum<G>(tree_sum(e));
      const f32x4 out = {e[0] * rcp, e[1] * rcp, e[2] * rcp, e[3] * rcp};
      if (col_ok && row < rows) st_stream(y + row * cols + 4 * j, out);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) q[u] = qn[u];
  }
}

// Occupancy targets (waves per SIMD) for the register-resident kernels: 4
// (128 VGPRs) up to 32 values per lane with 128-bit access and probability
// outputs; 2 (256 VGPRs) otherwise, where 32-bit access needs more address
// registers and log outputs keep the logits next to the exponentials, so
// nothing spills to scratch.  The one-pass split kernel runs at twice
// these (its chunks hold half as many values per lane).
template <int V, bool VEC4, int MODE>
constexpr int kRowWaves = (V <= 8 && VEC4 && !keeps_logits<MODE>()) ? 4 : 2;

// ---------------------------------------------------------------------------
// (b) One wavefront per row, cols <= 256*V (4*V elements per lane).
// Four wavefronts per workgroup work on four rows independently.
//
// `delay` (wall-clock ticks, 0 for none) is passed only for launches where
// every workgroup takes a single row set: each wavefront's stores wait until
// that long after the workgroup started, so that the launch's reads are
// over before its writes begin (HBM then serves them in two phases rather
// than interleaved).
//
// PH (probability outputs, 128-bit access): rows of a length that is not a
// multiple of 4 in 16-byte aligned x and y, each row accessed in the aligned
// strips around it (load_strip_ph); the row's phase is (row * cols) mod 4.
template <int V, bool VEC4, int MODE, bool PH = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(
    kRowWaves<V, VEC4, MODE>))) void k_wave_row(
    const float* x, float* y, const int64_t* labels, int64_t rows, int64_t cols, Clip clip,
    uint32_t delay) {
  static_assert(!PH || (VEC4 && !keeps_logits<MODE>()), "phase access: probability outputs");
  const uint64_t t0 = wall_clock();
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  for (int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wave; row < rows;
       row += static_cast<int64_t>(gridDim.x) * 4) {
    const float* xr = x + row * cols;
    const int64_t label = row_label<MODE>(labels, row);
    const int lim = static_cast<int>(cols);
    float v[4 * V];
    if constexpr (PH) {
      const int a = static_cast<int>((row * cols) & 3);
      load_strip_ph<V>(v, xr, a, opaque(lane), 64, lim);
      const RowShift rs = row_shift(seg_max<64>(array_max(v)), clip);
      const float s = seg_sum<64>(exp_strip<MODE>(v, rs));
      if (delay != 0) wait_until_after(t0 + delay, s);
      const float rcp = 1.0f / s;
      store_strip_ph<V>(v, [&](float ev) { return ev * rcp; }, y + row * cols, a, opaque(lane),
                        64, lim);
      continue;
    }
    load_strip<V, VEC4>(v, xr, opaque(lane), 64, lim);
    const LabelPick pick = pick_label<V, VEC4, MODE>(v, label, cols, 0, lim, lane, 64, lane == 0);
    const RowShift rs = row_shift(seg_max<64>(array_max(v)), clip);
    const float s = seg_sum<64>(exp_strip<MODE>(v, rs));
    if (delay != 0) wait_until_after(t0 + delay, s);
    finish_row<V, VEC4, MODE>(v, rs, s, y, row, cols, 0, lim, pick, opaque(lane), 64);
  }
}

// ---------------------------------------------------------------------------
// (c) One workgroup of NT threads per row, cols <= 4*V*NT.  `delay` and PH
// as for k_wave_row.
template <int NT, int V, bool VEC4, int MODE, bool PH = false>
__global__ __launch_bounds__(NT) void k_block_row(const float* x, float* y,
                                                  const int64_t* labels, int64_t rows,
                                                  int64_t cols, Clip clip, uint32_t delay) {
  static_assert(!PH || (VEC4 && !keeps_logits<MODE>()), "phase access: probability outputs");
  const uint64_t t0 = wall_clock();
  constexpr int NW = NT / 64;
  __shared__ float red_max[NW];
  __shared__ float red_sum[NW];
  const int tid = threadIdx.x;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const float* xr = x + row * cols;
    const int64_t label = row_label<MODE>(labels, row);
    const int lim = static_cast<int>(cols);
    float v[4 * V];
    if constexpr (PH) {
      const int a = static_cast<int>((row * cols) & 3);
      load_strip_ph<V>(v, xr, a, opaque(tid), NT, lim);
      const RowShift rs = row_shift(block_max<NW>(array_max(v), red_max), clip);
      const float s = block_sum<NW>(exp_strip<MODE>(v, rs), red_sum);
      if (delay != 0) wait_until_after(t0 + delay, s);
      const float rcp = 1.0f / s;
      store_strip_ph<V>(v, [&](float ev) { return ev * rcp; }, y + row * cols, a, opaque(tid),
                        NT, lim);
    } else if constexpr (MODE == kNllOut && VEC4) {
      // The loss needs only the row's (max, sum) and one logit.  The sums
      // are folded in as the loads land, and thread 0 reads the label's
      // logit itself (one more cache line per row), so no value has to stay
      // live after its exponential: two workgroups per CU still fit.  (With
      // 32-bit loads the fold needs more registers than that; those rows
      // take the reduction below.)
      // The row's loads go out first; the logit's load waits only for the
      // label, and is issued by every thread (one cache line per wavefront)
      // so that no branch makes the compiler wait for all of them.
      load_strip_flat<V, VEC4>(v, xr, tid, NT, lim);
      const bool bad = label < 0 || label >= cols;
      const float xl = xr[bad ? 0 : label];
      const float2 ms = lane_online(v, clip);
      const float m = block_max<NW>(ms.x, red_max);
      const float s =
          block_sum<NW>(lane_share(ms, row_shift(m == kNegInf ? 0.0f : m, clip)), red_sum);
      if (tid == 0)
        y[row] = bad ? __builtin_nanf("") : -log_out(xl, row_shift(m, clip), log_of_sum(s));
    } else {
      // (The online reduction of the split kernel measured slower here:
      // 23.2 us against 22.5 us on 512 rows of 32768.)
      load_strip<V, VEC4>(v, xr, opaque(tid), NT, lim);
      const LabelPick pick =
          pick_label<V, VEC4, MODE>(v, label, cols, 0, lim, tid, NT, tid == 0);
      const RowShift rs = row_shift(block_max<NW>(array_max(v), red_max), clip);
      // Log outputs of 32 values per lane keep the accurate exponential: with
      // the cheap one the compiler keeps more terms in flight, which needs
      // more than the 64 VGPRs of two workgroups per CU.
      constexpr int SE = (MODE == kLogOut && V >= 8) ? kExpAccurate : kSumExp;
      const float s = block_sum<NW>(exp_strip<MODE, 4 * V, SE>(v, rs), red_sum);
      if (delay != 0) wait_until_after(t0 + delay, s);
      finish_row<V, VEC4, MODE>(v, rs, s, y, row, cols, 0, lim, pick, opaque(tid), NT);
    }
  }
}

// ---------------------------------------------------------------------------
// (c, split) Rows longer than one workgroup's registers: a row is cut into
// chunks of CH = 4*V*NT columns, one workgroup per chunk (or per group of
// chunks in the two-pass kernels).  The row's workgroups combine their
// partial (max, sum) pairs through the row's entry of the exchange table
// (sm_exchange.hpp).
//
// A partial (m_g, s_g) is a chunk's max and its sum of exp(max(x - m_g, lo)).
// A chunk whose max is -inf stores s_g = its element count, so that merging
// gives count * e_lo, the clipped value of its -inf elements.  Merging a
// row's partials (every lane of a wavefront computes the same bits):
//     M = max_g m_g,   S = sum_g s_g * exp(max(m_g - M, lo)).
// Using the clip relative to m_g inside a partial changes S by at most
// cols * e^lo relative (below 1e-10 for any row that fits in memory, since
// lo <= -48), far under fp32 resolution.

// The row's entry for wavefront 0 of a workgroup (lane 0 joins it; the
// pointer is made uniform across the wavefront).  A miss is counted.
__device__ __forceinline__ uint64_t* wave_entry(const XchArgs& xa, int lrow, uint64_t deadline) {
  uint64_t e = 0;
  if (__lane_id() == 0) {
    uint64_t* p = row_entry(xa, lrow, deadline);
    if (p == nullptr) count_give_up(xa, xch::kDiagJoinGiveUps);
    e = reinterpret_cast<uint64_t>(p);
  }
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(e));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(e >> 32));
  return reinterpret_cast<uint64_t*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Merge of up to 64 partials held one per lane (lanes without one pass
// m = -inf, s = 0): the row's (M, S), the same bits on every lane.
template <int SE>
__device__ __forceinline__ float2 merge_lanes(float pm, float ps, Clip clip) {
  const float mrow = seg_max<64>(pm);
  const RowShift rs = row_shift(mrow, clip);
  const float term = ps == 0.0f ? 0.0f : ps * exp_shift_clip<SE>(pm, rs);
  return make_float2(mrow, seg_sum<64>(term));
}

// Polls the row's first `g` slots (one per lane) until none is empty, up to
// `deadline`.  Returns the slot (~0 for lanes past g); *ok is false after a
// time-out.
__device__ __forceinline__ uint64_t poll_slots(const uint64_t* slots, int g, uint64_t deadline,
                                               bool* ok) {
  const int lane = __lane_id();
  uint64_t q = ~0ull;
  while (true) {
    q = lane < g ? xch::ld_agent(&slots[lane]) : ~0ull;
    if (__builtin_amdgcn_ballot_w64(q == 0) == 0) return q;
    if (static_cast<int64_t>(wall_clock() - deadline) > 0) {
      *ok = false;
      return q;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// (m, s) of one chunk held in v (its max and sum of clipped exponentials
// against that max; s = count when the max is -inf).  For probability
// modes v is replaced by the exponentials.
template <int NW, int V, int MODE>
__device__ __forceinline__ float2 chunk_partial(float (&v)[4 * V], int lim, Clip clip,
                                                float* red_max, float* red_sum) {
  float m;
  float s;
  if constexpr (keeps_logits<MODE>()) {
    const float2 ms = lane_online(v, clip);
    m = block_max<NW>(ms.x, red_max);
    s = block_sum<NW>(lane_share(ms, row_shift(m == kNegInf ? 0.0f : m, clip)), red_sum);
  } else {
    m = block_max<NW>(array_max(v), red_max);
    s = block_sum<NW>(exp_strip<MODE>(v, row_shift(m == kNegInf ? 0.0f : m, clip)), red_sum);
  }
  if (m == kNegInf) s = static_cast<float>(lim);
  return make_float2(m, s);
}

// (c, split, two passes) for rows longer than a one-pass launch can hold.
// The launch has WPR <= 64 workgroups per row; workgroup w of a row takes
// the row's chunks w, w + WPR, ...  Pass 1 (k_split_stats) joins the row's
// entry and leaves each workgroup's merged partial in its slot; pass 2
// (k_split_apply) finds the entry, merges the row's WPR slots, writes the
// chunks' outputs, and the last workgroup of the row releases the entry.
// x is read twice.
template <int NT, int V, bool VEC4, int MODE>
__global__ __launch_bounds__(NT) void k_split_stats(const float* x, XchArgs xa, int64_t cols,
                                                    int wpr, int64_t chunks, Clip clip) {
  const uint64_t t0 = wall_clock();
  constexpr int NW = NT / 64;
  constexpr int64_t CH = int64_t(4) * V * NT;
  __shared__ float red_max[NW];
  __shared__ float red_sum[NW];
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int lrow = b / wpr;
  const int w = b - lrow * wpr;
  float m = kNegInf;
  float s = 0.0f;
  for (int64_t g = w; g < chunks; g += wpr) {
    const int64_t c0 = g * CH;
    const int lim = seg_len(cols, c0, CH);
    float v[4 * V];
    load_strip<V, VEC4>(v, x + lrow * cols + c0, tid, NT, lim);
    const float2 p = chunk_partial<NW, V, MODE>(v, lim, clip, red_max, red_sum);
    const float mm = fmaxf(m, p.x);
    if (mm == kNegInf) {
      s = s + p.y;
    } else {
      const RowShift rs = row_shift(mm, clip);
      const float a = s == 0.0f ? 0.0f : s * exp_shift_clip<exp_mode<MODE>()>(m, rs);
      s = a + p.y * exp_shift_clip<exp_mode<MODE>()>(p.x, rs);
    }
    m = mm;
    __syncthreads();  // red_max / red_sum are reused by the next chunk
  }
  if (tid < 64) {
    uint64_t* entry = wave_entry(xa, lrow, t0 + xa.limit_ticks);
    if (tid == 0 && entry != nullptr) xch::st_agent(&entry_slots(entry)[w], encode_pair(m, s));
  }
}

template <int NT, int V, bool VEC4, int MODE>
__global__ __launch_bounds__(NT) void k_split_apply(const float* x, float* y,
                                                    const int64_t* labels, XchArgs xa,
                                                    int64_t cols, int wpr, int64_t chunks,
                                                    Clip clip) {
  const uint64_t t0 = wall_clock();
  constexpr int64_t CH = int64_t(4) * V * NT;
  __shared__ float bcast[2];
  const int tid = threadIdx.x;
  const int lane = __lane_id();
  const int b = blockIdx.x;
  const int lrow = b / wpr;
  const int w = b - lrow * wpr;
  const int64_t label = row_label<MODE>(labels, lrow);
  uint64_t* entry = nullptr;  // wavefront 0 only
  if (tid < 64) {
    entry = wave_entry(xa, lrow, t0 + xa.limit_ticks);
    float2 ms = make_float2(__builtin_nanf(""), __builtin_nanf(""));
    if (entry != nullptr) {
      const uint64_t q = lane < wpr ? xch::ld_agent(&entry_slots(entry)[lane]) : ~0ull;
      const float pm = lane < wpr ? decode_m(q) : kNegInf;
      const float ps = lane < wpr ? decode_s(q) : 0.0f;
      ms = merge_lanes<exp_mode<MODE>()>(pm, ps, clip);
    }
    if (tid == 0) {
      bcast[0] = ms.x;
      bcast[1] = ms.y;
    }
  }
  __syncthreads();
  const RowShift rs = row_shift(bcast[0], clip);
  const float srow = bcast[1];
  for (int64_t g = w; g < chunks; g += wpr) {
    const int64_t c0 = g * CH;
    const int lim = seg_len(cols, c0, CH);
    float v[4 * V];
    load_strip<V, VEC4>(v, x + lrow * cols + c0, tid, NT, lim);
    if constexpr (!keeps_logits<MODE>()) {
#pragma unroll
      for (int i = 0; i < 4 * V; ++i) v[i] = exp_shift_clip<MODE>(v[i], rs);
    }
    const LabelPick pick =
        pick_label<V, VEC4, MODE>(v, label, cols, c0, lim, tid, NT, g == 0 && tid == 0);
    finish_row<V, VEC4, MODE>(v, rs, srow, y, lrow, cols, c0, lim, pick, tid, NT);
  }
  if (entry != nullptr && tid < 64) {
    // The slot reads have returned (the outputs above depend on them).
    uint32_t last = 0;
    if (tid == 0) last = depart_entry(entry, wpr, 1u) ? 1u : 0u;
    last = __builtin_amdgcn_readfirstlane(last);
    if (last) {
      if (lane < wpr) xch::st_agent(&entry_slots(entry)[lane], 0ull);
      if (tid == 0) release_entry(entry);
    }
  }
}

// ---------------------------------------------------------------------------
// (c, split, one pass) The G <= 64 workgroups of a row exchange partials in
// the middle of the kernel, so x is read from HBM exactly once.
//
// Workgroup (row, g) keeps e = exp(max(x - m_g, lo)) of its chunk in
// registers, joins the row's entry and publishes (m_g, s_g) in slot g.
// Wavefront 0 polls the row's G slots until none is empty, merges them into
// M and S, and every thread writes
//     y = max(e * exp(m_g - M), e_lo) / S
// (log outputs keep x instead of e and write y = max(x - M, lo) - ln S).
// For an element with x - M >= lo the rescaled e equals exp(x - M) >= e^lo;
// for x - M < lo it is below e^lo, so the max is exactly the clip of the
// definition.  A NaN element makes s_g, hence S and the whole row, NaN.
//
// After its slot reads have returned, each workgroup counts itself out of
// the entry; the last one clears the slots and frees the entry.  All
// exchange accesses are device-scope atomics, performed at the device's
// coherence point rather than in a per-XCD L2, so no cache writeback or
// invalidate is needed.  A wavefront issues memory operations in program
// order and not speculatively, so the output work, which depends on the
// loaded slots, never runs ahead of them.
//
// Progress: a row's workgroups have consecutive IDs and workgroups are
// dispatched in ID order, so the lowest unfinished row always has all of its
// chunks dispatched once G workgroup slots are free; every wait ends as long
// as G workgroups of the launch fit on the device at once.  Every wait is
// also bounded by the wall clock: a workgroup that gives up writes NaN for
// its chunk (and counts the give-up) instead of stalling the device.
//
// `delay` (wall-clock ticks after the workgroup started, 0 for none) holds
// the stores back until the launch's loads are expected to be done, so that
// HBM serves the reads and the writes of the launch in two phases instead of
// interleaving them.
//
// NLL outputs (one value per row) take no wait at all: the last workgroup
// of the row to depart does the merge.
//
// PH (probability outputs): rows whose length is not a multiple of 4, in
// 16-byte aligned x and y.  Chunk g then covers the row's columns
// [g*CH - a, (g+1)*CH - a) (clamped to the row), a = the row's phase, so
// every chunk but the first starts on a 16-byte boundary and only the row's
// two end strips straddle (load_strip_ph).  The launch has
// ceil((cols + 3) / CH) chunks per row; a row whose phase leaves its last
// chunk empty publishes an empty pair from it (count 0).
template <int NT, int V, bool VEC4, int MODE, bool PH = false>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(
    2 * kRowWaves<V, VEC4, MODE>))) void k_split_onepass(
    const float* x, float* y, const int64_t* labels, XchArgs xa, int64_t cols, int chunks,
    uint32_t delay, Clip clip) {
  static_assert(!PH || (VEC4 && !keeps_logits<MODE>()), "phase access: probability outputs");
  const uint64_t t0 = wall_clock();
  constexpr int NW = NT / 64;
  constexpr int64_t CH = int64_t(4) * V * NT;
  __shared__ float red_max[NW];
  __shared__ float red_sum[NW];
  __shared__ float bcast[2];
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int lrow = b / chunks;
  const int g = b - lrow * chunks;
  int64_t c0 = int64_t(g) * CH;
  int lim = seg_len(cols, c0, CH);
  int a = 0;  // phase of this chunk's first column (PH: the first chunk only)
  if constexpr (PH) {
    const int ra =
        static_cast<int>((reinterpret_cast<uintptr_t>(x + lrow * cols) >> 2) & 3);
    const int64_t s0 = int64_t(g) * CH - ra;
    const int64_t e0 = s0 + CH < cols ? s0 + CH : cols;
    c0 = s0 < 0 ? 0 : s0;
    lim = e0 > c0 ? static_cast<int>(e0 - c0) : 0;
    a = g == 0 ? ra : 0;
  }
  const float* xr = x + lrow * cols + c0;
  const int64_t label = row_label<MODE>(labels, lrow);

  constexpr bool ONLINE = !keeps_logits<MODE>() && online_exp<4 * V>();
  static_assert(!PH || ONLINE, "phase access: the online reduction");
  float v[4 * V];
  float mk[ONLINE ? 4 * V / kOnlineSub : 1];
  float2 part;
  if constexpr (ONLINE) {
    part = segment_online<NW, V, VEC4, MODE, PH>(v, mk, xr, tid, NT, lim, clip, red_max,
                                                 red_sum, a);
    if (part.x == kNegInf) part.y = static_cast<float>(lim);
  } else if constexpr (keeps_logits<MODE>()) {
    load_strip_flat<V, VEC4>(v, xr, tid, NT, lim);
  } else {
    load_strip<V, VEC4>(v, xr, tid, NT, lim);
  }
  // NLL outputs: every workgroup reads the row's label logit right after its
  // chunk's loads (one cache line per wavefront, after the label itself),
  // so the one that merges the row below already holds it, and the values
  // die as they are folded in.
  const bool bad_label = label < 0 || label >= cols;
  float xl = 0.0f;
  if constexpr (MODE == kNllOut) xl = x[lrow * cols + (bad_label ? 0 : label)];
  LabelPick pick{0.0f, false, false};
  if constexpr (MODE == kLogOut)
    pick = pick_label<V, VEC4, MODE>(v, label, cols, c0, lim, tid, NT, g == 0 && tid == 0);
  if constexpr (!ONLINE) part = chunk_partial<NW, V, MODE>(v, lim, clip, red_max, red_sum);
  const float m = part.x;
  const float s = part.y;
  const uint64_t deadline = t0 + xa.limit_ticks;

  if constexpr (MODE == kNllOut) {
    // One value per row: no workgroup waits.  Each publishes its pair and
    // then counts itself out; the slot store has completed before the count
    // (explicit wait), so the workgroup that brings the count to G sees all
    // G pairs.  That one merges them as above, writes the loss with the
    // label logit it read at the start, and frees the entry.
    if (tid < 64) {
      uint64_t* const entry = wave_entry(xa, lrow, deadline);
      if (entry == nullptr) {
        if (tid == 0) y[lrow] = __builtin_nanf("");
        return;
      }
      uint64_t* const slots = entry_slots(entry);
      uint32_t last = 0;
      if (tid == 0) {
        xch::st_agent(&slots[g], encode_pair(m, s));
        __builtin_amdgcn_s_waitcnt(0);
        last = depart_entry(entry, chunks, 1u) ? 1u : 0u;
      }
      last = __builtin_amdgcn_readfirstlane(last);
      if (last) {
        // Every pair was stored before its count, so none should read
        // empty; a slot that still does is read again (bounded), so the
        // merge does not rest on when a completed store becomes visible.
        bool ok = true;
        const uint64_t q = poll_slots(slots, chunks, deadline, &ok);
        const float2 ms = tid < chunks ? make_float2(decode_m(q), decode_s(q))
                                       : make_float2(kNegInf, 0.0f);
        const float2 rowms = merge_lanes<kExpAccurate>(ms.x, ms.y, clip);
        const float loss = (bad_label || !ok)
                               ? __builtin_nanf("")
                               : -log_out(xl, row_shift(rowms.x, clip), log_of_sum(rowms.y));
        if (tid == 0) {
          y[lrow] = loss;
          if (!ok) count_give_up(xa, xch::kDiagWaitGiveUps);
        }
        // The slot reads have returned (the loss depends on them).
        asm volatile("" : : "v"(loss));
        if (tid < chunks) xch::st_agent(&slots[tid], 0ull);
        if (tid == 0) release_entry(entry);
      }
    }
    return;
  }

  if (tid < 64) {
    uint64_t* const entry = wave_entry(xa, lrow, deadline);
    bool ok = entry != nullptr;
    uint64_t q = 0;
    uint32_t last = 0;
    if (ok) {
      uint64_t* const slots = entry_slots(entry);
      if (tid == 0) xch::st_agent(&slots[g], encode_pair(m, s));
      q = poll_slots(slots, chunks, deadline, &ok);
    }
    const float2 ms = (ok && tid < chunks) ? make_float2(decode_m(q), decode_s(q))
                                           : make_float2(kNegInf, 0.0f);
    const float2 rowms = merge_lanes<exp_mode<MODE>()>(ms.x, ms.y, clip);
    if (tid == 0) {
      if (!ok && entry != nullptr) count_give_up(xa, xch::kDiagWaitGiveUps);
      const float rcp = 1.0f / rowms.y;
      if constexpr (keeps_logits<MODE>()) {
        bcast[0] = ok ? rowms.x : __builtin_nanf("");  // M
        bcast[1] = ok ? rowms.y : __builtin_nanf("");  // S
      } else if constexpr (ONLINE) {
        bcast[0] = ok ? rowms.x : __builtin_nanf("");  // M
        bcast[1] = ok ? rcp : __builtin_nanf("");      // 1 / S
      } else {
        const RowShift rs = row_shift(rowms.x, clip);
        bcast[0] = ok ? exp_shift_clip<MODE>(m, rs) * rcp : __builtin_nanf("");  // e^(m_g-M)/S
        bcast[1] = ok ? clip.e_lo * rcp : __builtin_nanf("");                    // e_lo / S
      }
      // Count out once this wavefront's slot reads have returned (the
      // add's operand depends on them).  A workgroup that joined no entry
      // has nothing to count out of.
      uint32_t one = 1u;
      asm volatile("" : "+v"(one) : "v"(q));
      if (entry != nullptr) last = depart_entry(entry, chunks, one) ? 1u : 0u;
    }
    last = __builtin_amdgcn_readfirstlane(last);
    if (last) {
      if (tid < chunks) xch::st_agent(&entry_slots(entry)[tid], 0ull);
      if (tid == 0) release_entry(entry);
    }
  }
  __syncthreads();
  if (delay != 0) wait_until(t0 + delay);
  if constexpr (keeps_logits<MODE>()) {
    // v still holds the logits: y = c - ln S against the row's M.
    finish_row<V, VEC4, MODE>(v, row_shift(bcast[0], clip), bcast[1], y, lrow, cols, c0, lim,
                              pick, tid, NT);
  } else if constexpr (ONLINE) {
    store_online<V, VEC4, MODE, PH>(v, mk, row_shift(bcast[0], clip), bcast[1],
                                    y + lrow * cols + c0, opaque(tid), NT, lim, a);
  } else {
    float* yr = y + lrow * cols + c0;
    const float scale = bcast[0];
    const float floor_y = bcast[1];
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) v[i] = fmaxf(v[i] * scale, floor_y);
    store_strip<V, VEC4>(v, [](float ev) { return ev; }, yr, opaque(tid), NT, lim);
  }
}

// ---------------------------------------------------------------------------
// Diagnostics.

// e[i] = exp(max(x[i] - m[i], lo)), through the same device routine the
// softmax kernels use; MODE kExpRaw instead gives e[i] = v_exp_f32(x[i])
// (2^x), the hardware instruction those routines build on.
constexpr int kExpRaw = 16;
template <int MODE>
__global__ __launch_bounds__(256) void k_exp_probe(const float* x, const float* m,
                                                   float* e, int64_t n, Clip clip) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    if constexpr (MODE == kExpRaw)
      e[i] = __builtin_amdgcn_exp2f(x[i]);
    else
      e[i] = exp_shift_clip<MODE>(x[i], row_shift(m[i], clip));
  }
}

// Plain copy with 128-bit streaming accesses: the memory-bound ceiling that
// the paper compares softmax against (Sec. 2.6), for the same bytes moved.
constexpr int kCopyUnroll = 4;
__global__ __launch_bounds__(256) void k_copy4(const float* x, float* y, int64_t n4) {
  const int64_t step = static_cast<int64_t>(gridDim.x) * 256 * kCopyUnroll;
  int64_t i = static_cast<int64_t>(blockIdx.x) * 256 * kCopyUnroll + threadIdx.x;
  // Full groups: all loads in flight before the stores, no per-element guard.
  for (; i + (kCopyUnroll - 1) * 256 < n4; i += step) {
    f32x4 t[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) t[u] = ld_stream(x + 4 * (i + u * 256));
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) st_stream(y + 4 * (i + u * 256), t[u]);
  }
  // The last, partial group of this thread.
  for (int u = 0; u < kCopyUnroll; ++u) {
    const int64_t k = i + u * 256;
    if (k < n4) st_stream(y + 4 * k, ld_stream(x + 4 * k));
  }
}

__global__ __launch_bounds__(256) void k_copy1(const float* x, float* y, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256)
    y[i] = x[i];
}

}  // namespace smx
