// Fused softmax attention over small tiles on gfx950 matrix cores:
//
//   O_b = softmax_clip(scale * Q_b K_b^T) V_b        for every batch element b
//
// with Q_b [lq, d], K_b [lk, d], V_b [lk, dv], O_b [lq, dv], fp32, row-major
// and contiguous per batch.  The softmax step is the library's clipped row
// softmax over the keys (Sec. 1.1 Eq. (1), the clip of Sec. 1.2 Fig. 1, no
// clip as in Sec. 2.3 Fig. 4); around it are the two products of the DAM
// model's attention, whose softmax the paper optimises (Sec. 1).  The scores
// never leave registers: they are produced by one matrix-core product,
// normalised in place and consumed as the operand of the next.
//
// Mapping (v_mfma_f32_16x16x4f32: C[i][j] += sum_k A[i][k] B[k][j], with
// A[i][k] in lane i + 16k, B[k][j] in lane j + 16k, and C[i][j] in lane
// j + 16 (i / 4), register i % 4):
//
//   * A workgroup of 4 wavefronts takes one batch element and a block of up
//     to 64 queries; wavefront w takes queries 16w .. 16w+15 of the block.
//     Write lane = j + 16 g (j = lane % 16, g = lane / 16).
//   * Scores, transposed: S^T[key][query] = sum_t K[key][t] Q[query][t],
//     for NKT key tiles of 16.  The contraction index runs over d in blocks
//     of 16; within a block, lane g of step s holds t = 16 blk + 4 g + s, so
//     each lane loads 4 consecutive t of its key (A) and its query (B) with
//     one 128-bit load per block.  The order of the terms of a dot product
//     is a permutation of t; every product is still taken once.
//   * Accumulator register r of key tile kt in lane (j, g) holds the score
//     of query j and key 16 kt + 4 g + r.  A query's keys are spread over its
//     4 registers x NKT tiles and the 4 lanes j, j+16, j+32, j+48, so the
//     row max and row sum take a lane-local reduction and two cross-lane
//     swaps (permlane16, permlane32).  Keys past lk are masked out of both.
//   * The normalised weights are then exactly the A operand of P.V for the
//     contraction step (kt, r): lane (j, g) holds P[query j][key 16kt+4g+r],
//     and the B operand is V[key 16kt+4g+r][column 16 nt + j].  The output
//     accumulator of column tile nt holds O[query 4g + r][column 16 nt + j].
//
// Padding: queries past lq load zeros and store nothing; keys past lk get
// weight exactly 0 and load zero value rows; t past d loads zeros; columns
// past dv load zeros and store nothing.
#pragma once

#include "sm_device.hpp"

namespace smx {

typedef float f32x4m __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4m mfma16x16x4(float a, float b, f32x4m c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Buffer resources.  Every operand is addressed through a raw buffer
// resource over the batch element's (or the wave's) own rows with a 32-bit
// byte offset per lane, so a load needs one offset register and no 64-bit
// pointer arithmetic.  The hardware checks each access against the
// resource's size: loads past it return 0 and stores past it are dropped,
// which is how rows past lq and lk are padded and skipped.  Offsets are
// kept below 2^31: a resource never spans more than 64 rows of at most
// 65536 floats.
constexpr int kBufDword3 = 0x00020000;  // raw buffer, 32-bit data format
constexpr int kBufOff = 0x7ffffff0;     // an offset past any resource here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), static_cast<short>(0), bytes,
                                           kBufDword3);
}

// Four consecutive floats of a row at byte offset `off` (128-bit when VEC4,
// else four 32-bit loads), zero when `ok` is false, past the resource, or
// (32-bit loads) at or past the row's `left` remaining columns.  With VEC4
// the row length is a multiple of 4, so the four are all in the row or all
// out of it.
template <bool VEC4>
__device__ __forceinline__ f32x4m buf_load4(__amdgpu_buffer_rsrc_t r, int off, bool ok,
                                            int left = 4) {
  if constexpr (VEC4) {
    const int o = ok ? off : kBufOff;
    return __builtin_bit_cast(f32x4m, __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, 0));
  } else {
    f32x4m x;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = (ok & (i < left)) ? off + 4 * i : kBufOff;
      x[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, o, 0, 0));
    }
    return x;
  }
}

template <int NKT, bool VEC4, bool WIDE>
__global__ __launch_bounds__(256) void k_attention(const float* q, const float* k,
                                                   const float* v, float* o, int64_t batch,
                                                   int lq, int lk, int d, int dv, float scale,
                                                   Clip clip) {
  const int lane = __lane_id();
  const int j = lane & 15;
  const int g = lane >> 4;
  // The wave index is uniform across the wave; saying so keeps the buffer
  // resources built from it in scalar registers.
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int qblocks = (lq + 63) >> 6;
  const int64_t items = batch * qblocks;

  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t b = item / qblocks;
    const int q0 = static_cast<int>(item - b * qblocks) * 64 + 16 * w;  // this wave's queries
    if (q0 >= lq) continue;                       // wave-uniform; no barriers below
    const int nq = lq - q0 < 16 ? lq - q0 : 16;   // valid queries of this wave
    // The wave's 16 query rows of Q and O, and the batch element's K and V.
    const __amdgpu_buffer_rsrc_t rq =
        make_rsrc(q + (b * lq + q0) * static_cast<int64_t>(d), nq * d * 4);
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + b * lk * static_cast<int64_t>(d), lk * d * 4);
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + b * lk * static_cast<int64_t>(dv), lk * dv * 4);
    const __amdgpu_buffer_rsrc_t ro =
        make_rsrc(o + (b * lq + q0) * static_cast<int64_t>(dv), nq * dv * 4);

    // ---- scores S^T = K Q^T for this wave's 16 queries --------------------
    // Lane (j, g) reads query j and key 16 kt + j at columns t0 .. t0+3,
    // t0 = 16 blk + 4 g; columns past d (last block only) read as zero.
    const int qoff = (j * d + 4 * g) * 4;
    const int koff = (j * d + 4 * g) * 4;
    const int kstride = 16 * d * 4;               // one key tile
    f32x4m acc[NKT];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) acc[kt] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
    const int nblk = (d + 15) >> 4;               // uniform trip count for the matrix ops
    if (nblk > 0) {
      // Operands of blocks blk, blk+1 are in registers while block blk+2 is
      // loaded: two blocks of loads stay in flight behind the matrix ops.
      const int left0 = d - 4 * g, left1 = d - 16 - 4 * g;
      f32x4m qf0 = buf_load4<VEC4>(rq, qoff, left0 > 0, left0);
      f32x4m qf1 = buf_load4<VEC4>(rq, qoff + 64, (nblk > 1) & (left1 > 0), left1);
      f32x4m kf0[NKT], kf1[NKT];
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        kf0[kt] = buf_load4<VEC4>(rk, koff + kt * kstride, left0 > 0, left0);
        kf1[kt] = buf_load4<VEC4>(rk, koff + kt * kstride + 64, (nblk > 1) & (left1 > 0), left1);
      }
      for (int blk = 0; blk < nblk; ++blk) {
        const int left = d - 16 * (blk + 2) - 4 * g;
        const bool more = (blk + 2 < nblk) & (left > 0);
        const int step = 64 * (blk + 2);
        const f32x4m qn = buf_load4<VEC4>(rq, qoff + step, more, left);
        f32x4m kn[NKT];
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
          kn[kt] = buf_load4<VEC4>(rk, koff + kt * kstride + step, more, left);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
#pragma unroll
          for (int kt = 0; kt < NKT; ++kt) acc[kt] = mfma16x16x4(kf0[kt][s], qf0[s], acc[kt]);
        }
        qf0 = qf1;
        qf1 = qn;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt) {
          kf0[kt] = kf1[kt];
          kf1[kt] = kn[kt];
        }
      }
    }

    // ---- clipped softmax over the keys of query j -------------------------
    // Only the last key tile can hold keys past lk (NKT = ceil(lk / 16)).
    float e[4 * NKT];
    float m = -__builtin_inff();
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool key_ok = kt < NKT - 1 || 16 * kt + 4 * g + r < lk;
        const float sv = acc[kt][r] * scale;
        e[4 * kt + r] = sv;
        m = key_ok ? fmaxf(m, sv) : m;
      }
    }
    m = fmaxf(m, row16_partner(m));
    m = fmaxf(m, half32_partner(m));
    const RowShift rs = row_shift(m, clip);
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool key_ok = kt < NKT - 1 || 16 * kt + 4 * g + r < lk;
        const float ev = exp_shift_clip<WIDE ? kExpWide : kExpAccurate>(e[4 * kt + r], rs);
        e[4 * kt + r] = key_ok ? ev : 0.0f;
      }
    }
    float sum = tree_sum(e);
    sum = sum + row16_partner(sum);
    sum = sum + half32_partner(sum);
    const float rcp = 1.0f / sum;
#pragma unroll
    for (int i = 0; i < 4 * NKT; ++i) e[i] = e[i] * rcp;

    // ---- O = P V ----------------------------------------------------------
    // Contraction step i = 4 kt + r takes key 16 kt + 4 g + r in lane
    // (j, g): byte offset vlane + i' * dv * 4 with i' = 16 kt + r.  Keys past
    // lk fall outside the resource and read as zero.
    const int vlane = 4 * g * dv * 4;
    const int orow = 4 * g * dv * 4;              // O row 4 g + r of the wave
    // Full 64-column blocks with 128-bit access (VEC4): lane j takes
    // columns c0 + 4 j .. c0 + 4 j + 3, one per column tile u, so a lane's
    // four tiles are one 128-bit load of V and one 128-bit store of O.  The
    // block is done in two halves of 2 NKT contraction steps; the next
    // half's loads are in flight while this half's matrix ops run.
    constexpr int H = 2 * NKT;
    const int nfull = VEC4 ? dv >> 6 : 0;
    if (nfull > 0) {
      f32x4m va[H], vh[H];
#pragma unroll
      for (int i = 0; i < H; ++i)
        va[i] = buf_load4<true>(rv, vlane + ((16 * (i >> 2) + (i & 3)) * dv + 4 * j) * 4, true);
      for (int cb = 0; cb < nfull; ++cb) {
        const int c = 64 * cb + 4 * j;
#pragma unroll
        for (int i = 0; i < H; ++i) {
          const int ii = H + i;
          vh[i] = buf_load4<true>(rv, vlane + ((16 * (ii >> 2) + (ii & 3)) * dv + c) * 4, true);
        }
        __builtin_amdgcn_sched_barrier(0);
        f32x4m oacc[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) oacc[u] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < H; ++i) {
#pragma unroll
          for (int u = 0; u < 4; ++u) oacc[u] = mfma16x16x4(e[i], va[i][u], oacc[u]);
        }
        const bool next = cb + 1 < nfull;
#pragma unroll
        for (int i = 0; i < H; ++i)
          va[i] = buf_load4<true>(rv, vlane + ((16 * (i >> 2) + (i & 3)) * dv + c + 64) * 4, next);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < H; ++i) {
#pragma unroll
          for (int u = 0; u < 4; ++u) oacc[u] = mfma16x16x4(e[H + i], vh[i][u], oacc[u]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const f32x4m ov = {oacc[0][r], oacc[1][r], oacc[2][r], oacc[3][r]};
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(
              __attribute__((ext_vector_type(4))) unsigned, ov), ro, orow + (r * dv + c) * 4, 0, 0);
        }
      }
    }
    // The remaining columns (all of them without 128-bit access), one plain
    // 16-column tile at a time: lane j takes column c0 + j.  Columns past dv
    // would land in the next row, so their loads use an offset past the
    // resource, and their stores are skipped.
    for (int c0 = 64 * nfull; c0 < dv; c0 += 16) {
      const int c = c0 + j;
      const bool c_ok = c < dv;
      float vs[4 * NKT];
#pragma unroll
      for (int i = 0; i < 4 * NKT; ++i) {
        const int off = c_ok ? vlane + ((16 * (i >> 2) + (i & 3)) * dv + c) * 4 : kBufOff;
        vs[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rv, off, 0, 0));
      }
      __builtin_amdgcn_sched_barrier(0);
      f32x4m oa = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int i = 0; i < 4 * NKT; ++i) oa = mfma16x16x4(e[i], vs[i], oa);
      // Plain stores here: a 32-bit buffer store of an accumulator element
      // was compiled to store element 0 for every r by this toolchain.
      float* orow_p = o + (b * lq + q0 + 4 * g) * static_cast<int64_t>(dv) + c;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if ((q0 + 4 * g + r < lq) & c_ok)
          __builtin_nontemporal_store(oa[r], orow_p + static_cast<int64_t>(r) * dv);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// The same computation with K_b and V_b staged in LDS, for problems whose
// lk * (d + dv) floats fit in kAttnLdsBytes and whose rows allow 128-bit
// access (d % 4 == dv % 4 == 0, 16-byte aligned operands).  Four wavefronts
// take one batch element (and one block of 64 queries):
//
//   1. the 4 wavefronts copy K_b and V_b, which are contiguous, into LDS
//      with LDS-DMA loads (global_load_lds_dwordx4: 1 KiB per wavefront
//      instruction, no registers), while each wavefront loads its 16 query
//      rows into registers;
//   2. the score product reads its K operands from LDS, the weights stay in
//      registers as before, and the P.V product reads V from LDS;
//   3. a barrier ends the item before the next one overwrites the LDS.
//
// Each batch element's K and V cross HBM and L2 once, instead of once per
// wavefront, and the matrix-op operands come from LDS.  Two schedules:
//
//   * k_attention_lds: two workgroups of 4 wavefronts per CU, each with its
//     own 80 KiB of LDS, one item after another (copy, wait, compute).  The
//     two do not stay out of step, so copies and matrix ops overlap only
//     in part.
//   * k_attention_pp: one workgroup of 8 wavefronts per CU in two teams that
//     take turns: one computes an item while the other copies the next.
//     Used with d = dv = DC known at compile time (the DAM tile, DC = 200),
//     where the masks and branches of the d loops fold away, the matrix ops
//     issue back to back, and the last key tile (at most 2 keys) is scored
//     on the VALU; with d at run time one wavefront per SIMD computes too
//     slowly for this schedule.
constexpr int kAttnLdsBytes = 80 * 1024;  // one batch element's K_b and V_b
constexpr int kAttnMaxDQ = 224;           // d up to this keeps Q in registers
constexpr int kAttnQB = kAttnMaxDQ / 16;  // 16-wide blocks of d in registers

typedef __attribute__((address_space(3))) char attn_lds_char;

// `bytes` bytes from global memory at src into LDS at dst with LDS-DMA loads,
// spread over 4 wavefronts wt = 0..3: each instruction writes its 64 lanes'
// 16 bytes to consecutive LDS bytes from the (uniform) destination.  Whole
// 1 KiB chunks need no lane mask; in a partial last chunk the lanes past the
// end are off.
__device__ __forceinline__ void attn_copy_lds(float* dst, const float* src, int bytes, int wt,
                                              int lane) {
  attn_lds_char* dl = (attn_lds_char*)dst;
  const char* gs = reinterpret_cast<const char*>(src);
  int c = 1024 * wt;
  for (; c + 1024 <= bytes; c += 4096)
    __builtin_amdgcn_global_load_lds(gs + c + 16 * lane, dl + c, 16, 0, 0);
  if (c < bytes && c + 16 * lane < bytes)
    __builtin_amdgcn_global_load_lds(gs + c + 16 * lane, dl + c, 16, 0, 0);
}

// K_b and V_b into LDS at lk_s and lv_s (attn_copy_lds, K_b first).
__device__ __forceinline__ void attn_copy_kv(float* lk_s, float* lv_s, const float* kb,
                                             const float* vb, int kbytes, int vbytes, int wt,
                                             int lane) {
  attn_copy_lds(lk_s, kb, kbytes, wt, lane);
  attn_copy_lds(lv_s, vb, vbytes, wt, lane);
}

// A wavefront's nq <= 16 query rows q0 .. of batch element b into
// registers: block blk of lane (j, g) holds Q[q0 + j][16 blk + 4 g .. + 3].
// Rows past nq and columns past d read as zero (buffer range check and the
// offset mask).
template <int DC>
__device__ __forceinline__ void attn_load_q(f32x4m (&qf)[kAttnQB], const float* q, int64_t b,
                                            int q0, int nq, int lq, int d, int j, int g) {
  const __amdgpu_buffer_rsrc_t rq =
      make_rsrc(q + (b * lq + q0) * static_cast<int64_t>(d), nq * d * 4);
  const int qoff = (j * d + 4 * g) * 4;
  const int nblk = (d + 15) >> 4;
#pragma unroll
  for (int blk = 0; blk < kAttnQB; ++blk) {
    // With d known at compile time a block wholly inside d needs no mask.
    const bool in_d = (DC != 0 && 16 * blk + 16 <= d) || 16 * blk + 4 * g < d;
    qf[blk] = buf_load4<true>(rq, qoff + 64 * blk, (blk < nblk) & in_d);
  }
}

// The value product for d = dv = DC known at compile time, with the
// weights' exponentials taken inside it: sc holds the scaled scores of the
// wavefront's 16 queries (lane (j, g): query j, keys 16 kt + 4 g + r at
// 4 kt + r), rs the row shift of query j.  Contraction step i = 4 kt + r
// multiplies key 16 kt + 4 g + r's unnormalised weight into all dv columns
// (one 16x16x4 matrix op per 16 columns), and the next step's exponential
// is independent of this step's matrix ops, so its VALU work issues beside
// them instead of before the whole product.  O is scaled by 1 / sum when it
// is stored: the sum of query 4 g + r's weights comes from lane 4 g + r.
// Keys past lk have weight 0 and read the zero row after V_b.
template <int NKT, bool WIDE, int DC, bool VT>
__device__ __forceinline__ void attn_pv_stream(const float (&sc)[4 * NKT], const RowShift& rs,
                                               const float* lv_s, float* o, int64_t b, int q0,
                                               int nq, int lq, int lk, int j, int g) {
  constexpr int dv = DC;
  constexpr int NS = 4 * NKT;                  // contraction steps
  constexpr int NF = DC / 64;                  // 64-column blocks: 4 ops of 16 columns
  constexpr int NT = (DC - 64 * NF + 15) / 16; // 16-column tiles after them
  auto key_ok = [&](int i) {
    const int kt = i >> 2, r = i & 3;
    return kt < NKT - 1 || (!(VT && r >= 2) && 16 * kt + 4 * g + r < lk);
  };
  // A step whose smallest key (lane group 0) is past lk has zero weight in
  // every lane: its matrix ops are skipped (uniform).
  auto step_live = [&](int i) { return (i >> 2) < NKT - 1 || 16 * (i >> 2) + (i & 3) < lk; };
  auto vrow = [&](int i) {
    const int key = 16 * (i >> 2) + 4 * g + (i & 3);
    return ((i >> 2) < NKT - 1 || key < lk ? key : lk) * dv;
  };
  auto weight = [&](int i) {
    return key_ok(i) ? exp_shift_clip<WIDE ? kExpWide : kExpAccurate>(sc[i], rs) : 0.0f;
  };
  f32x4m oacc[NF][4];
  f32x4m ot[NT > 0 ? NT : 1];
#pragma unroll
  for (int cb = 0; cb < NF; ++cb)
#pragma unroll
    for (int u = 0; u < 4; ++u) oacc[cb][u] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int t = 0; t < NT; ++t) ot[t] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
  // Value operands of a step: lane j reads columns 64 cb + 4 j .. + 3 of
  // each block and column 64 NF + 16 t + j of each tile (inside V_b and the
  // zero row for every lane, so no mask).
  f32x4m va[2][NF > 0 ? NF : 1];
  float vt[2][NT > 0 ? NT : 1];
  auto load_v = [&](int i, int slot) {
    const float* row = lv_s + vrow(i);
#pragma unroll
    for (int cb = 0; cb < NF; ++cb)
      va[slot][cb] = *reinterpret_cast<const f32x4m*>(row + 64 * cb + 4 * j);
#pragma unroll
    for (int t = 0; t < NT; ++t) vt[slot][t] = row[64 * NF + 16 * t + j];
  };
  load_v(0, 0);
  float w_next = weight(0);
  float psum = 0.0f;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const float w = w_next;
    if (i + 1 < NS) {
      load_v(i + 1, (i + 1) & 1);
      w_next = weight(i + 1);
    }
    if (step_live(i)) {
      psum += w;
#pragma unroll
      for (int cb = 0; cb < NF; ++cb)
#pragma unroll
        for (int u = 0; u < 4; ++u) oacc[cb][u] = mfma16x16x4(w, va[i & 1][cb][u], oacc[cb][u]);
#pragma unroll
      for (int t = 0; t < NT; ++t) ot[t] = mfma16x16x4(w, vt[i & 1][t], ot[t]);
    }
  }
  float sum = psum + row16_partner(psum);
  sum = sum + half32_partner(sum);
  const float rcp = 1.0f / sum;
  float rq[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) rq[r] = __shfl(rcp, 4 * g + r);
  const __amdgpu_buffer_rsrc_t ro =
      make_rsrc(o + (b * lq + q0) * static_cast<int64_t>(dv), nq * dv * 4);
  const int orow = 4 * g * dv * 4;
#pragma unroll
  for (int cb = 0; cb < NF; ++cb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const f32x4m ov = {oacc[cb][0][r] * rq[r], oacc[cb][1][r] * rq[r], oacc[cb][2][r] * rq[r],
                         oacc[cb][3][r] * rq[r]};
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, ov), ro,
          orow + (r * dv + 64 * cb + 4 * j) * 4, 0, 0);
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int c = 64 * NF + 16 * t + j;
    float* orow_p = o + (b * lq + q0 + 4 * g) * static_cast<int64_t>(dv) + c;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if ((q0 + 4 * g + r < lq) & (c < dv))
        __builtin_nontemporal_store(ot[t][r] * rq[r], orow_p + static_cast<int64_t>(r) * dv);
    }
  }
}

// The weights and the value product for d at run time (DC = 0): e holds
// the scaled scores as in attn_pv_stream and becomes the normalised weights
// before the product.
template <int NKT, bool WIDE>
__device__ __forceinline__ void attn_pv_rows(float (&e)[4 * NKT], const RowShift& rs,
                                             const float* lv_s, float* o, int64_t b, int q0,
                                             int nq, int lq, int lk, int dv, int j, int g) {
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool key_ok = kt < NKT - 1 || 16 * kt + 4 * g + r < lk;
      const float ev = exp_shift_clip<WIDE ? kExpWide : kExpAccurate>(e[4 * kt + r], rs);
      e[4 * kt + r] = key_ok ? ev : 0.0f;
    }
  }
  float sum = tree_sum(e);
  sum = sum + row16_partner(sum);
  sum = sum + half32_partner(sum);
  const float rcp = 1.0f / sum;
#pragma unroll
  for (int i = 0; i < 4 * NKT; ++i) e[i] = e[i] * rcp;

  // ---- O = P V, V from LDS --------------------------------------------------
  // Contraction step i = 4 kt + r: key 16 kt + 4 g + r.  Keys past lk (only
  // in the last key tile) have weight 0; their value operand is row 0 zeroed
  // at use, since a stale value could be NaN.
  auto v_ok = [&](int i) { return (i >> 2) < NKT - 1 || 16 * (i >> 2) + 4 * g + (i & 3) < lk; };
  auto vrow = [&](int i) { return (v_ok(i) ? 16 * (i >> 2) + 4 * g + (i & 3) : 0) * dv; };
  // A step whose smallest key (lane group 0) is past lk has zero weight in
  // every lane: its matrix ops are skipped (a uniform branch; for DAM's 50
  // keys, 2 of the 16 steps).
  auto step_live = [&](int i) { return (i >> 2) < NKT - 1 || 16 * (i >> 2) + (i & 3) < lk; };
  const __amdgpu_buffer_rsrc_t ro =
      make_rsrc(o + (b * lq + q0) * static_cast<int64_t>(dv), nq * dv * 4);
  const int orow = 4 * g * dv * 4;
  const int nfull = dv >> 6;
  // Each 64-column block in four quarters of NKT contraction steps: the next
  // quarter's V rows (the next block's first, after the last) are read while
  // this quarter's matrix ops run; the key mask is applied at use.
  f32x4m vq[2][NKT];
  if (nfull > 0) {
#pragma unroll
    for (int i = 0; i < NKT; ++i)
      vq[0][i] = *reinterpret_cast<const f32x4m*>(lv_s + vrow(i) + 4 * j);
  }
  for (int cb = 0; cb < nfull; ++cb) {
    const int c = 64 * cb + 4 * j;
    f32x4m oacc[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) oacc[u] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int qi = 0; qi < 4; ++qi) {
      if (qi < 3) {
#pragma unroll
        for (int i = 0; i < NKT; ++i)
          vq[(qi + 1) & 1][i] =
              *reinterpret_cast<const f32x4m*>(lv_s + vrow((qi + 1) * NKT + i) + c);
      } else if (cb + 1 < nfull) {
#pragma unroll
        for (int i = 0; i < NKT; ++i)
          vq[0][i] = *reinterpret_cast<const f32x4m*>(lv_s + vrow(i) + c + 64);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NKT; ++i) {
        const int st = qi * NKT + i;
        if (step_live(st)) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            oacc[u] = mfma16x16x4(e[st], v_ok(st) ? vq[qi & 1][i][u] : 0.0f, oacc[u]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const f32x4m ov = {oacc[0][r], oacc[1][r], oacc[2][r], oacc[3][r]};
      __builtin_amdgcn_raw_buffer_store_b128(
          __builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, ov), ro,
          orow + (r * dv + c) * 4, 0, 0);
    }
  }
  // The remaining columns, one 16-column tile at a time: lane j takes column
  // c0 + j; a column past dv reads a masked operand.
  for (int c0 = 64 * nfull; c0 < dv; c0 += 16) {
    const int c = c0 + j;
    const bool c_ok = c < dv;
    f32x4m oa = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < 4 * NKT; ++i) {
      if (step_live(i)) {
        const float x = lv_s[vrow(i) + (c_ok ? c : 0)];
        oa = mfma16x16x4(e[i], (v_ok(i) & c_ok) ? x : 0.0f, oa);
      }
    }
    // Plain stores here: a 32-bit buffer store of an accumulator element
    // was compiled to store element 0 for every r by this toolchain.
    float* orow_p = o + (b * lq + q0 + 4 * g) * static_cast<int64_t>(dv) + c;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if ((q0 + 4 * g + r < lq) & c_ok)
        __builtin_nontemporal_store(oa[r], orow_p + static_cast<int64_t>(r) * dv);
    }
  }
}

// Scores, clipped softmax and O = P V for one wavefront's nq <= 16 queries
// q0 .. of batch element b, with K_b at lk_s and V_b at lv_s in LDS and the
// query rows in qf.  With DC != 0 (d = dv = DC), a zero row of dv + 16
// floats follows V_b, and padding keys read their values from it
// (attn_pv_stream).  With MID_SYNC the wavefront takes one workgroup barrier
// between the softmax and the value product (V_b still in flight when the
// scores start).
template <int NKT, bool WIDE, int DC, bool MID_SYNC = false>
__device__ __forceinline__ void attn_compute(const float* lk_s, const float* lv_s,
                                             const f32x4m (&qf)[kAttnQB], float* o, int64_t b,
                                             int q0, int nq, int lq, int lk, int d, int dv,
                                             float scale, Clip clip, int j, int g) {
  constexpr int QB = kAttnQB;
  const int nblk = (d + 15) >> 4;
  // With DC != 0 (the DAM tile; the host guarantees at most 2 keys in the
  // last key tile, lk <= 16 (NKT - 1) + 2) those keys' scores are dot
  // products on the VALU: lane (j, g) sums its own terms t = 16 blk + 4 g + s
  // of query j, interleaved with the other tiles' matrix ops, and the 4 lanes
  // of query j add their sums.  Only NMT tiles go through the matrix cores:
  // a 16-key tile for 2 keys cost as much as a full one (92.8 -> 82.6 us on
  // the DAM shape).
  constexpr bool VT = DC != 0 && NKT > 1;
  constexpr int NMT = VT ? NKT - 1 : NKT;  // key tiles on the matrix cores
  constexpr int NR = VT ? NKT + 1 : NKT;   // K operand rows per lane

  // ---- scores S^T = K Q^T, K from LDS ---------------------------------------
  f32x4m acc[NKT];
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt) acc[kt] = f32x4m{0.0f, 0.0f, 0.0f, 0.0f};
  float dot[2] = {0.0f, 0.0f};
  // Keys past lk read row 0: their scores are garbage (even NaN) but the
  // softmax below masks them.  Columns t past d would read the next row, and
  // 0 * NaN is NaN, so those operands are zeroed.  With VT, rows NMT and
  // NMT + 1 are the two tail keys (the same for every lane; a missing second
  // key reads the row after the last, masked the same way).
  int krow[NR];
#pragma unroll
  for (int kt = 0; kt < NR; ++kt) {
    const int key = (VT && kt >= NMT) ? 16 * NMT + (kt - NMT) : 16 * kt + j;
    krow[kt] = ((VT || kt < NKT - 1 || key < lk) ? key : 0) * d + 4 * g;
  }
  // The next block's K operands are read while this block's matrix ops run;
  // the d mask is applied at use, so no wait comes early.
  f32x4m kc[NR], kn[NR];
  if (nblk > 0) {
#pragma unroll
    for (int kt = 0; kt < NR; ++kt) kc[kt] = *reinterpret_cast<const f32x4m*>(lk_s + krow[kt]);
  }
#pragma unroll
  for (int blk = 0; blk < QB; ++blk) {
    if (blk < nblk) {  // uniform
      if (blk + 1 < nblk) {
#pragma unroll
        for (int kt = 0; kt < NR; ++kt)
          kn[kt] = *reinterpret_cast<const f32x4m*>(lk_s + krow[kt] + 16 * (blk + 1));
      }
      __builtin_amdgcn_sched_barrier(0);
      const bool t_ok = (DC != 0 && 16 * blk + 16 <= d) || 16 * blk + 4 * g < d;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int kt = 0; kt < NMT; ++kt)
          acc[kt] = mfma16x16x4(t_ok ? kc[kt][s] : 0.0f, qf[blk][s], acc[kt]);
        if constexpr (VT) {
#pragma unroll
          for (int u = 0; u < 2; ++u)
            dot[u] = __builtin_fmaf(qf[blk][s], t_ok ? kc[NMT + u][s] : 0.0f, dot[u]);
        }
      }
#pragma unroll
      for (int kt = 0; kt < NR; ++kt) kc[kt] = kn[kt];
    }
  }
  if constexpr (VT) {
    // The 4 lanes of query j add their partial sums; every lane then holds
    // the scores of keys 16 NMT and 16 NMT + 1, which the softmax reads as
    // registers 0 and 1 of the last tile (lane group 0; the others' keys
    // there are past lk and masked).
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      dot[u] = dot[u] + row16_partner(dot[u]);
      dot[u] = dot[u] + half32_partner(dot[u]);
    }
    acc[NKT - 1] = f32x4m{dot[0], dot[1], 0.0f, 0.0f};
  }

  // ---- clipped softmax over the keys of query j -----------------------------
  float e[4 * NKT];
  float m = -__builtin_inff();
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bool key_ok = kt < NKT - 1 || (!(VT && r >= 2) && 16 * kt + 4 * g + r < lk);
      const float sv = acc[kt][r] * scale;
      e[4 * kt + r] = sv;
      m = key_ok ? fmaxf(m, sv) : m;
    }
  }
  m = fmaxf(m, row16_partner(m));
  m = fmaxf(m, half32_partner(m));
  const RowShift rs = row_shift(m, clip);
  if constexpr (DC != 0) {
    if constexpr (MID_SYNC) __syncthreads();
    attn_pv_stream<NKT, WIDE, DC, VT>(e, rs, lv_s, o, b, q0, nq, lq, lk, j, g);
  } else {
    static_assert(!MID_SYNC, "the mid-item barrier is for the compile-time tile");
    attn_pv_rows<NKT, WIDE>(e, rs, lv_s, o, b, q0, nq, lq, lk, dv, j, g);
  }
}

// Two workgroups of 4 wavefronts per CU, each with its own 80 KiB of LDS:
// copy K_b and V_b, load Q, wait, compute, one item after another.  With
// DC != 0 the zero row after V_b is cleared once; no copy writes there.
template <int NKT, bool WIDE, int DC = 0>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_attention_lds(
    const float* q, const float* k, const float* v, float* o, int64_t batch, int lq, int lk,
    int d_in, int dv_in, float scale, Clip clip) {
  const int d = DC ? DC : d_in;
  const int dv = DC ? DC : dv_in;
  __shared__ __attribute__((aligned(16))) float lds[kAttnLdsBytes / 4];
  float* lk_s = lds;           // K_b: lk x d
  float* lv_s = lds + lk * d;  // V_b: lk x dv (16-byte aligned: d % 4 == 0)
  const int lane = __lane_id();
  const int j = lane & 15;
  const int g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int qblocks = (lq + 63) >> 6;
  const int64_t items = batch * qblocks;
  if constexpr (DC != 0) {
    for (int i = threadIdx.x; i < dv + 16; i += 256) lv_s[lk * dv + i] = 0.0f;
  }
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int64_t b = item / qblocks;
    const int q0 = static_cast<int>(item - b * qblocks) * 64 + 16 * w;
    const bool active = q0 < lq;  // wave-uniform
    const int nq = active ? (lq - q0 < 16 ? lq - q0 : 16) : 0;
    // The other workgroup on this CU is usually running its matrix ops on
    // the same SIMDs; a higher wave priority gets these copies and loads
    // issued first, so the memory work starts early (97.7 -> 95.6 us on the
    // DAM shape; raising the priority of the matrix-op loops instead made
    // it 104.4).
    __builtin_amdgcn_s_setprio(2);
    attn_copy_kv(lk_s, lv_s, k + b * lk * static_cast<int64_t>(d),
                 v + b * lk * static_cast<int64_t>(dv), lk * d * 4, lk * dv * 4, w, lane);
    f32x4m qf[kAttnQB];
    if (active) attn_load_q<DC>(qf, q, b, q0, nq, lq, d, j, g);
    __builtin_amdgcn_s_setprio(0);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies and loads
    __syncthreads();                // everyone's copies
    if (active)
      attn_compute<NKT, WIDE, DC>(lk_s, lv_s, qf, o, b, q0, nq, lq, lk, d, dv, scale, clip, j, g);
    __syncthreads();  // LDS is free for the next item
  }
}

// One workgroup of 8 wavefronts per CU in two teams of 4, with two 80 KiB
// LDS buffers.  The workgroup's items n = 0, 1, ... go to team n % 2 and
// buffer n % 2.  In phase n, team n % 2 computes item n while the other
// team copies item n + 1 (K, V into LDS, Q into its registers) and waits
// for it; a workgroup barrier ends the phase.  So each CU always has one
// item's copies in flight beside another's matrix ops, one wavefront of
// each team per SIMD.  Every wavefront passes the same barriers: one after
// the first copy, one per phase.  The team that copies has raised priority
// while it issues, as in k_attention_lds.
template <int NKT, bool WIDE, int DC = 0>
__global__ __launch_bounds__(512) void k_attention_pp(
    const float* q, const float* k, const float* v, float* o, int64_t batch, int lq, int lk,
    int d_in, int dv_in, float scale, Clip clip) {
  const int d = DC ? DC : d_in;
  const int dv = DC ? DC : dv_in;
  constexpr int kBuf = kAttnLdsBytes / 4;  // floats per buffer
  __shared__ __attribute__((aligned(16))) float lds[2 * kBuf];
  const int lane = __lane_id();
  const int j = lane & 15;
  const int g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int team = w >> 2;
  const int wt = w & 3;
  const int qblocks = (lq + 63) >> 6;
  const int64_t items = batch * qblocks;
  // Items of this workgroup: blockIdx.x + n gridDim.x (at least one).
  const int64_t n_items = (items - 1 - blockIdx.x) / gridDim.x + 1;
  if constexpr (DC != 0) {
    for (int i = threadIdx.x; i < dv + 16; i += 512) {
      lds[lk * (d + dv) + i] = 0.0f;
      lds[kBuf + lk * (d + dv) + i] = 0.0f;
    }
  }
  f32x4m qf[kAttnQB];
  auto where = [&](int64_t n, int64_t& b, int& q0, int& nq) {
    const int64_t item = blockIdx.x + n * gridDim.x;
    b = item / qblocks;
    q0 = static_cast<int>(item - b * qblocks) * 64 + 16 * wt;
    nq = q0 < lq ? (lq - q0 < 16 ? lq - q0 : 16) : 0;
  };
  auto stage_issue = [&](int64_t n) {
    int64_t b;
    int q0, nq;
    where(n, b, q0, nq);
    float* base = lds + (n & 1) * kBuf;
    __builtin_amdgcn_s_setprio(2);
    attn_copy_kv(base, base + lk * d, k + b * lk * static_cast<int64_t>(d),
                 v + b * lk * static_cast<int64_t>(dv), lk * d * 4, lk * dv * 4, wt, lane);
    if (nq > 0) attn_load_q<DC>(qf, q, b, q0, nq, lq, d, j, g);
    __builtin_amdgcn_s_setprio(0);
  };
  auto stage = [&](int64_t n) {
    stage_issue(n);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies and loads
  };
  // The first item has no compute to hide its copy behind.  Team 0 copies
  // K_0 and its query rows and starts the scores as soon as they land;
  // meanwhile team 1 copies V_0 alone, and item 1 only after V_0 has landed
  // (with item 1 in flight beside the scores as well, the launch took 0.9 us
  // longer).  Barriers: (A) K_0 is in LDS, (B) V_0 is in LDS (team 0 takes it
  // between its softmax and its value product), (C) item 1 is in LDS.
  {
    int64_t b;
    int q0, nq;
    where(0, b, q0, nq);
    if (team == 0) {
      __builtin_amdgcn_s_setprio(2);
      attn_copy_lds(lds, k + b * lk * static_cast<int64_t>(d), lk * d * 4, wt, lane);
      if (nq > 0) attn_load_q<DC>(qf, q, b, q0, nq, lq, d, j, g);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // (A)
      if (nq > 0)
        attn_compute<NKT, WIDE, DC, true>(lds, lds + lk * d, qf, o, b, q0, nq, lq, lk, d, dv,
                                          scale, clip, j, g);  // takes (B)
      else
        __syncthreads();  // (B)
    } else {
      __syncthreads();  // (A)
      __builtin_amdgcn_s_setprio(2);
      attn_copy_lds(lds + lk * d, v + b * lk * static_cast<int64_t>(dv), lk * dv * 4, wt, lane);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();  // (B)
      if (n_items > 1) stage_issue(1);
      __builtin_amdgcn_s_waitcnt(0);
    }
    __syncthreads();  // (C)
  }
  for (int64_t n = 1; n < n_items; ++n) {
    if (team == (n & 1)) {
      int64_t b;
      int q0, nq;
      where(n, b, q0, nq);
      const float* base = lds + (n & 1) * kBuf;
      if (nq > 0)
        attn_compute<NKT, WIDE, DC>(base, base + lk * d, qf, o, b, q0, nq, lq, lk, d, dv, scale,
                                    clip, j, g);
    } else if (n + 1 < n_items) {
      stage(n + 1);
    }
    __syncthreads();  // item n + 1 is in LDS; buffer n % 2 is free
  }
}

}  // namespace smx
