// HIP kernels for the clipped row softmax on gfx950.
//
// Every kernel computes, per row of a row-major [rows, cols] fp32 matrix,
//   y = exp(max(x - rowmax, -64)) / sum(exp(max(x - rowmax, -64)))
// in the order of the paper's optimised functor (Sec. 2.3, Fig. 4: row max,
// subtract, exp, row sum, scale by the reciprocal of the sum) with the clip
// of the reference functor (Sec. 1.2, Fig. 1).  Unlike that CPU functor, no
// kernel uses y as scratch: x is read from HBM once (twice for split rows)
// and y is written once.
//
//   k_packed      cols <= 64: a workgroup stages a tile of whole rows in LDS
//                 with 128-bit loads, then groups of G lanes reduce one row
//                 each with DPP, then the tile goes back out with 128-bit
//                 stores.
//   k_wave_row    cols <= 4096: one wavefront per row, the row held in VGPRs.
//   k_block_row   cols <= 32768: one workgroup per row, the row held in
//                 VGPRs, per-wave partials combined through LDS.
//   k_split_stats / k_split_apply   longer rows: G workgroups per row; the
//                 first pass writes a (max, sum) partial per chunk, the
//                 second merges them and writes the chunk's outputs.
//
// In-place calls (x == y) are safe in every kernel: each element is read
// into registers (or LDS) by the workgroup that later writes it, before any
// write to it, and no workgroup reads another's outputs.
#pragma once

#include "sm_device.hpp"

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

// Loads N = 4*V elements of one row (or chunk) into registers: element i of
// this lane sits at column base + lane_off + stride*i (scalar) or, for
// 128-bit loads, at base + 4*(lane_off + stride*j) + k with i = 4j + k.
// Columns at or past `limit` read as -inf.
template <int V, bool VEC4>
__device__ __forceinline__ void load_strip(float (&v)[4 * V], const float* row,
                                           int64_t base, int64_t lane_off,
                                           int64_t stride, int64_t limit) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int64_t c = base + 4 * (lane_off + stride * j);
      if (c < limit) {
        const float4 q = *reinterpret_cast<const float4*>(row + c);
        v[4 * j + 0] = q.x;
        v[4 * j + 1] = q.y;
        v[4 * j + 2] = q.z;
        v[4 * j + 3] = q.w;
      } else {
        v[4 * j + 0] = v[4 * j + 1] = v[4 * j + 2] = v[4 * j + 3] = kNegInf;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      const int64_t c = base + lane_off + stride * i;
      v[i] = (c < limit) ? row[c] : kNegInf;
    }
  }
}

template <int V, bool VEC4>
__device__ __forceinline__ bool strip_valid(int i, int64_t base, int64_t lane_off,
                                            int64_t stride, int64_t limit) {
  if constexpr (VEC4)
    return base + 4 * (lane_off + stride * (i >> 2)) < limit;
  else
    return base + lane_off + stride * i < limit;
}

// Replaces v by the clipped exponentials (0 for columns past `limit`) and
// returns this lane's pairwise partial sum.
template <int V, bool VEC4>
__device__ __forceinline__ float exp_strip(float (&v)[4 * V], float neg_m, int64_t base,
                                           int64_t lane_off, int64_t stride,
                                           int64_t limit) {
#pragma unroll
  for (int i = 0; i < 4 * V; ++i)
    v[i] = strip_valid<V, VEC4>(i, base, lane_off, stride, limit)
               ? exp_shift_clip(v[i], neg_m)
               : 0.0f;
  return tree_sum(v);
}

template <int V, bool VEC4>
__device__ __forceinline__ void store_strip(const float (&v)[4 * V], float scale,
                                            float* row, int64_t base, int64_t lane_off,
                                            int64_t stride, int64_t limit) {
  if constexpr (VEC4) {
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int64_t c = base + 4 * (lane_off + stride * j);
      if (c < limit) {
        float4 q;
        q.x = v[4 * j + 0] * scale;
        q.y = v[4 * j + 1] * scale;
        q.z = v[4 * j + 2] * scale;
        q.w = v[4 * j + 3] * scale;
        *reinterpret_cast<float4*>(row + c) = q;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4 * V; ++i) {
      const int64_t c = base + lane_off + stride * i;
      if (c < limit) row[c] = v[i] * scale;
    }
  }
}

// ---------------------------------------------------------------------------
// (a) Packed rows, cols <= G*EPL with G lanes per row.
//
// A 256-thread workgroup owns tiles of TILE = 4 * (256/G) consecutive rows.
// TILE is a multiple of 4, so a tile starts on a 16-byte boundary whenever
// x and y do, whatever cols is (cols = 50 gives 200-byte rows).
template <int G, int EPL, bool VEC4>
__global__ __launch_bounds__(256) void k_packed(const float* x, float* y, int64_t rows,
                                                int64_t cols) {
  constexpr int kRowsPerPass = 256 / G;
  constexpr int kPasses = 4;
  constexpr int kTile = kRowsPerPass * kPasses;
  __shared__ float tile[kTile * G * EPL];

  const int tid = threadIdx.x;
  const int ccols = static_cast<int>(cols);
  const int64_t ntiles = (rows + kTile - 1) / kTile;
  const int j = tid % G;

  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t row0 = t * kTile;
    const int nr = static_cast<int>(rows - row0 < kTile ? rows - row0 : kTile);
    const int n = nr * ccols;
    const float* xs = x + row0 * cols;
    float* ys = y + row0 * cols;

    if constexpr (VEC4) {
      const int n4 = n >> 2;
      for (int i = tid; i < n4; i += 256)
        reinterpret_cast<float4*>(tile)[i] = reinterpret_cast<const float4*>(xs)[i];
      for (int i = (n4 << 2) + tid; i < n; i += 256) tile[i] = xs[i];
    } else {
      for (int i = tid; i < n; i += 256) tile[i] = xs[i];
    }
    __syncthreads();

#pragma unroll
    for (int p = 0; p < kPasses; ++p) {
      const int r = p * kRowsPerPass + tid / G;
      const bool active = r < nr;
      float* tr = tile + r * ccols;
      float v[EPL];
#pragma unroll
      for (int k = 0; k < EPL; ++k) {
        const int c = j + G * k;
        v[k] = (active && c < ccols) ? tr[c] : kNegInf;
      }
      const float m = seg_max<G>(array_max(v));
      const float neg_m = -m;
#pragma unroll
      for (int k = 0; k < EPL; ++k) {
        const int c = j + G * k;
        v[k] = (active && c < ccols) ? exp_shift_clip(v[k], neg_m) : 0.0f;
      }
      const float s = seg_sum<G>(tree_sum(v));
      const float rcp = 1.0f / s;
#pragma unroll
      for (int k = 0; k < EPL; ++k) {
        const int c = j + G * k;
        if (active && c < ccols) tr[c] = v[k] * rcp;
      }
    }
    __syncthreads();

    if constexpr (VEC4) {
      const int n4 = n >> 2;
      for (int i = tid; i < n4; i += 256)
        reinterpret_cast<float4*>(ys)[i] = reinterpret_cast<const float4*>(tile)[i];
      for (int i = (n4 << 2) + tid; i < n; i += 256) ys[i] = tile[i];
    } else {
      for (int i = tid; i < n; i += 256) ys[i] = tile[i];
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// (b) One wavefront per row, cols <= 256*V (VEC4) or 256*V scalar elements.
// Four wavefronts per workgroup work on four rows independently.
template <int V, bool VEC4>
__global__ __launch_bounds__(256) void k_wave_row(const float* x, float* y, int64_t rows,
                                                  int64_t cols) {
  const int lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  for (int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wave; row < rows;
       row += static_cast<int64_t>(gridDim.x) * 4) {
    const float* xr = x + row * cols;
    float* yr = y + row * cols;
    float v[4 * V];
    load_strip<V, VEC4>(v, xr, 0, lane, 64, cols);
    const float m = seg_max<64>(array_max(v));
    const float neg_m = -m;
    const float s = seg_sum<64>(exp_strip<V, VEC4>(v, neg_m, 0, lane, 64, cols));
    const float rcp = 1.0f / s;
    store_strip<V, VEC4>(v, rcp, yr, 0, lane, 64, cols);
  }
}

// ---------------------------------------------------------------------------
// (c) One workgroup of NT threads per row, cols <= 4*V*NT.
template <int NT, int V, bool VEC4>
__global__ __launch_bounds__(NT) void k_block_row(const float* x, float* y, int64_t rows,
                                                  int64_t cols) {
  constexpr int NW = NT / 64;
  __shared__ float red_max[NW];
  __shared__ float red_sum[NW];
  const int tid = threadIdx.x;
  for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
    const float* xr = x + row * cols;
    float* yr = y + row * cols;
    float v[4 * V];
    load_strip<V, VEC4>(v, xr, 0, tid, NT, cols);
    const float m = block_max<NW>(array_max(v), red_max);
    const float neg_m = -m;
    const float s = block_sum<NW>(exp_strip<V, VEC4>(v, neg_m, 0, tid, NT, cols), red_sum);
    const float rcp = 1.0f / s;
    store_strip<V, VEC4>(v, rcp, yr, 0, tid, NT, cols);
  }
}

// ---------------------------------------------------------------------------
// (c, split) Rows longer than one workgroup's registers: G = ceil(cols/CH)
// workgroups per row, CH = 4*V*NT columns each.
//
// Pass 1 writes part[row*G + g] = (m_g, s_g): the chunk max and the chunk's
// sum of exp(max(x - m_g, -64)).  A chunk whose max is -inf stores s_g = its
// element count, so that the merge below gives count * e^-64, the clipped
// value of its -inf elements.
//
// Pass 2 merges a row's partials (every wavefront of the workgroup does the
// same merge, so all hold the same bits):  M = max_g m_g,
// S = sum_g s_g * exp(max(m_g - M, -64)), then writes
// y = exp(max(x - M, -64)) / S.  Using the clip relative to m_g inside a
// partial changes S by at most cols * e^-64 relative (below 1e-22 at any
// supported length), far under fp32 resolution.
template <int NT, int V, bool VEC4>
__global__ __launch_bounds__(NT) void k_split_stats(const float* x, float2* part,
                                                    int64_t rows, int64_t cols,
                                                    int64_t chunks) {
  constexpr int NW = NT / 64;
  constexpr int64_t CH = int64_t(4) * V * NT;
  __shared__ float red_max[NW];
  __shared__ float red_sum[NW];
  const int tid = threadIdx.x;
  const int64_t total = rows * chunks;
  for (int64_t b = blockIdx.x; b < total; b += gridDim.x) {
    const int64_t row = b / chunks;
    const int64_t g = b - row * chunks;
    const int64_t c0 = g * CH;
    const float* xr = x + row * cols;
    float v[4 * V];
    load_strip<V, VEC4>(v, xr, c0, tid, NT, cols);
    const float m = block_max<NW>(array_max(v), red_max);
    const bool empty_max = (m == kNegInf);
    const float neg_m = empty_max ? 0.0f : -m;
    float s = block_sum<NW>(exp_strip<V, VEC4>(v, neg_m, c0, tid, NT, cols), red_sum);
    if (empty_max) {
      const int64_t left = cols - c0;
      s = static_cast<float>(left < CH ? left : CH);
    }
    if (tid == 0) part[b] = make_float2(m, s);
  }
}

template <int NT, int V, bool VEC4>
__global__ __launch_bounds__(NT) void k_split_apply(const float* x, float* y,
                                                    const float2* part, int64_t rows,
                                                    int64_t cols, int64_t chunks) {
  constexpr int64_t CH = int64_t(4) * V * NT;
  const int tid = threadIdx.x;
  const int lane = __lane_id();
  const int64_t total = rows * chunks;
  for (int64_t b = blockIdx.x; b < total; b += gridDim.x) {
    const int64_t row = b / chunks;
    const int64_t g = b - row * chunks;
    const int64_t c0 = g * CH;
    const float* xr = x + row * cols;
    float* yr = y + row * cols;
    float v[4 * V];
    load_strip<V, VEC4>(v, xr, c0, tid, NT, cols);

    const float2* pr = part + row * chunks;
    float mm = kNegInf;
    for (int64_t l = lane; l < chunks; l += 64) mm = fmaxf(mm, pr[l].x);
    const float neg_big_m = -seg_max<64>(mm);
    float ss = 0.0f;
    for (int64_t l = lane; l < chunks; l += 64) {
      const float2 p = pr[l];
      ss = ss + p.y * exp_shift_clip(p.x, neg_big_m);
    }
    const float rcp = 1.0f / seg_sum<64>(ss);

#pragma unroll
    for (int i = 0; i < 4 * V; ++i)
      v[i] = exp_shift_clip(v[i], neg_big_m);
    store_strip<V, VEC4>(v, rcp, yr, c0, tid, NT, cols);
  }
}

// ---------------------------------------------------------------------------
// Diagnostics.

// e[i] = exp(max(x[i] - m[i], -64)), through the same device routine the
// softmax kernels use.
__global__ __launch_bounds__(256) void k_exp_probe(const float* x, const float* m,
                                                   float* e, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256)
    e[i] = exp_shift_clip(x[i], -m[i]);
}

// Plain copy with 128-bit accesses: the memory-bound ceiling that the paper
// compares softmax against (Sec. 2.6), for the same bytes moved.
constexpr int kCopyUnroll = 4;
__global__ __launch_bounds__(256) void k_copy4(const float4* x, float4* y, int64_t n4) {
  const int64_t step = static_cast<int64_t>(gridDim.x) * 256 * kCopyUnroll;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 * kCopyUnroll + threadIdx.x;
       i < n4; i += step) {
    float4 t[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int64_t k = i + u * 256;
      if (k < n4) t[u] = x[k];
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int64_t k = i + u * 256;
      if (k < n4) y[k] = t[u];
    }
  }
}

__global__ __launch_bounds__(256) void k_copy1(const float* x, float* y, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256)
    y[i] = x[i];
}

}  // namespace smx
