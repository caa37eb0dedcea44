/*
 * Straightforward single-thread fp32 CPU softmax -- TEST/BENCH INFRASTRUCTURE.
 *
 * This is NOT the parity oracle (that is the float64 numpy code beside it).
 * It is the plain CPU baseline timed next to the GPU: a row-major
 * [rows, cols] fp32 softmax with the row max shift and the lower clip of the
 * shifted logits at -64 (Sec. 1.2, Fig. 1; the max / subtract / exp / sum /
 * scale-by-reciprocal order of Sec. 2.3, Fig. 4), written as the obvious
 * three passes per row with libm expf, built with gcc -O2, no hand SIMD and
 * no threads.  Only bench.py's CPU-baseline leg calls it.
 */
#include <math.h>
#include <stdint.h>

#define CPU_BASELINE_CLIP_LO (-64.0f)

void cpu_softmax_fp32(const float* x, float* y, int64_t rows, int64_t cols)
{
    for (int64_t r = 0; r < rows; ++r) {
        const float* xr = x + r * cols;
        float* yr = y + r * cols;
        float m = -INFINITY;
        for (int64_t c = 0; c < cols; ++c)
            m = xr[c] > m ? xr[c] : m;
        float s = 0.0f;
        for (int64_t c = 0; c < cols; ++c) {
            float d = xr[c] - m;
            d = d < CPU_BASELINE_CLIP_LO ? CPU_BASELINE_CLIP_LO : d;
            float e = expf(d);
            yr[c] = e;
            s += e;
        }
        float inv = 1.0f / s;
        for (int64_t c = 0; c < cols; ++c)
            yr[c] *= inv;
    }
}
