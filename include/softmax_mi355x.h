/*
 * softmax_mi355x.h -- C ABI of the MI355X (gfx950) row-softmax library.
 *
 * The operation (Sec. 1.1, Eq. (1) of "Softmax Optimizations for Intel Xeon
 * Processor-based Platforms", with the reference functor's clip of the
 * shifted logits, Sec. 1.2 Fig. 1, and the row-major [batch_size,
 * num_classes] layout of the optimised functor, Sec. 2.3 Fig. 4):
 *
 *   for every row i of x (rows x cols, fp32, row-major, leading dim = cols):
 *     M_i  = max_j x[i,j]
 *     c_ij = max(x[i,j] - M_i, SOFTMAX_CLIP_LO)      (compare-select)
 *     y[i,j] = exp(c_ij) / sum_k exp(c_ik)
 *
 * Accuracy: every output is within 4e-6 relative of the exact value of the
 * formula above (derivation: the exp argument is carried in extended
 * precision, the row sum is a fixed-depth tree).  Measured by a dense scan
 * on MI355X against float64: v_exp_f32 (2^t) is within 0.783 ulp over every
 * fp32 t in [-126, 0], and the library's clipped exponential within
 * 1.269 ulp over every fp32 x - M in [-64, 0] (stated bound 1.5 ulp; the
 * scan is tests/test_gpu_exp_scan.py).
 * Outputs are bitwise deterministic for a given input, shape and alignment.
 *
 * Non-finite inputs: a NaN or +inf anywhere in a row, or a row of all -inf,
 * gives a row of NaN; a -inf entry among finite ones clips to e^-64 / S.
 *
 * All functions are thread-safe.  Only the entry points below are exported.
 */
#ifndef SOFTMAX_MI355X_H
#define SOFTMAX_MI355X_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SOFTMAX_API __attribute__((visibility("default")))

/* Lower bound applied to the shifted logit x - rowmax before exp by
 * softmax_fwd.  The paper's reference functor clips here (Sec. 1.2 Fig. 1;
 * purpose in Sec. 2.1) without printing the constant; this library's
 * default is -64, so no output is 0 and none is denormal for any row length
 * below 2^33.  softmax_fwd_clip takes the bound as an argument. */
#define SOFTMAX_CLIP_LO (-64.0f)

/* Largest bound softmax_fwd_clip accepts.  Two parts of the kernels rely on
 * a clipped exponential being negligible next to a row sum of at least 1:
 * the padding of a row's last partial vector (under 4096 entries) and the
 * chunk-local clip inside the partial sums of rows split over several
 * workgroups (cols entries).  At -48 each adds under cols * e^-48 (below
 * 1e-10 relative for any row that fits in memory). */
#define SOFTMAX_CLIP_MAX (-48.0f)

/* Return codes. */
#define SOFTMAX_OK 0
#define SOFTMAX_ERR_INVALID_ARG 1 /* bad size, null or overlapping pointer */
#define SOFTMAX_ERR_HIP 2         /* a HIP call or launch failed */
#define SOFTMAX_ERR_NOT_DEVICE 3  /* pointer is not memory the current
                                     device can use, or the byte range runs
                                     past its allocation */

/* Kernel families reported by softmax_plan(). */
#define SOFTMAX_KERNEL_NONE 0      /* rows*cols == 0: nothing is launched */
#define SOFTMAX_KERNEL_PACKED 1    /* cols <= 256 not taken by GROUP_ROWS
                                      (log and NLL outputs: cols <= 64):
                                      several rows per wavefront */
#define SOFTMAX_KERNEL_WAVE_ROW 2  /* cols <= 4096: one wavefront per row
                                      (rows that are not whole 16-byte
                                      strips: 128-bit access in the aligned
                                      strips around the row above 2048) */
#define SOFTMAX_KERNEL_BLOCK_ROW 3 /* cols <= 16380 (NLL outputs: 32768):
                                      one workgroup per row; also
                                      probability rows of 16385 to 24575
                                      columns in whole strips when the
                                      device has between 15/16 and 3 times
                                      as many compute units as there are
                                      rows (the split grid's third chunk
                                      would be partly empty) */
#define SOFTMAX_KERNEL_SPLIT_ROW 4 /* longer rows: several workgroups per row
                                      (chunks aligned to the row's phase for
                                      rows that are not whole strips) */
#define SOFTMAX_KERNEL_GROUP_ROWS 5 /* cols <= 256 in whole 16-byte strips
                                       (cols % 4 == 0, 16-byte aligned x and
                                       y), probability outputs: G lanes per
                                       row (G the power of two >= cols / 4),
                                       several rows per wavefront.  Past
                                       about one round of the device's
                                       resident workgroups, rows that fill
                                       less than 3/4 of the G lanes take
                                       PACKED instead, and so do rows of
                                       more than 64 columns, or that fill
                                       their lanes in part, while the grid
                                       takes one to 2.5 rounds (the choice
                                       depends on rows and the device) */

/*
 * softmax_fwd -- row-wise clipped softmax, fp32 in and out.
 *
 *   x      device pointer to rows*cols fp32 values, row-major (element (i,j)
 *          at x[i*cols + j]).  Read only.
 *   y      device pointer to rows*cols fp32 values, same layout; written.
 *          y == x (in place) is allowed; any other overlap of the two byte
 *          ranges is rejected.
 *   rows   number of rows (the paper's batch_size), >= 0.
 *   cols   number of classes per row (num_classes), >= 0.
 *   stream HIP stream to enqueue on (0 = the null stream).
 *
 * Ownership: x and y are allocated and owned by the caller and must be memory
 * the current HIP device can access (hipMalloc, torch CUDA tensors, managed
 * or pinned host memory); the call checks this and the byte ranges against
 * the allocations before launching.  No alignment is required: 128-bit
 * accesses are used when x and y are 16-byte aligned (and, above 64
 * columns, cols % 4 == 0); otherwise 32-bit accesses.
 *
 * Asynchrony: work is enqueued on `stream` and the call returns without
 * waiting; y is valid once the stream has reached that point.
 *
 * Scratch: no entry point of this library allocates memory, so callers
 * that cannot allocate (code under stream capture, serving loops,
 * harnesses that forbid hipMalloc) can call any of them.  Rows longer than
 * 16380 columns (NLL outputs: 32768) are split over several workgroups
 * (except the block rows above),
 * which combine partial
 * (max, sum) pairs
 * through a table of 4096 row entries held in a static device array
 * (2,359,552 bytes per device, part of the library's code object, zero at
 * rest).  Each launch takes as many consecutive entries as it has rows,
 * from a per-device cursor on the host (launch bases advance mod 4096); the
 * workgroups of a row meet at its entry: the first to arrive claims it on
 * the device, the last to leave frees it.  So calls on any number of
 * streams, graphs replayed at the same time, and a first call made under
 * stream capture need no allocation and no synchronisation, and launches
 * in flight together use disjoint entries as long as they hold fewer than
 * 4096 split rows between them.  Beyond that (or when one graph is
 * replayed on two streams at once) a row whose entry is still held waits
 * for it; the wait is bounded, and a row that gives up is written as NaN
 * and counted (softmax_exchange_status).
 *
 * Long rows are done in one pass when a row spans at most 64 workgroups
 * (chunks of 8192 columns up to cols = 65536, then chunks of 16384 up to
 * cols = 1048576 and, with 128-bit access only, chunks of 32768 up to
 * cols = 2097152; probability rows keep 8192-column chunks up to
 * cols = 524288 when the row count makes that take fewer launches or fill
 * the device better): the
 * workgroups of a row exchange their pairs in the middle of the kernel and
 * wait for each other.  Workgroups are dispatched in ID order, so this always
 * progresses while a row's workgroups can be resident together.  Longer rows
 * take two passes (x read twice).  Every wait is bounded (20 ms of wall
 * clock): a workgroup that gives up writes NaN for its outputs instead of
 * stalling the device, and counts itself in softmax_exchange_status().
 *
 * Store schedule: in the one-pass split-row launches with 128-bit access
 * (every workgroup resident at once, one chunk each, about 8 MiB read or
 * more) the stores
 * wait until the launch's reads are expected to be done (read bytes /
 * 7.6 TB/s + 0.3 us after the workgroup starts), so HBM serves the reads
 * and the writes as two phases; softmax_plan() reports the delay, and
 * softmax_fwd_planned() can set it for any kernel.  It changes no result.
 *
 * Returns SOFTMAX_OK, or SOFTMAX_ERR_INVALID_ARG (rows or cols < 0,
 * rows*cols*4 overflows int64, x or y null while rows*cols > 0, partial
 * overlap), SOFTMAX_ERR_NOT_DEVICE, or SOFTMAX_ERR_HIP (the HIP error is
 * kept for softmax_last_hip_error()).  On any error nothing is launched
 * except for SOFTMAX_ERR_HIP from a failed launch.  rows*cols == 0 returns
 * SOFTMAX_OK without touching the GPU.
 */
SOFTMAX_API int softmax_fwd(const float* x, float* y, int64_t rows, int64_t cols,
                            hipStream_t stream);

/*
 * softmax_fwd_clip -- softmax_fwd with the clip bound as an argument:
 *
 *     y[i,j] = exp(max(x[i,j] - M_i, clip_lo)) / sum_k exp(max(x[i,k] - M_i, clip_lo))
 *
 * clip_lo = -INFINITY turns the clip off, which is the paper's optimised
 * functor (Sec. 2.3 Fig. 4; dropping the reference functor's ValueClip is
 * the first optimisation of Sec. 2.1): then a -inf entry among finite ones
 * gives exactly 0 and outputs may be denormal or 0.  Any clip_lo <=
 * SOFTMAX_CLIP_MAX is accepted; bounds below -128 give the same fp32
 * results as no clip.  softmax_fwd(...) is softmax_fwd_clip(..., -64, ...)
 * bit for bit.
 *
 * Accuracy: every output is within 4e-6 relative plus 2^-148 absolute of
 * the exact value (the absolute term only matters for outputs below 2^-126,
 * which need clip_lo < -87).  All other arguments, the layout, ownership,
 * asynchrony, scratch and error codes are those of softmax_fwd; a NaN
 * clip_lo or one above SOFTMAX_CLIP_MAX returns SOFTMAX_ERR_INVALID_ARG
 * with nothing launched.
 */
SOFTMAX_API int softmax_fwd_clip(const float* x, float* y, int64_t rows, int64_t cols,
                                 float clip_lo, hipStream_t stream);

/*
 * softmax_fwd_approx -- softmax_fwd_clip with the cheap exponential the
 * paper proposes as further work (Sec. 4: approximations that trade a little
 * accuracy for speed): each e = exp(max(x - M, clip_lo)) is the single
 * instruction v_exp_f32(RN(RN(x - M) * RN(log2 e))) in fp32 instead of the
 * extended-precision argument of softmax_fwd.
 *
 * Accuracy (the stated, looser bound): every output y with exact value
 * y* >= 2^-126 satisfies |y - y*| <= (2e-6 + 1.5e-7 * min(|x - M|, |clip_lo|)) * y*:
 * the fp32 argument carries a relative error of about 1.33e-7 that the
 * exponential turns into 1.33e-7 * |x - M|, so it grows with the distance
 * from the row max (about 1.2e-5 at the -64 clip).  Outputs whose exact
 * value is below 2^-126 (only possible with clip_lo < -87) may be flushed
 * to 0.  Arguments, layout, errors and everything else are those of
 * softmax_fwd_clip.
 */
SOFTMAX_API int softmax_fwd_approx(const float* x, float* y, int64_t rows, int64_t cols,
                                   float clip_lo, hipStream_t stream);

/*
 * softmax_log_fwd -- the logarithm of the clipped row softmax:
 *
 *     y[i,j] = c_ij - ln(sum_k exp(c_ik)),   c_ij = max(x[i,j] - M_i, clip_lo)
 *
 * the log that follows softmax in training and that the reference functor's
 * clip exists for (Sec. 2.1), computed directly so that it stays exact
 * where the probability itself would underflow.  clip_lo as for
 * softmax_fwd_clip (-INFINITY: plain log-softmax; a -inf entry then gives
 * -inf).  The row sum takes the single-instruction exponential per term
 * (its error, weighted by the softmax, stays within the bound below), ln S
 * comes from v_log_f32, and c = x - M and c - ln S are fp32 operations.
 *
 * Accuracy: |y - y*| <= 2e-6 + 2.5e-7 * (|y*| + ln(cols)) against the exact
 * value y* (the sum's rounding and the logarithm's 1 ulp on log2 S).
 * Arguments, layout, NaN rules, errors and everything else are those of
 * softmax_fwd_clip; y == x (in place) is allowed.
 */
SOFTMAX_API int softmax_log_fwd(const float* x, float* y, int64_t rows, int64_t cols,
                                float clip_lo, hipStream_t stream);

/*
 * softmax_nll_fwd -- the negative log-likelihood of one label per row under
 * the clipped softmax, fused so that no probability or log is written:
 *
 *     loss[i] = ln(sum_k exp(c_ik)) - c_{i, labels[i]},
 *     c_ij = max(x[i,j] - M_i, clip_lo)
 *
 * that is minus softmax_log_fwd's output at the label: the training loss
 * that the log after softmax feeds, and the reason the reference functor
 * clips (Sec. 2.1).
 *
 *   x       device pointer, rows x cols fp32, row-major (as softmax_fwd)
 *   labels  device pointer, rows int64 class indices
 *   loss    device pointer, rows fp32; written.  May not overlap x or
 *           labels.
 *   clip_lo as for softmax_fwd_clip (-INFINITY: plain cross-entropy; a
 *           -inf logit at the label then gives +inf).
 *
 * A label outside [0, cols) gives a NaN loss (no error: labels are device
 * data).  A NaN in the row, a +inf, or a row of all -inf gives NaN.  x is
 * read once; the call writes 4 bytes per row.  rows == 0 returns SOFTMAX_OK
 * with nothing launched; cols == 0 with rows > 0 is SOFTMAX_ERR_INVALID_ARG
 * (no row can have a valid label).
 *
 * Accuracy: |loss - loss*| <= 2e-6 + 2.5e-7 * (|loss*| + ln(cols)), as for
 * softmax_log_fwd.  Ownership, asynchrony, scratch (rows longer than
 * 32768 columns) and error codes follow softmax_fwd_clip, except that in
 * the one-pass long-row kernel a row's workgroups do not wait for each
 * other: the last to finish merges the row's partial pairs, writes the loss
 * and returns the row's exchange state to rest.  With 128-bit access
 * those rows are cut into chunks of 32768 columns (1024-thread workgroups)
 * rather than the chunks softmax_plan() reports for softmax_fwd.
 */
SOFTMAX_API int softmax_nll_fwd(const float* x, const int64_t* labels, float* loss,
                                int64_t rows, int64_t cols, float clip_lo,
                                hipStream_t stream);

/* Limits of softmax_attention_fwd. */
#define SOFTMAX_ATTN_MAX_KEYS 64     /* lk: the keys of one row fit one set of tiles */
#define SOFTMAX_ATTN_MAX_DIM 65536   /* d and dv */

/*
 * softmax_attention_fwd -- fused softmax attention over small tiles, the
 * attention of the DAM model whose softmax the paper optimises (Sec. 1;
 * softmax is 18.5% of that model's time in Sec. 1.2 Fig. 2):
 *
 *   for every batch element b:
 *     S = scale * Q_b K_b^T                       [lq, lk]
 *     P = row-wise clipped softmax of S over the keys, bound clip_lo
 *         (the operation of softmax_fwd_clip, Sec. 1.1 Eq. (1), Sec. 1.2
 *         Fig. 1; -INFINITY for no clip, Sec. 2.3 Fig. 4)
 *     O_b = P V_b                                  [lq, dv]
 *
 *   q      device pointer, batch x lq x d fp32, row-major, contiguous
 *   k      device pointer, batch x lk x d fp32
 *   v      device pointer, batch x lk x dv fp32
 *   o      device pointer, batch x lq x dv fp32; written.  o may not overlap
 *          q, k or v.
 *   batch, lq >= 0; 1 <= lk <= SOFTMAX_ATTN_MAX_KEYS (when there is work);
 *   0 <= d, dv <= SOFTMAX_ATTN_MAX_DIM.  q and k may be NULL when d == 0
 *   (every score is then 0).
 *   scale  finite fp32 multiplier of Q K^T (1/sqrt(d) for the DAM model).
 *   clip_lo as for softmax_fwd_clip.
 *
 * The scores and weights never leave the registers: the two products run
 * on the matrix cores in fp32 (v_mfma_f32_16x16x4f32) and the softmax runs
 * on their accumulators.  On the DAM tile (d = dv = 200, 49 or 50 keys) the
 * scores of the last one or two keys are fp32 fma dot products on the
 * vector ALUs instead, and the value product takes the unnormalised
 * exponentials (O is scaled by 1 / sum at the end).  Accuracy: each score carries the rounding of a
 * d-term fp32 dot product, delta_i = (d+2)*2^-24 * max_k |scale| sum_t
 * |Q_it K_kt| for query i, so each weight is within a relative
 * 2*delta_i + 4e-6 of the exact weight, and each output within
 * (2*delta_i + 4e-6 + (lk+2)*2^-24) * sum_k P_ik |V_kc| + 2^-148.
 *
 * Ownership, asynchrony and error codes follow softmax_fwd: caller-owned
 * device memory, work enqueued on `stream`, SOFTMAX_ERR_INVALID_ARG for bad
 * sizes, a non-finite scale, a bad clip_lo, null or overlapping pointers,
 * SOFTMAX_ERR_NOT_DEVICE for memory the device cannot use.  batch, lq or
 * dv of 0 returns SOFTMAX_OK with nothing launched.  No scratch.
 */
SOFTMAX_API int softmax_attention_fwd(const float* q, const float* k, const float* v,
                                      float* o, int64_t batch, int64_t lq, int64_t lk,
                                      int64_t d, int64_t dv, float scale, float clip_lo,
                                      hipStream_t stream);

/* Static description of a return code.  Never NULL. */
SOFTMAX_API const char* softmax_strerror(int code);

/* hipError_t of the last SOFTMAX_ERR_HIP returned on this thread (0 if none). */
SOFTMAX_API int softmax_last_hip_error(void);

/* What softmax_fwd would launch for these arguments.  Host only: no HIP call,
 * no launch; x and y are only inspected for alignment and overlap. */
typedef struct softmax_plan_t {
  int32_t kernel;          /* SOFTMAX_KERNEL_* */
  int32_t vec_width;       /* 4: 128-bit loads and stores; 1: 32-bit */
  int32_t lanes_per_row;   /* lanes that share one row (or one chunk) */
  int32_t elems_per_lane;  /* elements each lane holds per row or chunk */
  int32_t block_threads;   /* threads per workgroup */
  int32_t launches;        /* kernel launches per call */
  int64_t chunks_per_row;  /* workgroups per row (split rows), else 1 */
  int64_t grid;            /* workgroups in each launch */
  int64_t workspace_bytes; /* bytes of the static exchange table (split rows), else 0 */
  int64_t store_delay_ns;  /* stores wait this long after a workgroup starts (0: none),
                              in the first launch; the library's schedule gives a
                              shorter last launch a delay for its own reads;
                              softmax_fwd_planned: -1 asks for the library's choice */
} softmax_plan_t;

/* The shape fields (kernel, vec_width, lanes_per_row, elems_per_lane,
 * block_threads, chunks_per_row) depend only on the arguments, except that
 * rows of at most 256 columns choose between GROUP_ROWS and PACKED, long
 * rows their chunk size, and rows of 16385 to 24575 columns between
 * BLOCK_ROW and SPLIT_ROW, by the device's resident workgroups or compute
 * units too;
 * grid, launches and store_delay_ns are those for the current device, and
 * 0 when no device is present (then the shape is the choice made from the
 * arguments alone).  No launch, no allocation (the first call on a device
 * queries its attributes). */
SOFTMAX_API int softmax_plan(const float* x, const float* y, int64_t rows, int64_t cols,
                             softmax_plan_t* plan);

/*
 * softmax_fwd_planned -- softmax_fwd with a caller-chosen kernel, for tuning
 * and for measuring the dispatch (the paper picks code per shape, Sec. 2.5;
 * this library picks one of its compiled instances by cols).  Fields read
 * from *plan:
 *   kernel          SOFTMAX_KERNEL_GROUP_ROWS (cols <= 256, cols % 4 == 0,
 *                   vec_width 4), _PACKED (cols <= 256), _WAVE_ROW (cols <=
 *                   4096, 2048 with 32-bit access), _BLOCK_ROW (cols <=
 *                   32768) or _SPLIT_ROW (any cols);
 *   vec_width       4 (needs 16-byte aligned x and y and, above 256
 *                   columns, cols % 4 == 0, except the row-phase shapes
 *                   the library itself picks for rows that are not whole
 *                   strips: wave or block rows of 2049 to 8189 columns,
 *                   split rows whose phase adds no chunk) or 1;
 *   block_threads, elems_per_lane   split rows only: 256 x 32 (chunks of
 *                   8192 columns), 512 x 32 (16384) or, with vec_width 4,
 *                   512 x 64 (32768); rows of more than 64 chunks take the
 *                   two-pass kernels, which only exist as 512 x 32;
 *   store_delay_ns  -1 for the library's store schedule, 0 for none, or a
 *                   delay up to 200000 (then the same for every launch).
 * The other fields are ignored.  The result is the same as softmax_fwd's to
 * within the accuracy bound (the summation order follows the kernel).
 * Returns SOFTMAX_ERR_INVALID_ARG, with nothing launched, for a plan the
 * library cannot run on these arguments; otherwise as softmax_fwd.
 */
SOFTMAX_API int softmax_fwd_planned(const float* x, float* y, int64_t rows, int64_t cols,
                                    const softmax_plan_t* plan, hipStream_t stream);

/*
 * softmax_exchange_status -- diagnostic, for the current device: how many
 * times a workgroup gave up waiting for its row's exchange entry (held by
 * another row too long) and for its row's partial pairs, since the library
 * was loaded, and how many of the 4096 entries are held right now (0
 * whenever no split-row work is running and none gave up).  Any of the
 * pointers may be NULL.  Synchronous (hipMemcpy); not for use under stream
 * capture.
 */
SOFTMAX_API int softmax_exchange_status(uint64_t* join_give_ups, uint64_t* wait_give_ups,
                                        int32_t* entries_in_use);

/*
 * softmax_exp_probe -- diagnostic: e[i] = exp(max(x[i] - m[i], clip_lo))
 * for 0 <= i < n, through the same device routine the softmax kernels use
 * for the clipped exp (Sec. 1.2 Fig. 1, the ValueClip then exp), with the
 * clip_lo rules of softmax_fwd_clip: the routine of softmax_fwd_clip when
 * approx == 0, that of softmax_fwd_approx when approx == 1.  approx == 2
 * gives e[i] = 2^x[i] from the bare v_exp_f32 instruction both routines
 * build on (m and clip_lo are then unused; m may be NULL).  x, m, e are
 * device fp32 arrays of n elements owned by the caller (e must not overlap
 * x or m).  Same error rules as softmax_fwd_clip; approx outside 0..2 is
 * SOFTMAX_ERR_INVALID_ARG.
 */
SOFTMAX_API int softmax_exp_probe(const float* x, const float* m, float* e, int64_t n,
                                  float clip_lo, int approx, hipStream_t stream);

/*
 * softmax_copy_probe -- diagnostic: y[i] = x[i] for 0 <= i < n with 128-bit
 * accesses when both are 16-byte aligned.  The memory-bound ceiling for the
 * same bytes softmax moves (the paper's memcpy comparison, Sec. 2.6).
 * x and y are caller-owned device arrays; y == x (each element read, then
 * written back, by the same thread: the traffic of an in-place softmax
 * with no arithmetic) is allowed, any other overlap is rejected.
 */
SOFTMAX_API int softmax_copy_probe(const float* x, float* y, int64_t n, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SOFTMAX_MI355X_H */
