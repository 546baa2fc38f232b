/*
 * niti.h -- C ABI of the MI355X (gfx950) NITI hot-path library, libniti.so.
 *
 * NITI ("Training Integer Neural Networks Using Integer-only Arithmetic",
 * arXiv 2009.13108) trains with int8 tensors that each carry one shared
 * int8 exponent (a block exponent, Section 3.1).  Every layer multiplies
 * int8 operands into int32 accumulators (Section 3.2), finds the effective
 * bitwidth of the largest accumulator over the whole tensor, and shifts the
 * tensor back to int8 with pseudo stochastic rounding (Algorithms 1-3).
 * Weight gradients are shifted to m_u bits and subtracted from the int8
 * weights (Section 3.3).  The loss gradient is formed in integers
 * (Section 3.5).
 *
 * Conventions shared by every entry point
 *   Memory      Every tensor pointer is a DEVICE pointer owned by the caller.
 *               The library never allocates or frees device memory.  Calls
 *               that need temporary device memory take a caller-provided
 *               workspace (ws, ws_bytes); niti_workspace_bytes() sizes it.
 *               Tensor and workspace pointers of the contraction, rounding,
 *               loss and update calls must be 16-byte aligned (hipMalloc and
 *               torch allocations are); others are rejected with
 *               NITI_ERR_ARG.
 *   Layout      Activations and errors are NHWC int8 (channels fastest),
 *               convolution weights are KRSC int8 (output channel, filter
 *               row, filter column, input channel), matrices are row-major.
 *               Exponents are int8 scalars in device memory, so a training
 *               step never waits on the host.
 *   Streams     Every call only enqueues work on `stream` (a hipStream_t,
 *               passed as void*; NULL is the default stream) and returns.
 *   Errors      Arguments are checked on the host before anything is
 *               enqueued; on error a negative niti_status is returned and
 *               no work is launched.  A failed launch returns NITI_ERR_HIP.
 *               Data-dependent conditions never fail a call: they set bits
 *               in niti_stats.flags.
 *   Stats       Calls that form a block exponent need a niti_stats block in
 *               device memory, zero-filled by the caller before its first
 *               use and kept per tensor (per layer and pass) afterwards.  It
 *               holds the result of the call and the library's working
 *               state; two calls in flight at once must not share one.
 *   Rounding    mode NITI_ROUND_PSR is Algorithm 3; NITI_ROUND_RTN rounds
 *               to nearest with ties away from zero (Section 4.3 uses it for
 *               activations and errors); NITI_ROUND_SR is the stochastic
 *               rounding Section 3.4 compares against: the magnitude
 *               x = q 2^bp + f is rounded up exactly when the top bp bits of
 *               a 64-bit draw r are below f (probability f / 2^bp), where
 *               r = SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) output
 *               number c * 2^40 + i + 1 of the stream seeded with
 *               stats.sr_seed, c = stats.calls before the call, i = the
 *               element's offset in its output tensor (NHWC activations and
 *               errors, KRSC weights, row-major matrices).  Convolution and
 *               matrix calls in this mode run on the general kernels.  A
 *               rounded magnitude that would reach 128 is held at 127, so
 *               outputs lie in [-127, 127].
 *   Speculation The library first rounds with the binary point that the
 *               same stats block reported last time (bp_hint), checks it
 *               against the true block maximum, and recomputes the output
 *               when they differ.  Results are identical either way; a
 *               miss only costs time and sets NITI_FLAG_HINT_MISS.
 */
#ifndef NITI_H
#define NITI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum niti_status {
    NITI_OK = 0,
    NITI_ERR_NULL = -1,        /* a required pointer is NULL               */
    NITI_ERR_SHAPE = -2,       /* a size is negative, zero where it must not be, or inconsistent */
    NITI_ERR_UNSUPPORTED = -3, /* valid but outside what the kernels cover, among them any
                                  operand, result or workspace part of 2^31 bytes or more
                                  (the kernels address with 32-bit offsets)            */
    NITI_ERR_WORKSPACE = -4,   /* workspace missing or smaller than needed */
    NITI_ERR_HIP = -5,         /* the HIP runtime reported an error        */
    NITI_ERR_ARG = -6          /* an enum or scalar argument is out of range */
} niti_status;

typedef enum niti_round_mode {
    NITI_ROUND_PSR = 0, /* pseudo stochastic rounding, Algorithm 3 */
    NITI_ROUND_RTN = 1, /* round to nearest, ties away from zero   */
    NITI_ROUND_SR = 2   /* stochastic rounding with a counter-based draw (Section 3.4) */
} niti_round_mode;

/* niti_stats.flags bits */
#define NITI_FLAG_ACC_BOUND 1u  /* reduction of 2^17 or more int8 products, so int32 sums may wrap (each product is
                                   at most 2^14 in magnitude); sums are kept mod 2^32 */
#define NITI_FLAG_EXP_RANGE 2u  /* an output exponent left [-128, 127] and was held at the end */
#define NITI_FLAG_LOSS_SA   4u  /* loss exponent below -54: evaluated at s_a = -54 (same int8 error) */
#define NITI_FLAG_HINT_MISS 8u  /* the speculated binary point was wrong; the output was recomputed */

/* Per-tensor statistics and working state, 128 bytes of device memory.
 * The "out" fields hold the result of the last call made with the block. */
typedef struct niti_stats {
    uint64_t max_abs;    /* out: largest magnitude over the whole result       */
    int32_t b;           /* out: effective bitwidth of max_abs (Section 3.2)   */
    int32_t bp;          /* out: binary point used, max(0, b - target)         */
    int32_t flags;       /* out: NITI_FLAG_* of this call                      */
    int32_t s_out;       /* out: output exponent formed by this call, if any   */
    int32_t bp_hint;     /* in/out: binary point tried first by the next call  */
    uint32_t calls;      /* out: calls made with this block                    */
    uint32_t misses;     /* out: calls whose first try was wrong               */
    uint32_t reserved0;
    /* Library working state.  A call accumulates its block maximum and
     * flags in slot (calls & 1) and clears the other slot for the next
     * call, so no completion counter or extra launch is needed. */
    uint64_t acc_max[2];
    uint32_t wflags[2];
    int32_t cur;         /* slot of the call in progress  */
    int32_t hint_used;   /* guess the call in progress tried */
    uint64_t sr_seed;    /* in: seed of the NITI_ROUND_SR draws (zero-filled is seed 0) */
    uint32_t sr_call;    /* draw index c of the call in progress */
    uint32_t reserved[11];
} niti_stats;

/* Convolution geometry.  Input x is NHWC [n][h][w][c]; filter is KRSC
 * [k][r][s][c]; output is NHWC [n][p][q][k] with
 * p = (h + 2 pad_h - r) / stride_h + 1 and q = (w + 2 pad_w - s) / stride_w + 1.
 * The kernels take stride_h == stride_w, at most 8 for the forward pass and
 * the weight gradient and at most 2 for the back-propagation (a strided first
 * layer, such as AlexNet's 11 x 11 stride-4 one, forms no input error in
 * Algorithm 1); other strides return NITI_ERR_UNSUPPORTED, and
 * niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, ...) is then 0. */
typedef struct niti_conv_desc {
    int64_t n, h, w, c;
    int64_t k, r, s;
    int32_t stride_h, stride_w;
    int32_t pad_h, pad_w;
} niti_conv_desc;

/* Operation ids for niti_workspace_bytes. */
#define NITI_OP_GEMM_FWD        0
#define NITI_OP_CONV_FWD        1
#define NITI_OP_CONV_BWD_DATA   2
#define NITI_OP_CONV_BWD_WEIGHT 3
#define NITI_OP_INT_CE_LOSS     4

/* Fully-connected / plain forward layer (Algorithm 1, forward loop;
 * Section 3.2).  C = round(A B^T) with A [M][K], B [N][K] and C [M][N],
 * all int8 row-major; the int32 products are optionally passed through ReLU,
 * then the block exponent is found over all of C and the tensor is shifted
 * by max(0, b - target_bits) and rounded.  *s_c = *s_a + *s_b + bp when all
 * three exponent pointers are given (all NULL otherwise).  M, N >= 1,
 * K >= 0 (A and B may be NULL when K == 0: C is then all zero),
 * target_bits in 1..31.  No workspace. */
niti_status niti_gemm_fwd(const int8_t *A, const int8_t *B, int8_t *C,
                          int64_t M, int64_t N, int64_t K,
                          const int8_t *s_a, const int8_t *s_b, int8_t *s_c,
                          int target_bits, int relu, niti_round_mode mode,
                          niti_stats *stats, void *stream);

/* Convolution forward (Algorithm 1, forward loop; Section 3.2 reduces it to
 * an implicit GEMM).  y = round(conv(x, w)), exponents as niti_gemm_fwd
 * with target 7.  Needs c % 4 == 0 (pad image channels with zeros).
 * Workspace: niti_workspace_bytes(NITI_OP_CONV_FWD, d, ...), zero for most
 * layers; layers with few channels (s*c <= 64) use it for a zero-padded
 * copy of x and for their filter rows widened to whole load windows.  Such
 * a layer reads x in place, without the copy, when the descriptor has no
 * padding and every filter window of an output row lies inside the input
 * row (for example an image stored with its zero border); the weight
 * gradient does the same. */
niti_status niti_conv_fwd(const niti_conv_desc *d, const int8_t *x, const int8_t *w,
                          int8_t *y, const int8_t *s_x, const int8_t *s_w, int8_t *s_y,
                          int relu, niti_round_mode mode, niti_stats *stats,
                          void *ws, size_t ws_bytes, void *stream);

/* Error back-propagation through a convolution (Algorithm 1,
 * e(l-1) = w(l) (x) e(l); Section 3.2): dx = round(adjoint of conv in x,
 * applied to dy) with target 7.  dy is NHWC [n][p][q][k], dx NHWC
 * [n][h][w][c].  The error exponent is not formed (Section 3.1: it cancels
 * out of the learning rule).  If relu_src (NHWC like dx, the int8 forward
 * activation of that layer) is given, dx is zeroed where relu_src <= 0
 * after rounding; the block exponent is taken before that mask.  Workspace:
 * niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, d, ...). */
niti_status niti_conv_bwd_data(const niti_conv_desc *d, const int8_t *dy, const int8_t *w,
                               int8_t *dx, const int8_t *relu_src, niti_round_mode mode,
                               niti_stats *stats, void *ws, size_t ws_bytes, void *stream);

/* niti_conv_bwd_data in two parts, for callers that take the filter
 * rearrangement off the back-propagation's critical path (Algorithm 1: the
 * filter w of layer l is fixed from its forward use until its update, so
 * it can be rearranged any time in between).  niti_conv_pack_bwd_data
 * writes the filter w (KRSC, device) rearranged per sub-pixel class into
 * packed (device, caller-owned, 16-byte aligned, at least
 * niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, d, ...) bytes); it stays
 * valid until w changes.  niti_conv_bwd_data_packed then computes what
 * niti_conv_bwd_data computes for that w, from packed and without a
 * workspace; packed_bytes is checked as above.  Same errors as
 * niti_conv_bwd_data (NITI_ERR_WORKSPACE for a short packed buffer). */
niti_status niti_conv_pack_bwd_data(const niti_conv_desc *d, const int8_t *w, void *packed,
                                    size_t packed_bytes, void *stream);
niti_status niti_conv_bwd_data_packed(const niti_conv_desc *d, const int8_t *dy,
                                      const void *packed, int8_t *dx, const int8_t *relu_src,
                                      niti_round_mode mode, niti_stats *stats,
                                      size_t packed_bytes, void *stream);

/* Weight gradient and discrete update (Algorithm 1, g(l) = a(l-1) (x) e(l)
 * then w <- w - g; Section 3.3).  g32 = sum over n, p, q of dy x x, exact
 * mod 2^32; b = B(g32); g = round(g32, max(0, b - mu)); w <- w - g held to
 * [-127, 127], in place.  mu in 1..8.  If g32_out is given it receives the
 * int32 gradient (KRSC).  Workspace:
 * niti_workspace_bytes(NITI_OP_CONV_BWD_WEIGHT, d, ...).  A fully-connected
 * layer is the case h = w = r = s = 1. */
niti_status niti_conv_bwd_weight(const niti_conv_desc *d, const int8_t *x, const int8_t *dy,
                                 int8_t *w, int32_t *g32_out, int mu, niti_round_mode mode,
                                 niti_stats *stats, void *ws, size_t ws_bytes, void *stream);

/* niti_conv_bwd_weight for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
 * the same computation and results, with the temporary memory (split
 * partial sums, the int32 gradient when g32_out is NULL, the padded input
 * copy of few-channel layers) taken from a fixed array of
 * NITI_NOALLOC_SCRATCH_BYTES inside the library instead of a workspace.
 * Each GPU that the library runs on holds its own copy of that array until
 * the process ends; the array's address on the current device is looked up
 * on the first call made on that device, so the current device must be the
 * device of `stream`.  The call allocates and frees nothing.  Calls whose
 * niti_workspace_bytes(NITI_OP_CONV_BWD_WEIGHT, d, ...) exceeds
 * NITI_NOALLOC_SCRATCH_BYTES return NITI_ERR_WORKSPACE before anything is
 * enqueued.  Every call on one GPU uses the same array: two such calls whose
 * work overlaps on one GPU (different streams, no ordering between them)
 * race and give wrong results; calls in order on one stream are safe.  No
 * part of the array needs to start at zero (every value a kernel reads from
 * it was written earlier in the same call).  Other errors as
 * niti_conv_bwd_weight. */
#define NITI_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
niti_status niti_conv_bwd_weight_noalloc(const niti_conv_desc *d, const int8_t *x, const int8_t *dy,
                                         int8_t *w, int32_t *g32_out, int mu, niti_round_mode mode,
                                         niti_stats *stats, void *stream);

/* Shift and round an int32 tensor (Algorithm 2 with Algorithm 3).  bp >= 0
 * rounds with that binary point (stats may be NULL; magnitudes are held at
 * 127); bp < 0 finds the block exponent first, bp = max(0, B(x) -
 * target_bits), which needs stats.  *s_out = *s_in + bp when both are
 * given.  n >= 0. */
niti_status niti_round_psr(const int32_t *x, int8_t *y, int64_t n, int bp, int target_bits,
                           niti_round_mode mode, const int8_t *s_in, int8_t *s_out,
                           niti_stats *stats, void *stream);

/* Integer cross-entropy gradient (Section 3.5).  logits [batch][classes]
 * int8 with exponent *s_logits; labels int32 in [0, classes).  Per sample:
 * s_a <= -7 uses t_i = 2^(1-2 s_a) + a_i 2^(1-s_a) + a_i^2 (second-order
 * Taylor series, scaled to integers and evaluated exactly in 128-bit
 * integers; below s_a = -54 the int8 result no longer depends on s_a, so
 * s_a = -54 is evaluated and NITI_FLAG_LOSS_SA is set); s_a > -7 uses
 * t_i = 1 << max(0, xhat_i - p) with xhat_i = floor(47274 a_i 2^(s_a-15))
 * and p = max(xhat) - 10.  Then e_i = t_i - [i == label] sum(t), and
 * err = round(e) with target 7 over the whole batch.  stats.b and stats.bp
 * are exact; below s_a = -22 the largest |e_i| can exceed 64 bits, and
 * stats.max_abs holds it shifted right by 2 (-22 - s_a) bits.  classes in
 * 1..65536.  Workspace (16 bytes per logit):
 * niti_workspace_bytes(NITI_OP_INT_CE_LOSS, NULL, batch, classes, 0). */
niti_status niti_int_ce_loss_grad(const int8_t *logits, const int8_t *s_logits,
                                  const int32_t *labels, int8_t *err, int64_t batch,
                                  int64_t classes, niti_round_mode mode, niti_stats *stats,
                                  void *ws, size_t ws_bytes, void *stream);

/* Discrete weight update from an int32 gradient (Section 3.3): b = B(g32),
 * g = round(g32, max(0, b - mu)), w <- w - g held to [-127, 127], in place.
 * mu in 1..8, n >= 0. */
niti_status niti_sgd_update(int8_t *w, const int32_t *g32, int64_t n, int mu,
                            niti_round_mode mode, niti_stats *stats, void *stream);

/* Bytes of workspace an operation needs (0 when none).  d is used by the
 * convolution ops, (M, N) = (batch, classes) by the loss. */
size_t niti_workspace_bytes(int op, const niti_conv_desc *d, int64_t M, int64_t N, int64_t K);

/* Human-readable name of a status code (static storage). */
const char *niti_status_str(niti_status s);

/* ---- Layer glue used by the experiments' networks (not contractions) ---- */

/* Input quantisation (Section 3): 8-bit pixels px, NCHW [n][c][h][w], become
 * int8 p >> 1 (exponent -7 for the caller to attach) in NHWC
 * [n][h][w][c_pad]; channels c..c_pad-1 are zero.  c_pad >= c. */
niti_status niti_quantize_u8(const uint8_t *px, int8_t *x, int64_t n, int64_t c, int64_t h,
                             int64_t w, int64_t c_pad, void *stream);

/* 2x2 stride-2 max pooling, NHWC, h and w even.  idx (one byte per output)
 * records the window position (0..3, row-major) of the first maximum.  The
 * exponent is unchanged. */
niti_status niti_maxpool2_fwd(const int8_t *x, int8_t *y, uint8_t *idx, int64_t n, int64_t h,
                              int64_t w, int64_t c, void *stream);

/* Backward of niti_maxpool2_fwd: dx (NHWC [n][h][w][c]) receives each dy at
 * its window's recorded position and zero elsewhere. */
niti_status niti_maxpool2_bwd(const int8_t *dy, const uint8_t *idx, int8_t *dx, int64_t n,
                              int64_t h, int64_t w, int64_t c, void *stream);

/* Backward ReLU on an int8 error: e[i] = 0 where a[i] <= 0, in place. */
niti_status niti_relu_mask(int8_t *e, const int8_t *a, int64_t n, void *stream);

/* Dropout (the VGG-small networks of Table 5 put it before their
 * classifier; the paper gives no integer form): element i of x (n int8
 * values, any layout) is kept when the top byte of draw (seed, call, i) of
 * the stochastic-rounding generator (see Rounding above) is at least
 * drop256, i.e. with probability 1 - drop256/256; y = x where kept, 0
 * elsewhere; keep[i] = 1 / 0 records the choice.  The kept values are
 * rescaled through the exponent: *s_y = *s_x + exp_add, held to
 * [-128, 127], when both are given (drop256 = 128 with exp_add = 1 is the
 * 1/(1 - p) = 2 of inverted dropout, exactly).  drop256 in 0..256, exp_add in
 * -8..8 (NITI_ERR_ARG otherwise); s_x and s_y both given or both NULL. */
niti_status niti_dropout_fwd(const int8_t *x, int8_t *y, uint8_t *keep, int64_t n, uint64_t seed,
                             uint32_t call, int drop256, const int8_t *s_x, int8_t *s_y, int exp_add,
                             void *stream);
/* Backward of niti_dropout_fwd: dx = dy where keep, 0 elsewhere. */
niti_status niti_dropout_bwd(const int8_t *dy, const uint8_t *keep, int8_t *dx, int64_t n, void *stream);

/* Size of niti_stats (128), for bindings. */
size_t niti_stats_bytes(void);

/* ---- Kernel timing (a profiling aid; no effect on results) ----
 * While enabled, calls record HIP event pairs on their own stream:
 *   NITI_TIMING_IGEMM   the implicit-GEMM kernel and its finishing launch of
 *                       every niti_gemm_fwd / niti_conv_fwd /
 *                       niti_conv_bwd_data(_packed) call;
 *   NITI_TIMING_WGRAD   the weight-gradient contraction kernel of every
 *                       niti_conv_bwd_weight call;
 *   NITI_TIMING_KERNEL  every contraction kernel launch alone (the main
 *                       implicit-GEMM or weight-gradient kernel), labelled
 *                       with the kernel and its template arguments;
 *   NITI_TIMING_SUM     the split-sum and maximum pass of a weight gradient;
 *   NITI_TIMING_UPDATE  the rounding and update pass of a weight gradient;
 *   NITI_TIMING_LOSS    the two launches of niti_int_ce_loss_grad.
 * niti_timing_enable(1) clears the record and starts, niti_timing_enable(0)
 * stops.  niti_timing_read waits for the recorded events and returns the
 * summed milliseconds and the number of records of a family;
 * niti_timing_record returns record i (in enqueue order) with its family,
 * label ("" when none; static storage) and milliseconds.  The record is
 * process-wide and not guarded against calls from several host threads at
 * once.  Return NITI_ERR_ARG for an unknown family or an index past the
 * end, NITI_ERR_HIP if an event fails. */
enum {
    NITI_TIMING_IGEMM = 0,
    NITI_TIMING_WGRAD = 1,
    NITI_TIMING_KERNEL = 2,
    NITI_TIMING_SUM = 3,
    NITI_TIMING_UPDATE = 4,
    NITI_TIMING_LOSS = 5
};
niti_status niti_timing_enable(int on);
niti_status niti_timing_read(int family, double *ms, int64_t *calls);
niti_status niti_timing_record(int64_t i, int *family, const char **name, double *ms);

/* ---- Matrix-core rate check (a measurement aid; no part of the method) ----
 * Runs `workgroups` workgroups of four waves; each wave issues iters x 8
 * int8 MFMAs (32x32x32: 65536 integer operations each) on register operands
 * in eight independent accumulator chains, then writes one int32 per lane
 * to out[workgroup * 256 + lane] (device, caller-owned, at least
 * workgroups * 256 elements).  Its rate is what int8 matrix work sustains
 * on this device with no memory traffic.  NITI_ERR_SHAPE for iters < 0 or
 * workgroups outside 1..2^20. */
niti_status niti_mfma_loop(int64_t iters, int64_t workgroups, int32_t *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* NITI_H */
