// Internal launch interfaces between the C ABI (niti_api.hip) and the
// kernels.  Nothing here is exported.
#pragma once

#include "niti_device.h"

namespace niti {

constexpr int kMaxProblems = 4;   // sub-pixel classes of a stride-2 back-propagation
constexpr int kMaxDgradStride = 2;  // back-propagation: stride^2 classes <= kMaxProblems
constexpr int kMaxConvStride = 8;   // forward and weight gradient
constexpr int kFixupGrid = 256;   // workgroups of the fix-up launch (one per compute unit)

// One implicit-GEMM problem (see igemm.hip for the index form).
struct IgemmProblem {
    const int8_t* act;   // NHWC activation operand [img][H][W][C]
    const int8_t* wgt;   // weight operand [Nout][R][L]
    int8_t* out;         // NHWC output tensor base
    const int8_t* mask;  // backward ReLU source, addressed like out (or NULL)
    int32_t M;           // output pixels of this problem: img * OHc * OWc
    int32_t Nout;        // output channels
    int32_t R, S, L, Lpad, Ktot;  // taps: R rows of S pixels; L = S*C bytes per tap row
    int32_t H, W, C;     // activation geometry
    int32_t OHc, OWc;    // this problem's output grid
    int32_t st, off_h, off_w;  // input row = out row * st + off (+ tap)
    int32_t OH, OW, ldo;       // output tensor rows, columns, channel stride
    int32_t os, oa, ob;        // out row = grid row * os + oa (cols: ob)
    int32_t tiles_m, tiles_n, tile_base;
    FastDiv div_ohw, div_ow;
    int64_t act_bytes;   // extent of act (bytes), for buffer bounds
    int64_t wgt_bytes;   // extent of wgt (bytes)
    int32_t win;         // act is a zero-padded image read in filter-row windows of L bytes
    // Stride-2 class (0, 0) whose three sibling classes have no filter taps:
    // with each stored piece the kernels also write zeros at the same
    // channels of pixel (oh, ow + 1) (bit 0), (oh + 1, ow) (bit 1) and
    // (oh + 1, ow + 1) (bit 2), inside the output tensor.
    int32_t zsib;
};

// Which zero siblings of output pixel (oh, ow) lie inside the tensor
// (bits as in IgemmProblem::zsib).
__device__ __forceinline__ uint32_t zero_siblings(const IgemmProblem& P, int oh, int ow) {
    const uint32_t c = ow + 1 < P.OW ? 1u : 0u, r = oh + 1 < P.OH ? 1u : 0u;
    return (uint32_t)P.zsib & (c | (r << 1) | ((r & c) << 2));
}
// Zeros over nv bytes at dst.
__device__ __forceinline__ void store_zero_bytes(int8_t* dst, int nv) {
    if (nv == 16 && (((uintptr_t)dst) & 15) == 0) {
        *(uint4*)dst = make_uint4(0, 0, 0, 0);
    } else if (nv == 4 && (((uintptr_t)dst) & 3) == 0) {
        *(uint32_t*)dst = 0u;
    } else {
        for (int e = 0; e < nv; e++) dst[e] = 0;
    }
}
// Zeros at the siblings in bits of the piece at output offset off.
__device__ __forceinline__ void store_zero_siblings(const IgemmProblem& P, int64_t off, uint32_t bits, int nv) {
    const int64_t row = (int64_t)P.OW * P.ldo;
    if (bits & 1u) store_zero_bytes(P.out + off + P.ldo, nv);
    if (bits & 2u) store_zero_bytes(P.out + off + row, nv);
    if (bits & 4u) store_zero_bytes(P.out + off + row + P.ldo, nv);
}

struct IgemmBatch {
    IgemmProblem p[kMaxProblems];
    int32_t nprob;
    int32_t total_tiles;
};

struct IgemmCtl {
    niti_stats* stats;
    ExpArgs ex;
    int32_t target;
    int32_t relu;
    int32_t mode;
    uint32_t static_flags;
};

hipError_t igemm_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream);
// Kernel timing hooks (timing.hip): begin returns a record index, or -1 when
// timing is off; end closes that record on the same stream.  name labels a
// NITI_TIMING_KERNEL record (a string that lives as long as the process:
// kernel_label() makes one from a format, once per distinct text).
int timing_begin(int family, hipStream_t s, const char* name = nullptr);
void timing_end(int idx, hipStream_t s);
bool timing_on();
const char* kernel_label(const char* fmt, ...);
// Few outputs, long reduction (igemm_small.hip): a single plain matrix
// product of at most 1024 rows.
bool igemm_small_eligible(const IgemmBatch& b);
hipError_t igemm_small_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream);
bool igemm_dma_eligible(const IgemmBatch& b);
hipError_t igemm_dma_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream);
// Weight operand resident in LDS (igemm_wres.hip): one problem, at most 128
// output channels, a short reduction.
bool igemm_wres_eligible(const IgemmBatch& b);
hipError_t igemm_wres_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream);

// Weight-gradient contraction.  The pixel reduction is split into `splits`
// ranges; split z stores its partial sums to part + z*K*ncol (with one split
// that is the final g32).
struct WgradProblem {
    const int8_t* x;   // NHWC [img][H][W][C]
    const int8_t* dy;  // NHWC [img][P][Q][K]
    int32_t* part;     // [splits][K][R*S*C]
    int32_t H, W, C, K, R, S, P, Q;
    int32_t sh, sw, ph, pw;
    int32_t L, ncol;   // L = S*C, ncol = R*L
    int32_t npix;      // img*P*Q
    int32_t chunk;     // pixels per split (multiple of 64)
    FastDiv div_pq, div_q, div_l, div_c;
    int64_t x_bytes, dy_bytes;  // extents, for buffer bounds
    int32_t win;       // x is a zero-padded image read in filter-row windows of Lw bytes
    int32_t Lw, ncol_w;         // window bytes per filter row, R*Lw
};

struct WgradPlan {
    int32_t tbk;     // output-channel tile
    int32_t splits;  // pixel ranges
    int32_t chunk;   // pixels per range
};

// groups: workgroups to aim for (256: one per CU for the general kernel;
// the DMA kernel keeps three per CU busy).
WgradPlan wgrad_plan(int64_t K, int64_t ncol, int64_t npix, int64_t groups);
hipError_t wgrad_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream);
bool wgrad_dma_eligible(const WgradProblem& p);
hipError_t wgrad_dma_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream);
// 3x3 filters, C and K multiples of 64: all nine taps of a channel chunk per
// workgroup (wgrad_tap.hip).
bool wgrad_tap_eligible(const WgradProblem& p);
WgradPlan wgrad_tap_plan(int64_t K, int64_t C, int64_t npix);
hipError_t wgrad_tap_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream);

// Elementwise / reduction passes.
hipError_t fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t max_abs_i32(const int32_t* x, int64_t n, niti_stats* st, hipStream_t s);
// Round with a fixed bp (stats may be NULL) or with the block bp derived
// from stats->acc_max (bp < 0), finalizing stats in the latter case.
hipError_t round_i32_run(const int32_t* x, int8_t* y, int64_t n, int bp, int target, int mode,
                         niti_stats* st, ExpArgs ex, hipStream_t s);
hipError_t reduce_max_run(const int32_t* part, int splits, int32_t* g32, int64_t n, niti_stats* st,
                          hipStream_t s);
hipError_t update_run(int8_t* w, const int32_t* g32, int64_t n, int mu, int mode, niti_stats* st,
                      uint32_t static_flags, hipStream_t s);
// ws: 16 bytes per logit (the 128-bit pre-rounding values).
hipError_t loss_run(const int8_t* logits, const int8_t* s_logits, const int32_t* labels,
                    int8_t* err, void* ws, int64_t batch, int64_t classes, int mode,
                    niti_stats* st, hipStream_t s);
// Back-propagation filters: wc[class][c][t][u][k] = w[k][r(t)][s(u)][c].
struct DgradClass {
    int32_t r0, s0, T, U;  // first tap and tap counts of the class
    int64_t offset;        // byte offset of this class's filter in the packed buffer
};
hipError_t repack_dgrad_run(const int8_t* w, int8_t* out, const DgradClass* cls, int ncls,
                            int K, int R, int S, int C, int sh, int sw, hipStream_t s);
hipError_t quantize_run(const uint8_t* px, int8_t* x, int64_t n, int64_t c, int64_t h, int64_t w,
                        int64_t cp, hipStream_t s);
hipError_t maxpool_fwd_run(const int8_t* x, int8_t* y, uint8_t* idx, int64_t n, int64_t h,
                           int64_t w, int64_t c, hipStream_t s);
hipError_t maxpool_bwd_run(const int8_t* dy, const uint8_t* idx, int8_t* dx, int64_t n, int64_t h,
                           int64_t w, int64_t c, hipStream_t s);
hipError_t relu_mask_run(int8_t* e, const int8_t* a, int64_t n, hipStream_t s);
hipError_t dropout_fwd_run(const int8_t* x, int8_t* y, uint8_t* keep, int64_t n, uint64_t seed, uint32_t call,
                           uint32_t drop256, const int8_t* s_x, int8_t* s_y, int exp_add, hipStream_t s);
hipError_t dropout_bwd_run(const int8_t* dy, const uint8_t* keep, int8_t* dx, int64_t n, hipStream_t s);
// Zero the pixels of out (NHWC, c % 4 == 0) whose sub-pixel class
// (y % st, x % st) has bit (y % st) * st + x % st set in mask.
hipError_t zero_classes_run(int8_t* out, int64_t n, int64_t h, int64_t w, int64_t c, int st, uint32_t mask,
                            hipStream_t s);
// Zero-padded copy of an NHWC image (C % 4 == 0): xp[n][Hp][Wp][C] with the
// input at rows ph.., columns pw..; everything else zero.
hipError_t pad_image_run(const int8_t* x, int8_t* xp, int64_t n, int64_t h, int64_t w, int64_t c, int64_t hp,
                         int64_t wp, int64_t ph, int64_t pw, hipStream_t s);
// Filter rows as zero-extended windows: wr[k][t], t < ktot: row t / lw, byte
// t % lw of w[k][row][S*C] (zero past S*C and past R rows).
// Padded image copy and window filter repack of a few-channel convolution in
// one launch.
hipError_t pad_repack_run(const int8_t* x, int8_t* xp, int64_t n, int64_t h, int64_t w, int64_t c, int64_t hp,
                          int64_t wp, int64_t ph, int64_t pw, const int8_t* wt, int8_t* wr, int64_t k, int64_t r,
                          int64_t sc, int64_t lw, int64_t ktot, hipStream_t s);

}  // namespace niti
