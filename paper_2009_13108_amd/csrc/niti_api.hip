// C ABI of libniti.so (declared in include/niti.h): argument checks on the
// host, problem set-up, and kernel launches.  Nothing here allocates device
// memory or waits on the device.
#include <limits.h>

#include <mutex>

#include "niti_internal.h"

// Temporary memory of niti_conv_bwd_weight_noalloc: one fixed array per GPU
// (each device that loads this library holds its own copy until the process
// ends).  In host code this name is only a handle for the runtime; the array's
// device address is resolved per device with hipGetSymbolAddress below and
// only that address is passed to kernels.
static __device__ __align__(256) uint8_t scratch[NITI_NOALLOC_SCRATCH_BYTES];

using namespace niti;

namespace {

constexpr int64_t kMaxBytes = (int64_t)1 << 31;  // 32-bit offsets inside kernels
// Reductions of at least this many int8 products may leave the int32 range
// (each product is at most 2^14 in magnitude); shorter ones cannot.
constexpr int64_t kAccBoundLen = (int64_t)1 << 17;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

inline bool too_big(int64_t a) { return a < 0 || a >= kMaxBytes; }
// Tensor and workspace pointers are read with 16-byte vector and buffer loads.
inline bool mis16(const void* p) { return ((uintptr_t)p & 15) != 0; }

inline hipStream_t as_stream(void* s) { return (hipStream_t)s; }

inline niti_status hip_status(hipError_t e) { return e == hipSuccess ? NITI_OK : NITI_ERR_HIP; }

inline uint32_t acc_flags(int64_t red_len) { return red_len >= kAccBoundLen ? NITI_FLAG_ACC_BOUND : 0u; }

bool valid_mode(niti_round_mode m) { return m == NITI_ROUND_PSR || m == NITI_ROUND_RTN || m == NITI_ROUND_SR; }

// Geometry checks shared by the three convolution passes.
niti_status check_conv(const niti_conv_desc* d, int64_t* P, int64_t* Q) {
    if (!d) return NITI_ERR_NULL;
    if (d->n < 1 || d->h < 1 || d->w < 1 || d->c < 1 || d->k < 1 || d->r < 1 || d->s < 1)
        return NITI_ERR_SHAPE;
    if (d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0) return NITI_ERR_SHAPE;
    const int64_t p = (d->h + 2 * (int64_t)d->pad_h - d->r);
    const int64_t q = (d->w + 2 * (int64_t)d->pad_w - d->s);
    if (p < 0 || q < 0) return NITI_ERR_SHAPE;
    *P = p / d->stride_h + 1;
    *Q = q / d->stride_w + 1;
    if (d->c % 4 != 0) return NITI_ERR_UNSUPPORTED;
    if (d->stride_h != d->stride_w || d->stride_h > kMaxConvStride) return NITI_ERR_UNSUPPORTED;
    if (too_big(d->n * d->h * d->w * d->c) || too_big(d->n * *P * *Q * d->k) ||
        too_big(d->k * d->r * d->s * d->c) || too_big(d->k * d->r * d->s * d->c * 4))
        return NITI_ERR_UNSUPPORTED;
    return NITI_OK;
}

// Layers with few channels (S*C <= 64, C % 64 != 0) read a zero-padded copy
// of their input in filter-row windows of lw bytes (igemm_dma.hip, wgrad_dma.hip).
// An input without padding whose rows already reach the last window (an
// image stored with its zero border) is read in place: no copy.
struct WinPlan {
    bool on;
    bool in_place;
    int64_t hp, wp, lw, ktot;
    int64_t xpad_bytes, wr_bytes;  // workspace pieces, 256-byte rounded (xpad_bytes 0 in place)
};

WinPlan win_plan(const niti_conv_desc* d, int64_t P, int64_t Q) {
    WinPlan w{};
    const int64_t sc = d->s * d->c;
    if (d->c % 64 == 0 || d->c % 4 != 0 || sc > 64) return w;
    w.lw = sc <= 16 ? 16 : (sc <= 32 ? 32 : 64);
    w.hp = d->h + 2 * (int64_t)d->pad_h;
    const int64_t need_w = (Q - 1) * d->stride_w + (w.lw + d->c - 1) / d->c;  // last window in its row
    w.wp = d->w + 2 * (int64_t)d->pad_w;
    if (need_w > w.wp) w.wp = need_w;
    w.ktot = round_up(d->r * w.lw, 64);
    const int64_t xb = d->n * w.hp * w.wp * d->c;
    if (too_big(xb) || too_big(d->k * w.ktot)) return w;
    (void)P;
    w.in_place = d->pad_h == 0 && d->pad_w == 0 && w.hp == d->h && w.wp == d->w;
    w.xpad_bytes = w.in_place ? 0 : round_up(xb, 256);
    w.wr_bytes = round_up(d->k * w.ktot, 256);
    w.on = true;
    return w;
}

void set_out_grid(IgemmProblem& p, int64_t n, int64_t ohc, int64_t owc) {
    p.OHc = (int32_t)ohc;
    p.OWc = (int32_t)owc;
    p.M = (int32_t)(n * ohc * owc);
    p.div_ohw = make_fastdiv((uint32_t)(ohc * owc));
    p.div_ow = make_fastdiv((uint32_t)owc);
}

}  // namespace

extern "C" {

size_t niti_stats_bytes(void) { return sizeof(niti_stats); }

const char* niti_status_str(niti_status s) {
    switch (s) {
        case NITI_OK: return "ok";
        case NITI_ERR_NULL: return "required pointer is NULL";
        case NITI_ERR_SHAPE: return "invalid or inconsistent sizes";
        case NITI_ERR_UNSUPPORTED: return "shape or layout not supported by the kernels";
        case NITI_ERR_WORKSPACE: return "workspace missing or too small";
        case NITI_ERR_HIP: return "HIP runtime error";
        case NITI_ERR_ARG: return "argument out of range";
    }
    return "unknown status";
}

// Weight-gradient problem for a checked descriptor; shared by the workspace
// query and the entry point so that both take the same decisions.
struct WgradSetup {
    WgradProblem p;
    WinPlan wp;
    bool win;
    bool tap;  // the nine-tap kernel
    WgradPlan plan;
};

WgradSetup wgrad_setup(const niti_conv_desc* d, int64_t P, int64_t Q) {
    WgradSetup r{};
    WgradProblem& p = r.p;
    const int64_t npix = d->n * P * Q;
    p.K = (int32_t)d->k;
    p.R = (int32_t)d->r;
    p.S = (int32_t)d->s;
    p.C = (int32_t)d->c;
    p.P = (int32_t)P;
    p.Q = (int32_t)Q;
    p.sh = d->stride_h;
    p.sw = d->stride_w;
    p.L = p.S * p.C;
    p.ncol = p.R * p.L;
    p.npix = (int32_t)npix;
    p.div_pq = make_fastdiv((uint32_t)(P * Q));
    p.div_q = make_fastdiv((uint32_t)Q);
    p.div_l = make_fastdiv((uint32_t)p.L);
    p.div_c = make_fastdiv((uint32_t)p.C);
    p.dy_bytes = npix * d->k;
    // Window mode (few channels): a zero-padded copy of x, read in filter-row windows.
    r.wp = win_plan(d, P, Q);
    if (r.wp.on) {
        p.H = (int32_t)r.wp.hp;
        p.W = (int32_t)r.wp.wp;
        p.ph = 0;
        p.pw = 0;
        p.x_bytes = d->n * r.wp.hp * r.wp.wp * d->c;
        p.win = 1;
        p.Lw = (int32_t)r.wp.lw;
        p.ncol_w = p.R * p.Lw;
        r.win = wgrad_dma_eligible(p);
    }
    if (!r.win) {
        p.H = (int32_t)d->h;
        p.W = (int32_t)d->w;
        p.ph = d->pad_h;
        p.pw = d->pad_w;
        p.x_bytes = d->n * d->h * d->w * d->c;
        p.win = 0;
        p.Lw = 0;
        p.ncol_w = 0;
    }
    r.tap = !r.win && wgrad_tap_eligible(p);
    r.plan = r.tap ? wgrad_tap_plan(d->k, d->c, npix)
                   : wgrad_plan(d->k, r.win ? p.ncol_w : p.ncol, npix, wgrad_dma_eligible(p) ? 768 : 256);
    return r;
}

size_t niti_workspace_bytes(int op, const niti_conv_desc* d, int64_t M, int64_t N, int64_t K) {
    (void)K;
    int64_t P = 0, Q = 0;
    if ((op == NITI_OP_CONV_FWD || op == NITI_OP_CONV_BWD_DATA || op == NITI_OP_CONV_BWD_WEIGHT) &&
        (!d || check_conv(d, &P, &Q) != NITI_OK))
        return 0;
    switch (op) {
        case NITI_OP_CONV_FWD: {
            const WinPlan w = win_plan(d, P, Q);
            return w.on ? (size_t)(w.xpad_bytes + w.wr_bytes) : 0;
        }
        case NITI_OP_CONV_BWD_DATA:
            if (d->stride_h > kMaxDgradStride) return 0;
            return (size_t)round_up(d->k * d->r * d->s * d->c, 256);
        case NITI_OP_CONV_BWD_WEIGHT: {
            const int64_t nw = d->k * d->r * d->s * d->c;
            const WgradSetup w = wgrad_setup(d, P, Q);
            return (size_t)(round_up(nw * 4, 256) +
                            (w.plan.splits > 1 ? round_up((int64_t)w.plan.splits * nw * 4, 256) : 0) +
                            (w.win ? w.wp.xpad_bytes : 0));
        }
        case NITI_OP_INT_CE_LOSS:
            return (M > 0 && N > 0) ? (size_t)round_up(M * N * 16, 256) : 0;
        default:
            return 0;
    }
}

niti_status niti_gemm_fwd(const int8_t* A, const int8_t* B, int8_t* C, int64_t M, int64_t N, int64_t K,
                          const int8_t* s_a, const int8_t* s_b, int8_t* s_c, int target_bits, int relu,
                          niti_round_mode mode, niti_stats* stats, void* stream) {
    if (!C || !stats) return NITI_ERR_NULL;
    if (M < 1 || N < 1 || K < 0) return NITI_ERR_SHAPE;
    if ((!A || !B) && K > 0) return NITI_ERR_NULL;
    if (mis16(A) || mis16(B) || mis16(C)) return NITI_ERR_ARG;
    if (target_bits < 1 || target_bits > 31 || !valid_mode(mode)) return NITI_ERR_ARG;
    const int nexp = (s_a != nullptr) + (s_b != nullptr) + (s_c != nullptr);
    if (nexp != 0 && nexp != 3) return NITI_ERR_NULL;
    if (too_big(M * K) || too_big(N * K) || too_big(M * N) || too_big(round_up(K, 16)))
        return NITI_ERR_UNSUPPORTED;
    IgemmBatch b{};
    b.nprob = 1;
    IgemmProblem& p = b.p[0];
    p.act = A;
    p.wgt = B;
    p.out = C;
    p.mask = nullptr;
    p.Nout = (int32_t)N;
    p.R = 1;
    p.S = 1;
    p.L = (int32_t)K;
    p.Lpad = (int32_t)round_up(K, 16);
    p.Ktot = p.Lpad;
    p.H = 1;
    p.W = 1;
    p.C = (int32_t)K;
    p.st = 1;
    p.off_h = 0;
    p.off_w = 0;
    set_out_grid(p, M, 1, 1);
    p.OH = 1;
    p.OW = 1;
    p.ldo = (int32_t)N;
    p.os = 1;
    p.oa = 0;
    p.ob = 0;
    p.act_bytes = M * K;
    p.wgt_bytes = N * K;
    IgemmCtl ctl{};
    ctl.stats = stats;
    ctl.ex = ExpArgs{s_a, s_b, s_c};
    ctl.target = target_bits;
    ctl.relu = relu ? 1 : 0;
    ctl.mode = mode;
    ctl.static_flags = acc_flags(K);
    return hip_status(igemm_run(b, ctl, as_stream(stream)));
}

niti_status niti_conv_fwd(const niti_conv_desc* d, const int8_t* x, const int8_t* w, int8_t* y,
                          const int8_t* s_x, const int8_t* s_w, int8_t* s_y, int relu, niti_round_mode mode,
                          niti_stats* stats, void* ws, size_t ws_bytes, void* stream) {
    int64_t P, Q;
    if (!d) return NITI_ERR_NULL;
    if (!x || !w || !y || !stats) return NITI_ERR_NULL;
    if (mis16(x) || mis16(w) || mis16(y) || mis16(ws)) return NITI_ERR_ARG;
    const int nexp = (s_x != nullptr) + (s_w != nullptr) + (s_y != nullptr);
    if (nexp != 0 && nexp != 3) return NITI_ERR_NULL;
    if (!valid_mode(mode)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, &P, &Q);
    if (s != NITI_OK) return s;
    const size_t need = niti_workspace_bytes(NITI_OP_CONV_FWD, d, 0, 0, 0);
    if (need > 0 && (!ws || ws_bytes < need)) return NITI_ERR_WORKSPACE;
    hipStream_t strm = as_stream(stream);
    IgemmCtl ctl{};
    ctl.stats = stats;
    ctl.ex = ExpArgs{s_x, s_w, s_y};
    ctl.target = 7;
    ctl.relu = relu ? 1 : 0;
    ctl.mode = mode;
    ctl.static_flags = acc_flags(d->r * d->s * d->c);

    IgemmBatch b{};
    b.nprob = 1;
    IgemmProblem& p = b.p[0];
    p.out = y;
    p.mask = nullptr;
    p.Nout = (int32_t)d->k;
    p.R = (int32_t)d->r;
    p.S = (int32_t)d->s;
    p.C = (int32_t)d->c;
    p.st = d->stride_h;
    set_out_grid(p, d->n, P, Q);
    p.OH = (int32_t)P;
    p.OW = (int32_t)Q;
    p.ldo = (int32_t)d->k;
    p.os = 1;
    p.oa = 0;
    p.ob = 0;

    const WinPlan wp = win_plan(d, P, Q);
    if (wp.on && mode != NITI_ROUND_SR) {
        // zero-padded input (unless read in place) and window-extended filter
        // rows in the workspace
        int8_t* xpad = wp.in_place ? nullptr : (int8_t*)ws;
        int8_t* wr = (int8_t*)ws + wp.xpad_bytes;
        p.act = wp.in_place ? x : xpad;
        p.wgt = wr;
        p.H = (int32_t)wp.hp;
        p.W = (int32_t)wp.wp;
        p.off_h = 0;
        p.off_w = 0;
        p.L = (int32_t)wp.lw;
        p.Lpad = p.L;
        p.Ktot = (int32_t)wp.ktot;
        p.act_bytes = d->n * wp.hp * wp.wp * d->c;
        p.wgt_bytes = d->k * wp.ktot;
        p.win = 1;
        if (igemm_dma_eligible(b)) {
            hipError_t e = pad_repack_run(x, xpad, wp.in_place ? 0 : d->n, d->h, d->w, d->c, wp.hp, wp.wp, d->pad_h,
                                          d->pad_w, w, wr, d->k, d->r, d->s * d->c, wp.lw, wp.ktot, strm);
            if (e != hipSuccess) return NITI_ERR_HIP;
            return hip_status(igemm_run(b, ctl, strm));
        }
    }
    p.act = x;
    p.wgt = w;
    p.H = (int32_t)d->h;
    p.W = (int32_t)d->w;
    p.off_h = -d->pad_h;
    p.off_w = -d->pad_w;
    p.L = (int32_t)(d->s * d->c);
    p.Lpad = (int32_t)round_up(p.L, 16);
    p.Ktot = p.R * p.Lpad;
    p.act_bytes = d->n * d->h * d->w * d->c;
    p.wgt_bytes = d->k * d->r * d->s * d->c;
    p.win = 0;
    return hip_status(igemm_run(b, ctl, strm));
}

namespace {

// The sub-pixel classes of a back-propagation (Algorithm 1's e(l-1) = w (x)
// e(l) over a strided filter: one implicit-GEMM problem per class of output
// pixels that sees the same filter taps) over the class filters packed at
// `packed`.
struct DgradPlan {
    DgradClass cls[kMaxProblems];
    int ncls = 0;
    IgemmBatch b{};
    uint32_t zero_mask = 0;  // classes without taps: exact zeros, written apart
    int8_t* dx = nullptr;
};

void plan_dgrad(const niti_conv_desc* d, int64_t P, int64_t Q, const int8_t* dy, const int8_t* packed, int8_t* dx,
                const int8_t* relu_src, DgradPlan& pl) {
    const int st = d->stride_h;
    const int K = (int)d->k, R = (int)d->r, S = (int)d->s, C = (int)d->c;
    DgradClass* cls = pl.cls;
    IgemmBatch& b = pl.b;
    int& ncls = pl.ncls;
    uint32_t& zero_mask = pl.zero_mask;
    pl.dx = dx;
    int64_t off = 0;
    for (int a = 0; a < st; a++) {
        for (int bb = 0; bb < st; bb++) {
            DgradClass& c = cls[ncls];
            c.r0 = (a + d->pad_h) % st;
            c.s0 = (bb + d->pad_w) % st;
            c.T = c.r0 < R ? (R - c.r0 + st - 1) / st : 0;
            c.U = c.s0 < S ? (S - c.s0 + st - 1) / st : 0;
            c.offset = off;
            off += (int64_t)C * c.T * c.U * K;
            const int64_t hc = a < d->h ? (d->h - a + st - 1) / st : 0;
            const int64_t wc = bb < d->w ? (d->w - bb + st - 1) / st : 0;
            ncls++;
            if (hc == 0 || wc == 0) continue;
            if (c.T == 0 || c.U == 0) {
                zero_mask |= 1u << (a * st + bb);
                continue;
            }
            IgemmProblem& p = b.p[b.nprob++];
            const int da = (a + d->pad_h - c.r0) / st;
            const int db = (bb + d->pad_w - c.s0) / st;
            p.act = dy;
            p.wgt = packed + c.offset;
            p.out = dx;
            p.mask = relu_src;
            p.Nout = C;
            p.R = c.T;
            p.S = c.U;
            p.L = c.U * K;
            p.Lpad = (int32_t)round_up(p.L, 16);
            p.Ktot = p.R * p.Lpad;
            p.H = (int32_t)P;
            p.W = (int32_t)Q;
            p.C = K;
            p.st = 1;
            p.off_h = da - c.T + 1;
            p.off_w = db - c.U + 1;
            set_out_grid(p, d->n, hc, wc);
            p.OH = (int32_t)d->h;
            p.OW = (int32_t)d->w;
            p.ldo = C;
            p.os = st;
            p.oa = a;
            p.ob = bb;
            p.act_bytes = d->n * P * Q * d->k;
            p.wgt_bytes = (int64_t)C * c.T * c.U * K;
        }
    }
    // A 1 x 1 stride-2 filter: only class (0, 0) has taps, and its kernel
    // writes the zeros of the other three classes beside its own pixels.
    if (st == 2 && b.nprob == 1 && b.p[0].oa == 0 && b.p[0].ob == 0 && zero_mask == 0xEu) {
        b.p[0].zsib = 7;
        zero_mask = 0;
    }
}

hipError_t pack_dgrad(const niti_conv_desc* d, const int8_t* w, int8_t* packed, const DgradPlan& pl,
                      hipStream_t stream) {
    const int st = d->stride_h;
    return repack_dgrad_run(w, packed, pl.cls, pl.ncls, (int)d->k, (int)d->r, (int)d->s, (int)d->c, st, st, stream);
}

// Zero classes, then the classes with taps (or, with none, an all-zero dx).
niti_status run_dgrad(const niti_conv_desc* d, DgradPlan& pl, niti_round_mode mode, niti_stats* stats,
                      void* stream) {
    const int st = d->stride_h;
    const int K = (int)d->k, R = (int)d->r, S = (int)d->s;
    IgemmBatch& b = pl.b;
    hipError_t e = zero_classes_run(pl.dx, d->n, d->h, d->w, d->c, st, pl.zero_mask, as_stream(stream));
    if (e != hipSuccess) return NITI_ERR_HIP;
    if (b.nprob == 0) {
        // No class has taps (a 1x1 filter that only ever sees padding): dx is
        // all zeros and the call's maximum is 0.
        e = max_abs_i32(nullptr, 0, stats, as_stream(stream));
        if (e != hipSuccess) return NITI_ERR_HIP;
        return hip_status(round_i32_run(nullptr, nullptr, 0, -1, 7, mode, stats, ExpArgs{nullptr, nullptr, nullptr},
                                        as_stream(stream)));
    }
    IgemmCtl ctl{};
    ctl.stats = stats;
    ctl.ex = ExpArgs{nullptr, nullptr, nullptr};
    ctl.target = 7;
    ctl.relu = 0;
    ctl.mode = mode;
    ctl.static_flags = acc_flags((int64_t)K * R * S);
    return hip_status(igemm_run(b, ctl, as_stream(stream)));
}

// Shared argument checks of the back-propagation entry points.
niti_status check_dgrad(const niti_conv_desc* d, const int8_t* dy, const void* packed, int8_t* dx,
                        const int8_t* relu_src, niti_round_mode mode, niti_stats* stats, size_t packed_bytes,
                        int64_t* P, int64_t* Q) {
    if (!d) return NITI_ERR_NULL;
    if (!dy || !packed || !dx || !stats) return NITI_ERR_NULL;
    if (mis16(dy) || mis16(packed) || mis16(dx) || mis16(relu_src)) return NITI_ERR_ARG;
    if (!valid_mode(mode)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, P, Q);
    if (s != NITI_OK) return s;
    if (d->stride_h > kMaxDgradStride) return NITI_ERR_UNSUPPORTED;
    if (packed_bytes < niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, d, 0, 0, 0)) return NITI_ERR_WORKSPACE;
    return NITI_OK;
}

}  // namespace

niti_status niti_conv_bwd_data(const niti_conv_desc* d, const int8_t* dy, const int8_t* w, int8_t* dx,
                               const int8_t* relu_src, niti_round_mode mode, niti_stats* stats, void* ws,
                               size_t ws_bytes, void* stream) {
    int64_t P, Q;
    if (!d) return NITI_ERR_NULL;
    if (!dy || !w || !dx || !stats) return NITI_ERR_NULL;
    if (mis16(dy) || mis16(w) || mis16(dx) || mis16(relu_src) || mis16(ws)) return NITI_ERR_ARG;
    if (!valid_mode(mode)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, &P, &Q);
    if (s != NITI_OK) return s;
    if (d->stride_h > kMaxDgradStride) return NITI_ERR_UNSUPPORTED;
    const size_t need = niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, d, 0, 0, 0);
    if (!ws || ws_bytes < need) return NITI_ERR_WORKSPACE;
    DgradPlan pl;
    plan_dgrad(d, P, Q, dy, (const int8_t*)ws, dx, relu_src, pl);
    if (pack_dgrad(d, w, (int8_t*)ws, pl, as_stream(stream)) != hipSuccess) return NITI_ERR_HIP;
    return run_dgrad(d, pl, mode, stats, stream);
}

niti_status niti_conv_pack_bwd_data(const niti_conv_desc* d, const int8_t* w, void* packed, size_t packed_bytes,
                                    void* stream) {
    int64_t P, Q;
    if (!d) return NITI_ERR_NULL;
    if (!w || !packed) return NITI_ERR_NULL;
    if (mis16(w) || mis16(packed)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, &P, &Q);
    if (s != NITI_OK) return s;
    if (d->stride_h > kMaxDgradStride) return NITI_ERR_UNSUPPORTED;
    if (packed_bytes < niti_workspace_bytes(NITI_OP_CONV_BWD_DATA, d, 0, 0, 0)) return NITI_ERR_WORKSPACE;
    DgradPlan pl;
    plan_dgrad(d, P, Q, nullptr, (const int8_t*)packed, nullptr, nullptr, pl);
    return hip_status(pack_dgrad(d, w, (int8_t*)packed, pl, as_stream(stream)));
}

niti_status niti_conv_bwd_data_packed(const niti_conv_desc* d, const int8_t* dy, const void* packed, int8_t* dx,
                                      const int8_t* relu_src, niti_round_mode mode, niti_stats* stats,
                                      size_t packed_bytes, void* stream) {
    int64_t P, Q;
    niti_status s = check_dgrad(d, dy, packed, dx, relu_src, mode, stats, packed_bytes, &P, &Q);
    if (s != NITI_OK) return s;
    DgradPlan pl;
    plan_dgrad(d, P, Q, dy, (const int8_t*)packed, dx, relu_src, pl);
    return run_dgrad(d, pl, mode, stats, stream);
}

niti_status niti_conv_bwd_weight(const niti_conv_desc* d, const int8_t* x, const int8_t* dy, int8_t* w,
                                 int32_t* g32_out, int mu, niti_round_mode mode, niti_stats* stats, void* ws,
                                 size_t ws_bytes, void* stream) {
    int64_t P, Q;
    if (!d) return NITI_ERR_NULL;
    if (!x || !dy || !w || !stats) return NITI_ERR_NULL;
    if (mis16(x) || mis16(dy) || mis16(w) || mis16(g32_out) || mis16(ws)) return NITI_ERR_ARG;
    if (mu < 1 || mu > 8 || !valid_mode(mode)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, &P, &Q);
    if (s != NITI_OK) return s;
    const int64_t nw = d->k * d->r * d->s * d->c;
    const int64_t npix = d->n * P * Q;
    if (too_big(npix)) return NITI_ERR_UNSUPPORTED;
    hipStream_t strm = as_stream(stream);
    const WgradSetup ws_ = wgrad_setup(d, P, Q);
    WgradProblem p = ws_.p;
    const bool win = ws_.win;
    const WinPlan& wp = ws_.wp;
    const WgradPlan& plan = ws_.plan;
    p.dy = dy;
    p.x = x;
    const int64_t g_bytes = g32_out ? 0 : round_up(nw * 4, 256);
    const int64_t p_bytes = plan.splits > 1 ? round_up((int64_t)plan.splits * nw * 4, 256) : 0;
    const int64_t x_bytes = win ? wp.xpad_bytes : 0;
    if (too_big(p_bytes)) return NITI_ERR_UNSUPPORTED;
    if (g_bytes + p_bytes + x_bytes > 0 && (!ws || ws_bytes < (size_t)(g_bytes + p_bytes + x_bytes)))
        return NITI_ERR_WORKSPACE;
    int32_t* g32 = g32_out ? g32_out : (int32_t*)ws;
    int32_t* part = plan.splits > 1 ? (int32_t*)((char*)ws + g_bytes) : g32;
    hipError_t e;
    if (win && !wp.in_place) {
        int8_t* xpad = (int8_t*)ws + g_bytes + p_bytes;
        e = pad_image_run(x, xpad, d->n, d->h, d->w, d->c, wp.hp, wp.wp, d->pad_h, d->pad_w, strm);
        if (e != hipSuccess) return NITI_ERR_HIP;
        p.x = xpad;
    }
    p.part = part;
    const int tix = timing_begin(NITI_TIMING_WGRAD, strm);
    if (ws_.tap)
        e = wgrad_tap_run(p, plan, strm);
    else
        e = wgrad_dma_eligible(p) ? wgrad_dma_run(p, plan, strm) : wgrad_run(p, plan, strm);
    timing_end(tix, strm);
    if (e != hipSuccess) return NITI_ERR_HIP;
    const int tsum = timing_on() ? timing_begin(NITI_TIMING_SUM, strm, kernel_label("split_sum<%d>", plan.splits)) : -1;
    e = reduce_max_run(part, plan.splits, g32, nw, stats, strm);
    timing_end(tsum, strm);
    if (e != hipSuccess) return NITI_ERR_HIP;
    const int tupd = timing_begin(NITI_TIMING_UPDATE, strm);
    e = update_run(w, g32, nw, mu, mode, stats, acc_flags(npix), strm);
    timing_end(tupd, strm);
    return hip_status(e);
}

namespace {

constexpr size_t kScratchBytes = NITI_NOALLOC_SCRATCH_BYTES;   // size of `scratch`
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device, once resolved

// Device address of this device's copy of `scratch`, resolved on the first
// call made on each device (with that device current).
niti_status scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return NITI_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return NITI_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return NITI_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return NITI_OK;
}

}  // namespace

niti_status niti_conv_bwd_weight_noalloc(const niti_conv_desc* d, const int8_t* x, const int8_t* dy, int8_t* w,
                                         int32_t* g32_out, int mu, niti_round_mode mode, niti_stats* stats,
                                         void* stream) {
    // The checks of niti_conv_bwd_weight that do not involve the workspace,
    // made here first so that a rejected call touches no device state.
    int64_t P, Q;
    if (!d) return NITI_ERR_NULL;
    if (!x || !dy || !w || !stats) return NITI_ERR_NULL;
    if (mis16(x) || mis16(dy) || mis16(w) || mis16(g32_out)) return NITI_ERR_ARG;
    if (mu < 1 || mu > 8 || !valid_mode(mode)) return NITI_ERR_ARG;
    niti_status s = check_conv(d, &P, &Q);
    if (s != NITI_OK) return s;
    if (too_big(d->n * P * Q)) return NITI_ERR_UNSUPPORTED;
    if (niti_workspace_bytes(NITI_OP_CONV_BWD_WEIGHT, d, 0, 0, 0) > kScratchBytes) return NITI_ERR_WORKSPACE;
    void* ws = nullptr;
    s = scratch_address(&ws);
    if (s != NITI_OK) return s;
    return niti_conv_bwd_weight(d, x, dy, w, g32_out, mu, mode, stats, ws, kScratchBytes, stream);
}

niti_status niti_round_psr(const int32_t* x, int8_t* y, int64_t n, int bp, int target_bits,
                           niti_round_mode mode, const int8_t* s_in, int8_t* s_out, niti_stats* stats,
                           void* stream) {
    if (n < 0) return NITI_ERR_SHAPE;
    if ((!x || !y) && n > 0) return NITI_ERR_NULL;
    if (mis16(x) || mis16(y)) return NITI_ERR_ARG;
    if (!valid_mode(mode) || bp > 31) return NITI_ERR_ARG;
    if ((s_in == nullptr) != (s_out == nullptr)) return NITI_ERR_NULL;
    if (bp < 0) {
        if (!stats) return NITI_ERR_NULL;
        if (target_bits < 1 || target_bits > 31) return NITI_ERR_ARG;
    }
    if (mode == NITI_ROUND_SR && !stats) return NITI_ERR_NULL;   // the draws' seed and index
    hipStream_t strm = as_stream(stream);
    if (bp < 0) {
        hipError_t e = max_abs_i32(x, n, stats, strm);
        if (e != hipSuccess) return NITI_ERR_HIP;
    }
    return hip_status(round_i32_run(x, y, n, bp, target_bits, mode, (bp < 0 || mode == NITI_ROUND_SR) ? stats : nullptr,
                                    ExpArgs{s_in, nullptr, s_out}, strm));
}

niti_status niti_int_ce_loss_grad(const int8_t* logits, const int8_t* s_logits, const int32_t* labels,
                                  int8_t* err, int64_t batch, int64_t classes, niti_round_mode mode,
                                  niti_stats* stats, void* ws, size_t ws_bytes, void* stream) {
    if (!logits || !s_logits || !labels || !err || !stats) return NITI_ERR_NULL;
    if (mis16(logits) || mis16(labels) || mis16(err) || mis16(ws)) return NITI_ERR_ARG;
    if (batch < 1 || classes < 1) return NITI_ERR_SHAPE;
    if (classes > 65536 || !valid_mode(mode)) return NITI_ERR_ARG;
    if (too_big(batch * classes * 16)) return NITI_ERR_UNSUPPORTED;
    const size_t need = niti_workspace_bytes(NITI_OP_INT_CE_LOSS, nullptr, batch, classes, 0);
    if (!ws || ws_bytes < need) return NITI_ERR_WORKSPACE;
    const int t = timing_begin(NITI_TIMING_LOSS, as_stream(stream));
    const hipError_t e = loss_run(logits, s_logits, labels, err, ws, batch, classes, mode, stats, as_stream(stream));
    timing_end(t, as_stream(stream));
    return hip_status(e);
}

niti_status niti_sgd_update(int8_t* w, const int32_t* g32, int64_t n, int mu, niti_round_mode mode,
                            niti_stats* stats, void* stream) {
    if (n < 0) return NITI_ERR_SHAPE;
    if (((!w || !g32) && n > 0) || !stats) return NITI_ERR_NULL;
    if (mis16(w) || mis16(g32)) return NITI_ERR_ARG;
    if (mu < 1 || mu > 8 || !valid_mode(mode)) return NITI_ERR_ARG;
    if (too_big(n * 4)) return NITI_ERR_UNSUPPORTED;
    hipStream_t strm = as_stream(stream);
    hipError_t e = max_abs_i32(g32, n, stats, strm);
    if (e != hipSuccess) return NITI_ERR_HIP;
    return hip_status(update_run(w, g32, n, mu, mode, stats, 0u, strm));
}

niti_status niti_quantize_u8(const uint8_t* px, int8_t* x, int64_t n, int64_t c, int64_t h, int64_t w,
                             int64_t c_pad, void* stream) {
    if (!px || !x) return NITI_ERR_NULL;
    if (n < 1 || c < 1 || h < 1 || w < 1 || c_pad < c) return NITI_ERR_SHAPE;
    if (too_big(n * h * w * c_pad)) return NITI_ERR_UNSUPPORTED;
    return hip_status(quantize_run(px, x, n, c, h, w, c_pad, as_stream(stream)));
}

niti_status niti_maxpool2_fwd(const int8_t* x, int8_t* y, uint8_t* idx, int64_t n, int64_t h, int64_t w,
                              int64_t c, void* stream) {
    if (!x || !y || !idx) return NITI_ERR_NULL;
    if (n < 1 || h < 2 || w < 2 || c < 1 || (h & 1) || (w & 1)) return NITI_ERR_SHAPE;
    if (too_big(n * h * w * c)) return NITI_ERR_UNSUPPORTED;
    return hip_status(maxpool_fwd_run(x, y, idx, n, h, w, c, as_stream(stream)));
}

niti_status niti_maxpool2_bwd(const int8_t* dy, const uint8_t* idx, int8_t* dx, int64_t n, int64_t h,
                              int64_t w, int64_t c, void* stream) {
    if (!dy || !idx || !dx) return NITI_ERR_NULL;
    if (n < 1 || h < 2 || w < 2 || c < 1 || (h & 1) || (w & 1)) return NITI_ERR_SHAPE;
    if (too_big(n * h * w * c)) return NITI_ERR_UNSUPPORTED;
    return hip_status(maxpool_bwd_run(dy, idx, dx, n, h, w, c, as_stream(stream)));
}

niti_status niti_dropout_fwd(const int8_t* x, int8_t* y, uint8_t* keep, int64_t n, uint64_t seed, uint32_t call,
                             int drop256, const int8_t* s_x, int8_t* s_y, int exp_add, void* stream) {
    if (n < 0) return NITI_ERR_SHAPE;
    if ((!x || !y || !keep) && n > 0) return NITI_ERR_NULL;
    if ((s_x == nullptr) != (s_y == nullptr)) return NITI_ERR_NULL;
    if (drop256 < 0 || drop256 > 256 || exp_add < -8 || exp_add > 8) return NITI_ERR_ARG;
    if (too_big(n)) return NITI_ERR_UNSUPPORTED;
    return hip_status(dropout_fwd_run(x, y, keep, n, seed, call, (uint32_t)drop256, s_x, s_y, exp_add,
                                      as_stream(stream)));
}

niti_status niti_dropout_bwd(const int8_t* dy, const uint8_t* keep, int8_t* dx, int64_t n, void* stream) {
    if (n < 0) return NITI_ERR_SHAPE;
    if ((!dy || !keep || !dx) && n > 0) return NITI_ERR_NULL;
    if (too_big(n)) return NITI_ERR_UNSUPPORTED;
    return hip_status(dropout_bwd_run(dy, keep, dx, n, as_stream(stream)));
}

niti_status niti_relu_mask(int8_t* e, const int8_t* a, int64_t n, void* stream) {
    if (n < 0) return NITI_ERR_SHAPE;
    if ((!e || !a) && n > 0) return NITI_ERR_NULL;
    if (too_big(n)) return NITI_ERR_UNSUPPORTED;
    return hip_status(relu_mask_run(e, a, n, as_stream(stream)));
}

}  // extern "C"
