// Implicit-GEMM int8 MFMA kernel for the forward contraction and the error
// back-propagation contraction of fully-connected and convolution layers
// (Algorithm 1; Section 3.2 reduces convolutions to matrix products), with
// the block-exponent epilogue fused in (optional ReLU, tensor-wide maximum,
// shift-and-round to int8, optional backward ReLU mask).
//
// Problem form.  out[m][n] = round( sum_kk  wgt[n][kk] * act_row(m)[kk] )
//   m  : output pixel (image, row, column) of an NHWC output grid,
//   n  : output channel,
//   kk : (tap row r, byte j of that tap row's segment) with the segment the
//        contiguous NHWC run of S input pixels x C channels (L = S*C bytes),
//        padded to Lpad (multiple of 16) so a 16-byte piece never crosses r.
// The activation row of pixel m is read straight from the NHWC input (no
// im2col buffer), with zero outside the image.  Forward convolution,
// stride-1 back-propagation (flipped, transposed filter) and each sub-pixel
// class of a strided back-propagation are all this form; a plain matrix
// product is the 1x1 case.
//
// Exponent handling.  The rounding shift depends on the maximum over the
// whole output tensor, which is known only when every tile is done.  The
// main launch computes every tile, folds its maximum into the
// tensor maximum and writes the tile rounded with the shift the same stats
// block reported last time.  The fix-up launch derives the
// true shift; when it matches, the output is already exact and the launch
// only finalizes the statistics; otherwise it recomputes every tile with the
// true shift.  Either way the result equals rounding the true accumulators
// with the true shift.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int BK = 64;       // K bytes per main-loop step
constexpr int PITCH = 80;    // LDS row pitch: 64 data bytes + 16 pad (bank spread)
constexpr int NTHREADS = 256;

struct Tile {
    int prob, tm, tn;
};

__device__ __forceinline__ Tile locate_tile(const IgemmBatch& b, int t) {
    Tile r{0, 0, 0};
    int p = 0;
#pragma unroll
    for (int i = 1; i < kMaxProblems; i++)
        if (i < b.nprob && t >= b.p[i].tile_base) p = i;
    const int local = t - b.p[p].tile_base;
    r.prob = p;
    r.tm = local / b.p[p].tiles_n;
    r.tn = local - r.tm * b.p[p].tiles_n;
    return r;
}

// 16 bytes from an address of unknown alignment.
__device__ __forceinline__ uint4 load16(const int8_t* p) {
    const uintptr_t a = (uintptr_t)p;
    if ((a & 15) == 0) return *(const uint4*)p;
    uint4 v;
    if ((a & 3) == 0) {
        const uint32_t* q = (const uint32_t*)p;
        v.x = q[0]; v.y = q[1]; v.z = q[2]; v.w = q[3];
        return v;
    }
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; i++)
        w[i] = (uint32_t)(uint8_t)p[4 * i] | ((uint32_t)(uint8_t)p[4 * i + 1] << 8) |
               ((uint32_t)(uint8_t)p[4 * i + 2] << 16) | ((uint32_t)(uint8_t)p[4 * i + 3] << 24);
    v.x = w[0]; v.y = w[1]; v.z = w[2]; v.w = w[3];
    return v;
}

// Bytes [lo, hi) of a 16-byte window starting at p (0 <= lo <= hi <= 16),
// zero elsewhere.  Only the valid bytes are touched.
__device__ __forceinline__ uint4 load16_partial(const int8_t* p, int lo, int hi) {
    uint32_t w[4] = {0, 0, 0, 0};
    for (int i = lo; i < hi; i++) w[i >> 2] |= (uint32_t)(uint8_t)p[i] << (8 * (i & 3));
    uint4 v;
    v.x = w[0]; v.y = w[1]; v.z = w[2]; v.w = w[3];
    return v;
}

// Per-thread view of one activation row (one output pixel).
struct ActRow {
    const int8_t* base;  // image base + (ih0*W + iw0)*C  (may point before the image)
    int ih0;             // input row of tap 0
    int jlo, jhi;        // valid byte range of a tap row segment: [-iw0*C, (W-iw0)*C)
    int valid;
};

template <int TBM>
__device__ __forceinline__ void setup_act_rows(const IgemmProblem& P, int tm, ActRow* rows) {
    // Thread t loads pieces t + 256*i: row (t + 256 i) / 4, piece (t & 3).
#pragma unroll
    for (int i = 0; i < TBM / 64; i++) {
        const int rloc = (threadIdx.x + NTHREADS * i) >> 2;
        const int m = tm * TBM + rloc;
        ActRow r;
        r.valid = m < P.M;
        const int mm = r.valid ? m : 0;
        const uint32_t img = fdiv((uint32_t)mm, P.div_ohw);
        const uint32_t rem = (uint32_t)mm - img * (uint32_t)(P.OHc * P.OWc);
        const uint32_t oh = fdiv(rem, P.div_ow);
        const uint32_t ow = rem - oh * (uint32_t)P.OWc;
        const int ih0 = (int)oh * P.st + P.off_h;
        const int iw0 = (int)ow * P.st + P.off_w;
        r.ih0 = ih0;
        r.jlo = -iw0 * P.C;
        r.jhi = (P.W - iw0) * P.C;
        r.base = P.act + (int64_t)img * P.H * P.W * P.C + ((int64_t)ih0 * P.W + iw0) * P.C;
        rows[i] = r;
    }
}

__device__ __forceinline__ uint4 load_act_piece(const IgemmProblem& P, const ActRow& row, int r, int j) {
    uint4 z = make_uint4(0, 0, 0, 0);
    const int ih = row.ih0 + r;
    if (!row.valid || r >= P.R || (unsigned)ih >= (unsigned)P.H) return z;
    const int lo = max(row.jlo, j), hi = min(min(row.jhi, P.L), j + 16);
    if (hi <= lo) return z;
    const int8_t* p = row.base + (int64_t)r * P.W * P.C + j;
    if (lo == j && hi == j + 16) return load16(p);
    return load16_partial(p, lo - j, hi - j);
}

__device__ __forceinline__ uint4 load_wgt_piece(const IgemmProblem& P, int n, int r, int j) {
    uint4 z = make_uint4(0, 0, 0, 0);
    if (n >= P.Nout || r >= P.R || j >= P.L) return z;
    const int8_t* p = P.wgt + ((int64_t)n * P.R + r) * P.L + j;
    if (j + 16 <= P.L) return load16(p);
    return load16_partial(p, 0, P.L - j);
}

// (r, j) of the 16-byte piece at K offset kk (uniform across the block).
__device__ __forceinline__ void split_k(const IgemmProblem& P, int kk, int& r, int& j) {
    r = kk / P.Lpad;
    j = kk - r * P.Lpad;
}

template <int TBM, int TBN>
struct Smem {
    int8_t a[2][TBN * PITCH];  // weight rows (output channels)
    int8_t b[2][TBM * PITCH];  // activation rows (output pixels)
};

// One tile: accumulate, then round/store (and fold the maximum).
template <int TBM, int TBN>
__device__ __forceinline__ void run_tile(const IgemmProblem& P, int tm, int tn, Smem<TBM, TBN>& sm,
                                         const RoundK& rk, int relu, int do_store, int do_max,
                                         uint64_t& tmax) {
    constexpr int WTM = TBM / 2;  // wave tile: pixels
    constexpr int WTN = TBN / 2;  // wave tile: channels
    constexpr int FM = WTM / 32;
    constexpr int FN = WTN / 32;
    constexpr int PA = TBN / 64;  // weight pieces per thread
    constexpr int PB = TBM / 64;  // activation pieces per thread

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const int piece = threadIdx.x & 3;

    ActRow rows[PB];
    setup_act_rows<TBM>(P, tm, rows);

    v16i acc[FN][FM];
#pragma unroll
    for (int a = 0; a < FN; a++)
#pragma unroll
        for (int b = 0; b < FM; b++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[a][b][e] = 0;

    const int nk = (P.Ktot + BK - 1) / BK;
    uint4 ra[PA], rb[PB];

    auto gload = [&](int kt) {
        const int kk = kt * BK + piece * 16;
        int r, j;
        split_k(P, kk, r, j);
#pragma unroll
        for (int i = 0; i < PA; i++) {
            const int n = tn * TBN + ((threadIdx.x + NTHREADS * i) >> 2);
            ra[i] = kk < P.Ktot ? load_wgt_piece(P, n, r, j) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < PB; i++)
            rb[i] = kk < P.Ktot ? load_act_piece(P, rows[i], r, j) : make_uint4(0, 0, 0, 0);
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < PA; i++) {
            const int row = (threadIdx.x + NTHREADS * i) >> 2;
            *(uint4*)&sm.a[buf][row * PITCH + piece * 16] = ra[i];
        }
#pragma unroll
        for (int i = 0; i < PB; i++) {
            const int row = (threadIdx.x + NTHREADS * i) >> 2;
            *(uint4*)&sm.b[buf][row * PITCH + piece * 16] = rb[i];
        }
    };

    if (nk > 0) {
        gload(0);
        sstore(0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; kt++) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < 2; ks++) {
            const int koff = ks * 32 + (lane >> 5) * 16;
            v4i fa[FN], fb[FM];
#pragma unroll
            for (int a = 0; a < FN; a++) {
                const int row = wn * WTN + a * 32 + (lane & 31);
                fa[a] = *(const v4i*)&sm.a[buf][row * PITCH + koff];
            }
#pragma unroll
            for (int b = 0; b < FM; b++) {
                const int row = wm * WTM + b * 32 + (lane & 31);
                fb[b] = *(const v4i*)&sm.b[buf][row * PITCH + koff];
            }
#pragma unroll
            for (int a = 0; a < FN; a++)
#pragma unroll
                for (int b = 0; b < FM; b++)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
        }
        if (kt + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }

    // Epilogue.  acc[a][b] element 4*jj + i sits at channel
    // n = tile_n + wn*WTN + a*32 + 8*jj + 4*(lane/32) + i and pixel
    // m = tile_m + wm*WTM + b*32 + lane%32: four consecutive channels of one
    // pixel, i.e. four consecutive bytes of the NHWC output.
#pragma unroll
    for (int b = 0; b < FM; b++) {
        const int m = tm * TBM + wm * WTM + b * 32 + (lane & 31);
        const bool mvalid = m < P.M;
        int64_t ooff = 0;
        uint32_t zs = 0;
        if (mvalid) {
            const uint32_t img = fdiv((uint32_t)m, P.div_ohw);
            const uint32_t rem = (uint32_t)m - img * (uint32_t)(P.OHc * P.OWc);
            const uint32_t i0 = fdiv(rem, P.div_ow);
            const uint32_t j0 = rem - i0 * (uint32_t)P.OWc;
            const int oh = (int)i0 * P.os + P.oa;
            const int ow = (int)j0 * P.os + P.ob;
            ooff = (((int64_t)img * P.OH + oh) * P.OW + ow) * P.ldo;
            if (P.zsib) zs = zero_siblings(P, oh, ow);
        }
#pragma unroll
        for (int a = 0; a < FN; a++) {
#pragma unroll
            for (int jj = 0; jj < 4; jj++) {
                const int n0 = tn * TBN + wn * WTN + a * 32 + 8 * jj + 4 * (lane >> 5);
                int32_t v[4];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    int32_t x = acc[a][b][4 * jj + i];
                    if (relu && x < 0) x = 0;
                    v[i] = x;
                }
                if (!mvalid || n0 >= P.Nout) continue;
                const int nv = min(4, P.Nout - n0);
                if (do_max) {
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        if (i < nv) {
                            const uint64_t mg = mag32(v[i]);
                            tmax = mg > tmax ? mg : tmax;
                        }
                }
                if (do_store) {
                    uint32_t packed = 0;
#pragma unroll
                    for (int i = 0; i < 4; i++)
                        packed |= (uint32_t)(uint8_t)round_i32_at(v[i], rk, (uint64_t)(ooff + n0 + i)) << (8 * i);
                    int8_t* dst = P.out + ooff + n0;
                    if (P.mask) {
                        const int8_t* ms = P.mask + ooff + n0;
#pragma unroll
                        for (int i = 0; i < 4; i++)
                            if (i < nv && ms[i] <= 0) packed &= ~(0xFFu << (8 * i));
                    }
                    if (nv == 4 && ((((uintptr_t)dst) & 3) == 0)) {
                        *(uint32_t*)dst = packed;
                    } else {
                        for (int i = 0; i < nv; i++) dst[i] = (int8_t)(packed >> (8 * i));
                    }
                }
            }
        }
        if (do_store && zs) {
            for (int a = 0; a < FN; a++)
                for (int jj = 0; jj < 4; jj++) {
                    const int n0 = tn * TBN + wn * WTN + a * 32 + 8 * jj + 4 * (lane >> 5);
                    if (n0 < P.Nout) store_zero_siblings(P, ooff + n0, zs, min(4, P.Nout - n0));
                }
        }
    }
}

// Main launch: every tile once, maximum folded in, output rounded with the
// shift guessed from the previous call (no output when there is no guess).
template <int TBM, int TBN>
__global__ __launch_bounds__(NTHREADS) void igemm_main(IgemmBatch batch, IgemmCtl ctl) {
    __shared__ Smem<TBM, TBN> sm;
    niti_stats* st = ctl.stats;
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    const int hint = st->bp_hint;
    begin_call(st, slot, hint);
    const Tile t = locate_tile(batch, blockIdx.x);
    RoundK rk = make_round(hint < 0 ? 0 : hint, ctl.mode);
    sr_key_current(rk, st);
    uint64_t tmax = 0;
    run_tile<TBM, TBN>(batch.p[t.prob], t.tm, t.tn, sm, rk, ctl.relu, hint >= 0, 1, tmax);
    __shared__ uint32_t red[NTHREADS / 64];
    block_publish_max32(st, slot, (uint32_t)tmax, red, snap);  // magnitudes <= 2^31
}

// Fix-up launch: the tensor maximum is final.  If the guessed shift was
// right there is nothing to redo; otherwise every tile is recomputed and
// rounded with the true shift.  Workgroup 0 then records the statistics and
// the output exponent.
template <int TBM, int TBN>
__global__ __launch_bounds__(NTHREADS) void igemm_fixup(IgemmBatch batch, IgemmCtl ctl) {
    __shared__ Smem<TBM, TBN> sm;
    niti_stats* st = ctl.stats;
    const CallState cs = shared_call_state(st);
    const int hint = cs.hint;
    const int bp = block_bp(cs.mx, ctl.target);
    if (bp != hint) {
        RoundK rk = make_round(bp, ctl.mode);
        sr_key_recorded(rk, st);
        for (int tt = blockIdx.x; tt < batch.total_tiles; tt += gridDim.x) {
            const Tile t = locate_tile(batch, tt);
            uint64_t dummy = 0;
            run_tile<TBM, TBN>(batch.p[t.prob], t.tm, t.tn, sm, rk, ctl.relu, 1, 0, dummy);
            __syncthreads();
        }
    }
    if (is_finisher()) finish_call(st, ctl.target, ctl.ex, ctl.static_flags, 1);
}

template <int TBM, int TBN>
hipError_t launch_igemm(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    int base = 0;
    for (int i = 0; i < b.nprob; i++) {
        IgemmProblem& p = b.p[i];
        p.tiles_m = (p.M + TBM - 1) / TBM;
        p.tiles_n = (p.Nout + TBN - 1) / TBN;
        p.tile_base = base;
        base += p.tiles_m * p.tiles_n;
    }
    b.total_tiles = base;
    const int tk = timing_on()
                       ? timing_begin(NITI_TIMING_KERNEL, stream, kernel_label("igemm_main<%d,%d>", TBM, TBN))
                       : -1;
    hipLaunchKernelGGL((igemm_main<TBM, TBN>), dim3(base), dim3(NTHREADS), 0, stream, b, ctl);
    timing_end(tk, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int fix_grid = base < kFixupGrid ? base : kFixupGrid;
    hipLaunchKernelGGL((igemm_fixup<TBM, TBN>), dim3(fix_grid), dim3(NTHREADS), 0, stream, b, ctl);
    return hipGetLastError();
}

}  // namespace

namespace {

hipError_t igemm_dispatch(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    // Stochastic rounding keys each draw by the element's offset in the
    // output, which only this kernel's epilogue carries.
    const bool sr = ctl.mode == NITI_ROUND_SR;
    if (!sr && igemm_small_eligible(b)) return igemm_small_run(b, ctl, stream);
    if (!sr && igemm_wres_eligible(b)) return igemm_wres_run(b, ctl, stream);
    if (!sr && igemm_dma_eligible(b)) return igemm_dma_run(b, ctl, stream);
    // All problems of a batch share the tile shape; pick it from the largest.
    int maxM = 0, maxN = 0;
    for (int i = 0; i < b.nprob; i++) {
        maxM = b.p[i].M > maxM ? b.p[i].M : maxM;
        maxN = b.p[i].Nout > maxN ? b.p[i].Nout : maxN;
    }
    // Small problems (a classifier head's back-propagation) get 64 x 64
    // tiles, so that more than a handful of CUs take part.
    int64_t tiles128 = 0;
    for (int i = 0; i < b.nprob; i++)
        tiles128 += (int64_t)((b.p[i].M + 127) / 128) * ((b.p[i].Nout + 127) / 128);
    if (tiles128 < 64) return launch_igemm<64, 64>(b, ctl, stream);
    (void)maxM;
    if (maxN <= 64) return launch_igemm<256, 64>(b, ctl, stream);
    return launch_igemm<128, 128>(b, ctl, stream);
}

}  // namespace

hipError_t igemm_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    const int t = timing_begin(NITI_TIMING_IGEMM, stream);
    const hipError_t e = igemm_dispatch(b, ctl, stream);
    timing_end(t, stream);
    return e;
}

}  // namespace niti
