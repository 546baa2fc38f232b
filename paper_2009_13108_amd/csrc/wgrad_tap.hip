// Weight-gradient contraction for 3x3 convolutions with channel counts that
// are multiples of 64 (Algorithm 1, g(l) = a(l-1) (x) e(l); Section 3.3):
//
//   g32[k][(r*3 + s)*C + c] = sum over pixels pix of dy[pix][k] * x[n][oh*sh - ph + r][ow*sw - pw + s][c]
//
// The nine taps of one channel chunk read the same input pixels, shifted.
// A workgroup therefore owns an output tile of 64 output channels x (all nine
// taps of a 32-channel chunk) and, per stage of 128 output pixels, loads the
// nine shifted 128-pixel x 32-byte slices and the 128 x 64-byte error slice.
// The nine slices of one stage touch the same few input rows at nearly the
// same time, so they meet in L2 instead of re-reading memory past it, which
// is what bounds a kernel that tiles the im2col columns independently.
//
// The pixel reduction is split over about one workgroup per CU and every
// workgroup writes its partial tile, which the split-sum pass reads back:
// that traffic is the workgroup count times the tile size.  A 32-channel
// chunk halves it against a 64-channel one, for 10% more operand loads per
// multiply-add (the error slice is shared by fewer taps' columns).
//
// Layout of a stage in LDS: nine x regions [128 pixels][32 bytes] (one per
// tap; eight consecutive rows are 256 contiguous bytes, so transpose reads
// need no swizzle) and one dy region [128 pixels][64 bytes] (16-byte chunks
// XOR-swizzled by pixel).  The MFMA operands come out of them with transpose
// reads (the same fragment reader as wgrad_dma.hip).  Eight waves, two per
// SIMD: wave w computes output channels k0 + 32*wk .. +31 x the 32 channels
// over pixel half ph of each stage ((wk, ph) from w % 4) for taps 0..4
// (w < 4) or 5..8 (w >= 4): per 32 pixels one error fragment and five or
// four input fragments feed as many MFMAs.  The two pixel halves' sums meet
// in LDS at the end.
//
// Issue cost.  Every instruction a wave issues besides its MFMAs holds the
// SIMD's MFMA pipe for a few cycles (about three and a half with one wave
// per SIMD, about two with two waves), so the kernel keeps the instruction
// count per MFMA low: two waves per SIMD, and only waves 0..3 load.
//
// Loads.  Wave w < 4 fills pixels 32w .. 32w+31 of the nine x regions and
// of the dy region (eleven direct-to-LDS loads of 1 KiB, issued as inline
// assembly so the compiler does not wait for the whole ring before each
// transpose read); a lane keeps the input offset of its pixel and a 9-bit
// mask of the taps that fall outside the image, so each tap's load is one
// add and one bit test.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int PIX = 128;                  // output pixels per stage
constexpr int NTAP = 9;
constexpr int CW = 32;                    // channels per tile
constexpr int XREG = PIX * CW;            // bytes of one [128 pixels][32 bytes] x region
constexpr int DOFF = NTAP * XREG;         // dy region [128 pixels][64 bytes]
constexpr int STAGE = DOFF + PIX * 64;
constexpr int LOADS = NTAP + 2;           // loads per wave and stage
constexpr uint32_t kOOB = 0x80000000u;

typedef __attribute__((address_space(3))) v2i lds_v2i;

template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Wait until this wave's LDS reads are done (lgkmcnt 0, other counters free).
__device__ __forceinline__ void wait_lds0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Chunk swizzle of 64-byte pixel rows: conflict-free transpose reads over 8
// consecutive pixels.
__device__ __forceinline__ int swz(int pix) { return (pix >> 1) & 3; }

// Lane byte offsets, within a region, of the two transpose reads that give a
// 32 x 32-pixel fragment: the lane gets 16 pixel bytes (pixels p0 +
// 16*(lane/32) ...) of column cbase + lane%32.  They depend on the lane, p0
// and cbase only, so a workgroup computes them once.
struct FragOff {
    int lo, hi;
};

// 64-byte rows (dy), swizzled.
__device__ __forceinline__ FragOff frag_off64(int p0, int cbase, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int chunk = (cbase >> 4) + (g & 1);
    const int prow = p0 + 16 * (g >> 1) + (j >> 1);
    const int half = (j & 1) * 8;
    FragOff f;
    f.lo = prow * 64 + ((chunk ^ swz(prow)) << 4) + half;
    f.hi = (prow + 8) * 64 + ((chunk ^ swz(prow + 8)) << 4) + half;
    return f;
}

// 32-byte rows (x), all 32 columns, unswizzled.
__device__ __forceinline__ FragOff frag_off32(int p0, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int prow = p0 + 16 * (g >> 1) + (j >> 1);
    const int col = ((g & 1) << 4) + (j & 1) * 8;
    FragOff f;
    f.lo = prow * 32 + col;
    f.hi = (prow + 8) * 32 + col;
    return f;
}

// Fragment at LDS byte addresses lo / hi plus off (a constant after
// unrolling, folded into the instructions' offset field).
__device__ __forceinline__ v4i tr_frag(uint32_t lo_addr, uint32_t hi_addr, int off) {
    const lds_v2i* lo = (const lds_v2i*)(uintptr_t)lo_addr;
    const lds_v2i* hi = (const lds_v2i*)(uintptr_t)hi_addr;
    const v2i a = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(lo + off / 8));
    const v2i b = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(hi + off / 8));
    v4i r;
    r[0] = a[0];
    r[1] = a[1];
    r[2] = b[0];
    r[3] = b[1];
    return r;
}

// Taps of a wave: wave w of eight runs on SIMD w % 4; waves w and w + 4 take
// taps 0..4 and 5..8 of the same output block and pixel half, so the two
// waves of a SIMD share its MFMA pipe, one issuing while the other waits.
// Only waves 0..3 load, so the loads' address work is not duplicated.
template <int TH>
struct TapHalf {
    static constexpr int T0 = TH ? 5 : 0;   // first tap
    static constexpr int N = TH ? 4 : 5;    // taps
};
constexpr int NTHREADS = 512;

template <int NS, int TH>
__device__ __forceinline__ void tap_body(const WgradProblem& P, int8_t* lds, int split, int c0, int k0, int pbeg,
                                         int pend, int nsteps) {
    constexpr int T0 = TapHalf<TH>::T0, NTW = TapHalf<TH>::N;
    constexpr bool LOADER = TH == 0;
    constexpr int NR = 2 * (NTW + 1);      // fragment reads per stage
    constexpr int NM = 2 * NTW;            // MFMAs per stage
    constexpr int NG = LOADER ? LOADS : NTW + 1;   // issue groups per step
    const int lane = threadIdx.x & 63;
    const int sub = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3);
    const int wk = sub & 1, ph = sub >> 1;

    const u32x4 xrs = raw_rsrc(P.x, (uint32_t)P.x_bytes);
    const u32x4 drs = raw_rsrc(P.dy, (uint32_t)P.dy_bytes);
    const uint32_t lds0 = lds_address(lds);

    // Loader lanes' rows: x pixel 32*sub + lane/2 (chunk lane%2; a 1 KiB block
    // of an x region is 32 rows of 32 bytes) and dy pixels 32*sub + 16*u +
    // lane/4 (chunk lane%4, swizzled; a block of the dy region is 16 rows).
    const int xrow = 32 * sub + (lane >> 1);
    const uint32_t xbyte = (uint32_t)((lane & 1) << 4);
    int drow[2];
    uint32_t dbyte[2];
#pragma unroll
    for (int u = 0; u < 2; u++) {
        drow[u] = 32 * sub + 16 * u + (lane >> 2);
        dbyte[u] = (uint32_t)(((lane & 3) ^ swz(drow[u])) << 4);
    }
    const uint32_t WC = (uint32_t)P.W * (uint32_t)P.C;

    // Addresses of one stage's loads: LDS stage base, input offset of the
    // lane's x pixel, the taps outside the image, error offsets.
    struct Issue {
        uint32_t st, base, outside, dv[2];
    };
    int next = 0;
    auto prep = [&]() {
        Issue q;
        q.st = lds0 + (uint32_t)((next % NS) * STAGE);
        const int pb = pbeg + next * PIX;
        const int pix = pb + xrow;
        const bool ok = next < nsteps && pix < pend;
        const uint32_t pp = ok ? (uint32_t)pix : 0u;
        const uint32_t n = fdiv(pp, P.div_pq);
        const uint32_t rem = pp - n * (uint32_t)(P.P * P.Q);
        const uint32_t oh = fdiv(rem, P.div_q);
        const uint32_t ow = rem - oh * (uint32_t)P.Q;
        const int h0 = (int)oh * P.sh - P.ph;
        const int w0 = (int)ow * P.sw - P.pw;
        uint32_t rows = 0, cols = 0;
#pragma unroll
        for (int r = 0; r < 3; r++) rows |= (uint32_t)((unsigned)(h0 + r) < (unsigned)P.H) << r;
#pragma unroll
        for (int s = 0; s < 3; s++) cols |= (uint32_t)((unsigned)(w0 + s) < (unsigned)P.W) << s;
        // bit r*3+s set: tap (r, s) outside the image (all taps for a pixel past the range)
        q.outside = ok ? ~((((rows & 1u) ? cols : 0u)) | (((rows & 2u) ? cols : 0u) << 3) |
                           (((rows & 4u) ? cols : 0u) << 6))
                       : ~0u;
        q.base = (uint32_t)(((int)n * P.H + h0) * P.W + w0) * (uint32_t)P.C + (uint32_t)c0 + xbyte;
#pragma unroll
        for (int u = 0; u < 2; u++) {
            const int dp = pb + drow[u];
            q.dv[u] = next < nsteps && dp < pend ? (uint32_t)dp * (uint32_t)P.K + (uint32_t)k0 + dbyte[u] : kOOB;
        }
        next++;
        return q;
    };
    // Load g of a stage: 0..8 this wave's block of the nine shifted input
    // slices, 9 and 10 its two blocks of the error slice.
    auto load = [&](const Issue& q, int g) {
        if (g < NTAP) {
            const uint32_t tap_off = (uint32_t)(g / 3) * WC + (uint32_t)(g % 3) * (uint32_t)P.C;
            const uint32_t v = (__builtin_amdgcn_ubfe(q.outside, (uint32_t)g, 1) << 31) | (q.base + tap_off);
            lds_dma16_at(xrs, q.st, (uint32_t)(g * XREG + sub * 1024), v, 0);
        } else {
            const int u = g - NTAP;
            lds_dma16_at(drs, q.st, (uint32_t)(DOFF + (2 * sub + u) * 1024), q.dv[u], 0);
        }
    };
    auto issue = [&]() {
        const Issue q = prep();
#pragma unroll
        for (int g = 0; g < LOADS; g++) load(q, g);
    };

    // Fragment offsets of this wave's two 32-pixel quarters (2*ph, 2*ph + 1).
    const FragOff fo_x[2] = {frag_off32(64 * ph, lane), frag_off32(64 * ph + 32, lane)};
    const FragOff fo_d[2] = {frag_off64(64 * ph, 32 * wk, lane), frag_off64(64 * ph + 32, 32 * wk, lane)};

    v16i acc[NTW];
#pragma unroll
    for (int t = 0; t < NTW; t++)
#pragma unroll
        for (int e = 0; e < 16; e++) acc[t][e] = 0;

    // Fragments of one stage: per 32-pixel quarter, the error fragment and
    // the input fragments of this wave's taps.  A stage's fragments are read
    // during the previous stage's MFMAs, so the LDS latency is hidden behind
    // them.
    struct Frags {
        v4i d[2];
        v4i x[2][NTW];
    };
    // Fragment read f of the stage at LDS address st: per quarter ks, the
    // error fragment, then the taps.
    auto read_one = [&](uint32_t st, int f, Frags& F) {
        const int ks = f / (NTW + 1), i = f % (NTW + 1);
        if (i == 0)
            F.d[ks] = tr_frag(st + fo_d[ks].lo, st + fo_d[ks].hi, DOFF);
        else
            F.x[ks][i - 1] = tr_frag(st + fo_x[ks].lo, st + fo_x[ks].hi, (T0 + i - 1) * XREG);
    };
    // Stage it: stage it + 1 has landed (every loader's loads, hence the
    // barrier) and every wave has its stage-it fragments in registers, so
    // stage it's slot takes stage it + NS; then stage it + 1 is read while
    // stage it's MFMAs run.  Loads, fragment reads and MFMAs of a step are
    // issued interleaved (scheduling barriers keep the order), so a load
    // waiting for the memory pipeline holds up no MFMA.
    auto step = [&](int it, const Frags& cur, Frags& nxt) {
        if (LOADER) wait_vm<(NS - 2) * LOADS>();
        wait_lds0();
        __builtin_amdgcn_s_barrier();
        Issue q;
        if (LOADER) q = prep();
        const uint32_t st1 = lds0 + (uint32_t)(((it + 1) % NS) * STAGE);
#pragma unroll
        for (int g = 0; g < NG; g++) {
            if (LOADER) load(q, g);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int f = (g * NR) / NG; f < ((g + 1) * NR) / NG; f++) read_one(st1, f, nxt);
#pragma unroll
            for (int m = (g * NM) / NG; m < ((g + 1) * NM) / NG; m++) {
                const int ks = m / NTW, t = m % NTW;
                acc[t] = __builtin_amdgcn_mfma_i32_32x32x32_i8(cur.x[ks][t], cur.d[ks], acc[t], 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    if (LOADER) {
#pragma unroll
        for (int s = 0; s < NS; s++) issue();
        wait_vm<(NS - 1) * LOADS>();
    }
    __builtin_amdgcn_s_barrier();
    Frags f0, f1;
#pragma unroll
    for (int f = 0; f < NR; f++) read_one(lds0, f, f0);
    int it = 0;
    for (; it + 1 < nsteps; it += 2) {
        step(it, f0, f1);
        step(it + 1, f1, f0);
    }
    if (it < nsteps) step(it, f0, f1);
    wait_vm<0>();
    wait_lds0();
    __syncthreads();   // the ring is free

    // The two pixel halves: wave (wk, 1, TH) hands its sums to wave
    // (wk, 0, TH) through LDS, slot [wk][tap][jj][lane] of 16 bytes, which
    // adds them to its own and stores.
    v4i* xch = (v4i*)lds;
    if (ph == 1) {
#pragma unroll
        for (int t = 0; t < NTW; t++)
#pragma unroll
            for (int jj = 0; jj < 4; jj++) {
                v4i q;
                q[0] = acc[t][4 * jj];
                q[1] = acc[t][4 * jj + 1];
                q[2] = acc[t][4 * jj + 2];
                q[3] = acc[t][4 * jj + 3];
                xch[((wk * NTAP + T0 + t) * 4 + jj) * 64 + lane] = q;
            }
    }
    __syncthreads();
    if (ph == 1) return;

    // acc[t] element 4*jj + i: channel c0 + 8*jj + 4*(lane/32) + i of tap
    // T0 + t, output channel k0 + 32*wk + lane%32: four consecutive columns
    // per store.
    int32_t* out = P.part + (int64_t)split * P.K * P.ncol + (int64_t)(k0 + 32 * wk + (lane & 31)) * P.ncol;
#pragma unroll
    for (int t = 0; t < NTW; t++)
#pragma unroll
        for (int jj = 0; jj < 4; jj++) {
            const v4i o = xch[((wk * NTAP + T0 + t) * 4 + jj) * 64 + lane];
            const int col = (T0 + t) * P.C + c0 + 8 * jj + 4 * (lane >> 5);
            *(int4*)(out + col) = make_int4(acc[t][4 * jj] + o[0], acc[t][4 * jj + 1] + o[1],
                                            acc[t][4 * jj + 2] + o[2], acc[t][4 * jj + 3] + o[3]);
        }
}

// Work items (split, tile), tile fastest, cut into eight equal consecutive
// runs, one per XCD (workgroup L runs on XCD L % 8), so the tiles of one pixel
// range share an XCD and its L2.
template <int NS>
__global__ __launch_bounds__(NTHREADS, 1) void wgrad_tap_kernel(WgradProblem P, int tiles_c, int tiles_k, int splits) {
    extern __shared__ __attribute__((aligned(1024))) int8_t lds[];
    const int ntiles = tiles_c * tiles_k;
    const int per_xcd = (ntiles * splits + 7) / 8;
    const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if ((blockIdx.x >> 3) >= per_xcd || item >= ntiles * splits) return;
    const int split = item / ntiles;
    const int tile = item - split * ntiles;
    const int c0 = (tile % tiles_c) * CW;
    const int k0 = (tile / tiles_c) * 64;
    const int pbeg = split * P.chunk;
    const int pend = min(P.npix, pbeg + P.chunk);
    const int nsteps = pend > pbeg ? (pend - pbeg + PIX - 1) / PIX : 0;
    if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 8) == 0)
        tap_body<NS, 0>(P, lds, split, c0, k0, pbeg, pend, nsteps);
    else
        tap_body<NS, 1>(P, lds, split, c0, k0, pbeg, pend, nsteps);
}

}  // namespace

bool wgrad_tap_eligible(const WgradProblem& p) {
    return !p.win && p.R == 3 && p.S == 3 && p.C % 64 == 0 && p.K % 64 == 0 && p.x_bytes > 0 &&
           p.x_bytes < ((int64_t)1 << 31) && p.dy_bytes > 0 && p.dy_bytes < ((int64_t)1 << 31);
}

WgradPlan wgrad_tap_plan(int64_t K, int64_t C, int64_t npix) {
    WgradPlan pl;
    pl.tbk = 64;
    const int64_t tiles = (K / 64) * (C / CW);
    const int64_t steps = (npix + PIX - 1) / PIX;
    // About 192 workgroups, at least two stages each.  A workgroup holds
    // most of its CU's LDS and registers, so a grid of one per CU would shut
    // out a kernel running beside it on another stream (the back-propagation
    // of a training step); leaving a quarter of the CUs free measured ~2%
    // faster steps than 256, 160, 224 or a floor of 192 / tiles.
    int64_t splits = (192 + tiles - 1) / tiles;
    const int64_t max_splits = steps / 2 > 1 ? steps / 2 : 1;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    const int64_t chunk_steps = (steps + splits - 1) / splits;
    pl.chunk = (int32_t)(chunk_steps * PIX);
    pl.splits = (int32_t)((steps + chunk_steps - 1) / chunk_steps);
    if (pl.splits < 1) pl.splits = 1;
    return pl;
}

hipError_t wgrad_tap_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream) {
    constexpr int NS = 3;
    constexpr int LDS = NS * STAGE;
    static_assert(LDS >= 2 * NTAP * 4 * 64 * 16, "exchange area");
    static bool attr_done = false;
    if (!attr_done) {
        hipError_t e = hipFuncSetAttribute((const void*)wgrad_tap_kernel<NS>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
        attr_done = true;
    }
    p.chunk = plan.chunk;
    const int tc = p.C / CW, tk = p.K / 64;
    const int64_t grid = (int64_t)8 * (((int64_t)tc * tk * plan.splits + 7) / 8);
    const int t = timing_on() ? timing_begin(NITI_TIMING_KERNEL, stream, kernel_label("wgrad_tap_kernel<%d>", NS)) : -1;
    hipLaunchKernelGGL((wgrad_tap_kernel<NS>), dim3((unsigned)grid), dim3(NTHREADS), LDS, stream, p, tc, tk, plan.splits);
    timing_end(t, stream);
    return hipGetLastError();
}

}  // namespace niti
