// Matrix products with few outputs and a long reduction (Algorithm 1's
// forward and back-propagation contractions of a classifier head: a batch of
// a few hundred samples against a few hundred to a few thousand classes).
//
//   out[m][n] = round( sum_k  wgt[n][k] * act[m][k] ),  k < L
//
// With so few outputs a tiled kernel runs on a handful of CUs and each of
// them walks the reduction step by step, paying a memory round trip per
// step.  Here a workgroup owns one 32 x 32 output tile and its eight waves
// take interleaved 32-byte slices of the reduction: every wave issues all
// of its operand loads at once (straight into MFMA operand registers, no
// LDS staging), runs its MFMAs, and the eight partial tiles are added in
// LDS.  The epilogue (optional ReLU, tensor maximum, shift-and-round,
// backward ReLU mask) and the exponent handling (rounding with the previous
// call's shift, then a fix-up launch that recomputes on a miss) are those of
// the other implicit-GEMM kernels.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int SW = 8;                 // waves per workgroup (reduction slices)
constexpr int ST = SW * 64;           // threads per workgroup
constexpr int KB = 8;                 // 32-byte reduction steps per wave and load batch
constexpr int RP = 36;                // LDS row pitch of a partial tile (ints; 16-byte aligned)
constexpr int MAX_M = 1024;           // eligibility: at most this many output rows

// 16 bytes of a row at byte k, zero past L (rows may be only byte aligned).
__device__ __forceinline__ v4i row_piece(const int8_t* row, int k, int L) {
    v4i r = {0, 0, 0, 0};
    if (k >= L) return r;
    const int8_t* p = row + k;
    const uintptr_t a = (uintptr_t)p;
    if (k + 16 <= L) {
        if ((a & 15) == 0) return *(const v4i*)p;
        if ((a & 7) == 0) {
            const int2 lo = *(const int2*)p, hi = *(const int2*)(p + 8);
            r[0] = lo.x;
            r[1] = lo.y;
            r[2] = hi.x;
            r[3] = hi.y;
            return r;
        }
        if ((a & 3) == 0) {
            const int* q = (const int*)p;
            r[0] = q[0];
            r[1] = q[1];
            r[2] = q[2];
            r[3] = q[3];
            return r;
        }
    }
    const int n = min(16, L - k);
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    for (int i = 0; i < n; i++) w[i >> 2] |= (uint32_t)(uint8_t)p[i] << (8 * (i & 3));
    r[0] = (int)w[0];
    r[1] = (int)w[1];
    r[2] = (int)w[2];
    r[3] = (int)w[3];
    return r;
}

// One 32 x 32 tile: reduce, add the slices, then (threads < 256, four
// consecutive channels of one row each) fold the maximum and store.
__device__ __forceinline__ void small_tile(const IgemmProblem& P, int tile, int32_t* red, const RoundK& rk,
                                           int relu, bool do_store, bool do_max, uint32_t& tmax) {
    const int tiles_n = (P.Nout + 31) >> 5;
    const int tm = tile / tiles_n, tn = tile - tm * tiles_n;
    const int m0 = tm * 32, n0 = tn * 32;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r32 = lane & 31, kh = (lane >> 5) * 16;
    const int L = P.L;
    // Operand rows of this lane (clamped into the tensor; rows past the edge
    // load zeros).
    const bool nok = n0 + r32 < P.Nout, mok = m0 + r32 < P.M;
    const int8_t* wrow = P.wgt + (int64_t)(nok ? n0 + r32 : 0) * L;
    const int8_t* arow = P.act + (int64_t)(mok ? m0 + r32 : 0) * L;
    const int Lw = nok ? L : 0, La = mok ? L : 0;

    v16i acc;
#pragma unroll
    for (int e = 0; e < 16; e++) acc[e] = 0;
    const int nks = (L + 31) >> 5;
    for (int ks0 = wave; ks0 < nks; ks0 += SW * KB) {
        v4i a[KB], b[KB];
#pragma unroll
        for (int j = 0; j < KB; j++) {
            const int k = (ks0 + j * SW) * 32 + kh;
            a[j] = row_piece(wrow, k, Lw);
            b[j] = row_piece(arow, k, La);
        }
#pragma unroll
        for (int j = 0; j < KB; j++) acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[j], b[j], acc, 0, 0, 0);
    }

    // acc element 4*jj + i: channel n0 + 8*jj + 4*(lane/32) + i, row m0 + lane%32.
    int32_t* mine = red + (wave * 32 + r32) * RP + 4 * (lane >> 5);
#pragma unroll
    for (int jj = 0; jj < 4; jj++) {
        v4i q;
        q[0] = acc[4 * jj];
        q[1] = acc[4 * jj + 1];
        q[2] = acc[4 * jj + 2];
        q[3] = acc[4 * jj + 3];
        *(v4i*)(mine + 8 * jj) = q;
    }
    __syncthreads();
    if (threadIdx.x < 256) {
        const int row = threadIdx.x >> 3, c4 = (threadIdx.x & 7) * 4;
        const int m = m0 + row, n = n0 + c4;
        v4i s = *(const v4i*)(red + row * RP + c4);
#pragma unroll
        for (int w = 1; w < SW; w++) s += *(const v4i*)(red + (w * 32 + row) * RP + c4);
        if (m < P.M && n < P.Nout) {
            const int nv = min(4, P.Nout - n);
            int32_t v[4] = {s[0], s[1], s[2], s[3]};
#pragma unroll
            for (int i = 0; i < 4; i++)
                if (relu && v[i] < 0) v[i] = 0;
            if (do_max) {
#pragma unroll
                for (int i = 0; i < 4; i++)
                    if (i < nv) tmax = max(tmax, mag32(v[i]));
            }
            if (do_store) {
                const int64_t off = (int64_t)m * P.ldo + n;
                uint32_t packed = 0;
#pragma unroll
                for (int i = 0; i < 4; i++) packed |= (uint32_t)(uint8_t)round_i32(v[i], rk) << (8 * i);
                if (P.mask) {
                    const int8_t* ms = P.mask + off;
                    for (int i = 0; i < nv; i++)
                        if (ms[i] <= 0) packed &= ~(0xFFu << (8 * i));
                }
                int8_t* dst = P.out + off;
                if (nv == 4 && (((uintptr_t)dst) & 3) == 0) {
                    *(uint32_t*)dst = packed;
                } else {
                    for (int i = 0; i < nv; i++) dst[i] = (int8_t)(packed >> (8 * i));
                }
            }
        }
    }
    __syncthreads();   // red is reused by the next tile
}

// Main launch: every tile once, the maximum folded in, the output rounded
// with the shift of the previous call (none stored without a guess).
__global__ __launch_bounds__(ST) void igemm_small_main(IgemmProblem P, IgemmCtl ctl) {
    __shared__ __attribute__((aligned(16))) int32_t red[SW * 32 * RP];
    __shared__ uint32_t wmax[ST / 64];
    niti_stats* st = ctl.stats;
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    const int hint = st->bp_hint;
    begin_call(st, slot, hint);
    const RoundK rk = make_round(hint < 0 ? 0 : hint, ctl.mode);
    uint32_t tmax = 0;
    small_tile(P, blockIdx.x, red, rk, ctl.relu, hint >= 0, true, tmax);
    block_publish_max32(st, slot, tmax, wmax, snap);  // magnitudes <= 2^31
}

// Fix-up launch: with the final maximum, recompute every tile when the
// guessed shift was wrong; workgroup 0 then finalizes the statistics.
__global__ __launch_bounds__(ST) void igemm_small_fixup(IgemmProblem P, IgemmCtl ctl, int ntiles) {
    __shared__ __attribute__((aligned(16))) int32_t red[SW * 32 * RP];
    niti_stats* st = ctl.stats;
    const CallState cs = shared_call_state(st);
    const int hint = cs.hint;
    const int bp = block_bp(cs.mx, ctl.target);
    if (bp != hint) {
        const RoundK rk = make_round(bp, ctl.mode);
        uint32_t dummy = 0;
        for (int t = blockIdx.x; t < ntiles; t += gridDim.x) small_tile(P, t, red, rk, ctl.relu, true, false, dummy);
    }
    if (is_finisher()) finish_call(st, ctl.target, ctl.ex, ctl.static_flags, 1);
}

}  // namespace

// A single plain matrix product: 1 x 1 taps over an unpadded, unstrided
// input whose rows are the L-byte reduction vectors, written densely
// (row stride = Nout), with at most MAX_M rows and few 128 x 128 tiles.
bool igemm_small_eligible(const IgemmBatch& b) {
    if (b.nprob != 1) return false;
    const IgemmProblem& p = b.p[0];
    if (p.M < 1 || p.M > MAX_M || p.Nout < 1 || p.L < 0) return false;
    if (p.R != 1 || p.S != 1 || p.C != p.L || p.win) return false;
    if (p.H != p.OHc || p.W != p.OWc || p.st != 1 || p.off_h != 0 || p.off_w != 0) return false;
    if (p.OH != p.OHc || p.OW != p.OWc || p.os != 1 || p.oa != 0 || p.ob != 0) return false;
    if (p.ldo != p.Nout || p.zsib) return false;
    const int64_t tiles128 = (int64_t)((p.M + 127) / 128) * ((p.Nout + 127) / 128);
    return tiles128 < 64;
}

hipError_t igemm_small_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    const IgemmProblem& p = b.p[0];
    const int ntiles = ((p.M + 31) / 32) * ((p.Nout + 31) / 32);
    const int tk = timing_begin(NITI_TIMING_KERNEL, stream, "igemm_small_main");
    hipLaunchKernelGGL(igemm_small_main, dim3(ntiles), dim3(ST), 0, stream, p, ctl);
    timing_end(tk, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int fix_grid = ntiles < kFixupGrid ? ntiles : kFixupGrid;
    hipLaunchKernelGGL(igemm_small_fixup, dim3(fix_grid), dim3(ST), 0, stream, p, ctl, ntiles);
    return hipGetLastError();
}

}  // namespace niti
