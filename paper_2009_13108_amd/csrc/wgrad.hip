// Weight-gradient contraction g32 = a(l-1) (x) e(l) (Algorithm 1; Section
// 3.3) on int8 MFMA.
//
//   g32[k][r][s*C + c] = sum over pixels (n, p, q) of
//                        dy[n][p][q][k] * x[n][p*sh - ph + r][q*sw - pw + s][c]
//
// The reduction runs over the N*P*Q output pixels, far longer than the
// output, so the pixel range may be split across workgroups: each group
// stores its partial tile to its own slice, and a bandwidth pass sums the
// slices (exact mod 2^32, independent of the split) while taking the
// tensor maximum.
//
// Both operands arrive pixel-major from NHWC memory (channels contiguous)
// while the MFMA wants each lane's 16 bytes along the reduction (pixels).
// Each thread therefore loads four pixels' dwords, transposes the 4x4 byte
// block in registers (v_perm_b32) and writes pixel-contiguous dwords into
// LDS; the MFMA fragments are then plain 16-byte LDS reads.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int BKP = 64;     // pixels per main-loop step
constexpr int PITCH = 80;   // LDS row pitch in bytes (64 + 16 pad)
constexpr int NTHREADS = 256;

// 4x4 byte transpose: in[i] holds bytes (row i, col 0..3); out[b] holds
// bytes (row 0..3, col b).
__device__ __forceinline__ void transpose4x4(const uint32_t in[4], uint32_t out[4]) {
    const uint32_t t0 = __builtin_amdgcn_perm(in[1], in[0], 0x05010400u);
    const uint32_t t1 = __builtin_amdgcn_perm(in[1], in[0], 0x07030602u);
    const uint32_t t2 = __builtin_amdgcn_perm(in[3], in[2], 0x05010400u);
    const uint32_t t3 = __builtin_amdgcn_perm(in[3], in[2], 0x07030602u);
    out[0] = __builtin_amdgcn_perm(t2, t0, 0x05040100u);
    out[1] = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    out[2] = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    out[3] = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

struct PixPos {
    int n, p, q;
};

__device__ __forceinline__ PixPos decode_pix(const WgradProblem& P, int pix) {
    PixPos r;
    r.n = (int)fdiv((uint32_t)pix, P.div_pq);
    const int rem = pix - r.n * P.P * P.Q;
    r.p = (int)fdiv((uint32_t)rem, P.div_q);
    r.q = rem - r.p * P.Q;
    return r;
}

__device__ __forceinline__ void next_pix(const WgradProblem& P, PixPos& x) {
    if (++x.q == P.Q) {
        x.q = 0;
        if (++x.p == P.P) {
            x.p = 0;
            ++x.n;
        }
    }
}

template <int TBK, int TBC>
__global__ __launch_bounds__(NTHREADS) void wgrad_kernel(WgradProblem P) {
    constexpr int WTK = TBK / 2, WTC = TBC / 2;
    constexpr int FK = WTK / 32, FC = WTC / 32;
    constexpr int XCD = TBC / 4;                 // column dwords per pixel row of the x tile
    constexpr int XGP = NTHREADS / XCD;          // 4-pixel groups per pass (x)
    constexpr int XPASS = (BKP / 4) / XGP;       // passes over the 16 pixel groups
    constexpr int DKD = TBK / 4;
    constexpr int DGP = NTHREADS / DKD;
    constexpr int DPASS = (BKP / 4) / DGP;

    __shared__ int8_t xs[2][TBC * PITCH];
    __shared__ int8_t ds[2][TBK * PITCH];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wk = wave & 1, wc = wave >> 1;
    const int c0 = blockIdx.x * TBC;
    const int k0 = blockIdx.y * TBK;
    const int pbeg = blockIdx.z * P.chunk;
    const int pend = min(P.npix, pbeg + P.chunk);

    // This thread's x column dword (fixed over the whole reduction).
    const int xcd = threadIdx.x % XCD, xg = threadIdx.x / XCD;
    const int col = c0 + 4 * xcd;
    const bool col_ok = col < P.ncol;
    int cr = 0, cs = 0, cc = 0;
    if (col_ok) {
        cr = (int)fdiv((uint32_t)col, P.div_l);
        const int j = col - cr * P.L;
        cs = (int)fdiv((uint32_t)j, P.div_c);
        cc = j - cs * P.C;
    }
    // This thread's dy channel dword.
    const int dkd = threadIdx.x % DKD, dg = threadIdx.x / DKD;
    const int kch = k0 + 4 * dkd;
    const bool k_ok = kch < P.K;  // K % 4 == 0 is not required: tail handled bytewise

    uint32_t xr[XPASS][4], dr[DPASS][4];

    auto gload = [&](int pix0) {
#pragma unroll
        for (int ps = 0; ps < XPASS; ps++) {
            const int pb = pix0 + 4 * (xg + ps * XGP);
            PixPos pp = decode_pix(P, pb < P.npix ? pb : 0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                uint32_t v = 0;
                const int pix = pb + i;
                if (col_ok && pix < pend) {
                    const int h = pp.p * P.sh - P.ph + cr;
                    const int w = pp.q * P.sw - P.pw + cs;
                    if ((unsigned)h < (unsigned)P.H && (unsigned)w < (unsigned)P.W)
                        v = *(const uint32_t*)(P.x + (((int64_t)pp.n * P.H + h) * P.W + w) * P.C + cc);
                }
                xr[ps][i] = v;
                next_pix(P, pp);
            }
        }
#pragma unroll
        for (int ps = 0; ps < DPASS; ps++) {
            const int pb = pix0 + 4 * (dg + ps * DGP);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                uint32_t v = 0;
                const int pix = pb + i;
                if (k_ok && pix < pend) {
                    const int8_t* src = P.dy + (int64_t)pix * P.K + kch;
                    if (kch + 4 <= P.K && (((uintptr_t)src) & 3) == 0) {
                        v = *(const uint32_t*)src;
                    } else {
                        for (int b = 0; b < 4 && kch + b < P.K; b++)
                            v |= (uint32_t)(uint8_t)src[b] << (8 * b);
                    }
                }
                dr[ps][i] = v;
            }
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int ps = 0; ps < XPASS; ps++) {
            uint32_t t[4];
            transpose4x4(xr[ps], t);
            const int pg = xg + ps * XGP;
#pragma unroll
            for (int b = 0; b < 4; b++) *(uint32_t*)&xs[buf][(4 * xcd + b) * PITCH + 4 * pg] = t[b];
        }
#pragma unroll
        for (int ps = 0; ps < DPASS; ps++) {
            uint32_t t[4];
            transpose4x4(dr[ps], t);
            const int pg = dg + ps * DGP;
#pragma unroll
            for (int b = 0; b < 4; b++) *(uint32_t*)&ds[buf][(4 * dkd + b) * PITCH + 4 * pg] = t[b];
        }
    };

    v16i acc[FC][FK];
#pragma unroll
    for (int a = 0; a < FC; a++)
#pragma unroll
        for (int b = 0; b < FK; b++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[a][b][e] = 0;

    const int nsteps = pend > pbeg ? (pend - pbeg + BKP - 1) / BKP : 0;
    gload(pbeg);
    sstore(0);
    __syncthreads();
    for (int it = 0; it < nsteps; it++) {
        const int buf = it & 1;
        if (it + 1 < nsteps) gload(pbeg + (it + 1) * BKP);
#pragma unroll
        for (int ks = 0; ks < 2; ks++) {
            const int koff = ks * 32 + (lane >> 5) * 16;
            v4i fa[FC], fb[FK];
#pragma unroll
            for (int a = 0; a < FC; a++)
                fa[a] = *(const v4i*)&xs[buf][(wc * WTC + a * 32 + (lane & 31)) * PITCH + koff];
#pragma unroll
            for (int b = 0; b < FK; b++)
                fb[b] = *(const v4i*)&ds[buf][(wk * WTK + b * 32 + (lane & 31)) * PITCH + koff];
#pragma unroll
            for (int a = 0; a < FC; a++)
#pragma unroll
                for (int b = 0; b < FK; b++)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
        }
        if (it + 1 < nsteps) sstore(buf ^ 1);
        __syncthreads();
    }

    // acc[a][b] element 4*jj + i: column c0 + wc*WTC + a*32 + 8*jj + 4*(lane/32) + i,
    // channel k0 + wk*WTK + b*32 + lane%32: four consecutive columns per store.
    int32_t* out = P.part + (int64_t)blockIdx.z * P.K * P.ncol;
#pragma unroll
    for (int b = 0; b < FK; b++) {
        const int k = k0 + wk * WTK + b * 32 + (lane & 31);
        if (k >= P.K) continue;
        int32_t* grow = out + (int64_t)k * P.ncol;
#pragma unroll
        for (int a = 0; a < FC; a++)
#pragma unroll
            for (int jj = 0; jj < 4; jj++) {
                const int cidx = c0 + wc * WTC + a * 32 + 8 * jj + 4 * (lane >> 5);
                if (cidx >= P.ncol) continue;
                int32_t* dst = grow + cidx;
                if ((((uintptr_t)dst) & 15) == 0 && cidx + 4 <= P.ncol) {
                    *(int4*)dst = make_int4(acc[a][b][4 * jj], acc[a][b][4 * jj + 1], acc[a][b][4 * jj + 2],
                                            acc[a][b][4 * jj + 3]);
                } else {
                    for (int i = 0; i < 4 && cidx + i < P.ncol; i++) dst[i] = acc[a][b][4 * jj + i];
                }
            }
    }
}

template <int TBK, int TBC>
hipError_t launch_wgrad(const WgradProblem& p, const WgradPlan& plan, hipStream_t stream) {
    const int tc = (p.ncol + TBC - 1) / TBC;
    const int tk = (p.K + TBK - 1) / TBK;
    const int t = timing_on()
                      ? timing_begin(NITI_TIMING_KERNEL, stream, kernel_label("wgrad_kernel<%d,%d>", TBK, TBC))
                      : -1;
    hipLaunchKernelGGL((wgrad_kernel<TBK, TBC>), dim3(tc, tk, plan.splits), dim3(NTHREADS), 0, stream, p);
    timing_end(t, stream);
    return hipGetLastError();
}

}  // namespace

// Split of the pixel reduction: about `groups` workgroups in all, but at
// least 8 steps of 64 pixels per workgroup.
WgradPlan wgrad_plan(int64_t K, int64_t ncol, int64_t npix, int64_t groups) {
    WgradPlan pl;
    pl.tbk = K <= 64 ? 64 : 128;
    const int64_t tiles = ((K + pl.tbk - 1) / pl.tbk) * ((ncol + 127) / 128);
    const int64_t steps = (npix + BKP - 1) / BKP;
    int64_t splits = (groups + tiles - 1) / tiles;
    const int64_t max_splits = steps / 8 > 1 ? steps / 8 : 1;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    const int64_t chunk_steps = (steps + splits - 1) / splits;
    pl.chunk = (int32_t)(chunk_steps * BKP);
    pl.splits = (int32_t)((steps + chunk_steps - 1) / chunk_steps);
    if (pl.splits < 1) pl.splits = 1;
    return pl;
}

hipError_t wgrad_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream) {
    p.chunk = plan.chunk;
    if (plan.tbk == 64) return launch_wgrad<64, 128>(p, plan, stream);
    return launch_wgrad<128, 128>(p, plan, stream);
}

}  // namespace niti
