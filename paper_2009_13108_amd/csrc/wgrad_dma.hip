// Weight-gradient contraction g32 = a(l-1) (x) e(l) (Algorithm 1; Section
// 3.3) with a DMA-fed LDS ring and LDS transpose reads, for layers whose
// channel counts are multiples of 16 (the general path is wgrad.hip).
//
//   g32[k][col] = sum over pixels pix of dy[pix][k] * X[pix][col],
//   col = (r*S + s)*C + c,  X[pix][col] = x[n][oh*sh - ph + r][ow*sw - pw + s][c]
//
// Both operands are stored in LDS pixel-major, exactly as they arrive from
// NHWC memory (a row per pixel: 128 columns or 64/128 channels, 16-byte
// chunks XOR-swizzled by pixel).  The MFMA wants each lane's 16 bytes along
// the reduction (pixels); ds_read_b64_tr_b8 delivers that directly: within a
// group of 16 lanes that each address 8 bytes of a pixel row, lane i < 8
// receives byte i of the even lanes' rows and lane 8 + i byte i of the odd
// lanes' rows.  With lanes 2q and 2q+1 addressing the two 8-byte halves of
// pixel row q, every lane gets one column over 8 pixels; two such reads give
// the 16 pixel bytes of a 32x32x32 fragment lane.
//
// Each workgroup reduces one pixel range for one output tile and stores the
// partial tile to its own slice; a bandwidth pass sums the slices.
//
// Window mode (few channels, S*C <= 64): x is a zero-padded copy of the
// input, and a filter row (r) is one window of Lw bytes (S pixels and zero
// columns past them), so column col = r*Lw + j of X is x_pad at pixel row
// oh*sh + r, byte (ow*sw)*C + j: always in bounds.  Only columns with j <
// S*C are stored, compacted to r*S*C + j.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int PIX = 64;                 // pixels per stage
constexpr uint32_t kOOB = 0x80000000u;

typedef __attribute__((address_space(3))) v2i lds_v2i;

template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Swizzle of a pixel row's 16-byte chunks: conflict-free transpose reads
// over 8 consecutive pixels for 128-byte rows and 64-byte rows.
template <int RB>
__device__ __forceinline__ int swz(int pix) {
    return RB == 128 ? (pix & 7) : ((pix >> 1) & 3);
}

template <int TBK, int TBC, int NS>
struct WCfg {
    static constexpr int XBLK = TBC * PIX / 1024;      // 1 KiB blocks of the X tile per stage
    static constexpr int DBLK = TBK * PIX / 1024;      // blocks of the dy tile
    static constexpr int BLOCKS = XBLK + DBLK;
    static constexpr int IPW = BLOCKS / 4;
    static constexpr int XBYTES = TBC * PIX;
    static constexpr int STAGE = (TBC + TBK) * PIX;
    static constexpr int LDS = NS * STAGE;
    static constexpr int WTK = TBK / 2, WTC = TBC / 2;  // 2 x 2 waves
    static constexpr int FK = WTK / 32, FC = WTC / 32;
    static_assert(BLOCKS % 4 == 0, "blocks per wave");
};

// One 32 x 32-pixel fragment from a pixel-major region with RB-byte rows:
// lane gets 16 pixel bytes (pixels p0 + 16*(lane/32) ...) of column cbase + lane%32.
template <int RB>
__device__ __forceinline__ v4i tr_fragment(const int8_t* region, int p0, int cbase, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int col0 = cbase + 16 * (g & 1);            // 16-column group of this lane group
    const int chunk = col0 >> 4;
    const int prow = p0 + 16 * (g >> 1) + (j >> 1);   // pixel row this lane addresses
    const int half = (j & 1) * 8;
    const int8_t* a0 = region + prow * RB + ((chunk ^ swz<RB>(prow)) << 4) + half;
    const int8_t* a1 = region + (prow + 8) * RB + ((chunk ^ swz<RB>(prow + 8)) << 4) + half;
    const v2i lo = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)a0);
    const v2i hi = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)a1);
    v4i r;
    r[0] = lo[0];
    r[1] = lo[1];
    r[2] = hi[0];
    r[3] = hi[1];
    return r;
}

// Workgroup order.  Workgroups go to the eight XCDs (each with its own L2)
// in turn by linear index, so workgroup L runs on XCD L % 8.  The work items
// (split, tile), tile fastest, are cut into eight equal consecutive runs, one
// per XCD: the output tiles of one pixel range, which read the same input
// pixels (shifted per tap) and the same errors, then mostly share an XCD and
// meet in its L2, and every XCD gets the same amount of work.
template <int TBK, int TBC, int NS>
__global__ __launch_bounds__(256, 1) void wgrad_dma_kernel(WgradProblem P, int tiles_c, int tiles_k, int splits) {
    using T = WCfg<TBK, TBC, NS>;
    extern __shared__ __attribute__((aligned(1024))) int8_t lds[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wk = wave & 1, wc = wave >> 1;
    const int ntiles = tiles_c * tiles_k;
    const int per_xcd = (ntiles * splits + 7) / 8;
    const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if ((blockIdx.x >> 3) >= per_xcd || item >= ntiles * splits) return;
    const int split = item / ntiles;
    const int tile = item - split * ntiles;
    const int c0 = (tile % tiles_c) * TBC;
    const int k0 = (tile / tiles_c) * TBK;
    const int pbeg = split * P.chunk;
    const int pend = min(P.npix, pbeg + P.chunk);
    const int nsteps = pend > pbeg ? (pend - pbeg + PIX - 1) / PIX : 0;

    // Loads go out as inline assembly (lds_dma16): with the load builtin the
    // compiler waits for the whole ring before every transpose read.
    const u32x4 xrs = raw_rsrc(P.x, (uint32_t)P.x_bytes);
    const u32x4 drs = raw_rsrc(P.dy, (uint32_t)P.dy_bytes);
    const uint32_t lds0 = lds_address(lds);

    // Per load instruction: pixel row within the stage, and the column /
    // channel this lane's chunk covers (fixed over the reduction).
    int prow[T::IPW];
    int tdh[T::IPW], tdw[T::IPW];   // X: tap displacement (r - ph, s - pw); dy: unused
    uint32_t toff[T::IPW];          // X: channel offset c; dy: channel k
    bool cok[T::IPW];
#pragma unroll
    for (int i = 0; i < T::IPW; i++) {
        const int blk = wave * T::IPW + i;   // uniform
        if (blk < T::XBLK) {
            // 128-byte rows: 8 pixels x 8 chunks per block
            const int p = blk * 8 + (lane >> 3);
            const int chunk = (lane & 7) ^ swz<TBC>(p);
            const int col = c0 + 16 * chunk;
            prow[i] = p;
            if (P.win) {
                cok[i] = col < P.ncol_w;
                const int cc = cok[i] ? col : 0;
                const int r = cc / P.Lw;
                tdh[i] = 0;
                tdw[i] = 0;
                toff[i] = (uint32_t)(r * P.W * P.C + (cc - r * P.Lw));
            } else {
                cok[i] = col < P.ncol;
                const int cc = cok[i] ? col : 0;
                const int r = (int)fdiv((uint32_t)cc, P.div_l);
                const int jj = cc - r * P.L;
                const int s = (int)fdiv((uint32_t)jj, P.div_c);
                tdh[i] = r - P.ph;
                tdw[i] = s - P.pw;
                toff[i] = (uint32_t)(jj - s * P.C);
            }
        } else {
            const int b = blk - T::XBLK;
            constexpr int PPB = 1024 / TBK;          // pixels per block
            constexpr int CPR = TBK / 16;            // chunks per row
            const int p = b * PPB + lane / CPR;
            const int chunk = (lane % CPR) ^ swz<TBK>(p);
            const int k = k0 + 16 * chunk;
            prow[i] = p;
            cok[i] = k < P.K;
            tdh[i] = 0;
            tdw[i] = 0;
            toff[i] = (uint32_t)k;
        }
    }

    int next = 0;
    auto issue = [&]() {
        const uint32_t st = lds0 + (uint32_t)((next % NS) * T::STAGE);
        const int pb = pbeg + next * PIX;
#pragma unroll
        for (int i = 0; i < T::IPW; i++) {
            const int blk = wave * T::IPW + i;
            const int pix = pb + prow[i];
            const bool pok = next < nsteps && pix < pend && cok[i];
            uint32_t off = kOOB;
            if (blk < T::XBLK) {
                if (pok) {
                    const int n = (int)fdiv((uint32_t)pix, P.div_pq);
                    const int rem = pix - n * P.P * P.Q;
                    const int oh = (int)fdiv((uint32_t)rem, P.div_q);
                    const int ow = rem - oh * P.Q;
                    const int ih = oh * P.sh + tdh[i];
                    const int iw = ow * P.sw + tdw[i];
                    if (P.win || ((unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W))
                        off = (uint32_t)(((n * P.H + ih) * P.W + iw) * P.C) + toff[i];
                }
                lds_dma16(xrs, st + blk * 1024, off, 0);
            } else {
                if (pok) off = (uint32_t)pix * (uint32_t)P.K + toff[i];
                lds_dma16(drs, st + blk * 1024, off, 0);
            }
        }
        next++;
    };

    v16i acc[T::FC][T::FK];
#pragma unroll
    for (int a = 0; a < T::FC; a++)
#pragma unroll
        for (int b = 0; b < T::FK; b++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[a][b][e] = 0;

#pragma unroll
    for (int s = 0; s < NS - 1; s++) issue();
    for (int it = 0; it < nsteps; it++) {
        wait_vm<(NS - 2) * T::IPW>();
        __builtin_amdgcn_s_barrier();
        issue();
        const int8_t* st = lds + (it % NS) * T::STAGE;
#pragma unroll
        for (int ks = 0; ks < 2; ks++) {
            v4i fa[T::FC], fb[T::FK];
#pragma unroll
            for (int a = 0; a < T::FC; a++) fa[a] = tr_fragment<TBC>(st, 32 * ks, wc * T::WTC + a * 32, lane);
#pragma unroll
            for (int b = 0; b < T::FK; b++)
                fb[b] = tr_fragment<TBK>(st + T::XBYTES, 32 * ks, wk * T::WTK + b * 32, lane);
#pragma unroll
            for (int a = 0; a < T::FC; a++)
#pragma unroll
                for (int b = 0; b < T::FK; b++)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
        }
    }
    wait_vm<0>();

    // acc[a][b] element 4*jj + i: column c0 + wc*WTC + a*32 + 8*jj + 4*(lane/32) + i,
    // channel k0 + wk*WTK + b*32 + lane%32: four consecutive columns per store.
    int32_t* out = P.part + (int64_t)split * P.K * P.ncol;
#pragma unroll
    for (int b = 0; b < T::FK; b++) {
        const int k = k0 + wk * T::WTK + b * 32 + (lane & 31);
        if (k >= P.K) continue;
        int32_t* grow = out + (int64_t)k * P.ncol;
#pragma unroll
        for (int a = 0; a < T::FC; a++)
#pragma unroll
            for (int jj = 0; jj < 4; jj++) {
                int cidx = c0 + wc * T::WTC + a * 32 + 8 * jj + 4 * (lane >> 5);
                if (P.win) {
                    // window column r*Lw + j -> stored column r*L + j, j < L (groups of 4 stay whole)
                    if (cidx >= P.ncol_w) continue;
                    const int r = cidx / P.Lw, j = cidx - r * P.Lw;
                    if (j >= P.L) continue;
                    cidx = r * P.L + j;
                }
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

template <int TBK, int TBC, int NS>
hipError_t launch(const WgradProblem& p, const WgradPlan& plan, hipStream_t stream) {
    using T = WCfg<TBK, TBC, NS>;
    static bool attr_done = false;
    if (!attr_done) {
        hipError_t e = hipFuncSetAttribute((const void*)wgrad_dma_kernel<TBK, TBC, NS>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS);
        if (e != hipSuccess) return e;
        attr_done = true;
    }
    const int tc = ((p.win ? p.ncol_w : p.ncol) + TBC - 1) / TBC;
    const int tk = (p.K + TBK - 1) / TBK;
    const int64_t grid = (int64_t)8 * (((int64_t)tc * tk * plan.splits + 7) / 8);
    const int t = timing_on() ? timing_begin(NITI_TIMING_KERNEL, stream,
                                             kernel_label("wgrad_dma_kernel<%d,%d,%d>", TBK, TBC, NS))
                              : -1;
    hipLaunchKernelGGL((wgrad_dma_kernel<TBK, TBC, NS>), dim3((unsigned)grid), dim3(256), T::LDS, stream, p, tc, tk,
                       plan.splits);
    timing_end(t, stream);
    return hipGetLastError();
}

}  // namespace

bool wgrad_dma_eligible(const WgradProblem& p) {
    const bool cols = p.win ? (p.Lw % 16 == 0 && p.L % 4 == 0 && p.ph == 0 && p.pw == 0) : p.C % 16 == 0;
    return cols && p.K % 16 == 0 && p.x_bytes > 0 && p.x_bytes < ((int64_t)1 << 31) && p.dy_bytes > 0 &&
           p.dy_bytes < ((int64_t)1 << 31);
}

hipError_t wgrad_dma_run(WgradProblem& p, const WgradPlan& plan, hipStream_t stream) {
    p.chunk = plan.chunk;
    if (plan.tbk == 64) return launch<64, 128, 4>(p, plan, stream);
    return launch<128, 128, 4>(p, plan, stream);
}

}  // namespace niti
