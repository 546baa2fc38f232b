// Implicit-GEMM int8 MFMA kernel with a multi-stage LDS ring filled by
// direct-to-LDS buffer loads (gfx950 buffer_load_dwordx4 ... lds).  Same
// problem form, epilogue and exponent speculation as igemm.hip, which keeps
// the general path (odd channel counts such as a 4-channel image layer).
//
// Two load modes keep the per-step address work uniform:
//   kGemm   plain matrix rows (H = W = 1, one tap): a lane's offset is fixed
//           and the K step adds a uniform amount;
//   kConv64 convolutions with C % 64 == 0: every 64-byte K step lies in one
//           filter tap (r, s) and channel block c0, all uniform, so a lane
//           only checks that its pixel's tap is inside the image;
//   kWin    convolutions with few channels (S*C <= 64) over a zero-padded
//           copy of the input: a filter row is one contiguous window of
//           L = 16, 32 or 64 bytes (S pixels, zero weights past them), a K
//           step covers 64/L filter rows, and every window is in bounds, so
//           a lane's offset is fixed and the step adds a uniform amount.
//
// Loads.  Each wave instruction moves 64 lanes x 16 bytes into one 1 KiB LDS
// block (lane l lands at block + 16 l); a block holds 16 operand rows of one
// 64-byte K step.  A lane whose piece is outside the image, past the tensor
// or past K uses an offset beyond the buffer's size, which the hardware
// answers with zeros.  Within a row the four 16-byte chunks are stored
// XOR-swizzled (position = chunk ^ f(row)) so the 32x32x32 MFMA fragment
// reads (16 bytes per lane, 8 lanes per bank cycle) hit distinct banks.
//
// Pipeline.  NS stages; stage k+NS-1 is issued while stage k is computed.
// Loads past the last K step are issued anyway (as zeros), so the wait
// count before each step is a constant.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int KSTEP = 64;  // K bytes per stage
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kGemm = 0;
constexpr int kConv64 = 1;
constexpr int kWin = 2;

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ (row >> 2)) & 3; }

template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// vmcnt <= N and lgkmcnt == 0 (this wave's LDS reads done).
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
    static_assert(N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0070);
}

template <int BM, int BN, int NS, int WGM, int WGN>
struct Cfg {
    static constexpr int NWAVES = WGM * WGN;
    static constexpr int NT = 64 * NWAVES;
    static constexpr int WTM = BM / WGM, WTN = BN / WGN;   // wave tile: pixels x channels
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int BLOCKS = (BM + BN) / 16;           // 1 KiB blocks per stage
    static constexpr int ABLK = BN / 16;                    // blocks holding weight rows
    // Weight blocks per wave: ABLK / NWAVES each, or (fewer blocks than
    // waves) one each for waves 0 .. ABLK-1.
    static constexpr bool W_EVEN = ABLK % NWAVES == 0;
    static constexpr int IPW_W = W_EVEN ? ABLK / NWAVES : 1;
    static constexpr int IPW_A = (BLOCKS - ABLK) / NWAVES;  // activation blocks per wave
    static_assert((BLOCKS - ABLK) % NWAVES == 0 && (W_EVEN || ABLK < NWAVES), "load split over waves");
    static constexpr int STAGE_BYTES = (BM + BN) * KSTEP;
    static constexpr int LDS_BYTES = NS * STAGE_BYTES;
    static constexpr int WGM_ = WGM, BN_ = BN;
    static_assert(BM * (BN + 16) <= LDS_BYTES, "output tile fits in the ring");
};

// Round one accumulator (Algorithm 3 in the closed form of niti_device.h,
// or nearest) with the tile's uniform shift; RELU: v is already
// non-negative.  Magnitudes are at most 2^31, so the 32-bit maximum is
// exact.  Returns the int8 in the low byte.
template <bool RELU, bool RTN>
__device__ __forceinline__ uint32_t round_acc(int32_t v, const RoundK& k, uint32_t& tmax) {
    const uint32_t x = RELU ? (uint32_t)v : (v < 0 ? 0u - (uint32_t)v : (uint32_t)v);
    tmax = x > tmax ? x : tmax;
    uint32_t q;
    if (RTN) {
        q = x >> k.bp;
        q = min(q + (k.bp ? __builtin_amdgcn_ubfe(x, k.bp - 1, 1) : 0u), 127u);
    } else {
        q = round_psr_mag_fast(x, k);
    }
    if (RELU) return q;
    const uint32_t sgn = (uint32_t)(v >> 31);
    return ((q ^ sgn) - sgn) & 0xFFu;
}

// Tile maximum and rounded bytes of the register accumulators; the bytes go
// to an LDS tile [BM][BN + 16] (row = tile pixel).
template <typename T, bool RELU, bool RTN>
__device__ __forceinline__ void epilogue_regs(v16i (&acc)[T::FN][T::FM], int8_t* lds, const RoundK& rk,
                                              int do_store, int do_max, uint64_t& tmax) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % T::WGM_, wn = wave / T::WGM_;
    constexpr int PITCH = T::BN_ + 16;
    uint32_t mx = 0;
#pragma unroll
    for (int b = 0; b < T::FM; b++) {
        const int row = wm * T::WTM + b * 32 + (lane & 31);
#pragma unroll
        for (int a = 0; a < T::FN; a++)
#pragma unroll
            for (int jj = 0; jj < 4; jj++) {
                uint32_t packed = 0;
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    int32_t v = acc[a][b][4 * jj + i];
                    if (RELU) v = v < 0 ? 0 : v;
                    packed |= round_acc<RELU, RTN>(v, rk, mx) << (8 * i);
                }
                if (do_store) {
                    const int col = wn * T::WTN + a * 32 + 8 * jj + 4 * (lane >> 5);
                    *(uint32_t*)(lds + row * PITCH + col) = packed;
                }
            }
    }
    if (do_max) tmax = (uint64_t)mx > tmax ? (uint64_t)mx : tmax;
}

// Out-of-tile accumulators are zero (their operand rows were zero-filled),
// so including them in the maximum is harmless.  The LDS tile is written to
// the output in 16-byte row pieces, with the backward ReLU mask applied.
template <typename T, int BM, int BN>
__device__ __forceinline__ void store_tile(const IgemmProblem& P, int tm, int tn, const int8_t* lds) {
    constexpr int PITCH = BN + 16;
    constexpr int PPR = BN / 16;  // pieces per row
    const bool dense = P.os == 1 && P.OHc == P.OH && P.OWc == P.OW;
    for (int idx = threadIdx.x; idx < BM * PPR; idx += T::NT) {
        const int row = idx / PPR, pc = idx - row * PPR;
        const int m = tm * BM + row;
        const int n0 = tn * BN + pc * 16;
        if (m >= P.M || n0 >= P.Nout) continue;
        int64_t ooff;
        const int nv = min(16, P.Nout - n0);
        if (dense) {
            ooff = (int64_t)m * P.ldo + n0;   // the output grid is the pixel grid
        } else {
            const uint32_t img = fdiv((uint32_t)m, P.div_ohw);
            const uint32_t rem = (uint32_t)m - img * (uint32_t)(P.OHc * P.OWc);
            const uint32_t i0 = fdiv(rem, P.div_ow);
            const uint32_t j0 = rem - i0 * (uint32_t)P.OWc;
            const int oh = (int)i0 * P.os + P.oa;
            const int ow = (int)j0 * P.os + P.ob;
            ooff = (((int64_t)img * P.OH + oh) * P.OW + ow) * P.ldo + n0;
            if (P.zsib) store_zero_siblings(P, ooff, zero_siblings(P, oh, ow), nv);
        }
        uint4 v = *(const uint4*)(lds + row * PITCH + pc * 16);
        int8_t* dst = P.out + ooff;
        const bool full = nv == 16 && (((uintptr_t)dst) & 15) == 0;
        if (P.mask) {
            const int8_t* ms = P.mask + ooff;
            uint32_t mw[4];
            if (full) {
                const uint4 mv = *(const uint4*)ms;
                mw[0] = mv.x; mw[1] = mv.y; mw[2] = mv.z; mw[3] = mv.w;
            } else {
                for (int q = 0; q < 4; q++) mw[q] = 0;
                for (int e = 0; e < nv; e++) mw[e >> 2] |= (uint32_t)(uint8_t)ms[e] << (8 * (e & 3));
            }
            uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int q = 0; q < 4; q++) vw[q] &= positive_bytes(mw[q]);
            v = make_uint4(vw[0], vw[1], vw[2], vw[3]);
        }
        if (full) {
            *(uint4*)dst = v;
        } else {
            const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
            for (int e = 0; e < nv; e++) dst[e] = (int8_t)(vw[e >> 2] >> (8 * (e & 3)));
        }
    }
}

template <int BM, int BN, int NS, int WGM, int WGN, int MODE>
__device__ __forceinline__ void dma_tile(const IgemmProblem& P, int tm, int tn, int8_t* lds, const RoundK& rk,
                                         int relu, int do_store, int do_max, uint64_t& tmax, niti_stats* snap_st,
                                         int snap_slot, uint64_t& snap) {
    using T = Cfg<BM, BN, NS, WGM, WGN>;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % WGM, wn = wave / WGM;

    const u32x4 act_rs = raw_rsrc(P.act, (uint32_t)P.act_bytes);
    const u32x4 wgt_rs = raw_rsrc(P.wgt, (uint32_t)P.wgt_bytes);

    // Per-lane row state for each load instruction: a wave issues IPW_W
    // weight blocks and IPW_A activation blocks per stage; wb / ab is the
    // lane's byte offset at K step 0 (kOOB for a row past the operand).
    const int lrow = lane >> 2;
    const uint32_t kpo = (uint32_t)(((lane & 3) ^ swz(lrow)) << 4);  // byte offset of this lane's chunk
    uint32_t wb[T::IPW_W], ab[T::IPW_A];
    uint32_t aux[T::IPW_A];   // kConv64: taps (bit r*S+s) outside the image; kWin: filter row of the piece
    const bool wload = T::W_EVEN || wave < T::ABLK;   // this wave loads weight blocks (uniform)
    const int wblk0 = T::W_EVEN ? wave * T::IPW_W : wave;
#pragma unroll
    for (int i = 0; i < T::IPW_W; i++) {
        const int n = tn * BN + (wblk0 + i) * 16 + lrow;
        wb[i] = (wload && n < P.Nout) ? (uint32_t)n * (uint32_t)P.Ktot + kpo : kOOB;
    }
#pragma unroll
    for (int i = 0; i < T::IPW_A; i++) {
        const int m = tm * BM + (wave * T::IPW_A + i) * 16 + lrow;
        aux[i] = 0;
        if (MODE == kGemm) {
            ab[i] = m < P.M ? (uint32_t)m * (uint32_t)P.C + kpo : kOOB;
        } else {
            const uint32_t mm = m < P.M ? (uint32_t)m : 0u;
            const uint32_t img = fdiv(mm, P.div_ohw);
            const uint32_t rem = mm - img * (uint32_t)(P.OHc * P.OWc);
            const uint32_t oh = fdiv(rem, P.div_ow);
            const uint32_t ow = rem - oh * (uint32_t)P.OWc;
            if (MODE == kWin) {
                const int rr = (int)kpo / P.L;              // filter row of this piece within a step
                const int j0 = (int)kpo - rr * P.L;
                aux[i] = (uint32_t)rr;
                ab[i] = m < P.M ? (uint32_t)(((img * (uint32_t)P.H + oh * (uint32_t)P.st + (uint32_t)rr) *
                                                  (uint32_t)P.W + ow * (uint32_t)P.st) * (uint32_t)P.C) + (uint32_t)j0
                                : kOOB;
            } else {
                const int h0 = (int)oh * P.st + P.off_h;
                const int w0 = (int)ow * P.st + P.off_w;
                ab[i] = (uint32_t)((int64_t)img * P.H * P.W * P.C + ((int64_t)h0 * P.W + w0) * P.C) + kpo;
                // taps (r, s) whose input pixel lies outside the image (all of
                // them for a row past M)
                uint32_t rows = 0, cols = 0, valid = 0;
                for (int r = 0; r < P.R; r++) rows |= (uint32_t)((unsigned)(h0 + r) < (unsigned)P.H) << r;
                for (int c = 0; c < P.S; c++) cols |= (uint32_t)((unsigned)(w0 + c) < (unsigned)P.W) << c;
                for (int r = 0; r < P.R; r++)
                    if ((rows >> r) & 1u) valid |= cols << (r * P.S);
                aux[i] = m < P.M ? ~valid : ~0u;
            }
        }
    }

    const int nk = (P.Ktot + KSTEP - 1) / KSTEP;
    // Scalar instructions issue at about one per cycle per CU, shared by all
    // waves, so the load side keeps its per-step uniform work small: the
    // lanes' current offsets cvw / cva change only at events (a filter tap
    // change, the last K step, the end of K), counted down by ev; between
    // events a step adds to the two uniform offsets kb (weights, and kGemm
    // activations) and sa (kConv64: channel offset within the tap; kWin:
    // window row offset).  The uniform part of an offset rides in the
    // instruction's SGPR offset; every lane offset that is not kOOB stays
    // inside its buffer together with it, and lanes whose piece is past K,
    // past R or outside the image get kOOB (zeros).
    const uint32_t lds0 = lds_address(lds);
    uint32_t wdst[T::IPW_W], adst[T::IPW_A];   // this wave's blocks in stage 0
#pragma unroll
    for (int i = 0; i < T::IPW_W; i++) wdst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)(wblk0 + i) * 1024u);
#pragma unroll
    for (int i = 0; i < T::IPW_A; i++)
        adst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)(T::ABLK + wave * T::IPW_A + i) * 1024u);
    const int cbs = __builtin_amdgcn_readfirstlane(MODE == kConv64 ? P.C / KSTEP : 1);
    const int ntap = __builtin_amdgcn_readfirstlane(P.R * P.S);
    const uint32_t da = __builtin_amdgcn_readfirstlane(
        MODE == kWin ? (uint32_t)(KSTEP / P.L) * (uint32_t)(P.W * P.C) : (uint32_t)KSTEP);
    const uint32_t klim = __builtin_amdgcn_readfirstlane(
        MODE == kGemm ? (uint32_t)(P.Ktot - (nk - 1) * KSTEP) : (MODE == kWin ? (uint32_t)(P.R - (nk - 1) * (KSTEP / P.L)) : 0u));
    uint32_t kb = 0, sa = 0, tapbase = 0;
    int ev = 0, tap = 0, ts = 0, ph = 0;
    uint32_t cvw[T::IPW_W], cva[T::IPW_A];
#pragma unroll
    for (int i = 0; i < T::IPW_W; i++) cvw[i] = wb[i];
    auto set_tap = [&]() {
#pragma unroll
        for (int i = 0; i < T::IPW_A; i++) cva[i] = (__builtin_amdgcn_ubfe(aux[i], (uint32_t)tap, 1) << 31) | (ab[i] + tapbase);
    };
    // last K step (kGemm: pieces past K; kWin: rows past R masked)
    auto last_step = [&]() {
        ph = 1;
        ev = 1;
#pragma unroll
        for (int i = 0; i < T::IPW_W; i++) cvw[i] = (MODE == kGemm && kpo >= klim) ? kOOB : wb[i];
#pragma unroll
        for (int i = 0; i < T::IPW_A; i++) cva[i] = (MODE == kGemm ? kpo >= klim : aux[i] >= klim) ? kOOB : ab[i];
    };
#pragma unroll
    for (int i = 0; i < T::IPW_A; i++) cva[i] = ab[i];
    if (nk <= 0) {
        ph = 2;
        ev = 1 << 30;
    } else if (MODE == kConv64) {
        set_tap();
        ev = cbs;
    } else {
        ev = nk - 1;
        if (ev == 0) last_step();
    }
    // Events are handled at the start of the issue that follows them.
    auto advance = [&]() {
        if (MODE == kConv64 && tap + 1 < ntap) {
            ++tap;
            if (++ts == P.S) {
                ts = 0;
                tapbase += (uint32_t)((P.W - P.S + 1) * P.C);
            } else {
                tapbase += (uint32_t)P.C;
            }
            set_tap();
            sa = 0;
            ev = cbs;
            return;
        }
        if (MODE != kConv64 && ph == 0) {
            last_step();
            return;
        }
        // Past the end of K the loads go on unchanged (the buffer bounds
        // keep them harmless): they keep the wait counts constant, and the
        // stages they fill are never multiplied.
        tap = 1 << 30;
        ph = 2;
        ev = 1 << 30;
    };
    // issue(j): load K step j (ring slot j % NS)
    auto issue = [&](int j) {
        if (ev == 0) advance();
        const uint32_t slot = (uint32_t)(j % NS) * (uint32_t)T::STAGE_BYTES;
        if (wload) {
#pragma unroll
            for (int i = 0; i < T::IPW_W; i++) lds_dma16_at(wgt_rs, wdst[i], slot, cvw[i], kb);
        }
#pragma unroll
        for (int i = 0; i < T::IPW_A; i++) lds_dma16_at(act_rs, adst[i], slot, cva[i], MODE == kGemm ? kb : sa);
        kb += KSTEP;
        sa += da;
        ev = __builtin_amdgcn_readfirstlane(ev - 1);
    };

    v16i acc[T::FN][T::FM];
#pragma unroll
    for (int a = 0; a < T::FN; a++)
#pragma unroll
        for (int b = 0; b < T::FM; b++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[a][b][e] = 0;

    int a_off[T::FN], b_off[T::FM], a_sw[T::FN], b_sw[T::FM];
#pragma unroll
    for (int a = 0; a < T::FN; a++) {
        const int row = wn * T::WTN + a * 32 + (lane & 31);
        a_off[a] = row * KSTEP;
        a_sw[a] = swz(row & 15);
    }
#pragma unroll
    for (int b = 0; b < T::FM; b++) {
        const int row = wm * T::WTM + b * 32 + (lane & 31);
        b_off[b] = BN * KSTEP + row * KSTEP;
        b_sw[b] = swz(row & 15);
    }

#pragma unroll
    for (int s = 0; s < NS - 1; s++) issue(s);

    // Register double buffer over the two 32-byte halves of a K step: the
    // second half's fragments are read while the first half's MFMAs run, and
    // the next stage's first half right after the barrier, before this
    // stage's second-half MFMAs.  Before each barrier a wave waits for its
    // own fragment reads (lgkmcnt 0), so once all waves pass it no read of
    // the stage that the next load overwrites is still in flight.
    auto read_half = [&](const int8_t* st, int ks, v4i (&fa)[T::FN], v4i (&fb)[T::FM]) {
        const int kp = (lane >> 5) + 2 * ks;
#pragma unroll
        for (int a = 0; a < T::FN; a++) fa[a] = *(const v4i*)(st + a_off[a] + ((kp ^ a_sw[a]) << 4));
#pragma unroll
        for (int b = 0; b < T::FM; b++) fb[b] = *(const v4i*)(st + b_off[b] + ((kp ^ b_sw[b]) << 4));
    };
    auto mma_half = [&](const v4i (&fa)[T::FN], const v4i (&fb)[T::FM]) {
#pragma unroll
        for (int a = 0; a < T::FN; a++)
#pragma unroll
            for (int b = 0; b < T::FM; b++)
                acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[a], fb[b], acc[a][b], 0, 0, 0);
    };
    // Loads per stage of this wave (uniform): the stage-exact wait counts.
    constexpr int LW = T::IPW_A + T::IPW_W, LA = T::IPW_A;
    v4i fa0[T::FN], fb0[T::FM], fa1[T::FN], fb1[T::FM];
    if (wload)
        wait_vm<(NS - 2) * LW>();
    else
        wait_vm<(NS - 2) * LA>();
    __builtin_amdgcn_s_barrier();
    read_half(lds, 0, fa0, fb0);
    for (int kt = 0; kt < nk; kt++) {
        const int8_t* st = lds + (kt % NS) * T::STAGE_BYTES;
        issue(kt + NS - 1);   // into the slot of stage kt - 1, which every wave has finished reading
        read_half(st, 1, fa1, fb1);
        mma_half(fa0, fb0);
        // (after the last step this reads a stage loaded past the end of K,
        // which no MFMA uses: it keeps the loop free of branches)
        if (wload)
            wait_vm_lgkm0<(NS - 2) * LW>();
        else
            wait_vm_lgkm0<(NS - 2) * LA>();
        __builtin_amdgcn_s_barrier();
        read_half(lds + ((kt + 1) % NS) * T::STAGE_BYTES, 0, fa0, fb0);
        mma_half(fa1, fb1);
    }
    // Drain the loads issued past the end before the ring is reused.
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    // Snapshot of the tensor maximum for the skip test of the publishing
    // thread: read now, used after the epilogue, so its latency is hidden
    // and it includes the workgroups that finished meanwhile.
    if (snap_st && threadIdx.x == 0) snap = load_acc(snap_st, snap_slot);

    // Epilogue.  acc[a][b] element 4*jj + i is channel
    // wn*WTN + a*32 + 8*jj + 4*(lane/32) + i of tile pixel wm*WTM + b*32 + lane%32.
    // Rounded bytes go to the (drained) LDS ring as a [BM][BN] tile, then
    // leave in 16-byte row pieces.
    const int mode_sel = (relu ? 1 : 0) | (rk.rtn ? 2 : 0);
    switch (mode_sel) {
        case 0: epilogue_regs<T, false, false>(acc, lds, rk, do_store, do_max, tmax); break;
        case 1: epilogue_regs<T, true, false>(acc, lds, rk, do_store, do_max, tmax); break;
        case 2: epilogue_regs<T, false, true>(acc, lds, rk, do_store, do_max, tmax); break;
        default: epilogue_regs<T, true, true>(acc, lds, rk, do_store, do_max, tmax); break;
    }
    if (!do_store) return;
    __syncthreads();
    store_tile<T, BM, BN>(P, tm, tn, lds);
    __syncthreads();
}

__device__ __forceinline__ void locate(const IgemmBatch& b, int t, int& prob, int& tm, int& tn) {
    int p = 0;
#pragma unroll
    for (int i = 1; i < kMaxProblems; i++)
        if (i < b.nprob && t >= b.p[i].tile_base) p = i;
    const int local = t - b.p[p].tile_base;
    prob = p;
    tm = local / b.p[p].tiles_n;
    tn = local - tm * b.p[p].tiles_n;
}

template <int BM, int BN, int NS, int WGM, int WGN, int MODE>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void igemm_dma_main(IgemmBatch batch, IgemmCtl ctl) {
    extern __shared__ __attribute__((aligned(1024))) int8_t dyn_lds[];
    niti_stats* st = ctl.stats;
    const int slot = call_slot(st);
    uint64_t snap = 0;
    const int hint = st->bp_hint;
    begin_call(st, slot, hint);
    int prob, tm, tn;
    locate(batch, blockIdx.x, prob, tm, tn);
    const RoundK rk = make_round(hint < 0 ? 0 : hint, ctl.mode);
    uint64_t tmax = 0;
    dma_tile<BM, BN, NS, WGM, WGN, MODE>(batch.p[prob], tm, tn, dyn_lds, rk, ctl.relu, hint >= 0, 1, tmax, st, slot,
                                         snap);
    // Accumulator magnitudes are at most 2^31: 32-bit reductions are exact.
    // The ring is drained and the tile stored: its first bytes serve the
    // reduction (no static LDS, so two 80 KiB workgroups fit one CU).
    block_publish_max32(st, slot, (uint32_t)tmax, (uint32_t*)dyn_lds, snap);
}

template <int BM, int BN, int NS, int WGM, int WGN, int MODE>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void igemm_dma_fixup(IgemmBatch batch, IgemmCtl ctl) {
    extern __shared__ __attribute__((aligned(1024))) int8_t dyn_lds[];
    niti_stats* st = ctl.stats;
    const CallState cs = shared_call_state(st, dyn_lds);
    const int hint = cs.hint;
    const int bp = block_bp(cs.mx, ctl.target);
    if (bp != hint) {
        const RoundK rk = make_round(bp, ctl.mode);
        for (int t = blockIdx.x; t < batch.total_tiles; t += gridDim.x) {
            int prob, tm, tn;
            locate(batch, t, prob, tm, tn);
            uint64_t dummy = 0, nosnap = 0;
            dma_tile<BM, BN, NS, WGM, WGN, MODE>(batch.p[prob], tm, tn, dyn_lds, rk, ctl.relu, 1, 0, dummy, nullptr, 0,
                                                 nosnap);
        }
    }
    if (is_finisher()) finish_call(st, ctl.target, ctl.ex, ctl.static_flags, 1);
}

template <int BM, int BN, int NS, int WGM, int WGN, int MODE>
hipError_t launch_dma(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    using T = Cfg<BM, BN, NS, WGM, WGN>;
    static bool attr_done = false;
    if (!attr_done) {
        hipError_t e = hipFuncSetAttribute((const void*)igemm_dma_main<BM, BN, NS, WGM, WGN, MODE>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS_BYTES);
        if (e != hipSuccess) return e;
        e = hipFuncSetAttribute((const void*)igemm_dma_fixup<BM, BN, NS, WGM, WGN, MODE>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, T::LDS_BYTES);
        if (e != hipSuccess) return e;
        attr_done = true;
    }
    int base = 0;
    for (int i = 0; i < b.nprob; i++) {
        IgemmProblem& p = b.p[i];
        p.tiles_m = (p.M + BM - 1) / BM;
        p.tiles_n = (p.Nout + BN - 1) / BN;
        p.tile_base = base;
        base += p.tiles_m * p.tiles_n;
    }
    b.total_tiles = base;
    const int tk = timing_on() ? timing_begin(NITI_TIMING_KERNEL, stream,
                                              kernel_label("igemm_dma_main<%d,%d,%d,%d,%d,%d>", BM, BN, NS, WGM,
                                                           WGN, MODE))
                               : -1;
    hipLaunchKernelGGL((igemm_dma_main<BM, BN, NS, WGM, WGN, MODE>), dim3(base), dim3(T::NT), T::LDS_BYTES, stream,
                       b, ctl);
    timing_end(tk, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int fix_grid = base < kFixupGrid ? base : kFixupGrid;
    hipLaunchKernelGGL((igemm_dma_fixup<BM, BN, NS, WGM, WGN, MODE>), dim3(fix_grid), dim3(T::NT), T::LDS_BYTES,
                       stream, b, ctl);
    return hipGetLastError();
}

int problem_mode(const IgemmProblem& p) {
    if (p.win) return kWin;
    if (p.H == 1 && p.W == 1 && p.R == 1 && p.off_h == 0 && p.off_w == 0 && p.L == p.C) return kGemm;
    return kConv64;
}

template <int MODE>
hipError_t run_mode(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    int64_t work = 0;
    int maxN = 0;
    for (int i = 0; i < b.nprob; i++) {
        work += (int64_t)b.p[i].M * b.p[i].Nout;
        maxN = b.p[i].Nout > maxN ? b.p[i].Nout : maxN;
    }
    // The largest tile that still gives most compute units a workgroup.
    if (maxN <= 64) return launch_dma<256, 64, 4, 8, 1, MODE>(b, ctl, stream);
    // 128 x 128 with eight 32 x 64 waves: two workgroups per CU (256 x 128
    // fits one, by registers) and four waves per SIMD to hide each other's
    // LDS and barrier waits.
    if (maxN <= 128) return launch_dma<128, 128, 4, 4, 2, MODE>(b, ctl, stream);
    if (work >= (int64_t)200 * 256 * 256) return launch_dma<256, 256, 3, 2, 4, MODE>(b, ctl, stream);
    if (work >= (int64_t)200 * 256 * 128) return launch_dma<256, 128, 4, 2, 2, MODE>(b, ctl, stream);
    return launch_dma<128, 128, 4, 4, 2, MODE>(b, ctl, stream);
}

}  // namespace

// True when every problem has whole 16-byte pieces handled by one of the two
// load modes and both operands are addressable with 32-bit buffer offsets.
bool igemm_dma_eligible(const IgemmBatch& b) {
    int mode = -1;
    for (int i = 0; i < b.nprob; i++) {
        const IgemmProblem& p = b.p[i];
        if (p.act_bytes <= 0 || p.act_bytes >= ((int64_t)1 << 31) || p.wgt_bytes <= 0 ||
            p.wgt_bytes >= ((int64_t)1 << 31))
            return false;
        const int m = problem_mode(p);
        if (mode >= 0 && m != mode) return false;
        mode = m;
        if (m == kGemm) {
            if (p.C % 16 != 0 || p.Ktot != p.C) return false;
        } else if (m == kWin) {
            if ((p.L != 16 && p.L != 32 && p.L != 64) || p.Ktot != (p.R * p.L + KSTEP - 1) / KSTEP * KSTEP ||
                p.off_h != 0 || p.off_w != 0)
                return false;
        } else {
            if (p.C % KSTEP != 0 || p.L != p.S * p.C || p.Lpad != p.L || p.Ktot != p.R * p.L || p.R * p.S > 32)
                return false;
        }
    }
    return true;
}

hipError_t igemm_dma_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    const int m = problem_mode(b.p[0]);
    if (m == kGemm) return run_mode<kGemm>(b, ctl, stream);
    if (m == kWin) return run_mode<kWin>(b, ctl, stream);
    return run_mode<kConv64>(b, ctl, stream);
}

}  // namespace niti
