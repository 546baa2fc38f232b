// Implicit-GEMM int8 MFMA kernel for layers whose whole weight operand fits
// in LDS (at most 128 output channels, a short reduction: the 3 x 3 layers
// at 56 x 56, the image layer, 1 x 1 projections).  Same problem form,
// epilogue and exponent speculation as igemm_dma.hip; the differences:
//
// * Each workgroup stages the weights once, [n][Ktot] with a row pitch of
//   Ktot + 16 bytes (rows land on different LDS banks for the fragment
//   reads), and keeps them for all its work.
// * A wave owns tasks of 32 output pixels x all channels.  The activation
//   operand goes from memory straight into the MFMA operand registers: for
//   the 32 x 32 x 32 int8 MFMA, lane l's 16 bytes are K bytes
//   16 * (l / 32) .. + 15 of a 32-byte half for pixel l % 32, which is one
//   16-byte buffer load per lane and half.  Loads run D K steps ahead of the
//   MFMAs (a register ring of D steps), across task boundaries.
// * There is no barrier in the K loop and waves never wait for each other:
//   a wave's epilogue overlaps other waves' MFMAs.
//
// Out-of-image taps and rows past the tensor load zeros through the buffer
// bounds (bit 31 set on the lane offset), as in igemm_dma.hip.
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int KSTEP = 64;
constexpr uint32_t kOOB = 0x80000000u;
constexpr int kConvW = 1;   // C % 64 == 0: a K step lies in one filter tap and channel block
constexpr int kWinW = 2;    // zero-padded image read in filter-row windows of L bytes
constexpr int NWAVES = 8;
constexpr int NT = 64 * NWAVES;

// Wait until this wave's vector memory operations (LDS DMA included) are done.
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// LDS bytes of the staged weights: NROWS rows of pitch Ktot + 16, in whole
// 1 KB blocks (the staging DMA writes 64 slots of 16 bytes at a time).
__host__ __device__ constexpr int wres_lds_bytes(int nrows, int ktot) { return (nrows * (ktot + 16) + 1023) / 1024 * 1024; }

// Round one accumulator (Algorithm 3, or nearest) with the call's uniform
// shift; RELU: the backward mask is applied later, the forward ReLU here.
// FAST: the closed form of niti_device.h.  Returns the int8 in the low
// byte.
template <bool RELU, bool RTN, bool FAST>
__device__ __forceinline__ uint32_t wr_round(int32_t v, const RoundK& k, uint32_t& tmax) {
    if (RELU) v = v < 0 ? 0 : v;
    const uint32_t x = RELU ? (uint32_t)v : (v < 0 ? 0u - (uint32_t)v : (uint32_t)v);
    tmax = x > tmax ? x : tmax;
    uint32_t q;
    if (RTN) {
        q = x >> k.bp;
        q += k.bp ? __builtin_amdgcn_ubfe(x, k.bp - 1, 1) : 0u;
        q = min(q, 127u);
    } else if (FAST) {
        q = round_psr_mag_fast(x, k);
    } else {
        q = x >> k.bp;
        const uint32_t thi = __builtin_amdgcn_ubfe(x, k.odd + k.h, k.h);
        const uint32_t rlo = __builtin_amdgcn_ubfe(x, k.odd, k.h);
        q = min(q + (thi > rlo ? 1u : 0u), 127u);
    }
    if (RELU) return q;
    const uint32_t sgn = (uint32_t)(v >> 31);
    return ((q ^ sgn) - sgn) & 0xFFu;
}

// Rounded bytes of one 32 x 32 accumulator fragment, regrouped so that each
// lane holds 16 consecutive channels of its pixel.  Element 4*jj + i of the
// fragment is channel 8*jj + 4*(lane/32) + i of pixel lane%32; after packing,
// word jj of lane l < 32 holds channels 8jj..8jj+3 and of lane l + 32
// channels 8jj+4..8jj+7.  Two half-wave swaps (lanes 32..63 of the first
// operand with lanes 0..31 of the second) leave lanes 0..31 with channels
// 0..15 and lanes 32..63 with channels 16..31, as words (w0, w2, w1, w3).
template <bool RELU, bool RTN, bool FAST>
__device__ __forceinline__ uint4 wr_round_fragment(const v16i& acc, const RoundK& rk, uint32_t& mx) {
    uint32_t w[4];
#pragma unroll
    for (int jj = 0; jj < 4; jj++) {
        uint32_t packed = 0;
#pragma unroll
        for (int i = 0; i < 4; i++) packed |= wr_round<RELU, RTN, FAST>(acc[4 * jj + i], rk, mx) << (8 * i);
        w[jj] = packed;
    }
    const auto s02 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
    return make_uint4(s02[0], s02[1], s13[0], s13[1]);
}

// Write 16 rounded channels (nv <= 16 valid) at out + off, with the
// backward ReLU mask (a byte is kept where the mask byte is positive);
// have_m: mpre holds the 16 mask bytes at off, loaded earlier.
__device__ __forceinline__ void wr_store16(const IgemmProblem& P, int64_t off, uint4 v, int nv,
                                           bool have_m = false, uint4 mpre = make_uint4(0, 0, 0, 0)) {
    int8_t* dst = P.out + off;
    const bool full = nv == 16 && (((uintptr_t)dst) & 15) == 0;
    if (P.mask) {
        const int8_t* ms = P.mask + off;
        uint32_t mw[4];
        if (full) {
            const uint4 mv = have_m ? mpre : *(const uint4*)ms;
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

template <int NF, int D>
struct WrCfg {
    static constexpr int NROWS = 32 * NF;   // weight rows staged (channels, zero past Nout)
    // waves per SIMD the register budget is set for: two workgroups per CU
    // for two channel fragments or a one-step lead, else one
    static constexpr int MINW = NF <= 2 ? 4 : 2;
};

// Tasks of one wave.  Workgroup b runs on XCD b % 8; the tasks are cut into
// eight contiguous ranges in proportion to the waves each XCD receives, and
// the waves of an XCD deal out its range in turn, so neighbouring pixels
// (which share input rows) are computed at the same time under one L2.
struct TaskList {
    int first, step, end;
};
__device__ __forceinline__ TaskList task_list(int tasks, int G, int b, int wave) {
    const int x = b & 7, bslot = b >> 3;
    const int q = G >> 3, r = G & 7;
    const int cnt = q + (x < r ? 1 : 0);
    const int cum0 = x * q + min(x, r);
    const int start = (int)((int64_t)tasks * cum0 / G);
    const int end = (int)((int64_t)tasks * (cum0 + cnt) / G);
    return {start + bslot * NWAVES + wave, cnt * NWAVES, end};
}

// The tasks of one wave.  D: K steps the loads run ahead (divides the step
// count nk); do_store / do_max as in igemm_dma.hip.
template <int NF, int MODE, int D>
__device__ __forceinline__ void wres_tasks(const IgemmProblem& P, const TaskList tl, int8_t* lds, const RoundK& rk,
                                           int relu, int do_store, int do_max, uint32_t& tmax, niti_stats* snap_st,
                                           int snap_slot, uint64_t& snap) {
    using T = WrCfg<NF, D>;
    const int lane = threadIdx.x & 63;
    const int hi = lane >> 5;   // which 16 bytes of a 32-byte half this lane feeds
    const int nk = (P.Ktot + KSTEP - 1) / KSTEP;
    const int groups = nk / D;
    const uint32_t kp = (uint32_t)(P.Ktot + 16);   // LDS row pitch

    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc((void*)P.act, 0, (int)P.act_bytes, 0x00020000);

    // ---- load side: lane state of the task being loaded (pixel base, taps
    // outside the image / window rows), the uniform cursor within it, and
    // the register ring.
    uint32_t ab = kOOB, aux = ~0u;     // kConvW: pixel base, invalid taps; kWinW: window base, row of h = 0
    uint32_t ab1 = kOOB, aux1 = 0;     // kWinW: window base and row for h = 1
    const int cbs = MODE == kConvW ? P.C / KSTEP : 1;
    const int rps = MODE == kWinW ? KSTEP / P.L : 1;
    auto lane_state = [&](int t) {
        const int m = t * 32 + (lane & 31);
        const bool in = t < tl.end && m < P.M;
        const uint32_t mm = in ? (uint32_t)m : 0u;
        const uint32_t img = fdiv(mm, P.div_ohw);
        const uint32_t rem = mm - img * (uint32_t)(P.OHc * P.OWc);
        const uint32_t oh = fdiv(rem, P.div_ow);
        const uint32_t ow = rem - oh * (uint32_t)P.OWc;
        if (MODE == kWinW) {
            // K bytes 32 h + 16 hi of each step: window row and byte
            const int kb0 = 16 * hi, kb1 = 32 + 16 * hi;
            const int r0 = kb0 / P.L, r1 = kb1 / P.L;
            const uint32_t pix = ((img * (uint32_t)P.H + oh * (uint32_t)P.st) * (uint32_t)P.W + ow * (uint32_t)P.st) *
                                 (uint32_t)P.C;
            ab = in ? pix + (uint32_t)(r0 * P.W * P.C + (kb0 - r0 * P.L)) : kOOB;
            ab1 = in ? pix + (uint32_t)(r1 * P.W * P.C + (kb1 - r1 * P.L)) : kOOB;
            aux = (uint32_t)r0;
            aux1 = (uint32_t)r1;
        } else {
            const int h0 = (int)oh * P.st + P.off_h;
            const int w0 = (int)ow * P.st + P.off_w;
            ab = (uint32_t)((int64_t)img * P.H * P.W * P.C + ((int64_t)h0 * P.W + w0) * P.C) + (uint32_t)(16 * hi);
            uint32_t rows = 0, cols = 0, valid = 0;
            for (int r = 0; r < P.R; r++) rows |= (uint32_t)((unsigned)(h0 + r) < (unsigned)P.H) << r;
            for (int c = 0; c < P.S; c++) cols |= (uint32_t)((unsigned)(w0 + c) < (unsigned)P.W) << c;
            for (int r = 0; r < P.R; r++)
                if ((rows >> r) & 1u) valid |= cols << (r * P.S);
            aux = in ? ~valid : ~0u;
        }
    };
    // uniform cursor: K step j of the task being loaded
    int j = 0, tap = 0, ts = 0, cb = 0;
    uint32_t tapbase = 0;
    auto load_step = [&](v4i (&b)[2]) {
        if (MODE == kWinW) {
            const uint32_t so = (uint32_t)(j * rps * P.W * P.C);
            const int rlim = P.R - j * rps;   // window rows at or past R load zeros
            const uint32_t v0 = (int)aux >= rlim ? kOOB : ab;
            const uint32_t v1 = (int)aux1 >= rlim ? kOOB : ab1;
            b[0] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(ars, v0, so, 0));
            b[1] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(ars, v1, so, 0));
        } else {
            const uint32_t v = (__builtin_amdgcn_ubfe(aux, (uint32_t)tap, 1) << 31) | (ab + tapbase);
            const uint32_t so = (uint32_t)(cb * KSTEP);
            b[0] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(ars, v, so, 0));
            b[1] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(ars, v, so + 32u, 0));
            if (++cb == cbs) {
                cb = 0;
                ++tap;
                if (++ts == P.S) {
                    ts = 0;
                    tapbase += (uint32_t)((P.W - P.S + 1) * P.C);
                } else {
                    tapbase += (uint32_t)P.C;
                }
            }
        }
        ++j;
    };
    auto next_task_cursor = [&](int t) {
        lane_state(t);
        j = 0; tap = 0; ts = 0; cb = 0;
        tapbase = 0;
    };

    // ---- the first task's first D steps go out before the weights, so that
    // both latencies overlap
    v4i bq[D][2];
    next_task_cursor(tl.first);
#pragma unroll
    for (int u = 0; u < D; u++) load_step(bq[u]);

    // ---- weights: rows [n][Ktot] into LDS with pitch kp, by DMA straight
    // from memory.  LDS 16-byte slot s is chunk s % spr of row s / spr
    // (spr = Ktot / 16 + 1: the last slot of a row is its pad); pad slots and
    // rows past Nout read past the buffer end, which loads zeros.  Each wave
    // instruction fills 64 consecutive slots.
    {
        const u32x4 wrs = raw_rsrc(P.wgt, (uint32_t)P.wgt_bytes);
        const uint32_t spr = (uint32_t)(P.Ktot / 16 + 1);
        const uint32_t nslots = (uint32_t)T::NROWS * spr;
        const uint32_t lds0 = lds_address(lds);
        const uint32_t step = (uint32_t)NT;   // slots per pass of the workgroup
        const uint32_t dn = step / spr, dc = step - dn * spr;
        uint32_t s0 = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x & ~63);
        uint32_t n = (s0 + lane) / spr, c = (s0 + lane) - n * spr;
        for (; s0 < nslots; s0 += step) {
            const bool data = n < (uint32_t)P.Nout && c + 1 < spr;
            lds_dma16_at(wrs, lds0, s0 * 16u, data ? n * (uint32_t)P.Ktot + c * 16u : kOOB, 0u);
            n += dn;
            c += dc;
            if (c >= spr) {
                c -= spr;
                ++n;
            }
        }
        wait_vm0();
    }
    __syncthreads();   // weights staged

    // fragment reads: channel row (a * 32 + lane % 32), K bytes 32 h + 16 hi of
    // the step at K byte kk.  The weights of a half step are read one half
    // step ahead (they are the same for every task: after a task's last step
    // come the first step's), so no MFMA waits for LDS.
    const int8_t* wrow = lds + (lane & 31) * kp + 16 * hi;
    auto read_wh = [&](int kk, int h, v4i (&w)[NF]) {
#pragma unroll
        for (int a = 0; a < NF; a++) w[a] = *(const v4i*)(wrow + a * 32 * (int)kp + kk + 32 * h);
    };
    v4i wn[NF];
    read_wh(0, 0, wn);
    v16i acc[NF];
    const int mode_sel = (relu ? 1 : 0) | (rk.rtn ? 2 : 0);
    const bool dense = P.os == 1 && P.OHc == P.OH && P.OWc == P.OW;
    for (int t = tl.first; t < tl.end; t += tl.step) {
#pragma unroll
        for (int a = 0; a < NF; a++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[a][e] = 0;
        // output offset of pixel t*32 + lane%32 (channels a*32 + 16*hi ..
        // + 15), and, for a back-propagation, the ReLU mask bytes there,
        // loaded now so that they arrive during the task's MFMAs
        const int m = t * 32 + (lane & 31);
        int64_t ooff = -1;
        if (m < P.M) {
            if (dense) {
                ooff = (int64_t)m * P.ldo;
            } else {
                const uint32_t img = fdiv((uint32_t)m, P.div_ohw);
                const uint32_t rem = (uint32_t)m - img * (uint32_t)(P.OHc * P.OWc);
                const uint32_t i0 = fdiv(rem, P.div_ow);
                const uint32_t j0 = rem - i0 * (uint32_t)P.OWc;
                const int oh = (int)i0 * P.os + P.oa;
                const int ow = (int)j0 * P.os + P.ob;
                ooff = (((int64_t)img * P.OH + oh) * P.OW + ow) * P.ldo;
            }
        }
        uint4 mpre[NF];
        bool mok[NF];
#pragma unroll
        for (int a = 0; a < NF; a++) {
            const int n0 = a * 32 + 16 * hi;
            mok[a] = do_store && P.mask && ooff >= 0 && n0 + 16 <= P.Nout &&
                     (((uintptr_t)(P.mask + ooff + n0)) & 15) == 0 && (((uintptr_t)(P.out + ooff + n0)) & 15) == 0;
            mpre[a] = mok[a] ? *(const uint4*)(P.mask + ooff + n0) : make_uint4(0, 0, 0, 0);
        }
        for (int g = 0; g < groups; g++) {
            // the loads issued in this group are for the next task's first steps
            if (g == groups - 1) next_task_cursor(t + tl.step);
#pragma unroll
            for (int u = 0; u < D; u++) {
                const int kk = (g * D + u) * KSTEP;
                int kn = kk + KSTEP;
                if (kn == P.Ktot) kn = 0;
#pragma unroll
                for (int h = 0; h < 2; h++) {
                    v4i wa[NF];
#pragma unroll
                    for (int a = 0; a < NF; a++) wa[a] = wn[a];
                    if (h == 0)
                        read_wh(kk, 1, wn);
                    else
                        read_wh(kn, 0, wn);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int a = 0; a < NF; a++)
                        acc[a] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wa[a], bq[u][h], acc[a], 0, 0, 0);
                }
                load_step(bq[u]);
            }
        }
        if (t + tl.step >= tl.end && snap_st && threadIdx.x == 0) snap = load_acc(snap_st, snap_slot);
        // epilogue
        uint32_t mx = 0;
#pragma unroll
        for (int a = 0; a < NF; a++) {
            uint4 v;
            switch (mode_sel) {
                case 0: v = wr_round_fragment<false, false, true>(acc[a], rk, mx); break;
                case 1: v = wr_round_fragment<true, false, true>(acc[a], rk, mx); break;
                case 2: v = wr_round_fragment<false, true, false>(acc[a], rk, mx); break;
                default: v = wr_round_fragment<true, true, false>(acc[a], rk, mx); break;
            }
            const int n0 = a * 32 + 16 * hi;
            if (do_store && ooff >= 0 && n0 < P.Nout)
                wr_store16(P, ooff + n0, v, min(16, P.Nout - n0), mok[a], mpre[a]);
        }
        if (do_max) tmax = mx > tmax ? mx : tmax;
    }
    // Zero siblings of the tasks' pixels (stride-2 classes without taps),
    // in a pass of their own so that they cost no registers in the main loop.
    if (do_store && P.zsib) {
        for (int t = tl.first; t < tl.end; t += tl.step) {
            const int m = t * 32 + (lane & 31);
            if (m >= P.M) continue;
            const uint32_t img = fdiv((uint32_t)m, P.div_ohw);
            const uint32_t rem = (uint32_t)m - img * (uint32_t)(P.OHc * P.OWc);
            const uint32_t i0 = fdiv(rem, P.div_ow);
            const uint32_t j0 = rem - i0 * (uint32_t)P.OWc;
            const int oh = (int)i0 * P.os + P.oa;
            const int ow = (int)j0 * P.os + P.ob;
            const int64_t ooff = (((int64_t)img * P.OH + oh) * P.OW + ow) * P.ldo;
            const uint32_t zs = zero_siblings(P, oh, ow);
            for (int a = 0; a < NF; a++) {
                const int n0 = a * 32 + 16 * hi;
                if (n0 < P.Nout) store_zero_siblings(P, ooff + n0, zs, min(16, P.Nout - n0));
            }
        }
    }
}

template <int NF, int MODE, int D>
__global__ __launch_bounds__(NT, (WrCfg<NF, D>::MINW)) void igemm_wres_main(IgemmBatch batch, IgemmCtl ctl, int tasks) {
    extern __shared__ __attribute__((aligned(1024))) int8_t dyn_lds[];
    niti_stats* st = ctl.stats;
    const int slot = call_slot(st);
    uint64_t snap = 0;
    const int hint = st->bp_hint;
    begin_call(st, slot, hint);
    const RoundK rk = make_round(hint < 0 ? 0 : hint, ctl.mode);
    uint32_t tmax = 0;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    wres_tasks<NF, MODE, D>(batch.p[0], task_list(tasks, gridDim.x, blockIdx.x, wave), dyn_lds, rk, ctl.relu,
                            hint >= 0, 1, tmax, st, slot, snap);
    // Accumulator magnitudes are at most 2^31: 32-bit reductions are exact.
    // After the barrier the weight rows are no longer read: their first
    // bytes serve the reduction.
    __syncthreads();
    block_publish_max32(st, slot, tmax, (uint32_t*)dyn_lds, snap);
}

template <int NF, int MODE, int D>
__global__ __launch_bounds__(NT, (WrCfg<NF, D>::MINW)) void igemm_wres_fixup(IgemmBatch batch, IgemmCtl ctl, int tasks) {
    extern __shared__ __attribute__((aligned(1024))) int8_t dyn_lds[];
    niti_stats* st = ctl.stats;
    const CallState cs = shared_call_state(st, dyn_lds);
    const int hint = cs.hint;
    const int bp = block_bp(cs.mx, ctl.target);
    if (bp != hint) {
        const RoundK rk = make_round(bp, ctl.mode);
        uint32_t dummy = 0;
        uint64_t nosnap = 0;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        wres_tasks<NF, MODE, D>(batch.p[0], task_list(tasks, gridDim.x, blockIdx.x, wave), dyn_lds, rk, ctl.relu, 1,
                                0, dummy, nullptr, 0, nosnap);
    }
    if (is_finisher()) finish_call(st, ctl.target, ctl.ex, ctl.static_flags, 1);
}

template <int NF, int MODE, int D>
hipError_t launch_wres(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    static bool attr_done = false;
    static int resident = 0;
    const IgemmProblem& p = b.p[0];
    const int lds = wres_lds_bytes(WrCfg<NF, D>::NROWS, p.Ktot);
    if (!attr_done) {
        constexpr int kMaxLds = 160 * 1024;
        hipError_t e = hipFuncSetAttribute((const void*)igemm_wres_main<NF, MODE, D>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds);
        if (e != hipSuccess) return e;
        e = hipFuncSetAttribute((const void*)igemm_wres_fixup<NF, MODE, D>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                kMaxLds);
        if (e != hipSuccess) return e;
        int dev = 0, cus = 0;
        e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        resident = cus > 0 ? cus : 1;
        attr_done = true;
    }
    // workgroups per CU: two when two weight copies fit the LDS and the
    // registers allow, else one
    const int per_cu = (WrCfg<NF, D>::MINW >= 4 && 2 * lds <= 160 * 1024) ? 2 : 1;
    const int tasks = (p.M + 31) / 32;
    int grid = (tasks + NWAVES - 1) / NWAVES;
    if (grid > per_cu * resident) grid = per_cu * resident;
    const int tk = timing_on() ? timing_begin(NITI_TIMING_KERNEL, stream,
                                              kernel_label("igemm_wres_main<%d,%d,%d>", NF, MODE, D))
                               : -1;
    hipLaunchKernelGGL((igemm_wres_main<NF, MODE, D>), dim3(grid), dim3(NT), lds, stream, b, ctl, tasks);
    timing_end(tk, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((igemm_wres_fixup<NF, MODE, D>), dim3(grid), dim3(NT), lds, stream, b, ctl, tasks);
    return hipGetLastError();
}

template <int NF, int MODE>
hipError_t launch_d(int d, IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    switch (d) {
        case 4: return launch_wres<NF, MODE, 4>(b, ctl, stream);
        case 3: return launch_wres<NF, MODE, 3>(b, ctl, stream);
        case 2: return launch_wres<NF, MODE, 2>(b, ctl, stream);
        default: return launch_wres<NF, MODE, 1>(b, ctl, stream);
    }
}

// Loads run D steps ahead; D divides the step count (so a task's last group
// of D steps loads exactly the next task's first D steps).
int pick_lead(int nk) {
    if (nk % 4 == 0) return 4;
    if (nk % 3 == 0) return 3;
    if (nk % 2 == 0) return 2;
    return 1;
}

int wres_mode(const IgemmProblem& p) {
    if (p.win) return kWinW;
    if (!(p.H == 1 && p.W == 1 && p.R == 1 && p.off_h == 0 && p.off_w == 0 && p.L == p.C)) return kConvW;
    return 0;   // plain matrix rows: not handled here
}

}  // namespace

// One problem (no sub-pixel classes), at most 128 output channels, the
// weight operand small enough to stage (two copies per CU for up to 64
// channels), and 32-bit buffer offsets for the activations.
bool igemm_wres_eligible(const IgemmBatch& b) {
    if (b.nprob != 1) return false;
    const IgemmProblem& p = b.p[0];
    const int mode = wres_mode(p);
    if (mode == 0 || p.Nout <= 0 || p.Nout > 128 || p.M <= 0) return false;
    if (p.act_bytes <= 0 || p.act_bytes >= ((int64_t)1 << 31)) return false;
    if (p.Ktot <= 0 || p.Ktot % KSTEP != 0) return false;
    if (mode == kWinW) {
        if ((p.L != 16 && p.L != 32 && p.L != 64) || p.Ktot != (p.R * p.L + KSTEP - 1) / KSTEP * KSTEP ||
            p.off_h != 0 || p.off_w != 0)
            return false;
    } else {
        if (p.C % KSTEP != 0 || p.L != p.S * p.C || p.Lpad != p.L || p.Ktot != p.R * p.L || p.R * p.S > 32)
            return false;
    }
    if (p.wgt_bytes < (int64_t)p.Nout * p.Ktot || p.wgt_bytes >= ((int64_t)1 << 31)) return false;
    const int nf = p.Nout <= 64 ? 2 : 4;
    if (p.Ktot > 8192) return false;
    const int lds = wres_lds_bytes(32 * nf, p.Ktot);
    return nf == 2 ? lds <= 80 * 1024 : lds <= 152 * 1024;
}

hipError_t igemm_wres_run(IgemmBatch& b, IgemmCtl ctl, hipStream_t stream) {
    const IgemmProblem& p = b.p[0];
    const int d = pick_lead(p.Ktot / KSTEP);
    const bool win = wres_mode(p) == kWinW;
    if (p.Nout <= 64) return win ? launch_d<2, kWinW>(d, b, ctl, stream) : launch_d<2, kConvW>(d, b, ctl, stream);
    return win ? launch_d<4, kWinW>(d, b, ctl, stream) : launch_d<4, kConvW>(d, b, ctl, stream);
}

}  // namespace niti
