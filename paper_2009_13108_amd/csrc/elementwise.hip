// Bandwidth-bound passes of the NITI step: the tensor-wide maximum, the
// shift-and-round of an int32 tensor (Algorithms 2 and 3), the discrete
// weight update (Section 3.3), the integer cross-entropy gradient (Section
// 3.5), the back-propagation filter repack and the layer glue (input
// quantisation, 2x2 max pooling, backward ReLU).
#include "niti_internal.h"

namespace niti {

namespace {

constexpr int kThreads = 256;

inline int grid_for(int64_t n, int per_thread = 4, int cap = 2048) {
    int64_t g = (n + (int64_t)kThreads * per_thread - 1) / ((int64_t)kThreads * per_thread);
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n && (((uintptr_t)(p + i)) & 15) == 0) {
            *(int4*)(p + i) = make_int4(v, v, v, v);
        } else {
            for (int64_t j = i; j < i + 4 && j < n; j++) p[j] = v;
        }
    }
}

// Accumulating launch of a call: the tensor maximum of x.
__global__ void max_abs_i32_kernel(const int32_t* x, int64_t n, niti_stats* st) {
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    begin_call(st, slot, -1);
    uint64_t m = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const uint64_t a = mag32(x[i]);
        m = a > m ? a : m;
    }
    __shared__ uint32_t red[kThreads / 64];
    block_publish_max32(st, slot, (uint32_t)m, red, snap);  // magnitudes <= 2^31
}

// Sum of the per-split partial weight gradients (exact mod 2^32) into g32,
// and the tensor maximum of the sum.  With one split the partial already is
// g32 and only the maximum is taken.  A workgroup covers 256 consecutive
// elements (4 per lane, 16-byte loads); its four waves take interleaved
// quarters of the splits with four loads in flight each, and add their sums
// in LDS.
__global__ __launch_bounds__(256) void reduce_max_kernel(const int32_t* part, int splits, int32_t* g32,
                                                         int64_t n, niti_stats* st) {
    __shared__ uint4 sum4[4][64];
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    begin_call(st, slot, -1);
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t i0 = (int64_t)blockIdx.x * 256 + 4 * lane;
    const bool vec = (n % 4) == 0 && i0 + 4 <= n;
    uint32_t acc[4] = {0, 0, 0, 0};
    if (vec) {
        uint4 a = make_uint4(0, 0, 0, 0), b = a, c = a, d = a;
        int z = wv;
        for (; z + 12 < splits; z += 16) {
            const uint4 pa = *(const uint4*)(part + (int64_t)z * n + i0);
            const uint4 pb = *(const uint4*)(part + (int64_t)(z + 4) * n + i0);
            const uint4 pc = *(const uint4*)(part + (int64_t)(z + 8) * n + i0);
            const uint4 pd = *(const uint4*)(part + (int64_t)(z + 12) * n + i0);
            a.x += pa.x; a.y += pa.y; a.z += pa.z; a.w += pa.w;
            b.x += pb.x; b.y += pb.y; b.z += pb.z; b.w += pb.w;
            c.x += pc.x; c.y += pc.y; c.z += pc.z; c.w += pc.w;
            d.x += pd.x; d.y += pd.y; d.z += pd.z; d.w += pd.w;
        }
        for (; z < splits; z += 4) {
            const uint4 pa = *(const uint4*)(part + (int64_t)z * n + i0);
            a.x += pa.x; a.y += pa.y; a.z += pa.z; a.w += pa.w;
        }
        acc[0] = a.x + b.x + c.x + d.x;
        acc[1] = a.y + b.y + c.y + d.y;
        acc[2] = a.z + b.z + c.z + d.z;
        acc[3] = a.w + b.w + c.w + d.w;
    } else {
        for (int e = 0; e < 4; e++) {
            const int64_t i = i0 + e;
            if (i >= n) break;
            for (int z = wv; z < splits; z += 4) acc[e] += (uint32_t)part[(int64_t)z * n + i];
        }
    }
    sum4[wv][lane] = make_uint4(acc[0], acc[1], acc[2], acc[3]);
    __syncthreads();
    uint64_t m = 0;
    if (wv == 0) {
        uint32_t v[4];
        const uint4 s0 = sum4[0][lane], s1 = sum4[1][lane], s2 = sum4[2][lane], s3 = sum4[3][lane];
        v[0] = s0.x + s1.x + s2.x + s3.x;
        v[1] = s0.y + s1.y + s2.y + s3.y;
        v[2] = s0.z + s1.z + s2.z + s3.z;
        v[3] = s0.w + s1.w + s2.w + s3.w;
        for (int e = 0; e < 4; e++) {
            const int64_t i = i0 + e;
            if (i >= n) break;
            if (splits > 1) g32[i] = (int32_t)v[e];
            const uint64_t a = mag32((int32_t)v[e]);
            m = a > m ? a : m;
        }
    }
    __shared__ uint32_t red[kThreads / 64];
    block_publish_max32(st, slot, (uint32_t)m, red, snap);  // magnitudes <= 2^31
}

// The same sum for few splits (NZ <= 8, n % 4 == 0): every lane owns four
// consecutive elements at a time and adds all NZ partials itself (NZ
// independent 16-byte loads in flight), striding over the tensor; one
// maximum per workgroup is folded in at the end.
template <int NZ>
__global__ __launch_bounds__(256) void reduce_max_flat_kernel(const int32_t* part, int32_t* g32, int64_t n,
                                                              niti_stats* st) {
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    begin_call(st, slot, -1);
    const int64_t nq = n >> 2;
    const int64_t step = (int64_t)gridDim.x * blockDim.x;
    uint64_t m = 0;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += step) {
        uint4 v[NZ];
#pragma unroll
        for (int z = 0; z < NZ; z++) v[z] = *(const uint4*)(part + (int64_t)z * n + 4 * q);
        uint4 a = v[0];
#pragma unroll
        for (int z = 1; z < NZ; z++) {
            a.x += v[z].x;
            a.y += v[z].y;
            a.z += v[z].z;
            a.w += v[z].w;
        }
        if (NZ > 1) *(uint4*)(g32 + 4 * q) = a;
        const uint64_t m01 = max(mag32((int32_t)a.x), mag32((int32_t)a.y));
        const uint64_t m23 = max(mag32((int32_t)a.z), mag32((int32_t)a.w));
        const uint64_t mq = max(m01, m23);
        m = mq > m ? mq : m;
    }
    __shared__ uint32_t red[kThreads / 64];
    block_publish_max32(st, slot, (uint32_t)m, red, snap);  // magnitudes <= 2^31
}

// The same sum for many splits (n % 4 == 0).  A workgroup of four waves works
// in groups of G waves; a group takes 256 consecutive elements at a time:
// each of its waves reads them as one 1 KiB row piece per split (lane l holds
// elements 4l .. 4l+3), member w adds splits w, w + G, ... with a batch of
// 16-byte loads in flight (sixteen for G = 1, eight for G = 4), and the G
// sums are added in LDS.  G is one below 32 splits (a wave holds a whole
// column of them in one batch of loads) and four above.  At most one workgroup per CU strides over the tensor, so the
// maximum costs one atomic per CU.
template <int G>
__global__ __launch_bounds__(256) void reduce_max_many_kernel(const int32_t* part, int splits, int32_t* g32,
                                                              int64_t n, niti_stats* st) {
    constexpr int NG = 4 / G;   // element groups per pass
    __shared__ uint4 sums[4][64];
    __shared__ uint32_t red[4];
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    begin_call(st, slot, -1);
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int gi = wv / G, wm = wv - gi * G;
    uint32_t m = 0;
    for (int64_t i0 = ((int64_t)blockIdx.x * NG + gi) * 256; i0 - gi * 256 < n; i0 += (int64_t)gridDim.x * NG * 256) {
        const int64_t i = i0 + 4 * lane;
        uint4 a = make_uint4(0, 0, 0, 0);
        if (i < n) {
            const int32_t* src = part + i;
            constexpr int B = G == 1 ? 16 : 8;   // loads per batch
            int z = wm;
            for (; z + (B - 1) * G < splits; z += B * G) {
                uint4 v[B];
#pragma unroll
                for (int u = 0; u < B; u++) v[u] = *(const uint4*)(src + (int64_t)(z + G * u) * n);
#pragma unroll
                for (int u = 0; u < B; u++) {
                    a.x += v[u].x;
                    a.y += v[u].y;
                    a.z += v[u].z;
                    a.w += v[u].w;
                }
            }
            for (; z < splits; z += G) {
                const uint4 v = *(const uint4*)(src + (int64_t)z * n);
                a.x += v.x;
                a.y += v.y;
                a.z += v.z;
                a.w += v.w;
            }
        }
        if (G > 1) {
            sums[wv][lane] = a;
            __syncthreads();
            if (wm == 0) {
#pragma unroll
                for (int h = 1; h < G; h++) {
                    const uint4 v = sums[wv + h][lane];
                    a.x += v.x;
                    a.y += v.y;
                    a.z += v.z;
                    a.w += v.w;
                }
            }
        }
        if (wm == 0 && i < n) {
            *(uint4*)(g32 + i) = a;
            const uint32_t mq =
                max(max(mag32((int32_t)a.x), mag32((int32_t)a.y)), max(mag32((int32_t)a.z), mag32((int32_t)a.w)));
            m = max(m, mq);
        }
        if (G > 1) __syncthreads();   // sums is rewritten by the next pass
    }
    block_publish_max32(st, slot, m, red, snap);  // magnitudes <= 2^31
}

// Rows of the strided back-propagation output that belong to sub-pixel
// classes with no filter taps are exact zeros: out[img][y][x][:] = 0 for every
// (y % st, x % st) whose bit (y % st) * st + x % st is set in mask.  One
// workgroup per output row; rows whose classes all have taps return at once.
__global__ void zero_classes_kernel(uint32_t* out, int32_t h, int32_t w, int32_t c4, int32_t st, uint32_t mask) {
    const uint32_t rid = blockIdx.x;   // img * h + y
    const int y = (int)(rid % (uint32_t)h);
    const uint32_t rowbits = (mask >> ((y % st) * st)) & ((1u << st) - 1u);
    if (rowbits == 0) return;
    const uint32_t len = (uint32_t)w * (uint32_t)c4;
    uint32_t* row = out + (size_t)rid * len;
    for (uint32_t i = threadIdx.x; i < len; i += blockDim.x) {
        const uint32_t x = c4 == 1 ? i : i / (uint32_t)c4;
        if ((rowbits >> (x % (uint32_t)st)) & 1u) row[i] = 0u;
    }
}

// bp_fixed >= 0: that binary point.  bp_fixed < 0: the block binary point of
// the call in progress; this is its finishing launch.
__global__ void round_i32_kernel(const int32_t* x, int8_t* y, int64_t n, int bp_fixed, int target,
                                 int mode, niti_stats* st, ExpArgs ex) {
    const int bp = bp_fixed >= 0 ? bp_fixed : block_bp(shared_call_state(st).mx, target);
    RoundK rk = make_round(bp, mode);
    if (bp_fixed >= 0)
        sr_key_current(rk, st);    // an explicit binary point: no accumulating launch, calls not counted
    else
        sr_key_recorded(rk, st);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        y[i] = round_i32_at(x[i], rk, (uint64_t)i);
    if (bp_fixed >= 0) {
        // Algorithm 2: s_q = s_q32 + bp, held to the int8 range.
        if (ex.s_out && is_finisher()) {
            int s = (int)*ex.s_a + bp;
            *ex.s_out = (int8_t)(s > 127 ? 127 : (s < -128 ? -128 : s));
        }
        return;
    }
    if (is_finisher()) finish_call(st, target, ex, 0u, 0);
}

// Discrete update, the finishing launch of its call:
// g = round(g32, max(0, B(g32) - mu)); w <- clamp(w - g).
__global__ void update_kernel(int8_t* __restrict__ w, const int32_t* __restrict__ g32, int64_t n, int mu, int mode,
                              niti_stats* st, uint32_t static_flags) {
    const int bp = block_bp(shared_call_state(st).mx, mu);
    RoundK rk = make_round(bp, mode);
    sr_key_recorded(rk, st);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // Groups of four weights (one 4-byte word of w, 16 bytes of g32), two
    // groups per thread and pass with both loads issued before any store.
    const bool vec = ((((uintptr_t)w) | ((uintptr_t)g32)) & 15) == 0;
    const int64_t nq = vec ? n >> 2 : 0;
    for (int64_t q0 = tid; q0 < nq; q0 += 2 * stride) {
        int4 g[2];
        uint32_t wv[2];
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const int64_t q = q0 + j * stride;
            g[j] = q < nq ? ((const int4*)g32)[q] : make_int4(0, 0, 0, 0);
            wv[j] = q < nq ? ((const uint32_t*)w)[q] : 0u;
        }
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const int64_t q = q0 + j * stride;
            if (q >= nq) continue;
            const int32_t gv[4] = {g[j].x, g[j].y, g[j].z, g[j].w};
            uint32_t out = 0;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                int v = (int)(int8_t)(wv[j] >> (8 * e)) - (int)round_i32_at(gv[e], rk, (uint64_t)(4 * q + e));
                v = v > 127 ? 127 : (v < -127 ? -127 : v);
                out |= (uint32_t)(uint8_t)v << (8 * e);
            }
            ((uint32_t*)w)[q] = out;
        }
    }
    for (int64_t i = 4 * nq + tid; i < n; i += stride) {
        int v = (int)w[i] - (int)round_i32_at(g32[i], rk, (uint64_t)i);
        v = v > 127 ? 127 : (v < -127 ? -127 : v);
        w[i] = (int8_t)v;
    }
    if (is_finisher()) finish_call(st, mu, ExpArgs{nullptr, nullptr, nullptr}, static_flags, 0);
}

// ---------------------------------------------------------------------------
// Integer cross-entropy gradient, one wave per sample (Section 3.5).
//
// The Taylor branch (s_a <= -7) is exact: t_i = 2^(1-2 s_a) + a_i 2^(1-s_a) +
// a_i^2 in 128-bit integers, which holds every value (row sums included) for
// s_a >= -54.  Below -54 the rounded int8 error does not depend on s_a any
// more (the three terms sit in disjoint bit ranges far from the binary
// point), so s_a = -54 is evaluated and NITI_FLAG_LOSS_SA is raised.  Values
// go to the workspace as 128-bit integers.  Below s_a = -22 the largest value
// can exceed 64 bits, so the block maximum is folded in shifted right by
// kLossShift(s_a) = 2 (-22 - s_a) bits (exact for the effective bitwidth:
// every nonzero row has a value of at least 2^(-2 s_a) > 2^shift).
constexpr int kLossMinSa = -54;
constexpr int kLossWideSa = -22;

typedef __int128 i128;
typedef unsigned __int128 u128;

__device__ __forceinline__ int loss_eval_sa(int s_a) { return s_a < kLossMinSa ? kLossMinSa : s_a; }
__device__ __forceinline__ int loss_max_shift(int s_a) { return s_a < kLossWideSa ? 2 * (kLossWideSa - s_a) : 0; }

__device__ __forceinline__ int64_t loss_xhat(int64_t a, int s_a) {
    const int64_t prod = 47274 * a;
    const int sh = 15 - s_a;
    if (sh >= 0) return prod >> sh;  // arithmetic shift: floor
    // s_a > 15: any left shift already separates distinct logits by more
    // than the 10-bit window, so one doubling gives the same t values.
    return prod * 2;
}

__device__ __forceinline__ u128 mag128(i128 v) { return v < 0 ? (u128)0 - (u128)v : (u128)v; }

__device__ __forceinline__ i128 wave_sum_i128(i128 v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t lo = (uint64_t)(u128)v, hi = (uint64_t)((u128)v >> 64);
        const uint64_t lo2 = __shfl_xor(lo, o, kWave), hi2 = __shfl_xor(hi, o, kWave);
        v += (i128)(((u128)hi2 << 64) | (u128)lo2);
    }
    return v;
}

// One term t_i of a row (Section 3.5); p is the row's offset (base-2 branch).
__device__ __forceinline__ i128 loss_term(int a, int s_a, int64_t p) {
    if (s_a <= -7) {
        const i128 ai = a;
        return ((i128)1 << (1 - 2 * s_a)) + (ai << (1 - s_a)) + ai * ai;
    }
    int64_t xt = loss_xhat(a, s_a) - p;
    xt = xt < 0 ? 0 : xt;
    return (i128)((int64_t)1 << xt);
}

// One wave per sample.  NPL > 0: every lane keeps its NPL entries (lane,
// lane + 64, ...) in registers, so the logits are read once and e128 is
// only written (classes <= 64 * NPL); NPL == 0 streams any number of classes
// through e128.
template <int NPL>
__global__ void loss_kernel(const int8_t* __restrict__ logits, const int8_t* __restrict__ s_logits,
                            const int32_t* __restrict__ labels, i128* __restrict__ e128, int64_t batch,
                            int64_t classes, niti_stats* st) {
    const int slot = call_slot(st);
    const uint64_t snap = max_snapshot(st, slot);
    begin_call(st, slot, -1);
    const int lane = threadIdx.x & 63;
    const int64_t sample = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
    const int s_in = (int)*s_logits;
    const int s_a = loss_eval_sa(s_in);
    const int msh = loss_max_shift(s_a);
    uint64_t m = 0;
    if (sample < batch) {
        const int8_t* a = logits + sample * classes;
        i128* e = e128 + sample * classes;
        const int32_t y = labels[sample];
        const bool taylor = s_a <= -7;
        if constexpr (NPL > 0) {
            // All NPL loads in flight at once: entries past the row read its
            // last entry (in bounds, unconditional) and are zeroed after.
            int av[NPL];
#pragma unroll
            for (int j = 0; j < NPL; j++) av[j] = (int)a[min((int64_t)(lane + 64 * j), classes - 1)];
#pragma unroll
            for (int j = 0; j < NPL; j++)
                if (lane + 64 * j >= classes) av[j] = 0;
            int64_t p = 0;
            if (!taylor) {
                int64_t mx = INT64_MIN;
#pragma unroll
                for (int j = 0; j < NPL; j++)
                    if (lane + 64 * j < classes) {
                        const int64_t xh = loss_xhat(av[j], s_a);
                        mx = xh > mx ? xh : mx;
                    }
                p = wave_max_i64(mx) - 10;
            }
            i128 t[NPL];
            i128 C = 0;
#pragma unroll
            for (int j = 0; j < NPL; j++) {
                t[j] = lane + 64 * j < classes ? loss_term(av[j], s_a, p) : (i128)0;
                C += t[j];
            }
            C = wave_sum_i128(C);
            // The owner of the label's entry subtracts C (a label outside
            // [0, classes) contributes no term).
            const bool own = y >= 0 && y < classes && (y & 63) == lane;
#pragma unroll
            for (int j = 0; j < NPL; j++) {
                const int i = lane + 64 * j;
                if (own && (y >> 6) == j) t[j] -= C;
                if (i < classes) {
                    e[i] = t[j];
                    const uint64_t mg = (uint64_t)(mag128(t[j]) >> msh);
                    m = mg > m ? mg : m;
                }
            }
        } else {
            int64_t p = 0;
            if (!taylor) {
                int64_t mx = INT64_MIN;
                for (int64_t i = lane; i < classes; i += 64) {
                    const int64_t xh = loss_xhat(a[i], s_a);
                    mx = xh > mx ? xh : mx;
                }
                p = wave_max_i64(mx) - 10;
            }
            i128 C = 0;
            for (int64_t i = lane; i < classes; i += 64) {
                const i128 t = loss_term(a[i], s_a, p);
                e[i] = t;
                C += t;
            }
            C = wave_sum_i128(C);
            // Lane i owns entries i, i+64, ...; the owner of the label's entry
            // subtracts C (a label outside [0, classes) contributes no term).
            if (y >= 0 && y < classes && (y & 63) == lane) e[y] -= C;
            for (int64_t i = lane; i < classes; i += 64) {
                const uint64_t mg = (uint64_t)(mag128(e[i]) >> msh);
                m = mg > m ? mg : m;
            }
        }
    }
    if (s_in < kLossMinSa && threadIdx.x == 0 && blockIdx.x == 0)
        atomicOr(&st->wflags[slot], NITI_FLAG_LOSS_SA);
    block_publish_max(st, slot, m, snap);
}

// Algorithm 3, nearest, or stochastic (the draw's top bp bits against the
// fraction; past 64 fraction bits, the draw against the fraction's top 64
// bits) on a 128-bit value with binary point bp <= 126.
__device__ __forceinline__ int8_t round_i128(i128 v, int bp, int mode, uint64_t draw) {
    const u128 x = mag128(v);
    u128 q = x >> bp;
    if (bp > 0) {
        const u128 f = x & (((u128)1 << bp) - 1);
        if (mode == NITI_ROUND_RTN) {
            q += (x >> (bp - 1)) & 1u;
        } else if (mode == NITI_ROUND_SR) {
            q += bp <= 64 ? ((u128)(draw >> (64 - bp)) < f ? 1u : 0u) : ((u128)draw < (f >> (bp - 64)) ? 1u : 0u);
        } else {
            const int odd = bp & 1, h = (bp - odd) >> 1;
            const u128 fe = f >> odd;
            q += (fe >> h) > (fe & (((u128)1 << h) - 1)) ? 1u : 0u;
        }
    }
    const int qi = q < 127 ? (int)q : 127;
    return (int8_t)(v < 0 ? -qi : qi);
}

// Rounds e128 with the call's block binary point (finishing launch); each
// thread issues its LR loads before any store.
constexpr int LR = 4;
__global__ void loss_round_kernel(const i128* __restrict__ e128, int8_t* __restrict__ err, int64_t n, int mode,
                                  const int8_t* __restrict__ s_logits, niti_stats* st) {
    const int msh = loss_max_shift(loss_eval_sa((int)*s_logits));
    const uint64_t mx = shared_call_state(st).mx;
    const int b = mx ? bitlen64(mx) + msh : 0;
    const int bp = b > 7 ? b - 7 : 0;
    RoundK rk = make_round(bp < 31 ? bp : 31, mode);
    sr_key_recorded(rk, st);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += LR * stride) {
        i128 v[LR];
#pragma unroll
        for (int j = 0; j < LR; j++) v[j] = i0 + j * stride < n ? e128[i0 + j * stride] : (i128)0;
#pragma unroll
        for (int j = 0; j < LR; j++)
            if (i0 + j * stride < n)
                err[i0 + j * stride] = round_i128(v[j], bp, mode,
                                                  rk.sr ? sr_draw(rk.sr_seed, rk.sr_call, (uint64_t)(i0 + j * stride)) : 0ull);
    }
    if (is_finisher()) finish_call(st, 7, ExpArgs{nullptr, nullptr, nullptr}, 0u, 0, msh);
}

// ---------------------------------------------------------------------------
// Back-propagation filters.  Class (a, b) of a stride (sh, sw) layer uses
// filter rows r = r0 + sh*(T-1-t) and columns s = s0 + sw*(U-1-u), so that
// the class is a stride-1 correlation over dy:
//   wc[c][t][u][k] = w[k][r0 + sh (T-1-t)][s0 + sw (U-1-u)][c].
struct DgradClasses {
    DgradClass c[kMaxProblems];
    int n;
};


// Tiled form: one workgroup per (tap of a class, 64-channel block c0,
// 64-filter block k0).  The [64 k][64 c] slice of w at that tap is staged in
// LDS (row pitch 68 bytes, so column reads spread over banks) and written
// transposed as 64-byte runs out[c][t][u][k0 .. k0+63].
__global__ __launch_bounds__(256) void repack_dgrad_tiled_kernel(const int8_t* w, int8_t* out, DgradClasses cl,
                                                                 int K, int R, int S, int C, int sh, int sw) {
    __shared__ uint32_t tile32[64 * 17];   // [64 k][68 bytes]
    uint8_t* tile = (uint8_t*)tile32;
    int f = blockIdx.x;                    // flat tap index over the classes (uniform)
    int ci = 0;
    for (; ci < cl.n; ci++) {
        const int nt = cl.c[ci].T * cl.c[ci].U;
        if (f < nt) break;
        f -= nt;
    }
    if (ci >= cl.n) return;
    const DgradClass d = cl.c[ci];
    const int t = f / d.U, u = f - t * d.U;
    const int r = d.r0 + sh * (d.T - 1 - t);
    const int s = d.s0 + sw * (d.U - 1 - u);
    const int c0 = blockIdx.y * 64, k0 = blockIdx.z * 64;
    const int i = threadIdx.x;
    {
        const int kl = i >> 2, cb = (i & 3) * 16;
        const int k = k0 + kl;
        uint32_t v[4] = {0u, 0u, 0u, 0u};
        if (k < K) {
            const int8_t* src = w + (((int64_t)k * R + r) * S + s) * C + c0 + cb;
            if (c0 + cb + 16 <= C && (((uintptr_t)src) & 15) == 0) {
                const uint4 q = *(const uint4*)src;
                v[0] = q.x;
                v[1] = q.y;
                v[2] = q.z;
                v[3] = q.w;
            } else {
                for (int j = 0; j < 16 && c0 + cb + j < C; j++) v[j >> 2] |= (uint32_t)(uint8_t)src[j] << (8 * (j & 3));
            }
        }
#pragma unroll
        for (int q = 0; q < 4; q++) tile32[kl * 17 + (cb >> 2) + q] = v[q];
    }
    __syncthreads();
    {
        const int cc = i >> 2, kb = (i & 3) * 16;
        const int c = c0 + cc;
        if (c < C) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < 16; j++) v[j >> 2] |= (uint32_t)tile[(kb + j) * 68 + cc] << (8 * (j & 3));
            int8_t* dst = out + d.offset + (((int64_t)c * d.T + t) * d.U + u) * K + k0 + kb;
            if (k0 + kb + 16 <= K && (((uintptr_t)dst) & 15) == 0) {
                *(uint4*)dst = make_uint4(v[0], v[1], v[2], v[3]);
            } else {
                for (int j = 0; j < 16 && k0 + kb + j < K; j++) dst[j] = (int8_t)(v[j >> 2] >> (8 * (j & 3)));
            }
        }
    }
}

// ---------------------------------------------------------------------------
__global__ void quantize_kernel(const uint8_t* px, int8_t* x, int64_t n, int64_t c, int64_t h,
                                int64_t w, int64_t cp) {
    const int64_t total = n * h * w * cp;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t ch = i % cp;
        int64_t pix = i / cp;
        const int64_t col = pix % w;
        pix /= w;
        const int64_t row = pix % h;
        const int64_t img = pix / h;
        int8_t v = 0;
        if (ch < c) v = (int8_t)(px[((img * c + ch) * h + row) * w + col] >> 1);
        x[i] = v;
    }
}

__global__ void maxpool_fwd_kernel(const int8_t* x, int8_t* y, uint8_t* idx, int64_t n, int64_t h,
                                   int64_t w, int64_t c) {
    const int64_t H2 = h / 2, W2 = w / 2, total = n * H2 * W2 * c;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t ch = i % c;
        int64_t t = i / c;
        const int64_t j = t % W2;
        t /= W2;
        const int64_t r = t % H2;
        const int64_t img = t / H2;
        const int8_t* b = x + ((img * h + 2 * r) * w + 2 * j) * c + ch;
        int8_t v[4] = {b[0], b[c], b[w * c], b[w * c + c]};
        int best = 0;
        for (int q = 1; q < 4; q++)
            if (v[q] > v[best]) best = q;
        y[i] = v[best];
        idx[i] = (uint8_t)best;
    }
}

__global__ void maxpool_bwd_kernel(const int8_t* dy, const uint8_t* idx, int8_t* dx, int64_t n,
                                   int64_t h, int64_t w, int64_t c) {
    // One thread per input element: it takes dy where its window picked it.
    const int64_t total = n * h * w * c;
    const int64_t W2 = w / 2, H2 = h / 2;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const int64_t ch = i % c;
        int64_t t = i / c;
        const int64_t col = t % w;
        t /= w;
        const int64_t row = t % h;
        const int64_t img = t / h;
        const int64_t o = ((img * H2 + row / 2) * W2 + col / 2) * c + ch;
        const int pos = (int)((row & 1) * 2 + (col & 1));
        dx[i] = idx[o] == pos ? dy[o] : (int8_t)0;
    }
}

// Zero-padded copy, one wave per padded row (image * hp + row): the lanes
// take the row's dwords 64 apart, each issuing all its loads before its
// stores; columns and rows outside the image are zeros.
constexpr int kPadU = 4;   // dwords per lane and pass
struct PadArgs {
    const uint32_t* x;
    uint32_t* xp;
    uint32_t len, rows;
    int32_t h, w, c4, hp, ph, pw;
};

__device__ __forceinline__ void pad_rows(const PadArgs& a, uint32_t blk) {
    const uint32_t* __restrict__ x = a.x;
    uint32_t* __restrict__ xp = a.xp;
    const uint32_t len = a.len, rows = a.rows;
    const int32_t h = a.h, w = a.w, c4 = a.c4, hp = a.hp, ph = a.ph, pw = a.pw;
    const uint32_t r = blk * 4u + (threadIdx.x >> 6);
    if (r >= rows) return;
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t img = r / (uint32_t)hp;
    const int row = (int)(r - img * (uint32_t)hp) - ph;
    const bool rowok = row >= 0 && row < h;
    // dword index in x of padded column 0 of this row (negative values are
    // never used: only in-image columns are read)
    const int64_t base = (((int64_t)img * h + row) * w - pw) * c4;
    const uint32_t lo = (uint32_t)(pw * c4), hi = (uint32_t)((pw + w) * c4);
    uint32_t* dst = xp + (size_t)r * len;
    for (uint32_t j0 = lane; j0 < len; j0 += 64u * kPadU) {
        uint32_t v[kPadU];
#pragma unroll
        for (int u = 0; u < kPadU; u++) {
            const uint32_t j = j0 + 64u * u;
            v[u] = (rowok && j >= lo && j < hi) ? x[base + j] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kPadU; u++) {
            const uint32_t j = j0 + 64u * u;
            if (j < len) dst[j] = v[u];
        }
    }
}

__global__ __launch_bounds__(256) void pad_image_kernel(PadArgs a) { pad_rows(a, blockIdx.x); }

// Window filter of few-channel layers: w [k][r][s*c] -> wr [k][ktot], each
// filter row r at r*lw (zero past s*c and past the r rows).
struct WinArgs {
    const int8_t* w;
    int8_t* wr;
    int64_t k, r, sc, lw, ktot;
};

__device__ __forceinline__ void repack_window(const WinArgs& a, int64_t first, int64_t stride) {
    const int64_t total = a.k * a.ktot;
    for (int64_t i = first; i < total; i += stride) {
        const int64_t kk = i / a.ktot, t = i - kk * a.ktot;
        const int64_t row = t / a.lw, j = t - row * a.lw;
        a.wr[i] = (row < a.r && j < a.sc) ? a.w[(kk * a.r + row) * a.sc + j] : (int8_t)0;
    }
}

// Both preparations of a few-channel convolution in one launch: workgroups
// below pad_blocks copy the padded image, the others repack the filter.
__global__ __launch_bounds__(256) void pad_repack_kernel(PadArgs pa, WinArgs wa, uint32_t pad_blocks) {
    if (blockIdx.x < pad_blocks) {
        pad_rows(pa, blockIdx.x);
    } else {
        const int64_t b = blockIdx.x - pad_blocks;
        repack_window(wa, b * blockDim.x + threadIdx.x, (int64_t)(gridDim.x - pad_blocks) * blockDim.x);
    }
}


__global__ void relu_mask_kernel(int8_t* e, const int8_t* a, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        if (a[i] <= 0) e[i] = 0;
}

// Dropout: element i is kept when the top byte of its draw (the stochastic
// rounding generator, keyed by seed, call and i) is at least drop256.
__global__ void dropout_fwd_kernel(const int8_t* x, int8_t* y, uint8_t* keep, int64_t n, uint64_t seed,
                                   uint32_t call, uint32_t drop256, const int8_t* s_x, int8_t* s_y, int exp_add) {
    if (s_x && blockIdx.x == 0 && threadIdx.x == 0) {
        const int s = (int)*s_x + exp_add;
        *s_y = (int8_t)(s > 127 ? 127 : (s < -128 ? -128 : s));
    }
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const uint32_t k = (uint32_t)(sr_draw(seed, call, (uint64_t)i) >> 56) >= drop256 ? 1u : 0u;
        keep[i] = (uint8_t)k;
        y[i] = k ? x[i] : (int8_t)0;
    }
}

__global__ void dropout_bwd_kernel(const int8_t* dy, const uint8_t* keep, int8_t* dx, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dx[i] = keep[i] ? dy[i] : (int8_t)0;
}

}  // namespace

hipError_t fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(n, 16)), dim3(kThreads), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t max_abs_i32(const int32_t* x, int64_t n, niti_stats* st, hipStream_t s) {
    hipLaunchKernelGGL(max_abs_i32_kernel, dim3(grid_for(n, 8, 256)), dim3(kThreads), 0, s, x, n, st);
    return hipGetLastError();
}

hipError_t round_i32_run(const int32_t* x, int8_t* y, int64_t n, int bp, int target, int mode,
                         niti_stats* st, ExpArgs ex, hipStream_t s) {
    hipLaunchKernelGGL(round_i32_kernel, dim3(grid_for(n, 8)), dim3(kThreads), 0, s, x, y, n, bp,
                       target, mode, st, ex);
    return hipGetLastError();
}

hipError_t reduce_max_run(const int32_t* part, int splits, int32_t* g32, int64_t n, niti_stats* st,
                          hipStream_t s) {
    if (n > 0 && n % 4 == 0 && splits >= 1 && splits <= 8) {
        // At most one workgroup per CU: each folds its maximum in with one
        // atomic, and atomics on the one address serialize.
        const int g = grid_for(n / 4, 1, 256);
#define NITI_FLAT(NZ)                                                                                             \
    case NZ:                                                                                                      \
        hipLaunchKernelGGL(reduce_max_flat_kernel<NZ>, dim3(g), dim3(256), 0, s, part, g32, n, st);               \
        break;
        switch (splits) {
            NITI_FLAT(1)
            NITI_FLAT(2)
            NITI_FLAT(3)
            NITI_FLAT(4)
            NITI_FLAT(5)
            NITI_FLAT(6)
            NITI_FLAT(7)
            NITI_FLAT(8)
        }
#undef NITI_FLAT
        return hipGetLastError();
    }
    if (n > 0 && n % 4 == 0 && splits > 8) {
        // waves per 256 elements: one below 32 splits, else four
        const int g = splits < 32 ? 1 : 4;
        const int64_t passes = (n + 256 * (4 / g) - 1) / (256 * (4 / g));
        const int64_t blocks = passes < 256 ? passes : 256;
#define NITI_MANY(G)                                                                                              \
    case G:                                                                                                       \
        hipLaunchKernelGGL(reduce_max_many_kernel<G>, dim3((unsigned)blocks), dim3(256), 0, s, part, splits, g32,  \
                           n, st);                                                                                \
        break;
        switch (g) {
            NITI_MANY(1)
            NITI_MANY(4)
        }
#undef NITI_MANY
        return hipGetLastError();
    }
    const int64_t blocks = (n + 255) / 256;
    hipLaunchKernelGGL(reduce_max_kernel, dim3((unsigned)(blocks > 0 ? blocks : 1)), dim3(256), 0, s, part, splits,
                       g32, n, st);
    return hipGetLastError();
}

hipError_t update_run(int8_t* w, const int32_t* g32, int64_t n, int mu, int mode, niti_stats* st,
                      uint32_t static_flags, hipStream_t s) {
    hipLaunchKernelGGL(update_kernel, dim3(grid_for(n, 8)), dim3(kThreads), 0, s, w, g32, n, mu, mode, st,
                       static_flags);
    return hipGetLastError();
}

hipError_t loss_run(const int8_t* logits, const int8_t* s_logits, const int32_t* labels, int8_t* err,
                    void* ws, int64_t batch, int64_t classes, int mode, niti_stats* st, hipStream_t s) {
    i128* e128 = (i128*)ws;
    const int per_block = kThreads / 64;
    const int64_t blocks = (batch + per_block - 1) / per_block;
    const dim3 grid((unsigned)(blocks > 0 ? blocks : 1));
    if (classes <= 64 * 16)
        hipLaunchKernelGGL(loss_kernel<16>, grid, dim3(kThreads), 0, s, logits, s_logits, labels, e128, batch,
                           classes, st);
    else
        hipLaunchKernelGGL(loss_kernel<0>, grid, dim3(kThreads), 0, s, logits, s_logits, labels, e128, batch,
                           classes, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n = batch * classes;
    hipLaunchKernelGGL(loss_round_kernel, dim3(grid_for(n, LR)), dim3(kThreads), 0, s, e128, err, n, mode,
                       s_logits, st);
    return hipGetLastError();
}

hipError_t repack_dgrad_run(const int8_t* w, int8_t* out, const DgradClass* cls, int ncls, int K, int R,
                            int S, int C, int sh, int sw, hipStream_t s) {
    DgradClasses cl;
    cl.n = ncls;
    int64_t total = 0;
    for (int i = 0; i < ncls; i++) {
        cl.c[i] = cls[i];
        total = cls[i].offset + (int64_t)C * cls[i].T * cls[i].U * K;
    }
    if (total <= 0) return hipSuccess;
    int taps = 0;
    for (int i = 0; i < ncls; i++) taps += cls[i].T * cls[i].U;
    if (taps <= 0) return hipSuccess;
    hipLaunchKernelGGL(repack_dgrad_tiled_kernel, dim3((unsigned)taps, (unsigned)((C + 63) / 64), (unsigned)((K + 63) / 64)),
                       dim3(256), 0, s, w, out, cl, K, R, S, C, sh, sw);
    return hipGetLastError();
}

hipError_t quantize_run(const uint8_t* px, int8_t* x, int64_t n, int64_t c, int64_t h, int64_t w,
                        int64_t cp, hipStream_t s) {
    const int64_t total = n * h * w * cp;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(quantize_kernel, dim3(grid_for(total, 4)), dim3(kThreads), 0, s, px, x, n, c, h, w,
                       cp);
    return hipGetLastError();
}

hipError_t maxpool_fwd_run(const int8_t* x, int8_t* y, uint8_t* idx, int64_t n, int64_t h, int64_t w,
                           int64_t c, hipStream_t s) {
    const int64_t total = n * (h / 2) * (w / 2) * c;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(grid_for(total, 4)), dim3(kThreads), 0, s, x, y, idx, n, h,
                       w, c);
    return hipGetLastError();
}

hipError_t maxpool_bwd_run(const int8_t* dy, const uint8_t* idx, int8_t* dx, int64_t n, int64_t h,
                           int64_t w, int64_t c, hipStream_t s) {
    const int64_t total = n * h * w * c;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(grid_for(total, 4)), dim3(kThreads), 0, s, dy, idx, dx, n,
                       h, w, c);
    return hipGetLastError();
}

namespace {
hipError_t pad_args(const int8_t* x, int8_t* xp, int64_t n, int64_t h, int64_t w, int64_t c, int64_t hp, int64_t wp,
                    int64_t ph, int64_t pw, PadArgs& a) {
    const int64_t rows = n * hp;
    const int64_t len = wp * (c / 4);
    if (rows * len >= ((int64_t)1 << 32) || rows >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    a.x = (const uint32_t*)x;
    a.xp = (uint32_t*)xp;
    a.len = (uint32_t)(len > 0 ? len : 0);
    a.rows = (uint32_t)(rows > 0 && len > 0 ? rows : 0);
    a.h = (int32_t)h;
    a.w = (int32_t)w;
    a.c4 = (int32_t)(c / 4);
    a.hp = (int32_t)hp;
    a.ph = (int32_t)ph;
    a.pw = (int32_t)pw;
    return hipSuccess;
}
}  // namespace

hipError_t pad_image_run(const int8_t* x, int8_t* xp, int64_t n, int64_t h, int64_t w, int64_t c, int64_t hp,
                         int64_t wp, int64_t ph, int64_t pw, hipStream_t s) {
    PadArgs a;
    hipError_t e = pad_args(x, xp, n, h, w, c, hp, wp, ph, pw, a);
    if (e != hipSuccess) return e;
    if (a.rows == 0) return hipSuccess;
    hipLaunchKernelGGL(pad_image_kernel, dim3((a.rows + 3) / 4), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t pad_repack_run(const int8_t* x, int8_t* xp, int64_t n, int64_t h, int64_t w, int64_t c, int64_t hp,
                          int64_t wp, int64_t ph, int64_t pw, const int8_t* wt, int8_t* wr, int64_t k, int64_t r,
                          int64_t sc, int64_t lw, int64_t ktot, hipStream_t s) {
    PadArgs a;
    hipError_t e = pad_args(x, xp, n, h, w, c, hp, wp, ph, pw, a);
    if (e != hipSuccess) return e;
    const WinArgs wa{wt, wr, k, r, sc, lw, ktot};
    const uint32_t pad_blocks = (a.rows + 3) / 4;
    const int64_t total = k * ktot;
    const uint32_t rep_blocks = total > 0 ? (uint32_t)grid_for(total, 4) : 0u;
    if (pad_blocks + rep_blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(pad_repack_kernel, dim3(pad_blocks + rep_blocks), dim3(kThreads), 0, s, a, wa, pad_blocks);
    return hipGetLastError();
}

hipError_t zero_classes_run(int8_t* out, int64_t n, int64_t h, int64_t w, int64_t c, int st, uint32_t mask,
                            hipStream_t s) {
    if (mask == 0 || n * h * w * c == 0) return hipSuccess;
    hipLaunchKernelGGL(zero_classes_kernel, dim3((uint32_t)(n * h)), dim3(kThreads), 0, s, (uint32_t*)out,
                       (int32_t)h, (int32_t)w, (int32_t)(c / 4), st, mask);
    return hipGetLastError();
}


hipError_t relu_mask_run(int8_t* e, const int8_t* a, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(relu_mask_kernel, dim3(grid_for(n, 4)), dim3(kThreads), 0, s, e, a, n);
    return hipGetLastError();
}

hipError_t dropout_fwd_run(const int8_t* x, int8_t* y, uint8_t* keep, int64_t n, uint64_t seed, uint32_t call,
                           uint32_t drop256, const int8_t* s_x, int8_t* s_y, int exp_add, hipStream_t s) {
    if (n <= 0 && !s_x) return hipSuccess;
    hipLaunchKernelGGL(dropout_fwd_kernel, dim3(grid_for(n > 0 ? n : 1, 4)), dim3(kThreads), 0, s, x, y, keep, n, seed,
                       call, drop256, s_x, s_y, exp_add);
    return hipGetLastError();
}

hipError_t dropout_bwd_run(const int8_t* dy, const uint8_t* keep, int8_t* dx, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(dropout_bwd_kernel, dim3(grid_for(n, 4)), dim3(kThreads), 0, s, dy, keep, dx, n);
    return hipGetLastError();
}

}  // namespace niti
