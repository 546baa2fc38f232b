// Device-side building blocks shared by the NITI kernels: magnitude
// rounding (Algorithm 3 and round-to-nearest), the effective bitwidth of a
// block maximum (Section 3.2), fast unsigned division for index decoding,
// wave reductions and the per-call statistics epilogue.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "niti.h"

namespace niti {

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Effective bitwidth B(v) of a magnitude: bits needed to write it (Section 3.2).
__host__ __device__ inline int bitlen64(uint64_t m) {
#ifdef __HIP_DEVICE_COMPILE__
    return m ? 64 - __clzll((long long)m) : 0;
#else
    return m ? 64 - __builtin_clzll(m) : 0;
#endif
}

// Binary point for a block: shift just enough that the maximum keeps
// `target` magnitude bits (Algorithm 1: max(0, b - 7); Section 3.3: b - m_u).
__host__ __device__ inline int block_bp(uint64_t mx, int target) {
    int bp = bitlen64(mx) - target;
    return bp < 0 ? 0 : bp;
}

// Constants of one rounding shift, uniform over a whole tensor.
struct RoundK {
    uint32_t bp;     // binary point (0..31 for int32 data, 0..63 for int64)
    uint32_t odd;    // 1 when bp is odd: the lowest fraction bit is dropped
    uint32_t h;      // half width of the (even) fraction
    uint64_t fmask;  // bp low bits
    uint64_t hmask;  // h low bits
    int rtn;         // 1: round to nearest instead
    int sr;          // 1: stochastic rounding (draws keyed by sr_seed, sr_call, element index)
    uint64_t sr_seed;
    uint32_t sr_call;
    // Closed form of the 32-bit rounding (round_psr_mag_fast): with
    // r = (x >> odd) & hmask, the rounded value is (x + r * k1 + c0) >> bp.
    int32_t k1;      // -(2^h + 1) * 2^odd
    int32_t c0;      // (2^2h - 2^h) * 2^odd
};

__host__ __device__ inline RoundK make_round(int bp, int mode) {
    RoundK k;
    k.bp = (uint32_t)bp;
    k.odd = (uint32_t)bp & 1u;
    k.h = ((uint32_t)bp - k.odd) >> 1;
    k.fmask = bp >= 64 ? ~0ull : ((1ull << bp) - 1ull);
    k.hmask = (1ull << k.h) - 1ull;
    k.rtn = mode == NITI_ROUND_RTN;
    k.sr = mode == NITI_ROUND_SR;
    k.sr_seed = 0;
    k.sr_call = 0;
    k.k1 = k.h < 16 ? -(int32_t)(((1u << k.h) + 1u) << k.odd) : 0;
    k.c0 = k.h < 16 ? (int32_t)((((1u << (2 * k.h)) - (1u << k.h))) << k.odd) : 0;
    return k;
}

// Algorithm 3 in closed form for 32-bit data.  Write the fraction (odd
// bit dropped) as thi * 2^h + rlo.  Adding (2^2h - 2^h - rlo (2^h + 1))
// 2^odd to x raises the integer part by one exactly when thi > rlo and
// leaves it otherwise, so q + up = (x + rlo * k1 + c0) >> bp.
// Magnitude form (x = |v| <= 2^31): exact for every bp <= 31.
__device__ __forceinline__ uint32_t round_psr_mag_fast(uint32_t x, const RoundK& k) {
    const uint32_t rlo = __builtin_amdgcn_ubfe(x, k.odd, k.h);
    const uint32_t z = (uint32_t)(__mul24((int32_t)rlo, k.k1) + k.c0);
    return min((x + z) >> k.bp, 127u);
}

// Pseudo stochastic rounding of an unsigned 32-bit magnitude (Algorithm 3):
// integer part q = x >> bp, fraction f = low bp bits (odd bp: its lowest
// bit dropped); q is bumped when the upper half of f exceeds the lower half,
// the lower half standing in for a random draw.  Held at 127.
__device__ __forceinline__ uint32_t round_mag32(uint32_t x, const RoundK& k) {
    if (!k.rtn) return round_psr_mag_fast(x, k);
    uint32_t q = x >> k.bp;
    q += k.bp ? ((x >> (k.bp - 1)) & 1u) : 0u;
    return q < 127u ? q : 127u;
}

__device__ __forceinline__ uint64_t round_mag64(uint64_t x, const RoundK& k) {
    uint64_t q = k.bp >= 64 ? 0 : (x >> k.bp);
    if (k.rtn) {
        q += k.bp ? ((x >> (k.bp - 1)) & 1ull) : 0ull;
    } else {
        uint64_t f = (x & k.fmask) >> k.odd;
        uint64_t thi = f >> k.h;
        uint64_t rlo = f & k.hmask;
        q += thi > rlo ? 1ull : 0ull;
    }
    return q < 127ull ? q : 127ull;
}

// Stochastic rounding (Section 3.4): round the magnitude up with
// probability f / 2^bp, the draw being output number call * 2^40 + idx + 1
// of a SplitMix64 stream (Steele, Lea and Flood, "Fast splittable
// pseudorandom number generators", OOPSLA 2014) seeded with seed.
__device__ __forceinline__ uint64_t sr_draw(uint64_t seed, uint32_t call, uint64_t idx) {
    uint64_t z = seed + ((((uint64_t)call) << 40) + idx + 1ull) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// |v| rounded with binary point bp <= 31: up exactly when the top bp bits of
// the draw are below the fraction; held at 127.
__device__ __forceinline__ uint32_t round_sr_mag32(uint32_t x, const RoundK& k, uint64_t idx) {
    uint32_t q = x >> k.bp;
    if (k.bp) {
        const uint32_t f = x & ((1u << k.bp) - 1u);
        q += (uint32_t)(sr_draw(k.sr_seed, k.sr_call, idx) >> (64 - k.bp)) < f ? 1u : 0u;
    }
    return q < 127u ? q : 127u;
}

__device__ __forceinline__ uint32_t mag32(int32_t v) {
    return v < 0 ? 0u - (uint32_t)v : (uint32_t)v;
}

__device__ __forceinline__ int8_t round_i32(int32_t v, const RoundK& k) {
    int32_t q = (int32_t)round_mag32(mag32(v), k);
    return (int8_t)(v < 0 ? -q : q);
}

// round_i32 with the element index that keys a stochastic draw.
__device__ __forceinline__ int8_t round_i32_at(int32_t v, const RoundK& k, uint64_t idx) {
    if (!k.sr) return round_i32(v, k);
    const int32_t q = (int32_t)round_sr_mag32(mag32(v), k, idx);
    return (int8_t)(v < 0 ? -q : q);
}

__device__ __forceinline__ int8_t round_i64(int64_t v, const RoundK& k) {
    uint64_t m = v < 0 ? 0ull - (uint64_t)v : (uint64_t)v;
    int32_t q = (int32_t)round_mag64(m, k);
    return (int8_t)(v < 0 ? -q : q);
}

// ---------------------------------------------------------------------------
// Unsigned division by a runtime-constant divisor d >= 1 for n < 2^31
// (multiply-high with a precomputed magic number, as in Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994).
struct FastDiv {
    uint32_t d;
    uint32_t mul;
    uint32_t shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d ? d : 1;
    uint32_t l = 0;
    while ((1ull << l) < f.d) l++;
    // mul = floor(2^32 (2^l - d) / d) + 1, quotient = (mulhi(n, mul) + n) >> l
    f.mul = (uint32_t)((((1ull << l) - f.d) << 32) / f.d + 1);
    f.shift = l;
    return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
    uint32_t t = __umulhi(n, f.mul);
    return (uint32_t)(((uint64_t)t + n) >> f.shift);
}

// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        uint64_t u = __shfl_xor(v, o, kWave);
        v = u > v ? u : v;
    }
    return v;
}

// ---------------------------------------------------------------------------
// Direct-to-LDS loads issued as inline assembly.  Kernels that read their
// LDS ring with transpose reads use these: the compiler cannot tell which
// ring stage a transpose read touches, so with the load builtin it waits for
// every direct-to-LDS load in flight before each read, which serializes the
// ring.  Issued this way the loads are invisible to its wait counting, and
// the kernel's own per-stage vmcnt waits and barriers order them.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (stride 0): base address and size in bytes; accesses
// at offsets >= bytes return zeros.  Uniform.
__device__ __forceinline__ u32x4 raw_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    u32x4 r;
    r.x = __builtin_amdgcn_readfirstlane((uint32_t)a);
    r.y = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xFFFFu);
    r.z = __builtin_amdgcn_readfirstlane(bytes);
    r.w = 0x00020000u;
    return r;
}

// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16 bytes per lane from offset voff + soff of the buffer to LDS address
// m0 + 16 * lane (m0 uniform).
__device__ __forceinline__ void lds_dma16(u32x4 rs, uint32_t m0, uint32_t voff, uint32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(rs), "s"(soff)
                 : "memory", "m0");
}

// The same with the LDS address given as the sum of two uniform values,
// formed directly in m0.
__device__ __forceinline__ void lds_dma16_at(u32x4 rs, uint32_t base, uint32_t off, uint32_t voff, uint32_t soff) {
    asm volatile("s_add_u32 m0, %0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %3, %4 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(base)), "s"(__builtin_amdgcn_readfirstlane(off)), "v"(voff),
                   "s"(rs), "s"(soff)
                 : "memory", "m0", "scc");
}

// Wave maximum of a 32-bit value with row-local DPP steps and four lane
// reads; the result is uniform.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
    return max(max(a, b), max(c, d));
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ int64_t wave_max_i64(int64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        int64_t u = __shfl_xor(v, o, kWave);
        v = u > v ? u : v;
    }
    return v;
}

// ---------------------------------------------------------------------------
// Statistics protocol.  A call made with a stats block runs an accumulating
// launch (every workgroup folds its maximum into acc_max[slot], slot =
// calls & 1) and later a finishing launch in which one thread derives b and
// bp, records them, clears the other slot for the next call and counts the
// call.  Each field is written only in a launch where no other workgroup
// reads it, so no completion counter is needed.

__device__ __forceinline__ int call_slot(const niti_stats* st) { return (int)(st->calls & 1u); }

__device__ __forceinline__ uint64_t load_acc(niti_stats* st, int slot) {
    return __hip_atomic_load(&st->acc_max[slot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The maximum of the call in progress: both slots and the slot index are
// read at once (one memory round trip instead of two dependent ones) and
// the current slot's value is selected.
__device__ __forceinline__ uint64_t load_cur_acc(niti_stats* st) {
    const uint64_t a0 = load_acc(st, 0), a1 = load_acc(st, 1);
    return (st->cur & 1) ? a1 : a0;
}

// The maximum of the call in progress and the guess that call tried, for a
// finishing launch: read by one thread of the workgroup and handed to the
// others through LDS.  All of a launch's requests go to the one stats
// address and queue behind each other, so one request per workgroup instead
// of one per wave keeps a launch whose guess was right short.  Every thread
// of the workgroup must call it; lds is 16 bytes of LDS the kernel may
// reuse afterwards.
struct CallState {
    uint64_t mx;
    int hint;
};
__device__ __forceinline__ CallState shared_call_state(niti_stats* st, void* lds) {
    uint64_t* sh = (uint64_t*)lds;
    if (threadIdx.x == 0) {
        sh[0] = load_cur_acc(st);
        sh[1] = (uint64_t)(uint32_t)st->hint_used;
    }
    __syncthreads();
    const CallState r{sh[0], (int)(uint32_t)sh[1]};
    __syncthreads();   // every thread has its copy before the LDS is reused
    return r;
}
// The same for kernels without LDS of their own (16 bytes of static LDS).
__device__ __forceinline__ CallState shared_call_state(niti_stats* st) {
    __shared__ uint64_t sh[2];
    return shared_call_state(st, sh);
}

// Snapshot of the tensor maximum taken when a workgroup starts (by thread 0,
// the one that publishes).  The maximum only grows, so a workgroup maximum
// not above the snapshot can be skipped without a fresh read at the end.
__device__ __forceinline__ uint64_t max_snapshot(niti_stats* st, int slot) {
    return threadIdx.x == 0 ? load_acc(st, slot) : 0ull;
}

// Fold a value into the tensor maximum (no-return atomic).
__device__ __forceinline__ void publish_max(niti_stats* st, int slot, uint64_t m, uint64_t snap) {
    if (m > snap) atomicMax((unsigned long long*)&st->acc_max[slot], (unsigned long long)m);
}

// Workgroup-wide maximum folded in by thread 0.  Every thread calls it;
// red is LDS scratch for one value per wave; snap is max_snapshot().
__device__ __forceinline__ void block_publish_max_in(niti_stats* st, int slot, uint64_t m, uint64_t* red,
                                                     uint64_t snap) {
    m = wave_max_u64(m);
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    if (lane == 0) red[wv] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int nw = (blockDim.x + kWave - 1) / kWave;
        uint64_t r = 0;
        for (int i = 0; i < nw; i++) r = red[i] > r ? red[i] : r;
        publish_max(st, slot, r, snap);
    }
}

// Workgroup maximum of values below 2^32 (32-bit wave reductions), folded in
// by thread 0 with one atomic; red is LDS scratch for one value per wave and
// snap a snapshot held by thread 0.
__device__ __forceinline__ void block_publish_max32(niti_stats* st, int slot, uint32_t m, uint32_t* red,
                                                    uint64_t snap) {
    m = wave_max_u32(m);
    const int wv = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[wv] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int nw = (blockDim.x + kWave - 1) / kWave;
        uint32_t r = 0;
        for (int i = 0; i < nw; i++) r = max(r, red[i]);
        publish_max(st, slot, r, snap);
    }
}

__device__ __forceinline__ void block_publish_max(niti_stats* st, int slot, uint64_t m, uint64_t snap) {
    __shared__ uint64_t red[16];
    block_publish_max_in(st, slot, m, red, snap);
}

// In the accumulating launch: workgroup 0 records the slot and the guess
// this call tries, for the finishing launch.
__device__ __forceinline__ void begin_call(niti_stats* st, int slot, int hint) {
    if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) {
        st->cur = slot;
        st->hint_used = hint;
        st->sr_call = st->calls;   // the draw index c of this call, for its later launches
    }
}

// The stochastic-rounding key of the call in progress, for a launch after
// the accumulating one (the finishing thread increments calls meanwhile, so
// the index recorded by begin_call is read instead).
__device__ __forceinline__ void sr_key_recorded(RoundK& k, const niti_stats* st) {
    if (k.sr) {
        k.sr_seed = st->sr_seed;
        k.sr_call = st->sr_call;
    }
}
// The same in the accumulating launch itself (calls does not change during it).
__device__ __forceinline__ void sr_key_current(RoundK& k, const niti_stats* st) {
    if (k.sr) {
        k.sr_seed = st->sr_seed;
        k.sr_call = st->calls;
    }
}

// Exponent operands of a call that forms an output exponent.
struct ExpArgs {
    const int8_t* s_a;  // first operand exponent (or NULL)
    const int8_t* s_b;  // second operand exponent (or NULL)
    int8_t* s_out;      // output exponent (or NULL: not formed)
};

// The finishing launch's single thread: derive b and bp from the tensor
// maximum, form the output exponent (Algorithm 2: s_q = s_q32 + bp), record
// the statistics, make bp the next call's first guess, clear the other
// slot and count the call.
// Every value it reads is loaded before any is used (one memory round trip).
// max_shift: the maximum was folded in shifted right by that many bits (its
// effective bitwidth is then bitlen + max_shift; see the integer loss).
__device__ inline void finish_call(niti_stats* st, int target, ExpArgs ex, uint32_t static_flags,
                                   int hinted, int max_shift = 0) {
    const uint64_t a0 = load_acc(st, 0), a1 = load_acc(st, 1);
    const uint32_t f0 = __hip_atomic_load(&st->wflags[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t f1 = __hip_atomic_load(&st->wflags[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int cur = st->cur & 1;
    const int hint_used = st->hint_used;
    const uint32_t misses = st->misses, calls = st->calls;
    const int sa = ex.s_out && ex.s_a ? (int)*ex.s_a : 0;
    const int sb = ex.s_out && ex.s_b ? (int)*ex.s_b : 0;
    const uint64_t mx = cur ? a1 : a0;
    const uint32_t wf = cur ? f1 : f0;
    const int b = mx ? bitlen64(mx) + max_shift : 0;
    const int bp = b > target ? b - target : 0;
    uint32_t fl = wf | static_flags;
    if (hinted && bp != hint_used) {
        fl |= NITI_FLAG_HINT_MISS;
        st->misses = misses + 1;
    }
    int s = 0;
    if (ex.s_out) {
        s = sa + sb + bp;
        if (s > 127) { s = 127; fl |= NITI_FLAG_EXP_RANGE; }
        if (s < -128) { s = -128; fl |= NITI_FLAG_EXP_RANGE; }
        *ex.s_out = (int8_t)s;
    }
    st->max_abs = mx;
    st->b = b;
    st->bp = bp;
    st->flags = (int32_t)fl;
    st->s_out = s;
    st->bp_hint = bp;
    st->acc_max[cur ^ 1] = 0;
    st->wflags[cur ^ 1] = 0;
    st->calls = calls + 1;
}

// 0xFF in every byte of m that is positive as an int8, 0x00 elsewhere (the
// backward ReLU mask of four packed bytes), without per-byte compares: the
// low seven bits plus 0x7F carry into bit 7 exactly when they are not all
// zero, and no byte carries into the next.
__device__ __forceinline__ uint32_t positive_bytes(uint32_t m) {
    const uint32_t nz = (m & 0x7F7F7F7Fu) + 0x7F7F7F7Fu;
    const uint32_t pos = nz & ~m & 0x80808080u;
    return pos | (pos - (pos >> 7));
}

__device__ __forceinline__ bool is_finisher() {
    return blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0;
}

}  // namespace niti
