// Kernel timing hooks: HIP event pairs recorded on a call's stream around
// its launches, summed per family or read one by one on request; and the
// int8 MFMA loop that measures the matrix cores' sustained rate.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "niti_internal.h"

namespace niti {

namespace {

struct Pair {
    hipEvent_t a, b;
};

bool g_on = false;
std::vector<Pair> g_pool;          // events created so far, reused after a restart
std::vector<int> g_family;         // family of pair i (i < g_used)
std::vector<const char*> g_name;   // kernel of pair i (NITI_TIMING_KERNEL) or NULL
size_t g_used = 0;

}  // namespace

const char* kernel_label(const char* fmt, ...) {
    static std::mutex mu;
    static std::unordered_map<std::string, std::string*> names;   // held for the process
    char buf[128];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    std::lock_guard<std::mutex> lock(mu);
    auto it = names.find(buf);
    if (it == names.end()) it = names.emplace(buf, new std::string(buf)).first;
    return it->second->c_str();
}

bool timing_on() { return g_on; }

int timing_begin(int family, hipStream_t s, const char* name) {
    if (!g_on) return -1;
    if (g_used == g_pool.size()) {
        Pair p{};
        if (hipEventCreate(&p.a) != hipSuccess) return -1;
        if (hipEventCreate(&p.b) != hipSuccess) {
            (void)hipEventDestroy(p.a);
            return -1;
        }
        g_pool.push_back(p);
        g_family.push_back(0);
        g_name.push_back(nullptr);
    }
    const int i = (int)g_used;
    if (hipEventRecord(g_pool[i].a, s) != hipSuccess) return -1;
    g_family[i] = family;
    g_name[i] = name;
    g_used++;
    return i;
}

void timing_end(int idx, hipStream_t s) {
    if (idx < 0) return;
    if (hipEventRecord(g_pool[idx].b, s) != hipSuccess) g_family[idx] = -1;  // dropped from the sums
}

}  // namespace niti

using namespace niti;

extern "C" {

niti_status niti_timing_enable(int on) {
    g_on = on != 0;
    if (g_on) g_used = 0;
    return NITI_OK;
}

niti_status niti_timing_read(int family, double* ms, int64_t* calls) {
    if (family < NITI_TIMING_IGEMM || family > NITI_TIMING_LOSS) return NITI_ERR_ARG;
    if (!ms || !calls) return NITI_ERR_NULL;
    double tot = 0.0;
    int64_t n = 0;
    for (size_t i = 0; i < g_used; i++) {
        if (g_family[i] != family) continue;
        if (hipEventSynchronize(g_pool[i].b) != hipSuccess) return NITI_ERR_HIP;
        float t = 0.f;
        if (hipEventElapsedTime(&t, g_pool[i].a, g_pool[i].b) != hipSuccess) return NITI_ERR_HIP;
        tot += t;
        n++;
    }
    *ms = tot;
    *calls = n;
    return NITI_OK;
}

niti_status niti_timing_record(int64_t i, int* family, const char** name, double* ms) {
    if (!family || !name || !ms) return NITI_ERR_NULL;
    if (i < 0 || (size_t)i >= g_used) return NITI_ERR_ARG;
    *family = g_family[i];
    *name = g_name[i] ? g_name[i] : "";
    *ms = -1.0;
    if (g_family[i] < 0) return NITI_OK;
    if (hipEventSynchronize(g_pool[i].b) != hipSuccess) return NITI_ERR_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, g_pool[i].a, g_pool[i].b) != hipSuccess) return NITI_ERR_HIP;
    *ms = t;
    return NITI_OK;
}

}  // extern "C"

namespace niti {
namespace {

// Eight independent 32x32x32 int8 MFMA chains per wave on register operands,
// `iters` rounds; the accumulators are summed into one word per lane so the
// work is kept.  Four waves per workgroup, one per SIMD.
__global__ __launch_bounds__(256) void mfma_loop_kernel(int64_t iters, int32_t* out, int64_t n_out) {
    const int t = (int)threadIdx.x;
    const v4i a = {t, 3 * t + 1, 5 * t + 2, 7 * t + 3};
    const v4i b = {11 * t + 4, 13 * t + 5, 17 * t + 6, 19 * t + 7};
    v16i acc[8];
#pragma unroll
    for (int j = 0; j < 8; j++) acc[j] = v16i{};
    for (int64_t i = 0; i < iters; i++) {
#pragma unroll
        for (int j = 0; j < 8; j++) acc[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[j], 0, 0, 0);
    }
    int32_t s = 0;
#pragma unroll
    for (int j = 0; j < 8; j++)
#pragma unroll
        for (int e = 0; e < 16; e++) s += acc[j][e];
    const int64_t o = (int64_t)blockIdx.x * 256 + t;
    if (o < n_out) out[o] = s;
}

}  // namespace
}  // namespace niti

extern "C" {

niti_status niti_mfma_loop(int64_t iters, int64_t workgroups, int32_t* out, void* stream) {
    if (!out) return NITI_ERR_NULL;
    if (iters < 0 || workgroups < 1 || workgroups > (1 << 20)) return NITI_ERR_SHAPE;
    hipLaunchKernelGGL(niti::mfma_loop_kernel, dim3((unsigned)workgroups), dim3(256), 0, (hipStream_t)stream, iters,
                       out, workgroups * 256);
    return hipGetLastError() == hipSuccess ? NITI_OK : NITI_ERR_HIP;
}

}  // extern "C"
