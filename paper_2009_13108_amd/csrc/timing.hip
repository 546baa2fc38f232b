// Kernel timing hooks: HIP event pairs recorded on a call's stream around
// its contraction launches, summed per family on request.  Host code only.
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
size_t g_used = 0;

}  // namespace

int timing_begin(int family, hipStream_t s) {
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
    }
    const int i = (int)g_used;
    if (hipEventRecord(g_pool[i].a, s) != hipSuccess) return -1;
    g_family[i] = family;
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
    if (family != NITI_TIMING_IGEMM && family != NITI_TIMING_WGRAD) return NITI_ERR_ARG;
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

}  // extern "C"
