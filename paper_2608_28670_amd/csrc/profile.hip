// Per-kernel-class timing with HIP events recorded on the launch stream.
// Enabled classes bracket each launch with a start/stop event pair drawn from
// a pool created at enable time; collect waits on the events and sums them.
#include <vector>

#include "hip_common.h"

namespace bc {

namespace {
struct ClassTimer {
    bool on = false;
    int used = 0;
    std::vector<hipEvent_t> start, stop;
};
ClassTimer g_timer[PROF_NCLASS];

void release(ClassTimer& t) {
    for (hipEvent_t e : t.start) (void)hipEventDestroy(e);
    for (hipEvent_t e : t.stop) (void)hipEventDestroy(e);
    t.start.clear();
    t.stop.clear();
    t.on = false;
    t.used = 0;
}
}  // namespace

void prof_begin(int cls, hipStream_t s) {
    ClassTimer& t = g_timer[cls];
    if (!t.on || t.used >= (int)t.start.size()) return;
    (void)hipEventRecord(t.start[t.used], s);
}

void prof_end(int cls, hipStream_t s) {
    ClassTimer& t = g_timer[cls];
    if (!t.on || t.used >= (int)t.start.size()) return;
    (void)hipEventRecord(t.stop[t.used], s);
    ++t.used;
}

}  // namespace bc

using namespace bc;

extern "C" {

int bc_profile_enable(int kernel_class, int max_launches) {
    clear_error();
    if (kernel_class < 0 || kernel_class >= PROF_NCLASS) return fail(BC_ERR_INVALID_ARG, "class %d", kernel_class);
    if (max_launches < 1 || max_launches > 1 << 20) return fail(BC_ERR_INVALID_ARG, "max_launches %d", max_launches);
    ClassTimer& t = g_timer[kernel_class];
    release(t);
    t.start.resize(max_launches);
    t.stop.resize(max_launches);
    for (int i = 0; i < max_launches; ++i) {
        if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess) {
            t.start.resize(i);
            t.stop.resize(i);
            release(t);
            return fail(BC_ERR_HIP, "hipEventCreate failed");
        }
    }
    t.on = true;
    return BC_OK;
}

int bc_profile_collect(int kernel_class, double* total_ms, int* launches) {
    clear_error();
    if (kernel_class < 0 || kernel_class >= PROF_NCLASS) return fail(BC_ERR_INVALID_ARG, "class %d", kernel_class);
    ClassTimer& t = g_timer[kernel_class];
    double sum = 0.0;
    for (int i = 0; i < t.used; ++i) {
        if (hipEventSynchronize(t.stop[i]) != hipSuccess) { release(t); return fail(BC_ERR_HIP, "event sync"); }
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess) { release(t); return fail(BC_ERR_HIP, "elapsed"); }
        sum += ms;
    }
    if (total_ms) *total_ms = sum;
    if (launches) *launches = t.used;
    release(t);
    return BC_OK;
}

}  // extern "C"
