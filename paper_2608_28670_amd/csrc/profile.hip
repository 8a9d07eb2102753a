// Per-kernel-class timing with HIP events on the launch stream.  Inside a
// prof_begin/prof_end bracket of an enabled class, each kernel launch takes
// the next start/stop pair of a pool created at enable time and is launched
// with hipExtLaunchKernelGGL, which records the kernel's own start and end
// into them; collect waits on the events and sums the intervals.
#include <vector>

#include "hip_common.h"

namespace bc {

namespace {
struct ClassTimer {
    bool on = false;
    int used = 0;
    std::vector<hipEvent_t> start, stop;
    std::vector<double> work;
};
ClassTimer g_timer[PROF_NCLASS];

void release(ClassTimer& t) {
    for (hipEvent_t e : t.start) (void)hipEventDestroy(e);
    for (hipEvent_t e : t.stop) (void)hipEventDestroy(e);
    t.start.clear();
    t.stop.clear();
    t.work.clear();
    t.on = false;
    t.used = 0;
}
}  // namespace

thread_local int g_pending = -1;   // class of the open bracket on this thread, -1 if none
thread_local double g_pending_work = 0.0;   // its work, until the first launch takes it

void prof_begin(int cls, hipStream_t, double work) {
    g_pending = g_timer[cls].on ? cls : -1;
    g_pending_work = work;
}

void prof_end(int, hipStream_t) { g_pending = -1; }

bool prof_any_enabled() {
    for (const ClassTimer& t : g_timer)
        if (t.on) return true;
    return false;
}

bool prof_take(hipEvent_t* start, hipEvent_t* stop) {
    if (g_pending < 0) return false;
    ClassTimer& t = g_timer[g_pending];
    if (!t.on || t.used >= (int)t.start.size()) return false;
    *start = t.start[t.used];
    *stop = t.stop[t.used];
    t.work[t.used] = g_pending_work;
    g_pending_work = 0.0;
    ++t.used;
    return true;
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
    t.work.assign(max_launches, 0.0);
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

int bc_profile_records(int kernel_class, float* ms_out, double* work_out, int max_out, int* launches) {
    clear_error();
    if (kernel_class < 0 || kernel_class >= PROF_NCLASS) return fail(BC_ERR_INVALID_ARG, "class %d", kernel_class);
    if (!ms_out || max_out < 0) return fail(BC_ERR_INVALID_ARG, "ms_out");
    ClassTimer& t = g_timer[kernel_class];
    const int n = t.used < max_out ? t.used : max_out;
    for (int i = 0; i < n; ++i) {
        if (hipEventSynchronize(t.stop[i]) != hipSuccess) { release(t); return fail(BC_ERR_HIP, "event sync"); }
        if (hipEventElapsedTime(&ms_out[i], t.start[i], t.stop[i]) != hipSuccess) { release(t); return fail(BC_ERR_HIP, "elapsed"); }
        if (work_out) work_out[i] = t.work[i];
    }
    if (launches) *launches = n;
    release(t);
    return BC_OK;
}

int bc_profile_times(int kernel_class, float* ms_out, int max_out, int* launches) {
    return bc_profile_records(kernel_class, ms_out, nullptr, max_out, launches);
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
