// Internal declarations shared by the host sources of libbarycache.
#pragma once

#include <cstdarg>
#include <cstddef>
#include <cstdint>

#include "../../include/bc.h"

namespace bc {

// Record a formatted message as this thread's last error and return `code`.
int fail(int code, const char* fmt, ...);
void clear_error();

constexpr int kMaxK = 8;

// Weights of Eqs. 8-12 for one node set, fp64; returns a bc_status.
int bary_weights(const double* s, int K, double t, const bc_bary_params& p, double* w);
bool params_valid(const bc_bary_params& p);

// sigma of step k of an S-step flow-matching (Euler) schedule with the time
// shift s: s u / (1 + (s - 1) u), u = 1 - k / S (s = 0 or 1: u itself).
inline double flow_sigma(int k, int S, double s) {
    const double u = 1.0 - (double)k / S;
    return (s == 0.0 || s == 1.0) ? u : s * u / (1.0 + (s - 1.0) * u);
}

}  // namespace bc

// Cache context handle (Sec. 3.2, Eq. 6): host metadata over caller storage.
struct bc_cache_ring {
    int K;
    int64_t numel;
    int dtype;
    char* storage;          // device address of slot 0
    int head;               // slot of the newest feature, -1 when empty
    int count;              // features held, <= K
    double coord[bc::kMaxK];
};
