// Exercise the library's host logic (weights, mask, plan, schedules) under
// AddressSanitizer and UndefinedBehaviorSanitizer: random and adversarial
// arguments, with the invariants every successful call must meet.  Built from
// the library's own plan.cpp by tests/test_host_plan.py; exits non-zero on a
// violated invariant (the sanitizers abort on a memory or UB error).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <random>
#include <vector>

#include "bc.h"

static int failures = 0;
#define CHECK(c, ...) do { if (!(c)) { ++failures; std::fprintf(stderr, __VA_ARGS__); std::fprintf(stderr, "\n"); } } while (0)

int main() {
    std::mt19937_64 g(2026);
    std::uniform_real_distribution<double> u01(0.0, 1.0);
    const double inf = std::numeric_limits<double>::infinity(), nan = std::numeric_limits<double>::quiet_NaN();
    int ok = 0, rejected = 0;
    // weights: random nodes and queries, every parameter mode
    for (int it = 0; it < 20000; ++it) {
        int K = 1 + (int)(g() % 8);
        std::vector<double> s(K), w(K, 0.0);
        for (int j = 0; j < K; ++j) s[j] = u01(g) * (it % 3 == 0 ? 1000.0 : 1.0);
        if (it % 2) std::sort(s.begin(), s.end()); else std::sort(s.rbegin(), s.rend());
        double t = (it % 5 == 0) ? s[g() % K] : u01(g) * 1.5 - 0.25;
        bc_bary_params p;
        bc_bary_params_default(&p);
        p.nodes = (it % 7 == 0) ? BC_NODES_LAGRANGE : BC_NODES_TRAPEZOID;
        p.clip_C = (it % 11 == 0) ? inf : 10.0;
        p.lambda = (it % 13 == 0) ? u01(g) : 0.0;
        p.blend = (it % 17 == 0) ? BC_BLEND_LITERAL : BC_BLEND_RECENT;
        int rc = bc_bary_weights_ex(s.data(), K, t, &p, w.data());
        if (rc == BC_OK) {
            double sum = 0.0, mag = 0.0;
            for (double v : w) { CHECK(std::isfinite(v), "non-finite weight"); sum += v; mag += std::fabs(v); }
            // unit sum up to rounding, which grows with the weights' magnitude
            // (a nearly cancelling normaliser gives large weights)
            if (p.blend == BC_BLEND_RECENT)
                CHECK(std::fabs(sum - 1.0) <= 1e-14 * K * mag + 1e-14, "sum %.17g, sum|w| %g", sum, mag);
            ++ok;
        } else {
            CHECK(rc == BC_ERR_DEGENERATE || rc == BC_ERR_INVALID_ARG, "rc %d", rc);
            CHECK(bc_last_error()[0] != 0, "empty error message");
            ++rejected;
        }
    }
    // adversarial weights arguments
    double s3[3] = {3.0, 2.0, 1.0}, w3[3];
    double bad[3] = {1.0, nan, 0.0}, dup[3] = {1.0, 1.0, 0.0};
    CHECK(bc_bary_weights(nullptr, 3, 4.0, w3) == BC_ERR_INVALID_ARG, "NULL nodes");
    CHECK(bc_bary_weights(s3, 3, 4.0, nullptr) == BC_ERR_INVALID_ARG, "NULL out");
    CHECK(bc_bary_weights(s3, 0, 4.0, w3) == BC_ERR_INVALID_ARG, "K=0");
    CHECK(bc_bary_weights(s3, 9, 4.0, w3) == BC_ERR_INVALID_ARG, "K=9");
    CHECK(bc_bary_weights(s3, -5, 4.0, w3) == BC_ERR_INVALID_ARG, "K<0");
    CHECK(bc_bary_weights(bad, 3, 4.0, w3) == BC_ERR_INVALID_ARG, "NaN node");
    CHECK(bc_bary_weights(dup, 3, 4.0, w3) == BC_ERR_INVALID_ARG, "duplicate node");
    CHECK(bc_bary_weights(s3, 3, nan, w3) == BC_ERR_INVALID_ARG, "NaN query");
    bc_bary_params pb;
    bc_bary_params_default(&pb);
    pb.nodes = 7;
    CHECK(bc_bary_weights_ex(s3, 3, 4.0, &pb, w3) == BC_ERR_INVALID_ARG, "bad mode");
    bc_bary_params_default(&pb);
    pb.lambda = 1.5;
    CHECK(bc_bary_weights_ex(s3, 3, 4.0, &pb, w3) == BC_ERR_INVALID_ARG, "lambda > 1");
    // masks
    for (int S = -2; S <= 1001; S += (S < 60 ? 1 : 97)) {
        for (int n = -1; n <= 7; ++n) {
            std::vector<uint8_t> m(S > 0 ? S : 1, 9);
            int rc = bc_make_mask(S, n, n & 1, m.data());
            if (rc == BC_OK) {
                CHECK(m[0] == 1, "mask[0]");
                for (int k = 0; k < S; ++k) CHECK(m[k] <= 1, "mask value");
            }
        }
    }
    CHECK(bc_make_mask(10, 3, 1, nullptr) == BC_ERR_INVALID_ARG, "NULL mask");
    // plans under random masks
    for (int it = 0; it < 3000; ++it) {
        int S = 1 + (int)(g() % 120), K = 1 + (int)(g() % 8);
        std::vector<uint8_t> m(S);
        for (int k = 0; k < S; ++k) m[k] = (g() % 3 == 0) ? 1 : 0;
        m[0] = (it % 50 == 0) ? 0 : 1;
        std::vector<bc_plan_step> out(S);
        int rc = bc_plan(S, m.data(), nullptr, K, nullptr, out.data());
        if (m[0] == 0) { CHECK(rc == BC_ERR_INVALID_ARG, "mask[0]=0 accepted"); continue; }
        CHECK(rc == BC_OK, "plan rc %d: %s", rc, bc_last_error());
        if (rc != BC_OK) continue;
        for (int k = 0; k < S; ++k) {
            const bc_plan_step& st = out[k];
            CHECK(st.count >= 1 && st.count <= K, "count");
            CHECK(st.head >= 0 && st.head < K, "head");
            if (!st.is_full) {
                double sum = 0.0;
                for (int j = 0; j < st.count; ++j) {
                    CHECK(st.slots[j] >= 0 && st.slots[j] < K, "slot");
                    sum += st.w[j];
                }
                CHECK(std::fabs(sum - 1.0) < 1e-9, "plan weights sum %g", sum);
            }
        }
    }
    std::vector<bc_plan_step> o1(4);
    uint8_t m4[4] = {1, 0, 1, 0};
    CHECK(bc_plan(4, m4, nullptr, 0, nullptr, o1.data()) == BC_ERR_INVALID_ARG, "plan K=0");
    CHECK(bc_plan(4, m4, nullptr, 9, nullptr, o1.data()) == BC_ERR_INVALID_ARG, "plan K=9");
    CHECK(bc_plan(0, m4, nullptr, 3, nullptr, o1.data()) == BC_ERR_INVALID_ARG, "plan S=0");
    CHECK(bc_plan(4, nullptr, nullptr, 3, nullptr, o1.data()) == BC_ERR_INVALID_ARG, "plan NULL mask");
    double coords_bad[4] = {0.0, 1.0, 1.0, 3.0};
    CHECK(bc_plan(4, m4, coords_bad, 3, nullptr, o1.data()) != BC_OK || true, "coords");
    // schedules
    for (int smp = -1; smp <= 3; ++smp) {
        for (int S = -1; S <= 1001; S += (S < 60 ? 1 : 113)) {
            std::vector<int32_t> tau(S > 0 ? S : 1);
            std::vector<double> tin(S > 0 ? S : 1);
            for (double shift : {0.0, 1.0, 7.0, -1.0, nan}) {
                int rc = bc_make_schedule_shifted(smp, S, shift, tau.data(), tin.data());
                if (rc != BC_OK) continue;
                for (int k = 0; k < S; ++k) {
                    CHECK(tau[k] >= 0 && tau[k] <= 999, "tau range");
                    CHECK(std::isfinite(tin[k]) && tin[k] >= 0.0 && tin[k] <= 1000.0, "time range");
                    if (k) CHECK(tau[k] <= tau[k - 1], "tau order");
                }
            }
        }
    }
    for (int c = -3; c < 10; ++c) CHECK(bc_status_str(c) != nullptr, "status string");
    std::printf("weights ok %d rejected %d; failures %d\n", ok, rejected, failures);
    return failures ? 1 : 0;
}
