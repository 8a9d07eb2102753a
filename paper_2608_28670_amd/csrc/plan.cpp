// Host side of the Barycentric Extrapolator: weights (Sec. 3.2, Eqs. 8-12),
// the equal-spaced full/forecast mask, the precomputed per-step plan, the
// step schedule and error reporting.  Plain C++17, fp64, no HIP dependency.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>

#include "common.h"

namespace bc {

static thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = 0; }

bool params_valid(const bc_bary_params& p) {
    if (p.nodes != BC_NODES_TRAPEZOID && p.nodes != BC_NODES_LAGRANGE) return false;
    if (p.blend != BC_BLEND_RECENT && p.blend != BC_BLEND_LITERAL) return false;
    if (std::isnan(p.clip_C) || !(p.clip_C > 0)) return false;
    if (!std::isfinite(p.eta) || p.eta < 0) return false;
    if (std::isnan(p.delta) || std::isinf(p.delta)) return false;
    if (!std::isfinite(p.lambda) || p.lambda < 0 || p.lambda > 1) return false;
    return true;
}

// delta_H of Sec. 3.2: 1.0 for H = 2, 0.95 for H = 3, 0.7 for H = 4; this
// library extends it with 1.0 for H = 1 and 0.7 for H > 4.
static double delta_of(int K) {
    if (K <= 2) return 1.0;
    if (K == 3) return 0.95;
    return 0.7;
}

int bary_weights(const double* s, int K, double t, const bc_bary_params& p, double* w) {
    if (K < 1 || K > kMaxK) return fail(BC_ERR_INVALID_ARG, "K=%d outside [1, %d]", K, kMaxK);
    if (!params_valid(p)) return fail(BC_ERR_INVALID_ARG, "invalid bc_bary_params");
    if (!std::isfinite(t)) return fail(BC_ERR_INVALID_ARG, "query time is not finite");
    for (int j = 0; j < K; ++j)
        if (!std::isfinite(s[j])) return fail(BC_ERR_INVALID_ARG, "node %d is not finite", j);

    double alpha[kMaxK];
    if (p.nodes == BC_NODES_TRAPEZOID) {
        if (K > 1) {
            bool up = true, down = true;
            for (int j = 0; j + 1 < K; ++j) {
                up = up && s[j] < s[j + 1];
                down = down && s[j] > s[j + 1];
            }
            if (!up && !down) return fail(BC_ERR_INVALID_ARG, "trapezoid nodes must be strictly monotone");
        }
    } else {
        for (int j = 0; j < K; ++j)
            for (int m = j + 1; m < K; ++m)
                if (s[j] == s[m]) return fail(BC_ERR_INVALID_ARG, "lagrange nodes %d and %d coincide", j, m);
    }

    int on_node = -1;
    if (p.nodes == BC_NODES_LAGRANGE)
        for (int j = 0; j < K; ++j)
            if (s[j] == t) on_node = j;

    if (on_node >= 0) {
        for (int j = 0; j < K; ++j) alpha[j] = (j == on_node) ? 1.0 : 0.0;
    } else {
        // Numerators: Eq. 9's (-1)^j c_j with Eq. 8's trapezoid c (j from 1),
        // or the classical barycentric weights of polynomial interpolation.
        double num[kMaxK];
        for (int j = 0; j < K; ++j) {
            if (p.nodes == BC_NODES_TRAPEZOID) {
                double c = (j == 0 || j == K - 1) ? 0.5 : 1.0;
                num[j] = (j % 2 == 0) ? -c : c;
            } else {
                double prod = 1.0;
                for (int m = 0; m < K; ++m)
                    if (m != j) prod *= (s[j] - s[m]);
                num[j] = 1.0 / prod;
            }
        }
        const double dlt = p.delta < 0 ? delta_of(K) : p.delta;
        double v[kMaxK];
        double total = 0.0, vmax = 0.0;
        for (int j = 0; j < K; ++j) {
            const double gap = t - s[j];
            double u = gap != 0.0 ? num[j] / gap
                                  : std::copysign(std::numeric_limits<double>::infinity(), num[j]);
            u = std::fmax(-p.clip_C, std::fmin(p.clip_C, u));                    // Eq. 10
            v[j] = u == 0.0 ? 0.0 : std::copysign(std::pow(std::fabs(u) + p.eta, dlt), u);  // Eq. 11
            total += v[j];
            vmax = std::fmax(vmax, std::fabs(v[j]));
        }
        if (!std::isfinite(total) || vmax == 0.0 || std::fabs(total) <= 1e-12 * vmax)
            return fail(BC_ERR_DEGENERATE, "normaliser %.17g vanishes or is not finite (K=%d, t=%.17g)",
                        total, K, t);
        for (int j = 0; j < K; ++j) alpha[j] = v[j] / total;
    }

    // Eq. 12 blend.
    const double lam = p.lambda;
    if (p.blend == BC_BLEND_RECENT) {
        for (int j = 0; j < K; ++j) w[j] = (1.0 - lam) * alpha[j];
        w[0] += lam;
    } else {
        for (int j = 0; j + 1 < K; ++j) w[j] = (1.0 - lam) * alpha[j];
        w[K - 1] = lam * alpha[K - 1];
    }
    return BC_OK;
}

}  // namespace bc

extern "C" {

const char* bc_status_str(int s) {
    switch (s) {
        case BC_OK: return "ok";
        case BC_ERR_INVALID_ARG: return "invalid argument";
        case BC_ERR_DEGENERATE: return "degenerate weights";
        case BC_ERR_STATE: return "invalid state";
        case BC_ERR_HIP: return "HIP error";
        case BC_ERR_UNSUPPORTED: return "unsupported shape";
        default: return "unknown status";
    }
}

const char* bc_last_error(void) { return bc::g_err; }

int bc_version(void) { return (1 << 16) | 0; }

void bc_bary_params_default(bc_bary_params* p) {
    if (!p) return;
    p->nodes = BC_NODES_TRAPEZOID;
    p->clip_C = 10.0;
    p->eta = 1e-12;
    p->delta = -1.0;
    p->lambda = 0.0;
    p->blend = BC_BLEND_RECENT;
}

int bc_bary_weights_ex(const double* t_nodes, int K, double t_query, const bc_bary_params* p, double* w_out) {
    bc::clear_error();
    if (!t_nodes || !w_out) return bc::fail(BC_ERR_INVALID_ARG, "NULL pointer");
    bc_bary_params d;
    bc_bary_params_default(&d);
    double tmp[bc::kMaxK];
    int st = bc::bary_weights(t_nodes, K, t_query, p ? *p : d, tmp);
    if (st != BC_OK) return st;
    std::memcpy(w_out, tmp, sizeof(double) * K);
    return BC_OK;
}

int bc_bary_weights(const double* t_nodes, int K, double t_query, double* w_out) {
    return bc_bary_weights_ex(t_nodes, K, t_query, nullptr, w_out);
}

int bc_make_mask(int S, int interval, int force_last, uint8_t* mask_out) {
    bc::clear_error();
    if (!mask_out) return bc::fail(BC_ERR_INVALID_ARG, "NULL mask");
    if (S < 1 || interval < 1) return bc::fail(BC_ERR_INVALID_ARG, "S=%d interval=%d must be >= 1", S, interval);
    for (int k = 0; k < S; ++k)
        mask_out[k] = (k % interval == 0 || (force_last && k == S - 1)) ? 1 : 0;
    return BC_OK;
}

int bc_plan(int S, const uint8_t* mask, const double* coords, int K, const bc_bary_params* p,
            bc_plan_step* out) {
    bc::clear_error();
    if (!mask || !out) return bc::fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (S < 1) return bc::fail(BC_ERR_INVALID_ARG, "S=%d", S);
    if (K < 1 || K > bc::kMaxK) return bc::fail(BC_ERR_INVALID_ARG, "K=%d outside [1, 8]", K);
    if (mask[0] != 1) return bc::fail(BC_ERR_INVALID_ARG, "the first step must be a full step");
    for (int k = 0; k < S; ++k)
        if (mask[k] > 1) return bc::fail(BC_ERR_INVALID_ARG, "mask[%d]=%d is not 0/1", k, mask[k]);
    bc_bary_params prm;
    bc_bary_params_default(&prm);
    if (p) prm = *p;
    if (!bc::params_valid(prm)) return bc::fail(BC_ERR_INVALID_ARG, "invalid bc_bary_params");

    int head = -1, count = 0;
    double node_coord[bc::kMaxK] = {0};
    for (int k = 0; k < S; ++k) {
        bc_plan_step& st = out[k];
        for (int j = 0; j < bc::kMaxK; ++j) { st.slots[j] = -1; st.w[j] = 0.0; }
        const double ck = coords ? coords[k] : (double)k;
        if (mask[k]) {
            head = (head + 1) % K;
            node_coord[head] = ck;
            count = count < K ? count + 1 : K;
            st.is_full = 1;
            st.count = count;
            st.head = head;
        } else {
            double s[bc::kMaxK];
            for (int j = 0; j < count; ++j) {
                const int slot = ((head - j) % K + K) % K;
                st.slots[j] = slot;
                s[j] = node_coord[slot];
            }
            int rc = bc::bary_weights(s, count, ck, prm, st.w);
            if (rc != BC_OK) {
                char msg[400];
                std::snprintf(msg, sizeof msg, "%s", bc_last_error());
                return bc::fail(rc, "step %d: %s", k, msg);
            }
            st.is_full = 0;
            st.count = count;
            st.head = head;
        }
    }
    return BC_OK;
}

int bc_make_schedule_shifted(int sampler, int S, double flow_shift, int32_t* tau_out, double* time_out) {
    bc::clear_error();
    if (S < 1 || S > 1000) return bc::fail(BC_ERR_INVALID_ARG, "S=%d outside [1, 1000]", S);
    if (sampler != BC_SAMPLER_DDIM && sampler != BC_SAMPLER_DPMPP2M && sampler != BC_SAMPLER_EULER)
        return bc::fail(BC_ERR_INVALID_ARG, "unknown sampler %d", sampler);
    if (!(flow_shift >= 0.0) || !std::isfinite(flow_shift))
        return bc::fail(BC_ERR_INVALID_ARG, "flow shift %g", flow_shift);
    for (int k = 0; k < S; ++k) {
        const int tau = 999 - (1000 * k) / S;
        if (tau_out) tau_out[k] = tau;
        if (time_out)
            time_out[k] = sampler == BC_SAMPLER_EULER ? 1000.0 * bc::flow_sigma(k, S, flow_shift) : (double)tau;
    }
    return BC_OK;
}

int bc_make_schedule(int sampler, int S, int32_t* tau_out, double* time_out) {
    return bc_make_schedule_shifted(sampler, S, 1.0, tau_out, time_out);
}

}  // extern "C"
