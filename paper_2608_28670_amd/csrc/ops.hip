// Small kernels around the block GEMMs and attention: LayerNorm + adaLN
// modulation, the skinny linear layers of the conditioning path, patch
// embedding, the final layer, sampler updates and element-wise helpers.
// All statistics and accumulations are fp32.
#include <type_traits>
#include <algorithm>
#include <cmath>

#include "ops.h"

namespace bc {

constexpr float kLnEps = 1e-6f;
constexpr int kMaxPatch = 256;

// ---------------------------------------------------------------------------
// LayerNorm + modulate: one wave per row, the row cached in registers as
// 4-element chunks (lane l holds chunks l, l + 64, ...), so every load is 16
// (fp32) or 8 (bf16) bytes and every store 8 (bf16) or 16 (fp32) bytes.
// Requires D % 4 == 0.
// ---------------------------------------------------------------------------
template <typename T> struct Vec4;
template <> struct Vec4<float> {
    __device__ static void load(const float* p, float* v) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(p);
        v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
    }
    __device__ static void store(float* p, const float* v) {
        *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
    }
};
template <> struct Vec4<bf16> {
    __device__ static void load(const bf16* p, float* v) {
        typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
        const u32x2_t w = *reinterpret_cast<const u32x2_t*>(p);
        v[0] = __uint_as_float(w[0] << 16); v[1] = __uint_as_float(w[0] & 0xffff0000u);
        v[2] = __uint_as_float(w[1] << 16); v[3] = __uint_as_float(w[1] & 0xffff0000u);
    }
    __device__ static void store(bf16* p, const float* v) {
        typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
        uint32_t w[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const bf16 lo = (bf16)v[2 * i], hi = (bf16)v[2 * i + 1];
            w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
        }
        *reinterpret_cast<u32x2_t*>(p) = u32x2_t{w[0], w[1]};
    }
};

// Each wave takes RPW consecutive rows: the next row's chunks are loaded
// while the current one is reduced, and the modulation vectors (one pair per
// sample) are loaded once per sample instead of once per row.
template <typename Tin_, typename Tout_, int NC, int RPW>
__global__ __launch_bounds__(256) void ln_mod_kernel(const elem_t<Tin_>* __restrict__ x, int64_t rows, int D,
                                                     const float* __restrict__ shift,
                                                     const float* __restrict__ scale, int64_t ld_mod, int rps,
                                                     elem_t<Tout_>* __restrict__ h) {
    typedef elem_t<Tin_> Tin;
    typedef elem_t<Tout_> Tout;
    const int lane = threadIdx.x & 63;
    const int64_t row0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW;
    if (row0 >= rows) return;
    const int nch = D >> 2;
    float v[2][NC][4], s4[NC][4], c4[NC][4];
    auto load_row = [&](int64_t row, float (&dst)[NC][4]) {
        const Tin* xr = x + row * D;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const int c = lane + 64 * j;
            if (c < nch) Vec4<Tin>::load(xr + 4 * c, dst[j]);
            else {
#pragma unroll
                for (int e = 0; e < 4; ++e) dst[j][e] = 0.f;
            }
        }
    };
    load_row(row0, v[0]);
    int64_t cur_b = -1;
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        const int64_t row = row0 + i;
        if (row >= rows) break;
        if (i + 1 < RPW && row + 1 < rows) load_row(row + 1, v[(i + 1) & 1]);
        const int64_t b = row / rps;
        if (b != cur_b) {
            cur_b = b;
            const float* sh = shift + b * ld_mod;
            const float* sc = scale + b * ld_mod;
#pragma unroll
            for (int j = 0; j < NC; ++j) {
                const int c = lane + 64 * j;
                if (c < nch) {
                    Vec4<float>::load(sh + 4 * c, s4[j]);
                    Vec4<float>::load(sc + 4 * c, c4[j]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) s4[j][e] = c4[j][e] = 0.f;
                }
            }
        }
        const float (&r)[NC][4] = v[i & 1];
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < NC; ++j) sum += (r[j][0] + r[j][1]) + (r[j][2] + r[j][3]);
        const float mean = wave_sum(sum) / (float)D;
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            if (lane + 64 * j < nch) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float d = r[j][e] - mean;
                    sq += d * d;
                }
            }
        }
        const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)D + kLnEps);
        Tout* hr = h + row * D;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const int c = lane + 64 * j;
            if (c < nch) {
                float o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = (r[j][e] - mean) * rstd * (1.0f + c4[j][e]) + s4[j][e];
                Vec4<Tout>::store(hr + 4 * c, o);
            }
        }
    }
}

template <typename Tin, typename Tout, int RPW>
static int run_ln_rows(const void* x, int64_t rows, int D, const float* shift, const float* scale, int64_t ld_mod,
                       int rps, void* h, hipStream_t s) {
    const int nc = (D / 4 + 63) / 64;
    dim3 g((unsigned)((rows + 4 * RPW - 1) / (4 * RPW))), b(256);
    const Tin* xi = static_cast<const Tin*>(x);
    Tout* ho = static_cast<Tout*>(h);
    if (nc <= 1) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 1, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else if (nc <= 2) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 2, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else if (nc <= 5) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 5, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else if (nc <= 8) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 8, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else if (nc <= 12) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 12, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else if (nc <= 16) launch_k(ln_mod_kernel<tag_t<Tin>, tag_t<Tout>, 16, RPW>, g, b, s, xi, rows, D, shift, scale, ld_mod, rps, ho);
    else return fail(BC_ERR_UNSUPPORTED, "LayerNorm width %d > 4096", D);
    return check_launch("ln_mod");
}

// Rows per wave: two (the second row's loads in flight while the first is
// reduced), four for rows of up to 1280 values when there are at least 8192
// of them (PixArt's 16 384 rows of 1152: 20.6 -> 18.6 us; DiT-XL/2's 4096
// rows are fastest with two: 7.7 us against 8.6 with four and 8.0 with one).
template <typename Tin, typename Tout>
static int run_ln(const void* x, int64_t rows, int D, const float* shift, const float* scale, int64_t ld_mod, int rps,
                  void* h, hipStream_t s) {
    if (D <= 1280 && rows >= 8192) return run_ln_rows<Tin, Tout, 4>(x, rows, D, shift, scale, ld_mod, rps, h, s);
    return run_ln_rows<Tin, Tout, 2>(x, rows, D, shift, scale, ld_mod, rps, h, s);
}

int launch_ln_mod(int in_dt, const void* x, int64_t rows, int D, const float* shift, const float* scale,
                  int64_t ld_mod, int rows_per_sample, int out_dt, void* h, hipStream_t s) {
    if (rows <= 0) return BC_OK;
    if (D % 4 || ld_mod % 4 || (reinterpret_cast<uintptr_t>(shift) | reinterpret_cast<uintptr_t>(scale)) % 16)
        return fail(BC_ERR_UNSUPPORTED, "LayerNorm needs D and the modulation rows in 16-byte units");
    prof_begin(PROF_LAYERNORM, s, (double)rows * D * (dtype_size(in_dt) + dtype_size(out_dt)));
    int rc;
    if (in_dt == BC_F32 && out_dt == BC_BF16) rc = run_ln<float, bf16>(x, rows, D, shift, scale, ld_mod, rows_per_sample, h, s);
    else if (in_dt == BC_F32) rc = run_ln<float, float>(x, rows, D, shift, scale, ld_mod, rows_per_sample, h, s);
    else if (out_dt == BC_BF16) rc = run_ln<bf16, bf16>(x, rows, D, shift, scale, ld_mod, rows_per_sample, h, s);
    else rc = run_ln<bf16, float>(x, rows, D, shift, scale, ld_mod, rows_per_sample, h, s);
    prof_end(PROF_LAYERNORM, s);
    return rc;
}

// ---------------------------------------------------------------------------
// Skinny linear on MFMA: a 16 x 16 output tile per wave (16 samples x 16
// output features); act(in) is staged in LDS in the weight dtype, the weights
// stream straight from HBM into the B operand.
// ---------------------------------------------------------------------------
template <typename T> struct SkMma;
template <> struct SkMma<bf16> {
    static constexpr int E = 8, KI = 32, KC = 1024;
    typedef bf16x8 frag;
    __device__ static f32x4 mma(const frag& a, const frag& b, const f32x4& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static frag load(const bf16* p) { return __builtin_bit_cast(frag, *reinterpret_cast<const u32x4*>(p)); }
    __device__ static frag zero() { return __builtin_bit_cast(frag, u32x4{0, 0, 0, 0}); }
};
template <> struct SkMma<float> {
    static constexpr int E = 1, KI = 4, KC = 512;
    typedef float frag;
    __device__ static f32x4 mma(frag a, frag b, const f32x4& c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static frag load(const float* p) { return *p; }
    __device__ static frag zero() { return 0.f; }
};

constexpr int kSkTiles = 4;   // 16-column tiles per wave
constexpr int kSkBatch = 8;   // k-steps of weight loads issued together

template <typename T_>
__global__ __launch_bounds__(256) void skinny_kernel(SkinnyArgs a) {
    typedef elem_t<T_> T;
    typedef SkMma<T> MM;
    constexpr int KC = MM::KC;
    constexpr int PAD = 16 / (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) T sIn[16][KC + PAD];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int Ntot = a.nseg * a.Nseg;
    const int nbase = blockIdx.x * (4 * kSkTiles * 16) + wave * kSkTiles * 16;
    const int r16 = lane & 15, kg = (lane >> 4) * MM::E;

    for (int b0 = 0; b0 < a.B; b0 += 16) {
        f32x4 acc[kSkTiles];
#pragma unroll
        for (int t = 0; t < kSkTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int kc0 = 0; kc0 < a.K; kc0 += KC) {
            const int kn = min(KC, a.K - kc0);
            __syncthreads();
            for (int i = tid; i < 16 * KC; i += 256) {
                const int bb = i / KC, k = i % KC;
                float v = 0.f;
                if (b0 + bb < a.B && k < kn) {
                    v = a.in[(int64_t)(b0 + bb) * a.ld_in + kc0 + k];
                    if (a.act_in == 1) v = silu(v);
                }
                sIn[bb][k] = (T)v;
            }
            __syncthreads();
            // Weight rows of this wave's tiles (NULL past the end).
            const T* wr[kSkTiles];
#pragma unroll
            for (int t = 0; t < kSkTiles; ++t) {
                const int ncol = nbase + t * 16;
                wr[t] = nullptr;
                if (ncol < Ntot) {
                    const int seg = ncol / a.Nseg;
                    const int nloc = ncol - seg * a.Nseg + r16;
                    wr[t] = static_cast<const T*>(a.W[seg]) + (int64_t)nloc * a.K + kc0;
                }
            }
            // kSkBatch k-steps of every tile's weights in flight before the MFMAs.
            for (int k0 = 0; k0 < kn; k0 += kSkBatch * MM::KI) {
                typename MM::frag wf[kSkTiles][kSkBatch];
#pragma unroll
                for (int t = 0; t < kSkTiles; ++t)
#pragma unroll
                    for (int u = 0; u < kSkBatch; ++u) {
                        const int k = k0 + u * MM::KI + kg;
                        wf[t][u] = (wr[t] && k < kn) ? MM::load(wr[t] + k) : MM::zero();
                    }
#pragma unroll
                for (int u = 0; u < kSkBatch; ++u) {
                    const int k = k0 + u * MM::KI;
                    if (k >= kn) break;
                    const typename MM::frag af = MM::load(&sIn[r16][k + kg]);
#pragma unroll
                    for (int t = 0; t < kSkTiles; ++t) acc[t] = MM::mma(af, wf[t][u], acc[t]);
                }
            }
        }
#pragma unroll
        for (int t = 0; t < kSkTiles; ++t) {
            const int ncol = nbase + t * 16;
            if (ncol >= Ntot) break;
            const int seg = ncol / a.Nseg;
            const int nloc = ncol - seg * a.Nseg + r16;
            const float bv = a.bias[seg] ? ld(static_cast<const T*>(a.bias[seg]) + nloc) : 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int bb = b0 + 4 * (lane >> 4) + r;
                if (bb >= a.B) continue;
                float v = acc[t][r] + bv;
                if (a.act_out == 1) v = silu(v);
                const int64_t o = (int64_t)bb * a.ld_out + ncol + r16;
                if (a.addend) v += a.addend[o];
                a.out[o] = v;
            }
        }
    }
}

int launch_skinny(int dt, const SkinnyArgs& a, hipStream_t s) {
    if (a.B <= 0 || a.nseg <= 0) return BC_OK;
    if (a.B > 64) return fail(BC_ERR_UNSUPPORTED, "conditioning batch %d > 64", a.B);
    if (a.nseg > kMaxSeg || a.Nseg % 16 || a.K % (dt == BC_BF16 ? 8 : 4))
        return fail(BC_ERR_UNSUPPORTED, "skinny linear segments=%d N=%d K=%d", a.nseg, a.Nseg, a.K);
    for (int i = 0; i < a.nseg; ++i)
        if (!a.W[i] || reinterpret_cast<uintptr_t>(a.W[i]) % 16)
            return fail(BC_ERR_INVALID_ARG, "skinny linear weight %d missing or misaligned", i);
    const int Ntot = a.nseg * a.Nseg;
    const unsigned grid = (unsigned)((Ntot + 4 * kSkTiles * 16 - 1) / (4 * kSkTiles * 16));
    if (dt == BC_BF16) skinny_kernel<bf16_tag><<<grid, 256, 0, s>>>(a);
    else skinny_kernel<float><<<grid, 256, 0, s>>>(a);
    return check_launch("skinny linear");
}

// ---------------------------------------------------------------------------
// Conditioning helpers
// ---------------------------------------------------------------------------
__global__ void step_sinusoid_kernel(int sampler, int S, int half, double shift, float* e) {
    const int k = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= half || k >= S) return;
    // Euler: 1000 sigma_k with the time shift (the device copy of flow_sigma).
    const double u = 1.0 - (double)k / S;
    const double sig = (shift == 0.0 || shift == 1.0) ? u : shift * u / (1.0 + (shift - 1.0) * u);
    const double t = sampler == BC_SAMPLER_EULER ? 1000.0 * sig : (double)(999 - (1000 * k) / S);
    const double f = exp(-log(10000.0) * (double)i / (double)half);
    const double ang = t * f;
    e[(int64_t)k * 2 * half + i] = (float)cos(ang);
    e[(int64_t)k * 2 * half + half + i] = (float)sin(ang);
}

int launch_step_sinusoid(int sampler, int S, int dim, double shift, float* e, hipStream_t s) {
    const int half = dim / 2;
    step_sinusoid_kernel<<<dim3((half + 127) / 128, S), 128, 0, s>>>(sampler, S, half, shift, e);
    return check_launch("sinusoid");
}

template <typename T_>
__global__ void build_cond_kernel(const float* temb, int S, int B, int D, const elem_t<T_>* table, const int64_t* labels,
                                  int n_rows, const float* add, float* c) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)S * B * D) return;
    const int n = (int)(i % D);
    const int64_t kb = i / D;
    const int b = (int)(kb % B), k = (int)(kb / B);
    float v = temb[(int64_t)k * D + n];
    if (labels) {
        int64_t lab = labels[b];
        lab = lab < 0 ? 0 : (lab >= n_rows ? n_rows - 1 : lab);   // out-of-range labels are clamped
        v += ld(table + lab * D + n);
    } else if (add) {
        v += add[(int64_t)b * D + n];
    }
    c[i] = v;
}

int launch_build_cond(int dt, const float* temb, int S, int B, int D, const void* table, const int64_t* labels,
                      int n_rows, const float* add, float* c, hipStream_t s) {
    const int64_t n = (int64_t)S * B * D;
    const unsigned g = (unsigned)((n + 255) / 256);
    if (dt == BC_BF16) build_cond_kernel<bf16_tag><<<g, 256, 0, s>>>(temb, S, B, D, static_cast<const bf16*>(table), labels, n_rows, add, c);
    else build_cond_kernel<float><<<g, 256, 0, s>>>(temb, S, B, D, static_cast<const float*>(table), labels, n_rows, add, c);
    return check_launch("build_cond");
}

template <typename T_>
__global__ void gather_silu_kernel(const float* c, int B, int D, RowList rows, int n, elem_t<T_>* out) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)n * B * D) return;
    const int d = (int)(i % D);
    const int64_t ib = i / D;
    const int b = (int)(ib % B), r = (int)(ib / B);
    st(out + i, silu(c[((int64_t)rows.row[r] * B + b) * D + d]));
}

int launch_gather_silu(int dt, const float* c, int B, int D, const RowList& rows, int n, void* out, hipStream_t s) {
    if (n <= 0) return BC_OK;
    if (n > kMaxSeg) return fail(BC_ERR_UNSUPPORTED, "gather of %d rows", n);
    const int64_t total = (int64_t)n * B * D;
    const unsigned g = (unsigned)((total + 255) / 256);
    if (dt == BC_BF16) gather_silu_kernel<bf16_tag><<<g, 256, 0, s>>>(c, B, D, rows, n, static_cast<bf16*>(out));
    else gather_silu_kernel<float><<<g, 256, 0, s>>>(c, B, D, rows, n, static_cast<float*>(out));
    return check_launch("gather_silu");
}

template <typename T_>
__global__ void add_label_kernel(const float* t, const elem_t<T_>* table, const int64_t* labels, int B, int D, int n_rows,
                                 float* c) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * D) return;
    const int b = (int)(i / D), n = (int)(i % D);
    int64_t lab = labels[b];
    lab = lab < 0 ? 0 : (lab >= n_rows ? n_rows - 1 : lab);   // out-of-range labels are clamped
    c[i] = t[i] + ld(table + lab * D + n);
}

int launch_add_label(int dt, const float* t, const void* table, const int64_t* labels, int B, int D, int n_rows,
                     float* c, hipStream_t s) {
    const int64_t n = (int64_t)B * D;
    const unsigned g = (unsigned)((n + 255) / 256);
    if (dt == BC_BF16) add_label_kernel<bf16_tag><<<g, 256, 0, s>>>(t, static_cast<const bf16*>(table), labels, B, D, n_rows, c);
    else add_label_kernel<float><<<g, 256, 0, s>>>(t, static_cast<const float*>(table), labels, B, D, n_rows, c);
    return check_launch("add_label");
}

struct TableArgs { const void* tab[kMaxSeg]; };

template <typename T_>
__global__ void add_tables_kernel(const float* vec, int64_t ld_vec, TableArgs ta, int nseg, int N, int B, float* out,
                                  int64_t ld_out) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * nseg * N) return;
    const int j = (int)(i % N);
    const int seg = (int)((i / N) % nseg);
    const int b = (int)(i / ((int64_t)N * nseg));
    out[(int64_t)b * ld_out + (int64_t)seg * N + j] = vec[(int64_t)b * ld_vec + j] + ld(static_cast<const T*>(ta.tab[seg]) + j);
}

int launch_add_tables(int dt, const float* vec, int64_t ld_vec, const void* const* tables, int nseg, int N, int B,
                      float* out, int64_t ld_out, hipStream_t s) {
    if (nseg > kMaxSeg) return fail(BC_ERR_UNSUPPORTED, "%d tables", nseg);
    TableArgs ta;
    for (int i = 0; i < nseg; ++i) ta.tab[i] = tables[i];
    const int64_t n = (int64_t)B * nseg * N;
    const unsigned g = (unsigned)((n + 255) / 256);
    if (dt == BC_BF16) add_tables_kernel<bf16_tag><<<g, 256, 0, s>>>(vec, ld_vec, ta, nseg, N, B, out, ld_out);
    else add_tables_kernel<float><<<g, 256, 0, s>>>(vec, ld_vec, ta, nseg, N, B, out, ld_out);
    return check_launch("add_tables");
}

template <typename E_>
__global__ void token_mean_kernel(const elem_t<E_>* x, int B, int T_, int D, float* out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * D) return;
    const int b = (int)(i / D), n = (int)(i % D);
    float acc = 0.f;
    for (int t = 0; t < T_; ++t) acc += ld(x + ((int64_t)b * T_ + t) * D + n);
    out[i] = acc / (float)T_;
}

int launch_token_mean(int dt, const void* x, int B, int T, int D, float* out, hipStream_t s) {
    const int64_t n = (int64_t)B * D;
    const unsigned g = (unsigned)((n + 255) / 256);
    if (dt == BC_BF16) token_mean_kernel<bf16_tag><<<g, 256, 0, s>>>(static_cast<const bf16*>(x), B, T, D, out);
    else token_mean_kernel<float><<<g, 256, 0, s>>>(static_cast<const float*>(x), B, T, D, out);
    return check_launch("token_mean");
}

template <typename Tin_, typename Tout_>
__global__ void convert_kernel(const elem_t<Tin_>* in, elem_t<Tout_>* out, int64_t n) {
    typedef elem_t<Tin_> Tin;
    typedef elem_t<Tout_> Tout;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        st(out + i, ld(in + i));
}

int launch_convert(int in_dt, const void* in, int out_dt, void* out, int64_t n, hipStream_t s) {
    if (n <= 0) return BC_OK;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    const unsigned g = (unsigned)blocks;
    if (in_dt == BC_F32 && out_dt == BC_BF16) convert_kernel<float, bf16_tag><<<g, 256, 0, s>>>(static_cast<const float*>(in), static_cast<bf16*>(out), n);
    else if (in_dt == BC_BF16 && out_dt == BC_F32) convert_kernel<bf16_tag, float><<<g, 256, 0, s>>>(static_cast<const bf16*>(in), static_cast<float*>(out), n);
    else return launch_copy(in, out, n * dtype_size(in_dt), s);
    return check_launch("convert");
}

// ---------------------------------------------------------------------------
// Patch embedding and the final layer
// ---------------------------------------------------------------------------
// One workgroup per token: gather its p*p*C patch values once (LDS), then
// each thread produces output features of the row.
template <typename T_, int kPatchRows>
__global__ __launch_bounds__(256) void patch_embed_kernel(const float* __restrict__ lat, LatentShape ls,
                                                          const elem_t<T_>* __restrict__ W, const elem_t<T_>* __restrict__ bias,
                                                          const elem_t<T_>* __restrict__ pos, int D, int lat_B, int rows,
                                                          float* __restrict__ x) {
    typedef elem_t<T_> T;
    // kPatchRows tokens per workgroup: each thread reads its columns' weight
    // rows once for all of them (the weights are [D, p*p*C], one row per
    // output column), and each output still sums its patch in order q = 0, 1, ...
    // Large patches (the video model's 64 values) take 16 tokens per
    // workgroup; small ones one, which keeps enough workgroups in flight.
    __shared__ float patch[kPatchRows][kMaxPatch];
    const int Tn = ls.tokens();
    const int row0 = blockIdx.x * kPatchRows;
    const int hp = ls.H / ls.p, wp = ls.W / ls.p;
    const int PD = ls.p * ls.p * ls.C;
    for (int i = threadIdx.x; i < kPatchRows * PD; i += blockDim.x) {
        const int r = i / PD, q = i - r * PD, row = row0 + r;
        float v = 0.f;
        if (row < rows) {
            const int bm = row / Tn, tok = row - bm * Tn;
            const int b = bm % lat_B;
            const int f = tok / (hp * wp), ti = (tok / wp) % hp, tj = tok % wp;
            const int ph = q / (ls.p * ls.C), pw = (q / ls.C) % ls.p, ch = q % ls.C;
            v = lat[((((int64_t)b * ls.C + ch) * ls.F + f) * ls.H + ti * ls.p + ph) * ls.W + tj * ls.p + pw];
        }
        patch[r][q] = v;
    }
    __syncthreads();
    for (int c = threadIdx.x; c < D; c += blockDim.x) {
        const T* wr = W + (int64_t)c * PD;
        float acc[kPatchRows];
#pragma unroll
        for (int r = 0; r < kPatchRows; ++r) acc[r] = 0.f;
        for (int q = 0; q < PD; ++q) {
            const float w = ld(wr + q);
#pragma unroll
            for (int r = 0; r < kPatchRows; ++r) acc[r] = __builtin_fmaf(patch[r][q], w, acc[r]);
        }
        const float bc = ld(bias + c);
#pragma unroll
        for (int r = 0; r < kPatchRows; ++r) {
            const int row = row0 + r;
            if (row < rows) {
                const int tok = row % Tn;
                x[(int64_t)row * D + c] = acc[r] + bc + ld(pos + (int64_t)tok * D + c);
            }
        }
    }
}

int launch_patch_embed(int dt, const float* lat, LatentShape ls, int B, int lat_B, const void* W, const void* bias,
                       const void* pos, int D, float* x, hipStream_t s) {
    if (ls.p * ls.p * ls.C > kMaxPatch) return fail(BC_ERR_UNSUPPORTED, "patch of %d values", ls.p * ls.p * ls.C);
    if (lat_B < 1 || lat_B > B) return fail(BC_ERR_INVALID_ARG, "latent batch %d for a model batch of %d", lat_B, B);
    const int rows = B * ls.tokens();
    if (rows <= 0) return BC_OK;
    auto go = [&](auto tpb) {
        constexpr int TPB = decltype(tpb)::value;
        const unsigned grid = (unsigned)((rows + TPB - 1) / TPB);
        if (dt == BC_BF16)
            patch_embed_kernel<bf16_tag, TPB><<<grid, 256, 0, s>>>(lat, ls, static_cast<const bf16*>(W),
                                                               static_cast<const bf16*>(bias),
                                                               static_cast<const bf16*>(pos), D, lat_B, rows, x);
        else
            patch_embed_kernel<float, TPB><<<grid, 256, 0, s>>>(lat, ls, static_cast<const float*>(W),
                                                                static_cast<const float*>(bias),
                                                                static_cast<const float*>(pos), D, lat_B, rows, x);
    };
    if (ls.p * ls.p * ls.C >= 32) go(std::integral_constant<int, 16>{});
    else go(std::integral_constant<int, 1>{});
    return check_launch("patch_embed");
}

__global__ void cfg_labels_kernel(const int64_t* labels, int B, int64_t null_id, int64_t* out) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < B) out[i] = labels[i];
    else if (i < 2 * B) out[i] = null_id;
}

int launch_cfg_labels(const int64_t* labels, int B, int64_t null_id, int64_t* out, hipStream_t s) {
    cfg_labels_kernel<<<1, 128, 0, s>>>(labels, B, null_id, out);
    return check_launch("cfg_labels");
}

// ---------------------------------------------------------------------------
// Sampler update
// ---------------------------------------------------------------------------
// Model output arrives in token layout [B*T, p*p*C_out] (the final linear's
// output); element (b, c, f, y, x) of the latent is read from token
// (f, y/p, x/p), feature ((y%p)*p + x%p)*C_out + c, which is unpatchify.
__global__ void sampler_kernel(SamplerCoef k, float* x, const float* out_tok, float* prev, LatentShape ls, int B,
                               int C_out, float cfg, int64_t uncond_off) {
    const int64_t S = (int64_t)ls.F * ls.H * ls.W;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * ls.C * S) return;
    const int xs = (int)(i % ls.W);
    const int ys = (int)((i / ls.W) % ls.H);
    const int f = (int)((i / ((int64_t)ls.W * ls.H)) % ls.F);
    const int64_t bc = i / S;
    const int c = (int)(bc % ls.C), b = (int)(bc / ls.C);
    const int hp = ls.H / ls.p, wp = ls.W / ls.p;
    const int tok = (f * hp + ys / ls.p) * wp + xs / ls.p;
    const int feat = ((ys % ls.p) * ls.p + xs % ls.p) * C_out + c;
    const int64_t o = ((int64_t)b * ls.tokens() + tok) * (ls.p * ls.p * C_out) + feat;
    float e = out_tok[o];
    if (uncond_off > 0) {
        const float u = out_tok[o + uncond_off];
        e = __builtin_fmaf(cfg, e - u, u);
    }
    sampler_update(k, x + i, e, prev ? prev + i : nullptr);
}

int launch_sampler(const SamplerCoef& k, float* x, const float* out_tok, float* prev, LatentShape ls, int B, int C_out,
                   hipStream_t s, float cfg, int64_t uncond_off) {
    const int64_t n = (int64_t)B * ls.C * ls.F * ls.H * ls.W;
    sampler_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(k, x, out_tok, prev, ls, B, C_out, cfg, uncond_off);
    return check_launch("sampler");
}

// ---------------------------------------------------------------------------
// QK RMSNorm + 3D rotary embedding: one wave per (row, head, q|k); lane i
// holds the pair (2i, 2i + 1) of the head, so the rotation is lane-local and
// the RMS is one wave reduction.
// ---------------------------------------------------------------------------
template <typename T_>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(elem_t<T_>* __restrict__ qkv, int64_t rows, int64_t ldr, int D,
                                                           int heads, int hd, const elem_t<T_>* __restrict__ wq,
                                                           const elem_t<T_>* __restrict__ wk, int L, int n_img, int gf,
                                                           int gh, int gw, float log2_theta, float q_scale) {
    typedef elem_t<T_> T;
    const int64_t wid = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (wid >= rows * heads * 2) return;   // whole waves
    const int qk = (int)(wid & 1);
    const int64_t rh = wid >> 1;
    const int h = (int)(rh % heads);
    const int64_t r = rh / heads;
    T* p = qkv + r * ldr + (int64_t)qk * D + (int64_t)h * hd;
    const bool act = 2 * lane < hd;
    float x0 = 0.f, x1 = 0.f;
    if (act) {
        x0 = ld(p + 2 * lane);
        x1 = ld(p + 2 * lane + 1);
    }
    const T* w = qk ? wk : wq;
    if (w) {
        float ss = x0 * x0 + x1 * x1;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
        const float inv = 1.0f / sqrtf(ss / (float)hd + 1e-6f);
        if (act) {
            x0 = x0 * inv * ld(w + 2 * lane);
            x1 = x1 * inv * ld(w + 2 * lane + 1);
        }
    }
    const int t = (int)(r % L);
    if (log2_theta > 0.f && t < n_img && act) {
        const int d_f = hd / 8, d_h = (hd - d_f) / 2, d_w = hd - d_f - d_h;
        const int e = 2 * lane;
        const int col = t % gw, row = (t / gw) % gh, fr = t / (gw * gh);
        int pos, j, da;
        if (e < d_f) { pos = fr; j = e / 2; da = d_f; }
        else if (e < d_f + d_h) { pos = row; j = (e - d_f) / 2; da = d_h; }
        else { pos = col; j = (e - d_f - d_h) / 2; da = d_w; }
        const float freq = exp2f(-(float)(2 * j) / (float)da * log2_theta);
        float sn, cs;
        sincosf((float)pos * freq, &sn, &cs);
        const float y0 = x0 * cs - x1 * sn, y1 = x0 * sn + x1 * cs;
        x0 = y0;
        x1 = y1;
    }
    if (act) {
        const float os = qk ? 1.f : q_scale;
        p[2 * lane] = (T)(x0 * os);
        p[2 * lane + 1] = (T)(x1 * os);
    }
}

// bf16 variant for head_dim = 8 * CPH with CPH a power of two (64, 128): one
// wave per (row, q|k) walks the row in 16-byte chunks, lane l taking chunks
// l, l + 64, ...  Since 64 is a multiple of CPH, lane l always holds the same
// four pairs (chunk l % CPH) of whichever head a chunk belongs to: it loads its
// eight norm scales and works out its four rotations once per row.  A head's
// RMS is a reduction over the CPH lanes that hold it.
template <int CPH, typename B_>
__global__ __launch_bounds__(256) void qk_norm_rope_row_kernel(elem_t<B_>* __restrict__ qkv, int64_t rows, int64_t ldr,
                                                               int D, const elem_t<B_>* __restrict__ wq,
                                                               const elem_t<B_>* __restrict__ wk, int L, int n_img, int gf,
                                                               int gh, int gw, float log2_theta, float q_scale) {
    constexpr int HD = 8 * CPH;
    const int64_t wid = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (wid >= rows * 2) return;   // whole waves
    const int qk = (int)(wid & 1);
    const int64_t r = wid >> 1;
    bf16* p = qkv + r * ldr + (int64_t)qk * D;
    const int nch = D / 8;
    const int e0 = (lane % CPH) * 8;   // first element of this lane's chunk within its head
    const bf16* w = qk ? wk : wq;
    float wv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) wv[k] = w ? ld(w + e0 + k) : 1.f;
    const int t = (int)(r % L);
    const bool rot = log2_theta > 0.f && t < n_img;
    float cs[4], sn[4];
    if (rot) {
        constexpr int d_f = HD / 8, d_h = (HD - d_f) / 2, d_w = HD - d_f - d_h;
        const int col = t % gw, row = (t / gw) % gh, fr = t / (gw * gh);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = e0 + 2 * q;
            int pos, j, da;
            if (e < d_f) { pos = fr; j = e / 2; da = d_f; }
            else if (e < d_f + d_h) { pos = row; j = (e - d_f) / 2; da = d_h; }
            else { pos = col; j = (e - d_f - d_h) / 2; da = d_w; }
            const float freq = exp2f(-(float)(2 * j) / (float)da * log2_theta);
            sincosf((float)pos * freq, &sn[q], &cs[q]);
        }
    }
    for (int c0 = 0; c0 < nch; c0 += 64) {
        const int c = c0 + lane;
        const bool act = c < nch;
        u32x4 u = u32x4{0u, 0u, 0u, 0u};
        if (act) u = *reinterpret_cast<const u32x4*>(p + (int64_t)c * 8);
        float v[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[2 * k] = __uint_as_float(u[k] << 16);
            v[2 * k + 1] = __uint_as_float(u[k] & 0xffff0000u);
        }
        if (w) {
            float ss = 0.f;
#pragma unroll
            for (int k = 0; k < 8; ++k) ss += v[k] * v[k];
#pragma unroll
            for (int o = 1; o < CPH; o <<= 1) ss += __shfl_xor(ss, o);
            const float inv = 1.0f / sqrtf(ss / (float)HD + 1e-6f);
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = v[k] * inv * wv[k];
        }
        if (rot) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float y0 = v[2 * q] * cs[q] - v[2 * q + 1] * sn[q];
                const float y1 = v[2 * q] * sn[q] + v[2 * q + 1] * cs[q];
                v[2 * q] = y0;
                v[2 * q + 1] = y1;
            }
        }
        if (act) {
            const float os = qk ? 1.f : q_scale;
            u32x4 o;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const bf16 lo = (bf16)(v[2 * k] * os), hi = (bf16)(v[2 * k + 1] * os);
                o[k] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
            }
            *reinterpret_cast<u32x4*>(p + (int64_t)c * 8) = o;
        }
    }
}

int launch_qk_norm_rope(int dt, void* qkv, int64_t rows, int64_t ld, int D, int heads, int head_dim, const void* wq,
                        const void* wk, int rows_per_sample, int n_img, int gf, int gh, int gw, double theta,
                        float q_scale, hipStream_t s) {
    const bool rope = theta > 0.0 && n_img > 0;
    if (!wq && !wk && !rope && q_scale == 1.f) return BC_OK;
    if (head_dim < 2 || head_dim > 128 || head_dim % 2 || heads * head_dim != D || rows_per_sample < 1 ||
        (rope && (head_dim % 32 || (int64_t)gf * gh * gw != n_img)))
        return fail(BC_ERR_INVALID_ARG, "qk_norm_rope: head_dim %d, grid %d x %d x %d for %d tokens", head_dim, gf, gh,
                    gw, n_img);
    const int64_t waves = rows * heads * 2;
    if (waves < 1) return BC_OK;
    const float l2t = rope ? (float)std::log2(theta) : 0.f;
    const bool aligned = reinterpret_cast<uintptr_t>(qkv) % 16 == 0 && ld % 8 == 0 && D % 8 == 0;
    if (dt == BC_BF16 && aligned && (head_dim == 128 || head_dim == 64)) {
        const unsigned gr = (unsigned)((rows * 2 + 3) / 4);
        bf16* q = static_cast<bf16*>(qkv);
        const bf16 *a = static_cast<const bf16*>(wq), *b = static_cast<const bf16*>(wk);
        const int ni = rope ? n_img : 0;
        if (head_dim == 128)
            qk_norm_rope_row_kernel<16, bf16_tag><<<gr, 256, 0, s>>>(q, rows, ld, D, a, b, rows_per_sample, ni, gf, gh, gw, l2t, q_scale);
        else
            qk_norm_rope_row_kernel<8, bf16_tag><<<gr, 256, 0, s>>>(q, rows, ld, D, a, b, rows_per_sample, ni, gf, gh, gw, l2t, q_scale);
        return check_launch("qk_norm_rope_row");
    }
    const unsigned g = (unsigned)((waves + 3) / 4);
    if (dt == BC_BF16)
        qk_norm_rope_kernel<bf16_tag><<<g, 256, 0, s>>>(static_cast<bf16*>(qkv), rows, ld, D, heads, head_dim,
                                                    static_cast<const bf16*>(wq), static_cast<const bf16*>(wk),
                                                    rows_per_sample, rope ? n_img : 0, gf, gh, gw, l2t, q_scale);
    else
        qk_norm_rope_kernel<float><<<g, 256, 0, s>>>(static_cast<float*>(qkv), rows, ld, D, heads, head_dim,
                                                     static_cast<const float*>(wq), static_cast<const float*>(wk),
                                                     rows_per_sample, rope ? n_img : 0, gf, gh, gw, l2t, q_scale);
    return check_launch("qk_norm_rope");
}

// ---------------------------------------------------------------------------
// Blockwise mode: gated adds of module outputs into the fp32 residual stream,
// 8 consecutive elements per thread (16-byte loads of the bf16 sites).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load8(const bf16* p, float* v) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[2 * k] = __uint_as_float(u[k] << 16);
        v[2 * k + 1] = __uint_as_float(u[k] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8(const float* p, float* v) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[k] = a[k];
        v[4 + k] = b[k];
    }
}

template <typename T_>
__global__ __launch_bounds__(256) void gated_add_kernel(const elem_t<T_>* __restrict__ site, int64_t n8, int D,
                                                        float* __restrict__ x, const float* __restrict__ gate,
                                                        int64_t ldg, int rows_per_gate) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n8) return;
    const int64_t e = i * 8, r = e / D;
    const int d = (int)(e - r * D);
    float v[8], xv[8], g[8];
    load8(site + e, v);
    load8(x + e, xv);
    if (gate) load8(gate + (r / rows_per_gate) * ldg + d, g);
    else {
#pragma unroll
        for (int k = 0; k < 8; ++k) g[k] = 1.f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) xv[k] = fmaf(g[k], v[k], xv[k]);
    *reinterpret_cast<f32x4*>(x + e) = f32x4{xv[0], xv[1], xv[2], xv[3]};
    *reinterpret_cast<f32x4*>(x + e + 4) = f32x4{xv[4], xv[5], xv[6], xv[7]};
}

int launch_gated_add(int dt, const void* site, int64_t rows, int D, float* x, const float* gate, int64_t ldg,
                     int rows_per_gate, hipStream_t s) {
    if (D % 8 || reinterpret_cast<uintptr_t>(site) % 16 || reinterpret_cast<uintptr_t>(x) % 16 ||
        (gate && (reinterpret_cast<uintptr_t>(gate) % 16 || ldg % 4)) || rows_per_gate < 1)
        return fail(BC_ERR_INVALID_ARG, "gated_add: D %d, alignment", D);
    const int64_t n8 = rows * D / 8;
    if (n8 < 1) return BC_OK;
    const unsigned g = (unsigned)((n8 + 255) / 256);
    if (dt == BC_BF16) gated_add_kernel<bf16_tag><<<g, 256, 0, s>>>(static_cast<const bf16*>(site), n8, D, x, gate, ldg, rows_per_gate);
    else gated_add_kernel<float><<<g, 256, 0, s>>>(static_cast<const float*>(site), n8, D, x, gate, ldg, rows_per_gate);
    return check_launch("gated_add");
}

template <typename T_>
__global__ __launch_bounds__(256) void blockwise_forecast_kernel(BlockwiseArgs a) {
    typedef elem_t<T_> T;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i * 8 >= a.numel) return;
    const int64_t e = i * 8, r = e / a.D;
    const int d = (int)(e - r * a.D);
    const T* st = static_cast<const T*>(a.storage);
    const float* mrow = a.mods + (r / a.rows_per_gate) * a.ldm + d;
    float xv[8];
    load8(a.x + e, xv);
    for (int s = 0; s < a.nsites; ++s) {
        float f[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int j = 0; j < a.count; ++j) {
            float v[8];
            load8(st + ((int64_t)s * a.K + a.slot[j]) * a.numel + e, v);
#pragma unroll
            for (int k = 0; k < 8; ++k) f[k] = fmaf(a.w[j], v[k], f[k]);
        }
        float g[8];
        if (a.goff[s] >= 0) load8(mrow + a.goff[s], g);
        else {
#pragma unroll
            for (int k = 0; k < 8; ++k) g[k] = 1.f;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) xv[k] = fmaf(g[k], f[k], xv[k]);
    }
    *reinterpret_cast<f32x4*>(a.x + e) = f32x4{xv[0], xv[1], xv[2], xv[3]};
    *reinterpret_cast<f32x4*>(a.x + e + 4) = f32x4{xv[4], xv[5], xv[6], xv[7]};
}

int launch_blockwise_forecast(int dt, const BlockwiseArgs& a, hipStream_t s) {
    if (a.D % 8 || a.numel % 8 || a.nsites < 1 || a.nsites > kMaxSites || a.count < 1 || a.count > a.K ||
        a.K > kMaxK || a.ldm % 4 || reinterpret_cast<uintptr_t>(a.storage) % 16 ||
        reinterpret_cast<uintptr_t>(a.x) % 16 || reinterpret_cast<uintptr_t>(a.mods) % 16)
        return fail(BC_ERR_INVALID_ARG, "blockwise forecast: %d sites, count %d of %d", a.nsites, a.count, a.K);
    for (int j = 0; j < a.count; ++j)
        if (a.slot[j] < 0 || a.slot[j] >= a.K) return fail(BC_ERR_INVALID_ARG, "blockwise forecast: slot %d", a.slot[j]);
    for (int q = 0; q < a.nsites; ++q)
        if (a.goff[q] >= 0 && a.goff[q] % 4)   // (negative: no gate)
            return fail(BC_ERR_INVALID_ARG, "blockwise forecast: gate offset %d", a.goff[q]);
    const int64_t n8 = a.numel / 8;
    const unsigned g = (unsigned)((n8 + 255) / 256);
    if (dt == BC_BF16) blockwise_forecast_kernel<bf16_tag><<<g, 256, 0, s>>>(a);
    else blockwise_forecast_kernel<float><<<g, 256, 0, s>>>(a);
    return check_launch("blockwise_forecast");
}

// ---------------------------------------------------------------------------
// Relative L1 change of the adaptive schedule's probe: 16-byte chunks of cur
// and prev, |cur - prev| and |prev| summed per thread, per wave (butterfly)
// and per workgroup in a fixed order; prev takes cur's bytes in the same pass.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void abs_sums(const u32x4& c, const u32x4& p, float& sd, float& sp, bf16*) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float cl = __uint_as_float(c[i] << 16), ch = __uint_as_float(c[i] & 0xffff0000u);
        const float pl = __uint_as_float(p[i] << 16), ph = __uint_as_float(p[i] & 0xffff0000u);
        sd += fabsf(cl - pl) + fabsf(ch - ph);
        sp += fabsf(pl) + fabsf(ph);
    }
}
__device__ __forceinline__ void abs_sums(const u32x4& c, const u32x4& p, float& sd, float& sp, float*) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float cf = __uint_as_float(c[i]), pf = __uint_as_float(p[i]);
        sd += fabsf(cf - pf);
        sp += fabsf(pf);
    }
}

template <typename T_>
__global__ __launch_bounds__(256) void rel_l1_kernel(const elem_t<T_>* __restrict__ cur, elem_t<T_>* __restrict__ prev, int64_t n,
                                                     float* __restrict__ part) {
    typedef elem_t<T_> T;
    constexpr int E = 16 / (int)sizeof(T);
    const int64_t nc = n / E;
    const u32x4* c4 = reinterpret_cast<const u32x4*>(cur);
    u32x4* p4 = reinterpret_cast<u32x4*>(prev);
    float sd = 0.f, sp = 0.f;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nc; i += (int64_t)gridDim.x * 256) {
        const u32x4 c = c4[i], p = p4[i];
        abs_sums(c, p, sd, sp, (T*)nullptr);
        p4[i] = c;
    }
    if (blockIdx.x == 0) {
        for (int64_t i = nc * E + threadIdx.x; i < n; i += 256) {
            const float c = ld(cur + i), p = ld(prev + i);
            sd += fabsf(c - p);
            sp += fabsf(p);
            prev[i] = cur[i];
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        sd += __shfl_xor(sd, o);
        sp += __shfl_xor(sp, o);
    }
    __shared__ float red[2][4];
    const int wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        red[0][wv] = sd;
        red[1][wv] = sp;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
        const float* r = red[threadIdx.x];
        part[2 * blockIdx.x + threadIdx.x] = ((r[0] + r[1]) + r[2]) + r[3];
    }
}

__global__ __launch_bounds__(256) void rel_l1_sum_kernel(const float* __restrict__ part, int nblk,
                                                         double* __restrict__ sums) {
    __shared__ double ra[256], rb[256];
    const int t = threadIdx.x;
    double a = 0.0, b = 0.0;
    for (int i = t; i < nblk; i += 256) {
        a += (double)part[2 * i];
        b += (double)part[2 * i + 1];
    }
    ra[t] = a;
    rb[t] = b;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (t < h) {
            ra[t] += ra[t + h];
            rb[t] += rb[t + h];
        }
        __syncthreads();
    }
    if (t < 2) sums[t] = t == 0 ? ra[0] : rb[0];
}

int launch_rel_l1(int dt, const void* cur, void* prev, int64_t n, float* part, double* sums, hipStream_t s) {
    if (n < 1) return fail(BC_ERR_INVALID_ARG, "rel_l1: n=%lld", (long long)n);
    if (reinterpret_cast<uintptr_t>(cur) % 16 || reinterpret_cast<uintptr_t>(prev) % 16)
        return fail(BC_ERR_INVALID_ARG, "rel_l1: buffers must be 16-byte aligned");
    const int64_t nc = n / (16 / (int64_t)dtype_size(dt));
    const int nblk = (int)std::min<int64_t>(kRelL1Blocks, std::max<int64_t>(1, (nc + 1023) / 1024));
    if (dt == BC_BF16)
        rel_l1_kernel<bf16_tag><<<nblk, 256, 0, s>>>(static_cast<const bf16*>(cur), static_cast<bf16*>(prev), n, part);
    else
        rel_l1_kernel<float><<<nblk, 256, 0, s>>>(static_cast<const float*>(cur), static_cast<float*>(prev), n, part);
    const int rc = check_launch("rel_l1");
    if (rc != BC_OK) return rc;
    rel_l1_sum_kernel<<<1, 256, 0, s>>>(part, nblk, sums);
    return check_launch("rel_l1_sum");
}

}  // namespace bc
