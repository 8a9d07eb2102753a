// Launchers of the small kernels around the block GEMMs and attention.
#pragma once

#include "hip_common.h"

namespace bc {

constexpr int kMaxSeg = 64;

// h[r, :] = LN(x[r, :]) * (1 + scale[b, :]) + shift[b, :] with b = r / rows_per_sample,
// LayerNorm without affine (eps 1e-6, fp32 statistics).  x: fp32 or `in_dt`,
// h: `out_dt`.  shift/scale rows are `ld_mod` floats apart.
int launch_ln_mod(int in_dt, const void* x, int64_t rows, int D, const float* shift, const float* scale,
                  int64_t ld_mod, int rows_per_sample, int out_dt, void* h, hipStream_t s);

// Skinny linear for per-sample vectors (B <= 64 rows), weights `dt`:
//   out[b, seg*Nseg + n] = act_out(sum_k act_in(in[b, k]) W_seg[n, k] + bias_seg[n])
// for each of `nseg` segments with their own W/bias; act: 0 none, 1 SiLU.
// `addend` (fp32 [B, nseg*Nseg] or NULL) is added after act_out.
struct SkinnyArgs {
    const void* W[kMaxSeg];
    const void* bias[kMaxSeg];
    int nseg, Nseg, K, B;
    const float* in;
    int64_t ld_in;
    float* out;
    int64_t ld_out;
    const float* addend;
    int act_in, act_out;
};
int launch_skinny(int dt, const SkinnyArgs& a, hipStream_t s);

// Timestep sinusoid e[b, :] = [cos(t f_i), sin(t f_i)], f_i = 10000^(-i/half), fp32 out.
int launch_sinusoid(double t, int B, int dim, float* e, hipStream_t s);

// c[b, :] = t[b, :] + table[labels[b], :] (table in `dt`).
int launch_add_label(int dt, const float* t, const void* table, const int64_t* labels, int B, int D, int n_rows,
                     float* c, hipStream_t s);

// out[b, seg*N + j] = vec[b, j] + table_seg[j]  (tables in `dt`, N entries each).
int launch_add_tables(int dt, const float* vec, int64_t ld_vec, const void* const* tables, int nseg, int N, int B,
                      float* out, int64_t ld_out, hipStream_t s);

// Mean over tokens: out[b, :] = mean_t x[b, t, :] (x in `dt`), fp32 out.
int launch_token_mean(int dt, const void* x, int B, int T, int D, float* out, hipStream_t s);

// Element-type conversion of n elements.
int launch_convert(int in_dt, const void* in, int out_dt, void* out, int64_t n, hipStream_t s);

struct LatentShape {
    int C, F, H, W, p;   // latent [B, C, F, H, W] (F = 1 for images), spatial patch p
    __host__ __device__ int tokens() const { return F * (H / p) * (W / p); }
};

// x[b, tok, :] = patchify(lat)[b, tok, :] W^T + bias + pos[tok, :], fp32 out.
int launch_patch_embed(int dt, const float* lat, LatentShape ls, int B, const void* W, const void* bias,
                       const void* pos, int D, float* x, hipStream_t s);

// Final layer on a feature [B*T, D] (fp32 or `feat_dt`): LN, modulate with
// shift/scale (fp32, rows ld_mod apart), linear to p*p*C_out (weights `dt`),
// scattered back to the latent layout out [B, C_out, F, H, W] (fp32).
int launch_final_layer(int feat_dt, const void* feat, int dt, const float* shift, const float* scale,
                       int64_t ld_mod, const void* W, const void* bias, LatentShape ls, int C_out, int B, int D,
                       float* out, hipStream_t s);

// Sampler update on fp32 latents x [B, C, S] from the model output [B, C_out, S]
// (first C channels used):
//   mode 0: x = c0 x + c1 e
//   mode 1 (DPM-Solver++(2M) data prediction): x0 = (x - c2 e) / c3;
//     D = c4 x0 + c5 prev; x = c0 x + c1 D; prev = x0 (prev may be NULL if c5 == 0)
//   mode 2: x = x0 computed as in mode 1 (final step)
struct SamplerCoef { float c[6]; int mode; };
int launch_sampler(const SamplerCoef& k, float* x, const float* eps, float* prev, int B, int C, int C_out,
                   int64_t S, hipStream_t s);

}  // namespace bc
