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

// Timestep sinusoid of every step k < S: e[k, :] = [cos(t_k f_i), sin(t_k f_i)],
// f_i = 10000^(-i/half), where t_k is the step's model time (999 - floor(1000k/S),
// or 1000 flow_sigma(k, S, shift) for the flow-matching Euler sampler); fp32 out.
int launch_step_sinusoid(int sampler, int S, int dim, double shift, float* e, hipStream_t s);

// Per-(step, sample) conditioning c[k*B + b, :] = temb[k, :] + extra, where
// extra is table[labels[b], :] (table in `dt`, if labels), or add[b, :] (fp32,
// if add), or nothing.
int launch_build_cond(int dt, const float* temb, int S, int B, int D, const void* table, const int64_t* labels,
                      int n_rows, const float* add, float* c, hipStream_t s);

// out[i*B + b, :] = SiLU(c[rows[i]*B + b, :]) in `dt`, for i < n (n <= 64).
struct RowList { int row[kMaxSeg]; };
int launch_gather_silu(int dt, const float* c, int B, int D, const RowList& rows, int n, void* out, hipStream_t s);

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
// Model batch B reads latent sample b % lat_B (lat_B < B: the same latents
// for both halves of a guided batch).
int launch_patch_embed(int dt, const float* lat, LatentShape ls, int B, int lat_B, const void* W, const void* bias,
                       const void* pos, int D, float* x, hipStream_t s);

// Labels of a guided batch: out[b] = labels[b], out[B + b] = null_id, b < B.
int launch_cfg_labels(const int64_t* labels, int B, int64_t null_id, int64_t* out, hipStream_t s);

// Sampler update on fp32 latents x [B, C, F, H, W] from the model output in
// token layout out_tok [B*T, p*p*C_out] (first C channels used):
//   mode 0: x = c0 x + c1 e
//   mode 1 (DPM-Solver++(2M) data prediction): x0 = (x - c2 e) / c3;
//     D = c4 x0 + c5 prev; x = c0 x + c1 D; prev = x0 (prev may be NULL if c5 == 0)
//   mode 2: x = x0 computed as in mode 1 (final step)
struct SamplerCoef { float c[6]; int mode; };
// Guided (uncond_off > 0): the output used is u + cfg (c - u), with c at the
// element's own position and u uncond_off elements further (the null-class
// half of the batch).
int launch_sampler(const SamplerCoef& k, float* x, const float* out_tok, float* prev, LatentShape ls, int B, int C_out,
                   hipStream_t s, float cfg = 1.f, int64_t uncond_off = 0);

// The update of one latent element from its model output e (the modes above).
__device__ __forceinline__ void sampler_update(const SamplerCoef& k, float* x, float e, float* prev) {
    const float xv = *x;
    if (k.mode == 0) {
        *x = k.c[0] * xv + k.c[1] * e;
        return;
    }
    const float x0 = (xv - k.c[2] * e) / k.c[3];
    if (k.mode == 2) {
        *x = x0;
        return;
    }
    const float d = k.c[5] != 0.f ? k.c[4] * x0 + k.c[5] * *prev : k.c[4] * x0;
    *x = k.c[0] * xv + k.c[1] * d;
    if (prev) *prev = x0;
}

// Queries and keys of the video model's attention, in place on the QKV
// buffer (rows of ld elements: q at columns [0, D), k at [D, 2D)): per head,
// RMSNorm with the scales wq / wk ([head_dim], or NULL for none; eps 1e-6,
// fp32), then for the first n_img rows of every rows_per_sample the 3D rotary
// embedding over a gf x gh x gw token grid (theta <= 0: none); the queries
// are then multiplied by q_scale (the attention's pre-scaled queries; 1:
// none).  head_dim <= 128, even; with the rotation a multiple of 32.
int launch_qk_norm_rope(int dt, void* qkv, int64_t rows, int64_t ld, int D, int heads, int head_dim, const void* wq,
                        const void* wk, int rows_per_sample, int n_img, int gf, int gh, int gw, double theta,
                        float q_scale, hipStream_t s);

// Blockwise mode.  x [rows, D] fp32 (rows of rows_per_gate tokens per sample):
//   gated add:  x += gate[r / rows_per_gate] (.) site   (gate rows ldg floats
//               apart; NULL: a gate of one), site [rows, D] in `dt`;
//   forecast:   x += sum_s gate_s[r / rows_per_gate] (.) sum_j w[j] site_s(slot[j])
//               over the nsites sites of storage [site][K slots][rows * D],
//               gate_s at goff[s] floats into the modulation row of the sample
//               (goff[s] < 0: a gate of one), accumulated in fp32.
constexpr int kMaxSites = 96;
struct BlockwiseArgs {
    const void* storage;
    int64_t numel;                 // rows * D
    int nsites, K, count;
    int slot[kMaxK];
    float w[kMaxK];
    int goff[kMaxSites];
    const float* mods;
    int64_t ldm;
    int rows_per_gate, D;
    int64_t rows;
    float* x;
};
int launch_gated_add(int dt, const void* site, int64_t rows, int D, float* x, const float* gate, int64_t ldg,
                     int rows_per_gate, hipStream_t s);
int launch_blockwise_forecast(int dt, const BlockwiseArgs& a, hipStream_t s);

// Change measure of the adaptive schedule: over n elements of `dt`,
// sums[0] = sum |cur - prev| and sums[1] = sum |prev| (fp32 per thread and
// workgroup, the kRelL1Blocks partials `part` [2 * kRelL1Blocks] then added in
// double in a fixed order: the same inputs give the same sums), and prev = cur
// afterwards.  cur and prev 16-byte aligned.
constexpr int kRelL1Blocks = 1024;
int launch_rel_l1(int dt, const void* cur, void* prev, int64_t n, float* part, double* sums, hipStream_t s);

// Final step fused over 16-token groups, for bf16 models whose (D, p*p*C_out)
// has an instantiated variant (final_step_supported): the stepwise feature
// sum_j w[j] src[j] (rounded to bf16 like the unfused forecast), LayerNorm +
// adaLN (fmod [B, 2D]: shift, scale), the final linear (W [NO, D], bias [NO])
// and the sampler update of the latent pixels the tokens cover.  Returns
// BC_ERR_UNSUPPORTED for other shapes (the caller then runs the separate
// kernels).
constexpr int kFinalMaxK = 4;   // cached features the fused final step takes
struct FinalStepArgs {
    const void* src[8];
    float w[8];
    int K;
    int src_f32;          // one fp32 feature (K = 1) instead of K bf16 ones
    int guided;           // features and modulation hold 2B samples, the second half unconditional
    float cfg;            // guidance scale (guided)
    int B, T, D, NO, C_out;
    const float* fmod;
    const void* W;
    const void* bias;
    SamplerCoef sc;
    float* x;
    float* prev;
    LatentShape ls;
};
bool final_step_supported(int dt, int D, int NO, int T);
int launch_final_step(const FinalStepArgs& a, hipStream_t s);

}  // namespace bc
