/*
 * bc.h -- C ABI of libbarycache, an MI355X (gfx950) implementation of the hot
 * path of BaryCache sampling for Diffusion Transformers.
 *
 * Paper: "Memory-Efficient Training-Free Acceleration of Diffusion
 * Transformers with BaryCache".  On a full step the sampler runs the DiT layer
 * stack (Sec. 3.1, Eqs. 4-5) and stores its output, the stepwise feature, in a
 * cache context of the H most recent outputs (Sec. 3.2, Eq. 6).  On every other
 * step it forecasts the feature as a weighted sum of the cached ones
 * (Sec. 3.3, Eq. 13) with barycentric weights built from the step times alone
 * (Sec. 3.2, Eqs. 7-12).  Here H is called K.
 *
 * Conventions for every call:
 *   - Return value: a bc_status code; nothing is thrown across the ABI.  On an
 *     error, bc_last_error() (per thread) holds a message.
 *   - All arguments are checked before any work is enqueued: a call that
 *     returns BC_ERR_INVALID_ARG, BC_ERR_DEGENERATE or BC_ERR_STATE has had no
 *     effect on device memory or on any handle.
 *   - Device pointers are device addresses in the current HIP device's memory;
 *     the caller owns and allocates every device buffer (weights, features,
 *     the ring storage, workspaces).  The library never allocates device
 *     memory.  Handles own host memory only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device work is enqueued on it and the call returns without waiting;
 *     buffers must stay valid until that work has completed.  Errors that
 *     arise while kernels run surface at the caller's next synchronisation.
 *   - Matrices are row-major.  Linear weights are [out, in] with the input
 *     dimension contiguous; a linear layer computes y = x W^T + b.
 *   - Node order: t_nodes[0] is the time of the most recent cached feature
 *     (s_1 of Sec. 3.2), t_nodes[K-1] the oldest; weights follow that order.
 */
#ifndef BC_H
#define BC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BC_OK = 0,
    BC_ERR_INVALID_ARG = 1,   /* bad pointer, size, shape, dtype or parameter */
    BC_ERR_DEGENERATE = 2,    /* Eq. 11's normaliser is zero or not finite */
    BC_ERR_STATE = 3,         /* e.g. forecasting from an empty cache */
    BC_ERR_HIP = 4,           /* a HIP runtime call or launch failed */
    BC_ERR_UNSUPPORTED = 5    /* a shape outside what the kernels handle */
} bc_status;

typedef enum { BC_F32 = 0, BC_BF16 = 1 } bc_dtype;

const char* bc_status_str(int status);
/* Message of the last failing call on this thread ("" if none). */
const char* bc_last_error(void);
/* ABI version, (major << 16) | minor. */
int bc_version(void);
/* Hash of the sources, headers and compiler flags the library was built from
 * (a NUL-terminated hex string owned by the library), so a caller can refuse a
 * library that is older than its sources. */
const char* bc_build_id(void);

/* ------------------------------------------------------------------------ */
/* Barycentric weights (host, fp64)                                          */
/* ------------------------------------------------------------------------ */

typedef enum {
    BC_NODES_TRAPEZOID = 0,   /* numerators (-1)^j c_j, c = (1/2, 1, ..., 1, 1/2): Eqs. 8-9 */
    BC_NODES_LAGRANGE = 1     /* classical weights 1 / prod_{m!=j}(s_j - s_m) (polynomial interpolation) */
} bc_node_mode;

typedef enum {
    BC_BLEND_RECENT = 0,      /* w = (1 - lambda) alpha + lambda e_1 (mix with the most recent feature) */
    BC_BLEND_LITERAL = 1      /* Eq. 12 as printed: [(1-lambda) alpha_1..alpha_{K-1}, lambda alpha_K] */
} bc_blend_mode;

typedef struct {
    int nodes;       /* bc_node_mode */
    double clip_C;   /* clip bound of Eq. 10 (paper: 10); +inf disables the clip */
    double eta;      /* the small constant of Eq. 11 (paper: 1e-12) */
    double delta;    /* exponent of Eq. 11; < 0 selects delta_K: 1 (K<=2), 0.95 (K=3), 0.7 (K>=4) */
    double lambda;   /* blend factor of Eq. 12, in [0, 1] */
    int blend;       /* bc_blend_mode */
} bc_bary_params;

/* Paper defaults: trapezoid nodes, C = 10, eta = 1e-12, delta = delta_K,
 * lambda = 0, RECENT blend (Sec. 3.2; lambda = 0 is the image setting of
 * Sec. 4.1). */
void bc_bary_params_default(bc_bary_params* p);

/* The weight vector W of Eq. 12 for K nodes and query time t_query (Sec. 3.2,
 * Eqs. 8-12: raw weights u_j = b_j / (t - s_j), clip to [-C, C], signed power
 * sgn(u)(|u| + eta)^delta, normalisation to unit sum, blend).
 *   t_nodes: host [K] fp64, newest first; trapezoid mode needs them strictly
 *            monotone, Lagrange mode distinct.  1 <= K <= 8.
 *   w_out:   host [K] fp64, same order.
 * A query equal to a node gives +-inf before the clip in trapezoid mode and
 * the unit vector of that node in Lagrange mode.
 * Errors: INVALID_ARG (NULL, K out of range, non-finite or badly ordered
 * nodes, parameters out of range), DEGENERATE (zero or non-finite normaliser;
 * w_out untouched). */
int bc_bary_weights(const double* t_nodes, int K, double t_query, double* w_out);
int bc_bary_weights_ex(const double* t_nodes, int K, double t_query,
                       const bc_bary_params* p, double* w_out);

/* Full/forecast mask of the equal-spaced schedule (Sec. 3.3 and the schedule
 * ablation, Table 5): mask_out[k] = 1 (full) iff k % interval == 0, or
 * force_last and k == S-1; else 0.  mask_out: host [S]. */
int bc_make_mask(int S, int interval, int force_last, uint8_t* mask_out);

/* One step of the precomputed plan.  A full step writes the new feature to
 * ring slot `head` and then holds `count` features; a forecast step combines
 * the `count` newest features, node j in slot slots[j] with weight w[j]
 * (newest first).  Unused entries are -1 / 0. */
typedef struct {
    int is_full;
    int count;
    int head;
    int slots[8];
    double w[8];
} bc_plan_step;

/* The whole plan of a sampling run: the weights depend only on the schedule,
 * so they are all computed before the loop (the paper's "online decoupling",
 * Sec. 1 and Sec. 3.2 "Get Key").
 *   mask:   host [S], mask[0] must be 1.
 *   coords: host [S] node coordinate of each step, or NULL for coords[k] = k.
 *   K:      ring slots (history length H), 1..8.
 *   p:      weight parameters, or NULL for the defaults; delta < 0 uses
 *           delta of the node count actually available at each step.
 *   out:    host [S].
 * Errors: INVALID_ARG, DEGENERATE (names the step in bc_last_error()). */
int bc_plan(int S, const uint8_t* mask, const double* coords, int K,
            const bc_bary_params* p, bc_plan_step* out);

/* ------------------------------------------------------------------------ */
/* Cache context: an in-place ring of K feature tensors (Sec. 3.2, Eq. 6)    */
/* ------------------------------------------------------------------------ */

typedef struct bc_cache_ring bc_cache_ring;

/* Wrap caller-owned device storage of K * numel elements of `dtype` (slot i
 * starts at element i * numel) as an empty ring.  The handle holds host
 * metadata only: head, count and the node time of each slot. */
int bc_cache_create(int K, int64_t numel, int dtype, void* dev_storage, bc_cache_ring** out);
int bc_cache_destroy(bc_cache_ring* r);
/* Forget every cached feature (count = 0); storage is untouched. */
int bc_cache_reset(bc_cache_ring* r);
/* Device address of the slot the next push will fill, so a producer can write
 * the feature there directly and push it without a copy. */
int bc_cache_next_slot(const bc_cache_ring* r, void** dev_ptr);
/* Insert a feature computed at node time t as the newest entry, evicting the
 * oldest once K are held (the sliding window of Sec. 3.2).  `feat` is a device
 * pointer to numel elements of the ring's dtype, or NULL (or the next slot's
 * own address) when the producer already wrote the next slot: then no device
 * work is enqueued; otherwise one copy is enqueued on `stream`. */
int bc_cache_push(bc_cache_ring* r, const void* feat, double t, void* stream);
/* Ring state: count, head, and for j < count the node time and slot of node j
 * (newest first).  Any output pointer may be NULL; arrays need K entries. */
int bc_cache_state(const bc_cache_ring* r, int* count, int* head, double* t_nodes, int* slots);

/* Forecast x_hat = sum_j w[j] * node_j (Eq. 13) over the `count` newest cached
 * features: one fused pass that reads each feature once and writes `out`
 * (numel elements of out_dtype) once, accumulating in fp32 with the weights
 * rounded to fp32.
 *   w: host [count] fp64, newest first; 1 <= count <= ring count.
 * Errors: INVALID_ARG, STATE (count exceeds what the ring holds). */
int bc_bary_extrapolate(const bc_cache_ring* r, const double* w, int count,
                        void* out, int out_dtype, void* stream);

/* ------------------------------------------------------------------------ */
/* The layer stack (Sec. 3.1, Eqs. 4-5)                                      */
/* ------------------------------------------------------------------------ */

typedef enum {
    BC_BLOCK_DIT = 0,     /* adaLN-Zero DiT block */
    BC_BLOCK_PIXART = 1,  /* DiT block + cross-attention to a text context; modulation = t6 + table */
    BC_BLOCK_DUAL = 2,    /* image and text streams, joint attention */
    BC_BLOCK_SINGLE = 3   /* one stream over [image | text] tokens, fused projections */
} bc_block_kind;

typedef struct {
    int kind;       /* bc_block_kind */
    int B;          /* samples */
    int T;          /* image tokens per sample */
    int D;          /* hidden width; D == heads * head_dim */
    int heads;
    int head_dim;   /* 16..128, a multiple of 8 */
    int mlp;        /* MLP hidden width */
    int T_txt;      /* DUAL / SINGLE: text tokens per sample, else 0 */
    int T_ctx;      /* PIXART: context tokens per sample, else 0 */
    int dtype;      /* weights and activations: BC_F32 or BC_BF16 */
    /* DUAL / SINGLE: 3D rotary embedding of the image tokens' queries and keys
     * (the video model's attention).  The T image tokens form an
     * rope_f x rope_h x rope_w grid in (frame, row, column) order; pair i of a
     * head (dims 2i, 2i+1) lies in the frame, row or column axis (head_dim/8,
     * 7 head_dim/16, 7 head_dim/16 dims) and turns by pos * theta^(-2j/d_axis),
     * j its pair index within the axis.  rope_theta <= 0: none (then the grid
     * is ignored); else the grid product must be T and head_dim % 32 == 0.
     * Text tokens are never rotated. */
    int rope_f, rope_h, rope_w;
    double rope_theta;
} bc_block_desc;

/* One stream's parameters, device pointers in the block's dtype.
 *   DIT / DUAL stream: w_mod [6D, D], b_mod [6D], w_qkv [3D, D], b_qkv [3D],
 *     w_o [D, D], b_o [D], w_fc1 [mlp, D], b_fc1 [mlp], w_fc2 [D, mlp], b_fc2 [D].
 *   PIXART: w_mod is the per-block table [6, D] (b_mod unused), the rest as DIT.
 *   SINGLE: w_mod [3D, D], b_mod [3D]; w_qkv is the fused input projection
 *     [3D + mlp, D] with bias b_qkv; w_o is the fused output projection
 *     [D, D + mlp] with bias b_o; the fc pointers are unused.
 *   q_norm, k_norm (DUAL / SINGLE, optional, both or neither): [head_dim]
 *     scales of the RMSNorm applied to every head of the stream's queries and
 *     keys before attention (x / sqrt(mean(x^2) + 1e-6) * scale), ahead of the
 *     rotary embedding. */
typedef struct {
    const void *w_mod, *b_mod;
    const void *w_qkv, *b_qkv;
    const void *w_o, *b_o;
    const void *w_fc1, *b_fc1;
    const void *w_fc2, *b_fc2;
    const void *q_norm, *k_norm;
} bc_stream_weights;

typedef struct {
    bc_stream_weights img;     /* the (image) stream */
    bc_stream_weights txt;     /* DUAL: the text stream */
    const void *wx_q, *bx_q;   /* PIXART cross-attention: query [D, D], [D] */
    const void *wx_kv, *bx_kv; /*   keys|values from the context [2D, D], [2D] */
    const void *wx_o, *bx_o;   /*   output [D, D], [D] */
} bc_block_weights;

/* Bytes of workspace bc_dit_block_forward needs for this shape. */
int bc_block_workspace_size(const bc_block_desc* d, size_t* bytes);

/* One block on the residual stream, in place (Eq. 4 with the running residual
 * stream as the residual).
 *   x:    device fp32.  DIT / PIXART / DUAL: [B, T, D] image tokens.
 *         SINGLE: [B, T + T_txt, D] (each sample's image tokens then its text).
 *   x_txt: DUAL: device fp32 [B, T_txt, D] text tokens, in place; else NULL.
 *   c:    device fp32 conditioning.  DIT / DUAL / SINGLE: [B, D], the vector
 *         the modulation linear reads through SiLU.  PIXART: [B, 6D], the
 *         shared t6 vector to which the block's table is added.
 *   ctx:  PIXART: device [B, T_ctx, D] projected text context (block dtype);
 *         the block derives its keys/values with wx_kv.  Else NULL.
 *   ws:   device workspace of at least bc_block_workspace_size bytes, 256-byte
 *         aligned.
 * Activations between the kernels are in the block dtype; the residual stream,
 * LayerNorm statistics, softmax and every accumulation are fp32.
 * Errors: INVALID_ARG, UNSUPPORTED (head_dim or widths the kernels do not
 * tile), HIP. */
int bc_dit_block_forward(const bc_block_desc* d, const bc_block_weights* w,
                         float* x, float* x_txt, const float* c, const void* ctx,
                         void* ws, size_t ws_bytes, void* stream);

/* bc_dit_block_forward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the workspace is a device array of bc_noalloc_scratch_bytes()
 * bytes (96 MiB) inside the library, one per GPU, held from the library's load
 * until the process ends; the call allocates nothing.  The caller still owns
 * x, x_txt, c, ctx and the weights; arguments as bc_dit_block_forward.  Calls
 * on one GPU share that array and leave their intermediates in it: calls that
 * overlap on one GPU (other streams or host threads) race, so serialise them.
 * Errors: as bc_dit_block_forward; INVALID_ARG when the shape needs more
 * workspace than the array holds (bc_block_workspace_size > the limit), before
 * anything is enqueued; HIP if the array's device address cannot be found. */
int bc_dit_block_forward_noalloc(const bc_block_desc* d, const bc_block_weights* w,
                                 float* x, float* x_txt, const float* c, const void* ctx, void* stream);
size_t bc_noalloc_scratch_bytes(void);

/* ------------------------------------------------------------------------ */
/* Whole model and the sampling loop (Sec. 3.3)                              */
/* ------------------------------------------------------------------------ */

typedef enum { BC_MODEL_DIT = 0, BC_MODEL_PIXART = 1, BC_MODEL_MMDIT = 2 } bc_model_kind;

typedef struct {
    int kind;          /* bc_model_kind */
    int depth;         /* DIT / PIXART blocks; MMDIT dual-stream blocks */
    int depth_single;  /* MMDIT single-stream blocks */
    int D, heads, head_dim, mlp;
    int in_ch, out_ch, patch;
    int frames, height, width;  /* latent size; frames = 1 for images (latent [B, C, H, W]) */
    int n_classes;     /* DIT: class table rows = n_classes + 1 (0: unconditional) */
    int ctx_tokens, ctx_dim;    /* PIXART text: [B, ctx_tokens, ctx_dim] */
    int txt_tokens;    /* MMDIT text: [B, txt_tokens, D] */
    int freq_dim;      /* timestep sinusoid width, even */
    int dtype;         /* BC_F32 or BC_BF16: weights, activations and the ring */
    double rope_theta; /* MMDIT: 3D rotary embedding of the image tokens over the
                          (frames, height/patch, width/patch) grid, as in
                          bc_block_desc; <= 0: none.  Other kinds: 0. */
    double flow_shift; /* EULER sampler: time shift of the flow-matching schedule,
                          sigma_k = s u / (1 + (s - 1) u) with u = 1 - k/S; model
                          time 1000 sigma_k.  0 or 1: none; else > 0. */
} bc_model_desc;

/* Device pointers in the model dtype.  Token features are patches in
 * (p_h, p_w, channel) order; tokens run over (frame,) row, column. */
typedef struct {
    const void *t_w1, *t_b1, *t_w2, *t_b2;        /* timestep MLP: [D, freq_dim], [D], [D, D], [D] */
    const void *patch_w, *patch_b, *pos;          /* [D, in_ch p p], [D], [T, D] */
    const void *y_table;                          /* DIT with classes: [n_classes + 1, D] */
    const void *t6_w, *t6_b;                      /* PIXART: [6D, D], [6D] */
    const void *cap_w1, *cap_b1, *cap_w2, *cap_b2;/* PIXART caption MLP: [D, ctx_dim], [D], [D, D], [D] */
    const void *txt_w, *txt_b;                    /* MMDIT pooled-text projection: [D, D], [D] */
    const void *final_w_mod, *final_b_mod;        /* DIT / MMDIT: [2D, D], [2D]; PIXART: table [2, D] */
    const void *final_w, *final_b;                /* [out_ch p p, D], [out_ch p p] */
    const bc_block_weights* blocks;               /* host array: depth (+ depth_single) blocks */
} bc_model_weights;

typedef struct bc_model bc_model;

/* Validate and copy a model description and its weight pointers (the host
 * array `blocks` is copied; the device weights are referenced, not copied). */
int bc_model_create(const bc_model_desc* d, const bc_model_weights* w, bc_model** out);
int bc_model_destroy(bc_model* m);

typedef enum { BC_SAMPLER_DDIM = 0, BC_SAMPLER_DPMPP2M = 1, BC_SAMPLER_EULER = 2 } bc_sampler;

/* The step schedule: tau_out[k] the integer timestep (999 - floor(1000k/S))
 * and time_out[k] the value fed to the timestep embedding (tau for the
 * noise-prediction samplers, 1000 (1 - k/S) for Euler).  Either may be NULL. */
int bc_make_schedule(int sampler, int S, int32_t* tau_out, double* time_out);
/* As bc_make_schedule, with the flow-matching time shift s of bc_model_desc
 * applied to the EULER model times (1000 s u / (1 + (s - 1) u), u = 1 - k/S;
 * s = 0 or 1: none).  Errors: INVALID_ARG for s < 0 or not finite. */
int bc_make_schedule_shifted(int sampler, int S, double flow_shift, int32_t* tau_out, double* time_out);

/* Bytes of workspace bc_sample needs for B samples and an S-step schedule
 * (the per-step conditioning of the whole schedule is held at once). */
int bc_sample_workspace_size(const bc_model* m, int B, int S, size_t* bytes);

/* The BaryCache sampling loop (Sec. 3.3): for k = 0..S-1, a full step
 * (mask[k] = 1) runs the layer stack and its last block writes the stepwise
 * feature straight into the ring's next slot (Eq. 6's insertion); a forecast
 * step builds the feature from the ring with the precomputed weights
 * (Eq. 13).  Both then run the final layer and the sampler update.  The whole
 * loop is enqueued on `stream` without any host synchronisation.
 *   mask:    host [S], mask[0] = 1.
 *   K, p:    ring history length (must equal the ring's K) and weight params
 *            (NULL = defaults); node coordinate of step k is k.
 *   ring:    holds K slots of B*T*D elements of the model dtype; reset here.
 *   latents: device fp32 [B, in_ch, (frames,) height, width]; in: x_T, out: the sample.
 *   labels:  DIT with classes: device int64 [B]; else NULL.
 *   text:    PIXART: device [B, ctx_tokens, ctx_dim]; MMDIT: device [B, txt_tokens, D]
 *            (model dtype); else NULL.
 *   ws:      device workspace of bc_sample_workspace_size(m, B, S) bytes, 256-byte aligned.
 * The conditioning of every step (timestep MLP, class or text terms, the
 * final layer's and the blocks' adaLN vectors) depends only on the schedule,
 * labels and text, so it is computed up front in batched launches.
 * Errors: INVALID_ARG, DEGENERATE (a forecast step's weights), UNSUPPORTED, HIP. */
int bc_sample(const bc_model* m, int B, int sampler, int S, const uint8_t* mask,
              int K, const bc_bary_params* p, bc_cache_ring* ring, float* latents,
              const int64_t* labels, const void* text, void* ws, size_t ws_bytes,
              void* stream);

/* bc_sample with classifier-free guidance, as the paper's class-to-image runs
 * use it (Sec. 4.1, scale 1.5): a class-conditional DiT runs on a model batch
 * of 2B samples, the B `labels` and then B copies of the null class (row
 * n_classes of the class table), both reading the same latents; the stepwise
 * feature, and so every ring slot, covers all 2B samples (ring slots of
 * 2B*T*D elements); the update takes out_u + cfg_scale (out_c - out_u).
 * Workspace: bc_sample_workspace_size(m, 2B, S) bytes; B <= 32.
 * Errors: as bc_sample; UNSUPPORTED for models without classes; INVALID_ARG
 * for a non-finite scale. */
int bc_sample_cfg(const bc_model* m, int B, int sampler, int S, const uint8_t* mask,
                  int K, const bc_bary_params* p, bc_cache_ring* ring, float* latents,
                  const int64_t* labels, float cfg_scale, void* ws, size_t ws_bytes,
                  void* stream);

/* Blockwise mode (Sec. 4.5, Tables 5 and 6; the blockwise ratio Br = 0): the
 * cache holds, instead of the stack's output, every module's output before its
 * gate: per DIT block the attention output projection and the MLP output
 * (2 sites), per PIXART block also the cross-attention output (3 sites).
 * The number of sites of a model (depth * sites per block). */
int bc_blockwise_sites(const bc_model* m, int* nsites);

/* The sampling loop in blockwise mode.  A full step (mask[k] = 1) runs the
 * blocks and writes each module output ([B*T, D], model dtype) into its site's
 * ring slot (head + 1) mod K before adding it, gated, to the residual stream.
 * A forecast step embeds the current latent and adds, block by block, every
 * site's forecast (Eq. 13, the plan's weights for all sites) times the current
 * step's gate (the cross-attention has none), in one pass; the stream is then
 * the stepwise feature for the final layer.  Br = 1 is bc_sample itself; ratios
 * in between are not defined by the paper and not provided.
 *   site_storage: device [nsites][K][B*T*D] elements of the model dtype,
 *                 caller-owned, 16-byte aligned (bc_blockwise_sites);
 *   site_bytes:   its size in bytes (INVALID_ARG if smaller than that).
 *   K:            1..8 slots per site.
 *   ws:           bc_sample_workspace_size(m, B, S) bytes.
 * Other arguments as bc_sample (no ring: the sites are the cache).
 * Errors: as bc_sample; UNSUPPORTED for MMDIT models. */
int bc_sample_blockwise(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K,
                        const bc_bary_params* p, void* site_storage, size_t site_bytes, float* latents,
                        const int64_t* labels, const void* text, void* ws, size_t ws_bytes,
                        void* stream);

/* Bytes of workspace bc_sample_adaptive needs: bc_sample's plus the previous
 * step's probe (B*T*D elements of the model dtype), the first block's
 * (shift, scale) for every step and sample (S*B*2*D floats) and 8 KiB of
 * reduction partials. */
int bc_sample_adaptive_workspace_size(const bc_model* m, int B, int S, size_t* bytes);

/* The sampling loop under the adaptive schedule of Sec. 4.5 (Table 5): the
 * full/forecast decision is taken during the run from a feature probe instead
 * of a fixed mask.  At every step the latent is embedded and the first block's
 * modulated LayerNorm LN(x)(1 + scale1) + shift1 (image stream of the first
 * dual block for MMDIT) is the probe; for k >= 1 its change is
 *   change[k] = sum |probe_k - probe_{k-1}| / sum |probe_{k-1}|
 * over all B*T*D elements (sums in fp32 per workgroup, combined in double;
 * 0/0 = 0, x/0 = +inf).  Changes accumulate (in double, on the host) since the
 * last full step; step k runs the layer stack when k == 0, k == S-1, or the sum
 * reaches ell, and a full step empties the sum.  Forecast steps use the plan of
 * the full steps taken so far (Eq. 8-13), so the run equals bc_sample under the
 * mask it realises.  ell = 0: every step full; ell = +inf: only the first and
 * last.
 *   ell:        threshold, >= 0 (+inf allowed).
 *   mask_out:   host uint8 [S]: the realised mask (1 = full step).
 *   change_out: host double [S] or NULL: change[k] (change[0] = 0).
 *   ws:         bc_sample_adaptive_workspace_size(m, B, S) bytes, 256-byte aligned.
 * Other arguments as bc_sample.  The decision needs the change on the host:
 * the call copies two doubles back and synchronises `stream` once per step
 * after the first, so it returns when the run has finished, and it cannot be
 * captured into a graph.  Errors: as bc_sample; INVALID_ARG for a NaN or
 * negative threshold or NULL mask_out; HIP if the read-back fails (mask_out
 * and change_out then hold the steps decided so far). */
int bc_sample_adaptive(const bc_model* m, int B, int sampler, int S, double ell, int K,
                       const bc_bary_params* p, bc_cache_ring* ring, float* latents,
                       const int64_t* labels, const void* text, void* ws, size_t ws_bytes,
                       void* stream, uint8_t* mask_out, double* change_out);

/* The same sampling run captured once as a HIP graph and replayed, for
 * callers whose loop is launch-bound (small models, short schedules).
 * bc_sample_graph_create runs nothing: it records into a graph exactly the
 * work bc_sample would enqueue with these arguments, on `stream`, which must
 * not be the null stream and must not be capturing; kernel timing
 * (bc_profile_enable) must be off.  The ring's host state is left as it was.
 * bc_sample_graph_launch replays the run on `stream` (any stream) and leaves
 * the ring's host state as bc_sample would.  Every replay reads x_T from and
 * writes the sample to the same `latents` buffer (refill it in between), and
 * reads the same labels, text, weights and workspace, which must stay
 * allocated and in place while the graph exists; the graph holds no device
 * memory of its own.  Replays on one ring and workspace must not overlap.
 * Errors: as bc_sample; STATE (timing on, or the stream already capturing);
 * HIP (capture, instantiation or launch). */
typedef struct bc_sample_graph bc_sample_graph;
int bc_sample_graph_create(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K,
                           const bc_bary_params* p, bc_cache_ring* ring, float* latents,
                           const int64_t* labels, const void* text, void* ws, size_t ws_bytes,
                           void* stream, bc_sample_graph** out);
int bc_sample_graph_launch(bc_sample_graph* g, void* stream);
int bc_sample_graph_destroy(bc_sample_graph* g);

/* ------------------------------------------------------------------------ */
/* Building blocks exposed for measurement and tests                         */
/* ------------------------------------------------------------------------ */

typedef enum {
    BC_EPI_BIAS = 0,        /* out = acc + b (out in the dtype) */
    BC_EPI_BIAS_GELU = 1,   /* out = GELU_tanh(acc + b) */
    BC_EPI_GATE_RES = 2     /* out(fp32) = res(fp32) + gate[row / rows_per_gate] * (acc + b) */
} bc_epilogue;

/* y = epilogue(A W^T) for A [M, K] and W [N, K] in `dtype` (MFMA tiles on
 * gfx950).  out: [M, N] in `dtype`, or fp32 for GATE_RES.  bias: [N] dtype.
 * res, gate: GATE_RES only: res fp32 [M, N] (may alias out), gate fp32
 * [M / rows_per_gate, N].  K must be a multiple of 8. */
int bc_linear(int M, int N, int K, const void* A, const void* W, const void* bias,
              void* out, int epilogue, const float* res, const float* gate,
              int rows_per_gate, int dtype, void* stream);

/* Scaled dot-product attention softmax(Q K^T / sqrt(d)) V per (sample, head):
 * q [B, Tq, H, d], k and v [B, Tk, H, d], out [B, Tq, H, d], all `dtype`. */
int bc_attention(int B, int H, int Tq, int Tk, int d, const void* q, const void* k,
                 const void* v, void* out, int dtype, void* ws, size_t ws_bytes, void* stream);
int bc_attention_workspace_size(int B, int H, int Tq, int Tk, int d, int dtype, size_t* bytes);
/* As bc_attention with pre-scaled queries, the form the sampling loop's
 * projections write (the attention of Eq. 4's blocks): q already holds
 * q log2(e) / sqrt(d), so softmax(Q K^T / sqrt(d)) = normalised 2^(q_stored
 * k^T), and the kernel exponentiates the MFMA output directly.  bf16 only;
 * the same shapes, layouts, workspace and errors as bc_attention. */
int bc_attention_prescaled(int B, int H, int Tq, int Tk, int d, const void* q, const void* k,
                           const void* v, void* out, int dtype, void* ws, size_t ws_bytes, void* stream);

/* Per-kernel timing with HIP events on the stream each kernel is launched on.
 * While enabled for a kernel class, every launch of that class is bracketed by
 * two events (at most max_launches).  bc_profile_collect waits for them and
 * returns the summed duration and the number of launches, then disables.
 * Classes: 0 forecast, 1 GEMM with GELU epilogue, 2 GEMM gated residual with
 * K <= N (attention output projection), 3 GEMM bias (QKV), 4 attention,
 * 5 layernorm-modulate, 6 GEMM gated residual with K > N (MLP down
 * projection), 7 device copy (the ring push's copy path). */
int bc_profile_enable(int kernel_class, int max_launches);
int bc_profile_collect(int kernel_class, double* total_ms, int* launches);
/* As bc_profile_collect, but writes each launch's duration in ms, in launch
 * order, to ms_out (host, max_out entries; later launches are dropped) and
 * their number to *launches. */
int bc_profile_times(int kernel_class, float* ms_out, int max_out, int* launches);
/* As bc_profile_times, and work_out[i] (host, may be NULL) receives launch i's
 * algorithmic work: 2 M N K FLOPs for a GEMM, 4 B H Tq Tk d FLOPs for
 * attention (Q K^T and P V), bytes read plus written for the forecast
 * (n (K s_in + s_out)), the LayerNorm (rows D (s_in + s_out)) and a copy
 * (2 bytes).  A launch that is not the first of its library call records 0. */
int bc_profile_records(int kernel_class, float* ms_out, double* work_out, int max_out, int* launches);

#ifdef __cplusplus
}
#endif

#endif /* BC_H */
