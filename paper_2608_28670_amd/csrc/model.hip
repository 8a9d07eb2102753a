// Orchestration of the hot path on one HIP stream: the DiT-family blocks
// (Sec. 3.1, Eq. 4 with the running residual stream), the whole denoiser, and
// the BaryCache sampling loop (Sec. 3.3).
//
// Nothing here computes; it validates, lays out the caller's workspace and
// enqueues kernels.  The loop needs no device-to-host synchronisation: the
// full/forecast mask, the ring bookkeeping and every forecast weight are known
// before the first launch (the weights depend only on the schedule).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "attention.h"
#include "gemm.h"
#include "ops.h"

namespace bc {

// ---------------------------------------------------------------------------
// Workspace carving (every sub-buffer 256-byte aligned)
// ---------------------------------------------------------------------------
struct Carver {
    char* base;
    size_t off = 0;
    explicit Carver(void* b) : base(static_cast<char*>(b)) {}
    template <typename P> P* take(size_t bytes) {
        off = (off + 255) & ~size_t(255);
        P* p = base ? reinterpret_cast<P*>(base + off) : nullptr;
        off += bytes;
        return p;
    }
};

struct BlockBufs {
    void* h;        // [R, D]        LayerNorm output / cast of the stream
    void* qkv;      // [R, 3D]       (image rows, then text rows)
    void* attn;     // [R, D + F] for single-stream blocks, else [R, D]
    void* mlp;      // [R, F]
};

// wide_attn: the attention buffer doubles as the single-stream block's
// [attention | GELU(mlp)] input (R x (D + F)); need_mlp: a separate MLP hidden
// buffer for DiT / PixArt / dual-stream blocks.
static void carve_block(Carver& c, int dt, int64_t R, int D, int F, bool wide_attn, bool need_mlp, BlockBufs& b) {
    const size_t sz = dtype_size(dt);
    b.h = c.take<char>(R * D * sz);
    b.qkv = c.take<char>(R * 3 * D * sz);
    b.attn = c.take<char>(R * (wide_attn ? D + F : D) * sz);
    b.mlp = need_mlp ? c.take<char>(R * F * sz) : nullptr;
}

// Where the last gated residual of a block goes: the stream itself, or the
// ring slot of the stepwise feature (only the first `keep` of every `seg`
// rows, in `dt`).
struct BlockOut {
    void* ptr = nullptr;
    int dt = BC_F32;
    int seg = 0, keep = 0;
};

static GemmArgs gated_args(const void* A, int64_t lda, const void* W, const void* bias, int M, int N, int K, float* x,
                           const float* gate, int64_t ldg, int rows_per_gate, const BlockOut* out = nullptr) {
    GemmArgs g = gemm_args(A, lda, W, K, M, N, K);
    g.e.bias = bias;
    g.e.res = x;
    g.e.ldr = N;
    g.e.gate = gate;
    g.e.ldg = ldg;
    g.e.rows_per_gate = rows_per_gate;
    if (out && out->ptr) {
        g.e.out = out->ptr;
        g.e.out_f32 = out->dt == BC_F32;
        g.e.seg = out->seg;
        g.e.keep = out->keep;
    } else {
        g.e.out = x;
        g.e.out_f32 = 1;
    }
    g.e.ldo = N;
    return g;
}

static int gated(int dt, const void* A, int64_t lda, const void* W, const void* bias, int M, int N, int K, float* x,
                 const float* gate, int64_t ldg, int rows_per_gate, const BlockOut* out, hipStream_t s) {
    return launch_gemm(dt, BC_EPI_GATE_RES, gated_args(A, lda, W, bias, M, N, K, x, gate, ldg, rows_per_gate, out), s);
}

static GemmArgs plain_args(const void* A, int64_t lda, const void* W, const void* bias, int M, int N, int K, void* out,
                           bool gelu) {
    GemmArgs g = gemm_args(A, lda, W, K, M, N, K);
    g.e.bias = bias;
    g.e.out = out;
    g.e.ldo = N;
    if (gelu) g.e.gelu_from = 0;
    return g;
}

static int plain(int dt, const void* A, int64_t lda, const void* W, const void* bias, int M, int N, int K, void* out,
                 bool gelu, hipStream_t s) {
    return launch_gemm(dt, BC_EPI_BIAS, plain_args(A, lda, W, bias, M, N, K, out, gelu), s);
}

#define BC_TRY(x) do { const int _rc = (x); if (_rc != BC_OK) return _rc; } while (0)

// Projection whose first q_cols output columns are attention queries: they
// leave the epilogue multiplied by the softmax scale log2(e) / sqrt(head_dim),
// rounded once, and the attention takes them as pre-scaled (q_cols = 0: no
// queries, or their scale is applied after a norm that follows).
static int qproj(int dt, const void* A, int64_t lda, const void* W, const void* bias, int M, int N, int K, void* out,
                 int q_cols, int head_dim, hipStream_t s) {
    GemmArgs g = gemm_args(A, lda, W, K, M, N, K);
    g.e.bias = bias;
    g.e.out = out;
    g.e.ldo = N;
    g.e.q_scale_to = q_cols;
    g.e.q_scale = attn_q_scale(head_dim);
    return launch_gemm(dt, BC_EPI_BIAS, g, s);
}

// One DiT or PixArt block on x [B*T, D] (fp32).  mod: [B, >= 6D] fp32 rows
// ld_mod apart, ordered (shift1, scale1, gate1, shift2, scale2, gate2).
// sites (blockwise mode): the block's module outputs before their gates
// (attention, PixArt's cross-attention, MLP) are written there ([B*T, D] in
// the block dtype) and then added to x with their gates.
static int dit_block(const bc_block_desc& d, const bc_block_weights& w, float* x, const float* mod, int64_t ld_mod,
                     const void* ctx_kv, const BlockBufs& bb, const BlockOut* out, hipStream_t s,
                     void* const* sites = nullptr) {
    const int dt = d.dtype, D = d.D, F = d.mlp, T = d.T;
    const int M = d.B * T;
    const bc_stream_weights& sw = w.img;
    BC_TRY(launch_ln_mod(BC_F32, x, M, D, mod, mod + D, ld_mod, T, dt, bb.h, s));
    AttnArgs a = {};
    const size_t esz = dtype_size(dt);
    a.q_scaled = 1;
    a.o0 = a.o1 = bb.attn; a.ldo = D;
    a.B = d.B; a.H = d.heads; a.d = d.head_dim;
    auto al = [](const void* p, int n) { return reinterpret_cast<uintptr_t>(p) % n == 0; };
    if (qkv_attention_supported(dt, T, d.head_dim, D) && d.heads * d.head_dim == D && al(sw.w_qkv, 16) &&
        al(sw.b_qkv, 8)) {
        // Short sequences (DiT-XL/2's 256 tokens): the QKV projection and the
        // self-attention of a (sample, head) in one workgroup, Q, K and V in LDS.
        a.Tq0 = a.Tk0 = T;
        a.x = bb.h; a.ldx = D; a.w_qkv = sw.w_qkv; a.b_qkv = sw.b_qkv; a.dmodel = D;
        BC_TRY(launch_qkv_attention(dt, a, s));
    } else {
        BC_TRY(qproj(dt, bb.h, D, sw.w_qkv, sw.b_qkv, M, 3 * D, D, bb.qkv, D, d.head_dim, s));
        a.q0 = a.q1 = bb.qkv; a.Tq0 = T; a.ldq = 3 * D;
        a.k0 = a.k1 = static_cast<char*>(bb.qkv) + D * esz; a.Tk0 = T; a.ldk = 3 * D;
        a.v0 = a.v1 = static_cast<char*>(bb.qkv) + 2 * D * esz; a.ldv = 3 * D;
        BC_TRY(launch_attention(dt, a, s));
    }
    if (sites) {
        BC_TRY(plain(dt, bb.attn, D, sw.w_o, sw.b_o, M, D, D, sites[0], false, s));
        BC_TRY(launch_gated_add(dt, sites[0], M, D, x, mod + 2 * D, ld_mod, T, s));
    } else {
        BC_TRY(gated(dt, bb.attn, D, sw.w_o, sw.b_o, M, D, D, x, mod + 2 * D, ld_mod, T, nullptr, s));
    }
    if (d.kind == BC_BLOCK_PIXART) {
        // Cross-attention to the text context: no norm, no gate.
        BC_TRY(launch_convert(BC_F32, x, dt, bb.h, (int64_t)M * D, s));
        BC_TRY(qproj(dt, bb.h, D, w.wx_q, w.bx_q, M, D, D, bb.qkv, D, d.head_dim, s));
        AttnArgs c = {};
        c.q_scaled = 1;
        c.q0 = c.q1 = bb.qkv; c.Tq0 = T; c.ldq = D;
        c.k0 = c.k1 = ctx_kv; c.Tk0 = d.T_ctx; c.ldk = 2 * D;
        c.v0 = c.v1 = static_cast<const char*>(ctx_kv) + D * esz; c.ldv = 2 * D;
        c.o0 = c.o1 = bb.attn; c.ldo = D;
        c.B = d.B; c.H = d.heads; c.d = d.head_dim;
        BC_TRY(launch_attention(dt, c, s));
        if (sites) {
            BC_TRY(plain(dt, bb.attn, D, w.wx_o, w.bx_o, M, D, D, sites[1], false, s));
            BC_TRY(launch_gated_add(dt, sites[1], M, D, x, nullptr, 0, T, s));
        } else {
            BC_TRY(gated(dt, bb.attn, D, w.wx_o, w.bx_o, M, D, D, x, nullptr, 0, T, nullptr, s));
        }
    }
    BC_TRY(launch_ln_mod(BC_F32, x, M, D, mod + 3 * D, mod + 4 * D, ld_mod, T, dt, bb.h, s));
    BC_TRY(plain(dt, bb.h, D, sw.w_fc1, sw.b_fc1, M, F, D, bb.mlp, true, s));
    if (sites) {
        void* site = sites[d.kind == BC_BLOCK_PIXART ? 2 : 1];
        BC_TRY(plain(dt, bb.mlp, F, sw.w_fc2, sw.b_fc2, M, D, F, site, false, s));
        return launch_gated_add(dt, site, M, D, x, mod + 5 * D, ld_mod, T, s);
    }
    return gated(dt, bb.mlp, F, sw.w_fc2, sw.b_fc2, M, D, F, x, mod + 5 * D, ld_mod, T, out, s);
}

// Dual-stream block: image x [B*T, D] and text xt [B*Tt, D], each with its own
// modulation; attention is joint over the image then text tokens of a sample.
static int dual_block(const bc_block_desc& d, const bc_block_weights& w, float* x, float* xt, const float* mi,
                      const float* mt, int64_t ld_mod, const BlockBufs& bb, hipStream_t s) {
    const int dt = d.dtype, D = d.D, F = d.mlp, T = d.T, Tt = d.T_txt;
    const int Mi = d.B * T, Mt = d.B * Tt;
    const size_t esz = dtype_size(dt);
    char* qkv_i = static_cast<char*>(bb.qkv);
    char* qkv_t = qkv_i + (int64_t)Mi * 3 * D * esz;
    char* at_i = static_cast<char*>(bb.attn);
    char* at_t = at_i + (int64_t)Mi * D * esz;
    // Queries leave pre-scaled: from the QKV epilogue, or after their RMSNorm.
    const float qs = attn_q_scale(d.head_dim);
    const bool qn_i = w.img.q_norm != nullptr, qn_t = w.txt.q_norm != nullptr;
    BC_TRY(launch_ln_mod(BC_F32, x, Mi, D, mi, mi + D, ld_mod, T, dt, bb.h, s));
    BC_TRY(qproj(dt, bb.h, D, w.img.w_qkv, w.img.b_qkv, Mi, 3 * D, D, qkv_i, qn_i ? 0 : D, d.head_dim, s));
    BC_TRY(launch_qk_norm_rope(dt, qkv_i, Mi, 3 * D, D, d.heads, d.head_dim, w.img.q_norm, w.img.k_norm, T, T,
                               d.rope_f, d.rope_h, d.rope_w, d.rope_theta, qn_i ? qs : 1.f, s));
    BC_TRY(launch_ln_mod(BC_F32, xt, Mt, D, mt, mt + D, ld_mod, Tt, dt, bb.h, s));
    BC_TRY(qproj(dt, bb.h, D, w.txt.w_qkv, w.txt.b_qkv, Mt, 3 * D, D, qkv_t, qn_t ? 0 : D, d.head_dim, s));
    BC_TRY(launch_qk_norm_rope(dt, qkv_t, Mt, 3 * D, D, d.heads, d.head_dim, w.txt.q_norm, w.txt.k_norm, Tt, 0, 0, 0,
                               0, 0.0, qn_t ? qs : 1.f, s));
    AttnArgs a = {};
    a.q_scaled = 1;
    a.q0 = qkv_i; a.q1 = qkv_t; a.Tq0 = T; a.Tq1 = Tt; a.ldq = 3 * D;
    a.k0 = qkv_i + D * esz; a.k1 = qkv_t + D * esz; a.Tk0 = T; a.Tk1 = Tt; a.ldk = 3 * D;
    a.v0 = qkv_i + 2 * D * esz; a.v1 = qkv_t + 2 * D * esz; a.ldv = 3 * D;
    a.o0 = at_i; a.o1 = at_t; a.ldo = D;
    a.B = d.B; a.H = d.heads; a.d = d.head_dim;
    BC_TRY(launch_attention(dt, a, s));
    // The output projections and the MLP: each text-stream GEMM shares a launch
    // with its image-stream counterpart (its tiles fill the image grid's last
    // round); the LayerNorm outputs and MLP hiddens hold image rows, then text rows.
    BC_TRY(launch_gemm_pair(dt, BC_EPI_GATE_RES,
                            gated_args(at_i, D, w.img.w_o, w.img.b_o, Mi, D, D, x, mi + 2 * D, ld_mod, T),
                            gated_args(at_t, D, w.txt.w_o, w.txt.b_o, Mt, D, D, xt, mt + 2 * D, ld_mod, Tt), s));
    char* h_i = static_cast<char*>(bb.h);
    char* h_t = h_i + (int64_t)Mi * D * esz;
    char* f_i = static_cast<char*>(bb.mlp);
    char* f_t = f_i + (int64_t)Mi * F * esz;
    BC_TRY(launch_ln_mod(BC_F32, x, Mi, D, mi + 3 * D, mi + 4 * D, ld_mod, T, dt, h_i, s));
    BC_TRY(launch_ln_mod(BC_F32, xt, Mt, D, mt + 3 * D, mt + 4 * D, ld_mod, Tt, dt, h_t, s));
    BC_TRY(launch_gemm_pair(dt, BC_EPI_BIAS, plain_args(h_i, D, w.img.w_fc1, w.img.b_fc1, Mi, F, D, f_i, true),
                            plain_args(h_t, D, w.txt.w_fc1, w.txt.b_fc1, Mt, F, D, f_t, true), s));
    return launch_gemm_pair(dt, BC_EPI_GATE_RES,
                            gated_args(f_i, F, w.img.w_fc2, w.img.b_fc2, Mi, D, F, x, mi + 5 * D, ld_mod, T),
                            gated_args(f_t, F, w.txt.w_fc2, w.txt.b_fc2, Mt, D, F, xt, mt + 5 * D, ld_mod, Tt), s);
}

// Single-stream block on x [B*(T+Tt), D]: mod (shift, scale, gate) [B, >= 3D].
static int single_block(const bc_block_desc& d, const bc_block_weights& w, float* x, const float* mod,
                        int64_t ld_mod, const BlockBufs& bb, const BlockOut* out, hipStream_t s) {
    const int dt = d.dtype, D = d.D, F = d.mlp, L = d.T + d.T_txt;
    const int M = d.B * L;
    const size_t esz = dtype_size(dt);
    BC_TRY(launch_ln_mod(BC_F32, x, M, D, mod, mod + D, ld_mod, L, dt, bb.h, s));
    // [qkv | GELU(mlp)]: the qkv part to its own buffer, the MLP part to
    // columns D.. of the output projection's input.
    GemmArgs g = gemm_args(bb.h, D, w.img.w_qkv, D, M, 3 * D + F, D);
    g.e.bias = w.img.b_qkv;
    g.e.out = bb.qkv;
    g.e.ldo = 3 * D;
    g.e.split = 3 * D;
    g.e.out2 = bb.attn;
    g.e.ldo2 = D + F;
    g.e.off2 = D;
    g.e.gelu_from = 3 * D;
    // Queries leave pre-scaled: from this epilogue, or after their RMSNorm.
    const bool qn = w.img.q_norm != nullptr;
    g.e.q_scale_to = qn ? 0 : D;
    g.e.q_scale = attn_q_scale(d.head_dim);
    BC_TRY(launch_gemm(dt, BC_EPI_BIAS, g, s));
    BC_TRY(launch_qk_norm_rope(dt, bb.qkv, M, 3 * D, D, d.heads, d.head_dim, w.img.q_norm, w.img.k_norm, L, d.T,
                               d.rope_f, d.rope_h, d.rope_w, d.rope_theta, qn ? attn_q_scale(d.head_dim) : 1.f, s));
    AttnArgs a = {};
    a.q_scaled = 1;
    a.q0 = a.q1 = bb.qkv; a.Tq0 = L; a.ldq = 3 * D;
    a.k0 = a.k1 = static_cast<char*>(bb.qkv) + D * esz; a.Tk0 = L; a.ldk = 3 * D;
    a.v0 = a.v1 = static_cast<char*>(bb.qkv) + 2 * D * esz; a.ldv = 3 * D;
    a.o0 = a.o1 = bb.attn; a.ldo = D + F;
    a.B = d.B; a.H = d.heads; a.d = d.head_dim;
    BC_TRY(launch_attention(dt, a, s));
    return gated(dt, bb.attn, D + F, w.img.w_o, w.img.b_o, M, D, D + F, x, mod + 2 * D, ld_mod, L, out, s);
}

static int check_block_desc(const bc_block_desc& d) {
    if (d.kind < BC_BLOCK_DIT || d.kind > BC_BLOCK_SINGLE) return fail(BC_ERR_INVALID_ARG, "block kind %d", d.kind);
    if (d.dtype != BC_F32 && d.dtype != BC_BF16) return fail(BC_ERR_INVALID_ARG, "dtype %d", d.dtype);
    if (d.B < 1 || d.T < 1 || d.D < 1 || d.heads < 1 || d.mlp < 1) return fail(BC_ERR_INVALID_ARG, "empty block shape");
    if (d.heads * d.head_dim != d.D) return fail(BC_ERR_INVALID_ARG, "heads*head_dim != D");
    if (d.T_txt < 0 || d.T_ctx < 0) return fail(BC_ERR_INVALID_ARG, "negative token count");
    if ((d.kind == BC_BLOCK_DUAL || d.kind == BC_BLOCK_SINGLE) ? d.T_txt < 1 && d.kind == BC_BLOCK_DUAL : d.T_txt != 0)
        return fail(BC_ERR_INVALID_ARG, "T_txt=%d does not fit block kind %d", d.T_txt, d.kind);
    if ((d.kind == BC_BLOCK_PIXART) != (d.T_ctx > 0)) return fail(BC_ERR_INVALID_ARG, "T_ctx only for PIXART");
    if (!attention_supported(d.head_dim)) return fail(BC_ERR_UNSUPPORTED, "head_dim %d", d.head_dim);
    if (d.dtype == BC_F32 && d.head_dim > 64) return fail(BC_ERR_UNSUPPORTED, "fp32 blocks need head_dim <= 64");
    if (d.rope_theta > 0.0) {
        if (d.kind != BC_BLOCK_DUAL && d.kind != BC_BLOCK_SINGLE)
            return fail(BC_ERR_INVALID_ARG, "rotary embedding only for DUAL / SINGLE blocks");
        if (d.rope_f < 1 || d.rope_h < 1 || d.rope_w < 1 || (int64_t)d.rope_f * d.rope_h * d.rope_w != d.T ||
            d.head_dim % 32 || !std::isfinite(d.rope_theta))
            return fail(BC_ERR_INVALID_ARG, "rotary grid %d x %d x %d for T=%d, head_dim %d", d.rope_f, d.rope_h,
                        d.rope_w, d.T, d.head_dim);
    }
    const int epc = d.dtype == BC_BF16 ? 8 : 4;
    if (d.D % 16 || d.mlp % epc || d.D > 4096) return fail(BC_ERR_UNSUPPORTED, "D=%d mlp=%d", d.D, d.mlp);
    return BC_OK;
}

static bool have(const void* p) { return p != nullptr; }

static int check_stream_weights(const bc_stream_weights& w, int kind) {
    if (have(w.q_norm) != have(w.k_norm)) return fail(BC_ERR_INVALID_ARG, "q_norm and k_norm go together");
    if (have(w.q_norm) && kind != BC_BLOCK_DUAL && kind != BC_BLOCK_SINGLE)
        return fail(BC_ERR_INVALID_ARG, "QK norm only for DUAL / SINGLE blocks");
    bool ok = have(w.w_mod) && have(w.w_qkv) && have(w.b_qkv) && have(w.w_o) && have(w.b_o);
    if (kind != BC_BLOCK_PIXART) ok = ok && have(w.b_mod);
    if (kind != BC_BLOCK_SINGLE) ok = ok && have(w.w_fc1) && have(w.b_fc1) && have(w.w_fc2) && have(w.b_fc2);
    return ok ? BC_OK : fail(BC_ERR_INVALID_ARG, "missing block weight");
}

static int check_block_weights(const bc_block_weights& w, int kind) {
    BC_TRY(check_stream_weights(w.img, kind));
    if (kind == BC_BLOCK_DUAL) BC_TRY(check_stream_weights(w.txt, kind));
    if (kind == BC_BLOCK_PIXART && !(have(w.wx_q) && have(w.bx_q) && have(w.wx_kv) && have(w.bx_kv) && have(w.wx_o) && have(w.bx_o)))
        return fail(BC_ERR_INVALID_ARG, "missing cross-attention weight");
    return BC_OK;
}

// Workspace of one standalone block call: block buffers, modulation vectors,
// and the PixArt context keys/values.
static size_t block_ws(const bc_block_desc& d, void* base, BlockBufs* bb, float** mod, float** mod_t, void** ctx_kv) {
    Carver c(base);
    const int64_t R = (int64_t)d.B * (d.T + d.T_txt);
    BlockBufs tmp;
    carve_block(c, d.dtype, R, d.D, d.mlp, d.kind == BC_BLOCK_SINGLE, d.kind != BC_BLOCK_SINGLE, bb ? *bb : tmp);
    float* m = c.take<float>((size_t)d.B * 6 * d.D * sizeof(float));
    float* mt = c.take<float>(d.kind == BC_BLOCK_DUAL ? (size_t)d.B * 6 * d.D * sizeof(float) : 0);
    void* kv = c.take<char>(d.kind == BC_BLOCK_PIXART ? (size_t)d.B * d.T_ctx * 2 * d.D * dtype_size(d.dtype) : 0);
    if (mod) *mod = m;
    if (mod_t) *mod_t = mt;
    if (ctx_kv) *ctx_kv = kv;
    return c.off + 256;
}

static SkinnyArgs skinny1(const void* W, const void* b, int N, int K, int B, const float* in, float* out,
                          int act_in, int act_out) {
    SkinnyArgs a;
    std::memset(&a, 0, sizeof a);
    a.W[0] = W; a.bias[0] = b;
    a.nseg = 1; a.Nseg = N; a.K = K; a.B = B;
    a.in = in; a.ld_in = K; a.out = out; a.ld_out = N;
    a.act_in = act_in; a.act_out = act_out;
    return a;
}

}  // namespace bc

// ---------------------------------------------------------------------------
// Model handle
// ---------------------------------------------------------------------------
struct bc_model {
    bc_model_desc d;
    bc_model_weights w;
    std::vector<bc_block_weights> blocks;
};

namespace bc {

struct SampleWs {
    BlockBufs bb;
    float *x, *x_img, *x_txt;                 // residual streams
    float *e, *t1, *temb;                     // per step: sinusoid, hidden, timestep embedding
    float *c;                                 // per (step, sample): conditioning vector
    void* sc;                                 // SiLU(c) (or SiLU(t) for PixArt) rows, model dtype
    float* fmod;                              // per (step, sample): final-layer (shift, scale)
    float *mods, *mods_s;                     // per (full step, sample): block modulation
    float* t6;                                // PixArt: per (full step, sample) t6
    float *pooled, *txtp;                     // MMDiT pooled text and its projection
    void *cap_h, *ctx, *ctx_kv;               // PixArt text context
    void* feat;                               // forecast output [B*T, D] (model dtype)
    float *out, *prev;                        // model output (token layout), DPM-Solver++ history
    int full_chunk;                           // full steps whose modulation is held at once
    size_t bytes;
    int64_t* labels2;     // labels of a guided batch (the conditional half, then the null class)
    // Adaptive schedule only: the previous step's probe [B*T, D] (model dtype),
    // the first block's (shift, scale) of every (step, sample) [S*B, 2D], and
    // the change measure's partial and final sums.
    void* probe;
    float *pmod, *part;
    double* sums;
};

static int64_t latent_spatial(const bc_model_desc& d) { return (int64_t)d.frames * d.height * d.width; }

static int model_tokens(const bc_model_desc& d) { return d.frames * (d.height / d.patch) * (d.width / d.patch); }

// Full steps whose block modulation is computed together: up to 256
// (step, sample) rows and at most kMaxSeg steps (one gather launch).
static int full_chunk_of(int B, int S) { return std::max(1, std::min({S, 256 / B, kMaxSeg})); }

static int64_t mod_width(const bc_model_desc& d) {
    return d.kind == BC_MODEL_MMDIT ? (int64_t)2 * d.depth * 6 * d.D : (int64_t)d.depth * 6 * d.D;
}

static SampleWs carve_sample(const bc_model_desc& d, int B, int S, void* base, bool adaptive = false) {
    Carver c(base);
    SampleWs w;
    const int T = model_tokens(d), D = d.D, F = d.mlp;
    const int Tt = d.kind == BC_MODEL_MMDIT ? d.txt_tokens : 0;
    const int64_t R = (int64_t)B * (T + Tt);
    const size_t esz = dtype_size(d.dtype);
    const size_t f4 = sizeof(float);
    carve_block(c, d.dtype, R, D, F, d.kind == BC_MODEL_MMDIT, true, w.bb);
    w.x = c.take<float>(R * D * f4);
    w.x_img = w.x;
    w.x_txt = nullptr;
    if (d.kind == BC_MODEL_MMDIT) {
        if (B == 1) {
            w.x_txt = w.x + (int64_t)T * D;            // one sample: [img | txt] is already the joint layout
        } else {
            w.x_img = c.take<float>((int64_t)B * T * D * f4);
            w.x_txt = c.take<float>((int64_t)B * Tt * D * f4);
        }
    }
    const int64_t SB = (int64_t)S * B;
    w.full_chunk = full_chunk_of(B, S);
    const int64_t FB = (int64_t)w.full_chunk * B;
    w.e = c.take<float>((size_t)S * d.freq_dim * f4);
    w.t1 = c.take<float>((size_t)S * D * f4);
    w.temb = c.take<float>((size_t)S * D * f4);
    w.c = c.take<float>((size_t)SB * D * f4);
    w.sc = c.take<char>((size_t)SB * D * esz);
    w.fmod = c.take<float>((size_t)SB * 2 * D * f4);
    w.mods = c.take<float>((size_t)FB * mod_width(d) * f4);
    w.mods_s = c.take<float>(d.kind == BC_MODEL_MMDIT ? (size_t)FB * d.depth_single * 3 * D * f4 : 0);
    w.t6 = c.take<float>(d.kind == BC_MODEL_PIXART ? (size_t)FB * 6 * D * f4 : 0);
    w.pooled = c.take<float>(d.kind == BC_MODEL_MMDIT ? (size_t)B * D * f4 : 0);
    w.txtp = c.take<float>(d.kind == BC_MODEL_MMDIT ? (size_t)B * D * f4 : 0);
    const bool px = d.kind == BC_MODEL_PIXART;
    w.cap_h = c.take<char>(px ? (size_t)B * d.ctx_tokens * D * esz : 0);
    w.ctx = c.take<char>(px ? (size_t)B * d.ctx_tokens * D * esz : 0);
    w.ctx_kv = c.take<char>(px ? (size_t)d.depth * B * d.ctx_tokens * 2 * D * esz : 0);
    w.feat = c.take<char>((size_t)B * T * D * esz);
    w.out = c.take<float>((size_t)B * d.out_ch * latent_spatial(d) * f4);
    w.prev = c.take<float>((size_t)B * d.in_ch * latent_spatial(d) * f4);
    w.labels2 = c.take<int64_t>((size_t)B * sizeof(int64_t));
    w.probe = c.take<char>(adaptive ? (size_t)B * T * D * esz : 0);
    w.pmod = c.take<float>(adaptive ? (size_t)SB * 2 * D * f4 : 0);
    w.part = c.take<float>(adaptive ? (size_t)kRelL1Blocks * 2 * f4 : 0);
    w.sums = c.take<double>(adaptive ? 2 * sizeof(double) : 0);
    w.bytes = c.off + 256;
    return w;
}

static bc_block_desc block_desc_of(const bc_model_desc& d, int B, int kind) {
    bc_block_desc b;
    b.kind = kind;
    b.B = B;
    b.T = model_tokens(d);
    b.D = d.D;
    b.heads = d.heads;
    b.head_dim = d.head_dim;
    b.mlp = d.mlp;
    b.T_txt = (kind == BC_BLOCK_DUAL || kind == BC_BLOCK_SINGLE) ? d.txt_tokens : 0;
    b.T_ctx = kind == BC_BLOCK_PIXART ? d.ctx_tokens : 0;
    b.dtype = d.dtype;
    const bool rope = d.kind == BC_MODEL_MMDIT && d.rope_theta > 0.0;
    b.rope_f = rope ? d.frames : 0;
    b.rope_h = rope ? d.height / d.patch : 0;
    b.rope_w = rope ? d.width / d.patch : 0;
    b.rope_theta = rope ? d.rope_theta : 0.0;
    return b;
}

// alpha_bar of the linear beta schedule 1e-4 .. 0.02 over 1000 steps.
static void alpha_bar(double* ab) {
    double p = 1.0;
    for (int i = 0; i < 1000; ++i) {
        p *= 1.0 - (1e-4 + (0.02 - 1e-4) * (double)i / 999.0);
        ab[i] = p;
    }
}

// Sampler coefficients of step k (see launch_sampler for their meaning).
static SamplerCoef sampler_coef(int sampler, int k, int S, const int32_t* tau, const double* ab, double* h_prev,
                                double shift) {
    SamplerCoef c;
    std::memset(&c, 0, sizeof c);
    if (sampler == BC_SAMPLER_EULER) {
        c.mode = 0;
        c.c[0] = 1.f;
        c.c[1] = (float)(flow_sigma(k + 1, S, shift) - flow_sigma(k, S, shift));
        return c;
    }
    const double a = ab[tau[k]];
    const double a2 = k + 1 < S ? ab[tau[k + 1]] : 1.0;
    if (sampler == BC_SAMPLER_DDIM) {
        c.mode = 0;
        c.c[0] = (float)std::sqrt(a2 / a);
        c.c[1] = (float)(std::sqrt(1.0 - a2) - std::sqrt(a2 * (1.0 - a) / a));
        return c;
    }
    // DPM-Solver++(2M), data prediction.
    const double al = std::sqrt(a), sg = std::sqrt(1.0 - a);
    c.c[2] = (float)sg;
    c.c[3] = (float)al;
    if (k == S - 1) {
        c.mode = 2;
        return c;
    }
    const double al2 = std::sqrt(a2), sg2 = std::sqrt(1.0 - a2);
    const double h = std::log(al2 / sg2) - std::log(al / sg);
    c.mode = 1;
    c.c[0] = (float)(sg2 / sg);
    c.c[1] = (float)(-al2 * (std::exp(-h) - 1.0));
    if (k == 0) {
        c.c[4] = 1.f;
        c.c[5] = 0.f;
    } else {
        const double r = *h_prev / h;
        c.c[4] = (float)(1.0 + 1.0 / (2.0 * r));
        c.c[5] = (float)(-1.0 / (2.0 * r));
    }
    *h_prev = h;
    return c;
}

}  // namespace bc

using namespace bc;

extern "C" {

int bc_block_workspace_size(const bc_block_desc* d, size_t* bytes) {
    clear_error();
    if (!d || !bytes) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    BC_TRY(check_block_desc(*d));
    *bytes = block_ws(*d, nullptr, nullptr, nullptr, nullptr, nullptr);
    return BC_OK;
}

int bc_dit_block_forward(const bc_block_desc* dp, const bc_block_weights* wp, float* x, float* x_txt, const float* c,
                         const void* ctx, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (!dp || !wp || !x || !c || !ws) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    const bc_block_desc& d = *dp;
    BC_TRY(check_block_desc(d));
    BC_TRY(check_block_weights(*wp, d.kind));
    if (d.kind == BC_BLOCK_DUAL && !x_txt) return fail(BC_ERR_INVALID_ARG, "dual-stream block needs x_txt");
    if (d.kind == BC_BLOCK_PIXART && !ctx) return fail(BC_ERR_INVALID_ARG, "PixArt block needs ctx");
    if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(BC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    BlockBufs bb;
    float *mod, *mod_t;
    void* kv;
    const size_t need = block_ws(d, ws, &bb, &mod, &mod_t, &kv);
    if (ws_bytes < need) return fail(BC_ERR_INVALID_ARG, "workspace %zu < %zu bytes", ws_bytes, need);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bc_block_weights& w = *wp;
    const int D = d.D;
    if (d.kind == BC_BLOCK_PIXART) {
        const void* tab = w.img.w_mod;
        BC_TRY(launch_add_tables(d.dtype, c, 6 * D, &tab, 1, 6 * D, d.B, mod, 6 * D, s));
        GemmArgs g = gemm_args(ctx, D, w.wx_kv, D, d.B * d.T_ctx, 2 * D, D);
        g.e.bias = w.bx_kv;
        g.e.out = kv;
        g.e.ldo = 2 * D;
        BC_TRY(launch_gemm(d.dtype, BC_EPI_BIAS, g, s));
        return dit_block(d, w, x, mod, 6 * D, kv, bb, nullptr, s);
    }
    const int nm = d.kind == BC_BLOCK_SINGLE ? 3 : 6;
    BC_TRY(launch_skinny(d.dtype, skinny1(w.img.w_mod, w.img.b_mod, nm * D, D, d.B, c, mod, 1, 0), s));
    if (d.kind == BC_BLOCK_DIT) return dit_block(d, w, x, mod, 6 * D, nullptr, bb, nullptr, s);
    if (d.kind == BC_BLOCK_SINGLE) return single_block(d, w, x, mod, 3 * D, bb, nullptr, s);
    BC_TRY(launch_skinny(d.dtype, skinny1(w.txt.w_mod, w.txt.b_mod, 6 * D, D, d.B, c, mod_t, 1, 0), s));
    return dual_block(d, w, x, x_txt, mod, mod_t, 6 * D, bb, s);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free block forward: the workspace of bc_dit_block_forward is a
// file-scope device array, so the call needs no allocation by the library or
// the caller.  Each GPU the library runs on holds its own copy of the array
// (kNoAllocScratchBytes) from module load until the process ends.  Host code
// never passes the array's name to a kernel (on the host it only stands in for
// the symbol): its device address is looked up once per device with
// hipGetSymbolAddress and kept.
// ---------------------------------------------------------------------------
namespace bc {

constexpr size_t kNoAllocScratchBytes = size_t(96) << 20;
constexpr int kNoAllocMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kNoAllocMaxDevices];

// Device address of `scratch` on the current device (looked up on the first
// call on that device).
static int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(BC_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kNoAllocMaxDevices) return fail(BC_ERR_UNSUPPORTED, "device %d", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(BC_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return BC_OK;
}

}  // namespace bc

extern "C" {

size_t bc_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

int bc_dit_block_forward_noalloc(const bc_block_desc* dp, const bc_block_weights* wp, float* x, float* x_txt,
                                 const float* c, const void* ctx, void* stream) {
    clear_error();
    if (!dp) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    BC_TRY(check_block_desc(*dp));
    const size_t need = block_ws(*dp, nullptr, nullptr, nullptr, nullptr, nullptr);
    if (need > kNoAllocScratchBytes)
        return fail(BC_ERR_INVALID_ARG, "this block needs %zu bytes of workspace; the allocation-free entry point "
                    "holds %zu", need, kNoAllocScratchBytes);
    void* ws = nullptr;
    BC_TRY(scratch_address(&ws));
    return bc_dit_block_forward(dp, wp, x, x_txt, c, ctx, ws, kNoAllocScratchBytes, stream);
}

int bc_model_create(const bc_model_desc* dp, const bc_model_weights* wp, bc_model** out) {
    clear_error();
    if (!dp || !wp || !out) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    const bc_model_desc& d = *dp;
    if (d.kind < BC_MODEL_DIT || d.kind > BC_MODEL_MMDIT) return fail(BC_ERR_INVALID_ARG, "model kind %d", d.kind);
    if (d.dtype != BC_F32 && d.dtype != BC_BF16) return fail(BC_ERR_INVALID_ARG, "dtype %d", d.dtype);
    if (d.depth < 1 || d.depth_single < 0 || (d.kind != BC_MODEL_MMDIT && d.depth_single != 0))
        return fail(BC_ERR_INVALID_ARG, "depth %d / %d", d.depth, d.depth_single);
    if (d.depth > kMaxSeg || d.depth_single > kMaxSeg || (d.kind == BC_MODEL_MMDIT && 2 * d.depth > kMaxSeg))
        return fail(BC_ERR_UNSUPPORTED, "too many blocks");
    if (d.in_ch < 1 || d.out_ch < d.in_ch || d.patch < 1 || d.frames < 1 || d.height % d.patch || d.width % d.patch ||
        d.height < 1 || d.width < 1)
        return fail(BC_ERR_INVALID_ARG, "latent/patch shape");
    if (d.freq_dim < 2 || d.freq_dim % 2 || d.freq_dim % (d.dtype == BC_BF16 ? 8 : 4))
        return fail(BC_ERR_INVALID_ARG, "freq_dim %d", d.freq_dim);
    if (d.n_classes < 0 || (d.kind != BC_MODEL_DIT && d.n_classes))
        return fail(BC_ERR_INVALID_ARG, "n_classes only for DIT");
    if (d.kind == BC_MODEL_PIXART && (d.ctx_tokens < 1 || d.ctx_dim < 1 || d.ctx_dim % 8))
        return fail(BC_ERR_INVALID_ARG, "PixArt context %d x %d", d.ctx_tokens, d.ctx_dim);
    if (d.kind == BC_MODEL_MMDIT && d.txt_tokens < 1) return fail(BC_ERR_INVALID_ARG, "MMDiT needs txt_tokens");
    if (d.rope_theta != 0.0 && (d.kind != BC_MODEL_MMDIT || !(d.rope_theta > 0.0) || !std::isfinite(d.rope_theta)))
        return fail(BC_ERR_INVALID_ARG, "rope_theta only for MMDIT, > 0 and finite");
    if (!(d.flow_shift >= 0.0) || !std::isfinite(d.flow_shift))
        return fail(BC_ERR_INVALID_ARG, "flow_shift %g", d.flow_shift);
    const int kinds[2] = {d.kind == BC_MODEL_DIT ? BC_BLOCK_DIT : d.kind == BC_MODEL_PIXART ? BC_BLOCK_PIXART : BC_BLOCK_DUAL,
                          BC_BLOCK_SINGLE};
    for (int k = 0; k < (d.kind == BC_MODEL_MMDIT ? 2 : 1); ++k) {
        bc_block_desc bd = block_desc_of(d, 1, kinds[k]);
        BC_TRY(check_block_desc(bd));
    }
    const bc_model_weights& w = *wp;
    bool ok = have(w.t_w1) && have(w.t_b1) && have(w.t_w2) && have(w.t_b2) && have(w.patch_w) && have(w.patch_b) &&
              have(w.pos) && have(w.final_w_mod) && have(w.final_w) && have(w.final_b) && have(w.blocks);
    if (d.kind != BC_MODEL_PIXART) ok = ok && have(w.final_b_mod);
    if (d.kind == BC_MODEL_DIT && d.n_classes) ok = ok && have(w.y_table);
    if (d.kind == BC_MODEL_PIXART)
        ok = ok && have(w.t6_w) && have(w.t6_b) && have(w.cap_w1) && have(w.cap_b1) && have(w.cap_w2) && have(w.cap_b2);
    if (d.kind == BC_MODEL_MMDIT) ok = ok && have(w.txt_w) && have(w.txt_b);
    if (!ok) return fail(BC_ERR_INVALID_ARG, "missing model weight");
    const int nb = d.depth + d.depth_single;
    for (int l = 0; l < nb; ++l) BC_TRY(check_block_weights(w.blocks[l], l < d.depth ? kinds[0] : BC_BLOCK_SINGLE));
    bc_model* m = new (std::nothrow) bc_model;
    if (!m) return fail(BC_ERR_INVALID_ARG, "out of host memory");
    m->d = d;
    m->w = w;
    m->blocks.assign(w.blocks, w.blocks + nb);
    m->w.blocks = m->blocks.data();
    *out = m;
    return BC_OK;
}

int bc_model_destroy(bc_model* m) {
    clear_error();
    delete m;
    return BC_OK;
}

int bc_sample_workspace_size(const bc_model* m, int B, int S, size_t* bytes) {
    clear_error();
    if (!m || !bytes) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (B < 1 || B > 64) return fail(BC_ERR_INVALID_ARG, "B=%d outside [1, 64]", B);
    if (S < 1 || S > 1000) return fail(BC_ERR_INVALID_ARG, "S=%d outside [1, 1000]", S);
    *bytes = carve_sample(m->d, B, S, nullptr).bytes;
    return BC_OK;
}

int bc_sample_adaptive_workspace_size(const bc_model* m, int B, int S, size_t* bytes) {
    clear_error();
    if (!m || !bytes) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (B < 1 || B > 64) return fail(BC_ERR_INVALID_ARG, "B=%d outside [1, 64]", B);
    if (S < 1 || S > 1000) return fail(BC_ERR_INVALID_ARG, "S=%d outside [1, 1000]", S);
    *bytes = carve_sample(m->d, B, S, nullptr, true).bytes;
    return BC_OK;
}

}  // extern "C"

// Pinned host memory for the adaptive schedule's per-step read-back of two
// doubles (a copy into pageable memory costs tens of microseconds more per
// step).  Allocated on the run's first read-back and freed when the run
// returns, so the library holds no host memory between calls.
struct PinnedReadback {
    double* buf = nullptr;
    double* get() {
        if (!buf) {
            void* p = nullptr;
            if (hipHostMalloc(&p, 256, hipHostMallocDefault) != hipSuccess) return nullptr;
            buf = static_cast<double*>(p);
        }
        return buf;
    }
    ~PinnedReadback() {
        if (buf) (void)hipHostFree(buf);
    }
};

// Blockwise mode: the module sites' ring storage, [site][slot][B*T*D].
struct BlockwiseIO {
    void* storage;
    size_t bytes;
};

// Module sites per block in blockwise mode (attention, PixArt's
// cross-attention, MLP).
static int sites_per_block(const bc_model_desc& d) { return d.kind == BC_MODEL_PIXART ? 3 : 2; }

// The adaptive schedule's threshold and outputs (host arrays of S entries).
struct AdaptiveIO {
    double ell;
    uint8_t* mask_out;
    double* change_out;   // may be NULL
};

// The loop of bc_sample; guided: classifier-free guidance with scale cfg over
// a model batch of 2B (labels, then the null class) for B latents.  With `ad`
// the mask is not given but decided step by step (adaptive schedule), which
// reads two sums back to the host at every step after the first.
static int sample_run(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K, const bc_bary_params* p,
                      bc_cache_ring* ring, float* latents, const int64_t* labels, const void* text, bool guided,
                      float cfg, void* ws, size_t ws_bytes, void* stream, const AdaptiveIO* ad = nullptr,
                      const BlockwiseIO* bw = nullptr) {
    if (!m || !(mask || ad) || !(ring || bw) || !latents || !ws) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (bw && (ad || guided || !bw->storage || reinterpret_cast<uintptr_t>(bw->storage) % 16))
        return fail(BC_ERR_INVALID_ARG, "blockwise mode: 16-byte aligned site storage, fixed mask, no guidance");
    if (bw && m->d.kind == BC_MODEL_MMDIT)
        return fail(BC_ERR_UNSUPPORTED, "blockwise mode is built for DiT and PixArt models");
    if (ad && (guided || !ad->mask_out || !(ad->ell >= 0.0)))
        return fail(BC_ERR_INVALID_ARG, "adaptive schedule: mask_out required, threshold >= 0, no guidance");
    const bc_model_desc& d = m->d;
    const int Bm = guided ? 2 * B : B;     // model batch
    if (B < 1 || Bm > 64) return fail(BC_ERR_INVALID_ARG, "B=%d outside [1, %d]", B, guided ? 32 : 64);
    if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(BC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    const int T = model_tokens(d), D = d.D;
    if (bw) {
        if (K < 1 || K > kMaxK) return fail(BC_ERR_INVALID_ARG, "K=%d outside [1, %d]", K, kMaxK);
        if (d.depth * sites_per_block(d) > kMaxSites) return fail(BC_ERR_UNSUPPORTED, "too many module sites");
        const size_t need = (size_t)d.depth * sites_per_block(d) * K * Bm * T * D * dtype_size(d.dtype);
        if (bw->bytes < need) return fail(BC_ERR_INVALID_ARG, "site storage %zu < %zu bytes", bw->bytes, need);
    } else {
        if (K != ring->K) return fail(BC_ERR_INVALID_ARG, "K=%d but the ring has %d slots", K, ring->K);
        if (ring->dtype != d.dtype || ring->numel != (int64_t)Bm * T * D)
            return fail(BC_ERR_INVALID_ARG, "ring must hold %lld elements of the model dtype per slot",
                        (long long)Bm * T * D);
    }
    if (d.kind == BC_MODEL_DIT && d.n_classes && !labels) return fail(BC_ERR_INVALID_ARG, "class labels required");
    if (d.kind != BC_MODEL_DIT && !text) return fail(BC_ERR_INVALID_ARG, "text input required");
    std::vector<int32_t> tau(S > 0 ? S : 1);
    std::vector<double> tin(S > 0 ? S : 1);
    BC_TRY(bc_make_schedule_shifted(sampler, S, d.flow_shift, tau.data(), tin.data()));
    if (S < 1 || S > 1000) return fail(BC_ERR_INVALID_ARG, "S=%d outside [1, 1000]", S);
    std::vector<bc_plan_step> plan(S);
    std::vector<uint8_t> amask(S, 1);      // adaptive: the mask decided so far
    if (!ad) BC_TRY(bc_plan(S, mask, nullptr, K, p, plan.data()));
    else BC_TRY(bc_plan(S, amask.data(), nullptr, K, p, plan.data()));   // validates K and p
    const SampleWs w = carve_sample(d, Bm, S, ws, ad != nullptr);
    if (ws_bytes < w.bytes) return fail(BC_ERR_INVALID_ARG, "workspace %zu < %zu bytes", ws_bytes, w.bytes);

    hipStream_t s = static_cast<hipStream_t>(stream);
    const int dt = d.dtype, Tt = d.kind == BC_MODEL_MMDIT ? d.txt_tokens : 0;
    const size_t esz = dtype_size(dt);
    const LatentShape ls{d.in_ch, d.frames, d.height, d.width, d.patch};
    double ab[1000];
    alpha_bar(ab);
    double h_prev = 0.0;
    if (ring) bc_cache_reset(ring);
    const bc_block_weights* blk = m->w.blocks;
    const bc_model_weights& mw = m->w;
    const bc_block_desc bd_main = block_desc_of(d, Bm, d.kind == BC_MODEL_DIT ? BC_BLOCK_DIT
                                                       : d.kind == BC_MODEL_PIXART ? BC_BLOCK_PIXART : BC_BLOCK_DUAL);
    const bc_block_desc bd_single = block_desc_of(d, Bm, BC_BLOCK_SINGLE);
    if (guided) BC_TRY(launch_cfg_labels(labels, B, d.n_classes, w.labels2, s));
    const int64_t* mlabels = guided ? w.labels2 : labels;

    // Per-run text context.
    if (d.kind == BC_MODEL_PIXART) {
        const int Mc = B * d.ctx_tokens;
        BC_TRY(plain(dt, text, d.ctx_dim, mw.cap_w1, mw.cap_b1, Mc, D, d.ctx_dim, w.cap_h, true, s));
        BC_TRY(plain(dt, w.cap_h, D, mw.cap_w2, mw.cap_b2, Mc, D, D, w.ctx, false, s));
        for (int l = 0; l < d.depth; ++l)
            BC_TRY(plain(dt, w.ctx, D, blk[l].wx_kv, blk[l].bx_kv, Mc, 2 * D, D,
                         static_cast<char*>(w.ctx_kv) + (int64_t)l * Mc * 2 * D * esz, false, s));
    } else if (d.kind == BC_MODEL_MMDIT) {
        BC_TRY(launch_token_mean(dt, text, B, Tt, D, w.pooled, s));
        BC_TRY(launch_skinny(dt, skinny1(mw.txt_w, mw.txt_b, D, D, B, w.pooled, w.txtp, 0, 0), s));
    }

    // Conditioning of every step, computed before the loop: it depends only on
    // the schedule, the labels and the text, never on the latents.
    BC_TRY(launch_step_sinusoid(sampler, S, d.freq_dim, d.flow_shift, w.e, s));
    for (int k0 = 0; k0 < S; k0 += 64) {
        const int n = std::min(64, S - k0);
        BC_TRY(launch_skinny(dt, skinny1(mw.t_w1, mw.t_b1, D, d.freq_dim, n, w.e + (int64_t)k0 * d.freq_dim,
                                         w.t1 + (int64_t)k0 * D, 0, 1), s));
        BC_TRY(launch_skinny(dt, skinny1(mw.t_w2, mw.t_b2, D, D, n, w.t1 + (int64_t)k0 * D, w.temb + (int64_t)k0 * D, 0, 0), s));
    }
    const bool lab = d.kind == BC_MODEL_DIT && d.n_classes;
    BC_TRY(launch_build_cond(dt, w.temb, S, Bm, D, lab ? mw.y_table : nullptr, lab ? mlabels : nullptr, d.n_classes + 1,
                             d.kind == BC_MODEL_MMDIT ? w.txtp : nullptr, w.c, s));
    if (d.kind == BC_MODEL_PIXART) {
        const void* ft[2] = {mw.final_w_mod, static_cast<const char*>(mw.final_w_mod) + D * esz};
        BC_TRY(launch_add_tables(dt, w.c, D, ft, 2, D, S * Bm, w.fmod, 2 * D, s));
    } else {
        for (int k0 = 0; k0 < S; k0 += kMaxSeg) {
            const int n = std::min(kMaxSeg, S - k0);
            RowList rl;
            for (int i = 0; i < n; ++i) rl.row[i] = k0 + i;
            BC_TRY(launch_gather_silu(dt, w.c, Bm, D, rl, n,
                                      static_cast<char*>(w.sc) + (int64_t)k0 * Bm * D * esz, s));
        }
        GemmArgs fg = gemm_args(w.sc, D, mw.final_w_mod, D, S * Bm, 2 * D, D);
        fg.e.bias = mw.final_b_mod;
        fg.e.out = w.fmod;
        fg.e.ldo = 2 * D;
        fg.e.out_f32 = 1;
        BC_TRY(launch_gemm(dt, BC_EPI_BIAS, fg, s));
    }
    if (ad) {
        // The probe's modulation, the first block's (shift, scale), for every
        // step: SiLU(c) times the first 2D rows of the first block's (image
        // stream) modulation weights; PixArt: t6's first 2D entries plus the
        // block's table.
        if (d.kind == BC_MODEL_PIXART) {
            for (int k0 = 0; k0 < S; k0 += kMaxSeg) {
                const int n = std::min(kMaxSeg, S - k0);
                RowList rl;
                for (int i = 0; i < n; ++i) rl.row[i] = k0 + i;
                BC_TRY(launch_gather_silu(dt, w.c, Bm, D, rl, n,
                                          static_cast<char*>(w.sc) + (int64_t)k0 * Bm * D * esz, s));
            }
        }
        const bool px = d.kind == BC_MODEL_PIXART;
        GemmArgs pg = gemm_args(w.sc, D, px ? mw.t6_w : blk[0].img.w_mod, D, S * Bm, 2 * D, D);
        pg.e.bias = px ? mw.t6_b : blk[0].img.b_mod;
        pg.e.out = w.pmod;
        pg.e.ldo = 2 * D;
        pg.e.out_f32 = 1;
        BC_TRY(launch_gemm(dt, BC_EPI_BIAS, pg, s));
        if (px) {
            const void* tab[1] = {blk[0].img.w_mod};
            BC_TRY(launch_add_tables(dt, w.pmod, 2 * D, tab, 1, 2 * D, S * Bm, w.pmod, 2 * D, s));
        }
    }
    // Steps whose block modulation is needed: the full steps (known up front
    // unless the schedule is adaptive), every step in blockwise mode (the gates
    // of the forecast module outputs).
    std::vector<int> full_steps;
    for (int k = 0; k < S && !ad; ++k)
        if (plan[k].is_full || bw) full_steps.push_back(k);
    // Full steps whose modulation is computed together (one at a time when
    // they are decided during the loop).
    const int chunk = ad ? 1 : w.full_chunk;
    const int64_t ldm = mod_width(d);
    const int64_t lds = (int64_t)d.depth_single * 3 * D;
    // Block modulation of a chunk of full steps: rows (i, b) for the i-th full
    // step of the chunk; w.sc is reused for the gathered SiLU(c) rows.
    auto chunk_mods = [&](int f0) -> int {
        const int n = std::min<int>(chunk, (int)full_steps.size() - f0);
        RowList rl;
        for (int i = 0; i < n; ++i) rl.row[i] = full_steps[f0 + i];
        // (PixArt has no class or text term in c, so c is the timestep
        // embedding and SiLU(c) is t6's input.)
        BC_TRY(launch_gather_silu(dt, w.c, Bm, D, rl, n, w.sc, s));
        const int rows = n * Bm;
        if (d.kind == BC_MODEL_PIXART) {
            GemmArgs tg = gemm_args(w.sc, D, mw.t6_w, D, rows, 6 * D, D);
            tg.e.bias = mw.t6_b;
            tg.e.out = w.t6;
            tg.e.ldo = 6 * D;
            tg.e.out_f32 = 1;
            BC_TRY(launch_gemm(dt, BC_EPI_BIAS, tg, s));
            std::vector<const void*> tabs(d.depth);
            for (int l = 0; l < d.depth; ++l) tabs[l] = blk[l].img.w_mod;
            return launch_add_tables(dt, w.t6, 6 * D, tabs.data(), d.depth, 6 * D, rows, w.mods, ldm, s);
        }
        GemmSeg sg;
        std::memset(&sg, 0, sizeof sg);
        sg.Nseg = 6 * D;
        int nseg = 0;
        for (int l = 0; l < d.depth; ++l) {
            sg.W[nseg] = blk[l].img.w_mod; sg.bias[nseg] = blk[l].img.b_mod; ++nseg;
            if (d.kind == BC_MODEL_MMDIT) { sg.W[nseg] = blk[l].txt.w_mod; sg.bias[nseg] = blk[l].txt.b_mod; ++nseg; }
        }
        GemmArgs mg = gemm_args(w.sc, D, nullptr, D, rows, nseg * 6 * D, D);
        mg.e.out = w.mods;
        mg.e.ldo = ldm;
        mg.e.out_f32 = 1;
        BC_TRY(launch_gemm_grouped(dt, mg, sg, nseg, s));
        if (d.kind == BC_MODEL_MMDIT && d.depth_single) {
            GemmSeg ss;
            std::memset(&ss, 0, sizeof ss);
            ss.Nseg = 3 * D;
            for (int l = 0; l < d.depth_single; ++l) {
                ss.W[l] = blk[d.depth + l].img.w_mod;
                ss.bias[l] = blk[d.depth + l].img.b_mod;
            }
            GemmArgs sgm = gemm_args(w.sc, D, nullptr, D, rows, (int)lds, D);
            sgm.e.out = w.mods_s;
            sgm.e.ldo = lds;
            sgm.e.out_f32 = 1;
            BC_TRY(launch_gemm_grouped(dt, sgm, ss, d.depth_single, s));
        }
        return BC_OK;
    };

    // The fused final step needs 16-byte aligned features (ring slots, or the
    // blockwise sampler's fp32 stream in the workspace) and weights (checked
    // here once) and an instantiated (D, p*p*C_out).
    const bool fused_final = final_step_supported(dt, D, d.patch * d.patch * d.out_ch, T) && (D <= 1280 || !(guided || bw)) &&
                             reinterpret_cast<uintptr_t>(mw.final_w) % 16 == 0 &&
                             (bw ? reinterpret_cast<uintptr_t>(w.x) % 16 == 0
                                 : reinterpret_cast<uintptr_t>(ring->storage) % 16 == 0 && (ring->numel * esz) % 16 == 0);
    auto final_args = [&](const SamplerCoef& sc, const float* fmod) {
        FinalStepArgs fa;
        std::memset(&fa, 0, sizeof fa);
        fa.guided = guided ? 1 : 0;
        fa.cfg = cfg;
        fa.B = B; fa.T = T; fa.D = D; fa.NO = d.patch * d.patch * d.out_ch; fa.C_out = d.out_ch;
        fa.fmod = fmod;
        fa.W = mw.final_w;
        fa.bias = mw.final_b;
        fa.sc = sc;
        fa.x = latents;
        fa.prev = w.prev;
        fa.ls = ls;
        return fa;
    };

    int full_index = 0;
    double acc = 0.0;   // adaptive: changes summed since the last full step
    PinnedReadback readback;
    for (int k = 0; k < S; ++k) {
        if (ad) {
            // Probe at this step's latent: the embedding (which a full step
            // then uses) and the first block's modulated LayerNorm.
            BC_TRY(launch_patch_embed(dt, latents, ls, Bm, B, mw.patch_w, mw.patch_b, mw.pos, D, w.x_img, s));
            BC_TRY(launch_ln_mod(BC_F32, w.x_img, (int64_t)Bm * T, D, w.pmod + (int64_t)k * Bm * 2 * D,
                                 w.pmod + (int64_t)k * Bm * 2 * D + D, 2 * D, T, dt, w.bb.h, s));
            const int64_t n = (int64_t)Bm * T * D;
            double change = 0.0;
            if (k == 0) {
                BC_TRY(launch_copy(w.bb.h, w.probe, n * (int64_t)esz, s));
            } else {
                BC_TRY(launch_rel_l1(dt, w.bb.h, w.probe, n, w.part, w.sums, s));
                double* sums = readback.get();
                if (!sums) return fail(BC_ERR_HIP, "adaptive change readback: no pinned host buffer");
                hipError_t e = hipMemcpyAsync(sums, w.sums, 2 * sizeof(double), hipMemcpyDeviceToHost, s);
                if (e == hipSuccess) e = hipStreamSynchronize(s);
                if (e != hipSuccess) return fail(BC_ERR_HIP, "adaptive change readback: %s", hipGetErrorString(e));
                change = sums[1] > 0.0 ? sums[0] / sums[1] : sums[0] == 0.0 ? 0.0 : INFINITY;
            }
            bool full = true;
            if (k > 0 && k < S - 1) {
                acc += change;
                full = acc >= ad->ell;
            }
            if (full) acc = 0.0;
            amask[k] = full ? 1 : 0;
            ad->mask_out[k] = amask[k];
            if (ad->change_out) ad->change_out[k] = change;
            // The plan of step k depends only on the steps up to k.
            BC_TRY(bc_plan(k + 1, amask.data(), nullptr, K, p, plan.data()));
            if (full) full_steps.push_back(k);
        }
        const bc_plan_step& st = plan[k];
        const float* fmod = w.fmod + (int64_t)k * Bm * 2 * D;
        const int NO = d.patch * d.patch * d.out_ch;
        if (bw) {
            // Blockwise: a full step runs the blocks, writing every module's
            // output into its site's slot; a skipped step embeds the latent and
            // adds every site's gated forecast in one pass.  The feature is the
            // fp32 stream.
            const int fi = full_index % chunk;
            if (fi == 0) BC_TRY(chunk_mods(full_index));
            ++full_index;
            const float* mods = w.mods + (int64_t)fi * Bm * ldm;
            const int nq = sites_per_block(d);
            const int64_t numel = (int64_t)Bm * T * D;
            BC_TRY(launch_patch_embed(dt, latents, ls, Bm, B, mw.patch_w, mw.patch_b, mw.pos, D, w.x, s));
            if (st.is_full) {
                for (int l = 0; l < d.depth; ++l) {
                    void* sp[3];
                    for (int q = 0; q < nq; ++q)
                        sp[q] = static_cast<char*>(bw->storage) +
                                (((int64_t)(l * nq + q) * K + st.head) * numel) * (int64_t)esz;
                    BC_TRY(dit_block(bd_main, blk[l], w.x, mods + (int64_t)l * 6 * D, ldm,
                                     d.kind == BC_MODEL_PIXART ? static_cast<char*>(w.ctx_kv) + (int64_t)l * B * d.ctx_tokens * 2 * D * esz : nullptr,
                                     w.bb, nullptr, s, sp));
                }
            } else {
                BlockwiseArgs a;
                std::memset(&a, 0, sizeof a);
                a.storage = bw->storage;
                a.numel = numel;
                a.nsites = d.depth * nq;
                a.K = K;
                a.count = st.count;
                for (int j = 0; j < st.count; ++j) {
                    a.slot[j] = st.slots[j];
                    a.w[j] = (float)st.w[j];
                }
                for (int l = 0; l < d.depth; ++l)
                    for (int q = 0; q < nq; ++q)
                        a.goff[l * nq + q] = q == 0 ? l * 6 * D + 2 * D : (q + 1 == nq ? l * 6 * D + 5 * D : -1);
                a.mods = mods;
                a.ldm = ldm;
                a.rows_per_gate = T;
                a.D = D;
                a.rows = (int64_t)Bm * T;
                a.x = w.x;
                BC_TRY(launch_blockwise_forecast(dt, a, s));
            }
            const SamplerCoef sc = sampler_coef(sampler, k, S, tau.data(), ab, &h_prev, d.flow_shift);
            if (fused_final) {
                // The stream itself is the feature: final layer and update in one pass.
                FinalStepArgs fa = final_args(sc, fmod);
                fa.src_f32 = 1;
                fa.K = 1;
                fa.src[0] = w.x;
                fa.w[0] = 1.f;
                BC_TRY(launch_final_step(fa, s));
                continue;
            }
            BC_TRY(launch_ln_mod(BC_F32, w.x, (int64_t)Bm * T, D, fmod, fmod + D, 2 * D, T, dt, w.bb.h, s));
            GemmArgs fg = gemm_args(w.bb.h, D, mw.final_w, D, Bm * T, NO, D);
            fg.e.bias = mw.final_b;
            fg.e.out = w.out;
            fg.e.ldo = NO;
            fg.e.out_f32 = 1;
            BC_TRY(launch_gemm(dt, BC_EPI_BIAS, fg, s));
            BC_TRY(launch_sampler(sc, latents, w.out, w.prev, ls, B, d.out_ch, s));
            continue;
        }
        const void* feat;
        if (st.is_full) {
            void* slot = nullptr;
            BC_TRY(bc_cache_next_slot(ring, &slot));
            BlockOut out;
            out.ptr = slot;
            out.dt = dt;
            // Block modulation of this full step (computed a chunk of full steps at a time).
            const int fi = full_index % chunk;
            if (fi == 0) BC_TRY(chunk_mods(full_index));
            ++full_index;
            const float* mods = w.mods + (int64_t)fi * Bm * ldm;
            const float* mods_s = w.mods_s + (int64_t)fi * Bm * lds;
            if (!ad)   // (the adaptive loop embedded the latent for its probe)
                BC_TRY(launch_patch_embed(dt, latents, ls, Bm, B, mw.patch_w, mw.patch_b, mw.pos, D, w.x_img, s));
            if (d.kind == BC_MODEL_MMDIT) {
                BC_TRY(launch_convert(dt, text, BC_F32, w.x_txt, (int64_t)B * Tt * D, s));
                for (int l = 0; l < d.depth; ++l)
                    BC_TRY(dual_block(bd_main, blk[l], w.x_img, w.x_txt, mods + (int64_t)2 * l * 6 * D,
                                      mods + (int64_t)(2 * l + 1) * 6 * D, ldm, w.bb, s));
                if (w.x_img != w.x) {   // regroup [img | txt] per sample for the single-stream blocks
                    for (int b = 0; b < B; ++b) {
                        BC_TRY(launch_copy(w.x_img + (int64_t)b * T * D, w.x + (int64_t)b * (T + Tt) * D, (int64_t)T * D * 4, s));
                        BC_TRY(launch_copy(w.x_txt + (int64_t)b * Tt * D, w.x + ((int64_t)b * (T + Tt) + T) * D, (int64_t)Tt * D * 4, s));
                    }
                }
                out.seg = T + Tt;
                out.keep = T;
                for (int l = 0; l < d.depth_single; ++l)
                    BC_TRY(single_block(bd_single, blk[d.depth + l], w.x, mods_s + (int64_t)l * 3 * D, lds, w.bb,
                                        l + 1 == d.depth_single ? &out : nullptr, s));
                if (d.depth_single == 0) {   // stack ends with a dual block: cache its image stream
                    BC_TRY(launch_convert(BC_F32, w.x_img, dt, slot, (int64_t)B * T * D, s));
                }
            } else {
                out.seg = T;
                out.keep = T;
                for (int l = 0; l < d.depth; ++l)
                    BC_TRY(dit_block(bd_main, blk[l], w.x, mods + (int64_t)l * 6 * D, ldm,
                                     d.kind == BC_MODEL_PIXART ? static_cast<char*>(w.ctx_kv) + (int64_t)l * B * d.ctx_tokens * 2 * D * esz : nullptr,
                                     w.bb, l + 1 == d.depth ? &out : nullptr, s));
            }
            BC_TRY(bc_cache_push(ring, nullptr, (double)k, stream));
            feat = slot;
        }
        const SamplerCoef sc = sampler_coef(sampler, k, S, tau.data(), ab, &h_prev, d.flow_shift);
        if (fused_final && (st.is_full || st.count <= kFinalMaxK)) {
            // Stepwise feature (the new slot, or the forecast from the ring), final
            // layer and sampler update in one pass over the tokens.
            FinalStepArgs fa = final_args(sc, fmod);
            if (st.is_full) {
                fa.K = 1;
                fa.src[0] = feat;
                fa.w[0] = 1.f;
            } else {
                fa.K = st.count;
                for (int j = 0; j < st.count; ++j) {
                    fa.src[j] = ring->storage + (int64_t)st.slots[j] * ring->numel * esz;
                    fa.w[j] = (float)st.w[j];
                }
            }
            BC_TRY(launch_final_step(fa, s));
            continue;
        }
        if (!st.is_full) {
            const void* src[kMaxK];
            float wf[kMaxK];
            for (int j = 0; j < st.count; ++j) {
                src[j] = ring->storage + (int64_t)st.slots[j] * ring->numel * esz;
                wf[j] = (float)st.w[j];
            }
            BC_TRY(launch_forecast(src, wf, st.count, ring->numel, dt, w.feat, dt, s));
            feat = w.feat;
        }
        // Final layer: LayerNorm + adaLN, then the linear to p*p*C_out per token
        // (token layout; the sampler reads it back through unpatchify).
        BC_TRY(launch_ln_mod(dt, feat, (int64_t)Bm * T, D, fmod, fmod + D, 2 * D, T, dt, w.bb.h, s));
        GemmArgs fg = gemm_args(w.bb.h, D, mw.final_w, D, Bm * T, NO, D);
        fg.e.bias = mw.final_b;
        fg.e.out = w.out;
        fg.e.ldo = NO;
        fg.e.out_f32 = 1;
        BC_TRY(launch_gemm(dt, BC_EPI_BIAS, fg, s));
        BC_TRY(launch_sampler(sc, latents, w.out, w.prev, ls, B, d.out_ch, s, cfg, guided ? (int64_t)B * T * NO : 0));
    }
    return BC_OK;
}

extern "C" {

int bc_sample(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K, const bc_bary_params* p,
              bc_cache_ring* ring, float* latents, const int64_t* labels, const void* text, void* ws,
              size_t ws_bytes, void* stream) {
    clear_error();
    return sample_run(m, B, sampler, S, mask, K, p, ring, latents, labels, text, false, 1.f, ws, ws_bytes, stream);
}

int bc_sample_cfg(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K, const bc_bary_params* p,
                  bc_cache_ring* ring, float* latents, const int64_t* labels, float cfg_scale, void* ws,
                  size_t ws_bytes, void* stream) {
    clear_error();
    if (!m) return fail(BC_ERR_INVALID_ARG, "NULL model");
    if (m->d.kind != BC_MODEL_DIT || m->d.n_classes <= 0)
        return fail(BC_ERR_UNSUPPORTED, "classifier-free guidance needs a class-conditional DiT");
    if (!labels) return fail(BC_ERR_INVALID_ARG, "class labels required");
    if (!std::isfinite(cfg_scale)) return fail(BC_ERR_INVALID_ARG, "guidance scale must be finite");
    return sample_run(m, B, sampler, S, mask, K, p, ring, latents, labels, nullptr, true, cfg_scale, ws, ws_bytes,
                      stream);
}

int bc_blockwise_sites(const bc_model* m, int* nsites) {
    clear_error();
    if (!m || !nsites) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (m->d.kind == BC_MODEL_MMDIT) return fail(BC_ERR_UNSUPPORTED, "blockwise mode is built for DiT and PixArt models");
    *nsites = m->d.depth * sites_per_block(m->d);
    return BC_OK;
}

int bc_sample_blockwise(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K,
                        const bc_bary_params* p, void* site_storage, size_t site_bytes, float* latents,
                        const int64_t* labels, const void* text, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (!site_storage) return fail(BC_ERR_INVALID_ARG, "NULL site storage");
    const BlockwiseIO io{site_storage, site_bytes};
    return sample_run(m, B, sampler, S, mask, K, p, nullptr, latents, labels, text, false, 1.f, ws, ws_bytes, stream,
                      nullptr, &io);
}

int bc_sample_adaptive(const bc_model* m, int B, int sampler, int S, double ell, int K, const bc_bary_params* p,
                       bc_cache_ring* ring, float* latents, const int64_t* labels, const void* text, void* ws,
                       size_t ws_bytes, void* stream, uint8_t* mask_out, double* change_out) {
    clear_error();
    if (!mask_out) return fail(BC_ERR_INVALID_ARG, "mask_out required");
    if (!(ell >= 0.0)) return fail(BC_ERR_INVALID_ARG, "threshold must be >= 0 (got %g)", ell);
    const AdaptiveIO io{ell, mask_out, change_out};
    return sample_run(m, B, sampler, S, nullptr, K, p, ring, latents, labels, text, false, 1.f, ws, ws_bytes, stream,
                      &io);
}

}  // extern "C"

// A captured sampling run: the instantiated graph and the ring's host state
// at the end of the run (restored on every replay).
struct bc_sample_graph {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    bc_cache_ring* ring = nullptr;
    bc_cache_ring final_state;
};

extern "C" {

int bc_sample_graph_create(const bc_model* m, int B, int sampler, int S, const uint8_t* mask, int K,
                           const bc_bary_params* p, bc_cache_ring* ring, float* latents, const int64_t* labels,
                           const void* text, void* ws, size_t ws_bytes, void* stream, bc_sample_graph** out) {
    clear_error();
    if (!out || !ring) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    *out = nullptr;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (!s) return fail(BC_ERR_INVALID_ARG, "graph capture needs a stream other than the null stream");
    if (prof_any_enabled()) return fail(BC_ERR_STATE, "kernel timing is enabled; collect it before capturing");
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) return fail(BC_ERR_HIP, "hipStreamIsCapturing failed");
    if (cs != hipStreamCaptureStatusNone) return fail(BC_ERR_STATE, "the stream is already capturing");
    const bc_cache_ring before = *ring;
    if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess)
        return fail(BC_ERR_HIP, "hipStreamBeginCapture failed");
    const int rc = bc_sample(m, B, sampler, S, mask, K, p, ring, latents, labels, text, ws, ws_bytes, stream);
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(s, &graph);
    const bc_cache_ring after = *ring;
    *ring = before;   // nothing ran: the ring's host state is as it was
    if (rc != BC_OK || ec != hipSuccess || !graph) {
        if (graph) (void)hipGraphDestroy(graph);
        (void)hipGetLastError();
        return rc != BC_OK ? rc : fail(BC_ERR_HIP, "stream capture failed: %s", hipGetErrorString(ec));
    }
    hipGraphExec_t exec = nullptr;
    const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    if (ei != hipSuccess) {
        (void)hipGraphDestroy(graph);
        return fail(BC_ERR_HIP, "hipGraphInstantiate failed: %s", hipGetErrorString(ei));
    }
    bc_sample_graph* g = new bc_sample_graph;
    g->graph = graph;
    g->exec = exec;
    g->ring = ring;
    g->final_state = after;
    *out = g;
    return BC_OK;
}

int bc_sample_graph_launch(bc_sample_graph* g, void* stream) {
    clear_error();
    if (!g) return fail(BC_ERR_INVALID_ARG, "NULL graph");
    const hipError_t e = hipGraphLaunch(g->exec, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(BC_ERR_HIP, "hipGraphLaunch failed: %s", hipGetErrorString(e));
    *g->ring = g->final_state;
    return BC_OK;
}

int bc_sample_graph_destroy(bc_sample_graph* g) {
    clear_error();
    if (!g) return BC_OK;
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    if (g->graph) (void)hipGraphDestroy(g->graph);
    delete g;
    return BC_OK;
}

}  // extern "C"
