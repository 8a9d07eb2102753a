// Attention launcher interface shared by the block orchestration.
#pragma once

#include "hip_common.h"

namespace bc {

// Rows of each operand come from two segments: position p < T0 of sample b is
// row b*T0 + p of segment 0, otherwise row b*T1 + (p - T0) of segment 1.  Head
// h occupies columns [h*d, (h+1)*d) of a row; ld* are row strides (elements).
struct AttnArgs {
    const void *q0, *q1;
    int Tq0, Tq1;
    int64_t ldq;
    const void *k0, *k1;
    int Tk0, Tk1;
    int64_t ldk;
    const void *v0, *v1;
    int64_t ldv;
    void *o0, *o1;
    int64_t ldo;
    int B, H, d;
    // 1: q was written already multiplied by attn_q_scale(d) (its producer
    // rounded q * scale once), so scores leave the MFMA in log2 units.
    int q_scaled;
    float scale_log2;   // set by the launcher
    // launch_qkv_attention only: the block input x [B*T, dmodel] (rows ldx
    // apart) and the QKV projection's weights w_qkv [3 dmodel, dmodel] and
    // bias b_qkv [3 dmodel] (may be NULL); q, k and v are not read.
    const void* x;
    int64_t ldx;
    const void* w_qkv;
    const void* b_qkv;
    int dmodel;
    float proj_q_scale;   // set by the launcher: attn_q_scale(d), which the q columns leave multiplied by
};

// Softmax scale in log2 units: log2(e) / sqrt(head_dim).
inline float attn_q_scale(int head_dim) { return 1.4426950408889634f / sqrtf((float)head_dim); }

bool attention_supported(int head_dim);
int launch_attention(int dtype, AttnArgs a, hipStream_t s);

// A block's QKV projection and its self-attention in one launch, one
// workgroup per (sample, head) holding the head's Q, K and V in LDS: for bf16,
// up to 256 tokens per sample, head dims 32, 64 and 72, dmodel a multiple of
// 64 (= H d).  Writes only the attention output (a.o0, rows ldo apart): the
// same arithmetic, in the same order, as the QKV GEMM with single-group
// tiles followed by launch_attention.
bool qkv_attention_supported(int dtype, int T, int head_dim, int dmodel);
int launch_qkv_attention(int dtype, AttnArgs a, hipStream_t s);

}  // namespace bc
