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
};

// Softmax scale in log2 units: log2(e) / sqrt(head_dim).
inline float attn_q_scale(int head_dim) { return 1.4426950408889634f / sqrtf((float)head_dim); }

bool attention_supported(int head_dim);
int launch_attention(int dtype, AttnArgs a, hipStream_t s);

}  // namespace bc
