// GEMM launcher interface shared by the block orchestration.
#pragma once

#include "hip_common.h"

namespace bc {

// Epilogue of y = A W^T.  Column c of row r gets v = acc + bias[c]; then
//   BIAS kind: v = q_scale * v if c < q_scale_to (attention queries written
//     pre-scaled); v = GELU(v) if c >= gelu_from; stored to out[r*ldo + c] (fp32
//     if out_f32, else the operand dtype) if c < split, else (operand dtype)
//     to out2[r*ldo2 + c - split + off2];
//   GATE_RES kind: v = res[r*ldr + c] + gate[(r / rows_per_gate)*ldg + c] * v
//     (gate NULL: a plain residual add),
//     stored to row (r / seg) * keep + r % seg of out (fp32 if out_f32, else
//     the operand dtype) when r % seg < keep, dropped otherwise.
struct GemmEpi {
    const void* bias;
    void* out;
    int64_t ldo;
    int out_f32;
    void* out2;
    int64_t ldo2;
    int split, off2, gelu_from;
    int q_scale_to;
    float q_scale;
    const float* res;
    int64_t ldr;
    const float* gate;
    int64_t ldg;
    int rows_per_gate;
    int seg, keep;
};

struct GemmArgs {
    const void* A;
    int64_t lda;
    const void* W;
    int64_t ldw;
    int M, N, K;
    GemmEpi e;
};

// Grouped weights: output columns [i*Nseg, (i+1)*Nseg) use W[i] ([Nseg, K],
// row stride ldw) and bias[i] (may be NULL).
constexpr int kMaxGemmSeg = 64;
struct GemmSeg {
    const void* W[kMaxGemmSeg];
    const void* bias[kMaxGemmSeg];
    int Nseg;
};

// Defaults: plain bias epilogue writing [M, N] densely to (unset) out.
GemmArgs gemm_args(const void* A, int64_t lda, const void* W, int64_t ldw, int M, int N, int K);
// epi: BC_EPI_BIAS (covers GELU via gelu_from) or BC_EPI_GATE_RES.
int launch_gemm(int dtype, int epi, const GemmArgs& g, hipStream_t s);
// Two GEMMs with the same epilogue kind in one launch when the second one's
// tiles fit the idle part of the first one's last round (the dual-stream
// blocks' text-stream projections beside the image-stream ones); otherwise
// two launches.
int launch_gemm_pair(int dtype, int epi, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s);
// Bias epilogue over nseg column segments (g.N is ignored; g.e.out / ldo
// describe the whole [M, nseg*Nseg] output).
int launch_gemm_grouped(int dtype, const GemmArgs& g, const GemmSeg& sg, int nseg, hipStream_t s);

}  // namespace bc
