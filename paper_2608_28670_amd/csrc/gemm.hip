// Dense linear layers of the DiT block, y = epilogue(A W^T), on MFMA.
//
// A [M, K] and W [N, K] are both K-contiguous (the nn.Linear layout), so both
// operands stream into LDS the same way.  A workgroup of 4 waves owns a
// BM x BN output tile and walks K in steps of 128 bytes (64 bf16 / 32 fp32):
// global -> registers (prefetch of the next step) -> LDS (double buffered,
// rows padded by 16 bytes so the 16-byte fragment reads of 16 lanes hit 16
// distinct bank groups) -> MFMA operands.  Each wave computes a
// (BM/2) x (BN/2) sub-tile as a grid of 16x16 MFMA tiles:
//   bf16: v_mfma_f32_16x16x32_bf16, lane l holds row l%16, k = 8(l/16)..+8;
//   fp32: v_mfma_f32_16x16x4_f32,   lane l holds row l%16, k = l/16;
// and accumulates in fp32; lane l ends with rows 4(l/16)..+4 of column l%16.
// The epilogue applies the bias and then one of: nothing, GELU (tanh form),
// or the gated residual x + g * y of the adaLN blocks.
#include "gemm.h"

namespace bc {

template <typename T> struct Mma;
template <> struct Mma<bf16> {
    static constexpr int E = 8;    // operand elements per lane
    static constexpr int KI = 32;  // k per instruction
    typedef bf16x8 frag;
    __device__ static __forceinline__ f32x4 mma(const frag& a, const frag& b, const f32x4& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const bf16* p) {
        return __builtin_bit_cast(frag, *reinterpret_cast<const u32x4*>(p));
    }
};
template <> struct Mma<float> {
    static constexpr int E = 1;
    static constexpr int KI = 4;
    typedef float frag;
    __device__ static __forceinline__ f32x4 mma(frag a, frag b, const f32x4& c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const float* p) { return *p; }
};

constexpr int kGemmThreads = 256;

template <typename T, int EPI, int BM, int BN>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(GemmArgs g) {
    constexpr int EPC = 16 / (int)sizeof(T);        // elements per 16-byte chunk
    constexpr int BK = 8 * EPC;                      // 128 bytes of K per step
    constexpr int LDK = BK + EPC;                    // padded LDS row (elements)
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int CA = BM * 8 / kGemmThreads;        // 16-byte chunks per thread per step
    constexpr int CB = BN * 8 / kGemmThreads;
    typedef Mma<T> MM;

    __shared__ __attribute__((aligned(16))) T sA[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) T sB[2][BN][LDK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // Tile order: consecutive workgroup ids go round-robin to the 8 XCDs; give
    // each XCD a contiguous range of tiles, then raster in groups of 8 row
    // tiles so neighbouring workgroups share A rows and W rows in L2.
    const int tiles_m = (g.M + BM - 1) / BM;
    const int tiles_n = (g.N + BN - 1) / BN;
    const int nwg = gridDim.x;
    int pid = blockIdx.x;
    if ((nwg & 7) == 0) pid = (pid & 7) * (nwg >> 3) + (pid >> 3);
    constexpr int GROUP_M = 8;
    const int group = GROUP_M * tiles_n;
    const int first_m = (pid / group) * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int tm = first_m + (pid % group) % gm;
    const int tn = (pid % group) / gm;
    const int bm = tm * BM, bn = tn * BN;

    const T* __restrict__ A = static_cast<const T*>(g.A);
    const T* __restrict__ W = static_cast<const T*>(g.W);

    u32x4 ra[CA], rb[CB];
    auto load_global = [&](int k0) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + i * kGemmThreads;
            const int row = c >> 3, kc = k0 + (c & 7) * EPC;
            const int grow = bm + row;
            if (grow < g.M && kc < g.K)
                ra[i] = *reinterpret_cast<const u32x4*>(A + (int64_t)grow * g.lda + kc);
            else
                ra[i] = u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + i * kGemmThreads;
            const int row = c >> 3, kc = k0 + (c & 7) * EPC;
            const int grow = bn + row;
            if (grow < g.N && kc < g.K)
                rb[i] = *reinterpret_cast<const u32x4*>(W + (int64_t)grow * g.ldw + kc);
            else
                rb[i] = u32x4{0, 0, 0, 0};
        }
    };
    auto store_lds = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + i * kGemmThreads;
            *reinterpret_cast<u32x4*>(&sA[buf][c >> 3][(c & 7) * EPC]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + i * kGemmThreads;
            *reinterpret_cast<u32x4*>(&sB[buf][c >> 3][(c & 7) * EPC]) = rb[i];
        }
    };

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (g.K + BK - 1) / BK;
    load_global(0);
    store_lds(0);
    __syncthreads();

    const int frow = lane & 15;
    const int fk = (lane >> 4) * MM::E;
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) load_global((kt + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK / MM::KI; ++kk) {
            typename MM::frag af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) af[i] = MM::load(&sA[cur][wm * WM + i * 16 + frow][kk * MM::KI + fk]);
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[j] = MM::load(&sB[cur][wn * WN + j * 16 + frow][kk * MM::KI + fk]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = MM::mma(af[i], bfr[j], acc[i][j]);
        }
        if (kt + 1 < nk) store_lds(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue -----------------------------------------------------------
    const GemmEpi& e = g.e;
    const T* __restrict__ bias = static_cast<const T*>(e.bias);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = bn + wn * WN + j * 16 + (lane & 15);
        if (col >= g.N) continue;
        const float bv = bias ? ld(bias + col) : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = bm + wm * WM + i * 16 + 4 * (lane >> 4) + r;
                if (row >= g.M) continue;
                float v = acc[i][j][r] + bv;
                if constexpr (EPI == BC_EPI_GATE_RES) {
                    const float gv = e.gate ? e.gate[(int64_t)(row / e.rows_per_gate) * e.ldg + col] : 1.f;
                    v = e.res[(int64_t)row * e.ldr + col] + gv * v;
                    const int b = row / e.seg, s = row - b * e.seg;
                    if (s < e.keep) {
                        const int64_t o = (int64_t)(b * e.keep + s) * e.ldo + col;
                        if (e.out_f32) static_cast<float*>(e.out)[o] = v;
                        else st(static_cast<T*>(e.out) + o, v);
                    }
                } else {
                    if (col >= e.gelu_from) v = gelu_tanh(v);
                    if (col < e.split) st(static_cast<T*>(e.out) + (int64_t)row * e.ldo + col, v);
                    else st(static_cast<T*>(e.out2) + (int64_t)row * e.ldo2 + (col - e.split + e.off2), v);
                }
            }
        }
    }
}

template <typename T, int EPI>
static int run_gemm(const GemmArgs& g, hipStream_t s) {
    constexpr int BM = 128, BN = 128;
    const int64_t tiles = (int64_t)((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
    if (tiles > 0x7fffffff) return fail(BC_ERR_UNSUPPORTED, "GEMM grid too large");
    gemm_kernel<T, EPI, BM, BN><<<dim3((unsigned)tiles), dim3(kGemmThreads), 0, s>>>(g);
    return check_launch("gemm");
}

int launch_gemm(int dtype, int epi, const GemmArgs& g, hipStream_t s) {
    if (g.M <= 0 || g.N <= 0) return BC_OK;
    const int epc = dtype == BC_BF16 ? 8 : 4;
    if (g.K <= 0 || g.K % epc || g.lda % epc || g.ldw % epc)
        return fail(BC_ERR_UNSUPPORTED, "GEMM K=%d, lda=%lld, ldw=%lld must be multiples of %d", g.K,
                    (long long)g.lda, (long long)g.ldw, epc);
    if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.W)) % 16)
        return fail(BC_ERR_UNSUPPORTED, "GEMM operands must be 16-byte aligned");
    const int cls = epi == BC_EPI_GATE_RES ? PROF_GEMM_GATE : g.e.gelu_from < g.N ? PROF_GEMM_GELU : PROF_GEMM_BIAS;
    prof_begin(cls, s);
    int rc;
    if (dtype == BC_BF16) {
        rc = epi == BC_EPI_GATE_RES ? run_gemm<bf16, BC_EPI_GATE_RES>(g, s) : run_gemm<bf16, BC_EPI_BIAS>(g, s);
    } else {
        rc = epi == BC_EPI_GATE_RES ? run_gemm<float, BC_EPI_GATE_RES>(g, s) : run_gemm<float, BC_EPI_BIAS>(g, s);
    }
    prof_end(cls, s);
    return rc;
}

GemmArgs gemm_args(const void* A, int64_t lda, const void* W, int64_t ldw, int M, int N, int K) {
    GemmArgs g;
    g.A = A; g.lda = lda; g.W = W; g.ldw = ldw;
    g.M = M; g.N = N; g.K = K;
    GemmEpi& e = g.e;
    e.bias = nullptr;
    e.out = nullptr; e.ldo = N; e.out_f32 = 0;
    e.out2 = nullptr; e.ldo2 = 0; e.split = N; e.off2 = 0;
    e.gelu_from = N;
    e.res = nullptr; e.ldr = N;
    e.gate = nullptr; e.ldg = N; e.rows_per_gate = 1;
    e.seg = M > 0 ? M : 1; e.keep = e.seg;
    return g;
}

}  // namespace bc

using namespace bc;

extern "C" int bc_linear(int M, int N, int K, const void* A, const void* W, const void* bias, void* out,
                         int epilogue, const float* res, const float* gate, int rows_per_gate, int dtype,
                         void* stream) {
    clear_error();
    if (!A || !W || !out) return fail(BC_ERR_INVALID_ARG, "NULL operand");
    if (M < 0 || N < 1 || K < 1) return fail(BC_ERR_INVALID_ARG, "M=%d N=%d K=%d", M, N, K);
    if (dtype != BC_F32 && dtype != BC_BF16) return fail(BC_ERR_INVALID_ARG, "dtype %d", dtype);
    if (epilogue < BC_EPI_BIAS || epilogue > BC_EPI_GATE_RES) return fail(BC_ERR_INVALID_ARG, "epilogue %d", epilogue);
    GemmArgs g = gemm_args(A, K, W, K, M, N, K);
    g.e.bias = bias;
    g.e.out = out;
    if (epilogue == BC_EPI_BIAS_GELU) g.e.gelu_from = 0;
    if (epilogue == BC_EPI_GATE_RES) {
        if (!res || !gate || rows_per_gate < 1) return fail(BC_ERR_INVALID_ARG, "gated residual needs res, gate, rows_per_gate");
        g.e.res = res;
        g.e.gate = gate;
        g.e.rows_per_gate = rows_per_gate;
        g.e.out_f32 = 1;
    }
    return launch_gemm(dtype, epilogue == BC_EPI_GATE_RES ? BC_EPI_GATE_RES : BC_EPI_BIAS, g,
                       static_cast<hipStream_t>(stream));
}
