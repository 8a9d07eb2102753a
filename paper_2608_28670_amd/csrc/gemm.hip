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

// GELU, tanh form: 0.5 x (1 + tanh(y)), y = sqrt(2/pi) (x + 0.044715 x^3).
// Since 0.5 (1 + tanh(y)) = 1 / (1 + exp(-2 y)), this is x / (1 + 2^z) with
// z = -2 log2(e) y = x (A + B x^2): one native exp2 and one reciprocal per
// element (2^z overflows to +inf for very negative x, giving 0 as it should).
__device__ __forceinline__ float gelu_tanh(float x) {
    constexpr float A = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
    constexpr float B = A * 0.044715f;
    const float z = x * __builtin_fmaf(B, x * x, A);
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

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

// Bias + GELU / gated-residual epilogue for a wave's TM x TN block of 16x16
// accumulators whose top-left output element is (row0, col0).
template <typename T, int EPI, int TM, int TN>
__device__ __forceinline__ void epilogue(const GemmArgs& g, const f32x4 (&acc)[TM][TN], int row0, int col0, int lane) {
    const GemmEpi& e = g.e;
    const T* __restrict__ bias = static_cast<const T*>(e.bias);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int col = col0 + j * 16 + (lane & 15);
        if (col >= g.N) continue;
        const float bv = bias ? ld(bias + col) : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = row0 + i * 16 + 4 * (lane >> 4) + r;
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
                    if (col < e.q_scale_to) v *= e.q_scale;
                    if (col >= e.gelu_from) v = gelu_tanh(v);
                    if (col >= e.split) st(static_cast<T*>(e.out2) + (int64_t)row * e.ldo2 + (col - e.split + e.off2), v);
                    else if (e.out_f32) static_cast<float*>(e.out)[(int64_t)row * e.ldo + col] = v;
                    else st(static_cast<T*>(e.out) + (int64_t)row * e.ldo + col, v);
                }
            }
        }
    }
}

// Tile shape: BM x BN per workgroup, a WAVES_M x WAVES_N grid of waves, each
// wave owning a (BM/WAVES_M) x (BN/WAVES_N) block of 16x16 MFMA tiles.
template <typename T_, int EPI, int BM, int BN, int WAVES_M, int WAVES_N>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_kernel(GemmArgs g) {
    typedef elem_t<T_> T;
    constexpr int NT = 64 * WAVES_M * WAVES_N;       // threads
    constexpr int EPC = 16 / (int)sizeof(T);        // elements per 16-byte chunk
    constexpr int BK = 8 * EPC;                      // 128 bytes of K per step
    constexpr int LDK = BK + EPC;                    // padded LDS row (elements)
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int CA = BM * 8 / NT;                  // 16-byte chunks per thread per step
    constexpr int CB = BN * 8 / NT;
    static_assert(CA * NT == BM * 8 && CB * NT == BN * 8, "tile must split evenly over threads");
    typedef Mma<T> MM;

    __shared__ __attribute__((aligned(16))) T sA[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) T sB[2][BN][LDK];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    // Tile order: consecutive workgroup ids go round-robin to the 8 XCDs; give
    // each XCD a contiguous range of tiles, then raster in groups of 8 row
    // tiles so neighbouring workgroups share A rows and W rows in L2.
    const int tiles_m = (g.M + BM - 1) / BM;
    const int tiles_n = (g.N + BN - 1) / BN;
    const int nwg = gridDim.x;
    const int pid = xcd_contiguous(blockIdx.x, nwg);
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
            const int c = tid + i * NT;
            const int row = c >> 3, kc = k0 + (c & 7) * EPC;
            const int grow = bm + row;
            if (grow < g.M && kc < g.K)
                ra[i] = *reinterpret_cast<const u32x4*>(A + (int64_t)grow * g.lda + kc);
            else
                ra[i] = u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + i * NT;
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
            const int c = tid + i * NT;
            *reinterpret_cast<u32x4*>(&sA[buf][c >> 3][(c & 7) * EPC]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + i * NT;
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

    epilogue<T, EPI, TM, TN>(g, acc, bm + wm * WM, bn + wn * WN, lane);
}

// ---------------------------------------------------------------------------
// bf16 main loop with direct-to-LDS loads.
//
// Operand tiles go from HBM straight into LDS with global_load_lds_dwordx4:
// one wave-wide instruction moves 8 rows x 128 bytes (each lane 16 bytes,
// lane i landing at M0 + 16 i), so no registers or ds_write instructions are
// spent on staging.  LDS rows are 128 bytes (64 k) with no padding; to keep
// the 16-byte fragment reads of 16 consecutive rows conflict-free, the 16-byte
// chunk c of row r is stored in slot c ^ ((r >> 1) & 7), which the loading
// lane realises by choosing which global chunk it fetches.  STAGES k-steps are
// in flight: after the barrier of step kt the loads of step kt + STAGES - 1
// are issued into the buffer step kt - 1 used, and the wait before each
// barrier only drains the loads of the step about to be consumed.
// Requires K % 64 == 0 (whole k-steps); rows past M or N are clamped to the
// last row, so they load valid memory and only feed outputs never stored.
// ---------------------------------------------------------------------------
// LDS slot permutation of row r (see above); SW selects among candidate maps.
template <int SW> __device__ __forceinline__ int swz_of(int row) {
    if constexpr (SW == 0) return (row >> 1) & 7;
    else if constexpr (SW == 1) return row & 7;
    else return 0;
}
__device__ __forceinline__ int swz(int row) { return swz_of<0>(row); }

// One wave-wide direct-to-LDS load: each lane's 16 bytes at `src` land at
// lds_base + 16 * lane.  Issued as inline assembly so that the only waits on
// it are the explicit vmcnt waits of the pipeline (the compiler would
// otherwise drain every outstanding load before each LDS read and barrier).
__device__ __forceinline__ void dma16(const void* src, const void* lds_base) {
    const unsigned m0 = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)lds_base);   // wave-uniform
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(m0) : "memory", "m0");
}

template <int N> __device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, bool SEG, int SW = 0>
__device__ __forceinline__ void gemm_dma_body(GemmArgs g, const GemmSeg* sg) {
    typedef bf16 T;
    typedef Mma<bf16> MM;
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int BK = 64;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int OA = BM / 8 / NW, OB = BN / 8 / NW;     // row octets per wave per step
    constexpr int L = OA + OB;                             // loads per wave per step
    static_assert(OA * 8 * NW == BM && OB * 8 * NW == BN, "octets must split over waves");

    __shared__ __attribute__((aligned(1024))) T sA[STAGES][BM * BK];
    __shared__ __attribute__((aligned(1024))) T sB[STAGES][BN * BK];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;

    const int tiles_m = (g.M + BM - 1) / BM;
    const int tiles_n = (g.N + BN - 1) / BN;
    const int nwg = gridDim.x;
    const int pid = xcd_contiguous(blockIdx.x, nwg);
    constexpr int GROUP_M = 8;
    const int group = GROUP_M * tiles_n;
    const int first_m = (pid / group) * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int tm = first_m + (pid % group) % gm;
    const int tn = (pid % group) / gm;
    const int bm = tm * BM, bn = tn * BN;
    if constexpr (SEG) {
        // Grouped GEMM: column block bn lies in segment bn / Nseg, whose own
        // weight matrix [Nseg, K] and bias hold its rows.
        const int seg = bn / sg->Nseg;
        const int off = seg * sg->Nseg;
        g.W = static_cast<const bf16*>(sg->W[seg]) - (int64_t)off * g.ldw;
        g.e.bias = sg->bias[seg] ? static_cast<const bf16*>(sg->bias[seg]) - off : nullptr;
    }

    // Per-lane global source of each of this wave's octets (k offset added per step).
    const T* srcA[OA];
    const T* srcB[OB];
    const int lrow = lane >> 3, lslot = lane & 7;
#pragma unroll
    for (int o = 0; o < OA; ++o) {
        const int r = (wave * OA + o) * 8 + lrow;
        const int grow = min(bm + r, g.M - 1);
        srcA[o] = static_cast<const T*>(g.A) + (int64_t)grow * g.lda + ((lslot ^ swz_of<SW>(r)) * 8);
    }
#pragma unroll
    for (int o = 0; o < OB; ++o) {
        const int r = (wave * OB + o) * 8 + lrow;
        const int grow = min(bn + r, g.N - 1);
        srcB[o] = static_cast<const T*>(g.W) + (int64_t)grow * g.ldw + ((lslot ^ swz_of<SW>(r)) * 8);
    }
    auto issue = [&](int kt, int buf) {
        const int k0 = kt * BK;
#pragma unroll
        for (int o = 0; o < OA; ++o)
            dma16(srcA[o] + k0, &sA[buf][(wave * OA + o) * 8 * BK]);
#pragma unroll
        for (int o = 0; o < OB; ++o)
            dma16(srcB[o] + k0, &sB[buf][(wave * OB + o) * 8 * BK]);
    };

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = g.K / BK;
#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p)
        if (p < nk) issue(p, p);

    const int frow = lane & 15, grp = lane >> 4;
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + STAGES - 2 < nk) wait_vmcnt<(STAGES - 2) * L>();
        else wait_vmcnt<0>();
        __syncthreads();
        if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
        const T* a = sA[kt % STAGES];
        const T* b = sB[kt % STAGES];
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            const int c = kk * 4 + grp;
            MM::frag af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WM + i * 16 + frow;
                af[i] = MM::load(a + r * BK + ((c ^ swz_of<SW>(r)) * 8));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = wn * WN + j * 16 + frow;
                bfr[j] = MM::load(b + r * BK + ((c ^ swz_of<SW>(r)) * 8));
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = MM::mma(af[i], bfr[j], acc[i][j]);
        }
    }

    epilogue<T, EPI, TM, TN>(g, acc, bm + wm * WM, bn + wn * WN, lane);
}

// ---------------------------------------------------------------------------
// Wide-tile bf16 kernel for one-round grids.
//
// Same direct-to-LDS staging and swizzle as above, with three changes:
//  * tiles need not be powers of two (e.g. 256 x 288 or 128 x 432, so that
//    the DiT-XL/2 and PixArt block GEMMs split into exactly 256 tiles or a
//    whole number of rounds over the 256 CUs); the (BM + BN) / 8 row octets
//    of a k-step are dealt round-robin to the waves, which need not get equal
//    counts (the pipeline waits count each wave's own loads);
//  * a wave owns a 64 x 144 (or 64 x 128) block, halving the LDS bytes read
//    per MFMA flop relative to 32 x 64;
//  * the MFMA operands are swapped (W rows as the instruction's A), so lane l
//    accumulates out[row][col..col+3] with row = l % 16 and
//    col = 4 (l / 16): the epilogue reads and writes four consecutive
//    columns per lane with one vector access.
// Host-side conditions: K % 64 == 0; lda, ldw % 8 == 0; every epilogue
// column index, stride and boundary (N, split, gelu_from, off2, ldo, ldo2,
// ldr, ldg) a multiple of 4 and the epilogue pointers 16-byte aligned.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st4(bf16* p, const float (&v)[4]) {
    bf16x4 q;
    q[0] = (bf16)v[0]; q[1] = (bf16)v[1]; q[2] = (bf16)v[2]; q[3] = (bf16)v[3];
    *reinterpret_cast<bf16x4*>(p) = q;
}
__device__ __forceinline__ void st4(float* p, const float (&v)[4]) {
    *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
}

// Residual of the gated-residual epilogue, loaded into registers at the start
// of the last k-step so that its latency hides behind the MFMAs, when a wave's
// share is small enough to sit beside the accumulators (at most 12 MFMA tiles);
// larger tiles read it in the epilogue.  The gate (one row per sample) is read
// in the epilogue from cache.
template <int EPI, int TM, int TN> struct EpiPrefetch {
    static constexpr bool early = EPI == BC_EPI_GATE_RES && TM * TN <= 12;
    f32x4 res[early ? TM : 1][early ? TN : 1];
    __device__ __forceinline__ void load(const GemmArgs& g, int row0, int col0, int lane, int jn) {
        if constexpr (early) {
            const GemmEpi& e = g.e;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int row = min(row0 + i * 16 + (lane & 15), g.M - 1);
                const float* rrow = e.res + (int64_t)row * e.ldr;
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if (j >= jn) break;
                    const int col = min(col0 + j * 16 + 4 * (lane >> 4), g.N - 4);
                    res[i][j] = *reinterpret_cast<const f32x4*>(rrow + col);
                }
            }
        }
    }
    __device__ __forceinline__ f32x4 get(const GemmArgs& g, int i, int j, int row, int col) const {
        if constexpr (early) return res[i][j];
        else return *reinterpret_cast<const f32x4*>(g.e.res + (int64_t)row * g.e.ldr + col);
    }
};

// Epilogue straight from the accumulators (gated residual; fp32 outputs of
// the plain epilogue).  jn: number of the TN column blocks this wave holds.

template <int EPI, int TM, int TN>
__device__ __forceinline__ void epilogue_t(const GemmArgs& g, const f32x4 (&acc)[TM][TN], int row0, int col0, int lane,
                                           int jn, const EpiPrefetch<EPI, TM, TN>& pf) {
    const GemmEpi& e = g.e;
    if constexpr (EPI == BC_EPI_GATE_RES) {
        // Rows outer: the row's destination (ring-slot remap) is worked out once.
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = row0 + i * 16 + (lane & 15);
            if (row >= g.M) continue;
            const int b = row / e.seg, sidx = row - b * e.seg;
            if (sidx >= e.keep) continue;
            const int64_t orow = (int64_t)(b * e.keep + sidx) * e.ldo;
            const float* grow = e.gate ? e.gate + (int64_t)(row / e.rows_per_gate) * e.ldg : nullptr;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                if (j >= jn) break;
                const int col = col0 + j * 16 + 4 * (lane >> 4);
                if (col >= g.N) continue;
                float v[4];
                const bf16* __restrict__ bias = static_cast<const bf16*>(e.bias);
                float bv[4] = {0.f, 0.f, 0.f, 0.f};
                if (bias) {
                    const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + col);
#pragma unroll
                    for (int r = 0; r < 4; ++r) bv[r] = (float)b4[r];
                }
                const f32x4 gv = grow ? *reinterpret_cast<const f32x4*>(grow + col) : f32x4{1.f, 1.f, 1.f, 1.f};
                const f32x4 rv = pf.get(g, i, j, row, col);
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = rv[r] + gv[r] * (acc[i][j][r] + bv[r]);
                if (e.out_f32) st4(static_cast<float*>(e.out) + orow + col, v);
                else st4(static_cast<bf16*>(e.out) + orow + col, v);
            }
        }
        return;
    }
    const bf16* __restrict__ bias = static_cast<const bf16*>(e.bias);
    const bool odd = (lane >> 4) & 1;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        if (j >= jn) break;
        const int col = col0 + j * 16 + 4 * (lane >> 4);
        const bool col_ok = col < g.N;
        float bv[4] = {0.f, 0.f, 0.f, 0.f};
        if (bias && col_ok) {
            const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + col);
#pragma unroll
            for (int r = 0; r < 4; ++r) bv[r] = (float)b4[r];
        }
        if (!col_ok) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = row0 + i * 16 + (lane & 15);
            if (row >= g.M) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = acc[i][j][r] + bv[r];
            if (col < e.q_scale_to) {
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] *= e.q_scale;
            }
            if (col >= e.gelu_from) {
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = gelu_tanh(v[r]);
            }
            if (col >= e.split) st4(static_cast<bf16*>(e.out2) + (int64_t)row * e.ldo2 + (col - e.split + e.off2), v);
            else if (e.out_f32) st4(static_cast<float*>(e.out) + (int64_t)row * e.ldo + col, v);
            else st4(static_cast<bf16*>(e.out) + (int64_t)row * e.ldo + col, v);
        }
    }
}

// LDS slot of 16-byte chunk c in row r for k-steps of BK = 64 (128-byte rows,
// 8 chunks) or BK = 32 (64-byte rows, 4 chunks): the 16 rows read by one
// fragment load fall on 16 distinct 16-byte bank groups.
template <int BK> __device__ __forceinline__ int wslot(int c, int r) {
    if constexpr (BK == 64) return c ^ ((r >> 1) & 7);
    else return c ^ ((r >> 2) & 3);
}

// KG > 1: split K inside the workgroup.  KG groups of WAVES_M x WAVES_N waves
// share the tile; a stage holds KG consecutive 64-wide k-blocks (one per
// group, each laid out as above), so every wave keeps a full accumulator over
// 1/KG of K.  The groups' partial tiles are then summed through LDS and group
// 0 applies the epilogue.  (For small outputs: 128 x 144 tiles of 2 x 2 waves
// of 64 x 80 / 64 x 64 in two groups keep eight waves per CU with large wave
// tiles where a one-round grid has only 256 tiles.)
// Wait until at most `later` groups of Q direct-to-LDS loads (issued after the
// group waited for) are outstanding; `later` >= LMAX waits for all.
template <int Q, int L = 0, int LMAX = 3> __device__ __forceinline__ void wait_groups(int later) {
    if constexpr (L >= LMAX) {
        wait_vmcnt<0>();
    } else {
        if (later <= L) {
            wait_vmcnt<L * Q>();
            return;
        }
        wait_groups<Q, L + 1, LMAX>(later);
    }
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int BK, int KG, int PIPE>
__device__ __forceinline__ void gemm_wide_body(GemmArgs g, int tile) {
    typedef bf16 T;
    typedef Mma<bf16> MM;
    constexpr int NWG = WAVES_M * WAVES_N;                // waves per K group
    constexpr int NW = NWG * KG;
    static_assert(BK == 64 || BK == 32, "k-step");
    static_assert(KG == 1 || KG == 2, "K groups");
    constexpr int CPR = BK / 8;                            // 16-byte chunks per LDS row
    constexpr int RPI = 64 / CPR;                          // rows per wave-wide load
    constexpr int WM = BM / WAVES_M, TM = WM / 16;
    // The BN / 16 column blocks are dealt to the WAVES_N wave columns as
    // evenly as possible (144 = 80 + 64 for two): TN is the larger share.
    constexpr int NBLK = BN / 16, TN = (NBLK + WAVES_N - 1) / WAVES_N, NREM = NBLK % WAVES_N;
    constexpr int GOCT = (BM + BN) / RPI;                  // wave-wide loads per group block
    constexpr int NOCT = GOCT * KG;                        // wave-wide loads per stage
    constexpr int QMAX = (NOCT + NW - 1) / NW;             // octets per wave (at most)
    static_assert(TM * 16 * WAVES_M == BM && BM % 16 == 0 && BN % 16 == 0, "tile shape");
    constexpr int GBLK = (BM + BN) * BK;                   // elements per group block: BM rows of A, then BN rows of W
    constexpr int STAGE = GBLK * KG;
    constexpr int OPITCH = BN + 8;                         // staged bf16 output row (16-byte pad)
    constexpr int SMEM0 = STAGES * STAGE > BM * OPITCH ? STAGES * STAGE : BM * OPITCH;
    // Gated epilogue through LDS (small tiles): an fp32 row-major copy of the
    // tile, FPITCH floats per row.
    constexpr int FPITCH = BN + 4;
    constexpr bool STAGE_GATED = EPI == BC_EPI_GATE_RES && BM * FPITCH * 4 <= 96 * 1024;
    constexpr int RED = STAGE_GATED ? BM * FPITCH * 2 : KG > 1 ? NWG * TM * TN * 64 * 4 * 2 : 0;   // in bf16 units
    constexpr int SMEM = SMEM0 > RED ? SMEM0 : RED;
    __shared__ __attribute__((aligned(1024))) T sm[SMEM];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kg = wave / NWG, wig = wave % NWG;
    const int wm = wig / WAVES_N, wn = wig % WAVES_N;
    const int jn = NREM == 0 ? TN : NBLK / WAVES_N + (wn < NREM ? 1 : 0);    // this wave's column blocks
    const int j0 = NREM == 0 ? wn * TN : wn * (NBLK / WAVES_N) + min(wn, NREM);

    const int tiles_m = (g.M + BM - 1) / BM;
    const int tiles_n = (g.N + BN - 1) / BN;
    constexpr int GROUP_M = 8;
    const int group = GROUP_M * tiles_n;
    const int first_m = (tile / group) * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int tm = first_m + (tile % group) % gm;
    const int tn = (tile % group) / gm;
    const int bm = tm * BM, bn = tn * BN;

    // Load o = wave + NW q of a stage fills rows RPI (o % GOCT) .. + RPI - 1 of
    // group block o / GOCT (A rows first, then W rows); lane L loads row
    // RPI (o % GOCT) + L / CPR into slot L % CPR, fetching the global chunk
    // that the swizzle puts there.
    const T* src[QMAX];
    const int lrow = lane / CPR, lslot = lane % CPR;
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
        const int o = min(wave + NW * q, NOCT - 1);
        const int og = o / GOCT, r = RPI * (o % GOCT) + lrow;
        const T* p;
        if (r < BM) p = static_cast<const T*>(g.A) + (int64_t)min(bm + r, g.M - 1) * g.lda;
        else p = static_cast<const T*>(g.W) + (int64_t)min(bn + r - BM, g.N - 1) * g.ldw;
        src[q] = p + og * BK + wslot<BK>(lslot, r) * 8;
    }
    const int nk = g.K / (BK * KG);                        // stages
    auto issue = [&](int kt, int buf) {
        const int k0 = kt * BK * KG;
#pragma unroll
        for (int q = 0; q < QMAX; ++q) {
            const int o = wave + NW * q;
            if (NOCT % NW == 0 || o < NOCT) dma16(src[q] + k0, &sm[buf * STAGE + (o / GOCT) * GBLK + (o % GOCT) * RPI * BK]);
        }
    };

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    EpiPrefetch<EPI, TM, TN> pf;
#pragma unroll
    for (int p = 0; p < STAGES - 1; ++p)
        if (p < nk) issue(p, p);
    // Loads this wave issues per k-step (waves below NOCT % NW get one more).
    const bool more = NOCT % NW == 0 || wave < NOCT % NW;
    const int frow = lane & 15, grp = lane >> 4;
    if constexpr (PIPE) {
        // Software-pipelined k loop: the barrier sits between the two 32-wide
        // halves of a k-step, so the fragments of the next step's first half
        // are read from LDS while this step's second-half MFMAs run, and the
        // second half's fragments while the first half's run.  Stage kt's
        // buffer is last read before the middle barrier of step kt, so the
        // loads of step kt + STAGES - 1 may overwrite it at the top of kt + 1.
        static_assert(KG == 1 && BK == 64 && STAGES >= 3 && STAGES <= 5, "pipelined k loop");
        // Fragments live across the loop as 32-bit words (a bf16 vector
        // carried around the loop is split into halves and re-packed with
        // byte permutes, which makes the MFMAs wait on the next reads).
        u32x4 fa[2][TM], fb[2][TN];
        auto read = [&](int kt, int kk, u32x4 (&a)[TM], u32x4 (&b)[TN]) {
            const T* st = sm + (kt % STAGES) * STAGE;
            const int c = kk * 4 + grp;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WM + i * 16 + frow;
                a[i] = *reinterpret_cast<const u32x4*>(st + r * BK + wslot<BK>(c, r) * 8);
            }
            // Waves with the smaller column share read their last block twice
            // rather than leaving a fragment conditionally unset.
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int r = BM + (j0 + (NREM != 0 && j >= jn ? jn - 1 : j)) * 16 + frow;
                b[j] = *reinterpret_cast<const u32x4*>(st + r * BK + wslot<BK>(c, r) * 8);
            }
        };
        // Unconditional: the accumulators past a wave's share (j >= jn) take
        // the duplicated block and are never stored; branch-free issue.
        auto mma = [&](const u32x4 (&a)[TM], const u32x4 (&b)[TN]) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = MM::mma(__builtin_bit_cast(MM::frag, b[j]), __builtin_bit_cast(MM::frag, a[i]), acc[i][j]);
        };
        // Stage j's loads are done once at most (loads issued after them) are
        // outstanding: min(STAGES - 2, nk - 1 - j) groups of QMAX (or QMAX - 1).
        auto wait_stage = [&](int j) {
            const int later = min(STAGES - 2, nk - 1 - j);
            if (more) wait_groups<QMAX, 0, STAGES - 1>(later);
            else wait_groups<QMAX - 1, 0, STAGES - 1>(later);
        };
        wait_stage(0);
        __syncthreads();
        read(0, 0, fa[0], fb[0]);
        // All but the last step; the last one (no next stage) is peeled so
        // that no control-flow merge sits between a step's second-half reads
        // and its MFMAs (the merged wait counts would make them wait).
        // In each half the fragment reads are issued first, ahead of the
        // MFMAs on the other buffer, so their latency hides behind them.
        for (int kt = 0; kt + 1 < nk; ++kt) {
            if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
            __builtin_amdgcn_sched_barrier(0);
            read(kt, 1, fa[1], fb[1]);
            mma(fa[0], fb[0]);
            __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);   // DS reads
            __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);   // MFMAs
            wait_stage(kt + 1);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
            read(kt + 1, 0, fa[0], fb[0]);
            mma(fa[1], fb[1]);
            __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);
        }
        if (EPI == BC_EPI_GATE_RES && !STAGE_GATED) pf.load(g, bm + wm * WM, bn + j0 * 16, lane, jn);
        read(nk - 1, 1, fa[1], fb[1]);
        mma(fa[0], fb[0]);
        mma(fa[1], fb[1]);
    } else
    for (int kt = 0; kt < nk; ++kt) {
        if (STAGES > 2 && kt + STAGES - 2 < nk) {
            if (more) wait_vmcnt<(STAGES - 2) * QMAX>();
            else wait_vmcnt<(STAGES - 2) * (QMAX - 1)>();
        } else {
            wait_vmcnt<0>();
        }
        __syncthreads();
        if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
        if (EPI == BC_EPI_GATE_RES && !STAGE_GATED && kg == 0 && kt == nk - 1) pf.load(g, bm + wm * WM, bn + j0 * 16, lane, jn);
        const T* st = sm + (kt % STAGES) * STAGE + kg * GBLK;
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            const int c = kk * 4 + grp;
            MM::frag af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int r = wm * WM + i * 16 + frow;
                af[i] = MM::load(st + r * BK + wslot<BK>(c, r) * 8);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                if (NREM != 0 && j >= jn) break;
                const int r = BM + (j0 + j) * 16 + frow;
                bfr[j] = MM::load(st + r * BK + wslot<BK>(c, r) * 8);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    if (NREM == 0 || j < jn) acc[i][j] = MM::mma(bfr[j], af[i], acc[i][j]);
        }
    }

    if constexpr (STAGE_GATED) {
        // The tile goes through LDS as fp32 rows (group 1's partial first, then
        // group 0 adds its own: a fixed order), and all waves then apply the
        // gated residual to whole rows, reading the residual and gate and
        // writing the stream as consecutive 16-byte chunks.
        const GemmEpi& e = g.e;
        float* ft = reinterpret_cast<float*>(sm);
        __syncthreads();   // every wave is done with the stage buffers
        for (int pass = KG - 1; pass >= 0; --pass) {
            if (kg == pass) {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if (j >= jn) break;
                    const int lc = (j0 + j) * 16 + 4 * (lane >> 4);
#pragma unroll
                    for (int i = 0; i < TM; ++i) {
                        f32x4* dst = reinterpret_cast<f32x4*>(ft + (wm * WM + i * 16 + (lane & 15)) * FPITCH + lc);
                        *dst = pass == KG - 1 ? acc[i][j] : *dst + acc[i][j];
                    }
                }
            }
            __syncthreads();
        }
        const bf16* __restrict__ bias = static_cast<const bf16*>(e.bias);
        constexpr int NT = 64 * NW, C4 = BN / 4;              // threads; 4-column chunks per tile row
        for (int q = tid; q < BM * C4; q += NT) {
            const int lr = q / C4, c4 = q - lr * C4;
            const int row = bm + lr, col = bn + c4 * 4;
            if (row >= g.M || col >= g.N) continue;
            const int b = row / e.seg, sidx = row - b * e.seg;
            if (sidx >= e.keep) continue;
            const f32x4 y = *reinterpret_cast<const f32x4*>(ft + lr * FPITCH + c4 * 4);
            const f32x4 rv = *reinterpret_cast<const f32x4*>(e.res + (int64_t)row * e.ldr + col);
            const f32x4 gv = e.gate ? *reinterpret_cast<const f32x4*>(e.gate + (int64_t)(row / e.rows_per_gate) * e.ldg + col)
                                    : f32x4{1.f, 1.f, 1.f, 1.f};
            float bv[4] = {0.f, 0.f, 0.f, 0.f};
            if (bias) {
                const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + col);
#pragma unroll
                for (int r = 0; r < 4; ++r) bv[r] = (float)b4[r];
            }
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = rv[r] + gv[r] * (y[r] + bv[r]);
            const int64_t o = (int64_t)(b * e.keep + sidx) * e.ldo + col;
            if (e.out_f32) st4(static_cast<float*>(e.out) + o, v);
            else st4(static_cast<bf16*>(e.out) + o, v);
        }
        return;
    }
    if constexpr (KG == 2) {
        // Group 1 hands its partial tile to group 0 through LDS.
        __syncthreads();   // every wave is done with the stage buffers
        f32x4* red = reinterpret_cast<f32x4*>(sm) + wig * TM * TN * 64 + lane;
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) red[(i * TN + j) * 64] = acc[i][j];
        }
        __syncthreads();
        if (kg == 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] += red[(i * TN + j) * 64];
        }
    }
    if constexpr (EPI == BC_EPI_BIAS) {
        if (!g.e.out_f32) {
            // bf16 outputs leave through LDS: the waves write their finished
            // values into a row-major copy of the tile, then the workgroup stores
            // it as consecutive 16-byte chunks of each row, so every store
            // instruction covers whole cache lines.  (Written straight from the
            // accumulators, 32-byte pieces of lines from all 256 one-round tiles
            // at once came back as about 1.5x the output bytes in HBM writes.)
            const GemmEpi& e = g.e;
            const bf16* __restrict__ bias = static_cast<const bf16*>(e.bias);
            __syncthreads();   // every wave is done with the stage buffers (and the reduction)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                if (j >= jn || kg != 0) break;
                const int lc = (j0 + j) * 16 + 4 * (lane >> 4);
                const int col = bn + lc;
                float bv[4] = {0.f, 0.f, 0.f, 0.f};
                if (bias && col < g.N) {
                    const bf16x4 b4 = *reinterpret_cast<const bf16x4*>(bias + col);
#pragma unroll
                    for (int r = 0; r < 4; ++r) bv[r] = (float)b4[r];
                }
                const bool act = col >= e.gelu_from;
                const float qs = col < e.q_scale_to ? e.q_scale : 1.f;
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    bf16x4 q;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float v = (acc[i][j][r] + bv[r]) * qs;
                        if (act) v = gelu_tanh(v);
                        q[r] = (bf16)v;
                    }
                    const int lr = wm * WM + i * 16 + (lane & 15);
                    *reinterpret_cast<bf16x4*>(sm + lr * OPITCH + lc) = q;
                }
            }
            __syncthreads();
            constexpr int NT = 64 * NW, CPRO = BN / 8;    // threads; 16-byte chunks per tile row
            for (int q = tid; q < BM * CPRO; q += NT) {
                const int lr = q / CPRO, c8 = q - lr * CPRO;
                const int row = bm + lr, col = bn + c8 * 8;
                if (row >= g.M || col >= g.N) continue;
                const u32x4 val = *reinterpret_cast<const u32x4*>(sm + lr * OPITCH + c8 * 8);
                bf16* dst = col >= e.split ? static_cast<bf16*>(e.out2) + (int64_t)row * e.ldo2 + (col - e.split + e.off2)
                                           : static_cast<bf16*>(e.out) + (int64_t)row * e.ldo + col;
                *reinterpret_cast<u32x4*>(dst) = val;
            }
            return;
        }
    }
    if (kg != 0) return;
    epilogue_t<EPI, TM, TN>(g, acc, bm + wm * WM, bn + j0 * 16, lane, jn, pf);
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int BK, int KG, int PIPE = 0>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N * KG) void gemm_wide_kernel(GemmArgs g) {
    gemm_wide_body<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, BK, KG, PIPE>(g, xcd_contiguous(blockIdx.x, gridDim.x));
}

// Two GEMMs in one grid: workgroups [0, tiles0) take the first (in the
// XCD-contiguous order over its own tiles), the rest the second, whose
// workgroups come last and are dealt round-robin to the XCDs, so its tiles
// fill the first one's last round.
template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int BK, int KG, int PIPE = 0>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N * KG) void gemm_wide_pair_kernel(GemmArgs g0, GemmArgs g1,
                                                                                     int tiles0) {
    const int b = blockIdx.x;
    const bool second = b >= tiles0;
    gemm_wide_body<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, BK, KG, PIPE>(second ? g1 : g0,
                                                                        second ? b - tiles0 : xcd_contiguous(b, tiles0));
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES = 2, int BK = 64, int KG = 1, int PIPE = 0>
static void launch_wide(const GemmArgs& g, hipStream_t s) {
    const unsigned tiles = (unsigned)(((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN));
    launch_k(gemm_wide_kernel<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, BK, KG, PIPE>, dim3(tiles),
             dim3(64 * WAVES_M * WAVES_N * KG), s, g);
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int SW = 0>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_dma_kernel(GemmArgs g) {
    gemm_dma_body<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, false, SW>(g, nullptr);
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_dma_seg_kernel(GemmArgs g, GemmSeg sg) {
    gemm_dma_body<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, true>(g, &sg);
}

template <int EPI, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int SW = 0>
static void launch_dma(const GemmArgs& g, hipStream_t s) {
    const unsigned tiles = (unsigned)(((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN));
    launch_k(gemm_dma_kernel<EPI, BM, BN, WAVES_M, WAVES_N, STAGES, SW>, dim3(tiles), dim3(64 * WAVES_M * WAVES_N), s, g);
}

template <typename T, int EPI, int BM, int BN, int WAVES_M, int WAVES_N>
static void launch_tile(const GemmArgs& g, hipStream_t s) {
    const unsigned tiles = (unsigned)(((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN));
    launch_k(gemm_kernel<tag_t<T>, EPI, BM, BN, WAVES_M, WAVES_N>, dim3(tiles), dim3(64 * WAVES_M * WAVES_N), s, g);
}

// The wide kernel's vector epilogue needs every column index and stride it
// touches to be a multiple of 4 and its pointers 16-byte aligned.
static bool wide_ok(const GemmArgs& g, int epi) {
    const GemmEpi& e = g.e;
    auto al = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    if (g.K % 64 || g.lda % 8 || g.ldw % 8 || g.N % 4 || e.ldo % 4 || !al(e.out)) return false;
    if (e.bias && reinterpret_cast<uintptr_t>(e.bias) % 8) return false;
    if (epi == BC_EPI_GATE_RES) return e.ldr % 4 == 0 && al(e.res) && (!e.gate || (e.ldg % 4 == 0 && al(e.gate)));
    // The plain epilogue pairs lanes into 8-column groups: N, the split and
    // GELU boundaries and the bf16 row strides and offsets are multiples of 8.
    if (g.N % 8 || e.ldo % 8) return false;
    if (e.gelu_from < g.N && e.gelu_from % 8) return false;
    if (e.q_scale_to > 0 && e.q_scale_to % 8) return false;
    if (e.split < g.N && (e.split % 8 || e.off2 % 8 || e.ldo2 % 8 || !al(e.out2))) return false;
    return true;
}

// Tile choice (measured on MI355X over the DiT-XL/2, PixArt and HunyuanVideo
// block shapes, see the design notes), for bf16 operands with whole 64-wide
// k-steps and an epilogue the wide kernel can vectorise:
//   * at least one full round of 256 x 288 tiles over the 256 CUs: 256 x 288
//     (8 waves of 64 x 144), or 256 x 256 when N is a multiple of 256 but not
//     of 288 (no ragged column tile);
//   * N a multiple of 432 with at least one round of 128 x 432 tiles (the
//     DiT-XL/2 QKV projection: exactly 256): 2 x 4 waves of 64 x 112 / 64 x 96;
//   * at most 256 tiles of 128 x 144 (the N = 1152 projections at M = 4096):
//     2 x 4 waves of 64 x 48 / 64 x 32 with four stages in flight (in the
//     model their weights come cold from HBM every block: 4 stages ran the
//     DiT-XL/2 sampler 7 % faster than 2) and the gated epilogue staged
//     through LDS; for the plain epilogue with K % 128 == 0, K split over two
//     groups of 2 x 2 waves (64 x 80 / 64 x 64) instead;
//   * otherwise 128 x 128 (8 waves of 32 x 64, two workgroups per CU).
// Other bf16 operands take the direct-to-LDS kernel with the scalar
// epilogue, or the register-staged kernel; fp32 the register-staged kernel.
template <typename T, int EPI>
static int run_gemm(const GemmArgs& g, hipStream_t s) {
    const int64_t tiles128 = (int64_t)((g.M + 127) / 128) * ((g.N + 127) / 128);
    if (tiles128 > 0x7fffffff) return fail(BC_ERR_UNSUPPORTED, "GEMM grid too large");
    if constexpr (sizeof(T) == 2) {
        const int64_t tiles288 = (int64_t)((g.M + 255) / 256) * ((g.N + 287) / 288);
        const int64_t tiles144 = (int64_t)((g.M + 127) / 128) * ((g.N + 143) / 144);
        const bool dma = g.K % 64 == 0 && g.lda % 8 == 0 && g.ldw % 8 == 0;
        if (dma && wide_ok(g, EPI)) {
            if (tiles288 >= 256) {
                if (g.N % 288 != 0 && g.N % 256 == 0) launch_wide<EPI, 256, 256, 4, 4>(g, s);
                else launch_wide<EPI, 256, 288, 4, 3>(g, s);
            } else if (g.N % 432 == 0 && (int64_t)((g.M + 127) / 128) * (g.N / 432) >= 256) {
                launch_wide<EPI, 128, 432, 4, 3>(g, s);
            } else if (tiles144 <= 256) {
                if (EPI == BC_EPI_BIAS && g.K % 128 == 0) launch_wide<EPI, 128, 144, 2, 2, 2, 64, 2>(g, s);
                else launch_wide<EPI, 128, 144, 4, 4, 4, 64, 1, 1>(g, s);
            } else {
                launch_wide<EPI, 128, 128, 4, 4>(g, s);
            }
        } else if (dma) {
            launch_dma<EPI, 128, 128, 4, 2, 2>(g, s);
        } else {
            launch_tile<T, EPI, 128, 128, 4, 2>(g, s);
        }
    } else {
        launch_tile<T, EPI, 128, 128, 2, 2>(g, s);
    }
    return check_launch("gemm");
}

int launch_gemm_grouped(int dtype, const GemmArgs& g0, const GemmSeg& sg, int nseg, hipStream_t s) {
    // Column segment i of the output uses weights sg.W[i] ([Nseg, K]) and bias sg.bias[i].
    if (g0.M <= 0 || nseg <= 0) return BC_OK;
    if (nseg > kMaxGemmSeg) return fail(BC_ERR_UNSUPPORTED, "%d GEMM segments", nseg);
    GemmArgs g = g0;
    g.N = nseg * sg.Nseg;
    const bool dma = dtype == BC_BF16 && g.K % 64 == 0 && g.ldw % 8 == 0 && g.lda % 8 == 0 && sg.Nseg % 128 == 0 &&
                     reinterpret_cast<uintptr_t>(g.A) % 16 == 0;
    if (dma) {
        for (int i = 0; i < nseg; ++i)
            if (reinterpret_cast<uintptr_t>(sg.W[i]) % 16) return fail(BC_ERR_UNSUPPORTED, "misaligned segment weight");
        prof_begin(PROF_GEMM_BIAS, s, 2.0 * g.M * (double)g.N * g.K);
        const unsigned tiles = (unsigned)(((g.M + 127) / 128) * (g.N / 128));
        launch_k(gemm_dma_seg_kernel<BC_EPI_BIAS, 128, 128, 4, 2, 2>, dim3(tiles), dim3(512), s, g, sg);
        prof_end(PROF_GEMM_BIAS, s);
        return check_launch("grouped gemm");
    }
    // One launch per segment, writing its column block of the output.
    for (int i = 0; i < nseg; ++i) {
        GemmArgs gi = g0;
        gi.N = sg.Nseg;
        gi.W = sg.W[i];
        gi.e.bias = sg.bias[i];
        gi.e.out = static_cast<char*>(g0.e.out) + (size_t)i * sg.Nseg * (g0.e.out_f32 ? 4 : dtype_size(dtype));
        const int rc = launch_gemm(dtype, BC_EPI_BIAS, gi, s);
        if (rc != BC_OK) return rc;
    }
    return BC_OK;
}

int launch_gemm(int dtype, int epi, const GemmArgs& g, hipStream_t s) {
    if (g.M <= 0 || g.N <= 0) return BC_OK;
    const int epc = dtype == BC_BF16 ? 8 : 4;
    if (g.K <= 0 || g.K % epc || g.lda % epc || g.ldw % epc)
        return fail(BC_ERR_UNSUPPORTED, "GEMM K=%d, lda=%lld, ldw=%lld must be multiples of %d", g.K,
                    (long long)g.lda, (long long)g.ldw, epc);
    if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.W)) % 16)
        return fail(BC_ERR_UNSUPPORTED, "GEMM operands must be 16-byte aligned");
    const int cls = epi == BC_EPI_GATE_RES ? (g.K > g.N ? PROF_GEMM_DOWN : PROF_GEMM_GATE)
                    : g.e.gelu_from < g.N ? PROF_GEMM_GELU : PROF_GEMM_BIAS;
    prof_begin(cls, s, 2.0 * g.M * (double)g.N * g.K);
    int rc;
    if (dtype == BC_BF16) {
        rc = epi == BC_EPI_GATE_RES ? run_gemm<bf16, BC_EPI_GATE_RES>(g, s) : run_gemm<bf16, BC_EPI_BIAS>(g, s);
    } else {
        rc = epi == BC_EPI_GATE_RES ? run_gemm<float, BC_EPI_GATE_RES>(g, s) : run_gemm<float, BC_EPI_BIAS>(g, s);
    }
    prof_end(cls, s);
    return rc;
}

// The first GEMM's tile choice must be 256 x 256 (as run_gemm picks it) and
// the second one's tiles must fit the idle part of the first one's last
// round; otherwise two launches.
int launch_gemm_pair(int dtype, int epi, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s) {
    if (g1.M <= 0 || g1.N <= 0) return launch_gemm(dtype, epi, g0, s);
    if (g0.M <= 0 || g0.N <= 0) return launch_gemm(dtype, epi, g1, s);
    auto wide = [&](const GemmArgs& g) {
        return dtype == BC_BF16 && g.K > 0 && g.K % 64 == 0 && g.lda % 8 == 0 && g.ldw % 8 == 0 &&
               (reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.W)) % 16 == 0 && wide_ok(g, epi);
    };
    const int64_t t0 = (int64_t)((g0.M + 255) / 256) * ((g0.N + 255) / 256);
    const int64_t t1 = (int64_t)((g1.M + 255) / 256) * ((g1.N + 255) / 256);
    const int64_t t288 = (int64_t)((g0.M + 255) / 256) * ((g0.N + 287) / 288);
    const int64_t idle = (t0 + 255) / 256 * 256 - t0;
    const bool big = t288 >= 256 && g0.N % 288 != 0 && g0.N % 256 == 0;
    if (!(wide(g0) && wide(g1) && big && t1 <= idle && t0 + t1 <= 0x7fffffff)) {
        const int rc = launch_gemm(dtype, epi, g0, s);
        return rc != BC_OK ? rc : launch_gemm(dtype, epi, g1, s);
    }
    const int cls = epi == BC_EPI_GATE_RES ? (g0.K > g0.N ? PROF_GEMM_DOWN : PROF_GEMM_GATE)
                    : g0.e.gelu_from < g0.N ? PROF_GEMM_GELU : PROF_GEMM_BIAS;
    prof_begin(cls, s, 2.0 * g0.M * (double)g0.N * g0.K + 2.0 * g1.M * (double)g1.N * g1.K);
    const dim3 grid((unsigned)(t0 + t1)), block(1024);
    if (epi == BC_EPI_GATE_RES)
        launch_k(gemm_wide_pair_kernel<BC_EPI_GATE_RES, 256, 256, 4, 4, 2, 64, 1, 0>, grid, block, s, g0, g1, (int)t0);
    else
        launch_k(gemm_wide_pair_kernel<BC_EPI_BIAS, 256, 256, 4, 4, 2, 64, 1, 0>, grid, block, s, g0, g1, (int)t0);
    prof_end(cls, s);
    return check_launch("gemm pair");
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
    e.q_scale_to = 0; e.q_scale = 1.f;
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
