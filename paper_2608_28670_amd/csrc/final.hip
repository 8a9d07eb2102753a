// The last part of every sampling step fused into one pass over the tokens:
// the stepwise feature (the barycentric forecast of Eq. 13, or the feature
// just computed), the final layer's LayerNorm + adaLN modulation and linear
// D -> p*p*C_out, and the sampler update of the latent pixels each token
// covers (unpatchify folded into the indexing).  A workgroup owns 16 tokens:
// in each wave, lane l holds token l % 16 and the 16-byte feature chunks
// 4 s + l / 16 of the wave's chunk steps s, which is exactly the A-operand layout of
// v_mfma_f32_16x16x32_bf16, so the normalised row feeds the MFMA without
// leaving registers.  A workgroup's waves split the row's D (four chunk steps
// each, twelve at D = 3072) and meet in LDS for the row statistics and the sum
// of their partial outputs.  The HBM traffic is the K cached features plus the
// latents; the feature, the LayerNorm output and the model output never touch
// memory.
#include "ops.h"

namespace bc {

namespace {

constexpr float kFinalEps = 1e-6f;

__device__ __forceinline__ float group4_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// CH = D / 32 chunk steps of a row, CW per wave over CH / CW waves (CW = 4;
// 12 for D = 3072: 8 waves, two per SIMD); NT = NO / 16 output tiles; KK =
// number of cached features.  With CW > 4 the modulation vectors
// and weight fragments are loaded per chunk step in the linear, after the
// statistics, instead of with the features (they would not fit the
// registers next to them).  Rows past the last token (B T not a multiple of
// 16) read the last row and update nothing.
// MODE 0: bf16 features.  MODE 1: the same for a guided batch of 2B samples,
// the second half unconditional: the workgroup computes the outputs of its
// 16 tokens in both halves and updates the B latents with u + cfg (c - u).
// MODE 2: one fp32 feature (the blockwise sampler's stream), normalised in
// fp32 as it is, like the LayerNorm kernel on an fp32 input.
template <int CH, int NT, int KK, int CW, int MODE>
__global__ __launch_bounds__(64 * (CH / CW)) void final_step_kernel(FinalStepArgs a) {
    constexpr int NWV = CH / CW;                        // waves per workgroup
    constexpr bool LATE = CW > 4;                       // modulation and weights loaded in the linear
    constexpr bool F32 = MODE == 2;
    static_assert(NWV * CW == CH, "D / 32 must be a multiple of the chunk steps per wave");
    static_assert(!F32 || KK == 1, "the fp32 feature is a single source");
    __shared__ float s_stat[NWV][16];
    __shared__ f32x4 s_out[NWV][NT][64];
    const int lane = threadIdx.x & 63, grp = lane >> 4, wave = threadIdx.x >> 6;
    const int64_t rows = (int64_t)a.B * a.T;
    const int64_t row0 = (int64_t)blockIdx.x * 16;
    const int64_t row = min(row0 + (lane & 15), rows - 1);
    const int D = CH * 32;
    const int sbeg = wave * CW;
    const bf16* W = static_cast<const bf16*>(a.W);

    // The outputs of this workgroup's 16 tokens in the model batch's half
    // that starts at feature row roff (sample offset boff); wave 0 returns
    // them in `res`.
    auto pass = [&](int64_t roff, int boff, f32x4 (&res)[NT]) __attribute__((always_inline)) {
        const int64_t frow = row + roff;
        // 1. This wave's feature chunks of the row, all K sources loaded at
        // once, combined in fp32 and rounded to bf16 (fp32 features are kept).
        // (Up to four chunk steps of all K sources are in flight at a time.)
        constexpr int CB = CW < 4 ? CW : 4;
        u32x4 raw[KK][CB];
        f32x4 rawf[F32 ? CB : 1][2];
        auto load_raw = [&](int s0) __attribute__((always_inline)) {
            if constexpr (F32) {
#pragma unroll
                for (int s = 0; s < CB; ++s) {
                    const float* p = static_cast<const float*>(a.src[0]) + frow * D + 32 * (sbeg + s0 + s) + 8 * grp;
                    rawf[s][0] = *reinterpret_cast<const f32x4*>(p);
                    rawf[s][1] = *reinterpret_cast<const f32x4*>(p + 4);
                }
            } else {
#pragma unroll
                for (int j = 0; j < KK; ++j)
#pragma unroll
                    for (int s = 0; s < CB; ++s)
                        raw[j][s] = *reinterpret_cast<const u32x4*>(static_cast<const bf16*>(a.src[j]) + frow * D +
                                                                    32 * (sbeg + s0 + s) + 8 * grp);
            }
        };
        load_raw(0);
        // The modulation vectors and the weight fragments do not depend on the
        // statistics: load them now, with the features.
        const int b = (int)(row / a.T) + boff;
        const float* shift = a.fmod + (int64_t)b * 2 * D;
        const float* scale = shift + D;
        constexpr int CP = LATE ? 1 : CW;               // chunk steps whose operands are preloaded
        f32x4 shv4[CP][2], scv4[CP][2];
        bf16x8 wf[CP][NT];
        auto load_ops = [&](int s, int slot) __attribute__((always_inline)) {
            const int d0 = 32 * (sbeg + s) + 8 * grp;
            shv4[slot][0] = *reinterpret_cast<const f32x4*>(shift + d0);
            shv4[slot][1] = *reinterpret_cast<const f32x4*>(shift + d0 + 4);
            scv4[slot][0] = *reinterpret_cast<const f32x4*>(scale + d0);
            scv4[slot][1] = *reinterpret_cast<const f32x4*>(scale + d0 + 4);
#pragma unroll
            for (int t = 0; t < NT; ++t)
                wf[slot][t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(W + (int64_t)(16 * t + (lane & 15)) * D + d0));
        };
        if constexpr (!LATE) {
#pragma unroll
            for (int s = 0; s < CW; ++s) load_ops(s, s);
        }
        u32x4 h[F32 ? 1 : CW];
        f32x4 hf[F32 ? CW : 1][2];
        float sum = 0.f;
#pragma unroll
        for (int s = 0; s < CW; ++s) {
            if (s > 0 && s % CB == 0) load_raw(s);
            if constexpr (F32) {
                hf[s][0] = rawf[s % CB][0];
                hf[s][1] = rawf[s % CB][1];
#pragma unroll
                for (int e = 0; e < 4; ++e) sum += hf[s][0][e] + hf[s][1][e];
            } else {
                float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < KK; ++j) {
                    float f[8];
                    unpack(raw[j][s % CB], f, static_cast<const bf16*>(nullptr));
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[e] += a.w[j] * f[e];
                }
                uint32_t wd[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bf16 lo = (bf16)acc[2 * q], hi = (bf16)acc[2 * q + 1];
                    sum += (float)lo + (float)hi;
                    wd[q] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
                }
                h[s] = u32x4{wd[0], wd[1], wd[2], wd[3]};
            }
        }
        auto feature = [&](int s, float (&f)[8]) __attribute__((always_inline)) {
            if constexpr (F32) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    f[e] = hf[s][0][e];
                    f[4 + e] = hf[s][1][e];
                }
            } else {
                unpack(h[s], f, static_cast<const bf16*>(nullptr));
            }
        };
        // 2. Row statistics: over the row's four lanes (l, l^16, l^32, l^48), then
        // over the waves through LDS; two passes (mean, centred squares).
        sum = group4_sum(sum);
        if (grp == 0) s_stat[wave][lane] = sum;
        __syncthreads();
        float mean = 0.f;
#pragma unroll
        for (int v = 0; v < NWV; ++v) mean += s_stat[v][lane & 15];
        mean /= (float)D;
        float sq = 0.f;
#pragma unroll
        for (int s = 0; s < CW; ++s) {
            float f[8];
            feature(s, f);
#pragma unroll
            for (int e = 0; e < 8; ++e) sq += (f[e] - mean) * (f[e] - mean);
        }
        sq = group4_sum(sq);
        __syncthreads();   // every wave has read the sums
        if (grp == 0) s_stat[wave][lane] = sq;
        __syncthreads();
        float var = 0.f;
#pragma unroll
        for (int v = 0; v < NWV; ++v) var += s_stat[v][lane & 15];
        var /= (float)D;
        const float rstd = 1.0f / sqrtf(var + kFinalEps);

        // 3. Normalise + modulate into MFMA operands; this wave's part of the
        // linear over its k-range, partial outputs summed through LDS.
        f32x4 out[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) out[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < CW; ++s) {
            const int q4 = LATE ? 0 : s;
            if constexpr (LATE) load_ops(s, 0);
            float f[8];
            feature(s, f);
            const float shv[8] = {shv4[q4][0][0], shv4[q4][0][1], shv4[q4][0][2], shv4[q4][0][3],
                                  shv4[q4][1][0], shv4[q4][1][1], shv4[q4][1][2], shv4[q4][1][3]};
            const float scv[8] = {scv4[q4][0][0], scv4[q4][0][1], scv4[q4][0][2], scv4[q4][0][3],
                                  scv4[q4][1][0], scv4[q4][1][1], scv4[q4][1][2], scv4[q4][1][3]};
            uint32_t wd[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bf16 lo = (bf16)((f[2 * q] - mean) * rstd * (1.0f + scv[2 * q]) + shv[2 * q]);
                const bf16 hi = (bf16)((f[2 * q + 1] - mean) * rstd * (1.0f + scv[2 * q + 1]) + shv[2 * q + 1]);
                wd[q] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
            }
            const bf16x8 af = __builtin_bit_cast(bf16x8, u32x4{wd[0], wd[1], wd[2], wd[3]});
#pragma unroll
            for (int t = 0; t < NT; ++t) out[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[q4][t], out[t], 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) s_out[wave][t][lane] = out[t];
        __syncthreads();
        if (wave == 0) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                res[t] = s_out[0][t][lane];
#pragma unroll
                for (int v = 1; v < NWV; ++v) res[t] += s_out[v][t][lane];
            }
        }
    };

    f32x4 out[NT];
    if constexpr (MODE == 1) {
        // The conditional outputs wait in LDS (not in registers) while the
        // unconditional half is computed.
        __shared__ f32x4 s_cond[NT][64];
        pass(0, 0, out);
        if (wave == 0) {
#pragma unroll
            for (int t = 0; t < NT; ++t) s_cond[t][lane] = out[t];
        }
        pass(rows, a.B, out);
        if (wave == 0) {
#pragma unroll
            for (int t = 0; t < NT; ++t) out[t] += a.cfg * (s_cond[t][lane] - out[t]);
        }
    } else {
        pass(0, 0, out);
    }
    if (wave != 0) return;

    // 4. Bias and the sampler update.  Lane l holds tokens row0 + 4 (l/16) + r
    // and output feature n = 16 t + l % 16 = ((py p + px) C_out + c).  (With
    // guidance the bias appears in both halves and cancels in c - u.)
    const LatentShape& ls = a.ls;
    const int p = ls.p, hp = ls.H / p, wp = ls.W / p;
    const int64_t S = (int64_t)ls.F * ls.H * ls.W;
    const bf16* bias = static_cast<const bf16*>(a.bias);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int n = 16 * t + (lane & 15);
        const int c = n % a.C_out, pp = n / a.C_out;
        if (c >= ls.C) continue;                        // output channels the sampler does not use
        const int py = pp / p, px = pp % p;
        const float bv = bias ? (float)bias[n] : 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t tr = row0 + 4 * grp + r;
            if (tr >= rows) continue;
            const int bb = (int)(tr / a.T), tok = (int)(tr % a.T);
            const int f = tok / (hp * wp), ty = (tok / wp) % hp, tx = tok % wp;
            const int64_t i = ((int64_t)bb * ls.C + c) * S + ((int64_t)f * ls.H + ty * p + py) * ls.W + tx * p + px;
            sampler_update(a.sc, a.x + i, out[t][r] + bv, a.prev ? a.prev + i : nullptr);
        }
    }
}

}  // namespace

// Instantiated (D / 32, NO / 16): D 1152 (DiT-XL/2, PixArt), 3072 (the video
// model) and 1280, 128 and 256 (small models), with 16 to 64 outputs per
// token; 1 to 4 cached features.
#define BC_FINAL_VARIANTS(X) X(36, 2) X(36, 4) X(40, 2) X(40, 4) X(96, 4) X(4, 1) X(4, 2) X(8, 1) X(8, 2) X(8, 4)

bool final_step_supported(int dt, int D, int NO, int T) {
    if (dt != BC_BF16 || D % 32 || NO % 16 || T < 1) return false;
    const int ch = D / 32, nt = NO / 16;
#define BC_FS_HAS(CH, NTT) if (ch == CH && nt == NTT) return true;
    BC_FINAL_VARIANTS(BC_FS_HAS)
#undef BC_FS_HAS
    return false;
}

template <int CH, int NT, int MODE>
static int launch_fs_mode(const FinalStepArgs& a, dim3 grid, hipStream_t s) {
    constexpr int CW = CH > 40 ? 12 : 4;
    const dim3 block(64 * (CH / CW));
    if constexpr (MODE == 2) {
        final_step_kernel<CH, NT, 1, CW, 2><<<grid, block, 0, s>>>(a);
    } else {
        switch (a.K) {
            case 1: final_step_kernel<CH, NT, 1, CW, MODE><<<grid, block, 0, s>>>(a); break;
            case 2: final_step_kernel<CH, NT, 2, CW, MODE><<<grid, block, 0, s>>>(a); break;
            case 3: final_step_kernel<CH, NT, 3, CW, MODE><<<grid, block, 0, s>>>(a); break;
            case 4: final_step_kernel<CH, NT, 4, CW, MODE><<<grid, block, 0, s>>>(a); break;
            default: return fail(BC_ERR_UNSUPPORTED, "fused final step: %d cached features", a.K);
        }
    }
    return check_launch("final step");
}

// Guided and blockwise runs exist for the class- and caption-conditioned
// models only (D <= 1280).
template <int CH, int NT>
static int launch_fs(const FinalStepArgs& a, dim3 grid, hipStream_t s) {
    if constexpr (CH <= 40) {
        if (a.src_f32) return launch_fs_mode<CH, NT, 2>(a, grid, s);
        if (a.guided) return launch_fs_mode<CH, NT, 1>(a, grid, s);
    } else {
        if (a.src_f32 || a.guided) return fail(BC_ERR_UNSUPPORTED, "fused final step: guided or fp32 feature at D %d", a.D);
    }
    return launch_fs_mode<CH, NT, 0>(a, grid, s);
}

int launch_final_step(const FinalStepArgs& a, hipStream_t s) {
    if (!final_step_supported(BC_BF16, a.D, a.NO, a.T) || a.K < 1 || a.K > kFinalMaxK ||
        a.NO != a.ls.p * a.ls.p * a.C_out || a.T != a.ls.tokens() || (a.src_f32 && (a.K != 1 || a.guided)))
        return fail(BC_ERR_UNSUPPORTED, "fused final step: D %d, NO %d, T %d, K %d", a.D, a.NO, a.T, a.K);
    const int64_t rows = (int64_t)a.B * a.T;
    const dim3 grid((unsigned)((rows + 15) / 16));
    const int ch = a.D / 32, nt = a.NO / 16;
#define BC_FS(CH, NTT) if (ch == CH && nt == NTT) return launch_fs<CH, NTT>(a, grid, s);
    BC_FINAL_VARIANTS(BC_FS)
#undef BC_FS
    return fail(BC_ERR_UNSUPPORTED, "fused final step: D %d, NO %d", a.D, a.NO);
}

}  // namespace bc
