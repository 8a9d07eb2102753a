// Device-side types and helpers shared by the HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <cstdint>

#include "common.h"

typedef __bf16 bf16;
// Kernel template arguments name the element type through a tag, so no kernel
// symbol carries the __bf16 type (its mangling, DF16b, is rejected or misread
// by the demanglers that profilers use): a kernel is instantiated with float
// or bf16_tag and declares its pointer parameters as elem_t<tag>*.
struct bf16_tag {};
template <typename X> struct ElemOf { typedef X type; };
template <> struct ElemOf<bf16_tag> { typedef __bf16 type; };
template <typename X> using elem_t = typename ElemOf<X>::type;
template <typename X> struct TagOf { typedef X type; };
template <> struct TagOf<__bf16> { typedef bf16_tag type; };
template <typename X> using tag_t = typename TagOf<X>::type;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte chunk

namespace bc {

// Element access in either storage type, always through fp32.
__device__ __forceinline__ float ld(const float* p) { return *p; }
__device__ __forceinline__ float ld(const bf16* p) { return (float)*p; }
__device__ __forceinline__ void st(float* p, float v) { *p = v; }
__device__ __forceinline__ void st(bf16* p, float v) { *p = (bf16)v; }   // round to nearest even

// 16-byte chunk <-> 8 (bf16) or 4 (fp32) values.
__device__ __forceinline__ void unpack(const u32x4& u, float* f, const bf16*) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void unpack(const u32x4& u, float* f, const float*) {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
}

// Workgroup id -> tile id with each XCD holding a contiguous range of tiles.
// The dispatcher deals workgroups round-robin to the 8 XCDs (workgroup i to
// XCD i % 8), so XCD x receives nwg / 8 workgroups, plus one more when
// x < nwg % 8; numbering those consecutively keeps neighbouring tiles, which
// share operands, in one XCD's L2.  A bijection on [0, nwg) for any nwg.
__device__ __forceinline__ int xcd_contiguous(int bid, int nwg) {
    const int q = nwg >> 3, r = nwg & 7;
    const int x = bid & 7, i = bid >> 3;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

template <typename T> struct ElemsPer16B { static constexpr int v = 16 / (int)sizeof(T); };

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// Wave-wide sum without LDS: DPP within each 16-lane row (lane ^ 1, lane ^ 2,
// rotate by 4 and by 8), then v_permlane16_swap / v_permlane32_swap across
// rows (with both operands equal they return the value of lane l and of lane
// l ^ 16, resp. l ^ 32, in their two results).  The result is read from lane
// 0 so every lane gets the same value.
template <int CTRL> __device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_f<0x124>(v);   // row_ror:4
    v += dpp_f<0x128>(v);   // row_ror:8 -> the 16-lane row's sum
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(b[0]) + __uint_as_float(b[1]);
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}

inline int dtype_size(int dt) { return dt == BC_BF16 ? 2 : 4; }

// Check a launch; returns BC_OK or BC_ERR_HIP with the message recorded.
int check_launch(const char* what);

// Kernel classes timed by bc_profile_*; see bc.h.
enum ProfClass { PROF_FORECAST = 0, PROF_GEMM_GELU = 1, PROF_GEMM_GATE = 2, PROF_GEMM_BIAS = 3,
                 PROF_ATTENTION = 4, PROF_LAYERNORM = 5, PROF_GEMM_DOWN = 6, PROF_COPY = 7, PROF_NCLASS = 8 };
// Open a timed bracket of class `cls`; `work` is the bracket's algorithmic
// work (FLOPs for GEMMs and attention, bytes moved for the memory-bound
// classes), recorded with the first launch inside it.
void prof_begin(int cls, hipStream_t s, double work = 0.0);
void prof_end(int cls, hipStream_t s);
// Next start/stop event pair of the class bracketed by prof_begin/prof_end on
// this thread, if that class is being timed.
bool prof_take(hipEvent_t* start, hipEvent_t* stop);
bool prof_any_enabled();                 // some kernel class is being timed

// Kernel launch that, inside a timed bracket, has the runtime stamp the
// kernel's own start and end into the class's events (the same interval a
// kernel trace reports), and is a plain launch otherwise.
template <typename... KArgs, typename... Args>
inline void launch_k(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s, Args... args) {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (!prof_take(&e0, &e1)) e0 = e1 = nullptr;
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e0, e1, 0, args...);
}

// ---- kernel launchers (each returns a bc_status) ---------------------------

// out[i] = sum_j w[j] * src[j][i] for i < n (Eq. 13), fp32 accumulation.
int launch_forecast(const void* const* src, const float* w, int K, int64_t n, int in_dt,
                    void* out, int out_dt, hipStream_t s);
int launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s);
int launch_fill_zero(void* dst, int64_t bytes, hipStream_t s);

}  // namespace bc
