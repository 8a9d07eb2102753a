// The forecast of Eq. 13, x_hat = sum_j w_j x_{f=-j}, as one memory-bound
// pass, and the cache-context (ring) ABI around it.
//
// Each thread owns U 16-byte vectors of the output; for each it loads the
// matching 16 bytes of all K cached features (every load issued before any
// arithmetic), accumulates in fp32 with the K weights held in SGPRs (kernel
// arguments), and stores once.  Algorithmic traffic is (K * in + out) bytes
// per element.  The weights are fp64 on the host, computed once per plan.
#include <cmath>
#include <cstring>
#include <new>

#include "hip_common.h"

namespace bc {

struct FcArgs {
    const void* src[kMaxK];
    float w[kMaxK];
    void* out;
    int64_t n;       // elements
};

constexpr int kThreads = 256;
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// The vector path works in units of one 16-byte input chunk per thread and
// step: 8 bf16 or 4 fp32 elements, so every load instruction of a wave reads
// 1 KiB of consecutive bytes of each cached feature.
template <typename Tin> struct Unit { static constexpr int el = 16 / (int)sizeof(Tin); };

template <typename Tin>
__device__ __forceinline__ void unpack_unit(const u32x4& raw, float* f) {
    if constexpr (sizeof(Tin) == 2) unpack(raw, f, (const bf16*)nullptr);
    else unpack(raw, f, (const float*)nullptr);
}

// Store EL fp32 values as EL elements of Tout (16 bytes for bf16 -> bf16 and
// fp32 -> fp32, 8 for fp32 -> bf16, 32 for bf16 -> fp32).
template <typename Tout, int EL>
__device__ __forceinline__ void store_unit(Tout* p, const float* f) {
    if constexpr (sizeof(Tout) == 2) {
        uint32_t w[EL / 2];
#pragma unroll
        for (int i = 0; i < EL / 2; ++i) {
            bf16 lo = (bf16)f[2 * i], hi = (bf16)f[2 * i + 1];
            w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
        }
        if constexpr (EL == 8) {
            u32x4 u = {w[0], w[1], w[2], w[3]};
            __builtin_nontemporal_store(u, reinterpret_cast<u32x4*>(p));
        } else {
            u32x2 u = {w[0], w[1]};
            __builtin_nontemporal_store(u, reinterpret_cast<u32x2*>(p));
        }
    } else {
        u32x4* q = reinterpret_cast<u32x4*>(p);
#pragma unroll
        for (int c = 0; c < EL / 4; ++c) {
            u32x4 a = {__float_as_uint(f[4 * c]), __float_as_uint(f[4 * c + 1]), __float_as_uint(f[4 * c + 2]),
                       __float_as_uint(f[4 * c + 3])};
            __builtin_nontemporal_store(a, q + c);
        }
    }
}

// Vector path: every pointer 16-byte aligned; covers the first n / EL * EL
// elements.  A thread owns U units, threads of a workgroup consecutive units.
template <int K, typename Tin_, typename Tout_, int U>
__global__ __launch_bounds__(kThreads) void forecast_vec_kernel(FcArgs a) {
    typedef elem_t<Tin_> Tin;
    typedef elem_t<Tout_> Tout;
    constexpr int EL = Unit<Tin>::el;
    const int64_t nv = a.n / EL;
    const int64_t v0 = (int64_t)blockIdx.x * (kThreads * U) + threadIdx.x;
    u32x4 raw[U][K];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t v = v0 + (int64_t)u * kThreads;
        if (v < nv) {
#pragma unroll
            for (int j = 0; j < K; ++j)
                raw[u][j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(static_cast<const Tin*>(a.src[j]) + v * EL));
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t v = v0 + (int64_t)u * kThreads;
        if (v < nv) {
            float acc[EL], x[EL];
            unpack_unit<Tin>(raw[u][0], x);
#pragma unroll
            for (int e = 0; e < EL; ++e) acc[e] = a.w[0] * x[e];
#pragma unroll
            for (int j = 1; j < K; ++j) {
                unpack_unit<Tin>(raw[u][j], x);
#pragma unroll
                for (int e = 0; e < EL; ++e) acc[e] = __builtin_fmaf(a.w[j], x[e], acc[e]);
            }
            store_unit<Tout, EL>(static_cast<Tout*>(a.out) + v * EL, acc);
        }
    }
}

// Element path: any alignment; handles [begin, n).
template <typename Tin_, typename Tout_>
__global__ __launch_bounds__(kThreads) void forecast_scalar_kernel(FcArgs a, int K, int64_t begin) {
    typedef elem_t<Tin_> Tin;
    typedef elem_t<Tout_> Tout;
    for (int64_t i = begin + (int64_t)blockIdx.x * kThreads + threadIdx.x; i < a.n;
         i += (int64_t)gridDim.x * kThreads) {
        float acc = 0.f;
        for (int j = 0; j < K; ++j) acc = __builtin_fmaf(a.w[j], ld(static_cast<const Tin*>(a.src[j]) + i), acc);
        st(static_cast<Tout*>(a.out) + i, acc);
    }
}

template <typename Tin, typename Tout, int U>
static void launch_vec(const FcArgs& a, int K, int64_t nv, hipStream_t s) {
    const int64_t blocks = (nv + kThreads * U - 1) / (kThreads * U);
    dim3 g((unsigned)blocks), b(kThreads);
    switch (K) {
#define BC_FC_CASE(KK) case KK: launch_k(forecast_vec_kernel<KK, tag_t<Tin>, tag_t<Tout>, U>, g, b, s, a); break;
        BC_FC_CASE(1) BC_FC_CASE(2) BC_FC_CASE(3) BC_FC_CASE(4)
        BC_FC_CASE(5) BC_FC_CASE(6) BC_FC_CASE(7) BC_FC_CASE(8)
#undef BC_FC_CASE
        default: break;
    }
}

template <typename Tin, typename Tout>
static int run_forecast(const FcArgs& a, int K, hipStream_t s) {
    // Large tensors: four 16-byte units per thread, all loads issued first;
    // small ones (below ~32M elements): one per thread, for more workgroups
    // in flight.
    constexpr int U = 4;
    constexpr int EL = Unit<Tin>::el;
    bool aligned = (reinterpret_cast<uintptr_t>(a.out) % 16) == 0;
    for (int j = 0; j < K; ++j) aligned = aligned && (reinterpret_cast<uintptr_t>(a.src[j]) % 16) == 0;
    int64_t done = 0;
    if (aligned) {
        const int64_t nv = a.n / EL;
        if (nv > 0) {
            if (nv / kThreads > 0x7fffffff) return fail(BC_ERR_UNSUPPORTED, "forecast of %lld elements is too large", (long long)a.n);
            if (a.n >= ((int64_t)32 << 20)) launch_vec<Tin, Tout, U>(a, K, nv, s);
            else launch_vec<Tin, Tout, 1>(a, K, nv, s);
            done = nv * EL;
        }
    }
    if (done < a.n) {
        const int64_t rest = a.n - done;
        int64_t blocks = (rest + kThreads - 1) / kThreads;
        if (blocks > 65536) blocks = 65536;
        launch_k(forecast_scalar_kernel<tag_t<Tin>, tag_t<Tout>>, dim3((unsigned)blocks), dim3(kThreads), s, a, K, done);
    }
    return check_launch("forecast");
}

int launch_forecast(const void* const* src, const float* w, int K, int64_t n, int in_dt,
                    void* out, int out_dt, hipStream_t s) {
    if (K < 1 || K > kMaxK) return fail(BC_ERR_INVALID_ARG, "K=%d outside [1, 8]", K);
    if (n <= 0) return BC_OK;
    FcArgs a;
    std::memset(&a, 0, sizeof a);
    for (int j = 0; j < K; ++j) { a.src[j] = src[j]; a.w[j] = w[j]; }
    a.out = out;
    a.n = n;
    int rc;
    prof_begin(PROF_FORECAST, s, (double)n * (K * dtype_size(in_dt) + dtype_size(out_dt)));
    if (in_dt == BC_BF16 && out_dt == BC_BF16) rc = run_forecast<bf16, bf16>(a, K, s);
    else if (in_dt == BC_BF16) rc = run_forecast<bf16, float>(a, K, s);
    else if (out_dt == BC_BF16) rc = run_forecast<float, bf16>(a, K, s);
    else rc = run_forecast<float, float>(a, K, s);
    prof_end(PROF_FORECAST, s);
    return rc;
}

// ---- plain copies and zero fills (byte streams) ------------------------------

// 16-byte chunks: each workgroup copies one contiguous run of 4 x 256
// chunks, each thread four of them (all four loads issued before the
// stores), non-temporal: a copied feature is not read again soon.  One pass
// over the grid (no grid-stride loop) measured 6.3 TB/s on a 805 MB copy
// against 5.1-5.5 TB/s for grid-stride variants.
constexpr int kCopyU = 4;
__global__ __launch_bounds__(kThreads) void copy16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n16) {
    const int64_t base = (int64_t)blockIdx.x * (kThreads * kCopyU) + threadIdx.x;
    u32x4 v[kCopyU];
#pragma unroll
    for (int u = 0; u < kCopyU; ++u)
        if (base + u * kThreads < n16) v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + base + u * kThreads));
#pragma unroll
    for (int u = 0; u < kCopyU; ++u)
        if (base + u * kThreads < n16) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4*>(dst + base + u * kThreads));
}
__global__ __launch_bounds__(kThreads) void copy1_kernel(const uint8_t* src, uint8_t* dst, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
        dst[i] = src[i];
}
__global__ __launch_bounds__(kThreads) void zero16_kernel(uint4* dst, int64_t n16) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += (int64_t)gridDim.x * kThreads)
        dst[i] = make_uint4(0, 0, 0, 0);
}
__global__ __launch_bounds__(kThreads) void zero1_kernel(uint8_t* dst, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
        dst[i] = 0;
}

static unsigned grid_for(int64_t items) {
    int64_t b = (items + kThreads - 1) / kThreads;
    if (b > 8192) b = 8192;
    if (b < 1) b = 1;
    return (unsigned)b;
}

int launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s) {
    if (bytes <= 0) return BC_OK;
    const bool vec = ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) | (uintptr_t)bytes) % 16) == 0;
    const int64_t blocks = (bytes / 16 + kThreads * kCopyU - 1) / (kThreads * kCopyU);
    if (vec && blocks > 0x7fffffff) return fail(BC_ERR_UNSUPPORTED, "copy of %lld bytes is too large", (long long)bytes);
    prof_begin(PROF_COPY, s, 2.0 * (double)bytes);
    if (vec)
        launch_k(copy16_kernel, dim3((unsigned)blocks), dim3(kThreads), s, static_cast<const uint4*>(src),
                 static_cast<uint4*>(dst), bytes / 16);
    else
        launch_k(copy1_kernel, dim3(grid_for(bytes)), dim3(kThreads), s, static_cast<const uint8_t*>(src),
                 static_cast<uint8_t*>(dst), bytes);
    prof_end(PROF_COPY, s);
    return check_launch("copy");
}

int launch_fill_zero(void* dst, int64_t bytes, hipStream_t s) {
    if (bytes <= 0) return BC_OK;
    if ((reinterpret_cast<uintptr_t>(dst) | (uintptr_t)bytes) % 16 == 0)
        zero16_kernel<<<grid_for(bytes / 16), kThreads, 0, s>>>(static_cast<uint4*>(dst), bytes / 16);
    else
        zero1_kernel<<<grid_for(bytes), kThreads, 0, s>>>(static_cast<uint8_t*>(dst), bytes);
    return check_launch("fill");
}

int check_launch(const char* what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BC_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
    return BC_OK;
}

}  // namespace bc

// ---------------------------------------------------------------------------
// Ring ABI
// ---------------------------------------------------------------------------
using namespace bc;

extern "C" {

int bc_cache_create(int K, int64_t numel, int dtype, void* dev_storage, bc_cache_ring** out) {
    clear_error();
    if (!out || !dev_storage) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (K < 1 || K > kMaxK) return fail(BC_ERR_INVALID_ARG, "K=%d outside [1, 8]", K);
    if (numel < 1) return fail(BC_ERR_INVALID_ARG, "numel=%lld", (long long)numel);
    if (dtype != BC_F32 && dtype != BC_BF16) return fail(BC_ERR_INVALID_ARG, "dtype=%d", dtype);
    bc_cache_ring* r = new (std::nothrow) bc_cache_ring;
    if (!r) return fail(BC_ERR_INVALID_ARG, "out of host memory");
    r->K = K;
    r->numel = numel;
    r->dtype = dtype;
    r->storage = static_cast<char*>(dev_storage);
    r->head = -1;
    r->count = 0;
    for (int j = 0; j < kMaxK; ++j) r->coord[j] = 0.0;
    *out = r;
    return BC_OK;
}

int bc_cache_destroy(bc_cache_ring* r) {
    clear_error();
    delete r;
    return BC_OK;
}

int bc_cache_reset(bc_cache_ring* r) {
    clear_error();
    if (!r) return fail(BC_ERR_INVALID_ARG, "NULL ring");
    r->head = -1;
    r->count = 0;
    return BC_OK;
}

static char* slot_ptr(const bc_cache_ring* r, int slot) {
    return r->storage + (int64_t)slot * r->numel * dtype_size(r->dtype);
}

int bc_cache_next_slot(const bc_cache_ring* r, void** dev_ptr) {
    clear_error();
    if (!r || !dev_ptr) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    *dev_ptr = slot_ptr(r, (r->head + 1) % r->K);
    return BC_OK;
}

int bc_cache_push(bc_cache_ring* r, const void* feat, double t, void* stream) {
    clear_error();
    if (!r) return fail(BC_ERR_INVALID_ARG, "NULL ring");
    if (!std::isfinite(t)) return fail(BC_ERR_INVALID_ARG, "node time is not finite");
    const int slot = (r->head + 1) % r->K;
    char* dst = slot_ptr(r, slot);
    if (feat && feat != dst) {
        int rc = launch_copy(feat, dst, r->numel * dtype_size(r->dtype), static_cast<hipStream_t>(stream));
        if (rc != BC_OK) return rc;
    }
    r->head = slot;
    r->coord[slot] = t;
    r->count = r->count < r->K ? r->count + 1 : r->K;
    return BC_OK;
}

int bc_cache_state(const bc_cache_ring* r, int* count, int* head, double* t_nodes, int* slots) {
    clear_error();
    if (!r) return fail(BC_ERR_INVALID_ARG, "NULL ring");
    if (count) *count = r->count;
    if (head) *head = r->head;
    for (int j = 0; j < r->count; ++j) {
        const int slot = ((r->head - j) % r->K + r->K) % r->K;
        if (t_nodes) t_nodes[j] = r->coord[slot];
        if (slots) slots[j] = slot;
    }
    return BC_OK;
}

int bc_bary_extrapolate(const bc_cache_ring* r, const double* w, int count, void* out, int out_dtype,
                        void* stream) {
    clear_error();
    if (!r || !w || !out) return fail(BC_ERR_INVALID_ARG, "NULL pointer");
    if (out_dtype != BC_F32 && out_dtype != BC_BF16) return fail(BC_ERR_INVALID_ARG, "out dtype %d", out_dtype);
    if (count < 1 || count > r->K) return fail(BC_ERR_INVALID_ARG, "count=%d outside [1, K=%d]", count, r->K);
    if (count > r->count) return fail(BC_ERR_STATE, "forecast over %d nodes but the ring holds %d", count, r->count);
    const void* src[kMaxK];
    float wf[kMaxK];
    for (int j = 0; j < count; ++j) {
        if (!std::isfinite(w[j])) return fail(BC_ERR_INVALID_ARG, "weight %d is not finite", j);
        src[j] = slot_ptr(r, ((r->head - j) % r->K + r->K) % r->K);
        wf[j] = (float)w[j];
    }
    return launch_forecast(src, wf, count, r->numel, r->dtype, out, out_dtype, static_cast<hipStream_t>(stream));
}

}  // extern "C"
