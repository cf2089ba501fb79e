// Internal helpers of the HIP library (gfx950 only).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "moe.h"

namespace moe {

// Element storage types: bf16 is kept as its 16-bit pattern.
typedef uint16_t bf16_t;

// MFMA operand / accumulator vector types.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
    return __uint_as_float(((uint32_t)h) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__device__ __forceinline__ float silu(float a) {
    return a / (1.0f + __expf(-a));
}

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(v, o, 64);
        if (lane >= o) v += u;
    }
    return v;
}

// Largest s in [0, n) with a[s] <= v, for non-decreasing a with a[0] <= v.
__device__ __forceinline__ int last_le(const int* a, int n, int v) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a[mid] <= v) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__host__ __device__ constexpr int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Launch-error check shared by the host wrappers.
inline int launch_status() {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? MOE_OK : MOE_ERR_DEVICE;
}

// Raise kernel F's dynamic-LDS limit to `bytes` on the current device.  The
// setting persists, so each device is configured once per size increase and
// later launches skip the runtime call.  The check, the runtime call and the
// record of the granted size happen under one lock per kernel, so concurrent
// callers never leave a smaller limit set than the one recorded.
template <auto F>
inline int allow_dynamic_lds(size_t bytes) {
    constexpr int kMaxDevices = 64;
    static std::mutex lock;
    static int granted[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MOE_ERR_DEVICE;
    std::lock_guard<std::mutex> guard(lock);
    if (granted[dev] >= (int)bytes) return MOE_OK;
    if (hipFuncSetAttribute((const void*)F, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes) != hipSuccess)
        return MOE_ERR_DEVICE;
    granted[dev] = (int)bytes;
    return MOE_OK;
}

// ---------------------------------------------------------------------------
// Internal launchers (one translation unit each); arguments already validated.
// ---------------------------------------------------------------------------
int launch_route_topk(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
                      int E, int k, int flags, float* logits, int32_t* idx, float* gate, void* ws,
                      hipStream_t s);
size_t route_ws_bytes(int dtype, int64_t T, int d, int E, int flags);

int launch_quantize_e4m3(const void* x, int dtype, int64_t rows, int cols, uint8_t* q, float* scales,
                         hipStream_t s);
int launch_route_topk_e4m3(const uint8_t* xq, const float* sx, const uint8_t* wq, const float* sw,
                           const float* bias, int64_t T, int d, int E, int k, int flags,
                           float* logits, int32_t* idx, float* gate, hipStream_t s);

// Tiled score kernel (score.hip): K chunks for a batch, 0 if the shape does not
// suit it; launch with S chunks (S == 1 writes scores + bias to out[T][E],
// S > 1 partial scores to out[S][T][E], to be summed in chunk order).
int score_tiles_split(int64_t T, int rowbytes, int E, bool allow_split);
int launch_score_tiles(bool fp8, const void* x, const void* w, const float* sx, const float* sw,
                       const float* bias, int64_t T, int rowbytes, int E, int S, float* out,
                       hipStream_t s);
// The bf16 tiled score kernel with one K chunk over 33-64 experts (MOE_ERR_SHAPE
// otherwise), finishing with the top-k and gates of its tokens (logits nullable:
// scores + bias stored there when given).
int launch_score_tiles_topk(const void* x, const void* w, const float* bias, int64_t T,
                            int rowbytes, int E, int k, int renorm, float* logits, int32_t* idx,
                            float* gate, hipStream_t s);
// Top-k and gates of given scores (route.hip): scores[T][E] read in place.
int launch_topk_given(const float* scores, int64_t T, int E, int k, int flags, int32_t* idx,
                      float* gate, hipStream_t s);

int launch_histogram(const int32_t* idx, int64_t T, int k, int E, int32_t* counts, int32_t* coact,
                     hipStream_t s);

struct PermuteTables {
    uint64_t hosts[MOE_MAX_E];          // bit j set iff GPU j hosts expert e
    int16_t slot_of[MOE_MAX_E];         // local slot of expert e, or -1
    int16_t expert_of_slot[MOE_MAX_GROUPS];
};

int launch_permute(const void* x, int dtype, const int32_t* idx, const float* gate,
                   const int32_t* counts, int64_t T, int d, int k, int E, const PermuteTables& tab,
                   int n_local, int G, int dev, void* x_perm, int64_t cap_rows,
                   int32_t* group_offsets, int32_t* row_token, float* row_gate, int32_t* token_row,
                   int32_t* send_counts, void* ws, hipStream_t s);
size_t permute_ws_bytes(int64_t T, int k, int E);
// Device address of the library's own permute scratch on the current device
// (MOE_PERMUTE_NOALLOC_MAX_WS bytes, 256-byte aligned).
int permute_scratch(void** ptr);

// a_rows (nullable): row p of the first product's input is row a_rows[p] of
// x_perm, which then holds a_total rows (the token rows; no packaged copy).
// lead > 0: the first `lead` of the n_groups groups hold lead_rows rows each,
// and offsets (n_groups - lead + 1 entries) counts the others' rows from row
// lead * lead_rows.
int launch_grouped_ffn(const void* x_perm, int dtype, const int32_t* offsets, int n_groups,
                       const void* const* w13, const void* const* w2, int d, int f,
                       int64_t cap_rows, void* y_perm, void* ws, hipStream_t s,
                       const int32_t* a_rows = nullptr, int64_t a_total = 0,
                       int products = MOE_FFN_GATE_UP | MOE_FFN_DOWN,
                       const void* combine = nullptr, int lead = 0, int lead_rows = 0);
// moe_grouped_ffn with every group streamed and the down product's chunk sum
// writing the gate-weighted combine (bf16)
int launch_grouped_ffn_combine(const void* x_perm, const int32_t* offsets, int n_groups,
                               const void* const* w13, const void* const* w2, int d, int f,
                               int64_t cap_rows, const int32_t* token_row, const float* gate,
                               const void* y_shared, int64_t T, int k, void* y, void* ws,
                               hipStream_t s);
size_t grouped_ffn_ws_bytes(int dtype, int64_t cap_rows, int d, int f, int n_groups);

// y_shared: n_shared slices of [T][d] (nullable: none)
int launch_combine(const void* y_perm, int dtype, const int32_t* token_row, const float* gate,
                   const void* y_shared, int n_shared, int64_t T, int d, int k, void* y,
                   hipStream_t s);

}  // namespace moe
