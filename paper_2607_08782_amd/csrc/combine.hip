// Gate-weighted sum of the selected experts' outputs (Sec. II-A of the
// Director paper), gathered back into token order (the return trip of
// Sec. II-B), plus always-on shared experts with weight 1 (one or more
// [T][d] slices of shared-expert output, added in slice order).
//
// Bandwidth-bound gather: each thread owns one 16-byte chunk of one token's
// output row, reads the k expert rows it needs (all loads issued together;
// assignments placed on other GPUs are skipped), accumulates in fp32 in
// ascending r, and stores once.
#include "common.h"

namespace moe {
namespace {

constexpr int COMBINE_THREADS = 256;

template <typename Elem, int V>
struct Vec;

template <>
struct Vec<bf16_t, 8> {
    typedef uint4 type;
    static __device__ __forceinline__ void load(const bf16_t* p, float* v) {
        const uint4 u = *(const uint4*)p;
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    static __device__ __forceinline__ void store(bf16_t* p, const float* v) {
        uint4 u;
        u.x = pack_bf16x2(v[0], v[1]);
        u.y = pack_bf16x2(v[2], v[3]);
        u.z = pack_bf16x2(v[4], v[5]);
        u.w = pack_bf16x2(v[6], v[7]);
        *(uint4*)p = u;
    }
};

template <>
struct Vec<float, 4> {
    static __device__ __forceinline__ void load(const float* p, float* v) {
        const float4 u = *(const float4*)p;
        v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
    }
    static __device__ __forceinline__ void store(float* p, const float* v) {
        *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
    }
};

template <>
struct Vec<bf16_t, 1> {
    static __device__ __forceinline__ void load(const bf16_t* p, float* v) { v[0] = bf16_to_f32(*p); }
    static __device__ __forceinline__ void store(bf16_t* p, const float* v) { *p = f32_to_bf16(v[0]); }
};

template <>
struct Vec<float, 1> {
    static __device__ __forceinline__ void load(const float* p, float* v) { v[0] = *p; }
    static __device__ __forceinline__ void store(float* p, const float* v) { *p = v[0]; }
};

// acc += the n_shared slices y_shared[s][t][col..] (slice stride `stride`
// elements), in slice order; more than one slice: four loads at a time, a slice
// past the last re-reading the last and dropped by a select.
template <typename Elem, int V>
__device__ __forceinline__ void add_shared(const Elem* __restrict__ y_shared, int n_shared,
                                           int64_t stride, int64_t off, float* acc) {
    if (n_shared == 1) {
        float w[V];
        Vec<Elem, V>::load(y_shared + off, w);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += w[i];
        return;
    }
    for (int s0 = 0; s0 < n_shared; s0 += 4) {
        float w[4][V];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int sl = s0 + j < n_shared ? s0 + j : n_shared - 1;
            Vec<Elem, V>::load(y_shared + sl * stride + off, w[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < V; ++i) acc[i] = s0 + j < n_shared ? acc[i] + w[j][i] : acc[i];
    }
}

// KM: k rounded up to a power of two (compile-time trip counts, no spills)
template <typename Elem, int V, int KM>
__global__ __launch_bounds__(COMBINE_THREADS) void combine_kernel(
    const Elem* __restrict__ y_perm, const int32_t* __restrict__ token_row,
    const float* __restrict__ gate, const Elem* __restrict__ y_shared, int n_shared, int64_t T,
    int d, int k, int chunks_per_row, Elem* __restrict__ y) {
    const int64_t gid = (int64_t)blockIdx.x * COMBINE_THREADS + threadIdx.x;
    const int64_t t = gid / chunks_per_row;
    const int c = (int)(gid - t * chunks_per_row);
    if (t >= T) return;
    const int col = c * V;
    // The k row indices and gates first, then every row load at once: an
    // assignment with no row here (or a slot past k) re-reads the token's first
    // row here (a cache hit) and is dropped by the select, so no load sits
    // behind a branch; a token with no row here loads none.
    int32_t p[KM];
    float g[KM];
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        const int rr = r < k ? r : k - 1;
        p[r] = r < k ? token_row[t * k + rr] : -1;
        g[r] = gate[t * k + rr];
    }
    int32_t first = -1;
#pragma unroll
    for (int r = KM - 1; r >= 0; --r) first = p[r] >= 0 ? p[r] : first;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
    if (first >= 0) {
        float v[KM][V];
#pragma unroll
        for (int r = 0; r < KM; ++r)
            Vec<Elem, V>::load(y_perm + (int64_t)(p[r] >= 0 ? p[r] : first) * d + col, v[r]);
#pragma unroll
        for (int r = 0; r < KM; ++r)
#pragma unroll
            for (int i = 0; i < V; ++i) acc[i] = p[r] >= 0 ? fmaf(g[r], v[r][i], acc[i]) : acc[i];
    }
    add_shared<Elem, V>(y_shared, n_shared, T * d, t * d + col, acc);
    Vec<Elem, V>::store(y + t * d + col, acc);
}

// Rows that are a whole number of wave widths (every lane of a wave serves the
// same token): the token's local rows are compacted in registers (ascending r,
// by selects, no indexed registers), their count is uniform across the wave,
// and one of KM + 1 straight paths issues exactly that many row loads at once.
// At k = 8 with about two local rows per token this issues a quarter of the
// loads of the kernel above; the sum is the same, in the same order.
template <typename Elem, int V, int N>
__device__ __forceinline__ void combine_rows(const Elem* __restrict__ y_perm, const int32_t* q,
                                             const float* h, int d, int col, float* acc) {
    if constexpr (N > 0) {
        float v[N][V];
#pragma unroll
        for (int j = 0; j < N; ++j) Vec<Elem, V>::load(y_perm + (int64_t)q[j] * d + col, v[j]);
#pragma unroll
        for (int j = 0; j < N; ++j)
#pragma unroll
            for (int i = 0; i < V; ++i) acc[i] = fmaf(h[j], v[j][i], acc[i]);
    }
}

template <typename Elem, int V, int KM>
__global__ __launch_bounds__(COMBINE_THREADS) void combine_compact_kernel(
    const Elem* __restrict__ y_perm, const int32_t* __restrict__ token_row,
    const float* __restrict__ gate, const Elem* __restrict__ y_shared, int n_shared, int64_t T,
    int d, int k, int chunks_per_row, Elem* __restrict__ y) {
    const int64_t gid = (int64_t)blockIdx.x * COMBINE_THREADS + threadIdx.x;
    const int64_t t = gid / chunks_per_row;
    const int c = (int)(gid - t * chunks_per_row);
    if (t >= T) return;                      // whole waves: T * chunks_per_row is a multiple of 64
    const int col = c * V;
    int32_t p[KM];
    float g[KM];
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        const int rr = r < k ? r : k - 1;
        p[r] = r < k ? token_row[t * k + rr] : -1;
        g[r] = gate[t * k + rr];
    }
    // slot j of the compacted list takes the r with p[r] >= 0 and j local rows before it
    int32_t q[KM];
    float h[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        q[j] = 0;
        h[j] = 0.f;
    }
    int n = 0;
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        const bool here = p[r] >= 0;
#pragma unroll
        for (int j = 0; j <= r; ++j) {
            const bool take = here && n == j;
            q[j] = take ? p[r] : q[j];
            h[j] = take ? g[r] : h[j];
        }
        n += here ? 1 : 0;
    }
    n = __builtin_amdgcn_readfirstlane(n);
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
    static_assert(KM > 2, "the compacting combine serves k > 2");
    switch (n) {
        case 0: break;
        case 1: combine_rows<Elem, V, 1>(y_perm, q, h, d, col, acc); break;
        case 2: combine_rows<Elem, V, 2>(y_perm, q, h, d, col, acc); break;
        case 3: combine_rows<Elem, V, 3>(y_perm, q, h, d, col, acc); break;
        case 4: combine_rows<Elem, V, 4>(y_perm, q, h, d, col, acc); break;
        default:
            // more than four rows: four at a time, in order (slots past n hold row
            // 0, which is loaded and dropped)
#pragma unroll
            for (int j0 = 0; j0 < KM; j0 += 4) {
                if (j0 < n) {
                    float v[4][V];
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        Vec<Elem, V>::load(y_perm + (int64_t)q[j0 + j] * d + col, v[j]);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int i = 0; i < V; ++i)
                            acc[i] = j0 + j < n ? fmaf(h[j0 + j], v[j][i], acc[i]) : acc[i];
                }
            }
            break;
    }
    add_shared<Elem, V>(y_shared, n_shared, T * d, t * d + col, acc);
    Vec<Elem, V>::store(y + t * d + col, acc);
}

template <typename Elem, int V, int KM>
int launch_k(const void* y_perm, const int32_t* token_row, const float* gate, const void* y_shared,
             int n_shared, int64_t T, int d, int k, void* y, hipStream_t s) {
    const int chunks = d / V;
    const int64_t blocks = ceil_div(T * chunks, COMBINE_THREADS);
    if constexpr (KM > 2) {
        if (chunks % 64 == 0) {
            hipLaunchKernelGGL((combine_compact_kernel<Elem, V, KM>), dim3((unsigned)blocks),
                               dim3(COMBINE_THREADS), 0, s, (const Elem*)y_perm, token_row, gate,
                               (const Elem*)y_shared, n_shared, T, d, k, chunks, (Elem*)y);
            return launch_status();
        }
    }
    hipLaunchKernelGGL((combine_kernel<Elem, V, KM>), dim3((unsigned)blocks), dim3(COMBINE_THREADS),
                       0, s, (const Elem*)y_perm, token_row, gate, (const Elem*)y_shared, n_shared,
                       T, d, k, chunks, (Elem*)y);
    return launch_status();
}

template <typename Elem, int V>
int launch_v(const void* y_perm, const int32_t* token_row, const float* gate, const void* y_shared,
             int n_shared, int64_t T, int d, int k, void* y, hipStream_t s) {
#define MOE_CK(KM) launch_k<Elem, V, KM>(y_perm, token_row, gate, y_shared, n_shared, T, d, k, y, s)
    if (k <= 2) return MOE_CK(2);
    if (k <= 4) return MOE_CK(4);
    if (k <= 8) return MOE_CK(8);
    return MOE_CK(MOE_MAX_K);
#undef MOE_CK
}

}  // namespace

int launch_combine(const void* y_perm, int dtype, const int32_t* token_row, const float* gate,
                   const void* y_shared, int n_shared, int64_t T, int d, int k, void* y,
                   hipStream_t s) {
    if (T == 0 || d == 0) return MOE_OK;
    if (!y_shared) n_shared = 0;
#define MOE_CV(E, V) launch_v<E, V>(y_perm, token_row, gate, y_shared, n_shared, T, d, k, y, s)
    if (dtype == MOE_BF16) return d % 8 == 0 ? MOE_CV(bf16_t, 8) : MOE_CV(bf16_t, 1);
    return d % 4 == 0 ? MOE_CV(float, 4) : MOE_CV(float, 1);
#undef MOE_CV
}

}  // namespace moe
