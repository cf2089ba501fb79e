// Per-expert workload counts and co-activation counts (Sec. VI-A of the
// Director paper: W counts the tokens routed to each expert and drives the
// per-GPU load of Eq. 1; co-activation is the signal for co-locating experts
// that fire together, Sec. I).
//
// Integer atomics only, so the result does not depend on scheduling: each
// workgroup accumulates in LDS, then adds its non-zero bins to global memory.
#include "common.h"

namespace moe {
namespace {

constexpr int HIST_THREADS = 256;
constexpr int LDS_COACT_MAX_E = 128;     // E*E int32 bins fit in 64 KiB of LDS
constexpr int DIRECT_MAX_TOKENS = 512;   // up to this many tokens one workgroup does it all

// Clears a[0..na) and b[0..nb) in one launch (b may be null).
__global__ void zero_i32_kernel(int32_t* __restrict__ a, int64_t na, int32_t* __restrict__ b,
                                int64_t nb) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < na + nb;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i < na) a[i] = 0;
        else b[i - na] = 0;
    }
}

// DIRECT: a single workgroup covers all tokens and stores its bins (zeros
// included), so the outputs need no clearing launch beforehand.
template <bool COACT, bool LDS_COACT, bool DIRECT = false>
__global__ __launch_bounds__(HIST_THREADS) void histogram_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, int32_t* __restrict__ counts,
    int32_t* __restrict__ coact) {
    __shared__ int32_t c_lds[MOE_MAX_E];
    extern __shared__ int32_t co_lds[];          // [E][E] when LDS_COACT
    for (int i = threadIdx.x; i < E; i += HIST_THREADS) c_lds[i] = 0;
    if (LDS_COACT)
        for (int i = threadIdx.x; i < E * E; i += HIST_THREADS) co_lds[i] = 0;
    __syncthreads();

    for (int64_t t = (int64_t)blockIdx.x * HIST_THREADS + threadIdx.x; t < T;
         t += (int64_t)gridDim.x * HIST_THREADS) {
        const int32_t* row = idx + t * k;
        int sel[MOE_MAX_K];
#pragma unroll
        for (int r = 0; r < MOE_MAX_K; ++r) {
            // out-of-range indices are ignored rather than written out of bounds
            if (r < k) sel[r] = row[r];
            if (r < k && (unsigned)sel[r] >= (unsigned)E) sel[r] = -1;
        }
#pragma unroll
        for (int r = 0; r < MOE_MAX_K; ++r) {
            if (r >= k) break;
            if (sel[r] < 0) continue;
            atomicAdd(&c_lds[sel[r]], 1);
            if (COACT) {
#pragma unroll
                for (int q = 0; q < MOE_MAX_K; ++q) {
                    if (q >= k) break;
                    if (sel[q] < 0) continue;
                    if (LDS_COACT) atomicAdd(&co_lds[sel[r] * E + sel[q]], 1);
                    else atomicAdd(&coact[(int64_t)sel[r] * E + sel[q]], 1);
                }
            }
        }
    }
    __syncthreads();
    if (DIRECT) {
        for (int i = threadIdx.x; i < E; i += HIST_THREADS) counts[i] = c_lds[i];
        if (LDS_COACT)
            for (int i = threadIdx.x; i < E * E; i += HIST_THREADS) coact[i] = co_lds[i];
        return;
    }
    for (int i = threadIdx.x; i < E; i += HIST_THREADS)
        if (c_lds[i]) atomicAdd(&counts[i], c_lds[i]);
    if (LDS_COACT)
        for (int i = threadIdx.x; i < E * E; i += HIST_THREADS)
            if (co_lds[i]) atomicAdd(&coact[i], co_lds[i]);
}

// Counts only, up to HF_MAX entries (T*k) in one workgroup: entry e = tid + j*1024
// (coalesced, all sixteen loads of a thread issued together from clamped
// indices), per-wave bins in LDS (atomics contend only within a wave), then the
// waves' bins summed and stored directly: one launch, no clearing pass.
constexpr int HF_THREADS = 1024;
constexpr int HF_PER = 16;
constexpr int HF_MAX = HF_THREADS * HF_PER;

__global__ __launch_bounds__(HF_THREADS) void histogram_flat_kernel(const int32_t* __restrict__ idx,
                                                                   int n, int E,
                                                                   int32_t* __restrict__ counts) {
    __shared__ int32_t bins[HF_THREADS / 64][MOE_MAX_E];
    const int tid = threadIdx.x, wave = tid >> 6;
    for (int i = tid; i < (HF_THREADS / 64) * MOE_MAX_E; i += HF_THREADS) (&bins[0][0])[i] = 0;
    int v[HF_PER];
#pragma unroll
    for (int j = 0; j < HF_PER; ++j) {
        const int e = tid + j * HF_THREADS;
        v[j] = idx[e < n ? e : 0];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < HF_PER; ++j) {
        const int e = tid + j * HF_THREADS;
        // out-of-range expert ids are ignored rather than counted out of bounds
        if (e < n && (unsigned)v[j] < (unsigned)E) atomicAdd(&bins[wave][v[j]], 1);
    }
    __syncthreads();
    for (int i = tid; i < E; i += HF_THREADS) {
        int c = 0;
#pragma unroll
        for (int w = 0; w < HF_THREADS / 64; ++w) c += bins[w][i];
        counts[i] = c;
    }
}

// Short batches with co-activation (T <= DIRECT_MAX_TOKENS, E <= LDS_COACT_MAX_E):
// one 1024-thread workgroup, E*E bins in LDS cleared and stored 16 bytes at a
// time; thread i takes assignment (t, r) = (i / k, i % k), loads the token's k
// ids together (KM = k rounded up to a power of two, compile-time) and adds row
// r of the token's k x k co-activation block.
constexpr int HD_THREADS = 1024;

template <int KM>
__global__ __launch_bounds__(HD_THREADS) void histogram_coact_direct_kernel(
    const int32_t* __restrict__ idx, int T, int k, int E, int32_t* __restrict__ counts,
    int32_t* __restrict__ coact) {
    extern __shared__ __attribute__((aligned(16))) int32_t co_lds[];   // [E][E]
    __shared__ int32_t c_lds[MOE_MAX_E];
    const int tid = threadIdx.x;
    const int nb = E * E;
    const int n4 = nb >> 2;
    for (int i = tid; i < n4; i += HD_THREADS) ((int4*)co_lds)[i] = make_int4(0, 0, 0, 0);
    for (int i = (n4 << 2) + tid; i < nb; i += HD_THREADS) co_lds[i] = 0;
    for (int i = tid; i < E; i += HD_THREADS) c_lds[i] = 0;
    __syncthreads();
    for (int a = tid; a < T * k; a += HD_THREADS) {
        const int t = a / k, r = a - t * k;
        int sel[KM];
#pragma unroll
        for (int q = 0; q < KM; ++q) sel[q] = idx[(int64_t)t * k + (q < k ? q : k - 1)];
        int e = sel[0];
#pragma unroll
        for (int q = 1; q < KM; ++q) e = q == r ? sel[q] : e;
        // out-of-range expert ids are ignored rather than counted out of bounds
        if ((unsigned)e >= (unsigned)E) continue;
        atomicAdd(&c_lds[e], 1);
#pragma unroll
        for (int q = 0; q < KM; ++q)
            if (q < k && (unsigned)sel[q] < (unsigned)E) atomicAdd(&co_lds[e * E + sel[q]], 1);
    }
    __syncthreads();
    if (((uintptr_t)coact & 15) == 0) {
        for (int i = tid; i < n4; i += HD_THREADS) ((int4*)coact)[i] = ((const int4*)co_lds)[i];
        for (int i = (n4 << 2) + tid; i < nb; i += HD_THREADS) coact[i] = co_lds[i];
    } else {
        for (int i = tid; i < nb; i += HD_THREADS) coact[i] = co_lds[i];
    }
    for (int i = tid; i < E; i += HD_THREADS) counts[i] = c_lds[i];
}

}  // namespace

int launch_histogram(const int32_t* idx, int64_t T, int k, int E, int32_t* counts, int32_t* coact,
                     hipStream_t s) {
    // counts of up to HF_MAX assignments: one workgroup, one launch
    if (!coact && T > 0 && T * k <= HF_MAX) {
        hipLaunchKernelGGL(histogram_flat_kernel, dim3(1), dim3(HF_THREADS), 0, s, idx,
                           (int)(T * k), E, counts);
        return launch_status();
    }
    // short batches (decode): one workgroup, bins stored directly, one launch
    if (T <= DIRECT_MAX_TOKENS && (!coact || E <= LDS_COACT_MAX_E)) {
        if (coact) {
            if (T == 0) {
                hipLaunchKernelGGL(zero_i32_kernel, dim3((unsigned)ceil_div((int64_t)E * (E + 1), 256)),
                                   dim3(256), 0, s, counts, (int64_t)E, coact, (int64_t)E * E);
                return launch_status();
            }
            const size_t lds = (size_t)E * E * sizeof(int32_t);
#define HD(KM) hipLaunchKernelGGL((histogram_coact_direct_kernel<KM>), dim3(1), dim3(HD_THREADS), \
                                  lds, s, idx, (int)T, k, E, counts, coact)
            if (k <= 2) HD(2);
            else if (k <= 4) HD(4);
            else if (k <= 8) HD(8);
            else HD(MOE_MAX_K);
#undef HD
        } else
            hipLaunchKernelGGL((histogram_kernel<false, false, true>), dim3(1), dim3(HIST_THREADS),
                               0, s, idx, T, k, E, counts, coact);
        return launch_status();
    }
    const int64_t ncoact = coact ? (int64_t)E * E : 0;
    int64_t zblocks = ceil_div((int64_t)E + ncoact, 256);
    if (zblocks > 1024) zblocks = 1024;
    hipLaunchKernelGGL(zero_i32_kernel, dim3((unsigned)zblocks), dim3(256), 0, s, counts,
                       (int64_t)E, coact, ncoact);
    if (T == 0) return launch_status();
    int64_t blocks = ceil_div(T, HIST_THREADS);
    if (!coact) {
        if (blocks > 512) blocks = 512;
        hipLaunchKernelGGL((histogram_kernel<false, false>), dim3((unsigned)blocks),
                           dim3(HIST_THREADS), 0, s, idx, T, k, E, counts, coact);
    } else if (E <= LDS_COACT_MAX_E) {
        // 64 workgroups: each flushes its non-zero E*E bins with global atomics, so
        // more workgroups add flush traffic (Qwen3-shaped prefill: 16 -> 25.1 us,
        // 32 -> 17.7, 64 -> 14.4, 128 and 256 -> 14.5, with the clearing launch)
        if (blocks > 64) blocks = 64;
        const size_t lds = (size_t)E * E * sizeof(int32_t);
        hipLaunchKernelGGL((histogram_kernel<true, true>), dim3((unsigned)blocks),
                           dim3(HIST_THREADS), lds, s, idx, T, k, E, counts, coact);
    } else {
        if (blocks > 512) blocks = 512;
        hipLaunchKernelGGL((histogram_kernel<true, false>), dim3((unsigned)blocks),
                           dim3(HIST_THREADS), 0, s, idx, T, k, E, counts, coact);
    }
    return launch_status();
}

}  // namespace moe
