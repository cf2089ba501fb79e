// Packaging of tokens for the experts placed on this GPU (Sec. II-B of the
// Director paper: tokens are packaged and sent to the GPUs that host their
// experts; Sec. VI-A: placement x[e][j], Eq. 1 load and Eq. 3 volume).
//
// A stable counting sort of the T*k assignments into local-expert groups,
// with no host round trip:
//   count    one wave per 64 tokens: per-slot membership bitmaps in LDS,
//            popcounts -> per-block counts
//   scan     one workgroup: replica ranges [lo, hi) per slot from the global
//            counts, group offsets, per-slot exclusive scan over blocks,
//            send counts per GPU
//   scatter  one wave per 64 tokens: rank = block base + popcount of the
//            lower lanes' bits; kept ranks get a row
//   gather   x_perm[p] = x[row_token[p]], 16-byte vector copies
// Every step is integer arithmetic, so the result is exact and unique.
#include "common.h"

namespace moe {
namespace {

constexpr int PERM_TOKENS = 64;          // one wave per block of 64 tokens

struct SlotTable {
    int16_t slot_of[MOE_MAX_E];
};

struct HostTable {
    uint64_t hosts[MOE_MAX_E];
    int16_t expert_of_slot[MOE_MAX_GROUPS];
};

__device__ __forceinline__ void build_bits(const int32_t* __restrict__ idx, int64_t T, int k, int E,
                                           const int16_t* __restrict__ slot_of, int n_local,
                                           unsigned long long* bits, int lane, int64_t t) {
    for (int s = lane; s < n_local; s += PERM_TOKENS) bits[s] = 0ull;
    __syncthreads();
    if (t < T) {
        for (int r = 0; r < k; ++r) {
            const int e = idx[t * k + r];
            if ((unsigned)e >= (unsigned)E) continue;
            const int s = slot_of[e];
            if (s >= 0) atomicOr(&bits[s], 1ull << lane);
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(PERM_TOKENS) void perm_count_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, SlotTable tab, int n_local,
    int32_t* __restrict__ blk_counts) {
    __shared__ unsigned long long bits[MOE_MAX_GROUPS];
    __shared__ int16_t slot_lds[MOE_MAX_E];
    const int lane = threadIdx.x;
    for (int e = lane; e < E; e += PERM_TOKENS) slot_lds[e] = tab.slot_of[e];
    const int64_t blk = blockIdx.x;
    build_bits(idx, T, k, E, slot_lds, n_local, bits, lane, blk * PERM_TOKENS + lane);
    for (int s = lane; s < n_local; s += PERM_TOKENS)
        blk_counts[blk * n_local + s] = __popcll(bits[s]);
}

__global__ __launch_bounds__(256) void perm_scan_kernel(
    const int32_t* __restrict__ counts, HostTable tab, int E, int n_local, int G, int dev,
    int64_t nblk, int32_t* __restrict__ blk_counts, int32_t* __restrict__ group_offsets,
    int32_t* __restrict__ lo_out, int32_t* __restrict__ send_counts) {
    __shared__ int32_t size_s[MOE_MAX_GROUPS];
    const int tid = threadIdx.x;
    const uint64_t below = dev == 0 ? 0ull : (~0ull >> (64 - dev));
    if (tid < n_local) {
        const int e = tab.expert_of_slot[tid];
        const int64_t c = counts[e];
        const uint64_t h = tab.hosts[e];
        const int n = __popcll(h);
        const int q = __popcll(h & below);
        const int64_t lo = (int64_t)q * c / n;
        const int64_t hi = (int64_t)(q + 1) * c / n;
        size_s[tid] = (int32_t)(hi - lo);
        lo_out[tid] = (int32_t)lo;
    }
    if (send_counts && tid < G) {
        const uint64_t below_j = tid == 0 ? 0ull : (~0ull >> (64 - tid));
        int64_t sum = 0;
        for (int e = 0; e < E; ++e) {
            const uint64_t h = tab.hosts[e];
            if (!((h >> tid) & 1ull)) continue;
            const int64_t c = counts[e];
            const int n = __popcll(h);
            const int q = __popcll(h & below_j);
            sum += (int64_t)(q + 1) * c / n - (int64_t)q * c / n;
        }
        send_counts[tid] = (int32_t)sum;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t run = 0;
        group_offsets[0] = 0;
        for (int s = 0; s < n_local; ++s) {
            run += size_s[s];
            group_offsets[s + 1] = run;
        }
    }
    // per-slot exclusive scan of block counts, one wave per slot at a time
    const int wave = tid >> 6, lane = tid & 63;
    for (int s = wave; s < n_local; s += 4) {
        int32_t running = 0;
        for (int64_t c0 = 0; c0 < nblk; c0 += 64) {
            const int64_t b = c0 + lane;
            const int32_t v = b < nblk ? blk_counts[b * n_local + s] : 0;
            int32_t incl = v;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int32_t u = __shfl_up(incl, o, 64);
                if (lane >= o) incl += u;
            }
            if (b < nblk) blk_counts[b * n_local + s] = running + incl - v;
            running += __shfl(incl, 63, 64);
        }
    }
}

__global__ __launch_bounds__(PERM_TOKENS) void perm_scatter_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ gate, int64_t T, int k, int E,
    SlotTable tab, int n_local, const int32_t* __restrict__ blk_base,
    const int32_t* __restrict__ lo_in, const int32_t* __restrict__ group_offsets,
    int32_t* __restrict__ row_token, float* __restrict__ row_gate,
    int32_t* __restrict__ token_row) {
    __shared__ unsigned long long bits[MOE_MAX_GROUPS];
    __shared__ int16_t slot_lds[MOE_MAX_E];
    const int lane = threadIdx.x;
    for (int e = lane; e < E; e += PERM_TOKENS) slot_lds[e] = tab.slot_of[e];
    const int64_t blk = blockIdx.x;
    const int64_t t = blk * PERM_TOKENS + lane;
    build_bits(idx, T, k, E, slot_lds, n_local, bits, lane, t);
    if (t >= T) return;
    const unsigned long long lower = (1ull << lane) - 1ull;
    for (int r = 0; r < k; ++r) {
        const int e = idx[t * k + r];
        int32_t p = -1;
        const int s = (unsigned)e < (unsigned)E ? (int)slot_lds[e] : -1;
        if (s >= 0) {
            const int32_t rank = blk_base[blk * n_local + s] + __popcll(bits[s] & lower);
            const int32_t lo = lo_in[s];
            const int32_t off = group_offsets[s];
            const int32_t size = group_offsets[s + 1] - off;
            if (rank >= lo && rank < lo + size) {
                p = off + (rank - lo);
                row_token[p] = (int32_t)t;
                row_gate[p] = gate[t * k + r];
            }
        }
        token_row[t * k + r] = p;
    }
}

// Short batches (at most SMALL_T tokens): count, scan and scatter in one
// workgroup, one wave per 64-token block, the same arithmetic as the three
// kernels above (so the same unique result), one launch instead of three.
constexpr int SMALL_T = 1024;
constexpr int SMALL_BLK = SMALL_T / PERM_TOKENS;

__global__ __launch_bounds__(SMALL_T) void perm_small_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ gate,
    const int32_t* __restrict__ counts, int64_t T, int k, int E, SlotTable st, HostTable ht,
    int n_local, int G, int dev, int32_t* __restrict__ group_offsets,
    int32_t* __restrict__ row_token, float* __restrict__ row_gate, int32_t* __restrict__ token_row,
    int32_t* __restrict__ send_counts) {
    __shared__ unsigned long long bits[SMALL_BLK][MOE_MAX_GROUPS];
    __shared__ int32_t base[SMALL_BLK][MOE_MAX_GROUPS];
    __shared__ int16_t slot_lds[MOE_MAX_E];
    __shared__ int32_t lo_s[MOE_MAX_GROUPS], size_s[MOE_MAX_GROUPS], off_s[MOE_MAX_GROUPS + 1];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nblk = (int)ceil_div(T, PERM_TOKENS);
    for (int e = tid; e < E; e += SMALL_T) slot_lds[e] = st.slot_of[e];
    for (int i = tid; i < SMALL_BLK * MOE_MAX_GROUPS; i += SMALL_T)
        bits[i / MOE_MAX_GROUPS][i % MOE_MAX_GROUPS] = 0ull;
    __syncthreads();
    const int64_t t = (int64_t)wave * PERM_TOKENS + lane;
    if (t < T) {
        for (int r = 0; r < k; ++r) {
            const int e = idx[t * k + r];
            if ((unsigned)e >= (unsigned)E) continue;
            const int sl = slot_lds[e];
            if (sl >= 0) atomicOr(&bits[wave][sl], 1ull << lane);
        }
    }
    __syncthreads();
    const uint64_t below = dev == 0 ? 0ull : (~0ull >> (64 - dev));
    if (tid < n_local) {
        int32_t run = 0;
        for (int b = 0; b < nblk; ++b) {
            base[b][tid] = run;
            run += __popcll(bits[b][tid]);
        }
        const int e = ht.expert_of_slot[tid];
        const int64_t c = counts[e];
        const uint64_t h = ht.hosts[e];
        const int n = __popcll(h);
        const int q = __popcll(h & below);
        const int64_t lo = (int64_t)q * c / n;
        lo_s[tid] = (int32_t)lo;
        size_s[tid] = (int32_t)((int64_t)(q + 1) * c / n - lo);
    }
    if (send_counts && tid >= SMALL_T - 64 && tid - (SMALL_T - 64) < G) {
        const int j = tid - (SMALL_T - 64);
        const uint64_t below_j = j == 0 ? 0ull : (~0ull >> (64 - j));
        int64_t sum = 0;
        for (int e = 0; e < E; ++e) {
            const uint64_t h = ht.hosts[e];
            if (!((h >> j) & 1ull)) continue;
            const int64_t c = counts[e];
            const int n = __popcll(h);
            const int q = __popcll(h & below_j);
            sum += (int64_t)(q + 1) * c / n - (int64_t)q * c / n;
        }
        send_counts[j] = (int32_t)sum;
    }
    __syncthreads();
    if (tid == 0) {
        int32_t run = 0;
        off_s[0] = 0;
        for (int sl = 0; sl < n_local; ++sl) {
            run += size_s[sl];
            off_s[sl + 1] = run;
        }
    }
    __syncthreads();
    for (int sl = tid; sl <= n_local; sl += SMALL_T) group_offsets[sl] = off_s[sl];
    if (t >= T) return;
    const unsigned long long lower = (1ull << lane) - 1ull;
    for (int r = 0; r < k; ++r) {
        const int e = idx[t * k + r];
        int32_t p = -1;
        const int sl = (unsigned)e < (unsigned)E ? (int)slot_lds[e] : -1;
        if (sl >= 0) {
            const int32_t rank = base[wave][sl] + __popcll(bits[wave][sl] & lower);
            const int32_t lo = lo_s[sl];
            if (rank >= lo && rank < lo + size_s[sl]) {
                p = off_s[sl] + (rank - lo);
                row_token[p] = (int32_t)t;
                row_gate[p] = gate[t * k + r];
            }
        }
        token_row[t * k + r] = p;
    }
}

template <typename U>
__global__ __launch_bounds__(256) void gather_rows_kernel(
    const U* __restrict__ x, const int32_t* __restrict__ row_token,
    const int32_t* __restrict__ total, int units_per_row, U* __restrict__ x_perm) {
    const int32_t N = *total;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int64_t p = (int64_t)blockIdx.x * 4 + wave; p < N; p += (int64_t)gridDim.x * 4) {
        const int64_t t = row_token[p];
        const U* src = x + t * units_per_row;
        U* dst = x_perm + p * units_per_row;
        for (int u = lane; u < units_per_row; u += 64) dst[u] = src[u];
    }
}

}  // namespace

size_t permute_ws_bytes(int64_t T, int k, int E) {
    (void)k;
    const int64_t nblk = ceil_div(T, PERM_TOKENS);
    const int64_t slots = E < MOE_MAX_GROUPS ? E : MOE_MAX_GROUPS;
    return (size_t)(nblk * slots + MOE_MAX_GROUPS) * sizeof(int32_t) + 256;
}

int launch_permute(const void* x, int dtype, const int32_t* idx, const float* gate,
                   const int32_t* counts, int64_t T, int d, int k, int E, const PermuteTables& tabs,
                   int n_local, int G, int dev, void* x_perm, int64_t cap_rows,
                   int32_t* group_offsets, int32_t* row_token, float* row_gate, int32_t* token_row,
                   int32_t* send_counts, void* ws, hipStream_t s) {
    const int64_t nblk = ceil_div(T, PERM_TOKENS);
    int32_t* lo_ws = (int32_t*)ws;
    int32_t* blk = lo_ws + MOE_MAX_GROUPS;
    SlotTable st;
    HostTable ht;
    for (int e = 0; e < MOE_MAX_E; ++e) {
        st.slot_of[e] = tabs.slot_of[e];
        ht.hosts[e] = tabs.hosts[e];
    }
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) ht.expert_of_slot[i] = tabs.expert_of_slot[i];

    if (T <= SMALL_T) {
        hipLaunchKernelGGL(perm_small_kernel, dim3(1), dim3(SMALL_T), 0, s, idx, gate, counts, T, k,
                           E, st, ht, n_local, G, dev, group_offsets, row_token, row_gate,
                           token_row, send_counts);
    } else {
        if (n_local > 0)
            hipLaunchKernelGGL(perm_count_kernel, dim3((unsigned)nblk), dim3(PERM_TOKENS), 0, s,
                               idx, T, k, E, st, n_local, blk);
        hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(256), 0, s, counts, ht, E, n_local, G,
                           dev, n_local > 0 ? nblk : (int64_t)0, blk, group_offsets, lo_ws,
                           send_counts);
        hipLaunchKernelGGL(perm_scatter_kernel, dim3((unsigned)nblk), dim3(PERM_TOKENS), 0, s,
                           idx, gate, T, k, E, st, n_local, blk, lo_ws, group_offsets, row_token,
                           row_gate, token_row);
    }
    if (nblk > 0 && n_local > 0 && d > 0) {
        const size_t row_bytes = (size_t)d * (dtype == MOE_BF16 ? 2 : 4);
        int64_t max_rows = cap_rows;
        if (max_rows > T * (int64_t)k) max_rows = T * (int64_t)k;
        int64_t blocks = ceil_div(max_rows, 4);
        if (blocks > 4096) blocks = 4096;
        if (blocks < 1) blocks = 1;
        const int32_t* total = group_offsets + n_local;
        if (row_bytes % 16 == 0)
            hipLaunchKernelGGL(gather_rows_kernel<uint4>, dim3((unsigned)blocks), dim3(256), 0, s,
                               (const uint4*)x, row_token, total, (int)(row_bytes / 16),
                               (uint4*)x_perm);
        else if (row_bytes % 4 == 0)
            hipLaunchKernelGGL(gather_rows_kernel<uint32_t>, dim3((unsigned)blocks), dim3(256), 0,
                               s, (const uint32_t*)x, row_token, total, (int)(row_bytes / 4),
                               (uint32_t*)x_perm);
        else
            hipLaunchKernelGGL(gather_rows_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0,
                               s, (const uint16_t*)x, row_token, total, (int)(row_bytes / 2),
                               (uint16_t*)x_perm);
    }
    return launch_status();
}

}  // namespace moe
