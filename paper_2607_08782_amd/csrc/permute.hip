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

// The k expert ids (and gates) of token t, every load issued before the first
// use: k ids behind one wait instead of k dependent round trips.  Lanes past
// k re-read id k-1 of the same row.
__device__ __forceinline__ void load_ids(const int32_t* __restrict__ idx, int64_t t, int k,
                                         int (&ev)[MOE_MAX_K]) {
#pragma unroll
    for (int r = 0; r < MOE_MAX_K; ++r) ev[r] = idx[t * k + (r < k ? r : k - 1)];
}

__device__ __forceinline__ void load_gates(const float* __restrict__ gate, int64_t t, int k,
                                           float (&gv)[MOE_MAX_K]) {
#pragma unroll
    for (int r = 0; r < MOE_MAX_K; ++r) gv[r] = gate[t * k + (r < k ? r : k - 1)];
}

// Bit `lane` of bits[s] set iff this lane's token has an assignment to local slot s.
__device__ __forceinline__ void set_bits(const int (&ev)[MOE_MAX_K], bool valid, int k, int E,
                                         const int16_t* slot_of, unsigned long long* bits,
                                         int lane) {
    if (!valid) return;
#pragma unroll
    for (int r = 0; r < MOE_MAX_K; ++r) {
        if (r >= k) break;
        const int e = ev[r];
        const int s = (unsigned)e < (unsigned)E ? (int)slot_of[e] : -1;
        if (s >= 0) atomicOr(&bits[s], 1ull << lane);
    }
}

// Rows of the replica range: of expert e's c assignments, the host of rank q
// among its n hosts takes [q c / n, (q+1) c / n).
__device__ __forceinline__ int64_t replica_lo(int q, int64_t c, int n) {
    return (int64_t)q * c / n;
}

// send_s[j] += rows GPU j receives from every expert it hosts; the counts of
// the E experts sit in cnt_s.  Integer adds, so the order does not matter.
__device__ __forceinline__ void add_send_counts(const int32_t* cnt_s, const uint64_t* hosts,
                                                int E, int tid, int nthr, int32_t* send_s) {
    for (int e = tid; e < E; e += nthr) {
        uint64_t h = hosts[e];
        const int64_t c = cnt_s[e];
        const int n = __popcll(h);
        for (int q = 0; h; ++q, h &= h - 1ull) {
            const int j = __builtin_ctzll(h);
            atomicAdd(&send_s[j], (int32_t)(replica_lo(q + 1, c, n) - replica_lo(q, c, n)));
        }
    }
}

// off[0] = 0, off[i + 1] = size[0] + ... + size[i] for i < n; one whole wave.
__device__ __forceinline__ void wave_offsets(const int32_t* size, int n, int32_t* off, int lane) {
    int32_t carry = 0;
    for (int c0 = 0; c0 < n; c0 += 64) {
        const int i = c0 + lane;
        const int32_t v = i < n ? size[i] : 0;
        int32_t incl = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int32_t u = __shfl_up(incl, o, 64);
            if (lane >= o) incl += u;
        }
        if (i < n) off[i + 1] = carry + incl;
        carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) off[0] = 0;
}

__global__ __launch_bounds__(PERM_TOKENS) void perm_count_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, SlotTable tab, int n_local,
    int32_t* __restrict__ blk_counts) {
    __shared__ unsigned long long bits[MOE_MAX_GROUPS];
    __shared__ int16_t slot_lds[MOE_MAX_E];
    const int lane = threadIdx.x;
    const int64_t blk = blockIdx.x;
    const int64_t t = blk * PERM_TOKENS + lane;
    int ev[MOE_MAX_K];
    if (t < T) load_ids(idx, t, k, ev);
    for (int e = lane; e < E; e += PERM_TOKENS) slot_lds[e] = tab.slot_of[e];
    for (int s = lane; s < n_local; s += PERM_TOKENS) bits[s] = 0ull;
    __syncthreads();
    set_bits(ev, t < T, k, E, slot_lds, bits, lane);
    __syncthreads();
    for (int s = lane; s < n_local; s += PERM_TOKENS)
        blk_counts[blk * n_local + s] = __popcll(bits[s]);
}

constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_WAVES = SCAN_THREADS / 64;
constexpr int SCAN_TILE = 8192;          // block counts staged in LDS per pass

__global__ __launch_bounds__(SCAN_THREADS) void perm_scan_kernel(
    const int32_t* __restrict__ counts, HostTable tab, int E, int n_local, int G, int dev,
    int64_t nblk, int32_t* __restrict__ blk_counts, int32_t* __restrict__ group_offsets,
    int32_t* __restrict__ lo_out, int32_t* __restrict__ send_counts) {
    __shared__ uint64_t hosts_s[MOE_MAX_E];
    __shared__ int32_t cnt_s[MOE_MAX_E];
    __shared__ int32_t size_s[MOE_MAX_GROUPS], carry_s[MOE_MAX_GROUPS];
    __shared__ int32_t send_s[MOE_MAX_G];
    __shared__ int32_t tile[SCAN_TILE];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (int e = tid; e < E; e += SCAN_THREADS) {
        cnt_s[e] = counts[e];
        hosts_s[e] = tab.hosts[e];
    }
    if (tid < MOE_MAX_G) send_s[tid] = 0;
    if (tid < MOE_MAX_GROUPS) carry_s[tid] = 0;
    __syncthreads();
    if (tid < n_local) {
        const int e = tab.expert_of_slot[tid];
        const uint64_t h = hosts_s[e];
        const int n = __popcll(h);
        const int q = dev == 0 ? 0 : __popcll(h & (~0ull >> (64 - dev)));
        const int64_t lo = replica_lo(q, cnt_s[e], n);
        size_s[tid] = (int32_t)(replica_lo(q + 1, cnt_s[e], n) - lo);
        lo_out[tid] = (int32_t)lo;
    }
    if (send_counts) add_send_counts(cnt_s, hosts_s, E, tid, SCAN_THREADS, send_s);
    __syncthreads();
    if (wave == 0) wave_offsets(size_s, n_local, group_offsets, lane);
    if (send_counts && tid < G) send_counts[tid] = send_s[tid];

    // Per-slot exclusive scan of the block counts [nblk][n_local], a tile of
    // whole block rows at a time: coalesced loads into LDS, one wave per slot
    // (each lane a run of rows), coalesced stores.
    if (n_local <= 0 || nblk <= 0) return;
    const int64_t rows_per = SCAN_TILE / n_local;
    for (int64_t r0 = 0; r0 < nblk; r0 += rows_per) {
        const int rows = (int)(nblk - r0 < rows_per ? nblk - r0 : rows_per);
        const int n = rows * n_local;
        int32_t* g = blk_counts + r0 * n_local;
        int32_t v[SCAN_TILE / SCAN_THREADS];
#pragma unroll
        for (int u = 0; u < SCAN_TILE / SCAN_THREADS; ++u) {
            const int i = u * SCAN_THREADS + tid;
            v[u] = g[i < n ? i : 0];
        }
#pragma unroll
        for (int u = 0; u < SCAN_TILE / SCAN_THREADS; ++u) tile[u * SCAN_THREADS + tid] = v[u];
        __syncthreads();
        const int per = (rows + 63) / 64;
        for (int s = wave; s < n_local; s += SCAN_WAVES) {
            const int b0 = lane * per;
            int32_t sum = 0;
            for (int i = 0; i < per; ++i)
                if (b0 + i < rows) sum += tile[(b0 + i) * n_local + s];
            int32_t incl = sum;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int32_t u = __shfl_up(incl, o, 64);
                if (lane >= o) incl += u;
            }
            int32_t run = carry_s[s] + incl - sum;
            for (int i = 0; i < per; ++i) {
                if (b0 + i < rows) {
                    int32_t* p = &tile[(b0 + i) * n_local + s];
                    const int32_t c = *p;
                    *p = run;
                    run += c;
                }
            }
            const int32_t total = __shfl(incl, 63, 64);
            if (lane == 0) carry_s[s] += total;
        }
        __syncthreads();
        for (int i = tid; i < n; i += SCAN_THREADS) g[i] = tile[i];
        __syncthreads();
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
    __shared__ int32_t base_s[MOE_MAX_GROUPS], lo_s[MOE_MAX_GROUPS], off_s[MOE_MAX_GROUPS + 1];
    const int lane = threadIdx.x;
    const int64_t blk = blockIdx.x;
    const int64_t t = blk * PERM_TOKENS + lane;
    int ev[MOE_MAX_K];
    float gv[MOE_MAX_K];
    if (t < T) {
        load_ids(idx, t, k, ev);
        load_gates(gate, t, k, gv);
    }
    for (int e = lane; e < E; e += PERM_TOKENS) slot_lds[e] = tab.slot_of[e];
    for (int s = lane; s < n_local; s += PERM_TOKENS) {
        bits[s] = 0ull;
        base_s[s] = blk_base[blk * n_local + s];
        lo_s[s] = lo_in[s];
    }
    for (int s = lane; s <= n_local; s += PERM_TOKENS) off_s[s] = group_offsets[s];
    __syncthreads();
    set_bits(ev, t < T, k, E, slot_lds, bits, lane);
    __syncthreads();
    if (t >= T) return;
    const unsigned long long lower = (1ull << lane) - 1ull;
#pragma unroll
    for (int r = 0; r < MOE_MAX_K; ++r) {
        if (r >= k) break;
        const int e = ev[r];
        int32_t p = -1;
        const int s = (unsigned)e < (unsigned)E ? (int)slot_lds[e] : -1;
        if (s >= 0) {
            const int32_t rank = base_s[s] + __popcll(bits[s] & lower);
            const int32_t lo = lo_s[s];
            if (rank >= lo && rank < lo + (off_s[s + 1] - off_s[s])) {
                p = off_s[s] + (rank - lo);
                row_token[p] = (int32_t)t;
                row_gate[p] = gv[r];
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
    __shared__ uint64_t hosts_s[MOE_MAX_E];
    __shared__ int32_t cnt_s[MOE_MAX_E], send_s[MOE_MAX_G];
    __shared__ int32_t lo_s[MOE_MAX_GROUPS], size_s[MOE_MAX_GROUPS], off_s[MOE_MAX_GROUPS + 1];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nblk = (int)ceil_div(T, PERM_TOKENS);
    const int64_t t = (int64_t)wave * PERM_TOKENS + lane;
    int ev[MOE_MAX_K];
    float gv[MOE_MAX_K];
    if (t < T) {
        load_ids(idx, t, k, ev);
        load_gates(gate, t, k, gv);
    }
    for (int e = tid; e < E; e += SMALL_T) {
        slot_lds[e] = st.slot_of[e];
        cnt_s[e] = counts[e];
        hosts_s[e] = ht.hosts[e];
    }
    if (tid < MOE_MAX_G) send_s[tid] = 0;
    for (int i = tid; i < SMALL_BLK * MOE_MAX_GROUPS; i += SMALL_T)
        bits[i / MOE_MAX_GROUPS][i % MOE_MAX_GROUPS] = 0ull;
    __syncthreads();
    set_bits(ev, t < T, k, E, slot_lds, bits[wave], lane);
    if (send_counts) add_send_counts(cnt_s, hosts_s, E, tid, SMALL_T, send_s);
    __syncthreads();
    if (tid < n_local) {
        int32_t run = 0;
        for (int b = 0; b < nblk; ++b) {
            base[b][tid] = run;
            run += __popcll(bits[b][tid]);
        }
        const int e = ht.expert_of_slot[tid];
        const uint64_t h = hosts_s[e];
        const int n = __popcll(h);
        const int q = dev == 0 ? 0 : __popcll(h & (~0ull >> (64 - dev)));
        const int64_t lo = replica_lo(q, cnt_s[e], n);
        lo_s[tid] = (int32_t)lo;
        size_s[tid] = (int32_t)(replica_lo(q + 1, cnt_s[e], n) - lo);
    }
    if (send_counts && tid < G) send_counts[tid] = send_s[tid];
    __syncthreads();
    if (wave == 0) wave_offsets(size_s, n_local, off_s, lane);
    __syncthreads();
    for (int sl = tid; sl <= n_local; sl += SMALL_T) group_offsets[sl] = off_s[sl];
    if (t >= T) return;
    const unsigned long long lower = (1ull << lane) - 1ull;
#pragma unroll
    for (int r = 0; r < MOE_MAX_K; ++r) {
        if (r >= k) break;
        const int e = ev[r];
        int32_t p = -1;
        const int sl = (unsigned)e < (unsigned)E ? (int)slot_lds[e] : -1;
        if (sl >= 0) {
            const int32_t rank = base[wave][sl] + __popcll(bits[wave][sl] & lower);
            const int32_t lo = lo_s[sl];
            if (rank >= lo && rank < lo + size_s[sl]) {
                p = off_s[sl] + (rank - lo);
                row_token[p] = (int32_t)t;
                row_gate[p] = gv[r];
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

// Scratch of moe_permute_noalloc: the per-block slot counts and replica
// offsets that moe_permute keeps in the caller's workspace, held instead in a
// device array of this library (one copy per GPU, kept until the process
// ends).  Every byte the kernels read is written earlier in the same call, so
// nothing needs clearing; calls that overlap on one GPU race on it.
static __device__ __align__(256) unsigned char scratch[MOE_PERMUTE_NOALLOC_MAX_WS];

}  // namespace

// Device address of `scratch` on the current device.  The array's name in host
// code is a host-side stand-in, not a device address, so the address is looked
// up once per device, with that device current, and kept.
int permute_scratch(void** ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex lock;
    static void* addr[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MOE_ERR_DEVICE;
    std::lock_guard<std::mutex> guard(lock);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return MOE_ERR_DEVICE;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return MOE_OK;
}

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
        hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(SCAN_THREADS), 0, s, counts, ht, E, n_local, G,
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
