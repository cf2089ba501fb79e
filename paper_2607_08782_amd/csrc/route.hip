// Gate scores and top-k routing (Sec. II-A of the Director paper: the gating
// network scores each expert for every token and the token is sent to the k
// best; the gate is replicated on every GPU, Sec. II-B).
//
// Each workgroup owns a block of tokens:
//   phase 1  scores for its tokens x all E experts into LDS
//            bf16: MFMA 16x16x32, K split over 16 waves, fixed-order reduction
//            (long batches over more than 32 experts use the tiled kernel of
//            score.hip instead; short batches over more than 16 experts the
//            per-wave partial tiles of route_wave_kernel, summed in a second
//            launch with the top-k);
//            f32:  plain FMA loops;  logits-in: read in place from global memory
//   phase 2  bias added, scores written back coalesced (if requested)
//   phase 3  a group of lanes per token: k rounds of a group-wide maximum, gates.
#include "common.h"
#include "topk.h"

namespace moe {
namespace {

constexpr int ROUTE_THREADS = TOPK_THREADS;
constexpr int ROUTE_MAX_SPLIT = 32;    // K chunks of the split score kernel

enum RouteMode { MODE_F32 = 1, MODE_LOGITS_IN = 2, MODE_PARTIALS = 3 };

}  // namespace
int route_split(int64_t T, int d, int E);
namespace {

// bf16 gate scores on MFMA 16x16x32.  A workgroup of 16 waves owns 16*RT
// tokens; wave w takes the K steps w, w+16, w+32, ... (32 elements each) for
// all RT token tiles and up to NTM expert tiles, with operand fragments loaded
// straight from global memory (the router matrix stays L2-resident), two K
// steps of loads in flight per wave.  Partial scores are reduced in LDS in a fixed order
// (four slices, each summed over its four waves in turn, then the slices in
// turn), so the scores are deterministic.
constexpr int RB_WAVES = 16;
constexpr int RB_THREADS = RB_WAVES * 64;
constexpr uint32_t RB_RSRC_WORD3 = 0x00020000;     // raw buffer, 32-bit data format
constexpr int RB_OOB = 0x7ffffff0;                 // an offset past every descriptor's range

__device__ __forceinline__ uint4 rb_load16(__amdgpu_buffer_rsrc_t r, int voff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

template <int RT, int NTM, int KM, int C>
__global__ __launch_bounds__(RB_THREADS) void route_bf16_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, const float* __restrict__ bias,
    int64_t T, int d, int E, int k, int renorm, float* __restrict__ logits,
    int32_t* __restrict__ idx, float* __restrict__ gate, int S, float* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    constexpr int ROWS = 16 * RT;
    const int E_pad = (E + 15) & ~15;
    const int ldS = E_pad + 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * ROWS;
    const int nt = (int)((T - t0) < ROWS ? (T - t0) : ROWS);
    const int NT = E_pad / 16;
    const int row = lane & 15, kq = (lane >> 4) * 8;

    // operands through buffer descriptors: rows past the block's tokens or past E
    // fall outside them and read as zero, and a masked lane (K past d, a tile past
    // the experts) gets an offset outside them too, so every load is issued
    // unconditionally and the compiler can keep several in flight
    const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(X + t0 * d), (short)0, nt * d * 2, RB_RSRC_WORD3);
    const __amdgpu_buffer_rsrc_t wrsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)W, (short)0, E * d * 2, RB_RSRC_WORD3);
    int xoff[RT], woff[NTM];
#pragma unroll
    for (int i = 0; i < RT; ++i) xoff[i] = ((i * 16 + row) * d + kq) * 2;
#pragma unroll
    for (int j = 0; j < NTM; ++j) woff[j] = ((j * 16 + row) * d + kq) * 2;   // j >= NT: rows >= E
    f32x4 acc[RT][NTM];
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
        for (int j = 0; j < NTM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // K chunk of this workgroup (blockIdx.y of S): steps [sbeg, send), 32 elements each
    const int nsteps_all = (d + 31) / 32;
    const int chunk = blockIdx.y;
    const int sbeg = (int)((int64_t)chunk * nsteps_all / S);
    const int send = (int)((int64_t)(chunk + 1) * nsteps_all / S);
    const int nsteps = send - sbeg;
    if (NTM <= 4) {
        // all tiles' fragments of one K step fit in registers: keep two steps of
        // loads in flight (ring of two register sets, alternating by step parity).
        // Loads past this wave's last step get out-of-range offsets (zeros, no
        // memory traffic), so the loop has no branches and the waits are exact.
        uint4 av[2][RT], bv[2][NTM];
        const int n_mine = wave < nsteps ? (nsteps - wave + RB_WAVES - 1) / RB_WAVES : 0;
        const int s0 = sbeg + wave;
        auto load = [&](int i, uint4* a_, uint4* b_) {
            const int k0 = (s0 + i * RB_WAVES) * 32;
            const bool kin = i < n_mine && k0 + kq < d;
#pragma unroll
            for (int r = 0; r < RT; ++r) a_[r] = rb_load16(xrsrc, kin ? xoff[r] + k0 * 2 : RB_OOB);
#pragma unroll
            for (int j = 0; j < NTM; ++j) b_[j] = rb_load16(wrsrc, kin ? woff[j] + k0 * 2 : RB_OOB);
        };
        // every tile, also those past the experts (their operands read as zero):
        // a branch here would make the compiler wait for every load in flight
        auto mma = [&](const uint4* a_, const uint4* b_) {
#pragma unroll
            for (int i = 0; i < RT; ++i)
#pragma unroll
                for (int j = 0; j < NTM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, a_[i]), __builtin_bit_cast(bf16x8, b_[j]),
                        acc[i][j], 0, 0, 0);
        };
        load(0, av[0], bv[0]);
        load(1, av[1], bv[1]);
        for (int i = 0; i < n_mine; i += 2) {
            mma(av[0], bv[0]);
            load(i + 2, av[0], bv[0]);
            mma(av[1], bv[1]);                    // zeros when i + 1 == n_mine
            load(i + 3, av[1], bv[1]);
        }
    } else {
        for (int step = sbeg + wave; step < send; step += RB_WAVES) {
            const int k0 = step * 32;
            const bool kin = k0 + kq < d;
            bf16x8 a[RT];
#pragma unroll
            for (int i = 0; i < RT; ++i)
                a[i] = __builtin_bit_cast(bf16x8, rb_load16(xrsrc, kin ? xoff[i] + k0 * 2 : RB_OOB));
#pragma unroll
            for (int jc = 0; jc < NTM; jc += 4) {
                if (jc >= NT) break;
                bf16x8 b[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    b[jj] = __builtin_bit_cast(bf16x8,
                                               rb_load16(wrsrc, kin ? woff[jc + jj] + k0 * 2 : RB_OOB));
#pragma unroll
                for (int i = 0; i < RT; ++i)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
                        if (jc + jj < NT)
                            acc[i][jc + jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                a[i], b[jj], acc[i][jc + jj], 0, 0, 0);
            }
        }
    }

    // fixed-order reduction in the MFMA output layout (one 16-byte LDS access per
    // tile and lane): slice g = wave & 3 receives waves g, g+4, g+8, g+12 in turn,
    // the four slices are added in order into slice 0, and the sums are laid out
    // row-major (over slices 1..3) for the epilogue.
    const int g = wave & 3, q = wave >> 2;
    const int nslice = ROWS * E_pad;                  // floats per slice
    f32x4* Sg = (f32x4*)smem + g * (nslice / 4);
    for (int pass = 0; pass < 4; ++pass) {
        if (q == pass) {
#pragma unroll
            for (int i = 0; i < RT; ++i)
#pragma unroll
                for (int j = 0; j < NTM; ++j) {
                    if (j >= NT) continue;
                    f32x4* p = Sg + (i * NT + j) * 64 + lane;
                    *p = pass == 0 ? acc[i][j] : *p + acc[i][j];
                }
        }
        __syncthreads();
    }
    {
        f32x4* s4 = (f32x4*)smem;
        const int n4 = nslice / 4;
        for (int c = tid; c < n4; c += RB_THREADS)
            s4[c] = ((s4[c] + s4[n4 + c]) + s4[2 * n4 + c]) + s4[3 * n4 + c];
    }
    __syncthreads();
    float* Sm = smem + nslice;
    for (int c = tid; c < ROWS * E_pad; c += RB_THREADS) {
        const int r = c / E_pad, e = c % E_pad;
        const int rr = r & 15;
        const int o = (((r >> 4) * NT + (e >> 4)) * 64 + (rr >> 2) * 16 + (e & 15)) * 4 + (rr & 3);
        Sm[r * ldS + e] = smem[o];
    }
    __syncthreads();
    if (S == 1) {
        // 1024 threads hold at least one lane group per token: one token per group
        finish_tokens<KM, C, 1>(Sm, ldS, nt, t0, E, k, renorm, bias, logits, idx, gate);
    } else {
        // partial scores of this K chunk: part[chunk][t][e]
        for (int c = tid; c < nt * E; c += RB_THREADS) {
            const int r = c / E, e = c % E;
            part[((int64_t)chunk * T + t0 + r) * E + e] = Sm[r * ldS + e];
        }
    }
}

// Partial bf16 gate scores of short batches (few token blocks, e.g. decode):
// one wave per (16 tokens, 16 experts, K chunk) on MFMA 16x16x32, every operand
// load of the chunk issued before the first product, and the 16 x 16 fp32
// partial tile stored straight from the accumulators into part[chunk][t][e]
// (no LDS, no barriers), so a batch of a few dozen tokens still spreads over
// about a thousand waves.  Rows past the batch or past E, and K past d, read as
// zero through the buffer descriptors.
constexpr int RW_WAVES = 4;            // waves per workgroup
constexpr int RW_STEPS = 8;            // 32-wide K steps of loads issued at once

__global__ __launch_bounds__(RW_WAVES * 64) void route_wave_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int64_t T, int d, int E, int S,
    float* __restrict__ part) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = (int64_t)blockIdx.x * RW_WAVES + (threadIdx.x >> 6);
    const int ET = (E + 15) / 16;
    const int64_t TT = (T + 15) / 16;
    if (wid >= TT * ET * S) return;                  // the whole wave leaves together
    const int c = (int)(wid % S);
    const int64_t tile = wid / S;
    const int e0 = (int)(tile % ET) * 16;
    const int64_t t0 = (tile / ET) * 16;
    const int nt = (int)((T - t0) < 16 ? (T - t0) : 16);
    const int ne = E - e0 < 16 ? E - e0 : 16;
    const int row = lane & 15, kq = (lane >> 4) * 8;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(X + t0 * d), (short)0, nt * d * 2, RB_RSRC_WORD3);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(W + (int64_t)e0 * d), (short)0, ne * d * 2, RB_RSRC_WORD3);
    const int nsteps_all = (d + 31) / 32;
    const int sbeg = (int)((int64_t)c * nsteps_all / S);
    const int send = (int)((int64_t)(c + 1) * nsteps_all / S);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = sbeg; s0 < send; s0 += RW_STEPS) {
        uint4 a[RW_STEPS], b[RW_STEPS];
#pragma unroll
        for (int i = 0; i < RW_STEPS; ++i) {
            const int k = (s0 + i) * 32 + kq;
            const int off = (s0 + i < send && k < d) ? (row * d + k) * 2 : RB_OOB;
            a[i] = rb_load16(xr, off);
            b[i] = rb_load16(wr, off);
        }
#pragma unroll
        for (int i = 0; i < RW_STEPS; ++i)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[i]),
                                                          __builtin_bit_cast(bf16x8, b[i]), acc,
                                                          0, 0, 0);
    }
    // accumulator element i of lane L: token 4 (L / 16) + i, expert L % 16
    if (row < ne) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * (lane >> 4) + i;
            if (r < nt) part[((int64_t)c * T + t0 + r) * E + e0 + row] = acc[i];
        }
    }
}

// fp32 scores (plain FMA loops), scores handed in (MOE_LOGITS_IN) or K-chunk
// partial scores to be summed: `tpb` tokens per workgroup of 256 threads, one
// token per top-k lane group (topk_tokens_per_block), so short batches still
// spread over many workgroups.  MAXS: the most chunks a partial-sum launch adds.
template <int MODE, int KM, int C, int MAXS = ROUTE_MAX_SPLIT>
__global__ __launch_bounds__(ROUTE_THREADS) void route_simple_kernel(
    const float* __restrict__ X, const float* __restrict__ W, const float* __restrict__ bias,
    int64_t T, int d, int E, int k, int renorm, float* __restrict__ logits,
    int32_t* __restrict__ idx, float* __restrict__ gate, int S, const float* __restrict__ part,
    int tpb) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    const int ldS = ((E + 15) & ~15) + 1;
    float* Sm = smem;
    const int tid = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * tpb;
    const int nt = (int)((T - t0) < tpb ? (T - t0) : tpb);
    if (MODE == MODE_F32) {
        for (int c = tid; c < tpb * E; c += ROUTE_THREADS) {
            const int r = c % tpb, e = c / tpb;
            float a = 0.f;
            if (r < nt) {
                const float* xr = X + (t0 + r) * d;
                const float* wr = W + (int64_t)e * d;
                for (int i = 0; i < d; ++i) a = fmaf(xr[i], wr[i], a);
            }
            Sm[r * ldS + e] = a;
        }
    } else if (MODE == MODE_PARTIALS) {
        // K chunks summed in chunk order.  Chunks are split only for short
        // batches, where a thread has few elements: per element, all
        // MAXS chunk loads go out together (unconditionally, clamped to
        // chunk S - 1 and masked by a 0/1 factor), one round trip per element
        const float* pb = part + t0 * E;
        const int64_t cs = T * E;                     // chunk stride
        for (int c = tid; c < nt * E; c += ROUTE_THREADS) {
            float x[MAXS];
#pragma unroll
            for (int ch = 0; ch < MAXS; ++ch) x[ch] = pb[(ch < S ? ch : S - 1) * cs + c];
            float sum = 0.f;
#pragma unroll
            for (int ch = 0; ch < MAXS; ++ch) sum = fmaf(x[ch], ch < S ? 1.0f : 0.0f, sum);
            const int r = c / E, e = c - r * E;
            Sm[r * ldS + e] = sum;
        }
    } else {
        // scores handed in: top-k straight from global memory
        topk_tokens<KM, C>(logits + t0 * E, E, nt, t0, E, k, renorm, idx, gate);
        return;
    }
    __syncthreads();
    finish_tokens<KM, C>(Sm, ldS, nt, t0, E, k, renorm, bias, logits, idx, gate);
}

// Token rows per workgroup of the bf16 score kernel, by expert count.
int route_rows(int E) {
    const int E_pad = (E + 15) & ~15;
    // E <= 16: 16 tokens per workgroup (the router rows are a few KB, so small
    // token blocks cost little re-reading, and a long batch then fills the chip
    // without splitting K and a second launch)
    return 16 * (E_pad <= 16 ? 1 : (E_pad <= 128 ? 2 : 1));
}

// Tokens per workgroup of route_simple_kernel: at most one pass of the top-k
// lane groups, and few enough that a short batch still spreads over >= 128
// workgroups (the chunk sums and the top-k are latency-bound per workgroup).
int simple_tokens_per_block(int64_t T, int E) {
    const int cap = topk_tokens_per_block(E);
    const int64_t want = ceil_div(T, 128);
    return want >= cap ? cap : (want < 1 ? 1 : (int)want);
}

template <int KM, int C>
int launch_kmv(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
              int E, int k, int flags, float* logits, int32_t* idx, float* gate, void* ws,
              hipStream_t s) {
    const int renorm = (flags & MOE_RENORM) ? 1 : 0;
    const int E_pad = (E + 15) & ~15;
    if (!(flags & MOE_LOGITS_IN) && dtype == MOE_BF16) {
        const int rows = route_rows(E);
        const int St = score_tiles_split(T, 2 * d, E, true);
        const int S = St > 0 ? St : route_split(T, d, E);
        const size_t lds = (size_t)4 * rows * (E_pad + 1) * sizeof(float);
        const dim3 grid((unsigned)ceil_div(T, rows), (unsigned)S), block(RB_THREADS);
        float* part = (float*)ws;
        if (St == 1 && E <= 64) {
            // long batch over 33-64 experts: the tiled score kernel with its top-k in
            // the same launch (scores + bias to `logits` when requested).  Wider E
            // keeps the separate top-k launch: there the workgroup's own top-k (more
            // lanes per token, more passes over its 64 tokens) cost more than the
            // launch it saves (E = 128: 33.4 -> 34.6 us, E = 256: 35 -> 45 us per call;
            // E = 64: 22.8 -> 21.5 us)
            return launch_score_tiles_topk(x, w, bias, T, 2 * d, E, k, renorm, logits, idx, gate,
                                           s);
        }
        if (St > 0) {
            // the tiled score kernel with its K split: partial scores to the workspace
            float* out = (St == 1 && logits) ? logits : part;
            const int st = launch_score_tiles(false, x, w, nullptr, nullptr, bias, T, 2 * d, E,
                                              St, out, s);
            if (st != MOE_OK) return st;
            if (St == 1) {
                const int tpb = simple_tokens_per_block(T, E);
                hipLaunchKernelGGL((route_simple_kernel<MODE_LOGITS_IN, KM, C>),
                                   dim3((unsigned)ceil_div(T, tpb)), dim3(ROUTE_THREADS), 0, s,
                                   nullptr, nullptr, nullptr, T, d, E, k, renorm, out, idx, gate, 1,
                                   nullptr, tpb);
                return launch_status();
            }
        } else if (S > 1 && E > 16) {
            const int64_t waves = ceil_div(T, 16) * ((E + 15) / 16) * S;
            hipLaunchKernelGGL(route_wave_kernel, dim3((unsigned)ceil_div(waves, RW_WAVES)),
                               dim3(RW_WAVES * 64), 0, s, (const bf16_t*)x, (const bf16_t*)w, T, d,
                               E, S, part);
        } else {
#define MOE_RB_LAUNCH(RT, NTM)                                                                  \
    do {                                                                                        \
        if (lds > 65536 && allow_dynamic_lds<route_bf16_kernel<RT, NTM, KM, C>>(lds) != MOE_OK)  \
            return MOE_ERR_DEVICE;                                                              \
        hipLaunchKernelGGL((route_bf16_kernel<RT, NTM, KM, C>), grid, block, lds, s,               \
                           (const bf16_t*)x, (const bf16_t*)w, bias, T, d, E, k, renorm,        \
                           logits, idx, gate, S, part);                                         \
    } while (0)
        if constexpr (C == 0) MOE_RB_LAUNCH(1, 1);          // E <= 16
        else if constexpr (C <= 2) MOE_RB_LAUNCH(2, 4);     // E <= 64
        else if constexpr (C == 3) MOE_RB_LAUNCH(2, 8);     // E <= 128
        else MOE_RB_LAUNCH(1, 16);
#undef MOE_RB_LAUNCH
        }
        if (S > 1) {
            const int tpb = simple_tokens_per_block(T, E);
            const size_t lds2 = (size_t)tpb * (E_pad + 1) * sizeof(float);
            // as few clamped chunk loads per score as the split needs
            if (S <= 16)
                hipLaunchKernelGGL((route_simple_kernel<MODE_PARTIALS, KM, C, 16>),
                                   dim3((unsigned)ceil_div(T, tpb)), dim3(ROUTE_THREADS), lds2, s,
                                   nullptr, nullptr, bias, T, d, E, k, renorm, logits, idx, gate, S,
                                   (const float*)part, tpb);
            else
                hipLaunchKernelGGL((route_simple_kernel<MODE_PARTIALS, KM, C, ROUTE_MAX_SPLIT>),
                                   dim3((unsigned)ceil_div(T, tpb)), dim3(ROUTE_THREADS), lds2, s,
                                   nullptr, nullptr, bias, T, d, E, k, renorm, logits, idx, gate, S,
                                   (const float*)part, tpb);
        }
        return launch_status();
    }
    const int tpb = simple_tokens_per_block(T, E);
    const size_t lds = (size_t)tpb * (E_pad + 1) * sizeof(float);
    const dim3 grid((unsigned)ceil_div(T, tpb)), block(ROUTE_THREADS);
    if (flags & MOE_LOGITS_IN)
        hipLaunchKernelGGL((route_simple_kernel<MODE_LOGITS_IN, KM, C>), grid, block, 0, s, nullptr,
                           nullptr, nullptr, T, d, E, k, renorm, logits, idx, gate, 1, nullptr,
                           tpb);
    else
        hipLaunchKernelGGL((route_simple_kernel<MODE_F32, KM, C>), grid, block, lds, s,
                           (const float*)x, (const float*)w, bias, T, d, E, k, renorm, logits,
                           idx, gate, 1, nullptr, tpb);
    return launch_status();
}

}  // namespace

// K chunks of the bf16 scores when there are few token blocks (decode batches);
// 1 = the one-launch kernel with the top-k in its epilogue.  More than 16
// experts: route_wave_kernel gets about 1024 waves of 16 x 16 tiles with at
// least two K steps each (Qwen3-30B-A3B-shaped decode routing 16.8 -> 11.9 us).
// At most 16 experts a 16-wide tile is mostly padding, and the block kernel
// splits K into chunks of at least four steps instead (its LDS reduction sums
// the waves of a block).
int route_split(int64_t T, int d, int E) {
    const int64_t blocks = ceil_div(T, route_rows(E));
    if (blocks <= 0 || blocks >= 128) return 1;
    const int nsteps = (d + 31) / 32;
    int64_t S;
    if (E <= 16) {
        S = ceil_div(256, blocks);
        if (S > 16) S = 16;
        if (S > nsteps / 4) S = nsteps / 4;
    } else {
        S = ceil_div(1024, ceil_div(T, 16) * ((E + 15) / 16));
        if (S > ROUTE_MAX_SPLIT) S = ROUTE_MAX_SPLIT;
        if (S > nsteps / 2) S = nsteps / 2;
    }
    return S < 1 ? 1 : (int)S;
}

size_t route_ws_bytes(int dtype, int64_t T, int d, int E, int flags) {
    if ((flags & MOE_LOGITS_IN) || dtype != MOE_BF16 || T <= 0) return 0;
    const int St = score_tiles_split(T, 2 * d, E, true);
    const int S = St > 0 ? St : route_split(T, d, E);
    // the tiled kernel with one chunk keeps its scores here when none are requested
    return (S > 1 || St == 1) ? (size_t)S * (size_t)T * (size_t)E * sizeof(float) : 0;
}

int launch_topk_given(const float* scores, int64_t T, int E, int k, int flags, int32_t* idx,
                      float* gate, hipStream_t s) {
    return launch_route_topk(nullptr, MOE_F32, nullptr, nullptr, T, 0, E, k,
                             (flags & MOE_RENORM) | MOE_LOGITS_IN, (float*)scores, idx, gate,
                             nullptr, s);
}

int launch_route_topk(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
                      int E, int k, int flags, float* logits, int32_t* idx, float* gate, void* ws,
                      hipStream_t s) {
    if (T == 0) return MOE_OK;
#define MOE_KC(KM, C) launch_kmv<KM, C>(x, dtype, w, bias, T, d, E, k, flags, logits, idx, gate, ws, s)
#define MOE_KMV(KM)                                                                              \
    switch (topk_class(E)) {                                                                     \
        case 0: return MOE_KC(KM, 0);                                                            \
        case 1: return MOE_KC(KM, 1);                                                            \
        case 2: return MOE_KC(KM, 2);                                                            \
        case 3: return MOE_KC(KM, 3);                                                            \
        default: return MOE_KC(KM, 4);                                                           \
    }
    if (k <= 2) MOE_KMV(2);
    if (k <= 4) MOE_KMV(4);
    if (k <= 8) MOE_KMV(8);
    MOE_KMV(16);
#undef MOE_KMV
#undef MOE_KC
}

}  // namespace moe
