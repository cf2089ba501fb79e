// Gate scores and top-k routing (Sec. II-A of the Director paper: the gating
// network scores each expert for every token and the token is sent to the k
// best; the gate is replicated on every GPU, Sec. II-B).
//
// Each workgroup owns a block of tokens:
//   phase 1  scores for its tokens x all E experts into LDS
//            bf16: MFMA 16x16x32, K split over 16 waves, fixed-order reduction;
//            f32:  plain FMA loops;  logits-in: read in place from global memory
//   phase 2  bias added, scores written back coalesced (if requested)
//   phase 3  a group of lanes per token: k rounds of a group-wide maximum, gates.
#include "common.h"

namespace moe {
namespace {

constexpr int ROUTE_THREADS = 256;
constexpr int ROUTE_MAX_SPLIT = 16;    // K chunks of the split score kernel

enum RouteMode { MODE_F32 = 1, MODE_LOGITS_IN = 2, MODE_PARTIALS = 3 };

}  // namespace
int route_split(int64_t T, int d, int E);
namespace {

// Top-k of one token by a group of L adjacent lanes (L in {4, ..., 64}, E <= 4L):
// lane g of the group holds the scores of experts g, g + L, g + 2L, g + 3L as
// 64-bit keys (order-preserving image of the fp32 score in the high half, the
// complement of the expert index in the low half), so "larger key" means larger
// score, ties to the lower index.  Each of the k rounds takes the group-wide
// maximum key by xor shuffles and retires it.
__host__ __device__ inline int topk_lanes(int E) {
    int L = 4;
    while (L * 4 < E) L *= 2;
    return L;
}

__device__ __forceinline__ uint32_t ord_f32(float x) {
    uint32_t u = __float_as_uint(x);
    if (u == 0x80000000u) u = 0u;                        // -0 ranks as +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float unord_f32(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o, 64);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), o, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Cross-lane moves inside a row of 16 lanes (DPP): quad_perm [1,0,3,2] and
// [2,3,0,1], half-row mirror (lane i <- 7 - i) and row mirror (i <- 15 - i).
// Applied in that order, each pairs every lane with one that holds the
// result of a disjoint lane set, so the four steps combine 4, 8, 16 lanes.
constexpr int DPP_QUAD_XOR1 = 0xB1, DPP_QUAD_XOR2 = 0x4E, DPP_HALF_MIRROR = 0x141,
              DPP_MIRROR = 0x140;

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, 0xf, 0xf, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Maximum over each aligned group of L lanes (L in {4, ..., 64}); every lane of
// the wave must be active.
__device__ __forceinline__ uint64_t group_max(uint64_t b, int L) {
    b = umax64(b, dpp_u64<DPP_QUAD_XOR1>(b));
    b = umax64(b, dpp_u64<DPP_QUAD_XOR2>(b));
    if (L >= 8) b = umax64(b, dpp_u64<DPP_HALF_MIRROR>(b));
    if (L >= 16) b = umax64(b, dpp_u64<DPP_MIRROR>(b));
    if (L >= 32) b = umax64(b, shfl_xor_u64(b, 16));
    if (L >= 64) b = umax64(b, shfl_xor_u64(b, 32));
    return b;
}

// Sum over each aligned group of L lanes, the same value on every lane.
__device__ __forceinline__ float group_sum(float v, int L) {
    v += dpp_f32<DPP_QUAD_XOR1>(v);
    v += dpp_f32<DPP_QUAD_XOR2>(v);
    if (L >= 8) v += dpp_f32<DPP_HALF_MIRROR>(v);
    if (L >= 16) v += dpp_f32<DPP_MIRROR>(v);
    if (L >= 32) v += __shfl_xor(v, 16, 64);
    if (L >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// `s` points at the token's E scores (LDS or global memory); every lane of the
// group must call (valid = false only masks the loads and stores).
template <int KM>
__device__ __forceinline__ void topk_group(const float* s, int E, int k, bool renorm, int L, int g,
                                           bool valid, int32_t* __restrict__ idx_out,
                                           float* __restrict__ gate_out) {
    uint64_t key[4];
    float sv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int e = g + i * L;
        key[i] = 0;
        sv[i] = 0.f;
        if (valid && e < E) {
            sv[i] = s[e];
            key[i] = ((uint64_t)ord_f32(sv[i]) << 32) | (uint64_t)(0xffffffffu - (uint32_t)e);
        }
    }
    float v[KM];
    int id[KM];
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        v[r] = 0.f;
        id[r] = 0;
        if (r < k) {
            uint64_t b = key[0] > key[1] ? key[0] : key[1];
            const uint64_t c = key[2] > key[3] ? key[2] : key[3];
            b = group_max(b > c ? b : c, L);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (key[i] == b) key[i] = 0;
            v[r] = unord_f32((uint32_t)(b >> 32));
            id[r] = (int)(0xffffffffu - (uint32_t)b);
        }
    }
    const float m = v[0];
    float denom = 0.f;
    if (renorm) {
#pragma unroll
        for (int j = 0; j < KM; ++j)
            if (j < k) denom += expf(v[j] - m);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (valid && g + i * L < E) denom += expf(sv[i] - m);
        denom = group_sum(denom, L);
    }
    if (valid && g == 0) {
        const float inv = 1.0f / denom;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
            if (j < k) {
                idx_out[j] = id[j];
                gate_out[j] = expf(v[j] - m) * inv;
            }
        }
    }
}

// Top-k of `nt` tokens whose scores sit at S[r * ldS + e] (LDS or global
// memory), by every lane of the workgroup in groups of topk_lanes(E).
template <int KM>
__device__ __forceinline__ void topk_tokens(const float* S, int ldS, int nt, int64_t t0, int E,
                                            int k, int renorm, int32_t* __restrict__ idx,
                                            float* __restrict__ gate) {
    const int L = topk_lanes(E);
    const int tid = threadIdx.x, groups = blockDim.x / L;
    const int grp = tid / L, g = tid % L;
    for (int base = 0; base < nt; base += groups) {
        const int r = base + grp;
        const bool valid = r < nt;
        const int64_t t = t0 + (valid ? r : 0);
        topk_group<KM>(S + (valid ? r : 0) * ldS, E, k, renorm != 0, L, g, valid, idx + t * k,
                       gate + t * k);
    }
}

// Bias, optional score store and top-k for the `nt` tokens whose scores sit in
// S[r * ldS + e] (LDS).
template <int KM>
__device__ __forceinline__ void finish_tokens(float* S, int ldS, int nt, int64_t t0, int E, int k,
                                              int renorm, const float* __restrict__ bias,
                                              float* __restrict__ logits,
                                              int32_t* __restrict__ idx, float* __restrict__ gate) {
    const int tid = threadIdx.x, nthr = blockDim.x;
    for (int c = tid; c < nt * E; c += nthr) {
        const int r = c / E, e = c % E;
        float v = S[r * ldS + e];
        if (bias) v += bias[e];
        S[r * ldS + e] = v;
        if (logits) logits[(t0 + r) * E + e] = v;
    }
    __syncthreads();
    topk_tokens<KM>(S, ldS, nt, t0, E, k, renorm, idx, gate);
}

// bf16 gate scores on MFMA 16x16x32.  A workgroup of 16 waves owns 16*RT
// tokens; wave w takes the K steps w, w+16, w+32, ... (32 elements each) for
// all RT token tiles and up to NTM expert tiles, with operand fragments loaded
// straight from global memory (the router matrix stays L2-resident), two K
// steps of loads in flight per wave.  Partial scores are reduced in LDS in a fixed order
// (four slices, each summed over its four waves in turn, then the slices in
// turn), so the scores are deterministic.
constexpr int RB_WAVES = 16;
constexpr int RB_THREADS = RB_WAVES * 64;

template <int RT, int NTM, int KM>
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

    const bf16_t* xbase = X + (t0 + row) * d + kq;       // token row `row` of tile 0
    const bf16_t* wbase = W + (int64_t)row * d + kq;     // expert row `row` of tile 0
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
        // loads in flight (ring of two register sets, alternating by step parity)
        uint4 av[2][RT], bv[2][NTM];
        auto load = [&](int step, uint4* a_, uint4* b_) {
            const int k0 = step * 32;
            const bool kin = k0 + kq < d;
#pragma unroll
            for (int i = 0; i < RT; ++i) {
                a_[i] = make_uint4(0, 0, 0, 0);
                if (kin && i * 16 + row < nt) a_[i] = *(const uint4*)(xbase + (int64_t)i * 16 * d + k0);
            }
#pragma unroll
            for (int j = 0; j < NTM; ++j) {
                b_[j] = make_uint4(0, 0, 0, 0);
                if (kin && j < NT && j * 16 + row < E)
                    b_[j] = *(const uint4*)(wbase + (int64_t)j * 16 * d + k0);
            }
        };
        auto mma = [&](const uint4* a_, const uint4* b_) {
#pragma unroll
            for (int i = 0; i < RT; ++i)
#pragma unroll
                for (int j = 0; j < NTM; ++j)
                    if (j < NT)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8, a_[i]), __builtin_bit_cast(bf16x8, b_[j]),
                            acc[i][j], 0, 0, 0);
        };
        const int n_mine = wave < nsteps ? (nsteps - wave + RB_WAVES - 1) / RB_WAVES : 0;
        const int s0 = sbeg + wave;
        if (n_mine > 0) load(s0, av[0], bv[0]);
        if (n_mine > 1) load(s0 + RB_WAVES, av[1], bv[1]);
        for (int i = 0; i < n_mine; i += 2) {
            mma(av[0], bv[0]);
            if (i + 2 < n_mine) load(s0 + (i + 2) * RB_WAVES, av[0], bv[0]);
            if (i + 1 < n_mine) {
                mma(av[1], bv[1]);
                if (i + 3 < n_mine) load(s0 + (i + 3) * RB_WAVES, av[1], bv[1]);
            }
        }
    } else {
        for (int step = sbeg + wave; step < send; step += RB_WAVES) {
            const int k0 = step * 32;
            const bool kin = k0 + kq < d;
            bf16x8 a[RT];
#pragma unroll
            for (int i = 0; i < RT; ++i) {
                uint4 v = make_uint4(0, 0, 0, 0);
                if (kin && i * 16 + row < nt) v = *(const uint4*)(xbase + (int64_t)i * 16 * d + k0);
                a[i] = __builtin_bit_cast(bf16x8, v);
            }
#pragma unroll
            for (int jc = 0; jc < NTM; jc += 4) {
                if (jc >= NT) break;
                bf16x8 b[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int j = jc + jj;
                    uint4 v = make_uint4(0, 0, 0, 0);
                    if (kin && j < NT && j * 16 + row < E)
                        v = *(const uint4*)(wbase + (int64_t)j * 16 * d + k0);
                    b[jj] = __builtin_bit_cast(bf16x8, v);
                }
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
        finish_tokens<KM>(Sm, ldS, nt, t0, E, k, renorm, bias, logits, idx, gate);
    } else {
        // partial scores of this K chunk: part[chunk][t][e]
        for (int c = tid; c < nt * E; c += RB_THREADS) {
            const int r = c / E, e = c % E;
            part[((int64_t)chunk * T + t0 + r) * E + e] = Sm[r * ldS + e];
        }
    }
}

// fp32 scores (plain FMA loops), scores handed in (MOE_LOGITS_IN) or K-chunk
// partial scores to be summed: `tpb` tokens per workgroup of 256 threads, one
// token per top-k lane group (route_tokens_per_block), so short batches still
// spread over many workgroups.
template <int MODE, int KM>
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
        // K chunks summed in chunk order
        for (int c = tid; c < nt * E; c += ROUTE_THREADS) {
            const int r = c / E, e = c % E;
            const float* p = part + (t0 + r) * E + e;
            const int64_t cs = T * E;                // chunk stride
            float v[ROUTE_MAX_SPLIT];
#pragma unroll
            for (int ch = 0; ch < ROUTE_MAX_SPLIT; ++ch) v[ch] = ch < S ? p[ch * cs] : 0.f;
            float sum = 0.f;
#pragma unroll
            for (int ch = 0; ch < ROUTE_MAX_SPLIT; ++ch) sum += v[ch];
            Sm[r * ldS + e] = sum;
        }
    } else {
        // scores handed in: top-k straight from global memory
        topk_tokens<KM>(logits + t0 * E, E, nt, t0, E, k, renorm, idx, gate);
        return;
    }
    __syncthreads();
    finish_tokens<KM>(Sm, ldS, nt, t0, E, k, renorm, bias, logits, idx, gate);
}

// Tokens per workgroup of route_simple_kernel: one per top-k lane group.
int route_tokens_per_block(int E) { return ROUTE_THREADS / topk_lanes(E); }

// Token rows per workgroup of the bf16 score kernel, by expert count.
int route_rows(int E) {
    const int E_pad = (E + 15) & ~15;
    return 16 * (E_pad <= 16 ? 4 : (E_pad <= 128 ? 2 : 1));
}

template <int KM>
int launch_km(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
              int E, int k, int flags, float* logits, int32_t* idx, float* gate, void* ws,
              hipStream_t s) {
    const int renorm = (flags & MOE_RENORM) ? 1 : 0;
    const int E_pad = (E + 15) & ~15;
    if (!(flags & MOE_LOGITS_IN) && dtype == MOE_BF16) {
        const int rows = route_rows(E);
        const int S = route_split(T, d, E);
        const size_t lds = (size_t)4 * rows * (E_pad + 1) * sizeof(float);
        const dim3 grid((unsigned)ceil_div(T, rows), (unsigned)S), block(RB_THREADS);
        float* part = (float*)ws;
#define MOE_RB_LAUNCH(RT, NTM)                                                                  \
    do {                                                                                        \
        if (lds > 65536 && allow_dynamic_lds<route_bf16_kernel<RT, NTM, KM>>(lds) != MOE_OK)  \
            return MOE_ERR_DEVICE;                                                              \
        hipLaunchKernelGGL((route_bf16_kernel<RT, NTM, KM>), grid, block, lds, s,               \
                           (const bf16_t*)x, (const bf16_t*)w, bias, T, d, E, k, renorm,        \
                           logits, idx, gate, S, part);                                         \
    } while (0)
        if (E_pad <= 16) MOE_RB_LAUNCH(4, 1);
        else if (E_pad <= 64) MOE_RB_LAUNCH(2, 4);
        else if (E_pad <= 128) MOE_RB_LAUNCH(2, 8);
        else MOE_RB_LAUNCH(1, 16);
#undef MOE_RB_LAUNCH
        if (S > 1) {
            const int tpb = route_tokens_per_block(E);
            const size_t lds2 = (size_t)tpb * (E_pad + 1) * sizeof(float);
            hipLaunchKernelGGL((route_simple_kernel<MODE_PARTIALS, KM>),
                               dim3((unsigned)ceil_div(T, tpb)), dim3(ROUTE_THREADS), lds2, s,
                               nullptr, nullptr, bias, T, d, E, k, renorm, logits, idx, gate, S,
                               (const float*)part, tpb);
        }
        return launch_status();
    }
    const int tpb = route_tokens_per_block(E);
    const size_t lds = (size_t)tpb * (E_pad + 1) * sizeof(float);
    const dim3 grid((unsigned)ceil_div(T, tpb)), block(ROUTE_THREADS);
    if (flags & MOE_LOGITS_IN)
        hipLaunchKernelGGL((route_simple_kernel<MODE_LOGITS_IN, KM>), grid, block, 0, s, nullptr,
                           nullptr, nullptr, T, d, E, k, renorm, logits, idx, gate, 1, nullptr,
                           tpb);
    else
        hipLaunchKernelGGL((route_simple_kernel<MODE_F32, KM>), grid, block, lds, s,
                           (const float*)x, (const float*)w, bias, T, d, E, k, renorm, logits,
                           idx, gate, 1, nullptr, tpb);
    return launch_status();
}

}  // namespace

// K chunks of the bf16 score kernel: enough workgroups to spread the hidden
// states over the chip when there are few token blocks (decode batches).
int route_split(int64_t T, int d, int E) {
    const int64_t blocks = ceil_div(T, route_rows(E));
    if (blocks <= 0 || blocks >= 128) return 1;
    const int nsteps = (d + 31) / 32;
    int64_t S = ceil_div(256, blocks);
    if (S > ROUTE_MAX_SPLIT) S = ROUTE_MAX_SPLIT;
    if (S > nsteps / 4) S = nsteps / 4;
    return S < 1 ? 1 : (int)S;
}

size_t route_ws_bytes(int dtype, int64_t T, int d, int E, int flags) {
    if ((flags & MOE_LOGITS_IN) || dtype != MOE_BF16 || T <= 0) return 0;
    const int S = route_split(T, d, E);
    return S > 1 ? (size_t)S * (size_t)T * (size_t)E * sizeof(float) : 0;
}

int launch_route_topk(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
                      int E, int k, int flags, float* logits, int32_t* idx, float* gate, void* ws,
                      hipStream_t s) {
    if (T == 0) return MOE_OK;
    if (k <= 2) return launch_km<2>(x, dtype, w, bias, T, d, E, k, flags, logits, idx, gate, ws, s);
    if (k <= 4) return launch_km<4>(x, dtype, w, bias, T, d, E, k, flags, logits, idx, gate, ws, s);
    if (k <= 8) return launch_km<8>(x, dtype, w, bias, T, d, E, k, flags, logits, idx, gate, ws, s);
    return launch_km<16>(x, dtype, w, bias, T, d, E, k, flags, logits, idx, gate, ws, s);
}

}  // namespace moe
