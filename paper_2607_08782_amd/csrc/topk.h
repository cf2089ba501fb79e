// Top-k routing of given scores (Sec. II-A: each token goes to its k best
// experts; gates are the softmax of the selected scores, or of all scores
// restricted to the selected ones).  Internal to the library.
//
// One token is handled by a group of L adjacent lanes; lane g of the group
// holds V scores, of experts g, g + L, ..., g + (V-1) L, as 64-bit keys: the
// high half an order-preserving image of the fp32 score, the low half the
// complement of the expert index, so "larger key" means larger score, ties to
// the lower index (and -0 ranks as +0).  Each lane sorts its keys once; each of
// the k rounds then takes the group-wide maximum of the lanes' leading keys and
// the lane holding it shifts its keys by one.  The shape (V, L) is fixed per
// class of E at compile time (no branches in the reductions), and a group works
// on NT tokens at once so a wave has independent chains to issue.
#pragma once

#include "common.h"

namespace moe {

constexpr int TOPK_THREADS = 256;

// Class of E: 0: E <= 16, 1: <= 32, 2: <= 64, 3: <= 128, 4: <= 256.
__host__ __device__ constexpr int topk_class(int E) {
    return E <= 16 ? 0 : E <= 32 ? 1 : E <= 64 ? 2 : E <= 128 ? 3 : 4;
}
template <int C> struct TopkShape {
    static constexpr int V = C <= 1 ? 4 : 8;                       // keys per lane
    static constexpr int L = C == 0 ? 4 : C <= 2 ? 8 : C == 3 ? 16 : 32;   // lanes per token
    static constexpr int NT = 2;                                   // tokens per group at once
};
// Tokens per 256-thread workgroup of the given-scores top-k: NT per lane group.
__host__ __device__ constexpr int topk_tokens_per_block_c(int C) {
    return 2 * (C == 0 ? 64 : C <= 2 ? 32 : C == 3 ? 16 : 8);
}

__device__ __forceinline__ uint32_t ord_f32(float x) {
    uint32_t u = __float_as_uint(x);
    if (u == 0x80000000u) u = 0u;
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
    const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)v, CTRL, 0xf, 0xf, true);
    const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(v >> 32), CTRL, 0xf, 0xf, true);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// Maximum over each aligned group of L lanes (L in {4, ..., 64}); every lane of
// the wave must be active.
template <int L>
__device__ __forceinline__ uint64_t group_max(uint64_t b) {
    b = umax64(b, dpp_u64<DPP_QUAD_XOR1>(b));
    b = umax64(b, dpp_u64<DPP_QUAD_XOR2>(b));
    if constexpr (L >= 8) b = umax64(b, dpp_u64<DPP_HALF_MIRROR>(b));
    if constexpr (L >= 16) b = umax64(b, dpp_u64<DPP_MIRROR>(b));
    if constexpr (L >= 32) b = umax64(b, shfl_xor_u64(b, 16));
    if constexpr (L >= 64) b = umax64(b, shfl_xor_u64(b, 32));
    return b;
}

// Sum over each aligned group of L lanes, the same value on every lane.
template <int L>
__device__ __forceinline__ float group_sum(float v) {
    v += dpp_f32<DPP_QUAD_XOR1>(v);
    v += dpp_f32<DPP_QUAD_XOR2>(v);
    if constexpr (L >= 8) v += dpp_f32<DPP_HALF_MIRROR>(v);
    if constexpr (L >= 16) v += dpp_f32<DPP_MIRROR>(v);
    if constexpr (L >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (L >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// Compare-exchange: a keeps the larger key.
__device__ __forceinline__ void cx64(uint64_t& a, uint64_t& b) {
    const bool sw = b > a;
    const uint64_t t = sw ? b : a;
    b = sw ? a : b;
    a = t;
}

// Sort V (4 or 8) keys descending in registers (Batcher's odd-even merge sort).
template <int V>
__device__ __forceinline__ void sort_keys(uint64_t (&k)[V]) {
    static_assert(V == 4 || V == 8, "sorting network for 4 or 8 keys");
    if constexpr (V == 4) {
        cx64(k[0], k[1]); cx64(k[2], k[3]);
        cx64(k[0], k[2]); cx64(k[1], k[3]);
        cx64(k[1], k[2]);
    } else {
        cx64(k[0], k[1]); cx64(k[2], k[3]); cx64(k[4], k[5]); cx64(k[6], k[7]);
        cx64(k[0], k[2]); cx64(k[1], k[3]); cx64(k[4], k[6]); cx64(k[5], k[7]);
        cx64(k[1], k[2]); cx64(k[5], k[6]);
        cx64(k[0], k[4]); cx64(k[1], k[5]); cx64(k[2], k[6]); cx64(k[3], k[7]);
        cx64(k[2], k[4]); cx64(k[3], k[5]);
        cx64(k[1], k[2]); cx64(k[3], k[4]); cx64(k[5], k[6]);
    }
}

// Top-k of NT tokens at once by one group of L lanes (the tokens' instruction
// streams interleave).  s[j] points at token j's E scores (LDS or global
// memory); every lane of the group must call (valid[j] = false only masks
// token j's loads and stores).  Each lane sorts its keys once; a round is then
// the group maximum over the lanes' leading keys, and the lane holding it
// shifts its keys by one.
template <int KM, int C, int NT>
__device__ __forceinline__ void topk_group(const float* const (&s)[NT], int E, int k, bool renorm,
                                           int g, const bool (&valid)[NT],
                                           int32_t* const (&idx_out)[NT],
                                           float* const (&gate_out)[NT]) {
    constexpr int V = TopkShape<C>::V, L = TopkShape<C>::L;
    uint64_t key[NT][V];
    float sv[NT][V];
    // every load is issued unconditionally from an in-bounds address (s[j][0]
    // exists) and masked afterwards, so the loads overlap instead of each
    // waiting behind a branch
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e = g + i * L;
            const bool ok = valid[j] && e < E;
            sv[j][i] = s[j][ok ? e : 0];
        }
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e = g + i * L;
            const bool ok = valid[j] && e < E;
            sv[j][i] = ok ? sv[j][i] : 0.f;
            key[j][i] = ok ? (((uint64_t)ord_f32(sv[j][i]) << 32) |
                              (uint64_t)(0xffffffffu - (uint32_t)e))
                           : 0;
        }
#pragma unroll
    for (int j = 0; j < NT; ++j) sort_keys<V>(key[j]);
    float v[NT][KM];
    int id[NT][KM];
#pragma unroll
    for (int r = 0; r < KM; ++r) {
        if (r < k) {
            uint64_t b[NT];
#pragma unroll
            for (int j = 0; j < NT; ++j) b[j] = group_max<L>(key[j][0]);
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const bool mine = key[j][0] == b[j];
#pragma unroll
                for (int i = 0; i < V - 1; ++i) key[j][i] = mine ? key[j][i + 1] : key[j][i];
                key[j][V - 1] = mine ? 0 : key[j][V - 1];
                v[j][r] = unord_f32((uint32_t)(b[j] >> 32));
                id[j][r] = (int)(0xffffffffu - (uint32_t)b[j]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                v[j][r] = 0.f;
                id[j][r] = 0;
            }
        }
    }
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const float m = v[j][0];
        float denom = 0.f;
        if (renorm) {
#pragma unroll
            for (int r = 0; r < KM; ++r)
                if (r < k) denom += expf(v[j][r] - m);
        } else {
#pragma unroll
            for (int i = 0; i < V; ++i)
                if (valid[j] && g + i * L < E) denom += expf(sv[j][i] - m);
            denom = group_sum<L>(denom);
        }
        if (valid[j] && g == 0) {
            const float inv = 1.0f / denom;
#pragma unroll
            for (int r = 0; r < KM; ++r) {
                if (r < k) {
                    idx_out[j][r] = id[j][r];
                    gate_out[j][r] = expf(v[j][r] - m) * inv;
                }
            }
        }
    }
}

// Top-k of `nt` tokens whose scores sit at S[r * ldS + e] (LDS or global
// memory), by every lane of the workgroup in groups of L lanes, NT tokens per
// group at a time.
template <int KM, int C, int NT = TopkShape<C>::NT>
__device__ __forceinline__ void topk_tokens(const float* S, int ldS, int nt, int64_t t0, int E,
                                            int k, int renorm, int32_t* __restrict__ idx,
                                            float* __restrict__ gate) {
    constexpr int L = TopkShape<C>::L;
    const int tid = threadIdx.x, groups = blockDim.x / L;
    const int grp = tid / L, g = tid % L;
    for (int base = 0; base < nt; base += groups * NT) {
        const float* sp[NT];
        bool valid[NT];
        int32_t* ip[NT];
        float* gp[NT];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int r = base + grp + j * groups;
            valid[j] = r < nt;
            const int rr = valid[j] ? r : 0;
            sp[j] = S + rr * ldS;
            ip[j] = idx + (t0 + rr) * k;
            gp[j] = gate + (t0 + rr) * k;
        }
        topk_group<KM, C, NT>(sp, E, k, renorm != 0, g, valid, ip, gp);
    }
}

// Bias, optional score store and top-k for the `nt` tokens whose scores sit in
// S[r * ldS + e] (LDS).
template <int KM, int C, int NT = TopkShape<C>::NT>
__device__ __forceinline__ void finish_tokens(float* S, int ldS, int nt, int64_t t0, int E, int k,
                                              int renorm, const float* __restrict__ bias,
                                              float* __restrict__ logits,
                                              int32_t* __restrict__ idx, float* __restrict__ gate) {
    const int tid = threadIdx.x, nthr = blockDim.x;
    // element c = r * E + e, walked without a division per element
    const int dr = nthr / E, de = nthr - dr * E;
    int r = tid / E, e = tid - r * E;
    for (; r < nt; r += dr, e += de) {
        if (e >= E) {
            e -= E;
            ++r;
            if (r >= nt) break;
        }
        float v = S[r * ldS + e];
        if (bias) v += bias[e];
        S[r * ldS + e] = v;
        if (logits) logits[(t0 + r) * E + e] = v;
    }
    __syncthreads();
    topk_tokens<KM, C, NT>(S, ldS, nt, t0, E, k, renorm, idx, gate);
}

inline int topk_tokens_per_block(int E) { return topk_tokens_per_block_c(topk_class(E)); }

}  // namespace moe
