// Gate scores and top-k routing (Sec. II-A of the Director paper: the gating
// network scores each expert for every token and the token is sent to the k
// best; the gate is replicated on every GPU, Sec. II-B).
//
// One workgroup of 256 threads owns 64 tokens:
//   phase 1  scores for the 64 tokens x all E experts into LDS
//            bf16: MFMA 16x16x32 (four waves x 16 tokens, router rows staged
//            through LDS once per workgroup and K step);
//            f32:  plain FMA loops;  logits-in: copied from global memory
//   phase 2  bias added, scores written back coalesced (if requested)
//   phase 3  one thread per token: insertion top-k over the LDS row, gates.
#include "common.h"

namespace moe {
namespace {

constexpr int ROUTE_TOKENS = 64;
constexpr int ROUTE_THREADS = 256;
constexpr int ROUTE_BK = 32;          // K per MFMA 16x16x32 step

enum RouteMode { MODE_BF16 = 0, MODE_F32 = 1, MODE_LOGITS_IN = 2 };

// "a ranks before b": larger score, or equal score and lower expert index.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
    return va > vb || (va == vb && ia < ib);
}

template <int KM>
__device__ void topk_row(const float* s, int E, int k, bool renorm, int32_t* idx_out,
                         float* gate_out) {
    float v[KM];
    int id[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) { v[j] = -__builtin_inff(); id[j] = 0x7fffffff; }
    float kth_v = -__builtin_inff();
    int kth_i = 0x7fffffff;
    for (int e = 0; e < E; ++e) {
        float x = s[e];
        if (!better(x, e, kth_v, kth_i)) continue;
#pragma unroll
        for (int j = 0; j < KM; ++j)
            if (j == k - 1) { v[j] = x; id[j] = e; }
#pragma unroll
        for (int j = KM - 1; j > 0; --j) {
            if (j < k && better(v[j], id[j], v[j - 1], id[j - 1])) {
                float tv = v[j]; v[j] = v[j - 1]; v[j - 1] = tv;
                int ti = id[j]; id[j] = id[j - 1]; id[j - 1] = ti;
            }
        }
#pragma unroll
        for (int j = 0; j < KM; ++j)
            if (j == k - 1) { kth_v = v[j]; kth_i = id[j]; }
    }
    const float m = v[0];
    float denom = 0.f;
    if (renorm) {
#pragma unroll
        for (int j = 0; j < KM; ++j)
            if (j < k) denom += expf(v[j] - m);
    } else {
        for (int e = 0; e < E; ++e) denom += expf(s[e] - m);
    }
    const float inv = 1.0f / denom;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        if (j < k) {
            idx_out[j] = id[j];
            gate_out[j] = expf(v[j] - m) * inv;
        }
    }
}

template <int MODE, int KM>
__global__ __launch_bounds__(ROUTE_THREADS) void route_kernel(
    const void* __restrict__ xv, const void* __restrict__ wv, const float* __restrict__ bias,
    int64_t T, int d, int E, int k, int renorm, float* __restrict__ logits,
    int32_t* __restrict__ idx, float* __restrict__ gate) {
    extern __shared__ float smem[];
    const int E_pad = (E + 15) & ~15;
    const int ldS = E_pad + 1;                   // odd stride: conflict-free row scans
    float* S = smem;                             // [64][ldS] scores
    bf16_t* Wst = (bf16_t*)(smem + ROUTE_TOKENS * ldS);   // [E_pad][ROUTE_BK] router slice (bf16)

    const int tid = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * ROUTE_TOKENS;
    const int nt = (int)((T - t0) < ROUTE_TOKENS ? (T - t0) : ROUTE_TOKENS);

    if (MODE == MODE_BF16) {
        const bf16_t* X = (const bf16_t*)xv;
        const bf16_t* W = (const bf16_t*)wv;
        const int wave = tid >> 6, lane = tid & 63;
        const int row = lane & 15;                 // token row of this lane's A fragment
        const int kq = (lane >> 4) * 8;            // K offset of this lane inside the 32-step
        const int64_t trow = t0 + wave * 16 + row;
        const bool row_ok = (wave * 16 + row) < nt;
        const int NT = E_pad / 16;                 // expert tiles (<= 16)
        f32x4 acc[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

        for (int k0 = 0; k0 < d; k0 += ROUTE_BK) {
            // stage W[0:E_pad, k0:k0+32] in LDS, 16 bytes per thread per pass
            const int chunks = E_pad * (ROUTE_BK / 8);
            for (int c = tid; c < chunks; c += ROUTE_THREADS) {
                const int e = c >> 2, kc = (c & 3) * 8;
                uint4 v = make_uint4(0, 0, 0, 0);
                if (e < E && k0 + kc < d) v = *(const uint4*)(W + (int64_t)e * d + k0 + kc);
                *(uint4*)(Wst + e * ROUTE_BK + kc) = v;
            }
            uint4 av = make_uint4(0, 0, 0, 0);
            if (row_ok && k0 + kq < d) av = *(const uint4*)(X + trow * d + k0 + kq);
            __syncthreads();
            const bf16x8 a = __builtin_bit_cast(bf16x8, av);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                if (j < NT) {
                    const uint4 bv = *(const uint4*)(Wst + (j * 16 + row) * ROUTE_BK + kq);
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        a, __builtin_bit_cast(bf16x8, bv), acc[j], 0, 0, 0);
                }
            }
            __syncthreads();
        }
        // C fragment: lane holds rows 4*(lane/16)+i, column lane%16
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (j < NT) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = wave * 16 + (lane >> 4) * 4 + i;
                    S[r * ldS + j * 16 + (lane & 15)] = acc[j][i];
                }
            }
        }
        __syncthreads();
    } else if (MODE == MODE_F32) {
        const float* X = (const float*)xv;
        const float* W = (const float*)wv;
        for (int c = tid; c < ROUTE_TOKENS * E; c += ROUTE_THREADS) {
            const int r = c % ROUTE_TOKENS, e = c / ROUTE_TOKENS;
            float a = 0.f;
            if (r < nt) {
                const float* xr = X + (t0 + r) * d;
                const float* wr = W + (int64_t)e * d;
                for (int i = 0; i < d; ++i) a = fmaf(xr[i], wr[i], a);
            }
            S[r * ldS + e] = a;
        }
        __syncthreads();
    } else {
        for (int c = tid; c < nt * E; c += ROUTE_THREADS) {
            const int r = c / E, e = c % E;
            S[r * ldS + e] = logits[(t0 + r) * E + e];
        }
        __syncthreads();
    }

    if (MODE != MODE_LOGITS_IN) {
        for (int c = tid; c < nt * E; c += ROUTE_THREADS) {
            const int r = c / E, e = c % E;
            float v = S[r * ldS + e];
            if (bias) v += bias[e];
            S[r * ldS + e] = v;
            if (logits) logits[(t0 + r) * E + e] = v;
        }
        __syncthreads();
    }

    if (tid < nt) {
        const int64_t t = t0 + tid;
        topk_row<KM>(S + tid * ldS, E, k, renorm != 0, idx + t * k, gate + t * k);
    }
}

template <int MODE>
int launch_mode(const void* x, const void* w, const float* bias, int64_t T, int d, int E, int k,
                int renorm, float* logits, int32_t* idx, float* gate, hipStream_t s) {
    const int E_pad = (E + 15) & ~15;
    size_t lds = (size_t)ROUTE_TOKENS * (E_pad + 1) * sizeof(float);
    if (MODE == MODE_BF16) lds += (size_t)E_pad * ROUTE_BK * sizeof(bf16_t);
    const dim3 grid((unsigned)ceil_div(T, ROUTE_TOKENS));
    const dim3 block(ROUTE_THREADS);
#define MOE_ROUTE_LAUNCH(KM)                                                                    \
    do {                                                                                        \
        if (lds > 65536 &&                                                                      \
            hipFuncSetAttribute((const void*)route_kernel<MODE, KM>,                            \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=        \
                hipSuccess)                                                                     \
            return MOE_ERR_DEVICE;                                                              \
        hipLaunchKernelGGL((route_kernel<MODE, KM>), grid, block, lds, s, x, w, bias, T, d, E,  \
                           k, renorm, logits, idx, gate);                                       \
    } while (0)
    if (k <= 2) MOE_ROUTE_LAUNCH(2);
    else if (k <= 4) MOE_ROUTE_LAUNCH(4);
    else if (k <= 8) MOE_ROUTE_LAUNCH(8);
    else MOE_ROUTE_LAUNCH(16);
#undef MOE_ROUTE_LAUNCH
    return launch_status();
}

}  // namespace

int launch_route_topk(const void* x, int dtype, const void* w, const float* bias, int64_t T, int d,
                      int E, int k, int flags, float* logits, int32_t* idx, float* gate,
                      hipStream_t s) {
    if (T == 0) return MOE_OK;
    const int renorm = (flags & MOE_RENORM) ? 1 : 0;
    if (flags & MOE_LOGITS_IN)
        return launch_mode<MODE_LOGITS_IN>(nullptr, nullptr, nullptr, T, d, E, k, renorm, logits,
                                           idx, gate, s);
    if (dtype == MOE_BF16)
        return launch_mode<MODE_BF16>(x, w, bias, T, d, E, k, renorm, logits, idx, gate, s);
    return launch_mode<MODE_F32>(x, w, bias, T, d, E, k, renorm, logits, idx, gate, s);
}

}  // namespace moe
