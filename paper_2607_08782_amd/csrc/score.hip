// Gate scores of long batches over many experts (Sec. II-A: the gating network
// scores every expert for every token), as a tiled GEMM:
//
//   bf16:  S[t][e] = sum_i x[t][i] w[e][i]
//   E4M3:  S[t][e] = s_x[t] s_w[e] sum_i q_x[t][i] q_w[e][i]    (the quantized
//          predictor's gate, Sec. V-A)
//
// plus bias.  The kernel streams the hidden states once: a workgroup
// owns 64 tokens x all experts (4 waves: 2 token halves x 2 expert halves), so
// each router row is read once per 64 tokens instead of once per 32 or 16, and
// both operands go straight from HBM/L2 into a ring of LDS stages (128 bytes of
// K per row per stage, `buffer_load ... lds`) with R - 1 stages in flight,
// which keeps enough bytes moving per CU to reach the HBM rate.  Rows past the
// batch or past E fall outside the buffer descriptors and read as zero.  The
// LDS rows are XOR-swizzled in 16-byte chunks (the loading lane fetches the
// chunk that belongs in its slot), so fragment reads are free of bank
// conflicts without padding.
//
// With one K chunk the workgroup stores its scores (bias added); with S > 1
// chunks it stores fp32 partial scores part[chunk][t][e], which the caller
// sums in chunk order.  The bf16 gate with one chunk can also finish with the
// top-k of its own 64 tokens (KM > 0): the scores go through LDS to the same
// top-k as for given scores, so no second launch reads them back.
#include "common.h"
#include "topk.h"

namespace moe {
namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int SC_BM = 64;          // tokens per workgroup
constexpr int SC_THREADS = 256;    // 4 waves
constexpr int SC_BKB = 128;        // bytes of K per row per stage
constexpr uint32_t SC_RSRC_WORD3 = 0x00020000;
constexpr int SC_OOB = 0x7fffff00;  // an offset past every descriptor's range: the store is dropped

// chunk position of 16-byte chunk c of LDS row r: c ^ sc_swz(r)
__device__ __forceinline__ int sc_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// wait until at most N of this wave's vector-memory loads are outstanding
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// KM > 0 (S == 1): top-k (k <= KM, top-k class C) of the workgroup's tokens
// into idx / gate after the scores; out (the scores) may then be null.
template <bool FP8, int NTW, int R, int KM = 0, int C = 0>
__global__ __launch_bounds__(SC_THREADS) void score_tiles_kernel(
    const uint8_t* __restrict__ x, const uint8_t* __restrict__ w, const float* __restrict__ sx,
    const float* __restrict__ sw, const float* __restrict__ bias, int64_t T, int rowbytes, int E,
    int S, float* __restrict__ out, int k = 0, int renorm = 0, int32_t* __restrict__ idx = nullptr,
    float* __restrict__ gate = nullptr) {
    extern __shared__ __attribute__((aligned(1024))) char lds[];
    constexpr int A_BYTES = SC_BM * SC_BKB;           // 8 KB
    constexpr int NB = 64 * NTW;                      // router rows per tile
    constexpr int B_BYTES = NB * SC_BKB;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int A_LOADS = A_BYTES / 1024 / 4;       // 1 KB direct loads per wave per stage
    constexpr int B_LOADS = B_BYTES / 1024 / 4;
    constexpr int P = A_LOADS + B_LOADS;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;
    const int64_t t0 = (int64_t)blockIdx.x * SC_BM;
    const int nt = (int)((T - t0) < SC_BM ? (T - t0) : SC_BM);
    const int chunk = blockIdx.y;
    const int nst_all = rowbytes / SC_BKB;
    const int st0 = (int)((int64_t)chunk * nst_all / S);
    const int nst = (int)((int64_t)(chunk + 1) * nst_all / S) - st0;

    const __amdgpu_buffer_rsrc_t arsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + t0 * rowbytes), (short)0, nt * rowbytes, SC_RSRC_WORD3);
    const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)w, (short)0, E * rowbytes, SC_RSRC_WORD3);
    // load i of a wave fills LDS rows 32 i + 8 wave + (lane / 8), chunk slot lane % 8,
    // from the operand row of the same index (row offsets in the per-lane offset, so
    // the descriptor's range check sees them), chunk (lane % 8) ^ sc_swz(row)
    const int drow = lane >> 3;
    const int voff0 = (8 * wave + drow) * rowbytes + (((lane & 7) ^ (drow ^ (wave & 1))) * 16);
    const int vstep = 32 * rowbytes;
    auto dma = [&](int s) {
        char* base = lds + (s % R) * STAGE;
        const int so = (st0 + s) * SC_BKB;
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                arsrc, (lds_void*)(base + (4 * i + wave) * 1024), 16, voff0 + i * vstep, so, 0, 0);
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                brsrc, (lds_void*)(base + A_BYTES + (4 * i + wave) * 1024), 16, voff0 + i * vstep,
                so, 0, 0);
    };

    // fragments: lane row r = lane % 32 of its 32-row tile, half h = lane / 32.
    // bf16 (32x32x16): sub-step q reads chunk 4h + q (elements 32h + 8q ..);
    // E4M3 (32x32x64): sub-step q reads chunks 4h + 2q, 4h + 2q + 1.  The same
    // K order for both operands, so the products sum over all of K.
    const int fr = lane & 31, h = lane >> 5;
    const int swz = sc_swz(fr);
    const int a_row = (wm * 32 + fr) * SC_BKB;
    const int b_row = A_BYTES + (wn * 32 * NTW + fr) * SC_BKB;
    int coff[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) coff[c] = ((4 * h + c) ^ swz) * 16;

    f32x16 acc[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

    // the lane's column terms (bias; the FP8 router-row scales), loaded before the
    // K loop: a load still pending at the stores made the compiler wait for every
    // earlier store before each one, serialising the epilogue
    float b_c[NTW], s_c[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        const int col = wn * 32 * NTW + j * 32 + fr;
        const int cc = col < E ? col : E - 1;
        b_c[j] = (S == 1 && bias) ? bias[cc] : 0.0f;
        s_c[j] = FP8 ? sw[cc] : 1.0f;
    }

    auto compute = [&](int slot) {
        const char* st = lds + slot * STAGE;
        if constexpr (FP8) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const uint4 a0 = *(const uint4*)(st + a_row + coff[2 * q]);
                const uint4 a1 = *(const uint4*)(st + a_row + coff[2 * q + 1]);
                const i32x8 a = {(int)a0.x, (int)a0.y, (int)a0.z, (int)a0.w,
                                 (int)a1.x, (int)a1.y, (int)a1.z, (int)a1.w};
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    const char* br = st + b_row + j * 32 * SC_BKB;
                    const uint4 b0 = *(const uint4*)(br + coff[2 * q]);
                    const uint4 b1 = *(const uint4*)(br + coff[2 * q + 1]);
                    const i32x8 b = {(int)b0.x, (int)b0.y, (int)b0.z, (int)b0.w,
                                     (int)b1.x, (int)b1.y, (int)b1.z, (int)b1.w};
                    acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[j], 0, 0, 0,
                                                                             127, 0, 127);
                }
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bf16x8 a = *(const bf16x8*)(st + a_row + coff[q]);
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    const bf16x8 b = *(const bf16x8*)(st + b_row + j * 32 * SC_BKB + coff[q]);
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
                }
            }
        }
    };

#pragma unroll
    for (int s = 0; s < R - 1; ++s)
        if (s < nst) dma(s);
    for (int t = 0; t < nst; ++t) {
        if (nst - 1 - t >= R - 2)
            wait_vm<(R - 2) * P>();       // stage t landed; the R - 2 after it may still fly
        else
            wait_vm<0>();
        // every wave's share of stage t is in; stage t-1 is free (its reads fed
        // MFMAs already).  A bare barrier: the fence of __syncthreads would wait
        // for all R - 1 stages in flight, draining the ring every step.
        asm volatile("s_barrier" ::: "memory");
        if (t + R - 1 < nst) dma(t + R - 1);
        compute(t % R);
    }

    // accumulator element r of a 32x32 tile: row 8 (r / 4) + 4 h + r % 4, column fr;
    // S == 1: out[t][e] = score + bias[e];  S > 1: out[chunk][t][e] = partial score.
    // Branch-free stores through a descriptor over the block's rows: an element past
    // the batch or past E gets an offset outside it and is dropped.
    float* o = out ? out + (S > 1 ? (int64_t)chunk * T * E : 0) + t0 * E : nullptr;
    const __amdgpu_buffer_rsrc_t orsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)o, (short)0, o ? nt * E * 4 : 0, SC_RSRC_WORD3);
    // fused top-k: the scores also go to an LDS tile [64][E_pad + 1] over the
    // ring, which every wave has finished reading once past this barrier
    const int ldS = ((E + 15) & ~15) + 1;
    float* const sc = (float*)lds;
    if constexpr (KM > 0) asm volatile("s_barrier" ::: "memory");
    float sx_r[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int row = wm * 32 + (r >> 2) * 8 + 4 * h + (r & 3);
        sx_r[r] = FP8 ? sx[t0 + (row < nt ? row : nt - 1)] : 1.0f;
    }
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        const int col = wn * 32 * NTW + j * 32 + fr;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + (r >> 2) * 8 + 4 * h + (r & 3);
            float v = acc[j][r];
            if (FP8) v = v * sx_r[r] * s_c[j];
            if (S == 1 && bias) v += b_c[j];
            const int off = (row < nt && col < E) ? (row * E + col) * 4 : SC_OOB;
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), orsrc, off, 0, 0);
            if constexpr (KM > 0)
                if (row < nt && col < E) sc[row * ldS + col] = v;
        }
    }
    if constexpr (KM > 0) {
        __syncthreads();
        topk_tokens<KM, C>(sc, ldS, nt, t0, E, k, renorm, idx, gate);
    }
}

template <bool FP8, int NTW, int R>
int launch_tiles(const uint8_t* x, const uint8_t* w, const float* sx, const float* sw,
                 const float* bias, int64_t T, int rowbytes, int E, int S, float* out,
                 hipStream_t s) {
    constexpr size_t lds = (size_t)R * (SC_BM * SC_BKB + 64 * NTW * SC_BKB);
    static_assert(lds <= 160 * 1024, "ring fits the LDS of a CU");
    if (lds > 65536 && allow_dynamic_lds<score_tiles_kernel<FP8, NTW, R>>(lds) != MOE_OK)
        return MOE_ERR_DEVICE;
    const dim3 grid((unsigned)ceil_div(T, SC_BM), (unsigned)S);
    hipLaunchKernelGGL((score_tiles_kernel<FP8, NTW, R>), grid, dim3(SC_THREADS), lds, s, x, w, sx,
                       sw, bias, T, rowbytes, E, S, out);
    return launch_status();
}

template <int NTW, int R, int KM, int C>
int launch_tiles_topk(const uint8_t* x, const uint8_t* w, const float* bias, int64_t T,
                      int rowbytes, int E, int k, int renorm, float* logits, int32_t* idx,
                      float* gate, hipStream_t s) {
    constexpr size_t ring = (size_t)R * (SC_BM * SC_BKB + 64 * NTW * SC_BKB);
    constexpr size_t tile = (size_t)SC_BM * (64 * NTW + 1) * sizeof(float);
    constexpr size_t lds = ring > tile ? ring : tile;
    static_assert(lds <= 160 * 1024, "ring fits the LDS of a CU");
    if (lds > 65536 &&
        allow_dynamic_lds<score_tiles_kernel<false, NTW, R, KM, C>>(lds) != MOE_OK)
        return MOE_ERR_DEVICE;
    hipLaunchKernelGGL((score_tiles_kernel<false, NTW, R, KM, C>), dim3((unsigned)ceil_div(T, SC_BM)),
                       dim3(SC_THREADS), lds, s, x, w, nullptr, nullptr, bias, T, rowbytes, E, 1,
                       logits, k, renorm, idx, gate);
    return launch_status();
}

template <int KM>
int launch_topk_by_width(const uint8_t* x, const uint8_t* w, const float* bias, int64_t T,
                         int rowbytes, int E, int k, int renorm, float* logits, int32_t* idx,
                         float* gate, hipStream_t s) {
    // 33-64 experts: one 64-wide tile, top-k class 2
    if (E > 64) return MOE_ERR_SHAPE;
    return launch_tiles_topk<1, 8, KM, 2>(x, w, bias, T, rowbytes, E, k, renorm, logits, idx,
                                          gate, s);
}

}  // namespace

// K chunks for the tiled score kernel, or 0 when the shape does not suit it:
// E > 32 (smaller E is cheap for the K-split kernel), whole 128-byte stages,
// and at least 128 token tiles (half a tile per CU or more; the DeepSeek-V2-Lite
// prefill batch of 8192 tokens: 22.1 -> 20.2 us against the block kernel).  One
// chunk: summing K-chunk partials in a second pass cost more than the
// parallelism it bought (that batch split in two: 27.1 us), and with fewer tiles
// the K-split kernel, which spreads a batch over more workgroups, measured faster
// (Qwen1.5-shaped batches).
int score_tiles_split(int64_t T, int rowbytes, int E, bool allow_split) {
    (void)allow_split;
    if (E <= 32 || E > MOE_MAX_E || rowbytes % SC_BKB != 0 || T <= 0) return 0;
    if ((int64_t)MOE_MAX_E * rowbytes >= ((int64_t)1 << 31)) return 0;   // 32-bit buffer offsets
    return ceil_div(T, SC_BM) >= 128 ? 1 : 0;
}

// Ring depth by tile width: one workgroup per CU, as many stages in flight as
// the LDS holds (the hidden states arrive at the rate bytes-in-flight / latency).
int launch_score_tiles(bool fp8, const void* x, const void* w, const float* sx, const float* sw,
                       const float* bias, int64_t T, int rowbytes, int E, int S, float* out,
                       hipStream_t s) {
    const uint8_t* xb = (const uint8_t*)x;
    const uint8_t* wb = (const uint8_t*)w;
#define MOE_SC(F)                                                                                   \
    if (E <= 64) return launch_tiles<F, 1, 8>(xb, wb, sx, sw, bias, T, rowbytes, E, S, out, s);     \
    if (E <= 128) return launch_tiles<F, 2, 6>(xb, wb, sx, sw, bias, T, rowbytes, E, S, out, s);    \
    return launch_tiles<F, 4, 3>(xb, wb, sx, sw, bias, T, rowbytes, E, S, out, s)
    if (fp8) {
        MOE_SC(true);
    }
    MOE_SC(false);
#undef MOE_SC
}

int launch_score_tiles_topk(const void* x, const void* w, const float* bias, int64_t T,
                            int rowbytes, int E, int k, int renorm, float* logits, int32_t* idx,
                            float* gate, hipStream_t s) {
    const uint8_t* xb = (const uint8_t*)x;
    const uint8_t* wb = (const uint8_t*)w;
#define MOE_ST(KM) \
    launch_topk_by_width<KM>(xb, wb, bias, T, rowbytes, E, k, renorm, logits, idx, gate, s)
    if (k <= 2) return MOE_ST(2);
    if (k <= 4) return MOE_ST(4);
    if (k <= 8) return MOE_ST(8);
    return MOE_ST(MOE_MAX_K);
#undef MOE_ST
}

}  // namespace moe
