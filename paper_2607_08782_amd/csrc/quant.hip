// Quantized routing predictor (Sec. V-A of the Director paper: a low-bit
// replica of the model, weights and activations quantized, whose gate scores
// rank experts almost as the full-precision gate does; its accuracy is the
// top-k match rate of Sec. VIII).  On gfx950 the natural low-bit format is
// FP8 E4M3, which the matrix cores multiply natively
// (v_mfma_scale_f32_32x32x64_f8f6f4).
//
//   quantize   one workgroup per row: |max| -> scale = max/448 (fp32), codes =
//              E4M3 round-to-nearest-even of x/scale (fp32 division), stored
//              as bytes; the row's largest magnitude maps to +-448
//   q-router   logits[t][e] = s_x[t] s_w[e] sum_i q_x[t][i] q_w[e][i] + b[e]:
//              32 tokens x all experts per workgroup, eight waves split K in
//              64-byte steps of the FP8 MFMA (unit block scales), partial
//              sums added in a fixed order in LDS (deterministic); top-k and
//              gates then run as for given scores.
#include "common.h"

namespace moe {
namespace {

constexpr int QTHREADS = 256;
constexpr int QR_TOKENS = 32;           // tokens per router workgroup (MFMA rows)
constexpr int QR_WAVES = 8;

typedef int i32x8 __attribute__((ext_vector_type(8)));

// E4M3 code of a finite fp32 value: nearest grid value, ties to the even code,
// magnitudes beyond 448 saturate; values rounding to zero give +0 (code 0).
__device__ __forceinline__ uint32_t e4m3_rne(float r) {
    const float a = fminf(fabsf(r), 448.0f);
    uint32_t code;
    if (a < 0.015625f) {                                   // below 2^-6: subnormal grid m * 2^-9
        code = (uint32_t)__builtin_rintf(a * 512.0f);      // 0..8 (8 is the smallest normal)
    } else {
        const int e = (int)((__float_as_uint(a) >> 23) & 0xff) - 127;   // -6 .. 8
        const float m = __builtin_rintf((__builtin_ldexpf(a, -e) - 1.0f) * 8.0f);   // exact, 0..8
        code = (uint32_t)((e + 7) * 8) + (uint32_t)m;      // m == 8 carries into the exponent
        if (code > 0x7eu) code = 0x7eu;
    }
    if (r < 0.0f && code != 0u) code |= 0x80u;
    return code;
}

template <typename T>
__device__ __forceinline__ float load_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_f32<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_f32<bf16_t>(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }

// Per-row maximum magnitude of a 256-thread workgroup (every thread gets it).
__device__ __forceinline__ float block_amax(float amax, float* red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    return amax;
}

__device__ __forceinline__ float row_scale(float amax) {
    return amax > 0.0f ? __fdiv_rn(amax, 448.0f) : 1.0f;
}

// Any width and alignment: one element per thread and step.
template <typename T>
__global__ __launch_bounds__(QTHREADS) void quantize_rows_kernel(const T* __restrict__ x, int64_t rows,
                                                                int cols, uint8_t* __restrict__ q,
                                                                float* __restrict__ scales) {
    __shared__ float red[QTHREADS / 64];
    const int tid = threadIdx.x;
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
        const T* xr = x + r * cols;
        float amax = 0.0f;
        for (int c = tid; c < cols; c += QTHREADS) amax = fmaxf(amax, fabsf(load_f32(xr, c)));
        const float s = row_scale(block_amax(amax, red));
        if (tid == 0) scales[r] = s;
        uint8_t* qr = q + r * cols;
        for (int c = tid; c < cols; c += QTHREADS) qr[c] = (uint8_t)e4m3_rne(__fdiv_rn(load_f32(xr, c), s));
    }
}

// Eight consecutive elements as fp32 (16-byte bf16 or 32-byte fp32 loads).
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
    const uint4 u = *(const uint4*)p;
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8(const float* p, float* v) {
    const float4 a = ((const float4*)p)[0], b = ((const float4*)p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ uint2 encode8(const float* v, float s) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        lo |= e4m3_rne(__fdiv_rn(v[i], s)) << (8 * i);
        hi |= e4m3_rne(__fdiv_rn(v[4 + i], s)) << (8 * i);
    }
    return make_uint2(lo, hi);
}

// cols % 8 == 0, rows 16-byte aligned (x) and 8-byte aligned (q): each thread
// owns 8-element chunks tid, tid + 256, ...; the first CH of them stay in
// registers between the maximum and the encoding, later ones are read again.
template <typename T, int CH>
__global__ __launch_bounds__(QTHREADS) void quantize_rows_vec_kernel(const T* __restrict__ x,
                                                                    int64_t rows, int cols,
                                                                    uint8_t* __restrict__ q,
                                                                    float* __restrict__ scales) {
    __shared__ float red[QTHREADS / 64];
    const int tid = threadIdx.x;
    const int nchunk = cols / 8;
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
        const T* xr = x + r * cols;
        float v[CH][8];
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = tid + i * QTHREADS;
            load8(xr + (c < nchunk ? c : 0) * 8, v[i]);     // in-bounds, masked below
        }
#pragma unroll
        for (int i = 0; i < CH; ++i)
            if (tid + i * QTHREADS < nchunk)
#pragma unroll
                for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(v[i][j]));
        for (int c = tid + CH * QTHREADS; c < nchunk; c += QTHREADS) {
            float t[8];
            load8(xr + c * 8, t);
#pragma unroll
            for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(t[j]));
        }
        const float s = row_scale(block_amax(amax, red));
        if (tid == 0) scales[r] = s;
        uint8_t* qr = q + r * cols;
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = tid + i * QTHREADS;
            if (c < nchunk) *(uint2*)(qr + c * 8) = encode8(v[i], s);
        }
        for (int c = tid + CH * QTHREADS; c < nchunk; c += QTHREADS) {
            float t[8];
            load8(xr + c * 8, t);
            *(uint2*)(qr + c * 8) = encode8(t, s);
        }
    }
}

// One workgroup: QR_TOKENS tokens x ET tiles of 32 experts.  Lane l of a wave
// holds token (or expert) row l % 32 and bytes [32 * (l / 32), +32) of a
// 64-byte K step; A and B use the same K order, so the sum runs over all K.
// Wave w takes the K steps w, w + QR_WAVES, ... with the next step's operands
// loaded while the current step's products run.
constexpr uint32_t QR_RSRC_WORD3 = 0x00020000;     // raw buffer, 32-bit data format
constexpr int QR_OOB = 0x7fffffc0;                 // an offset past every descriptor's range

__device__ __forceinline__ i32x8 qr_load32(__amdgpu_buffer_rsrc_t r, int voff) {
    const uint4 lo = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
    const uint4 hi = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 16, 0));
    return (i32x8){(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Operands of one 64-byte K step at byte kb: rows past the block's tokens or
// past E fall outside the descriptors and read as zero, so every load is
// issued unconditionally (the compiler keeps them in flight).
template <int ET>
__device__ __forceinline__ void qroute_load(__amdgpu_buffer_rsrc_t xr, __amdgpu_buffer_rsrc_t wr,
                                            int d, int row, int kb, bool valid, i32x8& a,
                                            i32x8 (&b)[ET]) {
    a = qr_load32(xr, valid ? row * d + kb : QR_OOB);
#pragma unroll
    for (int j = 0; j < ET; ++j) b[j] = qr_load32(wr, valid ? (j * 32 + row) * d + kb : QR_OOB);
}

template <int ET>
__global__ __launch_bounds__(QR_WAVES * 64) void qroute_kernel(
    const uint8_t* __restrict__ xq, const float* __restrict__ sx, const uint8_t* __restrict__ wq,
    const float* __restrict__ sw, const float* __restrict__ bias, int64_t T, int d, int E,
    float* __restrict__ logits) {
    __shared__ f32x16 red[2][ET][64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * QR_TOKENS;
    const int row = lane & 31, half = lane >> 5;
    const int nt = (int)((T - t0) < QR_TOKENS ? (T - t0) : QR_TOKENS);
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(xq + t0 * d), (short)0, nt * d, QR_RSRC_WORD3);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)wq, (short)0, E * d, QR_RSRC_WORD3);
    f32x16 acc[ET];
#pragma unroll
    for (int j = 0; j < ET; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    // wave w takes K steps w, w + QR_WAVES, ...; the loads of a step past its
    // last get out-of-range offsets (zeros, no memory traffic), so the loops
    // have no branches around loads and the compiler's waits stay exact
    const int ksteps = d / 64;
    const int n_mine = wave < ksteps ? (ksteps - wave + QR_WAVES - 1) / QR_WAVES : 0;
    const int koff = half * 32;
    auto mma = [&](const i32x8& a_, const i32x8 (&b_)[ET]) {
#pragma unroll
        for (int j = 0; j < ET; ++j)
            acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a_, b_[j], acc[j], 0, 0, 0, 127,
                                                                     0, 127);
    };
    auto kb_of = [&](int i) { return (wave + i * QR_WAVES) * 64 + koff; };
    if constexpr (ET <= 4) {
        // two steps of loads in flight (ring of two operand sets, by step parity)
        i32x8 a0, b0[ET], a1, b1[ET];
        qroute_load<ET>(xr, wr, d, row, kb_of(0), 0 < n_mine, a0, b0);
        qroute_load<ET>(xr, wr, d, row, kb_of(1), 1 < n_mine, a1, b1);
        for (int i = 0; i < n_mine; i += 2) {
            mma(a0, b0);
            qroute_load<ET>(xr, wr, d, row, kb_of(i + 2), i + 2 < n_mine, a0, b0);
            mma(a1, b1);                          // zeros when i + 1 == n_mine
            qroute_load<ET>(xr, wr, d, row, kb_of(i + 3), i + 3 < n_mine, a1, b1);
        }
    } else {
        // eight expert tiles: registers for one operand set
        i32x8 a, b[ET];
        qroute_load<ET>(xr, wr, d, row, kb_of(0), 0 < n_mine, a, b);
        for (int i = 0; i < n_mine; ++i) {
            mma(a, b);
            qroute_load<ET>(xr, wr, d, row, kb_of(i + 1), i + 1 < n_mine, a, b);
        }
    }
    // fixed-order reduction in the MFMA output layout: slice g = wave & 1
    // receives waves g, g+2, g+4, g+6 in turn, then the two slices are added.
    const int g = wave & 1, q = wave >> 1;
    for (int pass = 0; pass < QR_WAVES / 2; ++pass) {
        if (q == pass) {
#pragma unroll
            for (int j = 0; j < ET; ++j) {
                f32x16* p = &red[g][j][lane];
                *p = pass == 0 ? acc[j] : *p + acc[j];
            }
        }
        __syncthreads();
    }
    // item = (tile j, row quad rq, lane ln): rows 8 rq + 4 (ln / 32) + m, m < 4, of
    // expert column 32 j + ln % 32 (the accumulator layout of the 32x32 MFMA)
    const float* r0 = (const float*)&red[0][0][0];
    const float* r1 = (const float*)&red[1][0][0];
    for (int it = tid; it < ET * 256; it += QR_WAVES * 64) {
        const int j = it >> 8, rq = (it >> 6) & 3, ln = it & 63;
        const int e = j * 32 + (ln & 31);
        if (e >= E) continue;
        const int o = (j * 64 + ln) * 16 + rq * 4;
        const float4 a = *(const float4*)(r0 + o), b = *(const float4*)(r1 + o);
        const float s_w = sw[e], b_e = bias ? bias[e] : 0.0f;
        const float v[4] = {a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w};
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t t = t0 + rq * 8 + (ln >> 5) * 4 + m;
            if (t < T) {
                float x = v[m] * sx[t] * s_w;
                if (bias) x += b_e;
                logits[t * E + e] = x;
            }
        }
    }
}

}  // namespace

int launch_quantize_e4m3(const void* x, int dtype, int64_t rows, int cols, uint8_t* q, float* scales,
                         hipStream_t s) {
    if (rows == 0) return MOE_OK;
    const unsigned grid = (unsigned)(rows < 8192 ? rows : 8192);
    const size_t xb = dtype == MOE_BF16 ? 2 : 4;
    const bool vec = cols % 8 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 7) == 0 &&
                     ((size_t)cols * xb) % 16 == 0;
    if (vec) {
        const int per_thread = (int)ceil_div(cols / 8, QTHREADS);
#define QV(CH)                                                                                      \
    if (per_thread <= CH || CH == 4) {                                                              \
        if (dtype == MOE_BF16)                                                                      \
            hipLaunchKernelGGL((quantize_rows_vec_kernel<bf16_t, CH>), dim3(grid), dim3(QTHREADS), 0, \
                               s, (const bf16_t*)x, rows, cols, q, scales);                         \
        else                                                                                        \
            hipLaunchKernelGGL((quantize_rows_vec_kernel<float, CH>), dim3(grid), dim3(QTHREADS), 0,  \
                               s, (const float*)x, rows, cols, q, scales);                          \
        return launch_status();                                                                     \
    }
        QV(1) QV(2) QV(4)
#undef QV
    }
    if (dtype == MOE_BF16)
        hipLaunchKernelGGL(quantize_rows_kernel<bf16_t>, dim3(grid), dim3(QTHREADS), 0, s,
                           (const bf16_t*)x, rows, cols, q, scales);
    else
        hipLaunchKernelGGL(quantize_rows_kernel<float>, dim3(grid), dim3(QTHREADS), 0, s,
                           (const float*)x, rows, cols, q, scales);
    return launch_status();
}

int launch_route_topk_e4m3(const uint8_t* xq, const float* sx, const uint8_t* wq, const float* sw,
                           const float* bias, int64_t T, int d, int E, int k, int flags,
                           float* logits, int32_t* idx, float* gate, hipStream_t s) {
    if (T == 0) return MOE_OK;
    if (score_tiles_split(T, d, E, false) == 1) {  // long batch over many experts
        const int st = launch_score_tiles(true, xq, wq, sx, sw, bias, T, d, E, 1, logits, s);
        if (st != MOE_OK) return st;
        return launch_topk_given(logits, T, E, k, flags, idx, gate, s);
    }
    const unsigned grid = (unsigned)ceil_div(T, QR_TOKENS);
    const int et = (int)ceil_div(E, 32);
#define QR(N)                                                                                   \
    if (et <= N) {                                                                              \
        hipLaunchKernelGGL(qroute_kernel<N>, dim3(grid), dim3(QR_WAVES * 64), 0, s, xq, sx, wq, sw, \
                           bias, T, d, E, logits);                                              \
    } else
    QR(1) QR(2) QR(4) QR(8) {}
#undef QR
    const int st = launch_status();
    if (st != MOE_OK) return st;
    return launch_topk_given(logits, T, E, k, flags, idx, gate, s);
}

}  // namespace moe
