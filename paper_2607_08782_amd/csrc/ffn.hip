// Grouped SwiGLU expert FFN over ragged groups of rows (Sec. II-A of the
// Director paper: each expert is an FFN sub-network; Eq. 2 prices this step
// as the per-GPU compute latency f_comp of the rows a GPU receives).
//
// bf16 path, two launches of one persistent MFMA kernel:
//   1. H = SiLU(X W1^T) * (X W3^T)   gate and up tiles side by side in one
//                                     256-row weight tile, fused epilogue
//   2. Y = H W2^T
// Both products are "NT": every operand row is contiguous along K, so global
// loads, LDS stores and MFMA fragment reads are all 16-byte vectors.
//
// Kernel shape (gfx950, wave64):
//   workgroup 512 threads = 8 waves (4 x 2, two per SIMD), macro tile 256 rows
//   x 256 weight rows, K step 64, LDS double buffer (2 x 72 KiB), wave tile
//   64 x 128 on v_mfma_f32_32x32x16_bf16 (2 x 4 accumulator tiles), fragment
//   reads software-pipelined against the MFMAs.
//   The grid is persistent (one workgroup per CU).  Tiles are ordered
//   (group, n-tile, m-tile) and cut into eight contiguous chunks, one per XCD
//   (workgroups are dispatched round-robin over the XCDs), so the workgroups
//   sharing an L2 also share weight tiles.  Group sizes are read on the
//   device; empty groups produce no tiles, so their weights are never read.
#include "common.h"

namespace moe {
namespace {

constexpr int BM = 256;          // rows per tile
constexpr int BNW = 256;         // weight rows per tile
constexpr int BK = 64;           // K per stage
constexpr int LDK = BK + 8;      // LDS row stride in elements (144 B: conflict-free reads)
constexpr int WAVES_M = 4, WAVES_N = 2;
constexpr int GEMM_THREADS = WAVES_M * WAVES_N * 64;
constexpr int MS = BM / WAVES_M / 32;              // 32-row accumulator tiles per wave
constexpr int NS = BNW / WAVES_N / 32;             // 32-column accumulator tiles per wave
constexpr int ROWS_PER_PASS = GEMM_THREADS / 8;    // rows one pass of 16-byte loads covers
constexpr int A_PER = BM / ROWS_PER_PASS;          // 16-byte loads per thread per stage (A)
constexpr int B_PER = BNW / ROWS_PER_PASS;         // (B)
constexpr int NUM_XCD = 8;
constexpr uint32_t RSRC_WORD3 = 0x00020000;        // raw buffer: 32-bit data format

struct GemmArgs {
    const bf16_t* w[MOE_MAX_GROUPS];   // per-group weight matrix, rows contiguous along K
    const int32_t* offsets;            // [n_groups + 1] row offsets (device)
    const bf16_t* a;                   // [rows][K]
    bf16_t* out;                       // [rows][ldo]
    int n_groups;
    int K;                             // contraction length
    int N;                             // output columns per group (f for SWIGLU, d for PLAIN)
    int ldo;
    int up_row;                        // SWIGLU: first row of W3 inside w[s] (= f)
    int n_tiles;                       // output-column tiles per group
};

// B-tile row of the jj-th 32-wide accumulator column block of wave column wn.
// SwiGLU tiles hold 128 gate rows then the matching 128 up rows; a wave takes
// the same columns from both halves, so gate and up meet in its registers.
template <bool SWIGLU>
__device__ __forceinline__ int b_sub_row(int wn, int jj) {
    if (SWIGLU) {
        constexpr int HW = BNW / 2 / WAVES_N;
        return jj < NS / 2 ? wn * HW + jj * 32 : BNW / 2 + wn * HW + (jj - NS / 2) * 32;
    }
    return wn * (BNW / WAVES_N) + jj * 32;
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Persistent grouped NT GEMM.  Per tile: operands stream through per-tile
// buffer descriptors (rows past the group's end fall outside the descriptor and
// read as zero), are staged through registers into a double-buffered LDS
// stage, and MFMA fragments are double-buffered per 16-wide K sub-step, so the
// LDS reads of sub-step q+1 (including across the stage barrier) overlap the
// MFMAs of sub-step q.
template <bool SWIGLU>
__global__ __launch_bounds__(GEMM_THREADS) void grouped_gemm_kernel(GemmArgs args) {
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNW * LDK];
    __shared__ int s_off[MOE_MAX_GROUPS + 1];
    __shared__ int s_tstart[MOE_MAX_GROUPS + 1];
    __shared__ int s_cur[4];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;
    const int n_groups = args.n_groups;
    const int BN_OUT = SWIGLU ? BNW / 2 : BNW;      // output columns per tile

    for (int s = tid; s <= n_groups; s += GEMM_THREADS) s_off[s] = args.offsets[s];
    __syncthreads();
    if (tid == 0) {
        int acc = 0;
        s_tstart[0] = 0;
        for (int s = 0; s < n_groups; ++s) {
            const int rows = s_off[s + 1] - s_off[s];
            acc += (int)ceil_div(rows > 0 ? rows : 0, BM) * args.n_tiles;
            s_tstart[s + 1] = acc;
        }
    }
    __syncthreads();
    const int total = s_tstart[n_groups];
    const int nper = gridDim.x / NUM_XCD;
    const int xcd = blockIdx.x % NUM_XCD;
    const int widx = blockIdx.x / NUM_XCD;
    const int chunk = (total + NUM_XCD - 1) / NUM_XCD;
    const int t_begin = xcd * chunk;
    const int t_end = min(t_begin + chunk, total);
    const int KT = args.K / BK;
    const int K = args.K;
    const int kc = (tid & 7) * 8;
    const int voff = ((tid >> 3) * K + kc) * 2;
    const int vstep = ROWS_PER_PASS * K * 2;
    const int frag_col = (lane >> 5) * 32;
    const int frag_row = lane & 31;

    for (int L = t_begin + widx; L < t_end; L += nper) {
        if (tid == 0) {
            int s = 0;
            while (s + 1 < n_groups && s_tstart[s + 1] <= L) ++s;
            const int rows = s_off[s + 1] - s_off[s];
            const int mt = (int)ceil_div(rows, BM);
            const int local = L - s_tstart[s];
            const int nt = local / mt;
            s_cur[0] = s;
            s_cur[1] = (local - nt * mt) * BM;
            s_cur[2] = nt;
        }
        __syncthreads();
        const int g = s_cur[0];
        const int m0 = s_cur[1];
        const int n0 = s_cur[2] * BN_OUT;
        const int row0 = s_off[g] + m0;
        const int rows_valid = min(BM, s_off[g + 1] - row0);
        const bf16_t* __restrict__ W = args.w[g];

        const __amdgpu_buffer_rsrc_t arsrc = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(args.a + (int64_t)row0 * K), (short)0, rows_valid * K * 2, RSRC_WORD3);
        const int bvalid = min(BN_OUT, args.N - n0);
        const int bup = SWIGLU ? args.up_row + n0 : n0;
        const __amdgpu_buffer_rsrc_t brsrc_lo = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(W + (int64_t)n0 * K), (short)0, bvalid * K * 2, RSRC_WORD3);
        const __amdgpu_buffer_rsrc_t brsrc_hi = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(W + (int64_t)bup * K), (short)0, bvalid * K * 2, RSRC_WORD3);

        uint4 ra[A_PER], rb[B_PER];
        auto gload = [&](int kt) {
            const int so = kt * BK * 2;
#pragma unroll
            for (int i = 0; i < A_PER; ++i) ra[i] = buffer_load16(arsrc, voff + i * vstep, so);
#pragma unroll
            for (int i = 0; i < B_PER; ++i) {
                if (SWIGLU && i >= B_PER / 2)
                    rb[i] = buffer_load16(brsrc_hi, voff + (i - B_PER / 2) * vstep, so);
                else
                    rb[i] = buffer_load16(brsrc_lo, voff + i * vstep, so);
            }
        };
        auto sstore = [&](int buf) {
#pragma unroll
            for (int i = 0; i < A_PER; ++i)
                *(uint4*)&As[buf][((tid >> 3) + ROWS_PER_PASS * i) * LDK + kc] = ra[i];
#pragma unroll
            for (int i = 0; i < B_PER; ++i)
                *(uint4*)&Bs[buf][((tid >> 3) + ROWS_PER_PASS * i) * LDK + kc] = rb[i];
        };

        f32x16 acc[MS][NS];
#pragma unroll
        for (int mi = 0; mi < MS; ++mi)
#pragma unroll
            for (int jj = 0; jj < NS; ++jj)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mi][jj][r] = 0.f;

        const bf16_t* a_lds0 = &As[0][(wm * (BM / WAVES_M) + frag_row) * LDK + frag_col];
        const bf16_t* b_lds0 = &Bs[0][frag_row * LDK + frag_col];
        bf16x8 fa0[MS], fb0[NS], fa1[MS], fb1[NS];
        auto read = [&](int buf, int kk, bf16x8* fa, bf16x8* fb) {
#pragma unroll
            for (int mi = 0; mi < MS; ++mi)
                fa[mi] = *(const bf16x8*)(a_lds0 + buf * BM * LDK + mi * 32 * LDK + kk * 8);
#pragma unroll
            for (int jj = 0; jj < NS; ++jj)
                fb[jj] = *(const bf16x8*)(b_lds0 + buf * BNW * LDK + b_sub_row<SWIGLU>(wn, jj) * LDK +
                                          kk * 8);
        };
        auto mfma = [&](const bf16x8* fa, const bf16x8* fb) {
#pragma unroll
            for (int mi = 0; mi < MS; ++mi)
#pragma unroll
                for (int jj = 0; jj < NS; ++jj)
                    acc[mi][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mi], fb[jj],
                                                                          acc[mi][jj], 0, 0, 0);
        };

        // The K permutation inside a stage (lane half h, sub-step kk -> K offset
        // h*32 + kk*8) is the same for A and B, so the products sum over all K.
        gload(0);
        sstore(0);
        gload(KT > 1 ? 1 : 0);
        __syncthreads();
        read(0, 0, fa0, fb0);
        for (int t = 0; t < KT; ++t) {
            const int buf = t & 1;
            __builtin_amdgcn_iglp_opt(1);
            read(buf, 1, fa1, fb1);
            mfma(fa0, fb0);
            read(buf, 2, fa0, fb0);
            mfma(fa1, fb1);
            read(buf, 3, fa1, fb1);
            mfma(fa0, fb0);
            if (t + 1 < KT) {
                sstore(buf ^ 1);
                __syncthreads();
                gload(t + 2 < KT ? t + 2 : KT - 1);
                read(buf ^ 1, 0, fa0, fb0);
            }
            mfma(fa1, fb1);
        }
        __syncthreads();

        // epilogue: accumulator element r of a 32x32 tile sits at
        // row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
        const int col_in = lane & 31;
#pragma unroll
        for (int mi = 0; mi < MS; ++mi) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row_in = wm * (BM / WAVES_M) + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 +
                                   (r & 3);
                if (row_in >= rows_valid) continue;
                bf16_t* orow = args.out + (int64_t)(row0 + row_in) * args.ldo;
                if (SWIGLU) {
                    constexpr int HW = BNW / 2 / WAVES_N;
#pragma unroll
                    for (int j = 0; j < NS / 2; ++j) {
                        const int col = n0 + wn * HW + j * 32 + col_in;
                        if (col < args.N)
                            orow[col] = f32_to_bf16(silu(acc[mi][j][r]) * acc[mi][NS / 2 + j][r]);
                    }
                } else {
#pragma unroll
                    for (int jj = 0; jj < NS; ++jj) {
                        const int col = n0 + wn * (BNW / WAVES_N) + jj * 32 + col_in;
                        if (col < args.N) orow[col] = f32_to_bf16(acc[mi][jj][r]);
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 path: plain FMA loops, one thread per output element.
// ---------------------------------------------------------------------------
struct PtrTable {
    const float* p[MOE_MAX_GROUPS];
};

__device__ __forceinline__ int find_group(const int* off, int n_groups, int p) {
    int s = 0;
    while (s + 1 < n_groups && off[s + 1] <= p) ++s;
    return s;
}

__global__ __launch_bounds__(256) void ffn1_f32_kernel(const float* __restrict__ x,
                                                       const int32_t* __restrict__ offsets,
                                                       int n_groups, PtrTable w13, int d, int f,
                                                       float* __restrict__ h) {
    __shared__ int s_off[MOE_MAX_GROUPS + 1];
    for (int s = threadIdx.x; s <= n_groups; s += blockDim.x) s_off[s] = offsets[s];
    __syncthreads();
    const int64_t N = s_off[n_groups];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N * f;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int p = (int)(i / f), j = (int)(i % f);
        const int s = find_group(s_off, n_groups, p);
        const float* W = w13.p[s];
        const float* xr = x + (int64_t)p * d;
        float a = 0.f, b = 0.f;
        for (int q = 0; q < d; ++q) {
            a = fmaf(W[(int64_t)j * d + q], xr[q], a);
            b = fmaf(W[(int64_t)(f + j) * d + q], xr[q], b);
        }
        h[i] = a / (1.0f + expf(-a)) * b;
    }
}

__global__ __launch_bounds__(256) void ffn2_f32_kernel(const float* __restrict__ h,
                                                       const int32_t* __restrict__ offsets,
                                                       int n_groups, PtrTable w2, int d, int f,
                                                       float* __restrict__ y) {
    __shared__ int s_off[MOE_MAX_GROUPS + 1];
    for (int s = threadIdx.x; s <= n_groups; s += blockDim.x) s_off[s] = offsets[s];
    __syncthreads();
    const int64_t N = s_off[n_groups];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N * d;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int p = (int)(i / d), o = (int)(i % d);
        const int s = find_group(s_off, n_groups, p);
        const float* W = w2.p[s] + (int64_t)o * f;
        const float* hr = h + (int64_t)p * f;
        float acc = 0.f;
        for (int j = 0; j < f; ++j) acc = fmaf(W[j], hr[j], acc);
        y[i] = acc;
    }
}

int num_cus() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

}  // namespace

size_t grouped_ffn_ws_bytes(int dtype, int64_t cap_rows, int d, int f, int n_groups) {
    (void)d; (void)n_groups;
    const size_t esize = dtype == MOE_BF16 ? 2 : 4;
    return (size_t)cap_rows * (size_t)f * esize + 256;
}

int launch_grouped_ffn(const void* x_perm, int dtype, const int32_t* offsets, int n_groups,
                       const void* const* w13, const void* const* w2, int d, int f,
                       int64_t cap_rows, void* y_perm, void* ws, hipStream_t s) {
    if (cap_rows == 0) return MOE_OK;
    if (dtype == MOE_F32) {
        PtrTable t13, t2;
        for (int i = 0; i < MOE_MAX_GROUPS; ++i) {
            t13.p[i] = i < n_groups ? (const float*)w13[i] : nullptr;
            t2.p[i] = i < n_groups ? (const float*)w2[i] : nullptr;
        }
        float* h = (float*)ws;
        int64_t b1 = ceil_div(cap_rows * (int64_t)f, 256), b2 = ceil_div(cap_rows * (int64_t)d, 256);
        if (b1 > 4096) b1 = 4096;
        if (b2 > 4096) b2 = 4096;
        hipLaunchKernelGGL(ffn1_f32_kernel, dim3((unsigned)b1), dim3(256), 0, s,
                           (const float*)x_perm, offsets, n_groups, t13, d, f, h);
        hipLaunchKernelGGL(ffn2_f32_kernel, dim3((unsigned)b2), dim3(256), 0, s, (const float*)h,
                           offsets, n_groups, t2, d, f, (float*)y_perm);
        return launch_status();
    }
    const int grid = (num_cus() / NUM_XCD) * NUM_XCD;
    bf16_t* h = (bf16_t*)ws;
    GemmArgs a1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) a1.w[i] = i < n_groups ? (const bf16_t*)w13[i] : nullptr;
    a1.offsets = offsets;
    a1.a = (const bf16_t*)x_perm;
    a1.out = h;
    a1.n_groups = n_groups;
    a1.K = d;
    a1.N = f;
    a1.ldo = f;
    a1.up_row = f;
    a1.n_tiles = (int)ceil_div(f, BNW / 2);
    hipLaunchKernelGGL(grouped_gemm_kernel<true>, dim3(grid), dim3(GEMM_THREADS), 0, s, a1);
    GemmArgs a2 = a1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) a2.w[i] = i < n_groups ? (const bf16_t*)w2[i] : nullptr;
    a2.a = h;
    a2.out = (bf16_t*)y_perm;
    a2.K = f;
    a2.N = d;
    a2.ldo = d;
    a2.up_row = 0;
    a2.n_tiles = (int)ceil_div(d, BNW);
    hipLaunchKernelGGL(grouped_gemm_kernel<false>, dim3(grid), dim3(GEMM_THREADS), 0, s, a2);
    return launch_status();
}

}  // namespace moe
