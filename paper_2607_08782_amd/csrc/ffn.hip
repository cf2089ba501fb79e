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
//   workgroup 256 threads = 4 waves (2 x 2), macro tile 128 rows x 256 weight
//   rows, K step 64, LDS double buffer (2 x 55 KiB), wave tile 64 x 128 on
//   v_mfma_f32_32x32x16_bf16 (2 x 4 accumulator tiles).
//   The grid is persistent (one workgroup per CU).  Tiles are ordered
//   (group, n-tile, m-tile) and cut into eight contiguous chunks, one per XCD
//   (workgroups are dispatched round-robin over the XCDs), so the workgroups
//   sharing an L2 also share weight tiles.  Group sizes are read on the
//   device; empty groups produce no tiles, so their weights are never read.
#include "common.h"

namespace moe {
namespace {

constexpr int BM = 128;          // rows per tile
constexpr int BNW = 256;         // weight rows per tile
constexpr int BK = 64;           // K per stage
constexpr int LDK = BK + 8;      // LDS row stride in elements (144 B: conflict-free reads)
constexpr int GEMM_THREADS = 256;
constexpr int NUM_XCD = 8;

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
template <bool SWIGLU>
__device__ __forceinline__ int b_sub_row(int wn, int jj) {
    return SWIGLU ? ((jj >> 1) * 128 + wn * 64 + (jj & 1) * 32) : (wn * 128 + jj * 32);
}

template <bool SWIGLU>
__global__ __launch_bounds__(GEMM_THREADS) void grouped_gemm_kernel(GemmArgs args) {
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNW * LDK];
    __shared__ int s_off[MOE_MAX_GROUPS + 1];
    __shared__ int s_tstart[MOE_MAX_GROUPS + 1];
    __shared__ int s_cur[4];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;
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

        // per-thread global source rows: A rows (tid>>3) + 32*i, B rows (tid>>3) + 32*i
        const int kc = (tid & 7) * 8;
        const bf16_t* aptr[4];
        bool aok[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = (tid >> 3) + 32 * i;
            aok[i] = r < rows_valid;
            aptr[i] = args.a + (int64_t)(row0 + (aok[i] ? r : 0)) * K + kc;
        }
        const bf16_t* bptr[8];
        bool bok[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = (tid >> 3) + 32 * i;
            int col, wrow;
            if (SWIGLU) {
                col = n0 + (r & 127);
                wrow = (r < 128 ? 0 : args.up_row) + col;
            } else {
                col = n0 + r;
                wrow = col;
            }
            bok[i] = col < args.N;
            bptr[i] = W + (int64_t)(bok[i] ? wrow : 0) * K + kc;
        }

        uint4 ra[4], rb[8];
        auto gload = [&](int kt) {
            const int k0 = kt * BK;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                ra[i] = aok[i] ? *(const uint4*)(aptr[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                rb[i] = bok[i] ? *(const uint4*)(bptr[i] + k0) : make_uint4(0, 0, 0, 0);
        };
        auto sstore = [&](int buf) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *(uint4*)&As[buf][((tid >> 3) + 32 * i) * LDK + kc] = ra[i];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                *(uint4*)&Bs[buf][((tid >> 3) + 32 * i) * LDK + kc] = rb[i];
        };

        f32x16 acc[2][4];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mi][jj][r] = 0.f;

        gload(0);
        sstore(0);
        __syncthreads();
        const int frag_col = (lane >> 5) * 32;
        const int frag_row = lane & 31;
        for (int kt = 0; kt < KT; ++kt) {
            const int buf = kt & 1;
            if (kt + 1 < KT) gload(kt + 1);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                bf16x8 af[2], bfr[4];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
                    af[mi] = *(const bf16x8*)&As[buf][(wm * 64 + mi * 32 + frag_row) * LDK +
                                                      frag_col + kk * 8];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
                    bfr[jj] = *(const bf16x8*)&Bs[buf][(b_sub_row<SWIGLU>(wn, jj) + frag_row) * LDK +
                                                       frag_col + kk * 8];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
                        acc[mi][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[jj],
                                                                              acc[mi][jj], 0, 0, 0);
            }
            if (kt + 1 < KT) sstore(buf ^ 1);
            __syncthreads();
        }

        // epilogue: accumulator element r of a 32x32 tile sits at
        // row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
        const int col_in = lane & 31;
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row_in = wm * 64 + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (row_in >= rows_valid) continue;
                bf16_t* orow = args.out + (int64_t)(row0 + row_in) * args.ldo;
                if (SWIGLU) {
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const int col = n0 + wn * 64 + j * 32 + col_in;
                        if (col < args.N) orow[col] = f32_to_bf16(silu(acc[mi][j][r]) * acc[mi][2 + j][r]);
                    }
                } else {
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const int col = n0 + wn * 128 + jj * 32 + col_in;
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
