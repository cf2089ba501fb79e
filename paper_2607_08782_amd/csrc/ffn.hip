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
//   x 256 weight rows, K step 64, LDS double buffer (2 x 64 KiB, 128-byte rows
//   with XOR-swizzled 16-byte chunks), wave tile 64 x 128 on
//   v_mfma_f32_16x16x32_bf16 (4 x 8 accumulator tiles), fragment reads
//   software-pipelined against the MFMAs.  Under sustained load the part runs
//   at its board power limit, so the clock follows the energy spent per flop:
//   16x16x32 moves half the accumulator bytes per flop of 32x32x16 and runs
//   these loops at a higher clock.
//   The grid is persistent (one workgroup per CU).  Tiles are ordered
//   (group, n-tile, m-tile) and cut into eight contiguous chunks, one per XCD
//   (workgroups are dispatched round-robin over the XCDs), so the workgroups
//   sharing an L2 also share weight tiles.  A workgroup's tiles form one load
//   pipeline: the next tile's first stages are loaded during the current
//   tile's last step, so a tile starts without waiting for its operands.  The
//   epilogue stores 8 bytes per lane (four columns of one row, gathered by a
//   4 x 4 transpose inside each lane quad).  Group sizes are read on the
//   device; empty groups produce no tiles, so their weights are never read.
#include "common.h"

namespace moe {
namespace {

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = 256;          // rows per tile
constexpr int BNW = 256;         // weight rows per tile
constexpr int BK = 64;           // K per stage
constexpr int LDK = BK + 8;      // LDS row stride in elements (144 B: conflict-free reads)
constexpr int TLDK = BK;         // tiled kernel: 128-byte rows, 16-byte chunks XOR-swizzled
constexpr int WAVES_M = 4, WAVES_N = 2;
constexpr int GEMM_THREADS = WAVES_M * WAVES_N * 64;
constexpr int MS = BM / WAVES_M / 16;              // 16-row accumulator tiles per wave
constexpr int NS = BNW / WAVES_N / 16;             // 16-column accumulator tiles per wave
constexpr int NH = NS / 2;                         // column tiles per half sub-step
constexpr int ROWS_PER_PASS = GEMM_THREADS / 8;    // rows one pass of 16-byte loads covers
constexpr int A_PER = BM / ROWS_PER_PASS;          // 16-byte loads per thread per stage (A)
constexpr int B_PER = BNW / ROWS_PER_PASS;         // (B)
constexpr int NUM_XCD = 8;
// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_MFMA = 0x008, SG_VMEM_READ = 0x020, SG_DS_READ = 0x100, SG_DS_WRITE = 0x200;
constexpr uint32_t RSRC_WORD3 = 0x00020000;        // raw buffer: 32-bit data format
constexpr int A_OOB = 0x7fffff00;                  // offset past any descriptor: reads zero

// First row of group g.  The first `lead` groups hold lead_rows rows each (the
// shared experts' groups of moe_grouped_ffn_rows_shared, every token once); the
// offsets array gives the row ranges of the groups after them, counted from
// row lead * lead_rows, as moe_permute writes them.
__device__ __forceinline__ int group_start(const int32_t* offsets, int lead, int lead_rows, int g) {
    return g < lead ? g * lead_rows : lead * lead_rows + offsets[g - lead];
}

struct GemmArgs {
    const bf16_t* w[MOE_MAX_GROUPS];   // per-group weight matrix, rows contiguous along K
    const int32_t* offsets;            // [n_groups - lead + 1] row offsets (device), see group_start
    const bf16_t* a;                   // [rows][K]
    bf16_t* out;                       // [rows][ldo]
    int n_groups;                      // lead groups included
    int lead, lead_rows;               // leading groups of lead_rows rows each (group_start)
    int K;                             // contraction length
    int N;                             // output columns per group (f for SWIGLU, d for PLAIN)
    int ldo;
    int up_row;                        // SWIGLU: first row of W3 inside w[s] (= f)
    int n_tiles;                       // output-column tiles per group
    int* limits;                       // [2] row limits of the streamed groups of the gate/up and
                                       // the down product (small_limits): the gate/up launch
                                       // writes both, later launches read theirs; nullptr: the
                                       // limit is lim0
    int product;                       // 0 gate/up, 1 down
    int lim0;                          // row limit of streamed groups when limits is nullptr
    int down_tiles;                    // gate/up launch: the down product's column tiles
    float* part;                       // fp32 partial tiles for split K (nullptr: never split)
    int* split_info;                   // the kernel records its split factor here for the reduce
    int split_units;                   // workgroups split K aims to occupy (<= TILE_SPLIT_UNITS)
    const int32_t* a_rows;             // gather: row p of A is a[a_rows[p]] (a holds a_total rows)
    int a_total;
};

// With fewer tiles than half the workgroups (mid-sized groups: a few 256-row
// tiles, long K), each tile's K range may be cut into S chunks of at least
// TILE_SPLIT_MIN_STEPS stages; every (tile, chunk) unit writes an fp32 partial
// tile and split_reduce_kernel sums the chunks in order and applies the epilogue.
// S minimises (rounds of units) x (K stages per unit) plus the partial-tile
// round trip, about 1/20 of a stage per unit (256 KB written and read back).
constexpr int TILE_SPLIT_UNITS = 256;
constexpr int TILE_SPLIT_MIN_STEPS = 8;

// A short call (see small_limits) streams its groups of up to SMALL_ROWS_MAX rows
// through the split-K streaming kernel and tiles the rest; any other call tiles
// every group.  Without the row limits in the workspace (a call of at most
// SMALL_ROWS rows in all) every group is streamed.
constexpr int SMALL_ROWS = 64;
constexpr int SMALL_ROWS_MAX = 256;

__host__ __device__ __forceinline__ int tile_split(int total, int KT, int split_units) {
    if (total <= 0 || 2 * total > split_units) return 1;
    const int smax = min(split_units / total, KT / TILE_SPLIT_MIN_STEPS);
    int best = 1;
    int64_t best_cost = 20 * (int64_t)KT;
    for (int S = 2; S <= smax; ++S) {
        const int64_t rounds = ((int64_t)total * S + split_units - 1) / split_units;
        const int64_t cost = 20 * rounds * ((KT + S - 1) / S) + (int64_t)S * total;
        if (cost < best_cost) { best_cost = cost; best = S; }
    }
    return best;
}

// Which tiles split: with few tiles all of them; otherwise only the tiles of a
// last round that would fill at most half the workgroups (the round every
// other workgroup waits for).  Tiles [0, head) run whole; tiles
// [head, head + tail) run as S chunks each.
struct SplitPlan {
    int head, tail, S;
};

__host__ __device__ __forceinline__ SplitPlan split_plan(int total, int KT, int split_units) {
    SplitPlan p = {total, 0, 1};
    if (total <= 0) return p;
    const int rounds = total / split_units;
    const int rest = total - rounds * split_units;
    const int S = tile_split(rest, KT, split_units);
    if (S > 1) {
        p.head = total - rest;
        p.tail = rest;
        p.S = S;
    }
    return p;
}

// B-tile row of the jj-th 32-wide accumulator column block of wave column wn.
// SwiGLU tiles hold 128 gate rows then the matching 128 up rows; a wave takes
// the same columns from both halves, so gate and up meet in its registers.
template <bool SWIGLU>
__device__ __forceinline__ int b_sub_row(int wn, int jj) {
    if (SWIGLU) {
        constexpr int HW = BNW / 2 / WAVES_N;
        return jj < NS / 2 ? wn * HW + jj * 16 : BNW / 2 + wn * HW + (jj - NS / 2) * 16;
    }
    return wn * (BNW / WAVES_N) + jj * 16;
}

// 4 x 4 transpose inside each aligned quad of lanes: on entry lane 4 q + e holds
// v[r] = M[r][e] of its quad's block, on exit v[c] = M[e][c].  Two exchange
// stages (lane distance 1, then 2) with DPP quad permutations.
__device__ __forceinline__ float dpp_quad(float x, int ctrl_sel) {
    const int i = __float_as_int(x);
    return __int_as_float(ctrl_sel == 1 ? __builtin_amdgcn_mov_dpp(i, 0xB1, 0xF, 0xF, true)
                                        : __builtin_amdgcn_mov_dpp(i, 0x4E, 0xF, 0xF, true));
}

__device__ __forceinline__ void quad_transpose(float* v, int lane) {
    const bool o1 = (lane & 1) != 0, o2 = (lane & 2) != 0;
#pragma unroll
    for (int r = 0; r < 4; r += 2) {          // lanes e, e ^ 1 swap elements r ^ 1
        const float recv = dpp_quad(o1 ? v[r] : v[r + 1], 1);
        v[r] = o1 ? recv : v[r];
        v[r + 1] = o1 ? v[r + 1] : recv;
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {             // lanes e, e ^ 2 swap elements r ^ 2
        const float recv = dpp_quad(o2 ? v[r] : v[r + 2], 2);
        v[r] = o2 ? recv : v[r];
        v[r + 2] = o2 ? v[r + 2] : recv;
    }
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// s_tstart[g] = tiles of the groups before g, for g = 0..n_groups (a group of
// more than small_rows rows has ceil(rows / BM) * n_tiles tiles, others none);
// run by one whole wave.
__device__ __forceinline__ void tile_starts(const int* s_off, int n_groups, int small_rows,
                                            int n_tiles, int* s_tstart, int lane) {
    int carry = 0;
    for (int g0 = 0; g0 < n_groups; g0 += 64) {
        const int g = g0 + lane;
        const int rows = g < n_groups ? s_off[g + 1] - s_off[g] : 0;
        const int v = rows > small_rows ? (int)ceil_div(rows, BM) * n_tiles : 0;
        const int incl = wave_incl_scan(v, lane);
        if (g < n_groups) s_tstart[g + 1] = carry + incl;
        carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) s_tstart[0] = 0;
}

// Row limits of the streamed groups of the two products, run by one whole wave.
// When the groups above SMALL_ROWS rows make so few tiles (a quarter of the
// split units or fewer) that the tiled kernel would split K over them, its
// launch is short and latency-bound: every workgroup still runs several K
// stages of a 256 x 256 tile, on a fraction of the CUs.  Streaming every group
// of up to SMALL_ROWS_MAX rows instead spreads the weight reads over all CUs
// (a DeepSeek-V2-Lite-shaped decode step: 219 -> 188 us).  Otherwise the small
// groups join the tiled launch, whose rounds leave CUs free for their tiles,
// rather than stream in a launch of their own after it (the two run one after
// the other): DeepSeek-V2-Lite prefill FFN 364 -> 332 us, Qwen1.5 batch 137 ->
// 129 us, Qwen3 prefill 466 -> 459 us.
__device__ __forceinline__ void small_limits(const int* s_off, int n_groups, int tiles_up,
                                             int tiles_down, int split_units, int lane,
                                             int& lim_up, int& lim_down) {
    int mt = 0;                                      // 256-row tiles of the groups > SMALL_ROWS
    for (int g0 = 0; g0 < n_groups; g0 += 64) {
        const int g = g0 + lane;
        const int rows = g < n_groups ? s_off[g + 1] - s_off[g] : 0;
        mt += rows > SMALL_ROWS ? (int)ceil_div(rows, BM) : 0;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mt += __shfl_xor(mt, o, 64);
    lim_up = 4 * mt * tiles_up <= split_units ? SMALL_ROWS_MAX : 0;
    lim_down = 4 * mt * tiles_down <= split_units ? SMALL_ROWS_MAX : 0;
}

// Persistent grouped NT GEMM.  Per tile: operands stream through per-tile
// buffer descriptors (rows past the group's end fall outside the descriptor and
// read as zero), are staged through registers into a double-buffered LDS
// stage, and MFMA fragments are double-buffered per 16-wide K sub-step, so the
// LDS reads of sub-step q+1 (including across the stage barrier) overlap the
// MFMAs of sub-step q.
// GATHER: row p of A is row a_rows[p] of args.a (the token rows themselves, so
// the packaged copy of them is never materialised).
template <bool SWIGLU, bool GATHER = false>
__global__ __launch_bounds__(GEMM_THREADS) void grouped_gemm_kernel(GemmArgs args) {
    __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * TLDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNW * TLDK];
    __shared__ int s_off[MOE_MAX_GROUPS + 1];
    __shared__ int s_tstart[MOE_MAX_GROUPS + 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;
    const int n_groups = args.n_groups;
    const int BN_OUT = SWIGLU ? BNW / 2 : BNW;      // output columns per tile

    // the down launch reads its row limit from the gate/up launch (no group can
    // exceed SMALL_ROWS when there is nowhere to keep it)
    int lim = args.limits != nullptr && args.product == 1 ? args.limits[1] : args.lim0;
    for (int s = tid; s <= n_groups; s += GEMM_THREADS)
        s_off[s] = group_start(args.offsets, args.lead, args.lead_rows, s);
    __syncthreads();
    if (wave == 0) {
        if (args.limits != nullptr && args.product == 0) {
            int lim_down;
            small_limits(s_off, n_groups, args.n_tiles, args.down_tiles, args.split_units, lane, lim,
                         lim_down);
            if (blockIdx.x == 0 && lane == 0) {
                args.limits[0] = lim;
                args.limits[1] = lim_down;
            }
        }
        tile_starts(s_off, n_groups, lim, args.n_tiles, s_tstart, lane);
    }
    __syncthreads();
    const int KT = args.K / BK;
    const int K = args.K;
    const int total_tiles = s_tstart[n_groups];
    SplitPlan plan = {total_tiles, 0, 1};
    if (args.part != nullptr) plan = split_plan(total_tiles, KT, args.split_units);
    if (args.part != nullptr && blockIdx.x == 0 && tid == 0) *args.split_info = plan.S;
    // each XCD takes a contiguous chunk of the whole tiles and a contiguous
    // chunk of the split units, so every XCD carries the same share of both
    const int nper = gridDim.x / NUM_XCD;
    const int xcd = blockIdx.x % NUM_XCD;
    const int widx = blockIdx.x / NUM_XCD;
    const int hchunk = (plan.head + NUM_XCD - 1) / NUM_XCD;
    const int h_begin = min(xcd * hchunk, plan.head), h_end = min(h_begin + hchunk, plan.head);
    const int n_units = plan.tail * plan.S;
    const int uchunk = (n_units + NUM_XCD - 1) / NUM_XCD;
    const int s_begin = min(xcd * uchunk, n_units), s_end = min(s_begin + uchunk, n_units);
    const int n_head = h_end - h_begin, n_mine = n_head + (s_end - s_begin);
    const int kc = (tid & 7) * 8;
    const int voff = ((tid >> 3) * K + kc) * 2;
    const int vstep = ROWS_PER_PASS * K * 2;

    if (widx >= n_mine) return;

    // Tile coordinates, uniform across the workgroup: every thread derives them
    // from the plan in LDS, kept in scalar registers.  Whole tile, or unit
    // u = (split tile, K chunk).
    struct Tile {
        int g, row0, rows_valid, n0, kt0, nsteps, u, split;
    };
    auto tile_at = [&](int i) {
        Tile c;
        const bool split = i >= n_head;
        const int u = split ? s_begin + (i - n_head) : 0;
        const int L = split ? plan.head + u / plan.S : h_begin + i;
        const int S = split ? plan.S : 1;
        const int kchunk = split ? u - (u / plan.S) * plan.S : 0;
        const int kt0 = (int)((int64_t)kchunk * KT / S);
        const int s = last_le(s_tstart, n_groups, L);
        const int rows = s_off[s + 1] - s_off[s];
        const int mt = (int)ceil_div(rows, BM);
        const int local = L - s_tstart[s];
        const int nt = local / mt;
        const int row0 = s_off[s] + (local - nt * mt) * BM;
        c.g = __builtin_amdgcn_readfirstlane(s);
        c.row0 = __builtin_amdgcn_readfirstlane(row0);
        c.rows_valid = __builtin_amdgcn_readfirstlane(min(BM, s_off[s + 1] - row0));
        c.n0 = __builtin_amdgcn_readfirstlane(nt) * BN_OUT;
        c.kt0 = __builtin_amdgcn_readfirstlane(kt0);
        c.nsteps = __builtin_amdgcn_readfirstlane((int)((int64_t)(kchunk + 1) * KT / S) - kt0);
        c.u = __builtin_amdgcn_readfirstlane(u);
        c.split = __builtin_amdgcn_readfirstlane(split ? 1 : 0);
        return c;
    };
    // operand descriptors of a tile: rows past the group's end fall outside the
    // A descriptor and read as zero; gate and up halves of a SwiGLU weight tile
    struct Rsrc {
        __amdgpu_buffer_rsrc_t a, lo, hi;
    };
    auto rsrc_of = [&](const Tile& c) {
        Rsrc r;
        r.a = GATHER ? __builtin_amdgcn_make_buffer_rsrc((void*)args.a, (short)0, args.a_total * K * 2,
                                                         RSRC_WORD3)
                     : __builtin_amdgcn_make_buffer_rsrc((void*)(args.a + (int64_t)c.row0 * K), (short)0,
                                                         c.rows_valid * K * 2, RSRC_WORD3);
        const bf16_t* __restrict__ W = args.w[c.g];
        const int bvalid = min(BN_OUT, args.N - c.n0);
        const int bup = SWIGLU ? args.up_row + c.n0 : c.n0;
        r.lo = __builtin_amdgcn_make_buffer_rsrc((void*)(W + (int64_t)c.n0 * K), (short)0,
                                                 bvalid * K * 2, RSRC_WORD3);
        r.hi = __builtin_amdgcn_make_buffer_rsrc((void*)(W + (int64_t)bup * K), (short)0,
                                                 bvalid * K * 2, RSRC_WORD3);
        return r;
    };
    // per-thread A row offsets (GATHER: the token rows of the tile)
    auto a_offsets = [&](const Tile& c, int* av) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i) {
            if constexpr (GATHER) {
                const int rin = (tid >> 3) + ROWS_PER_PASS * i;
                av[i] = rin < c.rows_valid ? (args.a_rows[c.row0 + rin] * K + kc) * 2 : A_OOB;
            } else {
                av[i] = voff + i * vstep;
            }
        }
    };

    uint4 ra[A_PER], rb[B_PER];
    auto gload = [&](const Rsrc& r, const int* av, int kt) {
        const int so = kt * BK * 2;
#pragma unroll
        for (int i = 0; i < A_PER; ++i) ra[i] = buffer_load16(r.a, av[i], so);
#pragma unroll
        for (int i = 0; i < B_PER; ++i) {
            if (SWIGLU && i >= B_PER / 2)
                rb[i] = buffer_load16(r.hi, voff + (i - B_PER / 2) * vstep, so);
            else
                rb[i] = buffer_load16(r.lo, voff + i * vstep, so);
        }
    };
    // 16-byte chunk c of LDS row r sits at chunk c ^ (r & 7): conflict-free for the
    // stage stores (8 lanes per row) and for the 16-row fragment reads
    const int sc = ((tid & 7) ^ ((tid >> 3) & 7)) * 8;
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < A_PER; ++i)
            *(uint4*)&As[buf][((tid >> 3) + ROWS_PER_PASS * i) * TLDK + sc] = ra[i];
#pragma unroll
        for (int i = 0; i < B_PER; ++i)
            *(uint4*)&Bs[buf][((tid >> 3) + ROWS_PER_PASS * i) * TLDK + sc] = rb[i];
    };

    f32x4 acc[MS][NS];
    // v_mfma_f32_16x16x32_bf16 fragments: lane l holds row l % 16 of a 16-row
    // block and the 8 K elements 8 (l / 16) .. of a 32-wide sub-step, for A and
    // B alike, so every product sums over the same K
    const int frow = lane & 15;
    const int fsw = lane & 7;                         // the swizzle of rows frow (+ 16 m)
    const int fc0 = ((lane >> 4) ^ fsw) * 8, fc1 = ((4 + (lane >> 4)) ^ fsw) * 8;
    const bf16_t* a_lds0 = &As[0][(wm * (BM / WAVES_M) + frow) * TLDK];
    const bf16_t* b_lds0 = &Bs[0][frow * TLDK];
    // a 32-wide sub-step q runs as two halves (column tiles 0..NH-1, NH..NS-1);
    // the fragments of the next half are read while the current half multiplies
    bf16x8 fa0[MS], fa1[MS], fb0[NH], fb1[NH];
    auto read_a = [&](int buf, int q, bf16x8* fa) {
#pragma unroll
        for (int mi = 0; mi < MS; ++mi)
            fa[mi] = *(const bf16x8*)(a_lds0 + buf * BM * TLDK + mi * 16 * TLDK + (q ? fc1 : fc0));
    };
    auto read_b = [&](int buf, int q, int h, bf16x8* fb) {
#pragma unroll
        for (int j = 0; j < NH; ++j)
            fb[j] = *(const bf16x8*)(b_lds0 + buf * BNW * TLDK +
                                     b_sub_row<SWIGLU>(wn, h * NH + j) * TLDK + (q ? fc1 : fc0));
    };
    auto mfma = [&](const bf16x8* fa, const bf16x8* fb, int h) {
#pragma unroll
        for (int mi = 0; mi < MS; ++mi)
#pragma unroll
            for (int j = 0; j < NH; ++j)
                acc[mi][h * NH + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    fa[mi], fb[j], acc[mi][h * NH + j], 0, 0, 0);
    };

    // The workgroup's tiles form one pipeline: while a tile's last K steps run,
    // the next tile's first stage is loaded (in place of a repeat of the last
    // stage) and stored to the free LDS buffer, and its second stage is in flight
    // during the epilogue, so a tile starts without waiting for its operands.
    // pb: the LDS buffer that holds the current tile's first stage.
    int i = widx;
    Tile cur = tile_at(i);
    Rsrc rc = rsrc_of(cur);
    int avc[A_PER];
    a_offsets(cur, avc);
    int pb = 0;
    gload(rc, avc, cur.kt0);
    sstore(0);
    gload(rc, avc, cur.kt0 + (cur.nsteps > 1 ? 1 : 0));
    __syncthreads();
    for (;;) {
        const int inext = i + nper;
        const bool has_next = inext < n_mine;
        const Tile nxt = tile_at(has_next ? inext : i);
        const Rsrc rn = rsrc_of(nxt);
        int avn[A_PER];
        a_offsets(nxt, avn);
        // what the load after this tile's last stage fetches: the next tile's
        // first stage, or (last tile) this tile's last stage again (cached)
        const int kt_after = has_next ? nxt.kt0 : cur.kt0 + cur.nsteps - 1;
        const int nsteps = cur.nsteps;

#pragma unroll
        for (int mi = 0; mi < MS; ++mi)
#pragma unroll
            for (int jj = 0; jj < NS; ++jj)
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[mi][jj][r] = 0.f;

        read_a(pb, 0, fa0);
        read_b(pb, 0, 0, fb0);
        // Every step but the last runs one straight path, so the MFMAs after the
        // barrier (on fragments read before it) issue without waiting for the
        // next stage's reads; the last step is peeled off below.
        for (int t = 0; t + 1 < nsteps; ++t) {
            const int buf = pb ^ (t & 1);
            read_b(buf, 0, 1, fb1);
            mfma(fa0, fb0, 0);
            read_a(buf, 1, fa1);
            read_b(buf, 1, 0, fb0);
            mfma(fa0, fb1, 1);
            read_b(buf, 1, 1, fb1);
            mfma(fa1, fb0, 0);
            sstore(buf ^ 1);
            // issue order up to the barrier: each half's fragment reads at the head of
            // the MFMA batch before the one that uses them, the stage stores spread
            // over the last batch
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(SG_MFMA, 12, 0);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(SG_MFMA, 8, 0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_DS_WRITE, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(SG_MFMA, 4, 0);
            __syncthreads();
            {
                // stage t + 2 of this tile, or what follows its last stage
                const bool own = t + 2 < nsteps;
                Rsrc rl;
                rl.a = own ? rc.a : rn.a;
                rl.lo = own ? rc.lo : rn.lo;
                rl.hi = own ? rc.hi : rn.hi;
                int avl[A_PER];
#pragma unroll
                for (int q = 0; q < A_PER; ++q) avl[q] = own ? avc[q] : avn[q];
                gload(rl, avl, own ? cur.kt0 + t + 2 : kt_after);
            }
            read_a(buf ^ 1, 0, fa0);
            read_b(buf ^ 1, 0, 0, fb0);
            mfma(fa1, fb1, 1);
            // after the barrier: the next stage's first fragment reads, then its
            // global loads, each between MFMAs of the last half
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
            }
        }
        const int lbuf = pb ^ ((nsteps - 1) & 1);
        {
            read_b(lbuf, 0, 1, fb1);
            mfma(fa0, fb0, 0);
            read_a(lbuf, 1, fa1);
            read_b(lbuf, 1, 0, fb0);
            mfma(fa0, fb1, 1);
            read_b(lbuf, 1, 1, fb1);
            mfma(fa1, fb0, 0);
            mfma(fa1, fb1, 1);
        }
        if (has_next) {
            // the next tile's first stage into the LDS buffer this tile no longer
            // reads (with a one-stage tile the registers hold this tile's stage
            // again: load it first), its second stage into the registers
            if (nsteps == 1) gload(rn, avn, nxt.kt0);
            sstore(lbuf ^ 1);
            gload(rn, avn, nxt.kt0 + (nxt.nsteps > 1 ? 1 : 0));
        }
        __syncthreads();

        if (cur.split) {
            // fp32 partial tile of this K chunk, laid out [row][weight row of the
            // tile]; rows past the group fall outside the descriptor and are dropped
            const __amdgpu_buffer_rsrc_t prsrc = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(args.part + (int64_t)cur.u * BM * BNW), (short)0, cur.rows_valid * BNW * 4,
                RSRC_WORD3);
            const int lbase = ((wm * (BM / WAVES_M) + (lane >> 4) * 4) * BNW +
                               b_sub_row<SWIGLU>(wn, 0) + (lane & 15)) * 4;
#pragma unroll
            for (int mi = 0; mi < MS; ++mi)
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int jj = 0; jj < NS; ++jj) {
                        const int off = ((mi * 16 + r) * BNW + b_sub_row<SWIGLU>(0, jj)) * 4;
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mi][jj][r]), prsrc,
                                                              lbase, off, 0);
                    }
        } else {
            // epilogue: accumulator element r of a 16x16 tile sits at row 4 (lane / 16)
            // + r, column lane % 16; a 4 x 4 transpose inside each lane quad gives
            // lane 4 b + e of row group a the row 4 a + e, columns 4 b .. 4 b + 3,
            // stored as one 8-byte vector (a quarter of the store instructions of
            // 2-byte stores, whole 32-byte row segments per lane quad) through a
            // descriptor over the tile's rows (rows past the group are dropped)
            const int qa = lane >> 4, qb = (lane >> 2) & 3, qe = lane & 3;
            const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(args.out + (int64_t)cur.row0 * args.ldo), (short)0,
                cur.rows_valid * args.ldo * 2, RSRC_WORD3);
            auto store4 = [&](const float* v, int row_in, int col) {
                const uint2 w = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, w), orsrc,
                                                      (row_in * args.ldo + col) * 2, 0, 0);
            };
#pragma unroll
            for (int mi = 0; mi < MS; ++mi) {
                const int row_in = wm * (BM / WAVES_M) + mi * 16 + qa * 4 + qe;
                if (SWIGLU) {
                    constexpr int HW = BNW / 2 / WAVES_N;
#pragma unroll
                    for (int j = 0; j < NS / 2; ++j) {
                        float v[4];
#pragma unroll
                        for (int r = 0; r < 4; ++r) v[r] = silu(acc[mi][j][r]) * acc[mi][NS / 2 + j][r];
                        quad_transpose(v, lane);
                        const int col = cur.n0 + wn * HW + j * 16 + qb * 4;
                        if (col < args.N) store4(v, row_in, col);
                    }
                } else {
#pragma unroll
                    for (int jj = 0; jj < NS; ++jj) {
                        float v[4];
#pragma unroll
                        for (int r = 0; r < 4; ++r) v[r] = acc[mi][jj][r];
                        quad_transpose(v, lane);
                        const int col = cur.n0 + wn * (BNW / WAVES_N) + jj * 16 + qb * 4;
                        if (col < args.N) store4(v, row_in, col);
                    }
                }
            }
        }
        if (!has_next) break;
        i = inext;
        cur = nxt;
        rc = rn;
#pragma unroll
        for (int q = 0; q < A_PER; ++q) avc[q] = avn[q];
        pb = lbuf ^ 1;
    }
}

// ---------------------------------------------------------------------------
// Small groups (those of a short call up to SMALL_ROWS_MAX rows, see
// small_limits; every group of a call with the MOE_FFN_SMALL_GROUPS statement or
// of at most SMALL_ROWS rows in all): weight streaming with split-K.  Here the
// weights dominate the traffic (each weight byte is used by
// a handful of rows), so the aim is to read every weight byte once, from all
// CUs at once.  Work item = (group, 128 weight rows, K chunk, 64 rows); one
// workgroup per item, three per CU with three K steps of loads in flight
// each (four per CU cannot hold that ring without spilling), fp32 partial sums
// per K chunk.  HBM reads
// reach their rate only with many independent streams in flight (a read-only
// probe over 448 MiB: 4.3-5.1 TB/s with 224-448 workgroups, 5.4-5.7 TB/s with
// 896 or more), so the item is narrow in weight rows and covers a whole
// decode-sized group (a group of up to 64 rows reads its weights once).  A second kernel adds the
// chunks in a fixed order (so results are deterministic) and, for the gate/up
// product, applies SiLU(a) * b.
// The split factor S is derived on the device from the group sizes; both
// kernels derive the same plan from the same inputs.
// ---------------------------------------------------------------------------
constexpr int ST_M = 64;                 // rows per item (two 32-row MFMA tiles per wave)
constexpr int ST_N = 128;                // weight rows per item (32 per wave)
constexpr int ST_THREADS = 256;
constexpr int ST_WG_PER_CU = 3;
constexpr int ST_RING = 2;               // K steps of loads in flight beyond the one in LDS
constexpr int ST_A_PER = ST_M * 64 / 8 / ST_THREADS;   // 16-byte loads per thread per K step
constexpr int ST_B_PER = ST_N * 64 / 8 / ST_THREADS;
constexpr int SPLIT_MAX = 32;
constexpr int PART_FACTOR = 8;           // partial capacity = PART_FACTOR x bound on small rows
static_assert(ST_A_PER == 2 && ST_B_PER == 4, "streaming tile");

struct StreamArgs {
    const bf16_t* w[MOE_MAX_GROUPS];     // per group [N][K]
    const int32_t* offsets;              // as GemmArgs::offsets
    const bf16_t* a;                     // [rows][K]
    float* part;                         // [S][n_small][N]
    bf16_t* out;                         // reduce output [rows][ldo]
    int n_groups;                        // lead groups included
    int lead, lead_rows;                 // as in GemmArgs
    int K;
    int N;                               // weight rows (2f for gate/up, d for down)
    int ldo;
    int part_rows;                       // capacity of `part` in rows (S * n_small <= part_rows)
    int grid;                            // workgroups of the streaming launch
    const int32_t* a_rows;               // gather: row p of A is a[a_rows[p]] (a holds a_total rows)
    int a_total;
    const int* limits;                   // row limits written by the gate/up tiled launch (nullptr:
    int product;                         // lim0); this product's index, 0 gate/up, 1 down
    int lim0;                            // row limit of streamed groups when limits is nullptr
};

struct StreamPlan {
    int off[MOE_MAX_GROUPS + 1];
    int qbase[MOE_MAX_GROUPS + 1];       // compact row base of each small group
    int istart[MOE_MAX_GROUPS + 1];      // first work item of each group
    int n_small, S, total, n_tiles;
};

__device__ void make_stream_plan(const StreamArgs& a, StreamPlan& P, int nthreads) {
    const int lim = a.limits != nullptr ? a.limits[a.product] : a.lim0;
    for (int g = threadIdx.x; g <= a.n_groups; g += nthreads)
        P.off[g] = group_start(a.offsets, a.lead, a.lead_rows, g);
    __syncthreads();
    if (threadIdx.x < 64) {                          // one wave: prefix sums over the groups
        const int lane = threadIdx.x;
        const int nt = (int)ceil_div(a.N, ST_N);
        const int KT = a.K / 64;
        int rows_small = 0, base = 0;
        for (int g0 = 0; g0 < a.n_groups; g0 += 64) {
            const int g = g0 + lane;
            const int rows = g < a.n_groups ? P.off[g + 1] - P.off[g] : 0;
            const bool small = rows > 0 && rows <= lim;
            const int rs = small ? rows : 0;
            const int items = small ? (int)ceil_div(rows, ST_M) * nt : 0;
            const int irs = wave_incl_scan(rs, lane), iit = wave_incl_scan(items, lane);
            if (g < a.n_groups) {
                P.qbase[g] = rows_small + irs - rs;
                P.istart[g] = base + iit - items;    // scaled by S below
            }
            rows_small += __shfl(irs, 63, 64);
            base += __shfl(iit, 63, 64);
        }
        // split factor: as many K chunks as fit the grid in one round (every
        // workgroup streams one item; a partly filled extra round would leave
        // most of HBM idle)
        int S = base > 0 ? a.grid / base : 1;
        S = min(S, SPLIT_MAX);
        S = min(S, KT);
        if (rows_small > 0) S = min(S, a.part_rows / rows_small);
        S = max(S, 1);
        for (int g = lane; g < a.n_groups; g += 64) P.istart[g] *= S;
        if (lane == 0) {
            P.qbase[a.n_groups] = rows_small;
            P.istart[a.n_groups] = base * S;
            P.n_small = rows_small;
            P.S = S;
            P.total = base * S;
            P.n_tiles = nt;
        }
    }
    __syncthreads();
}

// One workgroup per item (64 rows x 128 weight rows x one K chunk); each wave
// takes 32 of the weight rows against both 32-row halves of the rows.  Loads
// are coalesced (8 lanes read one 128-byte row segment) and run ST_RING K
// steps ahead in registers; one LDS stage holds the step being multiplied.
// The partial-sum epilogue adds a uniform row offset per accumulator element to
// one per-lane pointer: with a 64-bit row offset per element and lane, the
// compiler kept all of them live across the item loop and spilled them to
// scratch (decode steps 5 % slower).
template <bool GATHER = false>
__global__ __launch_bounds__(ST_THREADS, ST_WG_PER_CU) void stream_gemm_kernel(StreamArgs args) {
    __shared__ __attribute__((aligned(16))) bf16_t As[ST_M * LDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[ST_N * LDK];
    __shared__ StreamPlan P;
    __shared__ int s_item[4];
    make_stream_plan(args, P, ST_THREADS);
    if (P.total == 0) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wg_per_xcd = gridDim.x / NUM_XCD;
    const int xcd = blockIdx.x % NUM_XCD;
    const int widx = blockIdx.x / NUM_XCD;
    const int chunk = (P.total + NUM_XCD - 1) / NUM_XCD;
    const int i_begin = xcd * chunk, i_end = min(i_begin + chunk, P.total);
    const int K = args.K, KT = K / 64, S = P.S;
    const int kc = (tid & 7) * 8;
    const int lrow = tid >> 3;                          // 0..31: row of this thread's loads
    const int voff = (lrow * K + kc) * 2;
    const int vstep = 32 * K * 2;
    const int frag_col = (lane >> 5) * 32, frag_row = lane & 31;

    for (int it = i_begin + widx; it < i_end; it += wg_per_xcd) {
        if (tid == 0) {
            const int lo = last_le(P.istart, args.n_groups, it);   // the item's group
            s_item[0] = lo;
            s_item[1] = it - P.istart[lo];
        }
        __syncthreads();
        const int g = __builtin_amdgcn_readfirstlane(s_item[0]);
        int local = __builtin_amdgcn_readfirstlane(s_item[1]);
        const int rows = __builtin_amdgcn_readfirstlane(P.off[g + 1] - P.off[g]);
        const int mt = (int)ceil_div(rows, ST_M);
        const int m = local % mt;
        local /= mt;
        const int c = local % S;
        const int n0 = (local / S) * ST_N;
        const int row0 = __builtin_amdgcn_readfirstlane(P.off[g]) + m * ST_M;
        const int rows_valid = min(ST_M, rows - m * ST_M);
        const int bvalid = min(ST_N, args.N - n0);
        const int kt0 = (int)((int64_t)c * KT / S), kt1 = (int)((int64_t)(c + 1) * KT / S);

        const __amdgpu_buffer_rsrc_t ar =
            GATHER ? __builtin_amdgcn_make_buffer_rsrc((void*)args.a, (short)0, args.a_total * K * 2,
                                                      RSRC_WORD3)
                   : __builtin_amdgcn_make_buffer_rsrc((void*)(args.a + (int64_t)row0 * K), (short)0,
                                                      rows_valid * K * 2, RSRC_WORD3);
        int avoff[ST_A_PER];
#pragma unroll
        for (int q = 0; q < ST_A_PER; ++q) {
            const int rin = lrow + 32 * q;
            avoff[q] = !GATHER ? voff + q * vstep
                       : rin < rows_valid ? (args.a_rows[row0 + rin] * K + kc) * 2 : A_OOB;
        }
        const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(args.w[g] + (int64_t)n0 * K), (short)0, bvalid * K * 2, RSRC_WORD3);

        uint4 ring_a[ST_RING + 1][ST_A_PER], ring_b[ST_RING + 1][ST_B_PER];
        auto load = [&](int kt, uint4* ra, uint4* rb) {
            const int so = kt * 128;
#pragma unroll
            for (int q = 0; q < ST_A_PER; ++q) ra[q] = buffer_load16(ar, avoff[q], so);
#pragma unroll
            for (int i = 0; i < ST_B_PER; ++i) rb[i] = buffer_load16(br, voff + i * vstep, so);
        };
        f32x16 acc0, acc1;
#pragma unroll
        for (int r = 0; r < 16; ++r) { acc0[r] = 0.f; acc1[r] = 0.f; }
        const int nsteps = kt1 - kt0;
#pragma unroll
        for (int u = 0; u <= ST_RING; ++u)
            if (u < nsteps) load(kt0 + u, ring_a[u], ring_b[u]);
        for (int t0 = 0; t0 < nsteps; t0 += ST_RING + 1) {
#pragma unroll
            for (int u = 0; u <= ST_RING; ++u) {
                const int t = t0 + u;
                if (t < nsteps) {
                    __syncthreads();                 // previous step's fragment reads are done
#pragma unroll
                    for (int q = 0; q < ST_A_PER; ++q)
                        *(uint4*)&As[(lrow + 32 * q) * LDK + kc] = ring_a[u][q];
#pragma unroll
                    for (int i = 0; i < ST_B_PER; ++i)
                        *(uint4*)&Bs[(lrow + 32 * i) * LDK + kc] = ring_b[u][i];
                    __syncthreads();
                    if (t + ST_RING + 1 < nsteps) load(kt0 + t + ST_RING + 1, ring_a[u], ring_b[u]);
#pragma unroll
                    for (int kk = 0; kk < 4; ++kk) {
                        const bf16x8 a0 = *(const bf16x8*)&As[frag_row * LDK + frag_col + kk * 8];
                        const bf16x8 a1 = *(const bf16x8*)&As[(32 + frag_row) * LDK + frag_col + kk * 8];
                        const bf16x8 bw = *(const bf16x8*)&Bs[(wave * 32 + frag_row) * LDK + frag_col + kk * 8];
                        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, bw, acc0, 0, 0, 0);
                        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, bw, acc1, 0, 0, 0);
                    }
                }
            }
        }

        // partial store: element r of a 32x32 tile is row 8*(r/4) + 4*(lane/32) + r%4, col lane%32
        float* prow = args.part + ((int64_t)c * P.n_small + P.qbase[g] + m * ST_M) * args.N + n0 +
                      wave * 32;
        const int cw = bvalid - wave * 32;           // valid columns of this wave
        if (frag_row < cw) {
            // one per-lane base pointer; the row offset of each r is uniform
            const int lr = (lane >> 5) * 4;
            float* pl = prow + (int64_t)lr * args.N + frag_row;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rc = (r >> 2) * 8 + (r & 3);
                const int64_t o = (int64_t)__builtin_amdgcn_readfirstlane(rc * args.N);
                const int64_t o32 = (int64_t)__builtin_amdgcn_readfirstlane((rc + 32) * args.N);
                if (rc + lr < rows_valid) pl[o] = acc0[r];
                if (rc + 32 + lr < rows_valid) pl[o32] = acc1[r];
            }
        }
        __syncthreads();                             // s_item and LDS reuse by the next item
    }
}

// Adds chunks [c, c + RU) of a partial sum to x (SWIGLU: the up half, `up`
// floats further on, to y), in chunk order.  All RU loads are issued before the
// first add: a chunk at or past S reads chunk S - 1 and its add is skipped, so
// a short split costs one load round trip instead of one per chunk.
template <bool SWIGLU, int RU>
__device__ __forceinline__ void add_chunk_batch(const float* pr, int64_t cstride, int up, int c,
                                                int S, float4& x, float4& y) {
    float4 v[RU], u[RU];
#pragma unroll
    for (int j = 0; j < RU; ++j) {
        const int cc = c + j < S ? c + j : S - 1;
        v[j] = *(const float4*)(pr + cc * cstride);
        if (SWIGLU) u[j] = *(const float4*)(pr + cc * cstride + up);
    }
#pragma unroll
    for (int j = 0; j < RU; ++j)
        if (c + j < S) {
            x.x += v[j].x; x.y += v[j].y; x.z += v[j].z; x.w += v[j].w;
            if (SWIGLU) { y.x += u[j].x; y.y += u[j].y; y.z += u[j].z; y.w += u[j].w; }
        }
}

// x (and y) = the sum of chunks 0 .. S-1 (S >= 1) in chunk order: batches of 8
// loads, the rest as one batch of 4 or 8.
template <bool SWIGLU>
__device__ __forceinline__ void add_chunks(const float* pr, int64_t cstride, int up, int S,
                                           float4& x, float4& y) {
    x = make_float4(0.f, 0.f, 0.f, 0.f);
    y = x;
    int c = 0;
    for (; c + 8 <= S; c += 8) add_chunk_batch<SWIGLU, 8>(pr, cstride, up, c, S, x, y);
    if (S - c > 4) add_chunk_batch<SWIGLU, 8>(pr, cstride, up, c, S, x, y);
    else if (c < S) add_chunk_batch<SWIGLU, 4>(pr, cstride, up, c, S, x, y);
}

// Sums, in chunk order, the K chunks of the tiled kernel's split tiles (fp32
// partial tiles [row][weight row]; SWIGLU: gate in tile columns [0, 128), up
// in [128, 256)) and applies the epilogue: out = SiLU(gate) * up, or the sum.
template <bool SWIGLU>
__device__ void tile_split_reduce(const GemmArgs& t, int* s_off, int* s_tstart) {
    const int n_groups = t.n_groups;
    for (int g = threadIdx.x; g <= n_groups; g += ST_THREADS)
        s_off[g] = group_start(t.offsets, t.lead, t.lead_rows, g);
    __syncthreads();
    const int lim = t.limits != nullptr ? t.limits[t.product] : t.lim0;
    if (threadIdx.x < 64) tile_starts(s_off, n_groups, lim, t.n_tiles, s_tstart, threadIdx.x);
    __syncthreads();
    const SplitPlan plan = split_plan(s_tstart[n_groups], t.K / BK, t.split_units);
    const int S = plan.S;
    if (S == 1) return;
    constexpr int BN_OUT = SWIGLU ? BNW / 2 : BNW;
    constexpr int C4 = BN_OUT / 4;
    const int64_t items = (int64_t)plan.tail * BM * C4;
    for (int64_t i = (int64_t)blockIdx.x * ST_THREADS + threadIdx.x; i < items;
         i += (int64_t)gridDim.x * ST_THREADS) {
        const int q = (int)(i / (BM * C4));          // split tile, counted from plan.head
        const int L = plan.head + q;
        const int rem = (int)(i - (int64_t)q * BM * C4);
        const int row = rem / C4, j = (rem - row * C4) * 4;
        const int g = last_le(s_tstart, n_groups, L);
        const int rows = s_off[g + 1] - s_off[g];
        const int mt = (int)ceil_div(rows, BM);
        const int local = L - s_tstart[g];
        const int nt = local / mt;
        const int m0 = (local - nt * mt) * BM;
        if (m0 + row >= rows) continue;
        const int n0 = nt * BN_OUT;
        if (n0 + j >= t.N) continue;
        float4 x, y;
        add_chunks<SWIGLU>(t.part + ((int64_t)q * S * BM + row) * BNW + j, (int64_t)BM * BNW,
                           BNW / 2, S, x, y);
        const float o[4] = {SWIGLU ? silu(x.x) * y.x : x.x, SWIGLU ? silu(x.y) * y.y : x.y,
                            SWIGLU ? silu(x.z) * y.z : x.z, SWIGLU ? silu(x.w) * y.w : x.w};
        uint2 pk;
        pk.x = pack_bf16x2(o[0], o[1]);
        pk.y = pack_bf16x2(o[2], o[3]);
        *(uint2*)(t.out + (int64_t)(s_off[g] + m0 + row) * t.ldo + n0 + j) = pk;
    }
}

template <bool SWIGLU>
__device__ __forceinline__ void stream_reduce(const StreamArgs& args, const StreamPlan& P);

// Fixed-order sum of the K chunks; SWIGLU: out[p][j] = SiLU(sum gate_j) * sum up_j
// with gate in partial columns [0, N/2) and up in [N/2, N).  The same launch
// finishes the tiled kernel's split tiles (tile_split_reduce).
template <bool SWIGLU>
__global__ __launch_bounds__(ST_THREADS) void split_reduce_kernel(StreamArgs args, GemmArgs targs) {
    __shared__ StreamPlan P;
    __shared__ int t_off[MOE_MAX_GROUPS + 1], t_tstart[MOE_MAX_GROUPS + 1];
    const int tsplit = targs.part != nullptr ? *targs.split_info : 1;   // used at the end
    // no group can be streamed (MOE_FFN_LARGE_GROUPS): no streaming plan to build
    if (args.limits != nullptr || args.lim0 > 0) {
        make_stream_plan(args, P, ST_THREADS);
        stream_reduce<SWIGLU>(args, P);
    }
    if (tsplit > 1) tile_split_reduce<SWIGLU>(targs, t_off, t_tstart);
}

template <bool SWIGLU>
__device__ __forceinline__ void stream_reduce(const StreamArgs& args, const StreamPlan& P) {
    const int n_small = P.n_small;
    if (n_small == 0) return;
    const int S = P.S;
    const int cols = SWIGLU ? args.N / 2 : args.N;
    const int chunks = cols / 4;                     // 4 output columns per item
    const int64_t total = (int64_t)n_small * chunks;
    const int64_t cstride = (int64_t)n_small * args.N;
    for (int64_t i = (int64_t)blockIdx.x * ST_THREADS + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * ST_THREADS) {
        const int q = (int)(i / chunks);
        const int c4 = (int)(i - (int64_t)q * chunks) * 4;
        // the row's group: groups without small rows share qbase with the next one
        const int g = last_le(P.qbase, args.n_groups, q);
        const int p = P.off[g] + (q - P.qbase[g]);
        float4 x, y;
        add_chunks<SWIGLU>(args.part + (int64_t)q * args.N + c4, cstride, cols, S, x, y);
        const float o0 = SWIGLU ? silu(x.x) * y.x : x.x, o1 = SWIGLU ? silu(x.y) * y.y : x.y;
        const float o2 = SWIGLU ? silu(x.z) * y.z : x.z, o3 = SWIGLU ? silu(x.w) * y.w : x.w;
        uint2 pk;
        pk.x = pack_bf16x2(o0, o1);
        pk.y = pack_bf16x2(o2, o3);
        *(uint2*)(args.out + (int64_t)p * args.ldo + c4) = pk;
    }
}

// The down product's chunk sum fused with the gate-weighted combine, for calls
// in which every group is streamed (no group above SMALL_ROWS rows): one
// thread per token and 4 output columns.  For each assignment r of token t, in
// ascending r, the row's output is summed over the K chunks in chunk order and
// rounded to bf16 (the value the chunk sum would store in y_perm), then added
// with its gate by fmaf; the shared experts' output is added last and the sum
// stored in bf16 -- the arithmetic of split_reduce_kernel followed by the
// combine, so the outputs are the same bits, without y_perm being written and
// read back or the combine's launch.
struct CombineArgs {
    const int32_t* token_row;            // [T][k]
    const float* gate;                   // [T][k]
    const bf16_t* y_shared;              // [T][d], nullable
    bf16_t* y;                           // [T][d]
    int64_t T;
    int k;
};

template <int KM>
__global__ __launch_bounds__(ST_THREADS) void stream_reduce_combine_kernel(StreamArgs args,
                                                                           CombineArgs cb) {
    __shared__ StreamPlan P;
    make_stream_plan(args, P, ST_THREADS);
    const int lim = args.limits != nullptr ? args.limits[args.product] : args.lim0;
    const int S = P.S;
    const int d = args.N;
    const int chunks = d / 4;
    const int64_t cstride = (int64_t)P.n_small * d;
    const int64_t total = cb.T * chunks;
    // CB chunks of every assignment are loaded together, KM * CB loads in flight
    constexpr int CB = 32 / KM > 0 ? 32 / KM : 1;
    for (int64_t i = (int64_t)blockIdx.x * ST_THREADS + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * ST_THREADS) {
        const int64_t t = i / chunks;
        const int c4 = (int)(i - t * chunks) * 4;
        // the partial row of each assignment here, or none
        int64_t off[KM];
        float g[KM];
        bool ok[KM];
        int64_t first = -1;
#pragma unroll
        for (int r = 0; r < KM; ++r) {
            const int rr = r < cb.k ? r : cb.k - 1;
            const int32_t p = r < cb.k ? cb.token_row[t * cb.k + rr] : -1;
            g[r] = cb.gate[t * cb.k + rr];
            ok[r] = false;
            off[r] = 0;
            if (p >= 0) {
                const int grp = last_le(P.off, args.n_groups, p);
                // a group above the streaming limit has no partial rows (outside the contract)
                ok[r] = P.off[grp + 1] - P.off[grp] <= lim;
                off[r] = (int64_t)(P.qbase[grp] + p - P.off[grp]) * d + c4;
            }
            if (ok[r] && first < 0) first = off[r];
        }
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        if (first >= 0) {
            float4 x[KM];
#pragma unroll
            for (int r = 0; r < KM; ++r) x[r] = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int c = 0; c < S; c += CB) {
                float4 v[KM][CB];
                // every load issued before the first add: an assignment not here
                // reads the first one's row and a chunk past S the last chunk,
                // both dropped below
#pragma unroll
                for (int r = 0; r < KM; ++r)
#pragma unroll
                    for (int j = 0; j < CB; ++j) {
                        const int cc = c + j < S ? c + j : S - 1;
                        v[r][j] = *(const float4*)(args.part + (ok[r] ? off[r] : first) + cc * cstride);
                    }
#pragma unroll
                for (int r = 0; r < KM; ++r)
#pragma unroll
                    for (int j = 0; j < CB; ++j)
                        if (c + j < S) {
                            x[r].x += v[r][j].x; x[r].y += v[r][j].y;
                            x[r].z += v[r][j].z; x[r].w += v[r][j].w;
                        }
            }
            // each row's bf16 value, as y_perm would hold it, added with its gate in
            // ascending r
#pragma unroll
            for (int r = 0; r < KM; ++r) {
                if (!ok[r]) continue;
                acc[0] = fmaf(g[r], bf16_to_f32(f32_to_bf16(x[r].x)), acc[0]);
                acc[1] = fmaf(g[r], bf16_to_f32(f32_to_bf16(x[r].y)), acc[1]);
                acc[2] = fmaf(g[r], bf16_to_f32(f32_to_bf16(x[r].z)), acc[2]);
                acc[3] = fmaf(g[r], bf16_to_f32(f32_to_bf16(x[r].w)), acc[3]);
            }
        }
        if (cb.y_shared) {
            const uint2 w = *(const uint2*)(cb.y_shared + t * d + c4);
            acc[0] += __uint_as_float(w.x << 16);
            acc[1] += __uint_as_float(w.x & 0xffff0000u);
            acc[2] += __uint_as_float(w.y << 16);
            acc[3] += __uint_as_float(w.y & 0xffff0000u);
        }
        uint2 pk;
        pk.x = pack_bf16x2(acc[0], acc[1]);
        pk.y = pack_bf16x2(acc[2], acc[3]);
        *(uint2*)(cb.y + t * d + c4) = pk;
    }
}

// ---------------------------------------------------------------------------
// fp32 path: plain FMA loops, one thread per output element.
// ---------------------------------------------------------------------------
struct PtrTable {
    const float* p[MOE_MAX_GROUPS];
};

// fp32 path (small layers): 16 x 16 output tiles within one group, operands
// staged through LDS in 32-wide K slices (coalesced loads); every output is still
// one fmaf chain over K in ascending order, as a thread per output would sum it.
constexpr int F32_T = 16, F32_K = 32;

__device__ __forceinline__ void f32_tile_plan(const int32_t* offsets, int lead, int lead_rows,
                                              int n_groups, int ncols, int* s_off, int* s_tstart) {
    for (int s = threadIdx.x; s <= n_groups; s += blockDim.x)
        s_off[s] = group_start(offsets, lead, lead_rows, s);
    __syncthreads();
    if (threadIdx.x == 0) {
        const int nt = (ncols + F32_T - 1) / F32_T;
        int t = 0;
        for (int g = 0; g < n_groups; ++g) {
            s_tstart[g] = t;
            t += (s_off[g + 1] - s_off[g] + F32_T - 1) / F32_T * nt;
        }
        s_tstart[n_groups] = t;
    }
    __syncthreads();
}

__global__ __launch_bounds__(256) void ffn1_f32_kernel(const float* __restrict__ x,
                                                       const int32_t* __restrict__ a_rows,
                                                       const int32_t* __restrict__ offsets,
                                                       int lead, int lead_rows, int n_groups,
                                                       PtrTable w13, int d, int f,
                                                       float* __restrict__ h) {
    __shared__ int s_off[MOE_MAX_GROUPS + 1], s_tstart[MOE_MAX_GROUPS + 1];
    __shared__ float xs[F32_T][F32_K + 1], gs[F32_T][F32_K + 1], us[F32_T][F32_K + 1];
    f32_tile_plan(offsets, lead, lead_rows, n_groups, f, s_off, s_tstart);
    const int tid = threadIdx.x, tr = tid / F32_T, tc = tid % F32_T;
    const int nt = (f + F32_T - 1) / F32_T;
    for (int tile = blockIdx.x; tile < s_tstart[n_groups]; tile += gridDim.x) {
        const int g = last_le(s_tstart, n_groups, tile);
        const int local = tile - s_tstart[g];
        const int row0 = s_off[g] + (local / nt) * F32_T, col0 = (local % nt) * F32_T;
        const int rows = min(F32_T, s_off[g + 1] - row0);
        const float* __restrict__ W = w13.p[g];
        float a = 0.f, b = 0.f;
        for (int q0 = 0; q0 < d; q0 += F32_K) {
            for (int e = tid; e < F32_T * F32_K; e += 256) {
                const int r = e / F32_K, q = e % F32_K;
                const bool kin = q0 + q < d;
                const int p = row0 + r;
                xs[r][q] = r < rows && kin ? x[(int64_t)(a_rows ? a_rows[p] : p) * d + q0 + q] : 0.f;
                gs[r][q] = col0 + r < f && kin ? W[(int64_t)(col0 + r) * d + q0 + q] : 0.f;
                us[r][q] = col0 + r < f && kin ? W[(int64_t)(f + col0 + r) * d + q0 + q] : 0.f;
            }
            __syncthreads();
            const int qn = min(F32_K, d - q0);
            for (int q = 0; q < qn; ++q) {
                a = fmaf(gs[tc][q], xs[tr][q], a);
                b = fmaf(us[tc][q], xs[tr][q], b);
            }
            __syncthreads();
        }
        if (tr < rows && col0 + tc < f)
            h[(int64_t)(row0 + tr) * f + col0 + tc] = a / (1.0f + expf(-a)) * b;
    }
}

__global__ __launch_bounds__(256) void ffn2_f32_kernel(const float* __restrict__ h,
                                                       const int32_t* __restrict__ offsets,
                                                       int lead, int lead_rows, int n_groups,
                                                       PtrTable w2, int d, int f,
                                                       float* __restrict__ y) {
    __shared__ int s_off[MOE_MAX_GROUPS + 1], s_tstart[MOE_MAX_GROUPS + 1];
    __shared__ float hs[F32_T][F32_K + 1], ws[F32_T][F32_K + 1];
    f32_tile_plan(offsets, lead, lead_rows, n_groups, d, s_off, s_tstart);
    const int tid = threadIdx.x, tr = tid / F32_T, tc = tid % F32_T;
    const int nt = (d + F32_T - 1) / F32_T;
    for (int tile = blockIdx.x; tile < s_tstart[n_groups]; tile += gridDim.x) {
        const int g = last_le(s_tstart, n_groups, tile);
        const int local = tile - s_tstart[g];
        const int row0 = s_off[g] + (local / nt) * F32_T, col0 = (local % nt) * F32_T;
        const int rows = min(F32_T, s_off[g + 1] - row0);
        const float* __restrict__ W = w2.p[g];
        float acc = 0.f;
        for (int j0 = 0; j0 < f; j0 += F32_K) {
            for (int e = tid; e < F32_T * F32_K; e += 256) {
                const int r = e / F32_K, j = e % F32_K;
                const bool kin = j0 + j < f;
                hs[r][j] = r < rows && kin ? h[(int64_t)(row0 + r) * f + j0 + j] : 0.f;
                ws[r][j] = col0 + r < d && kin ? W[(int64_t)(col0 + r) * f + j0 + j] : 0.f;
            }
            __syncthreads();
            const int jn = min(F32_K, f - j0);
            for (int j = 0; j < jn; ++j) acc = fmaf(ws[tc][j], hs[tr][j], acc);
            __syncthreads();
        }
        if (tr < rows && col0 + tc < d) y[(int64_t)(row0 + tr) * d + col0 + tc] = acc;
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

static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

static int64_t small_rows_bound(int64_t cap_rows, int n_groups) {
    const int64_t b = (int64_t)n_groups * SMALL_ROWS;
    return cap_rows < b ? cap_rows : b;
}

// fp32 partial tiles of the tiled kernel's split K (none when no group can be
// big enough for the tiled kernel)
static int64_t tile_part_bytes(int64_t cap_rows) {
    return cap_rows > SMALL_ROWS ? 256 + (int64_t)TILE_SPLIT_UNITS * BM * BNW * 4 : 0;
}

// workspace: [H: cap_rows x f bf16][streaming partials][tiled partial tiles]
size_t grouped_ffn_ws_bytes(int dtype, int64_t cap_rows, int d, int f, int n_groups) {
    if (dtype != MOE_BF16) return (size_t)cap_rows * (size_t)f * 4 + 256;
    const int64_t h = align256(cap_rows * (int64_t)f * 2);
    const int64_t ncols = 2 * (int64_t)f > d ? 2 * (int64_t)f : d;
    const int64_t part = align256((int64_t)PART_FACTOR * small_rows_bound(cap_rows, n_groups) * ncols * 4);
    return (size_t)(h + part + tile_part_bytes(cap_rows) + 256);
}

int launch_grouped_ffn(const void* x_perm, int dtype, const int32_t* offsets, int n_groups,
                       const void* const* w13, const void* const* w2, int d, int f,
                       int64_t cap_rows, void* y_perm, void* ws, hipStream_t s,
                       const int32_t* a_rows, int64_t a_total, int products,
                       const void* combine, int lead, int lead_rows) {
    if (cap_rows == 0) return MOE_OK;
    const bool up = (products & MOE_FFN_GATE_UP) != 0, down = (products & MOE_FFN_DOWN) != 0;
    // every group within SMALL_ROWS_MAX rows (the caller's statement): all of them are
    // streamed, so no tile, no split tile and no row limit to pass on, and the tiled
    // launches are left out
    const bool small = (products & MOE_FFN_SMALL_GROUPS) != 0;
    // every non-empty group above SMALL_ROWS_MAX rows (the caller's statement): none is
    // streamed, every group is tiled (row limit 0) and the streaming launches are left out
    const bool large = (products & MOE_FFN_LARGE_GROUPS) != 0;
    if (dtype == MOE_F32) {
        PtrTable t13, t2;
        for (int i = 0; i < MOE_MAX_GROUPS; ++i) {
            t13.p[i] = i < n_groups ? (const float*)w13[i] : nullptr;
            t2.p[i] = i < n_groups ? (const float*)w2[i] : nullptr;
        }
        float* h = (float*)ws;
        // tiles of 16 rows within a group: at most cap_rows / 16 + n_groups row tiles
        const int64_t mt = cap_rows / 16 + n_groups;
        int64_t b1 = mt * ceil_div(f, 16), b2 = mt * ceil_div(d, 16);
        if (b1 > 4096) b1 = 4096;
        if (b2 > 4096) b2 = 4096;
        if (up)
            hipLaunchKernelGGL(ffn1_f32_kernel, dim3((unsigned)b1), dim3(256), 0, s,
                               (const float*)x_perm, a_rows, offsets, lead, lead_rows, n_groups,
                               t13, d, f, h);
        if (down)
            hipLaunchKernelGGL(ffn2_f32_kernel, dim3((unsigned)b2), dim3(256), 0, s,
                               (const float*)h, offsets, lead, lead_rows, n_groups, t2, d, f,
                               (float*)y_perm);
        return launch_status();
    }
    const int cus = num_cus();
    const int grid = (cus / NUM_XCD) * NUM_XCD;
    bf16_t* h = (bf16_t*)ws;
    float* part = (float*)((char*)ws + align256(cap_rows * (int64_t)f * 2));
    const int64_t rmax = small_rows_bound(cap_rows, n_groups);
    const int64_t ncols = 2 * (int64_t)f > d ? 2 * (int64_t)f : d;
    // tiled split K: two split factors (one per product) and the two products'
    // streamed-group row limits in a 256-byte header, then the partial tiles
    char* tbase = tile_part_bytes(cap_rows) > 0
                      ? (char*)part + align256((int64_t)PART_FACTOR * rmax * ncols * 4)
                      : nullptr;
    float* tpart = tbase && !small ? (float*)(tbase + 256) : nullptr;
    int* tinfo = tbase && !small ? (int*)tbase : nullptr;
    const int sgrid = ((cus * ST_WG_PER_CU) / NUM_XCD) * NUM_XCD;
    const int64_t red_items = rmax * ((f > d ? f : d) / 4);
    int rgrid = (int)ceil_div(red_items, ST_THREADS);
    if (tpart != nullptr && rgrid < 2 * cus) rgrid = 2 * cus;   // room for split tiles
    if (rgrid > 4096) rgrid = 4096;
    // only split tiles to sum: four workgroups per CU, each thread a few items
    // (the idle workgroups of a larger grid cost more than the loop; gate/up
    // products 1-2 % faster at the Mixtral and Qwen3 prefill shapes)
    if (large) rgrid = 4 * cus;
    if (rgrid < 1) rgrid = 1;

    // gate/up product: tiled launch, then the streaming launch (the small groups of a
    // short call), then the chunk sums
    GemmArgs a1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i)
        a1.w[i] = up && i < n_groups ? (const bf16_t*)w13[i] : nullptr;
    a1.offsets = offsets;
    a1.lead = lead;
    a1.lead_rows = lead_rows;
    a1.a = (const bf16_t*)x_perm;
    a1.out = h;
    a1.n_groups = n_groups;
    a1.K = d;
    a1.N = f;
    a1.ldo = f;
    a1.up_row = f;
    a1.n_tiles = (int)ceil_div(f, BNW / 2);
    a1.limits = tinfo && !large ? tinfo + 2 : nullptr;
    a1.product = 0;
    a1.lim0 = small ? SMALL_ROWS_MAX : large ? 0 : SMALL_ROWS;
    a1.down_tiles = (int)ceil_div(d, BNW);
    a1.part = tpart;
    a1.split_info = tinfo;
    a1.split_units = grid < TILE_SPLIT_UNITS ? grid : TILE_SPLIT_UNITS;
    a1.a_rows = a_rows;
    a1.a_total = (int)a_total;
    if (up && !small && a_rows)
        hipLaunchKernelGGL((grouped_gemm_kernel<true, true>), dim3(grid), dim3(GEMM_THREADS), 0, s, a1);
    else if (up && !small)
        hipLaunchKernelGGL((grouped_gemm_kernel<true, false>), dim3(grid), dim3(GEMM_THREADS), 0, s, a1);
    StreamArgs s1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) s1.w[i] = a1.w[i];
    s1.offsets = offsets;
    s1.lead = lead;
    s1.lead_rows = lead_rows;
    s1.a = (const bf16_t*)x_perm;
    s1.part = part;
    s1.out = h;
    s1.n_groups = n_groups;
    s1.K = d;
    s1.N = 2 * f;
    s1.ldo = f;
    s1.part_rows = (int)(PART_FACTOR * rmax);
    s1.grid = sgrid;
    s1.a_rows = a_rows;
    s1.a_total = (int)a_total;
    s1.limits = a1.limits;
    s1.product = 0;
    s1.lim0 = a1.lim0;
    if (up) {
        if (!large && a_rows)
            hipLaunchKernelGGL(stream_gemm_kernel<true>, dim3(sgrid), dim3(ST_THREADS), 0, s, s1);
        else if (!large)
            hipLaunchKernelGGL(stream_gemm_kernel<false>, dim3(sgrid), dim3(ST_THREADS), 0, s, s1);
        hipLaunchKernelGGL(split_reduce_kernel<true>, dim3(rgrid), dim3(ST_THREADS), 0, s, s1, a1);
    }
    if (!down) return launch_status();

    // down product
    GemmArgs a2 = a1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) a2.w[i] = i < n_groups ? (const bf16_t*)w2[i] : nullptr;
    a2.a = h;
    a2.out = (bf16_t*)y_perm;
    a2.K = f;
    a2.N = d;
    a2.ldo = d;
    a2.up_row = 0;
    a2.n_tiles = (int)ceil_div(d, BNW);
    a2.split_info = tinfo ? tinfo + 1 : nullptr;
    a2.product = 1;
    a2.a_rows = nullptr;
    if (!small)
        hipLaunchKernelGGL((grouped_gemm_kernel<false, false>), dim3(grid), dim3(GEMM_THREADS), 0, s,
                           a2);
    StreamArgs s2 = s1;
    for (int i = 0; i < MOE_MAX_GROUPS; ++i) s2.w[i] = a2.w[i];
    s2.a = h;
    s2.out = (bf16_t*)y_perm;
    s2.K = f;
    s2.N = d;
    s2.ldo = d;
    s2.a_rows = nullptr;
    s2.product = 1;
    if (!large)
        hipLaunchKernelGGL(stream_gemm_kernel<false>, dim3(sgrid), dim3(ST_THREADS), 0, s, s2);
    if (combine == nullptr) {
        hipLaunchKernelGGL(split_reduce_kernel<false>, dim3(rgrid), dim3(ST_THREADS), 0, s, s2, a2);
        return launch_status();
    }
    // the down product's chunk sum writes the combined output (every group streamed)
    const CombineArgs& cb = *(const CombineArgs*)combine;
    int64_t cgrid = ceil_div(cb.T * (d / 4), ST_THREADS);
    if (cgrid > 4096) cgrid = 4096;
    if (cgrid < 1) cgrid = 1;
#define MOE_RC(KM)                                                                               \
    hipLaunchKernelGGL(stream_reduce_combine_kernel<KM>, dim3((unsigned)cgrid), dim3(ST_THREADS), \
                       0, s, s2, cb)
    if (cb.k <= 2) MOE_RC(2);
    else if (cb.k <= 4) MOE_RC(4);
    else if (cb.k <= 8) MOE_RC(8);
    else MOE_RC(MOE_MAX_K);
#undef MOE_RC
    return launch_status();
}

int launch_grouped_ffn_combine(const void* x_perm, const int32_t* offsets, int n_groups,
                               const void* const* w13, const void* const* w2, int d, int f,
                               int64_t cap_rows, const int32_t* token_row, const float* gate,
                               const void* y_shared, int64_t T, int k, void* y, void* ws,
                               hipStream_t s) {
    if (T == 0) return MOE_OK;
    CombineArgs cb;
    cb.token_row = token_row;
    cb.gate = gate;
    cb.y_shared = (const bf16_t*)y_shared;
    cb.y = (bf16_t*)y;
    cb.T = T;
    cb.k = k;
    if (cap_rows == 0) {
        // no local row: y is the shared experts' output (or zero), as the combine gives
        return launch_combine(nullptr, MOE_BF16, token_row, gate, y_shared, 1, T, d, k, y, s);
    }
    return launch_grouped_ffn(x_perm, MOE_BF16, offsets, n_groups, w13, w2, d, f, cap_rows,
                              nullptr, ws, s, nullptr, 0,
                              MOE_FFN_GATE_UP | MOE_FFN_DOWN | MOE_FFN_SMALL_GROUPS, &cb);
}

}  // namespace moe
