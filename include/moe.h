/*
 * moe.h -- C ABI of the MI355X (gfx950) library for one GPU's share of one
 * expert-parallel MoE layer, the layer whose routing statistics Director
 * (arXiv 2607.08782) turns into expert placements.
 *
 * The share runs five steps, one entry point each, all enqueued on the
 * caller's HIP stream:
 *   moe_route_topk        gate scores and top-k routing            (Sec. II-A)
 *   moe_expert_histogram  per-expert workload counts W, co-activation
 *                                                     (Sec. VI-A; Sec. I)
 *   moe_permute           packaging of tokens for the experts placed on this
 *                         GPU, with per-GPU send counts (Sec. II-B; Eq. 1, 3)
 *   moe_grouped_ffn       the experts' FFNs over ragged groups of rows
 *                                                              (Sec. II-A)
 *   moe_combine           gate-weighted sum of expert outputs  (Sec. II-A)
 *
 * Conventions for every entry point
 *   - Pointers named "device" point to caller-owned device memory; pointers
 *     named "host" point to host memory that is read during the call and not
 *     kept.  The library allocates nothing and never synchronises the
 *     stream; outputs are valid once the stream reaches the end of the call.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Matrices are row-major and densely packed.  Element type codes:
 *     MOE_F32 (float) and MOE_BF16 (bfloat16, round-to-nearest-even stored).
 *     Gate scores, logits and gates are always float; indices int32.
 *   - Arguments are validated before anything is enqueued.  A non-zero
 *     status means nothing was enqueued, except MOE_ERR_DEVICE, which
 *     reports a HIP launch error (the stream state is then unspecified).
 *   - Entry points are stateless and reentrant; concurrent calls on
 *     different streams must use different output and workspace buffers.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types */
#define MOE_F32  0
#define MOE_BF16 1

/* status codes */
#define MOE_OK            0
#define MOE_ERR_ARG       1   /* null pointer, negative size, k out of range, bad dtype/flags */
#define MOE_ERR_PLACEMENT 2   /* an expert with no host GPU, dev >= G, or more than c_max local experts */
#define MOE_ERR_SHAPE     3   /* unsupported d or f, cap_rows or workspace too small */
#define MOE_ERR_DEVICE    4   /* a HIP launch failed */

/* products of moe_grouped_ffn_products */
#define MOE_FFN_GATE_UP 1   /* h = SiLU(W1 x) * (W3 x), kept in the workspace */
#define MOE_FFN_DOWN    2   /* y = W2 h, from the workspace */
#define MOE_FFN_SMALL_GROUPS 4   /* hint: no group has more than 256 rows; all are streamed */
#define MOE_FFN_LARGE_GROUPS 8   /* hint: every non-empty group has more than 256 rows; none is streamed */

/* flags of moe_route_topk */
#define MOE_RENORM    1   /* gates = softmax over the k selected logits (else: full softmax, restricted) */
#define MOE_LOGITS_IN 2   /* skip the gate GEMM: `logits` is an input holding T*E scores */

/* limits */
#define MOE_MAX_E      256   /* experts per layer */
#define MOE_MAX_K      16    /* experts per token */
#define MOE_MAX_G      64    /* GPUs in the placement map */
#define MOE_MAX_GROUPS 128   /* local expert groups per moe_grouped_ffn call */
#define MOE_PERMUTE_NOALLOC_MAX_WS (4 << 20)   /* scratch bytes of moe_permute_noalloc */

/* Human-readable name of a status code (static string). */
const char* moe_status_string(int status);

/*
 * moe_route_topk -- gate scores and top-k routing (Sec. II-A: the gating
 * network scores every expert for each token and the token goes to the k
 * best; the gate is replicated on every GPU, Sec. II-B).
 *
 *   logits[t][e] = sum_i x[t][i] * w_router[e][i] + bias[e]     (fp32 accumulate)
 *   topk_idx[t][r] = r-th best expert of token t: descending logit; equal
 *                    logits (-0.0 == +0.0) go to the lower expert index
 *   topk_gate[t][r] = exp(l_r - l_0) / sum_{r'<k} exp(l_r' - l_0)  with MOE_RENORM,
 *                     else exp(l_r - l_0) / sum_{e<E} exp(l_e - l_0)
 *
 * x         device [T][d] of `dtype`        (unused with MOE_LOGITS_IN; may be NULL then)
 * w_router  device [E][d] of `dtype`        (unused with MOE_LOGITS_IN)
 * bias      device [E] float, nullable (= 0)
 * logits    device [T][E] float: output, or input with MOE_LOGITS_IN; nullable
 *           otherwise (then the scores are not stored)
 * topk_idx  device [T][k] int32 output;  topk_gate  device [T][k] float output
 * ws        device workspace of moe_route_topk_ws_bytes(dtype, T, d, E, flags)
 *           bytes, 256-byte aligned; may be NULL when that size is 0.  (Short
 *           batches split the gate GEMM over K across workgroups and keep the
 *           per-chunk fp32 partial scores here; they are summed in chunk order.)
 * Requires 1 <= E <= MOE_MAX_E, 1 <= k <= min(E, MOE_MAX_K), T >= 0,
 * d >= 1 and, for MOE_BF16, d % 8 == 0 and E * d * 2 < 2^31 (else
 * MOE_ERR_SHAPE).  Logits must be finite.
 * Scores are deterministic: the same inputs give bitwise the same outputs.
 */
int moe_route_topk(const void* x, int dtype, const void* w_router, const float* bias,
                   int64_t T, int d, int E, int k, int flags,
                   float* logits, int32_t* topk_idx, float* topk_gate,
                   void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes moe_route_topk needs (0 = none). */
size_t moe_route_topk_ws_bytes(int dtype, int64_t T, int d, int E, int flags);

/*
 * moe_expert_histogram -- per-expert workload counts (Sec. VI-A: W_{j,i}
 * counts tokens routed to expert i; this share routes all T tokens, so
 * counts[e] is the inner sum of Eq. 1) and co-activation counts (the signal
 * for co-locating experts activated together, Sec. I).
 *
 *   counts[e]   = #{(t, r) : topk_idx[t][r] == e}
 *   coact[a][b] = #{t : a and b both among topk_idx[t][0..k-1]}   (diag = counts)
 *
 * topk_idx  device [T][k] int32, values in [0, E), distinct within a row
 * counts    device [E] int32 output (overwritten)
 * coact     device [E][E] int32 output, nullable (not computed)
 * Results are exact integers and independent of scheduling.
 */
int moe_expert_histogram(const int32_t* topk_idx, int64_t T, int k, int E,
                         int32_t* counts, int32_t* coact, void* stream);

/* Workspace bytes moe_permute needs for T tokens, k and E. */
size_t moe_permute_ws_bytes(int64_t T, int k, int E);

/*
 * moe_permute -- package the tokens for the experts placed on GPU `dev`
 * (Sec. II-B: tokens are packaged and sent to the GPUs hosting their
 * experts; Sec. VI-A: placement x[e][j], every expert hosted at least once,
 * Eq. 6d, at most C_max experts per GPU, Eq. 6e).
 *
 * placement  HOST [E][G] uint8, x[e][j] = placement[e*G + j] != 0
 * Local slot s = the s-th expert, by ascending id, with x[e][dev] = 1;
 * n_local = number of local slots.  An expert with n_e hosts splits its
 * tokens (ascending token order, c_e = counts[e] of them) into contiguous
 * blocks: its q-th host by ascending GPU id serves ranks
 * [floor(q*c_e/n_e), floor((q+1)*c_e/n_e)).  (The paper allows replicas but
 * leaves the split open; this is the rule the library fixes.)
 *
 * Outputs (rows are grouped by slot, ascending token order inside a group):
 *   group_offsets device [n_local+1] int32: exclusive prefix sum of rows per slot;
 *                 N = group_offsets[n_local] rows are written
 *   x_perm        device [cap_rows][d] of `dtype`: x_perm[p] = x[row_token[p]]
 *   row_token     device [cap_rows] int32;  row_gate  device [cap_rows] float
 *   token_row     device [T][k] int32: row of assignment (t, r) here, or -1
 *   send_counts   device [G] int32, nullable: rows each GPU's hosts take,
 *                 i.e. Eq. 3's D_{dev,j} / d; equals Eq. 1's lambda_j when
 *                 no expert is replicated
 * counts  device [E] int32 from moe_expert_histogram on the same topk_idx.
 * c_max   0 = unchecked, else MOE_ERR_PLACEMENT if n_local > c_max.
 * ws      device workspace of at least moe_permute_ws_bytes(T, k, E) bytes,
 *         256-byte aligned.
 * Requires cap_rows >= T * min(k, n_local), G <= MOE_MAX_G, and for
 * MOE_BF16 d % 8 == 0.  Rows past N are left untouched.
 */
int moe_permute(const void* x, int dtype, const int32_t* topk_idx, const float* topk_gate,
                const int32_t* counts, int64_t T, int d, int k, int E,
                const uint8_t* placement, int G, int dev, int c_max,
                void* x_perm, int64_t cap_rows, int32_t* group_offsets,
                int32_t* row_token, float* row_gate, int32_t* token_row,
                int32_t* send_counts, void* ws, size_t ws_bytes, void* stream);

/*
 * moe_permute_noalloc -- moe_permute without a workspace argument, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  It packages the tokens
 * exactly as moe_permute does (same outputs, bit for bit) and keeps the
 * per-block counts it needs in a scratch array of this library: one copy per
 * GPU, MOE_PERMUTE_NOALLOC_MAX_WS (4 MiB) bytes, held until the process ends.
 * The call allocates nothing; its first call on a GPU looks up that GPU's
 * copy of the array.
 *
 * Arguments, outputs and errors as for moe_permute, without ws / ws_bytes.
 * Returns MOE_ERR_SHAPE when moe_permute_ws_bytes(T, k, E) exceeds
 * MOE_PERMUTE_NOALLOC_MAX_WS (more than about 524 000 tokens at 128 local
 * slots), and MOE_ERR_DEVICE if the scratch cannot be located on the current
 * device.  The scratch keeps the last call's contents; every call on one GPU
 * shares it, so calls that overlap in time on one GPU (different streams, or
 * different threads) race and must be serialised by the caller.
 */
int moe_permute_noalloc(const void* x, int dtype, const int32_t* topk_idx,
                        const float* topk_gate, const int32_t* counts, int64_t T, int d, int k,
                        int E, const uint8_t* placement, int G, int dev, int c_max, void* x_perm,
                        int64_t cap_rows, int32_t* group_offsets, int32_t* row_token,
                        float* row_gate, int32_t* token_row, int32_t* send_counts, void* stream);

/* Workspace bytes moe_grouped_ffn needs. */
size_t moe_grouped_ffn_ws_bytes(int dtype, int64_t cap_rows, int d, int f, int n_groups);

/*
 * moe_grouped_ffn -- every local expert's FFN on its group of rows
 * (Sec. II-A: experts are FFN sub-networks).  Experts are SwiGLU:
 *
 *   for each slot s and row p in [group_offsets[s], group_offsets[s+1]):
 *     a = W1_s x_perm[p],  b = W3_s x_perm[p]               (f values each)
 *     h = SiLU(a) * b,     SiLU(a) = a / (1 + exp(-a))
 *     y_perm[p] = W2_s h
 *
 * x_perm         device [cap_rows][d] of `dtype`
 * group_offsets  device [n_groups+1] int32, non-decreasing, offsets[0] = 0,
 *                offsets[n_groups] <= cap_rows (read on the device only)
 * w13            HOST array of n_groups device pointers; w13[s] is [2f][d]:
 *                rows 0..f-1 are W1_s (gate), rows f..2f-1 are W3_s (up)
 * w2             HOST array of n_groups device pointers; w2[s] is [d][f]
 * y_perm         device [cap_rows][d] of `dtype` output (rows past
 *                offsets[n_groups] untouched)
 * ws             device workspace, moe_grouped_ffn_ws_bytes(...) bytes,
 *                256-byte aligned
 * For MOE_BF16 the products accumulate in fp32 and h is rounded to bf16
 * before the second product.  Requires 1 <= n_groups <= MOE_MAX_GROUPS and
 * for MOE_BF16 d % 64 == 0, f % 64 == 0 and d, f < 2^22 (else MOE_ERR_SHAPE).
 * A shared (always-on) expert is the call with x_perm = x, one group and
 * group_offsets = {0, T}.
 */
int moe_grouped_ffn(const void* x_perm, int dtype, const int32_t* group_offsets, int n_groups,
                    const void* const* w13, const void* const* w2, int d, int f,
                    int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_products -- moe_grouped_ffn run one product at a time
 * (Sec. II-A: the expert FFN is the two products of the SwiGLU block), for
 * callers that schedule or time the two separately.  products is a mask:
 *   MOE_FFN_GATE_UP  h = SiLU(W1_s x_perm[p]) * (W3_s x_perm[p]) for every row,
 *                    kept in ws (with the call's group plan)
 *   MOE_FFN_DOWN     y_perm[p] = W2_s h[p], reading h and the plan from ws
 * MOE_FFN_GATE_UP | MOE_FFN_DOWN is exactly moe_grouped_ffn.  A
 * MOE_FFN_DOWN call must follow a MOE_FFN_GATE_UP call on the same stream
 * with the same ws, group_offsets (unchanged contents), n_groups, d, f and
 * cap_rows; ws must not be used in between.  The two calls in sequence give
 * bitwise the outputs of moe_grouped_ffn.  x_perm and w13 are read only with
 * MOE_FFN_GATE_UP (may be NULL otherwise), y_perm and w2 only with
 * MOE_FFN_DOWN.  Other arguments, requirements and errors as for
 * moe_grouped_ffn; products outside {1, 2, 3} give MOE_ERR_ARG.
 * Adding MOE_FFN_SMALL_GROUPS to products states that no group holds more
 * than 256 rows (true of a batch of at most 256 tokens: a token reaches an
 * expert at most once).  Every group then takes the weight-streaming kernels
 * and the call skips the launches of the tiled kernels.  Without the flag a
 * call streams every group of at most 256 rows when its groups above 64 rows
 * make few tiles (always so when no group holds more than 64 rows), and tiles
 * every group otherwise; so a call whose groups all hold at most 64 rows gives
 * bitwise the outputs it gives without the flag, and a group that the call
 * without the flag would tile sums its products in another order (same
 * tolerance).  Rows of a group that breaks the statement are left unwritten.  It must be passed the same way to
 * the MOE_FFN_GATE_UP and the MOE_FFN_DOWN call of one pair.
 * Adding MOE_FFN_LARGE_GROUPS instead states that every non-empty group holds
 * more than 256 rows (true of a shared expert's call over more than 256
 * tokens): every group then takes the tiled kernels and the call skips the
 * weight-streaming launches.  Such a call gives bitwise the outputs it gives
 * without the flag; a group that breaks the statement is still computed in
 * full, by the tiled kernels (its products summed in another order, same
 * tolerance).  It must be passed the same way to both calls of a pair; the
 * two hints together give MOE_ERR_ARG.
 */
int moe_grouped_ffn_products(const void* x_perm, int dtype, const int32_t* group_offsets,
                             int n_groups, const void* const* w13, const void* const* w2, int d,
                             int f, int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                             int products, void* stream);

/*
 * moe_grouped_ffn_combine -- moe_grouped_ffn followed by moe_combine, for calls
 * in which no group holds more than 256 rows (a batch of at most 256 tokens;
 * the MOE_FFN_SMALL_GROUPS statement): the expert outputs are combined inside the
 * down product's fixed-order sum of its K chunks (the gate-weighted sum of
 * Sec. II-A, the return trip of Sec. II-B), so y_perm is neither written nor
 * read back and the combine needs no launch of its own:
 *
 *   y[t] = sum_{r ascending, token_row[t][r] >= 0} topk_gate[t][r] * y_perm[token_row[t][r]]
 *          + y_shared[t]
 *
 * with y_perm[p] the bf16 value moe_grouped_ffn with MOE_FFN_SMALL_GROUPS would
 * store, summed in fp32 in the order moe_combine uses: bitwise that call
 * followed by moe_combine.
 * x_perm, group_offsets, n_groups, w13, w2, d, f, cap_rows and ws as for
 * moe_grouped_ffn; token_row, topk_gate, y_shared (nullable), T, k and y as for
 * moe_combine.  MOE_BF16 only (MOE_ERR_ARG otherwise).  Rows of a group that
 * holds more than 256 rows are left out of y.  If y_shared comes from another
 * stream, that stream must be joined before this call.
 */
int moe_grouped_ffn_combine(const void* x_perm, int dtype, const int32_t* group_offsets,
                            int n_groups, const void* const* w13, const void* const* w2, int d,
                            int f, int64_t cap_rows, const int32_t* token_row,
                            const float* topk_gate, const void* y_shared, int64_t T, int k,
                            void* y, void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_rows -- moe_grouped_ffn whose first product reads row p of
 * its input straight from the token rows, x[row_token[p]], instead of from a
 * packaged copy: the row map of the packaging step (Sec. II-B) is kept and the
 * copy of the rows, x_perm, is never written or read.  This is the one-GPU
 * part of fusing the dispatch gather into the expert GEMM; with moe_permute
 * called with d = 0 (row maps only) the outputs are bitwise identical to
 * moe_permute + moe_grouped_ffn.
 *
 * x          device [T][d] of `dtype`: the token rows
 * row_token  device [cap_rows] int32 (moe_permute's row map): entries of rows
 *            below group_offsets[n_groups] must lie in [0, T)
 * other arguments, workspace (moe_grouped_ffn_ws_bytes) and outputs as for
 * moe_grouped_ffn.  bf16 requires T * d * 2 < 2^31 (32-bit row offsets),
 * else MOE_ERR_SHAPE, and 16-byte aligned x.
 */
int moe_grouped_ffn_rows(const void* x, int64_t T, const int32_t* row_token, int dtype,
                         const int32_t* group_offsets, int n_groups, const void* const* w13,
                         const void* const* w2, int d, int f, int64_t cap_rows, void* y_perm,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_rows_products -- moe_grouped_ffn_rows with the products mask of
 * moe_grouped_ffn_products (one product at a time, and the MOE_FFN_SMALL_GROUPS
 * or MOE_FFN_LARGE_GROUPS statement, with the same meaning and the same
 * outputs): x and row_token are read only with MOE_FFN_GATE_UP (may be NULL
 * otherwise), y_perm and w2 only with MOE_FFN_DOWN.  Other arguments,
 * requirements and errors as for moe_grouped_ffn_rows; MOE_FFN_GATE_UP |
 * MOE_FFN_DOWN is exactly moe_grouped_ffn_rows.
 */
int moe_grouped_ffn_rows_products(const void* x, int64_t T, const int32_t* row_token, int dtype,
                                  const int32_t* group_offsets, int n_groups,
                                  const void* const* w13, const void* const* w2, int d, int f,
                                  int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                                  int products, void* stream);

/*
 * moe_grouped_ffn_rows_shared -- moe_grouped_ffn_rows_products with the
 * always-on shared experts (Sec. II-A: every token also passes through them)
 * computed in the same launches as the routed experts, as n_shared leading
 * groups of T rows each: one call instead of a second FFN call, so the tiles of
 * both fill the GPU together.  A shared expert of width m * f takes m groups
 * (its gate, up and down rows cut into m blocks of f: SwiGLU is elementwise in
 * h, and the down product sums over h, so the m outputs sum to the expert's).
 *
 *   group s < n_shared       rows [s T, (s+1) T), weights w13[s], w2[s]
 *   routed group g            rows n_shared T + [group_offsets[g], group_offsets[g+1]),
 *                             weights w13[n_shared + g], w2[n_shared + g]
 *
 * row_token  device [n_shared T + cap_rows] int32: the caller's entries for the
 *            shared rows (row s T + t is token t: 0, 1, ..., T-1 per group,
 *            written once and kept), then the routed rows' map (moe_permute's
 *            row_token written at row_token + n_shared T)
 * group_offsets  device [n_groups+1], the routed groups as moe_permute writes
 *            them (n_groups may be 0: only group_offsets[0] = 0 is then read)
 * w13, w2    HOST arrays of n_shared + n_groups device pointers, shared first
 * cap_rows   routed row capacity;  y_perm device [n_shared T + cap_rows][d]: group
 *            s's output in rows [s T, (s+1) T) (the n_shared slices that
 *            moe_combine_shared adds), routed rows from n_shared T
 * ws         moe_grouped_ffn_ws_bytes(dtype, n_shared T + cap_rows, d, f,
 *            n_shared + n_groups) bytes
 * products   as for moe_grouped_ffn_rows_products; the hints state the sizes of
 *            every group, shared ones included.
 * Requires 0 <= n_shared, 1 <= n_shared + n_groups <= MOE_MAX_GROUPS, T >= 1
 * when n_shared > 0 and n_shared T + cap_rows < 2^31; other requirements and
 * errors as for moe_grouped_ffn_rows.  With n_shared = 0 it is
 * moe_grouped_ffn_rows_products.
 */
int moe_grouped_ffn_rows_shared(const void* x, int64_t T, const int32_t* row_token, int dtype,
                                const int32_t* group_offsets, int n_groups, int n_shared,
                                const void* const* w13, const void* const* w2, int d, int f,
                                int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                                int products, void* stream);

/*
 * moe_combine -- gate-weighted sum of the experts' outputs (Sec. II-A) back
 * in token order (the return trip of Sec. II-B), plus shared experts with
 * weight 1:
 *
 *   y[t] = sum_{r ascending, token_row[t][r] >= 0} topk_gate[t][r] * y_perm[token_row[t][r]]
 *          + y_shared[t]
 *
 * y_perm    device [rows][d] of `dtype`, required when T > 0 (it may hold
 *           no rows that any token uses);  token_row device [T][k] int32
 * topk_gate device [T][k] float;  y_shared device [T][d] of `dtype`, nullable
 * y         device [T][d] of `dtype` output (fp32 accumulation, then stored).
 * Tokens with no local assignment get y_shared[t] (or 0).
 */
int moe_combine(const void* y_perm, int dtype, const int32_t* token_row, const float* topk_gate,
                const void* y_shared, int64_t T, int d, int k, void* y, void* stream);

/*
 * moe_combine_shared -- moe_combine with the shared experts' output in
 * n_shared slices (as moe_grouped_ffn_rows_shared leaves it), added after the
 * routed sum in slice order:
 *
 *   y[t] = sum_{r ascending, token_row[t][r] >= 0} topk_gate[t][r] * y_perm[token_row[t][r]]
 *          + y_shared[0][t] + y_shared[1][t] + ... + y_shared[n_shared-1][t]
 *
 * y_shared  device [n_shared][T][d] of `dtype` (NULL or n_shared = 0: none).
 * Requires 0 <= n_shared <= MOE_MAX_GROUPS; other arguments as for
 * moe_combine.  n_shared = 1 is exactly moe_combine.
 */
int moe_combine_shared(const void* y_perm, int dtype, const int32_t* token_row,
                       const float* topk_gate, const void* y_shared, int n_shared, int64_t T,
                       int d, int k, void* y, void* stream);

/*
 * moe_quantize_e4m3 -- per-row FP8 quantization for the quantized routing
 * predictor (Sec. V-A: a low-bit replica with weights and activations both
 * quantized; gfx950 multiplies OCP FP8 E4M3 natively).  For every row r:
 *
 *   scales[r] = max_i |x[r][i]| / 448          (fp32 division; 1 if the row is 0)
 *   q[r][i]   = E4M3(x[r][i] / scales[r])      (fp32 division, round to nearest,
 *                                               ties to even; |.| > 448 saturates)
 *
 * E4M3: 1 sign, 4 exponent bits (bias 7), 3 mantissa bits, subnormals, max 448,
 * no infinities; a value that rounds to zero is stored as +0 (code 0x00).
 * x       device [rows][cols] of `dtype` (MOE_F32 or MOE_BF16), finite
 * q       device [rows][cols] uint8 output;  scales device [rows] float output
 * Requires rows >= 0, cols >= 1.  Results are exact (bitwise reproducible).
 */
int moe_quantize_e4m3(const void* x, int dtype, int64_t rows, int cols, uint8_t* q,
                      float* scales, void* stream);

/*
 * moe_route_topk_e4m3 -- gate scores of the quantized predictor (Sec. V-A)
 * and their top-k, whose agreement with moe_route_topk's choice is the
 * predictor's accuracy (top-k match rate, Sec. VIII):
 *
 *   logits[t][e] = x_scale[t] * w_scale[e] * sum_i E4M3(xq[t][i]) * E4M3(wq[e][i])
 *                  + bias[e]
 *
 * then top-k and gates exactly as moe_route_topk does for given scores.
 * xq       device [T][d] uint8 E4M3 codes, x_scale device [T] float (from
 *          moe_quantize_e4m3 of the activations)
 * wq       device [E][d] uint8 E4M3 codes, w_scale device [E] float (of the
 *          router weights [E][d])
 * bias     device [E] float, nullable
 * logits   device [T][E] float output (required: the top-k reads it back)
 * topk_idx device [T][k] int32 output;  topk_gate device [T][k] float output
 * flags    MOE_RENORM or 0
 * Requires d % 64 == 0, xq and wq 16-byte aligned, 1 <= E <= MOE_MAX_E,
 * 1 <= k <= min(E, MOE_MAX_K), T >= 0.  The code products are exact in fp32;
 * their sum is accumulated in fp32 in a fixed order (deterministic).
 */
int moe_route_topk_e4m3(const uint8_t* xq, const float* x_scale, const uint8_t* wq,
                        const float* w_scale, const float* bias, int64_t T, int d, int E, int k,
                        int flags, float* logits, int32_t* topk_idx, float* topk_gate,
                        void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
