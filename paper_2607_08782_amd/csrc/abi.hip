// C ABI entry points: argument validation, placement map -> slot tables,
// then the launches of each step on the caller's stream.  Nothing here
// allocates device memory or synchronises.
#include <string.h>

#include "common.h"

namespace {

using namespace moe;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

const char* moe_status_string(int status) {
    switch (status) {
        case MOE_OK: return "ok";
        case MOE_ERR_ARG: return "invalid argument";
        case MOE_ERR_PLACEMENT: return "invalid placement map";
        case MOE_ERR_SHAPE: return "unsupported shape, capacity or workspace size";
        case MOE_ERR_DEVICE: return "HIP launch error";
        default: return "unknown status";
    }
}

size_t moe_route_topk_ws_bytes(int dtype, int64_t T, int d, int E, int flags) {
    if (T < 0 || d < 0 || E < 1) return 0;
    return route_ws_bytes(dtype, T, d, E, flags);
}

int moe_route_topk(const void* x, int dtype, const void* w_router, const float* bias, int64_t T,
                   int d, int E, int k, int flags, float* logits, int32_t* topk_idx,
                   float* topk_gate, void* ws, size_t ws_bytes, void* stream) {
    if (T < 0 || E < 1 || E > MOE_MAX_E || k < 1 || k > MOE_MAX_K || k > E) return MOE_ERR_ARG;
    if (flags & ~(MOE_RENORM | MOE_LOGITS_IN)) return MOE_ERR_ARG;
    if (T > (int64_t)0x7fffffff * 16) return MOE_ERR_ARG;
    if (T > 0 && (!topk_idx || !topk_gate)) return MOE_ERR_ARG;
    if (flags & MOE_LOGITS_IN) {
        if (T > 0 && !logits) return MOE_ERR_ARG;
    } else {
        if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
        if (d < 1) return MOE_ERR_ARG;
        if (T > 0 && (!x || !w_router)) return MOE_ERR_ARG;
        if (dtype == MOE_BF16) {
            if (d % 8) return MOE_ERR_SHAPE;
            // the router matrix is addressed through one 32-bit buffer descriptor
            if ((int64_t)E * d * 2 > 0x7fffffffLL) return MOE_ERR_SHAPE;
            if (!aligned16(x) || !aligned16(w_router)) return MOE_ERR_ARG;
        }
    }
    const size_t need = route_ws_bytes(dtype, T, d, E, flags);
    if (need > 0 && (!ws || ws_bytes < need || ((uintptr_t)ws & 255u))) return MOE_ERR_SHAPE;
    return launch_route_topk(x, dtype, w_router, bias, T, d, E, k, flags, logits, topk_idx,
                             topk_gate, ws, (hipStream_t)stream);
}

int moe_expert_histogram(const int32_t* topk_idx, int64_t T, int k, int E, int32_t* counts,
                         int32_t* coact, void* stream) {
    if (T < 0 || E < 1 || E > MOE_MAX_E || k < 1 || k > MOE_MAX_K || k > E) return MOE_ERR_ARG;
    if (!counts || (T > 0 && !topk_idx)) return MOE_ERR_ARG;
    return launch_histogram(topk_idx, T, k, E, counts, coact, (hipStream_t)stream);
}

size_t moe_permute_ws_bytes(int64_t T, int k, int E) {
    if (T < 0 || k < 1 || E < 1) return 0;
    return permute_ws_bytes(T, k, E);
}

}  // extern "C"

namespace {

// Validation shared by moe_permute and moe_permute_noalloc, and the slot /
// host tables built from the placement map.
int permute_check(const void* x, int dtype, const int32_t* topk_idx, const float* topk_gate,
                  const int32_t* counts, int64_t T, int d, int k, int E,
                  const uint8_t* placement, int G, int dev, int c_max, void* x_perm,
                  int64_t cap_rows, int32_t* group_offsets, int32_t* row_token,
                  float* row_gate, int32_t* token_row, PermuteTables& tab, int& n_local) {
    if (T < 0 || d < 0 || E < 1 || E > MOE_MAX_E || k < 1 || k > MOE_MAX_K || k > E)
        return MOE_ERR_ARG;
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
    if (T * (int64_t)k > 0x7fffffff) return MOE_ERR_ARG;
    if (!placement || !group_offsets || !counts || cap_rows < 0) return MOE_ERR_ARG;
    if (G < 1 || G > MOE_MAX_G || dev < 0 || dev >= G) return MOE_ERR_PLACEMENT;
    if (T > 0 && (!topk_idx || !topk_gate || !token_row)) return MOE_ERR_ARG;

    memset(&tab, 0, sizeof(tab));
    for (int e = 0; e < MOE_MAX_E; ++e) tab.slot_of[e] = -1;
    n_local = 0;
    for (int e = 0; e < E; ++e) {
        uint64_t h = 0;
        for (int j = 0; j < G; ++j)
            if (placement[(int64_t)e * G + j]) h |= 1ull << j;
        if (!h) return MOE_ERR_PLACEMENT;
        tab.hosts[e] = h;
        if ((h >> dev) & 1ull) {
            if (n_local >= MOE_MAX_GROUPS) return MOE_ERR_PLACEMENT;
            tab.slot_of[e] = (int16_t)n_local;
            tab.expert_of_slot[n_local] = (int16_t)e;
            ++n_local;
        }
    }
    if (c_max > 0 && n_local > c_max) return MOE_ERR_PLACEMENT;
    const int64_t need_rows = T * (int64_t)(k < n_local ? k : n_local);
    if (cap_rows < need_rows) return MOE_ERR_SHAPE;
    if (dtype == MOE_BF16 && d % 8) return MOE_ERR_SHAPE;
    if (need_rows > 0 && (!row_token || !row_gate || (d > 0 && (!x || !x_perm))))
        return MOE_ERR_ARG;
    return MOE_OK;
}

}  // namespace

extern "C" {

int moe_permute(const void* x, int dtype, const int32_t* topk_idx, const float* topk_gate,
                const int32_t* counts, int64_t T, int d, int k, int E, const uint8_t* placement,
                int G, int dev, int c_max, void* x_perm, int64_t cap_rows,
                int32_t* group_offsets, int32_t* row_token, float* row_gate, int32_t* token_row,
                int32_t* send_counts, void* ws, size_t ws_bytes, void* stream) {
    PermuteTables tab;
    int n_local = 0;
    const int st = permute_check(x, dtype, topk_idx, topk_gate, counts, T, d, k, E, placement, G,
                                 dev, c_max, x_perm, cap_rows, group_offsets, row_token, row_gate,
                                 token_row, tab, n_local);
    if (st != MOE_OK) return st;
    if (!ws || ws_bytes < permute_ws_bytes(T, k, E) || ((uintptr_t)ws & 255u)) return MOE_ERR_SHAPE;
    return launch_permute(x, dtype, topk_idx, topk_gate, counts, T, d, k, E, tab, n_local, G, dev,
                          x_perm, cap_rows, group_offsets, row_token, row_gate, token_row,
                          send_counts, ws, (hipStream_t)stream);
}

int moe_permute_noalloc(const void* x, int dtype, const int32_t* topk_idx,
                        const float* topk_gate, const int32_t* counts, int64_t T, int d, int k,
                        int E, const uint8_t* placement, int G, int dev, int c_max, void* x_perm,
                        int64_t cap_rows, int32_t* group_offsets, int32_t* row_token,
                        float* row_gate, int32_t* token_row, int32_t* send_counts, void* stream) {
    PermuteTables tab;
    int n_local = 0;
    const int st = permute_check(x, dtype, topk_idx, topk_gate, counts, T, d, k, E, placement, G,
                                 dev, c_max, x_perm, cap_rows, group_offsets, row_token, row_gate,
                                 token_row, tab, n_local);
    if (st != MOE_OK) return st;
    if (permute_ws_bytes(T, k, E) > (size_t)MOE_PERMUTE_NOALLOC_MAX_WS) return MOE_ERR_SHAPE;
    void* ws = nullptr;
    if (permute_scratch(&ws) != MOE_OK) return MOE_ERR_DEVICE;
    return launch_permute(x, dtype, topk_idx, topk_gate, counts, T, d, k, E, tab, n_local, G, dev,
                          x_perm, cap_rows, group_offsets, row_token, row_gate, token_row,
                          send_counts, ws, (hipStream_t)stream);
}

size_t moe_grouped_ffn_ws_bytes(int dtype, int64_t cap_rows, int d, int f, int n_groups) {
    if (cap_rows < 0 || d < 1 || f < 1) return 0;
    return grouped_ffn_ws_bytes(dtype, cap_rows, d, f, n_groups);
}

}  // extern "C"

namespace {

// Validation of a grouped FFN call that runs `products` (a mask of
// MOE_FFN_GATE_UP and MOE_FFN_DOWN): the operands of the products it runs.
int ffn_check(const void* x_perm, int dtype, const int32_t* group_offsets, int n_groups,
              const void* const* w13, const void* const* w2, int d, int f, int64_t cap_rows,
              const void* y_perm, const void* ws, size_t ws_bytes, int products) {
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
    if (products & ~(MOE_FFN_GATE_UP | MOE_FFN_DOWN | MOE_FFN_SMALL_GROUPS | MOE_FFN_LARGE_GROUPS))
        return MOE_ERR_ARG;
    if ((products & MOE_FFN_SMALL_GROUPS) && (products & MOE_FFN_LARGE_GROUPS)) return MOE_ERR_ARG;
    const bool up = products & MOE_FFN_GATE_UP, down = products & MOE_FFN_DOWN;
    if (!up && !down) return MOE_ERR_ARG;
    if (n_groups < 1 || n_groups > MOE_MAX_GROUPS || d < 1 || f < 1 || cap_rows < 0)
        return MOE_ERR_ARG;
    if (cap_rows > 0x7fffffff) return MOE_ERR_ARG;
    if (!group_offsets || (up && !w13) || (down && !w2)) return MOE_ERR_ARG;
    for (int s = 0; s < n_groups; ++s)
        if ((up && !w13[s]) || (down && !w2[s])) return MOE_ERR_ARG;
    if (cap_rows > 0 && ((up && !x_perm) || (down && !y_perm))) return MOE_ERR_ARG;
    if (dtype == MOE_BF16) {
        if (d % 64 || f % 64) return MOE_ERR_SHAPE;
        // a 256-row tile of either product spans 256 rows of d or f elements in 32-bit
        // byte offsets
        if ((int64_t)d * 512 > 0x7fffffffLL || (int64_t)f * 512 > 0x7fffffffLL) return MOE_ERR_SHAPE;
        if ((x_perm && !aligned16(x_perm)) || (y_perm && !aligned16(y_perm))) return MOE_ERR_ARG;
        for (int s = 0; s < n_groups; ++s)
            if ((up && !aligned16(w13[s])) || (down && !aligned16(w2[s]))) return MOE_ERR_ARG;
    }
    if (cap_rows > 0 &&
        (!ws || ws_bytes < grouped_ffn_ws_bytes(dtype, cap_rows, d, f, n_groups) ||
         ((uintptr_t)ws & 255u)))
        return MOE_ERR_SHAPE;
    return MOE_OK;
}

}  // namespace

extern "C" {

int moe_grouped_ffn(const void* x_perm, int dtype, const int32_t* group_offsets, int n_groups,
                    const void* const* w13, const void* const* w2, int d, int f, int64_t cap_rows,
                    void* y_perm, void* ws, size_t ws_bytes, void* stream) {
    const int both = MOE_FFN_GATE_UP | MOE_FFN_DOWN;
    const int st = ffn_check(x_perm, dtype, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                             y_perm, ws, ws_bytes, both);
    if (st != MOE_OK) return st;
    return launch_grouped_ffn(x_perm, dtype, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                              y_perm, ws, (hipStream_t)stream);
}

int moe_grouped_ffn_products(const void* x_perm, int dtype, const int32_t* group_offsets,
                             int n_groups, const void* const* w13, const void* const* w2, int d,
                             int f, int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                             int products, void* stream) {
    const int st = ffn_check(x_perm, dtype, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                             y_perm, ws, ws_bytes, products);
    if (st != MOE_OK) return st;
    return launch_grouped_ffn(x_perm, dtype, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                              y_perm, ws, (hipStream_t)stream, nullptr, 0, products);
}

int moe_grouped_ffn_combine(const void* x_perm, int dtype, const int32_t* group_offsets,
                            int n_groups, const void* const* w13, const void* const* w2, int d,
                            int f, int64_t cap_rows, const int32_t* token_row,
                            const float* topk_gate, const void* y_shared, int64_t T, int k,
                            void* y, void* ws, size_t ws_bytes, void* stream) {
    if (dtype != MOE_BF16) return MOE_ERR_ARG;
    if (T < 0 || k < 1 || k > MOE_MAX_K) return MOE_ERR_ARG;
    if (T > 0 && (!token_row || !topk_gate || !y)) return MOE_ERR_ARG;
    if (T > 0 && (!aligned16(y) || (y_shared && !aligned16(y_shared)))) return MOE_ERR_ARG;
    const int st = ffn_check(x_perm, dtype, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                             T > 0 ? y : nullptr, ws, ws_bytes,
                             MOE_FFN_GATE_UP | MOE_FFN_DOWN | MOE_FFN_SMALL_GROUPS);
    if (st != MOE_OK) return st;
    return launch_grouped_ffn_combine(x_perm, group_offsets, n_groups, w13, w2, d, f, cap_rows,
                                      token_row, topk_gate, y_shared, T, k, y, ws,
                                      (hipStream_t)stream);
}

int moe_grouped_ffn_rows_shared(const void* x, int64_t T, const int32_t* row_token, int dtype,
                                const int32_t* group_offsets, int n_groups, int n_shared,
                                const void* const* w13, const void* const* w2, int d, int f,
                                int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                                int products, void* stream) {
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
    if (products & ~(MOE_FFN_GATE_UP | MOE_FFN_DOWN | MOE_FFN_SMALL_GROUPS | MOE_FFN_LARGE_GROUPS))
        return MOE_ERR_ARG;
    if ((products & MOE_FFN_SMALL_GROUPS) && (products & MOE_FFN_LARGE_GROUPS)) return MOE_ERR_ARG;
    const bool up = products & MOE_FFN_GATE_UP, down = products & MOE_FFN_DOWN;
    if (!up && !down) return MOE_ERR_ARG;
    if (n_shared < 0 || n_groups < 0 || n_shared > MOE_MAX_GROUPS) return MOE_ERR_ARG;
    const int groups = n_shared + n_groups;
    if (T < 0 || groups < 1 || groups > MOE_MAX_GROUPS || d < 1 || f < 1 || cap_rows < 0)
        return MOE_ERR_ARG;
    if (n_shared > 0 && T < 1) return MOE_ERR_ARG;
    // every row, shared and routed, is addressed with 32-bit row indices
    if (cap_rows > 0x7fffffff || (int64_t)n_shared * T > 0x7fffffffLL - cap_rows)
        return MOE_ERR_ARG;
    const int64_t rows = (int64_t)n_shared * T + cap_rows;
    if (!group_offsets || (up && !w13) || (down && !w2)) return MOE_ERR_ARG;
    for (int s = 0; s < groups; ++s)
        if ((up && !w13[s]) || (down && !w2[s])) return MOE_ERR_ARG;
    if (rows > 0 && ((up && (!x || !row_token || T < 1)) || (down && !y_perm)))
        return MOE_ERR_ARG;
    if (dtype == MOE_BF16) {
        if (d % 64 || f % 64) return MOE_ERR_SHAPE;
        // token rows are addressed through 32-bit buffer offsets, and so is a
        // 256-row tile of either product
        if (T * (int64_t)d * 2 > 0x7fffffffLL) return MOE_ERR_SHAPE;
        if ((int64_t)d * 512 > 0x7fffffffLL || (int64_t)f * 512 > 0x7fffffffLL) return MOE_ERR_SHAPE;
        if ((x && !aligned16(x)) || (y_perm && !aligned16(y_perm))) return MOE_ERR_ARG;
        for (int s = 0; s < groups; ++s)
            if ((up && !aligned16(w13[s])) || (down && !aligned16(w2[s]))) return MOE_ERR_ARG;
    }
    if (rows > 0 &&
        (!ws || ws_bytes < grouped_ffn_ws_bytes(dtype, rows, d, f, groups) ||
         ((uintptr_t)ws & 255u)))
        return MOE_ERR_SHAPE;
    return launch_grouped_ffn(x, dtype, group_offsets, groups, w13, w2, d, f, rows, y_perm, ws,
                              (hipStream_t)stream, row_token, T, products, nullptr, n_shared,
                              (int)T);
}

int moe_grouped_ffn_rows_products(const void* x, int64_t T, const int32_t* row_token, int dtype,
                                  const int32_t* group_offsets, int n_groups,
                                  const void* const* w13, const void* const* w2, int d, int f,
                                  int64_t cap_rows, void* y_perm, void* ws, size_t ws_bytes,
                                  int products, void* stream) {
    if (n_groups < 1) return MOE_ERR_ARG;
    return moe_grouped_ffn_rows_shared(x, T, row_token, dtype, group_offsets, n_groups, 0, w13, w2,
                                       d, f, cap_rows, y_perm, ws, ws_bytes, products, stream);
}

int moe_grouped_ffn_rows(const void* x, int64_t T, const int32_t* row_token, int dtype,
                         const int32_t* group_offsets, int n_groups, const void* const* w13,
                         const void* const* w2, int d, int f, int64_t cap_rows, void* y_perm,
                         void* ws, size_t ws_bytes, void* stream) {
    return moe_grouped_ffn_rows_products(x, T, row_token, dtype, group_offsets, n_groups, w13, w2,
                                         d, f, cap_rows, y_perm, ws, ws_bytes,
                                         MOE_FFN_GATE_UP | MOE_FFN_DOWN, stream);
}

int moe_combine_shared(const void* y_perm, int dtype, const int32_t* token_row,
                       const float* topk_gate, const void* y_shared, int n_shared, int64_t T,
                       int d, int k, void* y, void* stream) {
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
    if (T < 0 || d < 1 || k < 1 || k > MOE_MAX_K) return MOE_ERR_ARG;
    if (n_shared < 0 || n_shared > MOE_MAX_GROUPS) return MOE_ERR_ARG;
    if (T > 0 && (!token_row || !topk_gate || !y || !y_perm)) return MOE_ERR_ARG;
    if (n_shared == 0) y_shared = nullptr;
    const int V = dtype == MOE_BF16 ? 8 : 4;
    if (d % V == 0 && (!aligned16(y) || (y_perm && !aligned16(y_perm)) ||
                       (y_shared && !aligned16(y_shared))))
        return MOE_ERR_ARG;
    return launch_combine(y_perm, dtype, token_row, topk_gate, y_shared, n_shared, T, d, k, y,
                          (hipStream_t)stream);
}

int moe_combine(const void* y_perm, int dtype, const int32_t* token_row, const float* topk_gate,
                const void* y_shared, int64_t T, int d, int k, void* y, void* stream) {
    return moe_combine_shared(y_perm, dtype, token_row, topk_gate, y_shared, 1, T, d, k, y,
                              stream);
}

int moe_quantize_e4m3(const void* x, int dtype, int64_t rows, int cols, uint8_t* q,
                      float* scales, void* stream) {
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_ARG;
    if (rows < 0 || cols < 1) return MOE_ERR_ARG;
    if (rows > 0 && (!x || !q || !scales)) return MOE_ERR_ARG;
    return launch_quantize_e4m3(x, dtype, rows, cols, q, scales, (hipStream_t)stream);
}

int moe_route_topk_e4m3(const uint8_t* xq, const float* x_scale, const uint8_t* wq,
                        const float* w_scale, const float* bias, int64_t T, int d, int E, int k,
                        int flags, float* logits, int32_t* topk_idx, float* topk_gate,
                        void* stream) {
    if (T < 0 || E < 1 || E > MOE_MAX_E || k < 1 || k > MOE_MAX_K || k > E) return MOE_ERR_ARG;
    if (flags & ~MOE_RENORM) return MOE_ERR_ARG;
    if (T > (int64_t)0x7fffffff * 16) return MOE_ERR_ARG;
    if (d < 64 || d % 64) return MOE_ERR_SHAPE;
    if (!wq || !w_scale) return MOE_ERR_ARG;
    if (T > 0 && (!xq || !x_scale || !logits || !topk_idx || !topk_gate)) return MOE_ERR_ARG;
    if (!aligned16(wq) || (xq && !aligned16(xq))) return MOE_ERR_ARG;
    return launch_route_topk_e4m3(xq, x_scale, wq, w_scale, bias, T, d, E, k, flags, logits,
                                  topk_idx, topk_gate, (hipStream_t)stream);
}

}  // extern "C"
