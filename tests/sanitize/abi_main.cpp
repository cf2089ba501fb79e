// Host sanitizer driver of the C ABI's argument validation (test
// infrastructure): every entry point is called with argument combinations its
// validation must refuse -- null pointers, negative or oversized sizes, bad
// dtypes, flags and placements, misaligned pointers, short workspaces -- and
// the workspace-size functions over a range of shapes including the extremes.
// None of these calls reaches a HIP API call, so the run needs no GPU.  Built
// with AddressSanitizer and UndefinedBehaviorSanitizer on the host code of the
// whole library; prints "abi sanitizer run: OK" when every status is the
// expected one.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "moe.h"

static int failures = 0;
#define EXPECT(call, want)                                                             \
    do {                                                                               \
        const int got_ = (call);                                                       \
        if (got_ != (want)) {                                                          \
            fprintf(stderr, "line %d: %s -> %d, expected %d\n", __LINE__, #call, got_, \
                    (int)(want));                                                      \
            ++failures;                                                                \
        }                                                                              \
    } while (0)

int main() {
    void* F = (void*)0x1000;                 // never dereferenced: every call fails validation
    void* W = (void*)0x100000;               // 256-byte aligned stand-in workspace
    const void* wp[2] = {(void*)0x1000, (void*)0x2000};
    const void* wnull[2] = {(void*)0x1000, nullptr};

    // moe_route_topk
    EXPECT(moe_route_topk(F, 1, F, nullptr, 4, 64, 8, 0, 1, (float*)F, (int32_t*)F, (float*)F,
                          nullptr, 0, nullptr), MOE_ERR_ARG);
    EXPECT(moe_route_topk(F, 1, F, nullptr, 4, 64, 300, 2, 1, (float*)F, (int32_t*)F, (float*)F,
                          nullptr, 0, nullptr), MOE_ERR_ARG);
    EXPECT(moe_route_topk(F, 7, F, nullptr, 4, 64, 8, 2, 1, (float*)F, (int32_t*)F, (float*)F,
                          nullptr, 0, nullptr), MOE_ERR_ARG);
    EXPECT(moe_route_topk(F, 1, F, nullptr, 4, 12, 8, 2, 1, (float*)F, (int32_t*)F, (float*)F,
                          nullptr, 0, nullptr), MOE_ERR_SHAPE);
    EXPECT(moe_route_topk(F, 1, F, nullptr, 4, 4194304, 256, 2, 1, (float*)F, (int32_t*)F,
                          (float*)F, nullptr, 0, nullptr), MOE_ERR_SHAPE);
    EXPECT(moe_route_topk(nullptr, 1, F, nullptr, 4, 64, 8, 2, 3, nullptr, (int32_t*)F,
                          (float*)F, nullptr, 0, nullptr), MOE_ERR_ARG);
    EXPECT(moe_route_topk(F, 1, F, nullptr, -1, 64, 8, 2, 1, (float*)F, (int32_t*)F, (float*)F,
                          nullptr, 0, nullptr), MOE_ERR_ARG);
    // moe_expert_histogram
    EXPECT(moe_expert_histogram((int32_t*)F, 4, 0, 8, (int32_t*)F, nullptr, nullptr), MOE_ERR_ARG);
    EXPECT(moe_expert_histogram(nullptr, 4, 2, 8, (int32_t*)F, nullptr, nullptr), MOE_ERR_ARG);
    // moe_permute and moe_permute_noalloc
    uint8_t pl[4 * 2] = {1, 0, 0, 1, 1, 1, 0, 0};         // expert 3 has no host
    EXPECT(moe_permute(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 10, 64, 2, 4, pl, 2, 0, 0, F,
                       20, (int32_t*)F, (int32_t*)F, (float*)F, (int32_t*)F, nullptr, W, 1 << 20,
                       nullptr), MOE_ERR_PLACEMENT);
    pl[7] = 1;
    EXPECT(moe_permute(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 10, 64, 2, 4, pl, 2, 2, 0, F,
                       20, (int32_t*)F, (int32_t*)F, (float*)F, (int32_t*)F, nullptr, W, 1 << 20,
                       nullptr), MOE_ERR_PLACEMENT);
    EXPECT(moe_permute(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 10, 64, 2, 4, pl, 2, 0, 0, F,
                       19, (int32_t*)F, (int32_t*)F, (float*)F, (int32_t*)F, nullptr, W, 1 << 20,
                       nullptr), MOE_ERR_SHAPE);
    EXPECT(moe_permute(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 10, 64, 2, 4, pl, 2, 0, 0, F,
                       20, (int32_t*)F, (int32_t*)F, (float*)F, (int32_t*)F, nullptr, W, 16,
                       nullptr), MOE_ERR_SHAPE);
    std::vector<uint8_t> big(128 * 1, 1);
    EXPECT(moe_permute_noalloc(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 600000, 64, 8, 128,
                               big.data(), 1, 0, 0, F, 600000LL * 8, (int32_t*)F, (int32_t*)F,
                               (float*)F, (int32_t*)F, nullptr, nullptr), MOE_ERR_SHAPE);
    EXPECT(moe_permute_noalloc(F, 1, (int32_t*)F, (float*)F, (int32_t*)F, 10, 12, 2, 4, pl, 2, 0,
                               0, F, 20, (int32_t*)F, (int32_t*)F, (float*)F, (int32_t*)F,
                               nullptr, nullptr), MOE_ERR_SHAPE);
    // moe_grouped_ffn and its variants
    EXPECT(moe_grouped_ffn(F, 1, (int32_t*)F, 0, wp, wp, 128, 64, 16, F, W, 1 << 30, nullptr),
           MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn(F, 1, (int32_t*)F, 2, wp, wp, 100, 64, 16, F, W, 1 << 30, nullptr),
           MOE_ERR_SHAPE);
    EXPECT(moe_grouped_ffn(F, 1, (int32_t*)F, 2, wnull, wp, 128, 64, 16, F, W, 1 << 30, nullptr),
           MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn(F, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16, F, W, 10, nullptr),
           MOE_ERR_SHAPE);
    EXPECT(moe_grouped_ffn_products(F, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16, F, W, 1 << 30, 4,
                                    nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_products(nullptr, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16, F, W,
                                    1 << 30, 1, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_combine(F, 0, (int32_t*)F, 2, wp, wp, 128, 64, 16, (int32_t*)F,
                                   (float*)F, nullptr, 8, 2, F, W, 1 << 30, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_combine(F, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16, (int32_t*)F,
                                   (float*)F, nullptr, 8, 17, F, W, 1 << 30, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows(F, 64, nullptr, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16, F, W,
                                1 << 30, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows(F, 20000000, (int32_t*)F, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16,
                                F, W, 1 << 30, nullptr), MOE_ERR_SHAPE);
    EXPECT(moe_grouped_ffn_rows_products(F, 64, (int32_t*)F, 1, (int32_t*)F, 2, wp, wp, 128, 64,
                                         16, F, W, 1 << 30, 3 | 4 | 8, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows_products(F, 64, nullptr, 1, (int32_t*)F, 2, wp, wp, 128, 64, 16,
                                         F, W, 1 << 30, 1, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows_shared(F, 64, (int32_t*)F, 1, (int32_t*)F, 2, -1, wp, wp, 128,
                                       64, 16, F, W, 1 << 30, 3, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows_shared(F, 0, (int32_t*)F, 1, (int32_t*)F, 0, 1, wp, wp, 128, 64,
                                       16, F, W, 1 << 30, 3, nullptr), MOE_ERR_ARG);
    EXPECT(moe_grouped_ffn_rows_shared(F, 1 << 20, (int32_t*)F, 1, (int32_t*)F, 0, 2, wp, wp, 128,
                                       64, (1LL << 31) - (1 << 20), F, W, 1 << 30, 3, nullptr),
           MOE_ERR_ARG);
    // moe_combine
    EXPECT(moe_combine(nullptr, 1, (int32_t*)F, (float*)F, nullptr, 4, 64, 2, F, nullptr),
           MOE_ERR_ARG);
    EXPECT(moe_combine(F, 1, (int32_t*)F, (float*)F, nullptr, 4, 64, 0, F, nullptr), MOE_ERR_ARG);
    EXPECT(moe_combine_shared(F, 1, (int32_t*)F, (float*)F, F, -1, 4, 64, 2, F, nullptr),
           MOE_ERR_ARG);
    EXPECT(moe_combine_shared(F, 1, (int32_t*)F, (float*)F, F, MOE_MAX_GROUPS + 1, 4, 64, 2, F,
                              nullptr), MOE_ERR_ARG);
    // quantized predictor
    EXPECT(moe_quantize_e4m3(F, 2, 4, 64, (uint8_t*)F, (float*)F, nullptr), MOE_ERR_ARG);
    EXPECT(moe_route_topk_e4m3((uint8_t*)F, (float*)F, (uint8_t*)F, (float*)F, nullptr, 4, 96, 8,
                               2, 1, (float*)F, (int32_t*)F, (float*)F, nullptr), MOE_ERR_SHAPE);
    // workspace sizes over a range of shapes, the extremes included
    const int64_t Ts[] = {0, 1, 63, 64, 65, 1023, 1024, 1025, 4096, 16384, 100000, 524000};
    const int Es[] = {1, 8, 60, 64, 128, 256};
    size_t acc = 0;
    for (int64_t T : Ts)
        for (int E : Es) {
            for (int dtype = 0; dtype < 2; ++dtype) {
                acc += moe_route_topk_ws_bytes(dtype, T, 2048, E, 1);
                acc += moe_route_topk_ws_bytes(dtype, T, 4096, E, 3);
            }
            acc += moe_permute_ws_bytes(T, 8, E);
            acc += moe_grouped_ffn_ws_bytes(1, T * 8, 4096, 14336, E < 128 ? E : 128);
            acc += moe_grouped_ffn_ws_bytes(0, T, 128, 256, 8);
        }
    EXPECT(moe_permute_ws_bytes(-1, 8, 8) == 0, 1);
    EXPECT(moe_grouped_ffn_ws_bytes(1, -5, 128, 64, 2) == 0, 1);
    for (int code = -2; code < 8; ++code) acc += moe_status_string(code)[0];
    if (failures) return 1;
    printf("abi sanitizer run: OK (%zu)\n", acc);
    return 0;
}
