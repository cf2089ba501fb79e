/* Host sanitizer driver of the CPU oracle (test infrastructure): every step of
 * the layer share on small seeded inputs and on its edge cases (no tokens,
 * one token, k = E, ties, replicas over three GPUs, an expert with no host,
 * rows exactly at capacity), built with AddressSanitizer and
 * UndefinedBehaviorSanitizer so that any out-of-bounds access, use of freed
 * memory or undefined arithmetic in the oracle ends the run with an error.
 * Prints "oracle sanitizer run: OK" when every check passes. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void orc_router_logits(const float* X, const float* Wr, const float* bias, int64_t T, int64_t d,
                       int64_t E, double* out);
int orc_topk(const float* logits, int64_t T, int E, int k, int renorm, int32_t* idx,
             double* gate);
void orc_histogram(const int32_t* idx, int64_t T, int k, int E, int64_t* counts, int64_t* coact);
int64_t orc_permute(const float* X, int64_t T, int64_t d, const int32_t* idx, const double* gate,
                    int k, int E, const uint8_t* placement, int G, int dev, int64_t cap_rows,
                    float* x_perm, int64_t* group_offsets, int64_t* row_token, double* row_gate,
                    int64_t* token_row, int64_t* send_counts);
void orc_expert_ffn(const float* x, int64_t n, int64_t d, int64_t f, const float* W13,
                    const float* W2, double* y);
void orc_combine(const double* y_perm, const int64_t* token_row, const double* gate,
                 const double* y_shared, int64_t T, int64_t d, int k, double* y);

static uint64_t rng = 88172645463325252ull;
static double urand(void) {
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0;
}

#define CHECK(c) do { if (!(c)) { fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); return 1; } } while (0)

/* One whole share: logits, top-k, histogram, permute on every GPU, FFN of each
 * local group, combine.  Returns 0 when the partition invariants hold. */
static int share(int64_t T, int d, int E, int k, int f, int G, int ties, int replicas) {
    float* X = malloc(sizeof(float) * (size_t)(T ? T : 1) * d);
    float* Wr = malloc(sizeof(float) * (size_t)E * d);
    float* b = malloc(sizeof(float) * (size_t)E);
    for (int64_t i = 0; i < T * d; ++i) X[i] = (float)(urand() * 2 - 1);
    for (int64_t i = 0; i < (int64_t)E * d; ++i) Wr[i] = ties ? 0.f : (float)(urand() * 0.1 - 0.05);
    for (int e = 0; e < E; ++e) b[e] = ties ? (float)(e % 2) : 0.f;
    double* L = malloc(sizeof(double) * (size_t)(T ? T : 1) * E);
    float* L32 = malloc(sizeof(float) * (size_t)(T ? T : 1) * E);
    orc_router_logits(X, Wr, b, T, d, E, L);
    for (int64_t i = 0; i < T * E; ++i) L32[i] = (float)L[i];
    int32_t* idx = malloc(sizeof(int32_t) * (size_t)(T ? T : 1) * k);
    double* gate = malloc(sizeof(double) * (size_t)(T ? T : 1) * k);
    CHECK(orc_topk(L32, T, E, k, 1, idx, gate) == 0);
    CHECK(orc_topk(L32, T, E, E + 1, 1, idx, gate) == -1);
    int64_t* counts = malloc(sizeof(int64_t) * (size_t)E);
    int64_t* coact = malloc(sizeof(int64_t) * (size_t)E * E);
    orc_histogram(idx, T, k, E, counts, coact);
    int64_t total = 0;
    for (int e = 0; e < E; ++e) total += counts[e];
    CHECK(total == T * k);
    uint8_t* pl = calloc((size_t)E * G, 1);
    for (int e = 0; e < E; ++e) pl[e * G + e % G] = 1;
    for (int e = 0; e < replicas && e < E; ++e)
        for (int j = 0; j < G; ++j) pl[e * G + j] = 1;
    int64_t kept = 0;
    for (int dev = 0; dev < G; ++dev) {
        int n_local = 0;
        for (int e = 0; e < E; ++e) n_local += pl[e * G + dev];
        int64_t cap = T * (k < n_local ? k : n_local);
        float* xp = malloc(sizeof(float) * (size_t)(cap ? cap : 1) * d);
        int64_t* go = malloc(sizeof(int64_t) * (size_t)(n_local + 1));
        int64_t* rt = malloc(sizeof(int64_t) * (size_t)(cap ? cap : 1));
        double* rg = malloc(sizeof(double) * (size_t)(cap ? cap : 1));
        int64_t* tr = malloc(sizeof(int64_t) * (size_t)(T ? T : 1) * k);
        int64_t* sc = malloc(sizeof(int64_t) * (size_t)G);
        int64_t rows = orc_permute(X, T, d, idx, gate, k, E, pl, G, dev, cap, xp, go, rt, rg, tr, sc);
        CHECK(rows >= 0 && rows <= cap && go[n_local] == rows && sc[dev] == rows);
        kept += rows;
        /* FFN of every local group and the combine */
        float* W13 = malloc(sizeof(float) * (size_t)2 * f * d);
        float* W2 = malloc(sizeof(float) * (size_t)d * f);
        for (int64_t i = 0; i < 2LL * f * d; ++i) W13[i] = (float)(urand() * 0.1 - 0.05);
        for (int64_t i = 0; i < (int64_t)d * f; ++i) W2[i] = (float)(urand() * 0.1 - 0.05);
        double* yp = malloc(sizeof(double) * (size_t)(rows ? rows : 1) * d);
        for (int s = 0; s < n_local; ++s)
            orc_expert_ffn(xp + go[s] * d, go[s + 1] - go[s], d, f, W13, W2, yp + go[s] * d);
        double* y = malloc(sizeof(double) * (size_t)(T ? T : 1) * d);
        orc_combine(yp, tr, gate, NULL, T, d, k, y);
        free(xp); free(go); free(rt); free(rg); free(tr); free(sc); free(W13); free(W2);
        free(yp); free(y);
    }
    CHECK(kept == T * k);
    /* an expert with no host is refused */
    memset(pl, 0, (size_t)E * G);
    {
        int64_t go[2], sc[8];
        CHECK(orc_permute(NULL, T, 0, idx, gate, k, E, pl, G, 0, 0, NULL, go, NULL, NULL, NULL, sc) < 0);
    }
    free(X); free(Wr); free(b); free(L); free(L32); free(idx); free(gate); free(counts);
    free(coact); free(pl);
    return 0;
}

int main(void) {
    int rc = 0;
    rc |= share(0, 16, 8, 2, 8, 2, 0, 0);        /* no tokens */
    rc |= share(1, 16, 8, 2, 8, 2, 0, 1);        /* one token */
    rc |= share(37, 24, 6, 6, 16, 3, 0, 2);      /* k = E, replicas on every GPU */
    rc |= share(64, 32, 8, 3, 16, 1, 1, 0);      /* all-equal scores: ties everywhere */
    rc |= share(130, 40, 20, 4, 24, 3, 0, 3);    /* ragged sizes, three GPUs */
    if (rc) return 1;
    printf("oracle sanitizer run: OK\n");
    return 0;
}
