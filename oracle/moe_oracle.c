/*
 * moe_oracle.c -- TEST INFRASTRUCTURE, not part of the product.
 *
 * A plain, slow, obviously correct CPU oracle of one GPU's share of one
 * expert-parallel MoE layer, as used by Director (arXiv 2607.08782):
 *   gate scores -> top-k -> per-expert workload counts -> packaging of the
 *   tokens for the locally placed experts -> expert FFN -> gate-weighted sum.
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  It shares no code, header, table or helper with the
 * HIP library; neither side includes or links the other.
 *
 * Arithmetic: every floating-point value is accumulated in double.  Inputs
 * arrive as float arrays (bf16 inputs are passed as their exact float
 * upcasts).  Sums run over the index in ascending order, with no blocking,
 * no reordering and no fusion.  OpenMP only splits independent outputs
 * (tokens or rows) across threads, which cannot change any result.
 *
 * Parity status: every function is pinned by the CPU test-suite
 * (library routines, closed forms, brute force on tiny inputs, invariants).
 * The replica split rule in orc_permute is a convention the paper leaves open
 * (the floor rule read here); it is pinned by its partition invariants and by
 * a hand-worked example of that rule (tests/golden/replica_split_hand_example.json).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------------------
 * Gate scores (Sec. II-A: the gating network scores every expert for every
 * token; the gate is replicated on each GPU in expert parallelism, Sec. II-B).
 * The gating network is a linear layer with bias:
 *     logits[t][e] = sum_{i=0}^{d-1} X[t][i] * Wr[e][i] + bias[e]
 * X is [T][d] row-major, Wr is [E][d] row-major, bias is [E] (nullable = 0).
 * ------------------------------------------------------------------------- */
void orc_router_logits(const float* X, const float* Wr, const float* bias,
                       int64_t T, int64_t d, int64_t E, double* logits)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t e = 0; e < E; ++e) {
            double acc = 0.0;
            for (int64_t i = 0; i < d; ++i)
                acc += (double)X[t * d + i] * (double)Wr[e * d + i];
            if (bias) acc += (double)bias[e];
            logits[t * E + e] = acc;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Top-k selection and gate values (Sec. II-A: top-k routing on the relevance
 * scores; the outputs are later weighted by the gate scores).
 *
 * Selection works on the fp32 logits given (the precision the GPU decides in).
 * Repeat k times: among the experts not yet chosen, take the e with the
 * largest logit; on equal logits the lower expert index wins.  Comparison is
 * IEEE float comparison, so -0.0 equals +0.0.  idx[t][r] is the r-th choice,
 * i.e. descending logit, then ascending index.
 *
 * Gates, in double:
 *   renorm != 0: softmax over the k selected logits,
 *                g_r = exp(l_r - m) / sum_{r'} exp(l_{r'} - m), m = l[idx_0]
 *   renorm == 0: softmax over all E logits, restricted to the selected ones.
 * Returns 0, or -1 if k is not in [1, E] or E > 4096.
 * ------------------------------------------------------------------------- */
int orc_topk(const float* logits, int64_t T, int E, int k, int renorm,
             int32_t* idx, double* gate)
{
    if (k < 1 || k > E || E > 4096) return -1;
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const float* l = logits + t * E;
        char taken[4096];
        memset(taken, 0, (size_t)E);
        for (int r = 0; r < k; ++r) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || l[e] > l[best]) best = e;  /* strict: ties keep the lower index */
            }
            taken[best] = 1;
            idx[t * k + r] = best;
        }
        double m = (double)l[idx[t * k]];
        double denom = 0.0;
        if (renorm) {
            for (int r = 0; r < k; ++r) denom += exp((double)l[idx[t * k + r]] - m);
        } else {
            for (int e = 0; e < E; ++e) denom += exp((double)l[e] - m);
        }
        for (int r = 0; r < k; ++r)
            gate[t * k + r] = exp((double)l[idx[t * k + r]] - m) / denom;
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Workload counts (Sec. VI-A, "Request Workload": W_{j,i} counts the tokens
 * routed to expert i; this share routes all T tokens, so counts[e] is the
 * inner sum of Eq. (1)).  Co-activation counts (the signal for co-locating
 * experts that are activated together, Sec. I):
 *   counts[e]   = #{(t, r) : idx[t][r] = e}
 *   coact[a][b] = #{t : a in S_t and b in S_t}, S_t = {idx[t][0..k-1]}
 * coact is [E][E] row-major and nullable.
 * ------------------------------------------------------------------------- */
void orc_histogram(const int32_t* idx, int64_t T, int k, int E,
                   int64_t* counts, int64_t* coact)
{
    for (int e = 0; e < E; ++e) counts[e] = 0;
    if (coact) for (int64_t i = 0; i < (int64_t)E * E; ++i) coact[i] = 0;
    for (int64_t t = 0; t < T; ++t) {
        for (int r = 0; r < k; ++r) {
            int a = idx[t * k + r];
            counts[a] += 1;
            if (coact)
                for (int q = 0; q < k; ++q)
                    coact[(int64_t)a * E + idx[t * k + q]] += 1;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Packaging of tokens for the experts placed on GPU `dev` (Sec. II-B: tokens
 * are packaged and sent to the GPUs hosting their experts; Sec. VI-A:
 * placement x[e][j] in {0,1}, every expert hosted at least once, Eq. (6d);
 * the volume sent to GPU j is Eq. (3) divided by the per-token size d).
 *
 * placement is [E][G] row-major, x[e][j] = placement[e*G + j].
 * Local slot s = the s-th expert, by ascending id, with x[e][dev] = 1.
 *
 * The paper lets an expert have several hosts (Eq. 6d) but does not say how
 * its tokens are split among them.  Reading used here: let A_e be the tokens
 * that chose e, in ascending token order, c_e = |A_e|, n_e = sum_j x[e][j];
 * the q-th host of e (hosts counted by ascending GPU id) serves the ranks
 * [floor(q*c_e/n_e), floor((q+1)*c_e/n_e)) of A_e.
 *
 * Outputs (all caller-allocated):
 *   group_offsets[n_local+1]  exclusive prefix sum of the rows kept per slot
 *   row_token[rows], row_gate[rows], x_perm[rows][d] (x_perm nullable)
 *   token_row[T*k]            row of assignment (t, r) on this GPU, or -1
 *   send_counts[G]            rows each GPU's hosts take (Eq. (3) / d);
 *                             with no replicas this is lambda_j of Eq. (1)
 * Returns the number of local rows, or
 *   -1 bad argument, -2 an expert with no host, -3 rows exceed cap_rows.
 * ------------------------------------------------------------------------- */
int64_t orc_permute(const float* X, int64_t T, int64_t d,
                    const int32_t* idx, const double* gate, int k, int E,
                    const uint8_t* placement, int G, int dev,
                    int64_t cap_rows, float* x_perm,
                    int64_t* group_offsets, int64_t* row_token, double* row_gate,
                    int64_t* token_row, int64_t* send_counts)
{
    if (T < 0 || d < 0 || k < 1 || E < 1 || G < 1 || dev < 0 || dev >= G) return -1;

    int64_t* count = (int64_t*)calloc((size_t)E, sizeof(int64_t));
    int64_t* lo = (int64_t*)calloc((size_t)E, sizeof(int64_t));
    int64_t* hi = (int64_t*)calloc((size_t)E, sizeof(int64_t));
    int* slot = (int*)malloc((size_t)E * sizeof(int));
    int64_t* seen = (int64_t*)calloc((size_t)E, sizeof(int64_t));
    if (!count || !lo || !hi || !slot || !seen) { free(count); free(lo); free(hi); free(slot); free(seen); return -1; }

    for (int64_t t = 0; t < T; ++t)
        for (int r = 0; r < k; ++r) count[idx[t * k + r]] += 1;

    for (int j = 0; j < G; ++j) send_counts[j] = 0;
    int n_local = 0;
    int64_t bad = 0;
    for (int e = 0; e < E; ++e) {
        int n_e = 0;
        for (int j = 0; j < G; ++j) n_e += placement[(int64_t)e * G + j] ? 1 : 0;
        if (n_e == 0) { bad = -2; break; }
        int q = 0;
        for (int j = 0; j < G; ++j) {
            if (!placement[(int64_t)e * G + j]) continue;
            int64_t a = (int64_t)q * count[e] / n_e;
            int64_t b = (int64_t)(q + 1) * count[e] / n_e;
            send_counts[j] += b - a;
            if (j == dev) { lo[e] = a; hi[e] = b; }
            ++q;
        }
        slot[e] = placement[(int64_t)e * G + dev] ? n_local++ : -1;
    }
    if (bad) { free(count); free(lo); free(hi); free(slot); free(seen); return bad; }

    group_offsets[0] = 0;
    for (int e = 0, s = 0; e < E; ++e)
        if (slot[e] >= 0) { group_offsets[s + 1] = group_offsets[s] + (hi[e] - lo[e]); ++s; }
    int64_t rows = group_offsets[n_local];
    if (rows > cap_rows) { free(count); free(lo); free(hi); free(slot); free(seen); return -3; }

    for (int64_t t = 0; t < T; ++t) {
        for (int r = 0; r < k; ++r) {
            int e = idx[t * k + r];
            int64_t rho = seen[e]++;          /* rank of t in A_e */
            int64_t p = -1;
            if (slot[e] >= 0 && rho >= lo[e] && rho < hi[e]) {
                p = group_offsets[slot[e]] + (rho - lo[e]);
                row_token[p] = t;
                row_gate[p] = gate[t * k + r];
                if (x_perm) memcpy(x_perm + p * d, X + t * d, (size_t)d * sizeof(float));
            }
            token_row[t * k + r] = p;
        }
    }
    free(count); free(lo); free(hi); free(slot); free(seen);
    return rows;
}

/* ---------------------------------------------------------------------------
 * One expert FFN on n rows (Sec. II-A: each expert is an FFN sub-network).
 * The expert form is SwiGLU:
 *     a = W1 x,  b = W3 x,  h_j = SiLU(a_j) * b_j,  SiLU(a) = a / (1 + e^{-a}),
 *     y = W2 h.
 * W13 is [2f][d] row-major: rows 0..f-1 are W1 (gate), rows f..2f-1 are W3
 * (up).  W2 is [d][f] row-major.  x is [n][d], y is [n][d].
 * ------------------------------------------------------------------------- */
void orc_expert_ffn(const float* x, int64_t n, int64_t d, int64_t f,
                    const float* W13, const float* W2, double* y)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n; ++p) {
        double* h = (double*)malloc((size_t)(f > 0 ? f : 1) * sizeof(double));
        const float* xp = x + p * d;
        for (int64_t j = 0; j < f; ++j) {
            double a = 0.0, b = 0.0;
            for (int64_t i = 0; i < d; ++i) {
                a += (double)W13[j * d + i] * (double)xp[i];
                b += (double)W13[(f + j) * d + i] * (double)xp[i];
            }
            h[j] = a / (1.0 + exp(-a)) * b;
        }
        for (int64_t o = 0; o < d; ++o) {
            double acc = 0.0;
            for (int64_t j = 0; j < f; ++j) acc += (double)W2[o * f + j] * h[j];
            y[p * d + o] = acc;
        }
        free(h);
    }
}

/* ---------------------------------------------------------------------------
 * Gate-weighted sum (Sec. II-A: the selected experts' outputs are combined by
 * a weighted sum with the gate scores; Sec. II-B: the results return to the
 * token's GPU).  Shared (always-on) experts enter with weight 1:
 *     y[t] = sum_{r ascending, token_row[t][r] >= 0} gate[t][r] * y_perm[token_row[t][r]]
 *            + y_shared[t]
 * y_perm is [rows][d]; y_shared is [T][d] and nullable.
 * ------------------------------------------------------------------------- */
void orc_combine(const double* y_perm, const int64_t* token_row, const double* gate,
                 const double* y_shared, int64_t T, int64_t d, int k, double* y)
{
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int r = 0; r < k; ++r) {
                int64_t p = token_row[t * k + r];
                if (p >= 0) acc += gate[t * k + r] * y_perm[p * d + i];
            }
            if (y_shared) acc += y_shared[t * d + i];
            y[t * d + i] = acc;
        }
    }
}

/* Threads of the oracle's OpenMP loops from now on (the benchmark times it at
 * one thread as well as at all host threads). */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Number of OpenMP threads the oracle runs with (reported by the benchmark). */
int orc_num_threads(void)
{
    int n = 1;
    #pragma omp parallel
    {
        #pragma omp single
        {
#ifdef _OPENMP
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
