/*
 * Oracle for the MoE expert stage -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct CPU code for what the GPU path computes. Only the
 * tests, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product library never does. It shares no code, header or helper with the GPU
 * library.
 *
 * What it follows (Huang, Lin, Lee, "Efficient CPU-GPU Collaborative Inference
 * for MoE-based LLMs on Memory-Limited Systems"):
 *   - Section I (MoE layer): a router picks experts for the input, the layer output
 *     is the gate-weighted sum of the chosen experts' outputs. The router formula
 *     is not printed; the reading used is softmax over all expert logits, top-k
 *     selection with ties to the lower expert id, then renormalisation of the k
 *     selected probabilities.
 *   - Table II: top-2 routing; 340 MB / 152 MB per expert, i.e. three d x f
 *     matrices of 2-byte weights, read as a SwiGLU expert
 *     y = W2 (SiLU(W1 x) * (W3 x)).
 *   - Section III-A: hits and misses compute the same expert function; the cache
 *     changes where an expert runs, not what it computes, so this oracle has no
 *     notion of host or device.
 *
 * Precision: inputs are fp32 (bf16 weights widen exactly to fp32). Every dot
 * product and sum is accumulated in double and rounded to float at each named
 * intermediate (g, u, h, y_e, out). Router logits stay in double for selection
 * and for the gate weights, which are rounded to float once.
 *
 * OpenMP only splits independent output rows across threads; each row's sum is a
 * single sequential loop, so results do not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int oracle_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Router logits l_i = sum_j W_r[i, j] x_j, W_r row-major [n, d]. */
void oracle_router_logits(const float *x, const float *wr, int d, int n, double *logits)
{
    for (int i = 0; i < n; i++) {
        double acc = 0.0;
        for (int j = 0; j < d; j++)
            acc += (double)wr[(size_t)i * d + j] * (double)x[j];
        logits[i] = acc;
    }
}

/* Softmax over all n logits (shifted by the maximum). */
static void softmax_all(const double *l, int n, double *p)
{
    double m = l[0];
    for (int i = 1; i < n; i++)
        if (l[i] > m) m = l[i];
    double z = 0.0;
    for (int i = 0; i < n; i++) {
        p[i] = exp(l[i] - m);
        z += p[i];
    }
    for (int i = 0; i < n; i++) p[i] /= z;
}

/* Order a chosen set by (logit descending, expert id ascending) and derive the
 * renormalised gate weights w_j = p_{S_j} / sum_{i in S} p_i. */
static void order_and_weigh(const double *l, const double *p, int k, const int32_t *set,
                            int32_t *idx, float *w)
{
    int32_t s[256];
    for (int r = 0; r < k; r++) s[r] = set[r];
    /* selection sort by the ordering key */
    for (int a = 0; a < k; a++) {
        int best = a;
        for (int b = a + 1; b < k; b++) {
            if (l[s[b]] > l[s[best]] || (l[s[b]] == l[s[best]] && s[b] < s[best])) best = b;
        }
        int32_t t = s[a]; s[a] = s[best]; s[best] = t;
    }
    double denom = 0.0;
    for (int r = 0; r < k; r++) denom += p[s[r]];
    for (int r = 0; r < k; r++) {
        idx[r] = s[r];
        w[r] = (float)(p[s[r]] / denom);
    }
}

/*
 * Router gating (Section I MoE layer; Table II top-K).
 *   l = W_r x; p = softmax(l); S = the k largest logits, ties to the lower id;
 *   idx ordered by (l desc, id asc); w = p_S / sum(p_S).
 * gap_out (nullable) receives l_(k) - l_(k+1), the margin between the last chosen
 * and the best unchosen logit (+inf when k == n). logits_out (nullable, [n]).
 * Requires 1 <= k <= n <= 256. Returns 0, or -1 on bad sizes.
 */
int oracle_router(const float *x, const float *wr, int d, int n, int k,
                  int32_t *idx, float *w, double *logits_out, double *gap_out)
{
    if (n < 1 || n > 256 || k < 1 || k > n || d < 1) return -1;
    double l[256], p[256];
    int chosen[256];
    int32_t set[256];
    oracle_router_logits(x, wr, d, n, l);
    softmax_all(l, n, p);
    for (int i = 0; i < n; i++) chosen[i] = 0;
    for (int r = 0; r < k; r++) {
        int best = -1;
        for (int i = 0; i < n; i++) {
            if (chosen[i]) continue;
            if (best < 0 || l[i] > l[best]) best = i;   /* strict: lower id wins ties */
        }
        chosen[best] = 1;
        set[r] = best;
    }
    order_and_weigh(l, p, k, set, idx, w);
    if (gap_out) {
        double best_out = -INFINITY;
        int any = 0;
        for (int i = 0; i < n; i++)
            if (!chosen[i] && (!any || l[i] > best_out)) { best_out = l[i]; any = 1; }
        *gap_out = any ? l[idx[k - 1]] - best_out : INFINITY;
    }
    if (logits_out)
        for (int i = 0; i < n; i++) logits_out[i] = l[i];
    return 0;
}

/* Same gate weights for a caller-given expert set (used when several sets are
 * correct because of a near-tie: the values are then checked for the set the
 * other side chose). Returns -1 if the set has duplicates or ids out of range. */
int oracle_router_forced(const float *x, const float *wr, int d, int n, int k,
                         const int32_t *set, int32_t *idx, float *w)
{
    if (n < 1 || n > 256 || k < 1 || k > n || d < 1) return -1;
    double l[256], p[256];
    for (int a = 0; a < k; a++) {
        if (set[a] < 0 || set[a] >= n) return -1;
        for (int b = 0; b < a; b++)
            if (set[a] == set[b]) return -1;
    }
    oracle_router_logits(x, wr, d, n, l);
    softmax_all(l, n, p);
    order_and_weigh(l, p, k, set, idx, w);
    return 0;
}

/*
 * One SwiGLU expert (Table II size reading):
 *   g = W1 x, u = W3 x (rows of length d), h_i = SiLU(g_i) u_i = g_i / (1 + e^{-g_i}) u_i,
 *   y = W2 h (rows of length f).
 * slab: bf16 bit patterns, W1 [f, d] | W3 [f, d] | W2 [d, f], row-major.
 */
void oracle_expert(const float *x, const uint16_t *slab, int d, int f, float *y)
{
    const uint16_t *w1 = slab;
    const uint16_t *w3 = slab + (size_t)f * d;
    const uint16_t *w2 = slab + (size_t)2 * f * d;
    float *h = (float *)malloc(sizeof(float) * (size_t)f);
    if (!h) return;
#pragma omp parallel for schedule(static)
    for (int i = 0; i < f; i++) {
        double g = 0.0, u = 0.0;
        const uint16_t *r1 = w1 + (size_t)i * d;
        const uint16_t *r3 = w3 + (size_t)i * d;
        for (int j = 0; j < d; j++) {
            g += widen_bf16(r1[j]) * (double)x[j];
            u += widen_bf16(r3[j]) * (double)x[j];
        }
        float gf = (float)g, uf = (float)u;
        double silu = (double)gf / (1.0 + exp(-(double)gf));
        h[i] = (float)(silu * (double)uf);
    }
#pragma omp parallel for schedule(static)
    for (int i = 0; i < d; i++) {
        double acc = 0.0;
        const uint16_t *r2 = w2 + (size_t)i * f;
        for (int c = 0; c < f; c++) acc += widen_bf16(r2[c]) * (double)h[c];
        y[i] = (float)acc;
    }
    free(h);
}

/*
 * Weighted combine: out = sum_j w_j y_j (+ y_shared with weight 1 when given).
 * ys: [k][d] expert outputs in the order of w.
 */
void oracle_combine(const float *ys, const float *w, int k, int d, const float *y_shared, float *out)
{
    for (int i = 0; i < d; i++) {
        double acc = 0.0;
        for (int j = 0; j < k; j++) acc += (double)w[j] * (double)ys[(size_t)j * d + i];
        if (y_shared) acc += (double)y_shared[i];
        out[i] = (float)acc;
    }
}

/*
 * One token through one MoE layer: router, the chosen experts, combine.
 * slabs: n pointers (expert e's slab). shared_slab may be NULL (f_shared ignored).
 * forced_set (nullable, [k]): evaluate this expert set instead of the router's.
 * Outputs idx[k], w[k], out[d]; gap_out as in oracle_router (nullable).
 */
int oracle_moe_token(const float *x, const float *wr, const uint16_t *const *slabs,
                     const uint16_t *shared_slab, int d, int f, int f_shared, int n, int k,
                     const int32_t *forced_set, int32_t *idx, float *w, float *out,
                     double *gap_out)
{
    int rc = forced_set ? oracle_router_forced(x, wr, d, n, k, forced_set, idx, w)
                        : oracle_router(x, wr, d, n, k, idx, w, NULL, gap_out);
    if (rc) return rc;
    float *ys = (float *)malloc(sizeof(float) * (size_t)k * d);
    float *ysh = NULL;
    if (!ys) return -2;
    for (int j = 0; j < k; j++) oracle_expert(x, slabs[idx[j]], d, f, ys + (size_t)j * d);
    if (shared_slab && f_shared > 0) {
        ysh = (float *)malloc(sizeof(float) * (size_t)d);
        if (!ysh) { free(ys); return -2; }
        oracle_expert(x, shared_slab, d, f_shared, ysh);
    }
    oracle_combine(ys, w, k, d, ysh, out);
    free(ys);
    free(ysh);
    return 0;
}
