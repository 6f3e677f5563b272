/*
 * oracle/carith.c -- TEST INFRASTRUCTURE ONLY (the CPU oracle).
 *
 * The canonical single-precision arithmetic of the BASE scoring path, written
 * plainly: every operation is one IEEE-754 binary32 operation, rounded to
 * nearest-even, in the order stated here.  fmaf() is the single-rounding
 * fused multiply-add of C99; nothing else is fused (this file is built with
 * -ffp-contract=off).  The paper fixes no arithmetic order for its scores;
 * the order below is this implementation's reading of "scores computed in
 * fp32 in a fixed reduction order", and a HIP kernel that claims bit-exact
 * parity must compute exactly this sequence.
 *
 * Nothing here is shared with the HIP library: only tests, the smoke check
 * and the CPU-baseline leg of the benchmark load it.
 *
 * Contents (paper passages each follows):
 *   cexp        exp(x) for the predictor and the router softmax
 *               (Sec. 3.4, eq. log_energy_predictor; Sec. 3.1 router weights)
 *   cdot        fixed-order dot product
 *   route       router logits, top-K, normalised weights (Sec. 3.1; Sec. 3.5)
 *   predict     per routed pair cost w^2 exp(a_u.z_bar + b_u)   (Sec. 3.4)
 *   aggregate   batch score D_hat_u (Sec. 3.4; App. "Custom GPU Kernels")
 *   gates       router-score gates for executed experts (Sec. 3.5)
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define LANES 64          /* partial sums of a dot product */
#define GROUP 4           /* consecutive elements owned by one partial sum */
#define STRIDE (LANES * GROUP)

/* ---------------------------------------------------------------- cexp ---
 * Cody & Waite range reduction (W. J. Cody, W. Waite, "Software Manual for
 * the Elementary Functions", 1980) followed by the degree-7 Taylor polynomial
 * of e^r on |r| <= ln2/2, evaluated by Horner's rule with fused steps:
 *   x  <- min(max(x, -86), 88)           (results stay normal and finite)
 *   n  <- rint(x * log2(e))
 *   r  <- fma(-n, C1, x); r <- fma(-n, C2, r)    with C1 + C2 ~ ln 2,
 *         C1 = ln 2 with its low 9 significand bits cleared (n*C1 is exact)
 *   p  <- 1/7!;  p <- fma(p, r, 1/k!) for k = 6..0
 *   return p * 2^n
 * All constants are the binary32 values nearest to the stated reals.
 */
static const float CX_LOG2E = 1.44269504088896341f;   /* 0x3FB8AA3B */
static float cx_c1(void) { uint32_t u = 0x3F317200u; float f; memcpy(&f, &u, 4); return f; }
static float cx_c2(void) { uint32_t u = 0x35BFBE8Eu; float f; memcpy(&f, &u, 4); return f; }

float orc_cexp(float x)
{
    static const float inv_fact[8] = {
        1.0f, 1.0f, 0.5f, 0.166666666666666667f, 0.0416666666666666667f,
        0.00833333333333333333f, 0.00138888888888888889f,
        0.000198412698412698413f};
    const float c1 = cx_c1(), c2 = cx_c2();
    x = fminf(fmaxf(x, -86.0f), 88.0f);
    float t = x * CX_LOG2E;
    float n = rintf(t);
    float r = fmaf(-n, c1, x);
    r = fmaf(-n, c2, r);
    float p = inv_fact[7];
    for (int k = 6; k >= 0; --k)
        p = fmaf(p, r, inv_fact[k]);
    return ldexpf(p, (int)n);
}

void orc_cexp_array(const float *x, float *y, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) y[i] = orc_cexp(x[i]);
}

/* ---------------------------------------------------------------- cdot ---
 * dot(p, q) over d elements, d a multiple of 256.  Partial sum j (0..63)
 * owns elements 256m + 4j + r (r = 0..3) and accumulates them in ascending
 * element order with fmaf starting from +0.  The 64 partial sums are then
 * combined by a halving tree: for h = 32, 16, 8, 4, 2, 1 the sum j < h
 * becomes s[j] + s[j + h]; the result is s[0].
 */
float orc_cdot(const float *p, const float *q, int d)
{
    float s[LANES];
    for (int j = 0; j < LANES; ++j) {
        float acc = 0.0f;
        for (int m = 0; m * STRIDE < d; ++m)
            for (int r = 0; r < GROUP; ++r) {
                int k = m * STRIDE + j * GROUP + r;
                acc = fmaf(p[k], q[k], acc);
            }
        s[j] = acc;
    }
    for (int h = LANES / 2; h >= 1; h /= 2)
        for (int j = 0; j < h; ++j)
            s[j] = s[j] + s[j + h];
    return s[0];
}

/* all-pairs dots: out[i * nq + e] = cdot(P[i], Q[e]) */
void orc_cdot_matrix(const float *P, int np_, const float *Q, int nq, int d,
                     float *out)
{
    for (int i = 0; i < np_; ++i)
        for (int e = 0; e < nq; ++e)
            out[(int64_t)i * nq + e] = orc_cdot(P + (int64_t)i * d,
                                                Q + (int64_t)e * d, d);
}

/* halving-tree sum of the values v[j], j < 64 (absent values are +0) */
static float tree64(float *s)
{
    for (int h = LANES / 2; h >= 1; h /= 2)
        for (int j = 0; j < h; ++j)
            s[j] = s[j] + s[j + h];
    return s[0];
}

/* (a, ia) ranks before (b, ib) in the order (value desc, index asc) */
static int ranks_before(float a, int ia, float b, int ib)
{
    return (a > b) || (a == b && ia < ib);
}

/* ---------------------------------------------------------------- route ---
 * logits[t][e] = cdot(x_t, Wr[e]) + beta[e]     (beta may be NULL)
 * R_t = the K experts first in the order (logit desc, index asc).
 * eps_k = cexp(l[R_t[k]] - l[R_t[0]]).
 * norm_topk = 1: S = ((eps_0 + eps_1) + eps_2) + ...   (top-K only)
 * norm_topk = 0: S = sum over all E experts of cexp(l_e - l[R_t[0]]),
 *                partial j sums e = j, j+64, j+128, j+192 in that order,
 *                then the halving tree of cdot.
 * w_k = eps_k / S.
 */
void orc_route(const float *x, int B, int d, const float *Wr,
               const float *beta, int E, int K, int norm_topk,
               float *logits, int32_t *ids, float *w)
{
    /* tokens are independent: the loop may run on several host threads
       (OpenMP) with results identical to one thread */
#pragma omp parallel for schedule(static)
    for (int t = 0; t < B; ++t) {
        const float *xt = x + (int64_t)t * d;
        float *lt = logits + (int64_t)t * E;
        for (int e = 0; e < E; ++e) {
            float v = orc_cdot(xt, Wr + (int64_t)e * d, d);
            if (beta) v = v + beta[e];
            lt[e] = v;
        }
        int32_t *it = ids + (int64_t)t * K;
        /* selection by repeated extraction of the first-ranked remaining */
        for (int k = 0; k < K; ++k) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                int taken = 0;
                for (int q = 0; q < k; ++q) taken |= (it[q] == e);
                if (taken) continue;
                if (best < 0 || ranks_before(lt[e], e, lt[best], best))
                    best = e;
            }
            it[k] = best;
        }
        float lmax = lt[it[0]];
        float eps[64];
        for (int k = 0; k < K; ++k) eps[k] = orc_cexp(lt[it[k]] - lmax);
        float S;
        if (norm_topk) {
            S = 0.0f;
            for (int k = 0; k < K; ++k) S = S + eps[k];
        } else {
            float s[LANES];
            for (int j = 0; j < LANES; ++j) {
                float acc = 0.0f;
                for (int e = j; e < E; e += LANES)
                    acc = acc + orc_cexp(lt[e] - lmax);
                s[j] = acc;
            }
            S = tree64(s);
        }
        for (int k = 0; k < K; ++k) w[(int64_t)t * K + k] = eps[k] / S;
    }
}

/* -------------------------------------------------------------- predict ---
 * ss = cdot(x_t, x_t); inv = ss > 0 ? 1 / sqrt(ss) : 0      (z_bar = x * inv)
 * s_hat = cdot(x_t, A[u]) * inv;  s_hat = s_hat + b[u]      (a_u . z_bar + b_u)
 * cost = (w * w) * cexp(s_hat)
 */
void orc_predict(const float *x, int B, int d, const float *A,
                 const float *b, int K, const int32_t *ids, const float *w,
                 float *cost, float *inv_norm)
{
#pragma omp parallel for schedule(static)
    for (int t = 0; t < B; ++t) {
        const float *xt = x + (int64_t)t * d;
        float ss = orc_cdot(xt, xt, d);
        float inv = 0.0f;
        if (ss > 0.0f) {
            float rt = sqrtf(ss);
            inv = 1.0f / rt;
        }
        if (inv_norm) inv_norm[t] = inv;
        for (int k = 0; k < K; ++k) {
            int u = ids[(int64_t)t * K + k];
            float s = orc_cdot(xt, A + (int64_t)u * d, d) * inv;
            s = s + b[u];
            float wk = w[(int64_t)t * K + k];
            float w2 = wk * wk;
            cost[(int64_t)t * K + k] = w2 * orc_cexp(s);
        }
    }
}

/* ------------------------------------------------------------ aggregate ---
 * D_hat[u] = sum over tokens t with u in R_t of cost(t, u).
 * Tokens are taken in chunks of 64 (chunk c = tokens 64c .. 64c+63); inside
 * a chunk, position j holds cost(64c + j, u) if that token routes u and +0
 * otherwise, and the chunk sum is the halving tree of cdot.  Chunk sums are
 * added in ascending chunk order: D = ((s_0 + s_1) + s_2) + ...
 * count[u] = number of tokens that route u.
 */
void orc_aggregate(int B, int K, int E, const int32_t *ids,
                   const float *cost, float *scores, int32_t *counts)
{
    for (int u = 0; u < E; ++u) {
        float D = 0.0f;
        int cnt = 0;
        for (int c = 0; c * LANES < B; ++c) {
            float s[LANES];
            for (int j = 0; j < LANES; ++j) {
                int t = c * LANES + j;
                s[j] = 0.0f;
                if (t >= B) continue;
                for (int k = 0; k < K; ++k)
                    if (ids[(int64_t)t * K + k] == u) {
                        s[j] = cost[(int64_t)t * K + k];
                        ++cnt;
                    }
            }
            float cs = tree64(s);
            D = (c == 0) ? cs : D + cs;
        }
        scores[u] = D;
        counts[u] = cnt;
    }
}

/* ---------------------------------------------------------------- gates ---
 * Gate numerators of a token for the experts it executes, and the two
 * denominators of Sec. 3.5:
 *   num_j = cexp(l[v_j] - l[R_t[0]])
 *   paper  : g_j = num_j / S, S the router's own denominator (as in route)
 *   renorm : g_j = num_j / (((num_0 + num_1) + ...) over executed j)
 */
void orc_gates(const float *lt, const int32_t *rt, int E, int K,
               int norm_topk, const int32_t *exec, int n_exec, int renorm,
               float *g)
{
    float lmax = lt[rt[0]];
    float num[64];
    for (int j = 0; j < n_exec; ++j) num[j] = orc_cexp(lt[exec[j]] - lmax);
    float S;
    if (renorm) {
        S = 0.0f;
        for (int j = 0; j < n_exec; ++j) S = S + num[j];
    } else if (norm_topk) {
        S = 0.0f;
        for (int k = 0; k < K; ++k) S = S + orc_cexp(lt[rt[k]] - lmax);
    } else {
        float s[LANES];
        for (int j = 0; j < LANES; ++j) {
            float acc = 0.0f;
            for (int e = j; e < E; e += LANES)
                acc = acc + orc_cexp(lt[e] - lmax);
            s[j] = acc;
        }
        S = tree64(s);
    }
    for (int j = 0; j < n_exec; ++j) g[j] = num[j] / S;
}
