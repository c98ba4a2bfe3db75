/*
 * Plain CPU oracle of the LiLiCorr draft-correlation path.
 *
 * TEST INFRASTRUCTURE ONLY: this file is compiled by gcc and called (through oracle/__init__.py)
 * from tests/, from the smoke check and from the benchmark's CPU-baseline leg, and from nothing
 * else. It shares no code, header or constant with the HIP library.
 *
 * Every quantity is computed from its definition in double precision, single-threaded, with
 * plain loops. Inputs are widened exactly (bf16 -> float -> double); outputs are rounded to
 * float once, at the end of each call, so chained calls see float arrays at every call boundary.
 *
 * Readings of points the paper leaves open (listed again in the design notes):
 *  - top-K order: value descending, ties by lower token id; -0 and +0 compare equal;
 *  - cosine with a zero vector is 0, and a zero vector normalises to zeros;
 *  - y = e W with W[i][j] (i = input dimension, row-vector convention);
 *  - without an anchor the anchor scores are taken as all zero (slot 0 then commits its
 *    rank-0 candidate, the drafter's own argmax);
 *  - the walk breaks ties toward the lower candidate index;
 *  - logp_weight (lambda) adds lambda * logp to the walk's node scores; lambda = 0 is the
 *    paper's rule.
 *
 * Return value of every function: 0 on success, -1 on an argument that breaks the stated
 * preconditions (nothing is then written).
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

static double widen(const void *base, int dtype, int64_t i)
{
    if (dtype == ORACLE_F32)
        return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* ---------------------------------------------------------------------------------------------
 * Step 1: vocabulary-wide log-normalisation and top-K candidates.
 *
 * The candidate pool is the drafter's K most probable tokens at each slot (Sec. 3.2); the
 * serving kernel normalises the logits over the whole vocabulary in the same pass that extracts
 * the candidates (implementation appendix, "Serving"). Here:
 *     lse = m + log(sum_v exp(x_v - m)),  m = max_v x_v
 *     the K candidates are the first K entries of all v sorted by (x_v desc, v asc),
 *     logp_k = x_{id_k} - lse.
 * ------------------------------------------------------------------------------------------- */

struct sort_ctx {
    const double *x;
};

static int cmp_desc_then_id(const void *pa, const void *pb, void *arg)
{
    const struct sort_ctx *c = (const struct sort_ctx *)arg;
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    double xa = c->x[a], xb = c->x[b];
    if (xa > xb)
        return -1;
    if (xa < xb)
        return 1;
    return (a < b) ? -1 : (a > b) ? 1 : 0;
}

int oracle_topk(const void *logits, int dtype, int64_t N, int64_t B, int64_t V, int K,
                int32_t *ids, float *logp)
{
    if (!logits || !ids || !logp || N < 0 || B < 0 || V < 1 || K < 1 || K > V)
        return -1;
    if (dtype != ORACLE_F32 && dtype != ORACLE_BF16)
        return -1;
    double *x = (double *)malloc(sizeof(double) * (size_t)V);
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)V);
    if (!x || !order) {
        free(x);
        free(order);
        return -1;
    }
    int rc = 0;
    for (int64_t row = 0; row < N * B; ++row) {
        for (int64_t v = 0; v < V; ++v)
            x[v] = widen(logits, dtype, row * V + v);
        double m = -INFINITY;
        for (int64_t v = 0; v < V; ++v)
            if (x[v] > m)
                m = x[v];
        if (!(m > -INFINITY) || isinf(m) || isnan(m)) {
            rc = -1; /* a slot needs at least one finite logit */
            break;
        }
        double s = 0.0;
        for (int64_t v = 0; v < V; ++v)
            s += exp(x[v] - m);
        double lse = m + log(s);

        for (int64_t v = 0; v < V; ++v)
            order[v] = (int32_t)v;
        struct sort_ctx ctx = {x};
        qsort_r(order, (size_t)V, sizeof(int32_t), cmp_desc_then_id, &ctx);
        for (int k = 0; k < K; ++k) {
            ids[row * K + k] = order[k];
            logp[row * K + k] = (float)(x[order[k]] - lse);
        }
    }
    free(x);
    free(order);
    return rc;
}

/* ---------------------------------------------------------------------------------------------
 * Step 2: candidate in/out vectors.
 *
 * Each candidate gets an out vector and an in vector, each normalised to unit L2 norm (Sec. 3.2;
 * the two linear heads of the implementation appendix). The trained head is not available; its
 * last linear layers are stood in for by u = E[id] W, then v = u / ||u||.
 * ------------------------------------------------------------------------------------------- */

static void project_normalise(const double *e, const float *W, int d, float *out)
{
    double *u = (double *)calloc((size_t)d, sizeof(double));
    for (int j = 0; j < d; ++j) {
        double acc = 0.0;
        for (int i = 0; i < d; ++i)
            acc += e[i] * (double)W[(size_t)i * d + j];
        u[j] = acc;
    }
    double ss = 0.0;
    for (int j = 0; j < d; ++j)
        ss += u[j] * u[j];
    double norm = sqrt(ss);
    for (int j = 0; j < d; ++j)
        out[j] = (norm > 0.0) ? (float)(u[j] / norm) : 0.0f;
    free(u);
}

int oracle_candidate_vectors(const int32_t *ids, const void *E, int e_dtype, int64_t V, int d,
                             const float *W_in, const float *W_out, int64_t N, int64_t B, int K,
                             float *in_vec, float *out_vec)
{
    if (!ids || !E || !W_in || !W_out || !in_vec || !out_vec || V < 1 || d < 1 || N < 0 ||
        B < 0 || K < 1)
        return -1;
    if (e_dtype != ORACLE_F32 && e_dtype != ORACLE_BF16)
        return -1;
    int64_t M = N * B * (int64_t)K;
    for (int64_t c = 0; c < M; ++c)
        if (ids[c] < 0 || ids[c] >= V)
            return -1;
    double *e = (double *)malloc(sizeof(double) * (size_t)d);
    for (int64_t c = 0; c < M; ++c) {
        for (int i = 0; i < d; ++i)
            e[i] = widen(E, e_dtype, (int64_t)ids[c] * d + i);
        project_normalise(e, W_in, d, in_vec + c * d);
        project_normalise(e, W_out, d, out_vec + c * d);
    }
    free(e);
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Step 3: pair matching scores, Eq. (pair):
 *     phi(s, k, k') = sigma * cos(out_{s,k}, in_{s+1,k'})
 * S[n][t][k][k'] couples slot t (out) with slot t+1 (in), t = 0..B-2. With an anchor out vector
 * the anchor pair is S0[n][k'] = sigma * cos(anchor_out[n], in[n][0][k']).
 * ------------------------------------------------------------------------------------------- */

static double cosine(const float *a, const float *b, int d)
{
    double ab = 0.0, aa = 0.0, bb = 0.0;
    for (int i = 0; i < d; ++i) {
        ab += (double)a[i] * (double)b[i];
        aa += (double)a[i] * (double)a[i];
        bb += (double)b[i] * (double)b[i];
    }
    if (aa == 0.0 || bb == 0.0)
        return 0.0;
    return ab / (sqrt(aa) * sqrt(bb));
}

int oracle_pair_scores(const float *in_vec, const float *out_vec, const float *anchor_out,
                       int64_t N, int64_t B, int K, int d, float sigma, float *S, float *S0)
{
    if (!in_vec || !out_vec || N < 0 || B < 1 || K < 1 || d < 1)
        return -1;
    if (B > 1 && !S)
        return -1;
    if (anchor_out && !S0)
        return -1;
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t t = 0; t + 1 < B; ++t)
            for (int k = 0; k < K; ++k)
                for (int kk = 0; kk < K; ++kk) {
                    const float *o = out_vec + ((n * B + t) * K + k) * (int64_t)d;
                    const float *i = in_vec + ((n * B + t + 1) * K + kk) * (int64_t)d;
                    S[((n * (B - 1) + t) * K + k) * K + kk] =
                        (float)((double)sigma * cosine(o, i, d));
                }
        if (anchor_out)
            for (int kk = 0; kk < K; ++kk) {
                const float *i = in_vec + ((n * B + 0) * K + kk) * (int64_t)d;
                S0[n * K + kk] = (float)((double)sigma * cosine(anchor_out + n * d, i, d));
            }
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Step 4: greedy left-to-right walk (Sec. 3.5) with the local log-likelihood of Eq. (localar).
 *     z_t[k] = phi(t-1, c_{t-1}, k) + lambda * logp[t][k],   c_t = argmax_k z_t[k]
 *     logq[t] = z_t[c_t] - log sum_k exp(z_t[k])
 * Slot 0 uses the anchor scores S0 (all zero when no anchor is given). Ties go to the lowest k.
 * draft[t] = ids[t][c_t], choice[t] = c_t.
 * The node score z is formed in float with one rounding (fmaf), the precision the GPU kernel
 * takes its argmax in; with lambda = 0 (the paper's rule, z = phi alone) the logp term is absent
 * and z is the float score itself. logq is then evaluated in double from those float scores.
 * ------------------------------------------------------------------------------------------- */

int oracle_greedy_walk(const float *S, const float *S0, const float *logp, const int32_t *ids,
                       int64_t N, int64_t B, int K, float logp_weight, int32_t *draft,
                       int32_t *choice, float *logq)
{
    if (!logp || !ids || !draft || N < 0 || B < 1 || K < 1)
        return -1;
    if (B > 1 && !S)
        return -1;
    float *z = (float *)malloc(sizeof(float) * (size_t)K);
    for (int64_t n = 0; n < N; ++n) {
        int prev = -1;
        for (int64_t t = 0; t < B; ++t) {
            for (int k = 0; k < K; ++k) {
                float pair;
                if (t == 0)
                    pair = S0 ? S0[n * K + k] : 0.0f;
                else
                    pair = S[((n * (B - 1) + (t - 1)) * K + prev) * K + k];
                z[k] = (logp_weight == 0.0f) ? pair
                                              : fmaf(logp_weight, logp[(n * B + t) * K + k], pair);
            }
            int best = 0;
            for (int k = 1; k < K; ++k)
                if (z[k] > z[best])
                    best = k;
            double m = (double)z[best];
            double s = 0.0;
            for (int k = 0; k < K; ++k)
                s += exp((double)z[k] - m);
            draft[n * B + t] = ids[(n * B + t) * K + best];
            if (choice)
                choice[n * B + t] = best;
            if (logq)
                logq[n * B + t] = (float)((double)z[best] - (m + log(s)));
            prev = best;
        }
    }
    free(z);
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Exact max-path decode (decode-rule appendix, Eq. pathscore): the path c = (c_0 .. c_{B-1})
 * that maximises the sum of its matching terms
 *     g(c) = P_0[c_0] + sum_{t=1}^{B-1} phi(t-1, c_{t-1}, c_t)   (+ lambda sum_t logp[t][c_t])
 * with P_0 = S0, or all zero without an anchor (slot 0's candidate is then free). Sweeping left
 * to right, best[k] is the score of the best path ending at candidate k of the current slot and
 * from[t][k] the predecessor it came through; the path is then traced back from the best
 * candidate of the last slot. Ties go to the lowest index, for predecessors and for the final
 * candidate: among all maximising paths this returns the one that is smallest when read from the
 * last slot backwards.
 * Path sums and comparisons are in double: each float term is widened exactly and every partial
 * sum is rounded once, in the order of the sum above (the lambda term, an exact product of two
 * floats in double, is added after the matching term of its slot). The maximiser is therefore the
 * exact one unless two path sums differ by less than the double rounding of the partial sums
 * (about B * 2^-53 * max |partial sum|).
 * logq[t] is Eq. (localar) along the returned path, z_t[k] = P_t(c_{t-1}, k) (+ lambda logp), the
 * node score of the greedy walk, logq[t] = z_t[c_t] - log sum_k exp z_t[k], in double from the
 * float z; score[n] = g of the returned path, rounded once to float.
 * ------------------------------------------------------------------------------------------- */

int oracle_viterbi_walk(const float *S, const float *S0, const float *logp, const int32_t *ids,
                        int64_t N, int64_t B, int K, float logp_weight, int32_t *draft,
                        int32_t *choice, float *logq, float *score)
{
    if (!logp || !ids || !draft || N < 0 || B < 1 || K < 1)
        return -1;
    if (B > 1 && !S)
        return -1;
    const double lam = (double)logp_weight;
    double *best = (double *)malloc(sizeof(double) * (size_t)K);
    double *next = (double *)malloc(sizeof(double) * (size_t)K);
    float *z = (float *)malloc(sizeof(float) * (size_t)K);
    int *from = (int *)malloc(sizeof(int) * (size_t)(B * K));
    int *path = (int *)malloc(sizeof(int) * (size_t)B);
    for (int64_t n = 0; n < N; ++n) {
        for (int k = 0; k < K; ++k) {
            double v = S0 ? (double)S0[n * K + k] : 0.0;
            if (logp_weight != 0.0f)
                v += lam * (double)logp[(n * B + 0) * K + k];
            best[k] = v;
        }
        for (int64_t t = 1; t < B; ++t) {
            const float *St = S + (n * (B - 1) + (t - 1)) * K * (int64_t)K;
            for (int k = 0; k < K; ++k) {
                double bv = best[0] + (double)St[0 * K + k];
                int bp = 0;
                for (int p = 1; p < K; ++p) {
                    const double v = best[p] + (double)St[p * K + k];
                    if (v > bv) {
                        bv = v;
                        bp = p;
                    }
                }
                if (logp_weight != 0.0f)
                    bv += lam * (double)logp[(n * B + t) * K + k];
                next[k] = bv;
                from[t * K + k] = bp;
            }
            memcpy(best, next, sizeof(double) * (size_t)K);
        }
        int c = 0;
        for (int k = 1; k < K; ++k)
            if (best[k] > best[c])
                c = k;
        if (score)
            score[n] = (float)best[c];
        path[B - 1] = c;
        for (int64_t t = B - 1; t >= 1; --t)
            path[t - 1] = from[t * K + path[t]];
        for (int64_t t = 0; t < B; ++t) {
            for (int k = 0; k < K; ++k) {
                float pair;
                if (t == 0)
                    pair = S0 ? S0[n * K + k] : 0.0f;
                else
                    pair = S[((n * (B - 1) + (t - 1)) * K + path[t - 1]) * K + k];
                z[k] = (logp_weight == 0.0f) ? pair
                                              : fmaf(logp_weight, logp[(n * B + t) * K + k], pair);
            }
            double m = -INFINITY;
            for (int k = 0; k < K; ++k)
                if ((double)z[k] > m)
                    m = (double)z[k];
            double s = 0.0;
            for (int k = 0; k < K; ++k)
                s += exp((double)z[k] - m);
            const int ct = path[t];
            draft[n * B + t] = ids[(n * B + t) * K + ct];
            if (choice)
                choice[n * B + t] = ct;
            if (logq)
                logq[n * B + t] = (float)((double)z[ct] - (m + log(s)));
        }
    }
    free(best);
    free(next);
    free(z);
    free(from);
    free(path);
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Candidate confidence features (implementation appendix, node construction): five scalars per
 * candidate, read from the drafter's distribution at its slot. For candidate k (rank k, 0-based)
 * of a row of K top-K log-probabilities logp[0..K-1] (sorted, rank 0 the most likely):
 *     feat[k] = { logp[k], exp(logp[k]), logp[0] - logp[k], k / (K-1) (0 when K = 1), [k == 0] }
 * Readings: the gap to the most likely token is taken as the non-negative difference, and the
 * rank in [0, 1] as k / (K-1). Computed in double from the float log-probabilities.
 * ------------------------------------------------------------------------------------------- */

int oracle_candidate_features(const float *logp, int64_t rows, int K, float *feat)
{
    if (!logp || !feat || rows < 0 || K < 1)
        return -1;
    for (int64_t r = 0; r < rows; ++r) {
        const double top = (double)logp[r * K];
        for (int k = 0; k < K; ++k) {
            const double lp = (double)logp[r * K + k];
            float *f = feat + (r * K + k) * 5;
            f[0] = (float)lp;
            f[1] = (float)exp(lp);
            f[2] = (float)(top - lp);
            f[3] = K > 1 ? (float)((double)k / (double)(K - 1)) : 0.0f;
            f[4] = k == 0 ? 1.0f : 0.0f;
        }
    }
    return 0;
}
