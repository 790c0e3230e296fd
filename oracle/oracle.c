/*
 * Elbow-routed MoE layer: plain CPU oracle (fp64).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load this library.  It shares no code, header, table or helper
 * with the GPU library; the two meet only on the seeded input arrays.
 *
 * Everything is written as the paper defines it, in double precision, with plain loops:
 *
 *   routing (Section 2 "Elbow-Based Routing", Section 2.1 "Capped Expert Selection",
 *            Appendix A.1 Algorithm 1 "Elbow Detection via Kneedle Approximation"):
 *     p = softmax(l); sort p descending; p_min, p_max; normalise each sorted point to
 *     the unit square; deviation D_i from the reference line; e = argmax D;
 *     k = min(e + 1, K).
 *   expert FFN: OLMoE's SwiGLU MLP, FFN(x) = W_down (silu(W_gate x) * (W_up x)).
 *   layer:      y_t = [residual_t +] sum_{j<k_t} w_{t,j} FFN_{id_{t,j}}(x_t).
 *
 * Readings of the paper that this file fixes (the paper is silent or garbled there):
 *   - orientation of the normalised curve: Algorithm 1 prints p'_i = (p_i - p_min)/(R+eps)
 *     with p sorted descending, which makes D strictly decreasing and k = 1 for every
 *     input.  The elbow-angle definition (Section 2.3) puts the first normalised point at
 *     (0,0) and the last at (1,1), so the curve is flipped to increasing:
 *     p'_i = (p_max - p_(i)) / (p_max - p_min + eps).  D_i is then the depth of sorted
 *     point i below the chord joining the first and last sorted points.
 *   - eps = 1e-8 by default (the paper does not give its value); a parameter here.
 *   - argmax ties go to the smallest index (so a curve with no point below the chord
 *     gives e = 0, k = 1).
 *   - e in Algorithm 1 is 0-based and the algorithm returns e + 1; Section 2.1 caps that
 *     count at K.
 *   - the sort key is (logit descending, expert id ascending): softmax is strictly
 *     increasing, so this is the descending order of p with ties broken by lower id.
 *   - the weight of a selected expert is its full-softmax probability p, not
 *     renormalised over the selected set (renorm = 1 renormalises instead).
 *   - fixed top-K routing (the paper's baseline) is the same path with k = K.
 *
 *   - elbow angle (Section 2.3): taken as 180 degrees when the elbow is the first point.
 *   - tail randomisation (Section 2.2): the random tail is drawn from the experts outside
 *     the elbow's selection with one caller-supplied uniform value per (token, expert).
 *
 * Parity pins for every function here live in tests/test_oracle_*.py (hand-worked
 * curves, exact-rational brute force, invariants, the load-balance theorem, and special
 * cases that reduce to library routines).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MODE_ELBOW 0
#define ORC_MODE_TOPK 1

int orc_version(void) { return 2; }

/* Order indices by (key descending, index ascending): a plain insertion sort. */
static void order_desc(const double *key, int N, int *sigma)
{
    for (int i = 0; i < N; ++i) sigma[i] = i;
    for (int i = 1; i < N; ++i) {
        int cur = sigma[i];
        int j = i - 1;
        while (j >= 0) {
            int prev = sigma[j];
            int before = key[prev] > key[cur] || (key[prev] == key[cur] && prev < cur);
            if (before) break;
            sigma[j + 1] = prev;
            --j;
        }
        sigma[j + 1] = cur;
    }
}

/*
 * Steps after the sort (Algorithm 1, from p_min/p_max to the returned k, and the cap of
 * Section 2.1), on one token's probabilities p[N] and its order sigma.
 * Writes k, ids[0..K), w[0..K) (padding -1 / 0), and diagnostics:
 *   e_out      argmax index (0-based, uncapped; -1 in top-K mode)
 *   margin     D_{e} - max{D_i : min(i+1, K) != k}  (+inf when no such i, or top-K mode)
 *   competitor the i attaining that max (-1 if none)
 */
static void select_experts(const double *p, const int *sigma, int N, int K, double eps,
                           int mode, int renorm, int *k_out, int *ids, double *w,
                           int *e_out, double *margin, int *competitor)
{
    int k;
    int e = -1;
    double mg = INFINITY;
    int comp = -1;
    if (mode == ORC_MODE_TOPK) {
        k = K;
    } else {
        double D[N > 0 ? N : 1];
        double p_max = p[sigma[0]];
        double p_min = p[sigma[N - 1]];
        double denom = p_max - p_min + eps;
        for (int i = 0; i < N; ++i) {
            double pn = (p_max - p[sigma[i]]) / denom;   /* normalised probability */
            double xn = (double)i / (double)(N - 1);     /* normalised index */
            D[i] = pn - xn;                              /* deviation from the line */
        }
        e = 0;
        for (int i = 1; i < N; ++i)
            if (D[i] > D[e]) e = i;                      /* first index wins ties */
        k = e + 1 < K ? e + 1 : K;
        for (int i = 0; i < N; ++i) {
            int ki = i + 1 < K ? i + 1 : K;
            if (ki == k) continue;
            double gap = D[e] - D[i];
            if (gap < mg) { mg = gap; comp = i; }
        }
    }
    double sel = 0.0;
    for (int j = 0; j < k; ++j) sel += p[sigma[j]];
    for (int j = 0; j < K; ++j) {
        if (j < k) {
            ids[j] = sigma[j];
            w[j] = renorm ? p[sigma[j]] / sel : p[sigma[j]];
        } else {
            ids[j] = -1;
            w[j] = 0.0;
        }
    }
    *k_out = k;
    if (e_out) *e_out = e;
    if (margin) *margin = mg;
    if (competitor) *competitor = comp;
}

static int check_params(long T, int N, int K, double eps, int mode)
{
    if (T < 0 || N < 2 || K < 1 || K > N || !(eps >= 0.0)) return 1;
    if (mode != ORC_MODE_ELBOW && mode != ORC_MODE_TOPK) return 1;
    return 0;
}

/*
 * Route T tokens from fp32 logits [T, N] (row-major).  Outputs k[T], ids[T, K], w[T, K];
 * e, margin and competitor [T] are optional (NULL to skip).  Returns 0, or 1 on invalid
 * arguments, 2 if a row has no finite logit.
 */
int orc_route(const float *logits, long T, int N, int K, double eps, int mode, int renorm,
              int *k, int *ids, double *w, int *e, double *margin, int *competitor)
{
    if (check_params(T, N, K, eps, mode)) return 1;
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (long t = 0; t < T; ++t) {
        double l[N], p[N];
        int sigma[N];
        for (int j = 0; j < N; ++j) l[j] = (double)logits[t * N + j];
        /* softmax (Section 2; Algorithm 1, first step) */
        double mx = -INFINITY;
        for (int j = 0; j < N; ++j) if (l[j] > mx) mx = l[j];
        if (!isfinite(mx)) { bad = 1; continue; }
        double s = 0.0;
        for (int j = 0; j < N; ++j) { p[j] = exp(l[j] - mx); s += p[j]; }
        for (int j = 0; j < N; ++j) p[j] /= s;
        /* descending sort; ties (equal logits) by lower expert id */
        order_desc(l, N, sigma);
        select_experts(p, sigma, N, K, eps, mode, renorm, &k[t], ids + t * K, w + t * K,
                       e ? &e[t] : NULL, margin ? &margin[t] : NULL,
                       competitor ? &competitor[t] : NULL);
    }
    return bad ? 2 : 0;
}

/*
 * Same selection on given probability vectors p[T, N] (no softmax): the sort key is p
 * itself, ties by lower id.  Used to pin the selection rule on exact curves.
 */
int orc_route_from_probs(const double *p, long T, int N, int K, double eps, int mode,
                         int renorm, int *k, int *ids, double *w, int *e, double *margin,
                         int *competitor)
{
    if (check_params(T, N, K, eps, mode)) return 1;
    for (long t = 0; t < T; ++t) {
        int sigma[N];
        order_desc(p + t * N, N, sigma);
        select_experts(p + t * N, sigma, N, K, eps, mode, renorm, &k[t], ids + t * K,
                       w + t * K, e ? &e[t] : NULL, margin ? &margin[t] : NULL,
                       competitor ? &competitor[t] : NULL);
    }
    return 0;
}

/*
 * Elbow angle (Section 2.3): the angle at the elbow point (x'_e, p'_e) of the normalised
 * curve between the first normalised point (0,0) and the last (1,1):
 *   theta = arccos( v1 . v2 / (|v1| |v2|) ),  v1 = (-x'_e, -p'_e),  v2 = (1 - x'_e, 1 - p'_e),
 * with e the uncapped elbow index (the argmax of D over all i, first index on ties) and
 * p'_e the flipped normalisation of the routing step.  In degrees.  When e = 0 the elbow
 * point is the first point itself and v1 = 0: the angle is taken as 180 degrees (a curve
 * with no point below the chord has no elbow).
 */
static void elbow_angle_one(const double *p, const int *sigma, int N, double eps, int *e_out,
                            double *theta)
{
    double hi = p[sigma[0]];
    double lo = p[sigma[N - 1]];
    double R = hi - lo + eps;
    int e = 0;
    double best = 0.0; /* D_0 = 0 */
    for (int i = 1; i < N; ++i) {
        double yi = (hi - p[sigma[i]]) / R;         /* normalised probability */
        double xi = (double)i / (double)(N - 1);   /* normalised index */
        if (yi - xi > best) { best = yi - xi; e = i; }
    }
    double xe = (double)e / (double)(N - 1);
    double ye = (hi - p[sigma[e]]) / R;
    double v1x = -xe, v1y = -ye, v2x = 1.0 - xe, v2y = 1.0 - ye;
    double n1 = sqrt(v1x * v1x + v1y * v1y), n2 = sqrt(v2x * v2x + v2y * v2y);
    double th;
    if (e == 0 || n1 == 0.0 || n2 == 0.0) {
        th = 180.0;
    } else {
        double c = (v1x * v2x + v1y * v2y) / (n1 * n2);
        if (c > 1.0) c = 1.0;
        if (c < -1.0) c = -1.0;
        th = acos(c) * (180.0 / acos(-1.0));
    }
    *e_out = e;
    *theta = th;
}

/* softmax of one row of fp32 logits into p (fp64); returns 0 if no logit is finite */
static int softmax_row(const float *lrow, int N, double *l, double *p)
{
    for (int j = 0; j < N; ++j) l[j] = (double)lrow[j];
    double mx = -INFINITY;
    for (int j = 0; j < N; ++j) if (l[j] > mx) mx = l[j];
    if (!isfinite(mx)) return 0;
    double s = 0.0;
    for (int j = 0; j < N; ++j) { p[j] = exp(l[j] - mx); s += p[j]; }
    for (int j = 0; j < N; ++j) p[j] /= s;
    return 1;
}

/* Elbow index e[T] (uncapped) and angle theta[T] (degrees) from fp32 logits [T, N]. */
int orc_elbow_angle(const float *logits, long T, int N, double eps, int *e, double *theta)
{
    if (T < 0 || N < 2 || !(eps >= 0.0)) return 1;
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (long t = 0; t < T; ++t) {
        double l[N], p[N];
        int sigma[N];
        if (!softmax_row(logits + t * N, N, l, p)) { bad = 1; continue; }
        order_desc(l, N, sigma);
        elbow_angle_one(p, sigma, N, eps, &e[t], &theta[t]);
    }
    return bad ? 2 : 0;
}

/* The same on given probability vectors p[T, N] (sort key p, ties by lower id). */
int orc_elbow_angle_from_probs(const double *p, long T, int N, double eps, int *e,
                               double *theta)
{
    if (T < 0 || N < 2 || !(eps >= 0.0)) return 1;
    for (long t = 0; t < T; ++t) {
        int sigma[N];
        order_desc(p + t * N, N, sigma);
        elbow_angle_one(p + t * N, sigma, N, eps, &e[t], &theta[t]);
    }
    return 0;
}

/*
 * Tail randomisation (Section 2.2, the signal/noise check): the elbow's k = min(e + 1, K)
 * experts keep ranks 0..k-1; the other K - k slots are filled with experts drawn uniformly
 * from those outside the elbow's selection (equivalently, from the ranks >= k).  The draw is
 * an input: rand[T, N] holds one value per (token, expert); the drawn experts are the K - k
 * non-selected ones with the smallest rand (ties: lower id), in increasing order of rand.
 * Weights are the experts' own probabilities p (renorm = 1: over the K experts).
 * Outputs k_elbow[T] (where the random tail starts), ids[T, K], w[T, K]: all K slots are
 * filled.
 */
int orc_route_tail_random(const float *logits, const float *rand, long T, int N, int K,
                          double eps, int renorm, int *k_elbow, int *ids, double *w)
{
    if (check_params(T, N, K, eps, ORC_MODE_ELBOW)) return 1;
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (long t = 0; t < T; ++t) {
        double l[N], p[N];
        int sigma[N], kk;
        double wtmp[K];
        int itmp[K];
        if (!softmax_row(logits + t * N, N, l, p)) { bad = 1; continue; }
        order_desc(l, N, sigma);
        select_experts(p, sigma, N, K, eps, ORC_MODE_ELBOW, 0, &kk, itmp, wtmp, NULL, NULL,
                       NULL);
        int used[N];
        for (int c = 0; c < N; ++c) used[c] = 0;
        for (int j = 0; j < kk; ++j) used[sigma[j]] = 1;
        for (int j = 0; j < K; ++j) {
            int c;
            if (j < kk) {
                c = sigma[j];
            } else {
                c = -1;
                for (int q = 0; q < N; ++q) {
                    if (used[q]) continue;
                    if (c < 0 || rand[t * N + q] < rand[t * N + c]) c = q;
                }
                used[c] = 1;
            }
            ids[t * K + j] = c;
            w[t * K + j] = p[c];
        }
        if (renorm) {
            double s = 0.0;
            for (int j = 0; j < K; ++j) s += w[t * K + j];
            for (int j = 0; j < K; ++j) w[t * K + j] /= s;
        }
        k_elbow[t] = kk;
    }
    return bad ? 2 : 0;
}

/* Router logits of one token, l = W_r x (the router is a bias-free linear layer). */
static void logits_one(const float *x, const float *Wr, int d, int N, double *out)
{
    for (int n = 0; n < N; ++n) {
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc += (double)Wr[(long)n * d + c] * (double)x[c];
        out[n] = acc;
    }
}

/* Router logits for T tokens: out[T, N] (fp64). */
void orc_router_logits(const float *x, const float *Wr, long T, int d, int N, double *out)
{
#pragma omp parallel for schedule(static)
    for (long t = 0; t < T; ++t) logits_one(x + t * d, Wr, d, N, out + t * N);
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/*
 * One expert's SwiGLU MLP on one token: out[d] = W_down (silu(W_gate x) * (W_up x)).
 * Wgu is that expert's [2m, d] block (gate rows first), Wd its [d, m] block.
 */
static void expert_ffn(const float *x, const float *Wgu, const float *Wd, int d, int m,
                       double *h, double *out)
{
    for (int i = 0; i < m; ++i) {
        double g = 0.0, u = 0.0;
        const float *wg = Wgu + (long)i * d;
        const float *wu = Wgu + (long)(m + i) * d;
        for (int c = 0; c < d; ++c) {
            g += (double)wg[c] * (double)x[c];
            u += (double)wu[c] * (double)x[c];
        }
        h[i] = silu(g) * u;
    }
    for (int r = 0; r < d; ++r) {
        double acc = 0.0;
        const float *wd = Wd + (long)r * m;
        for (int i = 0; i < m; ++i) acc += (double)wd[i] * h[i];
        out[r] = acc;
    }
}

/*
 * Expert part of the layer for a list of tokens, given their routing:
 *   y[r] = [residual[tok_r] +] sum_{j<k[r]} w[r, j] * FFN_{ids[r, j]}(x[tok_r])
 * tok[n_tok] indexes rows of x [T, d]; k/ids/w are per listed token ([n_tok], [n_tok, K]).
 * Accumulation over j is in rank order, in double.  Returns 0 or 1 on a bad expert id.
 */
int orc_moe_experts(const float *x, const float *Wgu, const float *Wd, const float *residual,
                    long T, int d, int N, int m, int K, const long *tok, long n_tok,
                    const int *k, const int *ids, const double *w, double *y)
{
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (long r = 0; r < n_tok; ++r) {
        long t = tok[r];
        if (t < 0 || t >= T) { bad = 1; continue; }
        double *h = (double *)malloc(sizeof(double) * (size_t)m);
        double *o = (double *)malloc(sizeof(double) * (size_t)d);
        double *acc = y + r * d;
        for (int c = 0; c < d; ++c) acc[c] = residual ? (double)residual[t * d + c] : 0.0;
        for (int j = 0; j < k[r]; ++j) {
            int ex = ids[r * K + j];
            if (ex < 0 || ex >= N) { bad = 1; break; }
            expert_ffn(x + t * d, Wgu + (long)ex * 2 * m * d, Wd + (long)ex * d * m, d, m, h, o);
            for (int c = 0; c < d; ++c) acc[c] += w[r * K + j] * o[c];
        }
        free(h);
        free(o);
    }
    return bad;
}

/*
 * Whole layer for a list of tokens: router logits (fp64), routing on those logits,
 * then the expert part.  Routing outputs and the fp64 logits are returned for the
 * listed tokens.  Returns 0, 1 on invalid arguments, 2 on a row with no finite logit.
 */
int orc_moe_forward(const float *x, const float *Wr, const float *Wgu, const float *Wd,
                    const float *residual, long T, int d, int N, int m, int K, double eps,
                    int mode, int renorm, const long *tok, long n_tok, double *y,
                    double *logits, int *k, int *ids, double *w, double *margin)
{
    if (check_params(T, N, K, eps, mode) || d < 1 || m < 1) return 1;
    for (long r = 0; r < n_tok; ++r)
        if (tok[r] < 0 || tok[r] >= T) return 1;
    int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
    for (long r = 0; r < n_tok; ++r) {
        long t = tok[r];
        logits_one(x + t * d, Wr, d, N, logits + r * N);
        double l[N], p[N];
        int sigma[N];
        double mx = -INFINITY;
        for (int j = 0; j < N; ++j) { l[j] = logits[r * N + j]; if (l[j] > mx) mx = l[j]; }
        if (!isfinite(mx)) { bad = 1; continue; }
        double s = 0.0;
        for (int j = 0; j < N; ++j) { p[j] = exp(l[j] - mx); s += p[j]; }
        for (int j = 0; j < N; ++j) p[j] /= s;
        order_desc(l, N, sigma);
        select_experts(p, sigma, N, K, eps, mode, renorm, &k[r], ids + r * K, w + r * K,
                       NULL, margin ? &margin[r] : NULL, NULL);
    }
    if (bad) return 2;
    return orc_moe_experts(x, Wgu, Wd, residual, T, d, N, m, K, tok, n_tok, k, ids, w, y);
}

/*
 * Dispatch view of a routing: the expert-major token lists that a variable-k layer runs its
 * expert MLPs over (each token t appears once in the list of each of its k_t experts).
 *   counts[e]     = #{(t, j < k_t) : ids[t, j] = e}; their sum is sum_t k_t
 *   offsets[e]    = counts[0] + ... + counts[e-1]  (offsets[N] = sum_t k_t)
 *   row_token[r]  = the token of row r; rows of expert e are its tokens in increasing order
 *   inv[t, j]     = the row of (t, j) for j < k_t, -1 otherwise
 * Returns 0, or 1 if an id outside [0, N) is selected.
 */
int orc_dispatch(const int *k, const int *ids, long T, int N, int K, int *counts, int *offsets,
                 int *row_token, int *inv)
{
    for (int e = 0; e < N; ++e) counts[e] = 0;
    for (long t = 0; t < T; ++t)
        for (int j = 0; j < K; ++j) {
            inv[t * K + j] = -1;
            if (j >= k[t]) continue;
            int e = ids[t * K + j];
            if (e < 0 || e >= N) return 1;
            counts[e] += 1;
        }
    offsets[0] = 0;
    for (int e = 0; e < N; ++e) offsets[e + 1] = offsets[e] + counts[e];
    for (int e = 0; e < N; ++e) {
        int r = offsets[e];
        for (long t = 0; t < T; ++t)          /* tokens in increasing order */
            for (int j = 0; j < k[t] && j < K; ++j)
                if (ids[t * K + j] == e) {
                    row_token[r] = (int)t;
                    inv[t * K + j] = r;
                    ++r;
                }
    }
    return 0;
}
