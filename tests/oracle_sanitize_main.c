/*
 * Host-only driver for a sanitizer build of the CPU oracle (oracle/oracle.c), compiled by
 * tests/test_oracle_sanitize.py with AddressSanitizer and UndefinedBehaviorSanitizer.
 * It calls every oracle entry point on small seeded inputs, including the edge cases the
 * oracle handles (empty batches, K = 1 and K = N, tied and -inf logits, optional outputs
 * left NULL, invalid arguments), and checks the documented return codes.  Any out-of-bounds
 * access or undefined behaviour aborts the process with the sanitizer's report.
 * No routing arithmetic here: only input generation and return-code checks.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int orc_route(const float *logits, long T, int N, int K, double eps, int mode, int renorm,
              int *k, int *ids, double *w, int *e, double *margin, int *competitor);
int orc_route_from_probs(const double *p, long T, int N, int K, double eps, int mode,
                         int renorm, int *k, int *ids, double *w, int *e, double *margin,
                         int *competitor);
int orc_elbow_angle(const float *logits, long T, int N, double eps, int *e, double *theta);
int orc_elbow_angle_from_probs(const double *p, long T, int N, double eps, int *e,
                               double *theta);
int orc_route_tail_random(const float *logits, const float *rand, long T, int N, int K,
                          double eps, int renorm, int *k_elbow, int *ids, double *w);
void orc_router_logits(const float *x, const float *Wr, long T, int d, int N, double *out);
int orc_moe_experts(const float *x, const float *Wgu, const float *Wd, const float *residual,
                    long T, int d, int N, int m, int K, const long *tok, long n_tok,
                    const int *k, const int *ids, const double *w, double *y);
int orc_moe_forward(const float *x, const float *Wr, const float *Wgu, const float *Wd,
                    const float *residual, long T, int d, int N, int m, int K, double eps,
                    int mode, int renorm, const long *tok, long n_tok, double *y,
                    double *logits, int *k, int *ids, double *w, double *margin);
int orc_dispatch(const int *k, const int *ids, long T, int N, int K, int *counts, int *offsets,
                 int *row_token, int *inv);

static unsigned long long g_state = 0x9E3779B97F4A7C15ull;

/* uniform in [0, 1) from a 64-bit linear congruential step (Knuth's MMIX constants) */
static double uni(void)
{
    g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(g_state >> 11) * (1.0 / 9007199254740992.0);
}

static int g_fail = 0;

static void expect(int got, int want, const char *what)
{
    if (got != want) {
        fprintf(stderr, "FAIL %s: returned %d, expected %d\n", what, got, want);
        g_fail = 1;
    }
}

/* Exact-size heap buffers, so that any access past the end is caught. */
static void *buf(size_t n, size_t sz) { return calloc(n ? n : 1, sz); }

/* logits: kind 0 Gaussian-ish, 1 quantised (many ties), 2 with -inf entries */
static void fill_logits(float *l, long T, int N, int kind)
{
    for (long t = 0; t < T; ++t)
        for (int j = 0; j < N; ++j) {
            double v = (uni() + uni() + uni() - 1.5) * 3.0;
            if (kind == 1) v = floor(v * 2.0) / 2.0;
            if (kind == 2 && j != (int)(t % N) && uni() < 0.3) v = -INFINITY;
            l[t * N + j] = (float)v;
        }
}

static void routing_cases(void)
{
    const int Ns[] = {2, 3, 16, 64};
    const long T = 37;
    for (int a = 0; a < 4; ++a) {
        const int N = Ns[a];
        const int Ks[] = {1, N < 8 ? N : 8, N};
        float *l = buf(T * N, sizeof(float));
        float *r = buf(T * N, sizeof(float));
        double *p = buf(T * N, sizeof(double));
        for (int b = 0; b < 3; ++b) {
            const int K = Ks[b];
            int *k = buf(T, sizeof(int)), *ids = buf(T * K, sizeof(int));
            int *e = buf(T, sizeof(int)), *comp = buf(T, sizeof(int));
            double *w = buf(T * K, sizeof(double)), *mg = buf(T, sizeof(double));
            double *th = buf(T, sizeof(double));
            int *cnt = buf(N, sizeof(int)), *off = buf(N + 1, sizeof(int));
            int *rt = buf(T * K, sizeof(int)), *inv = buf(T * K, sizeof(int));
            for (int kind = 0; kind < 3; ++kind) {
                fill_logits(l, T, N, kind);
                for (long i = 0; i < T * N; ++i) r[i] = (float)uni();
                for (int mode = 0; mode < 2; ++mode)
                    for (int rn = 0; rn < 2; ++rn) {
                        expect(orc_route(l, T, N, K, 1e-8, mode, rn, k, ids, w, e, mg, comp), 0,
                               "orc_route");
                        expect(orc_route(l, T, N, K, 0.0, mode, rn, k, ids, w, NULL, NULL, NULL),
                               0, "orc_route (no optional outputs)");
                        expect(orc_dispatch(k, ids, T, N, K, cnt, off, rt, inv), 0,
                               "orc_dispatch");
                    }
                expect(orc_elbow_angle(l, T, N, 1e-8, e, th), 0, "orc_elbow_angle");
                for (int rn = 0; rn < 2; ++rn)
                    expect(orc_route_tail_random(l, r, T, N, K, 1e-8, rn, k, ids, w), 0,
                           "orc_route_tail_random");
            }
            /* probability rows: a softmax-free curve with ties and zeros */
            for (long t = 0; t < T; ++t) {
                double s = 0.0;
                for (int j = 0; j < N; ++j) {
                    double v = floor(uni() * 4.0);
                    p[t * N + j] = v;
                    s += v;
                }
                if (s == 0.0) p[t * N] = s = 1.0;
                for (int j = 0; j < N; ++j) p[t * N + j] /= s;
            }
            expect(orc_route_from_probs(p, T, N, K, 1e-8, 0, 0, k, ids, w, e, mg, comp), 0,
                   "orc_route_from_probs");
            expect(orc_route_from_probs(p, T, N, K, 1e-8, 1, 1, k, ids, w, NULL, NULL, NULL), 0,
                   "orc_route_from_probs (top-K, renormalised)");
            expect(orc_elbow_angle_from_probs(p, T, N, 1e-8, e, th), 0,
                   "orc_elbow_angle_from_probs");
            /* empty batch */
            expect(orc_route(l, 0, N, K, 1e-8, 0, 0, k, ids, w, e, mg, comp), 0, "orc_route T=0");
            expect(orc_dispatch(k, ids, 0, N, K, cnt, off, rt, inv), 0, "orc_dispatch T=0");
            /* an id outside [0, N) is reported */
            expect(orc_route(l, 1, N, K, 1e-8, 1, 0, k, ids, w, NULL, NULL, NULL), 0,
                   "orc_route T=1");
            ids[0] = N;
            expect(orc_dispatch(k, ids, 1, N, K, cnt, off, rt, inv), 1, "orc_dispatch bad id");
            free(k); free(ids); free(e); free(comp); free(w); free(mg); free(th);
            free(cnt); free(off); free(rt); free(inv);
        }
        /* invalid arguments and a row with no finite logit */
        int k1[1], id1[64], e1[1];
        double w1[64], th1[1];
        expect(orc_route(l, 1, N, 0, 1e-8, 0, 0, k1, id1, w1, NULL, NULL, NULL), 1, "K = 0");
        expect(orc_route(l, 1, N, N + 1, 1e-8, 0, 0, k1, id1, w1, NULL, NULL, NULL), 1, "K > N");
        expect(orc_route(l, 1, N, 1, -1.0, 0, 0, k1, id1, w1, NULL, NULL, NULL), 1, "eps < 0");
        expect(orc_route(l, 1, N, 1, 1e-8, 7, 0, k1, id1, w1, NULL, NULL, NULL), 1, "bad mode");
        for (int j = 0; j < N; ++j) l[j] = -INFINITY;
        expect(orc_route(l, 1, N, 1, 1e-8, 0, 0, k1, id1, w1, NULL, NULL, NULL), 2,
               "all -inf row");
        expect(orc_elbow_angle(l, 1, N, 1e-8, e1, th1) != 0, 1, "angle of an all -inf row");
        free(l); free(r); free(p);
    }
    float l1[1] = {0.f};
    int k1[1], id1[1];
    double w1[1];
    expect(orc_route(l1, 1, 1, 1, 1e-8, 0, 0, k1, id1, w1, NULL, NULL, NULL), 1, "N = 1");
}

static void layer_cases(void)
{
    const long T = 6;
    const int d = 16, N = 4, m = 8, K = 2;
    float *x = buf(T * d, sizeof(float)), *Wr = buf(N * d, sizeof(float));
    float *Wgu = buf((size_t)N * 2 * m * d, sizeof(float)), *Wd = buf((size_t)N * d * m, sizeof(float));
    float *res = buf(T * d, sizeof(float));
    for (long i = 0; i < T * d; ++i) { x[i] = (float)(uni() - 0.5); res[i] = (float)uni(); }
    for (long i = 0; i < (long)N * d; ++i) Wr[i] = (float)(uni() - 0.5);
    for (long i = 0; i < (long)N * 2 * m * d; ++i) Wgu[i] = (float)(uni() - 0.5);
    for (long i = 0; i < (long)N * d * m; ++i) Wd[i] = (float)(uni() - 0.5);
    double *lg = buf(T * N, sizeof(double));
    orc_router_logits(x, Wr, T, d, N, lg);
    orc_router_logits(x, Wr, 0, d, N, lg);
    const long tok[3] = {5, 0, 3};
    const long n_tok = 3;
    double *y = buf(n_tok * d, sizeof(double)), *lo = buf(n_tok * N, sizeof(double));
    double *w = buf(n_tok * K, sizeof(double)), *mg = buf(n_tok, sizeof(double));
    int *k = buf(n_tok, sizeof(int)), *ids = buf(n_tok * K, sizeof(int));
    for (int mode = 0; mode < 2; ++mode)
        for (int rn = 0; rn < 2; ++rn) {
            expect(orc_moe_forward(x, Wr, Wgu, Wd, res, T, d, N, m, K, 1e-8, mode, rn, tok,
                                   n_tok, y, lo, k, ids, w, mg), 0, "orc_moe_forward");
            expect(orc_moe_forward(x, Wr, Wgu, Wd, NULL, T, d, N, m, K, 1e-8, mode, rn, tok,
                                   n_tok, y, lo, k, ids, w, mg), 0,
                   "orc_moe_forward (no residual)");
            expect(orc_moe_experts(x, Wgu, Wd, res, T, d, N, m, K, tok, n_tok, k, ids, w, y), 0,
                   "orc_moe_experts");
        }
    expect(orc_moe_experts(x, Wgu, Wd, NULL, T, d, N, m, K, tok, 0, k, ids, w, y), 0,
           "orc_moe_experts n_tok=0");
    ids[0] = N;
    k[0] = K;
    expect(orc_moe_experts(x, Wgu, Wd, NULL, T, d, N, m, K, tok, n_tok, k, ids, w, y), 1,
           "orc_moe_experts bad id");
    free(x); free(Wr); free(Wgu); free(Wd); free(res); free(lg); free(y); free(lo); free(w);
    free(mg); free(k); free(ids);
}

int main(void)
{
    routing_cases();
    layer_cases();
    if (g_fail) return 1;
    printf("oracle sanitizer run: ok\n");
    return 0;
}
