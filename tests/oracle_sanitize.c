/*
 * Driver for a sanitized build of the CPU oracle (AddressSanitizer and UndefinedBehaviorSanitizer,
 * built and run by tests/test_oracle_sanitize.py).  It includes the oracle's single source file and
 * calls every exported function on small models with odd sizes (a 5-class head, non-power-of-two
 * dilations, one and two embedding taps, the bf16, int8 and approximate-nonlinearity modes, chunked
 * runs that resume a state, every sampling rule, the conditioning network), so that an
 * out-of-bounds access, a leak or undefined arithmetic anywhere on those paths ends the run with
 * a sanitizer report and a nonzero exit.
 */
#include <stdio.h>

#include "../oracle/wn_oracle.c"

static unsigned long long rng = 88172645463325252ull;
static float frand(void) { /* xorshift64, uniform in [-1, 1) */
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (float)((rng >> 11) * (1.0 / 9007199254740992.0)) * 2.0f - 1.0f;
}
static float *fill(size_t n, float scale) {
    float *p = malloc(sizeof(float) * (n ? n : 1));
    for (size_t i = 0; i < n; ++i) p[i] = scale * frand();
    return p;
}

static int run_model(int L, int r, int s, int a, const int *dil, int taps, int fmt, int ax) {
    oracle_model m;
    memset(&m, 0, sizeof(m));
    m.n_layers = L; m.r = r; m.s = s; m.a = a; m.dilations = dil; m.initial_sample = a / 2;
    m.weight_format = fmt; m.embed_taps = taps; m.approx_nonlin = ax;
    float *e = fill((size_t)taps * a * r, 0.5f), *be = fill(r, 0.1f), *wp = fill((size_t)L * 2 * r * r, 0.3f);
    float *wc = fill((size_t)L * 2 * r * r, 0.3f), *bg = fill((size_t)L * 2 * r, 0.1f);
    float *wr = fill((size_t)L * r * r, 0.3f), *br = fill((size_t)L * r, 0.1f), *wk = fill((size_t)L * s * r, 0.3f);
    float *bk = fill(s, 0.1f), *wl = fill((size_t)a * s, 0.3f), *bl = fill(a, 0.1f), *wo = fill((size_t)a * a, 0.3f);
    float *bo = fill(a, 0.1f);
    m.embed = e; m.b_embed = be; m.w_prev = wp; m.w_cur = wc; m.b_gate = bg; m.w_res = wr; m.b_res = br;
    m.w_skip = wk; m.b_skip = bk; m.w_relu = wl; m.b_relu = bl; m.w_out = wo; m.b_out = bo;
    const long long T = 23;
    float *cond = fill((size_t)T * L * 2 * r, 1.0f), *u = malloc(sizeof(float) * T);
    for (long long t = 0; t < T; ++t) u[t] = 0.5f * (frand() + 1.0f);
    int *ys = malloc(sizeof(int) * T), *yt = malloc(sizeof(int) * T);
    double *lg = malloc(sizeof(double) * T * a), *mg = malloc(sizeof(double) * T);
    int rc = oracle_run(&m, NULL, 0, T, cond, u, NULL, ys, lg, mg);
    if (rc == 0) rc = oracle_run(&m, NULL, 1, T, cond, u, ys, yt, lg, mg);
    /* a chunked run on an explicit state */
    oracle_state st;
    st.hist = malloc(sizeof(double) * (size_t)(oracle_history_len(&m) > 0 ? oracle_history_len(&m) : 1));
    oracle_reset(&m, &st);
    if (rc == 0) rc = oracle_run(&m, &st, 0, 7, cond, u, NULL, ys, lg, mg);
    if (rc == 0) rc = oracle_run(&m, &st, 0, T - 7, cond + 7 * L * 2 * r, u + 7, NULL, ys + 7, NULL, NULL);
    for (int mode = 0; mode <= 4 && rc == 0; ++mode)
        rc = oracle_run_sampled(&m, NULL, 0, T, cond, u, NULL, ys, lg, mg, mode, 0.7, a > 2 ? 3 : 1);
    for (int t = 0; t < T && rc == 0; ++t) {
        double p[512], margin;
        if (oracle_draw_nl(ax, a, lg + (size_t)t * a, u[t], p, &margin) < 0) rc = -3;
    }
    free(st.hist);
    free(e); free(be); free(wp); free(wc); free(bg); free(wr); free(br); free(wk); free(bk); free(wl); free(bl);
    free(wo); free(bo); free(cond); free(u); free(ys); free(yt); free(lg); free(mg);
    return rc;
}

static int run_conditioning(void) {
    oracle_cond_model c;
    c.n_features = 7; c.h1 = 5; c.h2 = 6;
    float *w1 = fill((size_t)2 * 3 * 5 * 2 * 7, 0.3f), *b1 = fill(2 * 3 * 5, 0.1f);
    float *w2 = fill((size_t)2 * 3 * 6 * 2 * 10, 0.3f), *b2 = fill(2 * 3 * 6, 0.1f);
    c.w1 = w1; c.b1 = b1; c.w2 = w2; c.b2 = b2;
    const long long Tf = 9, Ta = 9 * 16000 / 256;
    float *x = fill((size_t)Tf * 7, 1.0f);
    double *out = malloc(sizeof(double) * (size_t)Ta * 12);
    int rc = oracle_condition(&c, Tf, x, Ta, 256, 16000, out);
    if (rc == 0 && oracle_condition(&c, Tf, x, Ta + 100, 256, 16000, out) != -1) rc = -4; /* past the frames */
    free(w1); free(b1); free(w2); free(b2); free(x); free(out);
    return rc;
}

int main(void) {
    const int d4[] = {1, 2, 4, 8}, d3[] = {3, 1, 7}, d1[] = {1};
    int rc = 0;
    if (!rc) rc = run_model(4, 16, 32, 256, d4, 1, 0, 0);
    if (!rc) rc = run_model(3, 5, 7, 5, d3, 2, 0, 0);
    if (!rc) rc = run_model(3, 6, 4, 7, d3, 1, 1, 1);
    if (!rc) rc = run_model(1, 3, 2, 2, d1, 2, 1, 0);
    if (!rc) rc = run_model(3, 5, 7, 5, d3, 2, 2, 0);
    if (!rc) rc = run_model(4, 16, 32, 256, d4, 1, 2, 1);
    if (!rc) rc = run_conditioning();
    double xs[64], ys[64];
    for (int i = 0; i < 64; ++i) xs[i] = (i - 32) * 0.37;
    for (int which = 0; which < 3; ++which) oracle_approx_nonlin(which, xs, ys, 64);
    float f[5] = {1.0f, -0.0f, 3.4e38f, 1e-40f, 0.333f}, g[5];
    oracle_round_bf16_array(f, g, 5);
    float zrow[6] = {0, 0, 0, 1e-30f, -2.5f, 7.0f}, codes[6], sc[2];
    oracle_quantize_rows_i8(zrow, 2, 3, codes, sc);
    if (oracle_param_count(40, 64, 256, 256) != 1630528) rc = -5;
    printf("oracle sanitize driver: rc=%d\n", rc);
    return rc == 0 ? 0 : 1;
}
