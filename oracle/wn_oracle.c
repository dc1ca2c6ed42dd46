/*
 * CPU oracle for autoregressive WaveNet sample generation (Deep Voice,
 * arXiv 1702.07825).  TEST INFRASTRUCTURE ONLY: the GPU library never links,
 * loads or calls this file; only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg do.
 *
 * Plain, slow, sequential C in double precision.  It follows the equations of
 * the paper's Appendix A.1 ("Auto-regressive WaveNet") for one timestep, in the
 * per-layer order the paper's CPU-implementation section lists (sample
 * embedding, then per layer the two halves of the dilated convolution, the gated
 * activation, the residual 1x1 and the skip accumulation, then the two output
 * 1x1 convolutions and the softmax), and it keeps one history buffer per layer
 * so that nothing is recomputed (Section 5, "Optimizing Inference").
 *
 * Readings of the paper taken here:
 *  - residual: x^(j) = x^(j-1) + W_res h^(j) + B_res (appendix equation; the CPU
 *    section's x^(j) = W_res h^(j) + B_res is read as shorthand);
 *  - input embedding, one tap: x^(0)_t = E[y_{t-1}] + B_embed; two taps (the
 *    sample embedding of Section 5.1, the appendix's initial 2x1 convolution over
 *    the one-hot input): x^(0)_t = E_prev[y_{t-2}] + E_cur[y_{t-1}] + B_embed,
 *    where y_{t-2} at t = 0 lies before the input and contributes nothing (zero
 *    left padding, as for every layer's history);
 *  - every layer's history is zero before the first step (zero left padding);
 *    y_{-1} = initial_sample;
 *  - gate split: rows 0..r-1 of W_prev, W_cur, B and L feed tanh, rows r..2r-1
 *    feed the sigmoid;
 *  - skip: q^(0) = B_skip, q^(j) = q^(j-1) + W_skip^(j) h^(j), z_s = relu(q^(l));
 *  - direct sampling: y = min{k : u < C_k} with C_k = p_0 + ... + p_k and
 *    C_{a-1} taken as 1, i.e. y = #{k <= a-2 : C_k <= u}.  The decision is
 *    taken in fp32 (the precision of the paper's inference kernels): C_k is
 *    computed in double, rounded to float, and compared with the fp32 uniform.
 *    The margin min_k |u - C_k| (double, k <= a-2) is reported so that callers
 *    can tell which draws no rounding difference of a float implementation can
 *    change.
 *  - the other sampling rules (oracle_sample): top k keeps every class whose P
 *    is at least the k-th largest P (ties kept); the mean E_P[y] is taken to the
 *    nearest class index, halves up.
 *  - approximate nonlinearities (approx_nonlin = 1; Appendix C): the gate's tanh
 *    and sigmoid through e~(x) = 1 + |x| + 0.5658 x^2 + 0.143 x^4 as
 *    sign(x) (e~ - 1/e~) / (e~ + 1/e~) and e~ / (1 + e~) (x >= 0) or 1 / (1 + e~)
 *    (x < 0), and every e^x of the softmax and the sampling rules through the
 *    2^x bit pattern: y = x / ln 2, z = y - floor(y), the float whose bits are the
 *    integer part of (y + 126 + g(z)) 2^23 with g the appendix's rational fit of
 *    2^z - z; 0 where y <= -126 (the pattern has no exponent left);
 *  - bf16 weight storage: every matrix (W_prev, W_cur, W_res, W_skip, W_relu,
 *    W_out and the embedding table) is rounded to bfloat16 with round-to-
 *    nearest-even and used as the exact value of that bfloat16; biases stay fp32.
 *  - int8 weight storage (the paper stores int16 weights for its CPU kernels,
 *    Section 5.1, and names lower-precision weights as further work; it gives no
 *    scaling scheme): every matrix and the embedding table are stored per row
 *    as int8 codes with one fp32 scale, s = max|w| / 127 rounded to fp32 and
 *    code = round-half-even(w / s) (the quotient taken in double) in
 *    [-127, 127]; a zero row has s = 0 and zero codes.  The weight used is the
 *    exact product code * s; biases stay fp32.
 *
 * Layouts: every matrix is row-major [out][in]; conditioning is [T][l][2r].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int n_layers, r, s, a;
    const int *dilations;     /* [n_layers], each >= 1 */
    int initial_sample;       /* y_{-1} */
    int weight_format;        /* 0: the fp32 weights; 1: matrices rounded to bf16; 2: int8 codes
                                 with a per-row scale (see above) */
    int embed_taps;           /* 1 or 2 */
    int approx_nonlin;        /* 0: exact tanh, sigmoid, exp; 1: the approximations of Appendix C */
    const float *embed;       /* [taps][a][r]: the last tap embeds y_{t-1}, tap 0 of two y_{t-2} */
    const float *b_embed;     /* [r] */
    const float *w_prev;      /* [l][2r][r] */
    const float *w_cur;       /* [l][2r][r] */
    const float *b_gate;      /* [l][2r] */
    const float *w_res;       /* [l][r][r] */
    const float *b_res;       /* [l][r] */
    const float *w_skip;      /* [l][s][r] */
    const float *b_skip;      /* [s] */
    const float *w_relu;      /* [a][s] */
    const float *b_relu;      /* [a] */
    const float *w_out;       /* [a][a] */
    const float *b_out;       /* [a] */
} oracle_model;

/* Generator state of one stream: per-layer histories and the last sample. */
typedef struct {
    long long t;              /* steps already taken */
    int last_sample;          /* y_{t-1} */
    int prev_sample;          /* y_{t-2}, or -1 at t = 0 (no input before the first) */
    double *hist;             /* sum(d) * r doubles, layer j at offset r * sum_{i<j} d_i */
} oracle_state;

/* Round an fp32 value to bfloat16 (round to nearest, ties to even) and return it as float. */
static float round_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) { /* inf or nan: truncate, keep nan quiet */
        if (u & 0x007fffffu) u |= 0x00400000u;
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u = (u + 0x7fffu + lsb) & 0xffff0000u;
    }
    float g;
    memcpy(&g, &u, 4);
    return g;
}

float oracle_round_bf16(float f) { return round_bf16(f); }

/* int8 codes (as floats) and per-row scales of every matrix of a model, made at the start of a run
 * in weight format 2; NULL pointers in the other formats. */
typedef struct {
    float *embed, *w_prev, *w_cur, *w_res, *w_skip, *w_relu, *w_out;
    float *s_embed, *s_prev, *s_cur, *s_res, *s_skip, *s_relu, *s_out;
} oracle_i8;

/* Weight idx of a matrix whose rows hold `cols` inputs, as the model uses it: the fp32 value p[idx],
 * its bf16 rounding, or the product of its int8 code and its row's scale. */
static double wv(const oracle_model *m, const float *p, const float *codes, const float *scale, long cols, long idx) {
    if (m->weight_format == 2) return (double)codes[idx] * (double)scale[idx / cols];
    float f = p[idx];
    if (m->weight_format == 1) f = round_bf16(f);
    return (double)f;
}

/*
 * int8 codes of a row-major [rows][cols] matrix with one scale per row: s = max|w| / 127 rounded to
 * fp32, code = round-half-even(w / s) with the quotient in double, clamped to [-127, 127]; a row
 * of zeros gets s = 0 and codes 0.  The weight it stands for is code * s, exactly.
 */
void oracle_quantize_rows_i8(const float *w, long long rows, long long cols, float *codes, float *scale) {
    for (long long i = 0; i < rows; ++i) {
        const float *row = w + i * cols;
        double mx = 0.0;
        for (long long k = 0; k < cols; ++k)
            if (fabs((double)row[k]) > mx) mx = fabs((double)row[k]);
        const float sc = (float)(mx / 127.0);
        scale[i] = sc;
        for (long long k = 0; k < cols; ++k) {
            double c = sc > 0.0f ? nearbyint((double)row[k] / (double)sc) : 0.0;
            if (c > 127.0) c = 127.0;
            if (c < -127.0) c = -127.0;
            codes[i * cols + k] = (float)c;
        }
    }
}

static void free_i8(oracle_i8 *q) {
    free(q->embed); free(q->w_prev); free(q->w_cur); free(q->w_res); free(q->w_skip); free(q->w_relu); free(q->w_out);
    free(q->s_embed); free(q->s_prev); free(q->s_cur); free(q->s_res); free(q->s_skip); free(q->s_relu); free(q->s_out);
}

/* The int8 codes and scales of every matrix of m.  Returns 0, or -2 on allocation failure. */
static int make_i8(const oracle_model *m, oracle_i8 *q) {
    const long long L = m->n_layers, r = m->r, s = m->s, a = m->a, taps = m->embed_taps;
    struct { const float *w; long long rows, cols; float **codes, **scale; } mats[] = {
        {m->embed, taps * a, r, &q->embed, &q->s_embed},   {m->w_prev, L * 2 * r, r, &q->w_prev, &q->s_prev},
        {m->w_cur, L * 2 * r, r, &q->w_cur, &q->s_cur},    {m->w_res, L * r, r, &q->w_res, &q->s_res},
        {m->w_skip, L * s, r, &q->w_skip, &q->s_skip},     {m->w_relu, a, s, &q->w_relu, &q->s_relu},
        {m->w_out, a, a, &q->w_out, &q->s_out},
    };
    memset(q, 0, sizeof(*q));
    for (size_t i = 0; i < sizeof(mats) / sizeof(mats[0]); ++i) {
        *mats[i].codes = malloc(sizeof(float) * (size_t)(mats[i].rows * mats[i].cols));
        *mats[i].scale = malloc(sizeof(float) * (size_t)mats[i].rows);
        if (!*mats[i].codes || !*mats[i].scale) { free_i8(q); return -2; }
        oracle_quantize_rows_i8(mats[i].w, mats[i].rows, mats[i].cols, *mats[i].codes, *mats[i].scale);
    }
    return 0;
}

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* Appendix C: e~(x), a stand-in for e^|x| that gives good tanh and sigmoid values. */
static double e_tilde(double x) {
    const double a = fabs(x);
    return 1.0 + a + 0.5658 * x * x + 0.143 * x * x * x * x;
}
static double tanh_approx(double x) {
    const double e = e_tilde(x);
    const double t = (e - 1.0 / e) / (e + 1.0 / e);
    return x < 0.0 ? -t : (x > 0.0 ? t : 0.0);
}
static double sigmoid_approx(double x) {
    const double e = e_tilde(x);
    return x >= 0.0 ? e / (1.0 + e) : 1.0 / (1.0 + e);
}
/* Appendix C: e^x through the fp32 bit pattern of 2^(x / ln 2). */
static double exp_approx(double x) {
    const double y = x / log(2.0);
    if (y <= -126.0) return 0.0;
    const double z = y - floor(y);
    const double g = -4.7259162 + 27.7280233 / (4.84252568 - z) - 1.49012907 * z;
    const double v = (y + 126.0 + g) * 8388608.0;
    if (v >= 4294967295.0) return INFINITY;
    const uint32_t bits = (uint32_t)v;  /* integer part */
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}
static double tanh_nl(int ax, double x) { return ax ? tanh_approx(x) : tanh(x); }
static double sigmoid_nl(int ax, double x) { return ax ? sigmoid_approx(x) : sigmoid(x); }
static double exp_nl(int ax, double x) { return ax ? exp_approx(x) : exp(x); }

/* Array forms of the three approximations, for the tests that pin them. */
void oracle_approx_nonlin(int which, const double *x, double *out, long long n) {
    for (long long i = 0; i < n; ++i)
        out[i] = which == 0 ? tanh_approx(x[i]) : (which == 1 ? sigmoid_approx(x[i]) : exp_approx(x[i]));
}

long long oracle_history_len(const oracle_model *m) {
    long long n = 0;
    for (int j = 0; j < m->n_layers; ++j) n += m->dilations[j];
    return n * m->r;
}

void oracle_reset(const oracle_model *m, oracle_state *st) {
    st->t = 0;
    st->last_sample = m->initial_sample;
    st->prev_sample = -1;
    memset(st->hist, 0, sizeof(double) * (size_t)oracle_history_len(m));
}

/*
 * One timestep t of one stream: consumes y_{t-1} = st->last_sample (and, with two
 * embedding taps, y_{t-2} = st->prev_sample) and the conditioning of step t
 * ([l][2r]), writes the a = 256 logits of step t and advances the histories.
 * Returns 0 or -1 on allocation failure.
 */
static int oracle_step(const oracle_model *m, const oracle_i8 *q8, oracle_state *st, const float *cond_t,
                       double *logits) {
    const int L = m->n_layers, r = m->r, s = m->s, a = m->a;
    double *x = malloc(sizeof(double) * r), *xn = malloc(sizeof(double) * r);
    double *act = malloc(sizeof(double) * 2 * r), *h = malloc(sizeof(double) * r);
    double *q = malloc(sizeof(double) * s), *za = malloc(sizeof(double) * a);
    if (!x || !xn || !act || !h || !q || !za) {
        free(x); free(xn); free(act); free(h); free(q); free(za);
        return -1;
    }
    /* Sample embedding: x^(0) = E_cur[y_{t-1}] (+ E_prev[y_{t-2}]) + B_embed. */
    const long cur = (long)(m->embed_taps - 1) * a;  /* first row of the current tap's table */
    for (int c = 0; c < r; ++c) {
        x[c] = wv(m, m->embed, q8->embed, q8->s_embed, r, (cur + st->last_sample) * r + c) + (double)m->b_embed[c];
        if (m->embed_taps == 2 && st->prev_sample >= 0) x[c] += wv(m, m->embed, q8->embed, q8->s_embed, r, (long)st->prev_sample * r + c);
    }
    /* q^(0) = B_skip. */
    for (int k = 0; k < s; ++k) q[k] = (double)m->b_skip[k];

    long long hoff = 0;
    for (int j = 0; j < L; ++j) {
        const int d = m->dilations[j];
        double *slot = st->hist + hoff + (st->t % d) * r;   /* holds x^(j-1)_{t-d} */
        /* a = W_prev x_{t-d} + W_cur x_t + B + L  (the two halves of the width-2 dilated conv) */
        for (int o = 0; o < 2 * r; ++o) {
            double ap = 0.0, ac = 0.0;
            for (int c = 0; c < r; ++c) {
                ap += wv(m, m->w_prev, q8->w_prev, q8->s_prev, r, ((long)j * 2 * r + o) * r + c) * slot[c];
                ac += wv(m, m->w_cur, q8->w_cur, q8->s_cur, r, ((long)j * 2 * r + o) * r + c) * x[c];
            }
            act[o] = ap + ac + (double)m->b_gate[(long)j * 2 * r + o] + (double)cond_t[(long)j * 2 * r + o];
        }
        /* gated activation: h = tanh(a[0:r]) * sigmoid(a[r:2r]) */
        for (int c = 0; c < r; ++c) h[c] = tanh_nl(m->approx_nonlin, act[c]) * sigmoid_nl(m->approx_nonlin, act[r + c]);
        /* history: x^(j-1)_t replaces x^(j-1)_{t-d} (it is read again at t+d) */
        for (int c = 0; c < r; ++c) slot[c] = x[c];
        /* skip contribution: q += W_skip^(j) h */
        for (int k = 0; k < s; ++k) {
            double acc = 0.0;
            for (int c = 0; c < r; ++c) acc += wv(m, m->w_skip, q8->w_skip, q8->s_skip, r, ((long)j * s + k) * r + c) * h[c];
            q[k] += acc;
        }
        /* residual: x^(j) = x^(j-1) + W_res h + B_res */
        for (int o = 0; o < r; ++o) {
            double acc = 0.0;
            for (int c = 0; c < r; ++c) acc += wv(m, m->w_res, q8->w_res, q8->s_res, r, ((long)j * r + o) * r + c) * h[c];
            xn[o] = x[o] + acc + (double)m->b_res[(long)j * r + o];
        }
        memcpy(x, xn, sizeof(double) * r);
        hoff += (long long)d * r;
    }
    /* output: z_s = relu(q); z_a = relu(W_relu z_s + B_relu); logits = W_out z_a + B_out */
    for (int k = 0; k < s; ++k) q[k] = q[k] > 0.0 ? q[k] : 0.0;
    for (int i = 0; i < a; ++i) {
        double acc = 0.0;
        for (int k = 0; k < s; ++k) acc += wv(m, m->w_relu, q8->w_relu, q8->s_relu, s, (long)i * s + k) * q[k];
        acc += (double)m->b_relu[i];
        za[i] = acc > 0.0 ? acc : 0.0;
    }
    for (int i = 0; i < a; ++i) {
        double acc = 0.0;
        for (int k = 0; k < a; ++k) acc += wv(m, m->w_out, q8->w_out, q8->s_out, a, (long)i * a + k) * za[k];
        logits[i] = acc + (double)m->b_out[i];
    }
    free(x); free(xn); free(act); free(h); free(q); free(za);
    st->t += 1;
    return 0;
}

/*
 * Direct sampling from softmax(logits) with the uniform u (Appendix A.4,
 * "Sampling from Output Distribution": direct sampling; the softmax is the
 * max-subtracted form of the performance-model appendix).  Writes the
 * probabilities if prob != NULL and the margin if margin != NULL.
 */
static int draw_nl(int ax, int a, const double *logits, float u, double *prob, double *margin) {
    double mx = logits[0];
    for (int i = 1; i < a; ++i) if (logits[i] > mx) mx = logits[i];
    double z = 0.0;
    for (int i = 0; i < a; ++i) z += exp_nl(ax, logits[i] - mx);
    double cdf = 0.0, best = 1e300;
    int y = 0;
    for (int k = 0; k < a; ++k) {
        double p = exp_nl(ax, logits[k] - mx) / z;
        if (prob) prob[k] = p;
        cdf += p;
        if (k <= a - 2) {
            if ((float)cdf <= u) y += 1;
            double gap = fabs((double)u - cdf);
            if (gap < best) best = gap;
        }
    }
    if (margin) *margin = best;
    return y;
}

int oracle_draw(int a, const double *logits, float u, double *prob, double *margin) {
    return draw_nl(0, a, logits, u, prob, margin);
}

/* oracle_draw with the approximate exp of Appendix C when ax = 1. */
int oracle_draw_nl(int ax, int a, const double *logits, float u, double *prob, double *margin) {
    return draw_nl(ax, a, logits, u, prob, margin);
}

/*
 * The other ways of using the output distribution that the paper lists beside
 * direct sampling (Appendix A.4, "Sampling from Output Distribution"), each
 * taken from its definition there:
 *   mode 0  direct:       draw from P                      (oracle_draw above)
 *   mode 1  temperature:  draw from P^(1/t) / Z, i.e. from softmax(logits / t)
 *   mode 2  top k:        draw from P restricted to the classes whose P is at
 *                         least the k-th largest P (ties at the k-th are kept),
 *                         renormalised; P is ordered as the logits are
 *   mode 3  mode:         argmax P (the smallest index among equal maxima)
 *   mode 4  mean:         E_P[y] = sum_k k P(k), taken to the nearest class
 *                         index (halves go up); the paper gives no rounding
 * A draw is an inverse CDF as in oracle_draw: y = #{k <= a-2 : C_k <= u} with
 * the CDF rounded to float, where C_k sums the distribution actually sampled.
 * *margin receives how far the result is from changing: the distance of u from
 * the nearest C_k (modes 0-2), also the gap between the k-th and (k+1)-th
 * largest logits (mode 2, k < a), the gap between the two largest logits
 * (mode 3), or the distance of the mean from the nearest half-integer (mode 4).
 * Returns the index, or -1 for an invalid mode, temperature or k.
 */
static int sample_nl(int ax, int a, const double *logits, float u, int mode, double temperature, int top_k,
                     double *margin) {
    if (mode == 0) return draw_nl(ax, a, logits, u, NULL, margin);
    if (mode < 0 || mode > 4 || (mode == 1 && !(temperature > 0.0)) || (mode == 2 && (top_k < 1 || top_k > a)))
        return -1;
    double *w = malloc(sizeof(double) * (size_t)a);
    if (!w) return -1;
    int y = 0;
    double best = 1e300;
    if (mode == 3) {
        for (int k = 1; k < a; ++k) if (logits[k] > logits[y]) y = k;
        for (int k = 0; k < a; ++k) {
            double gap = logits[y] - logits[k];
            if (k != y && gap < best) best = gap;
        }
    } else {
        /* weights proportional to the distribution sampled */
        double mx = -1e300;
        for (int k = 0; k < a; ++k) {
            double v = (mode == 1) ? logits[k] / temperature : logits[k];
            if (v > mx) mx = v;
        }
        for (int k = 0; k < a; ++k) w[k] = exp_nl(ax, ((mode == 1) ? logits[k] / temperature : logits[k]) - mx);
        int last_kept = a - 1;
        if (mode == 2) {
            /* the k-th largest logit, by selection over a sorted copy */
            double *srt = malloc(sizeof(double) * (size_t)a);
            if (!srt) { free(w); return -1; }
            memcpy(srt, logits, sizeof(double) * (size_t)a);
            for (int i = 1; i < a; ++i) {  /* insertion sort, descending */
                double v = srt[i];
                int j = i - 1;
                while (j >= 0 && srt[j] < v) { srt[j + 1] = srt[j]; --j; }
                srt[j + 1] = v;
            }
            const double kth = srt[top_k - 1];
            if (top_k < a) best = kth - srt[top_k];
            free(srt);
            for (int k = 0; k < a; ++k) if (logits[k] < kth) w[k] = 0.0;
            while (last_kept > 0 && w[last_kept] == 0.0) --last_kept;
        }
        double z = 0.0;
        for (int k = 0; k < a; ++k) z += w[k];
        if (mode == 4) {
            double mean = 0.0;
            for (int k = 0; k < a; ++k) mean += (double)k * (w[k] / z);
            y = (int)floor(mean + 0.5);
            if (y > a - 1) y = a - 1;
            best = fabs(mean - (floor(mean) + 0.5));
        } else {
            double cdf = 0.0;
            for (int k = 0; k < a; ++k) {
                cdf += w[k] / z;
                if (k <= a - 2) {
                    if ((float)cdf <= u) y += 1;
                    double gap = fabs((double)u - cdf);
                    if (gap < best) best = gap;
                }
            }
            if (y > last_kept) y = last_kept;  /* only by rounding: C at the last kept class is 1 */
        }
    }
    free(w);
    if (margin) *margin = best;
    return y;
}

int oracle_sample(int a, const double *logits, float u, int mode, double temperature, int top_k, double *margin) {
    return sample_nl(0, a, logits, u, mode, temperature, top_k, margin);
}

/* oracle_sample with the approximate exp of Appendix C when ax = 1. */
int oracle_sample_nl(int ax, int a, const double *logits, float u, int mode, double temperature, int top_k,
                     double *margin) {
    return sample_nl(ax, a, logits, u, mode, temperature, top_k, margin);
}

/*
 * Run T steps of one stream.
 *   mode 0 (generate): y_{t} is drawn from step t's distribution with u[t] and
 *                      fed back; samples_out[t] receives it.
 *   mode 1 (teacher forcing): step t consumes y_in[t-1] (y_in[-1] is the state's
 *                      last sample); samples_out, if given, receives the draw that
 *                      u[t] would make from step t's distribution.
 * Draws follow oracle_sample's rule (sample_mode, temperature, top_k); margin_out
 * receives its margins.  logits_out [T][a] (double), margin_out [T] may be NULL.
 * u may be NULL in mode 1.  If st is NULL a fresh zero state is used.  Returns
 * 0, -1 (bad arguments) or -2 (allocation failure).
 */
int oracle_run_sampled(const oracle_model *m, oracle_state *st, int mode, long long T,
                       const float *cond, const float *u, const int *y_in,
                       int *samples_out, double *logits_out, double *margin_out,
                       int sample_mode, double temperature, int top_k) {
    if (!m || T < 0 || (mode != 0 && mode != 1) || m->embed_taps < 1 || m->embed_taps > 2 ||
        (m->approx_nonlin != 0 && m->approx_nonlin != 1) || m->weight_format < 0 || m->weight_format > 2)
        return -1;
    if (mode == 0 && !u) return -1;
    if (mode == 1 && !y_in) return -1;
    oracle_state local;
    double *own = NULL;
    if (!st) {
        own = malloc(sizeof(double) * (size_t)(oracle_history_len(m) > 0 ? oracle_history_len(m) : 1));
        if (!own) return -2;
        local.hist = own;
        oracle_reset(m, &local);
        st = &local;
    }
    double *lg = malloc(sizeof(double) * m->a);
    if (!lg) { free(own); return -2; }
    oracle_i8 q8;
    memset(&q8, 0, sizeof(q8));
    if (m->weight_format == 2 && make_i8(m, &q8) != 0) { free(lg); free(own); return -2; }
    const long long per_step = (long long)m->n_layers * 2 * m->r;
    for (long long t = 0; t < T; ++t) {
        if (oracle_step(m, &q8, st, cond + t * per_step, lg) != 0) { free(lg); free(own); free_i8(&q8); return -2; }
        if (logits_out) memcpy(logits_out + t * m->a, lg, sizeof(double) * m->a);
        int y = 0;
        double mg = 0.0;
        if (u) y = sample_nl(m->approx_nonlin, m->a, lg, u[t], sample_mode, temperature, top_k, &mg);
        if (y < 0) { free(lg); free(own); free_i8(&q8); return -1; }
        if (margin_out) margin_out[t] = u ? mg : 0.0;
        if (samples_out) samples_out[t] = y;
        st->prev_sample = st->last_sample;
        st->last_sample = (mode == 0) ? y : y_in[t];
    }
    free(lg);
    free(own);
    free_i8(&q8);
    return 0;
}

/* oracle_run_sampled with direct sampling. */
int oracle_run(const oracle_model *m, oracle_state *st, int mode, long long T,
               const float *cond, const float *u, const int *y_in,
               int *samples_out, double *logits_out, double *margin_out) {
    return oracle_run_sampled(m, st, mode, T, cond, u, y_in, samples_out, logits_out, margin_out, 0, 1.0, m ? m->a : 0);
}

/* Number of parameters of the layout above (the paper's model-size estimate). */
long long oracle_param_count(int n_layers, int r, int s, int a) {
    long long L = n_layers;
    long long per_layer = 2LL * (2 * r) * r + 2 * r + (long long)r * r + r + (long long)s * r;
    return (long long)a * r + r + L * per_layer + s + (long long)a * s + a + (long long)a * a + a;
}

/* FLOPs per generated sample, the performance-model appendix's final equation. */
double oracle_flops_per_sample(int n_layers, int r, int s, int a, double f_div, double f_exp) {
    double L = n_layers, R = r, S = s, A = a;
    return L * (10.0 * R * R + 11.0 * R + 2.0 * R * (f_div + f_exp)) + S * (2.0 * R * L + 2.0) +
           A * (2.0 * S + 2.0 * A + 3.0) + A * (3.0 + f_div + f_exp);
}

/* Vector form of the bf16 rounding above. */
void oracle_round_bf16_array(const float *in, float *out, long long n) {
    for (long long i = 0; i < n; ++i) out[i] = round_bf16(in[i]);
}

/*
 * Conditioning network (Appendix A.2, "Conditioning Network"): the per-layer
 * conditioning L of every audio step from linguistic features at the frame
 * rate.  Two bidirectional QRNN layers with fo-pooling and width-2
 * convolutions, then the channels of the two directions interleaved, then
 * upsampling to the audio rate by repetition.  A unidirectional layer computes,
 * over the frames in its own order,
 *     h~_t = tanh(W_h * x + B_h), o_t = sigma(W_o * x + B_o), f_t = sigma(W_f * x + B_f)
 *     h_t  = f_t h_{t-1} + (1 - f_t) h~_t   (h before the first frame is 0)
 *     z_t  = o_t h_t
 * where W * x is the width-2 convolution over [x_{t'}, x_t], t' the frame before
 * t in that order (zero before the first).  The backward layer runs on the
 * reversed frames, so its previous frame is t + 1.  Readings taken here: the
 * convolution is causal in each direction's own order; the bidirectional output
 * stacks forward then backward channels; after the second layer output channel
 * 2k + d is channel k of direction d, and the 2 h2 = l * 2r channels of an audio
 * step are layer j's L in block j; audio step tau repeats frame
 * floor(tau * frame_rate / audio_rate).
 */
typedef struct {
    int n_features;     /* F */
    int h1, h2;         /* channels per direction of layer 1 and layer 2 */
    const float *w1;    /* [2][3 h1][2][F]: direction, gate row (blocks h~, o, f), tap (0: previous frame, 1: current), input */
    const float *b1;    /* [2][3 h1] */
    const float *w2;    /* [2][3 h2][2][2 h1] */
    const float *b2;    /* [2][3 h2] */
} oracle_cond_model;

/* One bidirectional QRNN layer over T frames of `in` channels: out [T][2h], forward channels first. */
static void oracle_qrnn_layer(long long T, int in, int h, const double *x, const float *w, const float *b,
                              double *out) {
    for (int dir = 0; dir < 2; ++dir) {
        const float *wd = w + (size_t)dir * 3 * h * 2 * in;
        const float *bd = b + (size_t)dir * 3 * h;
        for (int k = 0; k < h; ++k) {
            double hprev = 0.0;
            for (long long s = 0; s < T; ++s) {
                const long long t = dir == 0 ? s : T - 1 - s;
                const long long tp = dir == 0 ? t - 1 : t + 1;
                double a[3];
                for (int gt = 0; gt < 3; ++gt) {
                    const float *row = wd + (size_t)(gt * h + k) * 2 * in;
                    double acc = bd[gt * h + k];
                    if (tp >= 0 && tp < T)
                        for (int i = 0; i < in; ++i) acc += (double)row[i] * x[(size_t)tp * in + i];
                    for (int i = 0; i < in; ++i) acc += (double)row[in + i] * x[(size_t)t * in + i];
                    a[gt] = acc;
                }
                const double ht = tanh(a[0]), o = sigmoid(a[1]), f = sigmoid(a[2]);
                const double hc = f * hprev + (1.0 - f) * ht;
                out[(size_t)t * 2 * h + (size_t)dir * h + k] = o * hc;
                hprev = hc;
            }
        }
    }
}

/*
 * cond [Ta][2 h2] (double) from features [Tf][F].  Returns 0, -1 (bad
 * arguments, or an audio step past the last frame) or -2 (allocation failure).
 */
int oracle_condition(const oracle_cond_model *m, long long Tf, const float *features, long long Ta,
                     int frame_rate, int audio_rate, double *cond) {
    if (!m || Tf < 1 || Ta < 0 || frame_rate < 1 || audio_rate < 1 || m->n_features < 1 || m->h1 < 1 || m->h2 < 1)
        return -1;
    if (Ta > 0 && (Ta - 1) * (long long)frame_rate / audio_rate >= Tf) return -1;
    const int F = m->n_features, h1 = m->h1, h2 = m->h2;
    double *x = malloc(sizeof(double) * (size_t)Tf * F);
    double *z1 = malloc(sizeof(double) * (size_t)Tf * 2 * h1);
    double *z2 = malloc(sizeof(double) * (size_t)Tf * 2 * h2);
    if (!x || !z1 || !z2) { free(x); free(z1); free(z2); return -2; }
    for (long long i = 0; i < Tf * F; ++i) x[i] = features[i];
    oracle_qrnn_layer(Tf, F, h1, x, m->w1, m->b1, z1);
    oracle_qrnn_layer(Tf, 2 * h1, h2, z1, m->w2, m->b2, z2);
    for (long long tau = 0; tau < Ta; ++tau) {
        const long long t = tau * (long long)frame_rate / audio_rate;
        for (int k = 0; k < h2; ++k)
            for (int dir = 0; dir < 2; ++dir)
                cond[(size_t)tau * 2 * h2 + 2 * k + dir] = z2[(size_t)t * 2 * h2 + (size_t)dir * h2 + k];
    }
    free(x); free(z1); free(z2);
    return 0;
}
