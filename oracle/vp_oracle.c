/*
 * vp_oracle.c -- fp64 CPU oracle of the VGGT-Prime routed global-attention
 * layer.  TEST INFRASTRUCTURE ONLY: this code is the parity reference for the
 * GPU library and is used only by the tests, the smoke check and the CPU
 * baseline timing of the benchmark.  It shares no code with the GPU path.
 *
 * Everything is computed in double precision from the stored input values
 * (fp32 arrays; bf16 inputs are widened exactly before they arrive here),
 * straight from the definitions, with no tiling and no online softmax.
 * Threads only split independent work (rows, heads); every reduction runs
 * serially in index order, so results are deterministic.
 *
 * Layouts: Q, K, V are [N, H, d] row-major, N = S * P tokens of all views;
 * the row of head h for token i starts at (i * H + h) * d.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define OR_MODE_MEAN 0
#define OR_MODE_SURR 1
#define OR_MODE_FULL 2

/* ---------------------------------------------------------------- threads */

typedef void (*or_body)(void *ctx, int64_t lo, int64_t hi);
typedef struct {
    or_body body;
    void *ctx;
    int64_t lo, hi;
} or_chunk;

static void *or_thread_main(void *p) {
    or_chunk *c = (or_chunk *)p;
    if (c->lo < c->hi) c->body(c->ctx, c->lo, c->hi);
    return NULL;
}

static int or_nthreads(int requested) {
    if (requested > 0) return requested;
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

/* Run body over [0, n) split into contiguous chunks, one per thread. */
static void or_parallel_for(int64_t n, int nthreads, or_body body, void *ctx) {
    int T = or_nthreads(nthreads);
    if (T > n) T = (int)(n > 0 ? n : 1);
    if (T <= 1) {
        if (n > 0) body(ctx, 0, n);
        return;
    }
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * T);
    or_chunk *ch = (or_chunk *)malloc(sizeof(or_chunk) * T);
    for (int t = 0; t < T; ++t) {
        ch[t].body = body;
        ch[t].ctx = ctx;
        ch[t].lo = n * t / T;
        ch[t].hi = n * (t + 1) / T;
        pthread_create(&th[t], NULL, or_thread_main, &ch[t]);
    }
    for (int t = 0; t < T; ++t) pthread_join(th[t], NULL);
    free(th);
    free(ch);
}

int or_threads_used(int requested) { return or_nthreads(requested); }

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* ------------------------------------------------ router pooling (Eq.1-2) */
/*
 * Gated attention pooling of the queries of head h (Section 4.1, Eq.1, a
 * pooling module from attention-based multiple-instance learning):
 *   a_{h,i} = sum_l w_h[l] * tanh((W_h q_{h,i})_l) * sigmoid((U_h q_{h,i})_l)
 *   alpha_h = softmax over all N tokens of a_h
 *   q_pool_h = sum_i alpha_{h,i} q_{h,i}                               (Eq.2)
 * W_h, U_h are [L, d]; w_h is [L]; no biases appear in Eq.1.
 */
typedef struct {
    const float *Q, *W, *U, *w;
    int64_t N;
    int H, d, L;
    double *a; /* [H, N] */
} pool_ctx;

static void pool_logits_body(void *p, int64_t lo, int64_t hi) {
    pool_ctx *c = (pool_ctx *)p;
    for (int64_t idx = lo; idx < hi; ++idx) {
        int h = (int)(idx / c->N);
        int64_t i = idx % c->N;
        const float *q = c->Q + (i * c->H + h) * (int64_t)c->d;
        const float *Wh = c->W + (int64_t)h * c->L * c->d;
        const float *Uh = c->U + (int64_t)h * c->L * c->d;
        const float *wh = c->w + (int64_t)h * c->L;
        double a = 0.0;
        for (int l = 0; l < c->L; ++l) {
            double x = 0.0, y = 0.0;
            for (int k = 0; k < c->d; ++k) {
                x += (double)Wh[l * c->d + k] * (double)q[k];
                y += (double)Uh[l * c->d + k] * (double)q[k];
            }
            a += (double)wh[l] * tanh(x) * sigmoid(y);
        }
        c->a[(int64_t)h * c->N + i] = a;
    }
}

/* q_pool [H, d]; optional a_out / alpha_out [H, N] (pre-softmax logits, weights). */
void or_router_pool(const float *Q, int64_t N, int H, int d, int L, const float *W,
                    const float *U, const float *w, double *q_pool, double *a_out,
                    double *alpha_out, int nthreads) {
    double *a = (double *)malloc(sizeof(double) * (size_t)N * H);
    pool_ctx c = {Q, W, U, w, N, H, d, L, a};
    or_parallel_for(N * H, nthreads, pool_logits_body, &c);
    for (int h = 0; h < H; ++h) {
        const double *ah = a + (int64_t)h * N;
        double mx = -INFINITY;
        for (int64_t i = 0; i < N; ++i)
            if (ah[i] > mx) mx = ah[i];
        double sum = 0.0;
        for (int64_t i = 0; i < N; ++i) sum += exp(ah[i] - mx);
        double *qp = q_pool + (int64_t)h * d;
        for (int k = 0; k < d; ++k) qp[k] = 0.0;
        for (int64_t i = 0; i < N; ++i) {
            double alpha = exp(ah[i] - mx) / sum;
            if (alpha_out) alpha_out[(int64_t)h * N + i] = alpha;
            const float *q = Q + (i * H + h) * (int64_t)d;
            for (int k = 0; k < d; ++k) qp[k] += alpha * (double)q[k];
        }
        if (a_out) memcpy(a_out + (int64_t)h * N, ah, sizeof(double) * N);
    }
    free(a);
}

/* --------------------------- single-query attention and saliency (Eq.3) */
/*
 * The pooled query attends over all N keys of all views (Section 4.1):
 *   t_{h,j} = scale * (q_pool_h . k_{h,j}),   r_h = softmax_j(t_h)
 *   s_h = max_j r_h(j)                                                 (Eq.3)
 * and, reusing r_h (Section 4.3, Eq.5; Algorithm 1 mean branch):
 *   C_h = r_h V_h,     mean_h = (1/N) sum_j v_{h,j}
 */
typedef struct {
    const float *K, *V;
    int64_t N;
    int H, d;
    const double *q_pool;
    double scale;
    double *r_out, *s, *C, *mean;
} route_ctx;

static void route_body(void *p, int64_t lo, int64_t hi) {
    route_ctx *c = (route_ctx *)p;
    int64_t N = c->N;
    int H = c->H, d = c->d;
    double *t = (double *)malloc(sizeof(double) * N);
    for (int64_t h = lo; h < hi; ++h) {
        const double *qp = c->q_pool + h * d;
        for (int64_t j = 0; j < N; ++j) {
            const float *k = c->K + (j * H + h) * (int64_t)d;
            double dot = 0.0;
            for (int e = 0; e < d; ++e) dot += qp[e] * (double)k[e];
            t[j] = c->scale * dot;
        }
        double mx = -INFINITY;
        for (int64_t j = 0; j < N; ++j)
            if (t[j] > mx) mx = t[j];
        double sum = 0.0;
        for (int64_t j = 0; j < N; ++j) sum += exp(t[j] - mx);
        double smax = 0.0;
        double *C = c->C + h * d, *mean = c->mean + h * d;
        for (int e = 0; e < d; ++e) C[e] = mean[e] = 0.0;
        for (int64_t j = 0; j < N; ++j) {
            double r = exp(t[j] - mx) / sum;
            if (c->r_out) c->r_out[h * N + j] = r;
            if (r > smax) smax = r;
            const float *v = c->V + (j * H + h) * (int64_t)d;
            for (int e = 0; e < d; ++e) {
                C[e] += r * (double)v[e];
                mean[e] += (double)v[e];
            }
        }
        for (int e = 0; e < d; ++e) mean[e] /= (double)N;
        c->s[h] = smax;
    }
    free(t);
}

void or_router_route(const float *K, const float *V, int64_t N, int H, int d,
                     const double *q_pool, double scale, double *r_out, double *s,
                     double *C, double *mean, int nthreads) {
    route_ctx c = {K, V, N, H, d, q_pool, scale, r_out, s, C, mean};
    or_parallel_for(H, nthreads, route_body, &c);
}

/* ------------------------------------------------ linear-logit mode router */
/*
 * Mode router of the synthetic workloads (not a construct of the paper): a
 * linear map of a 1024-vector to H*3 logits, logits[r] = W_r[r] . u + b_r[r],
 * row r = h * 3 + m with m in (MEAN, SURR, FULL).
 */
void or_router_logits(const float *u, const float *Wr, const float *br, int R, int Din,
                      double *logits) {
    for (int r = 0; r < R; ++r) {
        double acc = 0.0;
        for (int c = 0; c < Din; ++c) acc += (double)Wr[(int64_t)r * Din + c] * (double)u[c];
        logits[r] = acc + (double)br[r];
    }
}

/* --------------------------------------------------- mode assignment (Eq.4) */
/*
 * rule 0 (threshold, Eq.4): FULL if s >= tau_high; MEAN if s <= tau_low;
 *   SURR strictly between.  The thresholds arrive as fp32 and are widened.
 * rule 1 (argmax over the three logits of a head): the first maximal index.
 * rules 2 and 3: the two-branch ablation of the compute-mode study (no
 *   surrogate, only mean pooling and full attention): rule 2 is FULL if
 *   s >= tau_high, else MEAN; rule 3 compares only the MEAN and FULL logits,
 *   MEAN on a tie.
 * A NaN score sends the head to FULL (the paper is silent; FULL is exact).
 */
void or_assign(const double *scores, int H, int rule, float tau_low, float tau_high,
               uint8_t *modes) {
    for (int h = 0; h < H; ++h) {
        if (rule == 0 || rule == 2) {
            double s = scores[h];
            if (isnan(s) || s >= (double)tau_high)
                modes[h] = OR_MODE_FULL;
            else if (rule == 2 || s <= (double)tau_low)
                modes[h] = OR_MODE_MEAN;
            else
                modes[h] = OR_MODE_SURR;
        } else if (rule == 1) {
            const double *lg = scores + (int64_t)h * 3;
            int best = 0, bad = isnan(lg[0]);
            for (int m = 1; m < 3; ++m) {
                if (isnan(lg[m])) bad = 1;
                if (lg[m] > lg[best]) best = m;
            }
            modes[h] = bad ? OR_MODE_FULL : (uint8_t)best;
        } else {
            const double *lg = scores + (int64_t)h * 3;
            const double mean_l = lg[OR_MODE_MEAN], full_l = lg[OR_MODE_FULL];
            if (isnan(mean_l) || isnan(full_l))
                modes[h] = OR_MODE_FULL;
            else
                modes[h] = full_l > mean_l ? OR_MODE_FULL : OR_MODE_MEAN;
        }
    }
}

/* --------------------------------------------- FULL mode (Algorithm 1, eq) */
/*
 * Exact softmax attention of head h over all N tokens of all views
 * (Algorithm 1, first branch): for query row i,
 *   l_j = (q_{h,i} . k_{h,j}) * scale,  p = softmax(l),  y_i = sum_j p_j v_{h,j}
 * Two passes per row (max, then exponentials), scale = 1/sqrt(d).
 */
typedef struct {
    const float *Q, *K, *V;
    int64_t N;
    int H, d, h;
    const int64_t *rows;
    double scale;
    double *Y;
} full_ctx;

static void full_body(void *p, int64_t lo, int64_t hi) {
    full_ctx *c = (full_ctx *)p;
    int64_t N = c->N;
    int H = c->H, d = c->d, h = c->h;
    double *l = (double *)malloc(sizeof(double) * N);
    for (int64_t r = lo; r < hi; ++r) {
        int64_t i = c->rows ? c->rows[r] : r;
        const float *q = c->Q + (i * H + h) * (int64_t)d;
        double mx = -INFINITY;
        for (int64_t j = 0; j < N; ++j) {
            const float *k = c->K + (j * H + h) * (int64_t)d;
            double dot = 0.0;
            for (int e = 0; e < d; ++e) dot += (double)q[e] * (double)k[e];
            l[j] = dot * c->scale;
            if (l[j] > mx) mx = l[j];
        }
        double sum = 0.0;
        double *y = c->Y + r * d;
        for (int e = 0; e < d; ++e) y[e] = 0.0;
        for (int64_t j = 0; j < N; ++j) {
            double pj = exp(l[j] - mx);
            sum += pj;
            const float *v = c->V + (j * H + h) * (int64_t)d;
            for (int e = 0; e < d; ++e) y[e] += pj * (double)v[e];
        }
        for (int e = 0; e < d; ++e) y[e] /= sum;
    }
    free(l);
}

/* Y [nrows, d]; rows == NULL means rows 0..nrows-1. */
void or_full_rows(const float *Q, const float *K, const float *V, int64_t N, int H, int d,
                  int h, const int64_t *rows, int64_t nrows, double scale, double *Y,
                  int nthreads) {
    full_ctx c = {Q, K, V, N, H, d, h, rows, scale, Y};
    or_parallel_for(nrows, nthreads, full_body, &c);
}

/* --------------------------------------- SURR mode (Section 4.3, Eq.5-7) */
/*
 * Learned surrogate attention of head h for token i:
 *   z = [v_{h,i}; C_h]                       (value first, then context)
 *   gamma = sigmoid(MLP_gamma(z)),  delta = MLP_delta(z)               (Eq.6)
 *   y_i = C_h + gamma (.) delta                                        (Eq.7)
 * Each MLP is Linear(2d -> L) -> act -> Linear(L -> d), with biases;
 * act 0 = GELU (erf form), act 1 = ReLU.  w1 is [L, 2d], w2 is [d, L].
 * variant 0: Eq.7 as above; 2: the "no residual" ablation of the component
 * study, y_i = C_h; 3: identity added, y_i = v_{h,i} + C_h + gamma (.) delta.
 * (The "mean context" ablation is variant 0 with C_h replaced by the value
 * mean, done by the caller.)
 */
typedef struct {
    const float *V;
    int64_t N;
    int H, d, h, L, act, variant;
    const double *C;
    const float *gw1, *gb1, *gw2, *gb2, *dw1, *db1, *dw2, *db2;
    const int64_t *rows;
    double *Y;
} surr_ctx;

static double act_fn(double x, int act) {
    if (act == 1) return x > 0.0 ? x : 0.0;
    return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
}

static void mlp(const double *z, int din, int L, int dout, const float *w1, const float *b1,
                const float *w2, const float *b2, int act, double *hid, double *out) {
    for (int l = 0; l < L; ++l) {
        double acc = (double)b1[l];
        for (int c = 0; c < din; ++c) acc += (double)w1[(int64_t)l * din + c] * z[c];
        hid[l] = act_fn(acc, act);
    }
    for (int k = 0; k < dout; ++k) {
        double acc = (double)b2[k];
        for (int l = 0; l < L; ++l) acc += (double)w2[(int64_t)k * L + l] * hid[l];
        out[k] = acc;
    }
}

static void surr_body(void *p, int64_t lo, int64_t hi) {
    surr_ctx *c = (surr_ctx *)p;
    int d = c->d, L = c->L;
    double *z = (double *)malloc(sizeof(double) * (2 * d + 2 * L + 2 * d));
    double *hid = z + 2 * d, *g = hid + L, *dl = g + d;
    for (int64_t r = lo; r < hi; ++r) {
        int64_t i = c->rows ? c->rows[r] : r;
        const float *v = c->V + (i * c->H + c->h) * (int64_t)d;
        for (int e = 0; e < d; ++e) {
            z[e] = (double)v[e];
            z[d + e] = c->C[e];
        }
        double *y = c->Y + r * d;
        if (c->variant == 2) {   /* no residual correction: the context alone */
            for (int e = 0; e < d; ++e) y[e] = c->C[e];
            continue;
        }
        mlp(z, 2 * d, L, d, c->gw1, c->gb1, c->gw2, c->gb2, c->act, hid, g);
        mlp(z, 2 * d, L, d, c->dw1, c->db1, c->dw2, c->db2, c->act, hid, dl);
        for (int e = 0; e < d; ++e) {
            y[e] = c->C[e] + sigmoid(g[e]) * dl[e];
            if (c->variant == 3) y[e] += z[e];   /* identity added: v + Eq.7 */
        }
    }
    free(z);
}

/* Weights passed for head h only (already offset by the caller). */
void or_surr_rows(const float *V, int64_t N, int H, int d, int h, int L, int act, int variant,
                  const double *C_h, const float *gw1, const float *gb1, const float *gw2,
                  const float *gb2, const float *dw1, const float *db1, const float *dw2,
                  const float *db2, const int64_t *rows, int64_t nrows, double *Y,
                  int nthreads) {
    surr_ctx c = {V, N, H, d, h, L, act, variant, C_h, gw1, gb1, gw2, gb2, dw1, db1, dw2, db2,
                  rows, Y};
    or_parallel_for(nrows, nthreads, surr_body, &c);
}

/* ------------------------------------- linear attention (compute-mode study) */
/*
 * The linear-attention alternative to the surrogate that the compute-mode
 * ablation evaluates (the kernelised attention of Katharopoulos et al.,
 * with its feature map phi(x) = elu(x) + 1): for query row i of head h,
 *   w_j = phi(q_{h,i}) . phi(k_{h,j}),  y_i = sum_j w_j v_{h,j} / sum_j w_j
 * over all N tokens of all views (non-causal), computed from this definition
 * row by row (no factorisation).
 */
typedef struct {
    const float *Q, *K, *V;
    int64_t N;
    int H, d, h;
    const int64_t *rows;
    double *Y;
} lin_ctx;

static double elu1(double x) { return x > 0.0 ? x + 1.0 : exp(x); }

static void lin_body(void *p, int64_t lo, int64_t hi) {
    lin_ctx *c = (lin_ctx *)p;
    const int d = c->d;
    double *fq = (double *)malloc(sizeof(double) * 2 * d);
    double *acc = fq + d;
    for (int64_t r = lo; r < hi; ++r) {
        const int64_t i = c->rows ? c->rows[r] : r;
        const float *q = c->Q + (i * c->H + c->h) * (int64_t)d;
        for (int e = 0; e < d; ++e) {
            fq[e] = elu1((double)q[e]);
            acc[e] = 0.0;
        }
        double den = 0.0;
        for (int64_t j = 0; j < c->N; ++j) {
            const float *k = c->K + (j * c->H + c->h) * (int64_t)d;
            const float *v = c->V + (j * c->H + c->h) * (int64_t)d;
            double wj = 0.0;
            for (int e = 0; e < d; ++e) wj += fq[e] * elu1((double)k[e]);
            den += wj;
            for (int e = 0; e < d; ++e) acc[e] += wj * (double)v[e];
        }
        double *y = c->Y + r * d;
        for (int e = 0; e < d; ++e) y[e] = acc[e] / den;
    }
    free(fq);
}

void or_linattn_rows(const float *Q, const float *K, const float *V, int64_t N, int H, int d,
                     int h, const int64_t *rows, int64_t nrows, double *Y, int nthreads) {
    lin_ctx c = {Q, K, V, N, H, d, h, rows, Y};
    or_parallel_for(nrows, nthreads, lin_body, &c);
}

/* ------------------------------------------ dense block around the layer */
/*
 * Algorithm 1, steps (1), (3) and (4): the normalisations, the rotary
 * positional encoding applied inside QKV_h(., P), and the FFN activation.
 * (The linear layers are plain matrix products; the Python side uses a
 * library matmul for them.)
 */

/* LN: y = (x - mean) / sqrt(var + eps) * g + b per row of D values, mean and
 * the biased variance taken in index order. */
typedef struct {
    const double *X;
    int64_t N;
    int D;
    const float *g, *b;
    double eps;
    double *Y;
} ln_ctx;

static void ln_body(void *p, int64_t lo, int64_t hi) {
    ln_ctx *c = (ln_ctx *)p;
    for (int64_t i = lo; i < hi; ++i) {
        const double *x = c->X + i * c->D;
        double mean = 0.0, var = 0.0;
        for (int k = 0; k < c->D; ++k) mean += (double)x[k];
        mean /= c->D;
        for (int k = 0; k < c->D; ++k) var += ((double)x[k] - mean) * ((double)x[k] - mean);
        var /= c->D;
        const double r = 1.0 / sqrt(var + c->eps);
        for (int k = 0; k < c->D; ++k)
            c->Y[i * c->D + k] = ((double)x[k] - mean) * r * (double)c->g[k] + (double)c->b[k];
    }
}

void or_layernorm(const double *X, int64_t N, int D, const float *g, const float *b, double eps,
                  double *Y, int nthreads) {
    ln_ctx c = {X, N, D, g, b, eps, Y};
    or_parallel_for(N, nthreads, ln_body, &c);
}

/* 2D rotary encoding, in place on T [N, H, d] (d a multiple of 4).  The d
 * features of a head split into two halves of d/2: the first is rotated by
 * the token's row coordinate pos[i][0], the second by its column coordinate
 * pos[i][1].  Within a half of m = d/2 features, feature j and feature
 * j + m/2 (j < m/2) form a plane rotated by the angle p * base^(-2j/m):
 *   (u, w) -> (u cos a - w sin a, u sin a + w cos a). */
typedef struct {
    double *T;
    int64_t N;
    int H, d;
    const int32_t *pos;
    double base;
} rope_ctx;

static void rope_body(void *p, int64_t lo, int64_t hi) {
    rope_ctx *c = (rope_ctx *)p;
    const int m = c->d / 2, q = m / 2;
    for (int64_t i = lo; i < hi; ++i)
        for (int h = 0; h < c->H; ++h)
            for (int half = 0; half < 2; ++half) {
                const double coord = (double)c->pos[2 * i + half];
                double *t = c->T + (i * c->H + h) * (int64_t)c->d + half * m;
                for (int j = 0; j < q; ++j) {
                    const double a = coord * pow(c->base, -2.0 * j / (double)m);
                    const double u = t[j], w = t[j + q];
                    t[j] = u * cos(a) - w * sin(a);
                    t[j + q] = u * sin(a) + w * cos(a);
                }
            }
}

void or_rope2d(double *T, int64_t N, int H, int d, const int32_t *pos, double base,
               int nthreads) {
    rope_ctx c = {T, N, H, d, pos, base};
    or_parallel_for(N, nthreads, rope_body, &c);
}

/* GELU with the exact normal CDF: x * (1 + erf(x / sqrt 2)) / 2, in place. */
void or_gelu(double *X, int64_t n) {
    for (int64_t i = 0; i < n; ++i) X[i] = 0.5 * X[i] * (1.0 + erf(X[i] / sqrt(2.0)));
}

/* ------------------------------------------- distillation targets (Eq.8) */
/*
 * Teacher attention of head h with every query attending all N keys:
 * A[k][q] = exp(l_qk - m_q) / sum_k' exp(l_qk' - m_q), l_qk = scale q_q . k_k,
 * m_q = max_k l_qk.  Eq.8 max-pools it over queries: p[k] = max_q A[k][q].
 * Pass 1 (independent queries): m_q and the row sum s_q.  Pass 2 (independent
 * keys; all keys, or the listed ones): the maximum over every query.
 */
typedef struct {
    const float *Q, *K;
    int64_t N;
    int H, d, h;
    double scale;
    double *m, *s;
    const int64_t *keys;
    double *p;
} colmax_ctx;

static double qk_dot(const colmax_ctx *c, int64_t q, int64_t k) {
    const float *a = c->Q + (q * c->H + c->h) * (int64_t)c->d;
    const float *b = c->K + (k * c->H + c->h) * (int64_t)c->d;
    double dot = 0.0;
    for (int e = 0; e < c->d; ++e) dot += (double)a[e] * (double)b[e];
    return dot * c->scale;
}

static void rowstat_body(void *p, int64_t lo, int64_t hi) {
    colmax_ctx *c = (colmax_ctx *)p;
    double *row = (double *)malloc(sizeof(double) * (c->N > 0 ? c->N : 1));
    for (int64_t q = lo; q < hi; ++q) {
        double m = -INFINITY;
        for (int64_t k = 0; k < c->N; ++k) {
            row[k] = qk_dot(c, q, k);
            if (row[k] > m) m = row[k];
        }
        double s = 0.0;
        for (int64_t k = 0; k < c->N; ++k) s += exp(row[k] - m);
        c->m[q] = m;
        c->s[q] = s;
    }
    free(row);
}

static void colmax_body(void *p, int64_t lo, int64_t hi) {
    colmax_ctx *c = (colmax_ctx *)p;
    for (int64_t i = lo; i < hi; ++i) {
        const int64_t k = c->keys ? c->keys[i] : i;
        double best = 0.0;
        for (int64_t q = 0; q < c->N; ++q) {
            const double a = exp(qk_dot(c, q, k) - c->m[q]) / c->s[q];
            if (a > best) best = a;
        }
        c->p[i] = best;
    }
}

void or_attention_colmax(const float *Q, const float *K, int64_t N, int H, int d, int h,
                         double scale, const int64_t *keys, int64_t nkeys, double *p,
                         int nthreads) {
    double *m = (double *)malloc(sizeof(double) * 2 * (N > 0 ? N : 1));
    colmax_ctx c = {Q, K, N, H, d, h, scale, m, m + N, keys, p};
    or_parallel_for(N, nthreads, rowstat_body, &c);
    or_parallel_for(keys ? nkeys : N, nthreads, colmax_body, &c);
    free(m);
}

/* -------------------------------------------------------- token merging
 * Token merging before the routed attention.  The paper combines its layer
 * with ToMe (as FastVGGT uses it, at merging ratios of 75 % and 90 %) and
 * gives no steps of its own; the steps here are ToMe's bipartite soft
 * matching (Bolya et al., ICLR 2023) applied to the layer's Q, K, V:
 *   metric  m_i = bf16(sum over heads of K_{i,h}): the head sum in fp32, in
 *           head order, rounded once to bf16 (ToMe matches tokens by their
 *           keys; rounding the metric fixes the precision in which both
 *           implementations take their decisions);
 *   split   destinations: every token of view 0, the nspecial special tokens
 *           of every view, and in views 1.. the patches whose index within
 *           the view's patches is a multiple of g, g the smallest stride
 *           that leaves at least M sources; sources: all other tokens;
 *   match   each source's most similar destination by cosine similarity
 *           (the first in token order on ties; 0 for a zero vector);
 *   select  the M sources with the largest similarity are merged (the lower
 *           token index first on ties);
 *   rows    the kept tokens (destinations and unmerged sources) in token
 *           order are the rows of the merged sequence; a merged source joins
 *           its destination's row;
 *   merge   a row is the mean of its tokens; unmerging gives every token its
 *           row's output.
 * --------------------------------------------------------------------- */

/* x rounded to bf16 (nearest, ties to even), as a double. */
static double bf16_rne(float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof(u));
    if ((u & 0x7f800000u) != 0x7f800000u) u += 0x7fffu + ((u >> 16) & 1u);
    u &= 0xffff0000u;
    float y;
    memcpy(&y, &u, sizeof(y));
    return (double)y;
}

void or_tome_metric(const float *K, int64_t N, int H, int d, double *m) {
    for (int64_t i = 0; i < N; ++i)
        for (int e = 0; e < d; ++e) {
            float s = 0.f;
            for (int h = 0; h < H; ++h) s += K[(i * H + h) * (int64_t)d + e];
            m[i * d + e] = bf16_rne(s);
        }
}

/* Destination flags; returns g, or -1 when fewer than M sources exist. */
int64_t or_tome_split(int64_t S, int64_t P, int64_t nspecial, int64_t M, uint8_t *is_dst) {
    const int64_t np = P - nspecial;
    if (S < 1 || np < 1 || M < 0) return -1;
    int64_t g = 1;
    for (; g <= np; ++g) {
        const int64_t ndst = (np + g - 1) / g;
        if ((S - 1) * (np - ndst) >= M) break;
    }
    if (g > np) return -1;
    for (int64_t v = 0; v < S; ++v)
        for (int64_t j = 0; j < P; ++j) {
            const int64_t k = j - nspecial;
            is_dst[v * P + j] = (uint8_t)(v == 0 || k < 0 || k % g == 0);
        }
    return g;
}

typedef struct {
    const double *m;
    int d;
    const int64_t *dst;   /* destination tokens, ascending */
    int64_t ndst;
    const double *dnorm;  /* |m| of each destination */
    const int64_t *src;   /* sources to match */
    int64_t *best;        /* [nsrc] most similar destination token */
    double *score;        /* [nsrc] its cosine similarity */
} tome_ctx;

static double vnorm(const double *x, int d) {
    double s = 0.0;
    for (int e = 0; e < d; ++e) s += x[e] * x[e];
    return sqrt(s);
}

static void match_body(void *p, int64_t lo, int64_t hi) {
    tome_ctx *c = (tome_ctx *)p;
    for (int64_t i = lo; i < hi; ++i) {
        const double *a = c->m + c->src[i] * c->d;
        const double na = vnorm(a, c->d);
        int64_t best = -1;
        double bs = 0.0;
        for (int64_t j = 0; j < c->ndst; ++j) {
            const double *b = c->m + c->dst[j] * c->d;
            double dot = 0.0;
            for (int e = 0; e < c->d; ++e) dot += a[e] * b[e];
            const double cs = (na == 0.0 || c->dnorm[j] == 0.0) ? 0.0 : dot / (na * c->dnorm[j]);
            if (best < 0 || cs > bs) {
                bs = cs;
                best = c->dst[j];
            }
        }
        c->best[i] = best;
        c->score[i] = bs;
    }
}

void or_tome_match(const double *m, int64_t N, int d, const uint8_t *is_dst, const int64_t *src,
                   int64_t nsrc, int64_t *best, double *score, int nthreads) {
    int64_t ndst = 0;
    for (int64_t t = 0; t < N; ++t) ndst += is_dst[t];
    int64_t *dst = (int64_t *)malloc(sizeof(int64_t) * (ndst > 0 ? ndst : 1));
    double *dn = (double *)malloc(sizeof(double) * (ndst > 0 ? ndst : 1));
    for (int64_t t = 0, j = 0; t < N; ++t)
        if (is_dst[t]) {
            dst[j] = t;
            dn[j] = vnorm(m + t * d, d);
            ++j;
        }
    tome_ctx c = {m, d, dst, ndst, dn, src, best, score};
    or_parallel_for(nsrc, nthreads, match_body, &c);
    free(dst);
    free(dn);
}

typedef struct {
    double score;
    int64_t tok;
    int64_t pos;
} tome_item;

static int by_score(const void *x, const void *y) {
    const tome_item *a = (const tome_item *)x, *b = (const tome_item *)y;
    if (a->score > b->score) return -1;
    if (a->score < b->score) return 1;
    return a->tok < b->tok ? -1 : (a->tok > b->tok ? 1 : 0);
}

/* merged[i] = 1 for the M sources ranked first by (similarity desc, token asc). */
void or_tome_select(const int64_t *src, const double *score, int64_t nsrc, int64_t M,
                    uint8_t *merged) {
    tome_item *it = (tome_item *)malloc(sizeof(tome_item) * (nsrc > 0 ? nsrc : 1));
    for (int64_t i = 0; i < nsrc; ++i) {
        it[i].score = score[i];
        it[i].tok = src[i];
        it[i].pos = i;
        merged[i] = 0;
    }
    qsort(it, (size_t)nsrc, sizeof(tome_item), by_score);
    for (int64_t i = 0; i < M && i < nsrc; ++i) merged[it[i].pos] = 1;
    free(it);
}

/* row[t]: the merged-sequence row of every token; returns the row count. */
int64_t or_tome_rows(int64_t N, const int64_t *src, const int64_t *best, const uint8_t *merged,
                     int64_t nsrc, int64_t *row) {
    int64_t *into = (int64_t *)malloc(sizeof(int64_t) * (N > 0 ? N : 1));
    for (int64_t t = 0; t < N; ++t) into[t] = -1;
    for (int64_t i = 0; i < nsrc; ++i)
        if (merged[i]) into[src[i]] = best[i];
    int64_t r = 0;
    for (int64_t t = 0; t < N; ++t)
        if (into[t] < 0) row[t] = r++;
    for (int64_t t = 0; t < N; ++t)
        if (into[t] >= 0) row[t] = row[into[t]];
    free(into);
    return r;
}

/* Xm[r] = mean of X[t] over the tokens t with row[t] = r; X is [N, F]. */
void or_tome_merge(const float *X, int64_t N, int64_t F, const int64_t *row, int64_t nrows,
                   double *Xm) {
    int64_t *cnt = (int64_t *)calloc((size_t)(nrows > 0 ? nrows : 1), sizeof(int64_t));
    memset(Xm, 0, sizeof(double) * (size_t)(nrows * F));
    for (int64_t t = 0; t < N; ++t) {
        double *y = Xm + row[t] * F;
        const float *x = X + t * F;
        for (int64_t f = 0; f < F; ++f) y[f] += (double)x[f];
        cnt[row[t]]++;
    }
    for (int64_t r = 0; r < nrows; ++r)
        for (int64_t f = 0; f < F; ++f) Xm[r * F + f] /= (double)cnt[r];
    free(cnt);
}
