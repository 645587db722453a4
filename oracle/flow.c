/*
 * Plain CPU oracle of the streaming flow-decoder chunk step (fp64).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or constant with the
 * GPU library; the two meet only in the float32 weight blob and the seeded
 * inputs (data).
 *
 * What it computes.  The flow decoder turns the token encoder's features mu
 * into mel frames by conditional flow matching: starting from Gaussian noise
 * x_0 it integrates dx/dt = v(x, t) from t = 0 to 1 in n_steps explicit Euler
 * steps, where the velocity is the classifier-free-guided combination of a
 * DiT estimator evaluated on the conditional input (x, mu, speaker, prompt
 * mel) and on the unconditional one (x and zeros): Motivation ("Where the
 * time goes": a CFM solve with CFG x2 per second of speech) and the adapter
 * declaration (Design, "Adapter": n_steps = 10 solver steps).  Streaming
 * runs the estimator on one call of f_call frames at a time; every attention
 * of every block at every solver step also attends to that step's carried
 * keys and values of earlier frames.  The carry C follows Eq. carry exactly:
 * after a call the live cache is H = (this call's retained frames) || C, and
 * when its extent exceeds L = f_retained + f_prompt it is cut back to
 * H[0 : f_retained] || H[ext - f_prompt : ext] (prepend order: the mutable
 * history window before the immutable prompt tail).  A turn starts with a
 * prompt pass that attends only to itself and leaves the prompt's keys and
 * values as the whole carry (Design, "State rule": a turn transition writes
 * base state into the carry).  The attended extents are then f_prompt,
 * f_prompt + f_chunk, ... up to L (Eq. catalog; {302, 352, 402}).
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - the estimator is a DiT: input Linear(4 n_mel -> dim) of x | mu | spk |
 *     cond; blocks of adaLN-modulated multi-head self-attention and a GELU
 *     (tanh form) MLP with gated residuals; a modulated final LayerNorm and
 *     Linear(dim -> n_mel).  LayerNorm has no affine part, eps 1e-6.  The
 *     modulation of step i is Linear(SiLU(e(t_i))) where e is a two-layer
 *     SiLU MLP of the sinusoidal embedding of 1000 t (cos half, then sin half,
 *     frequencies 10000^(-j/half)).  Attention scores are q.k / sqrt(64);
 *   - the time grid is the cosine schedule t_i = 1 - cos(pi/2 * i/n_steps);
 *   - guidance: v = (1 + w) v_cond - w v_uncond with w = cfg_rate; the
 *     unconditional input keeps x and zeros mu, spk and cond;
 *   - a call of n frames retains its first f_chunk frames when n >= f_chunk
 *     (the rest are the lookahead, presented again by the next call) and
 *     retains nothing when n < f_chunk (a flush that ends the turn); all n
 *     frames attend to each other and to the carry;
 *   - noise: x_0 of the frame with index tau since the turn start (prompt
 *     frames first), mel pair j, is temperature * Box-Muller of the first two
 *     words of Philox4x64-10 at counter (tau, j, 2, 0), key (seed, stream key);
 *   - with bf16 parameters the weights of the estimator's Linear layers that
 *     run per solver step (in, qkv, o, fc1, fc2, out) are rounded to bfloat16;
 *     the arithmetic stays fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

float oc_round_bf16(float x);
void oc_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
double oc_u01(uint64_t x);
void oc_box_muller(double u0, double u1, double* g0, double* g1);

typedef struct {
    int n_mel, dim, heads, depth, mlp, t_dim, n_steps;
    int f_prompt, f_retained, f_chunk, f_call;
    double cfg_rate, temperature;
} ocf_arch;

/* y[r][o] = b[o] + sum_i W[o][i] x[r][i], W in PyTorch layout [out][in]. */
typedef struct {
    const double* W;
    const double* b;
    int out, in;
} ocf_lin;

typedef struct {
    ocf_arch a;
    double* w;                 /* the blob in fp64 */
    ocf_lin t1, t2, in, fada, out;
    ocf_lin *ada, *qkv, *o, *fc1, *fc2;
    double* t;                 /* [n_steps + 1] */
    double* mods;              /* [n_steps][depth][6 dim] */
    double* fmods;             /* [n_steps][2 dim] */
    int cap;                   /* frames a carry can hold: L + f_chunk */
    double *K, *V;             /* [n_steps][depth][2 branches][cap][dim], Eq. carry order */
    int len;                   /* frames in every carry */
    int prompt;                /* prompt frames of the turn */
    int64_t pos;               /* frame index (since the turn start) of the next call's first frame */
    double* spk;               /* [n_mel] */
    uint64_t seed, key;
} ocf_stream;

/* ----------------------------------------------------------- primitives */

static void linear(const ocf_lin* L, int rows, const double* x, double* y)
{
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; r++) {
        const double* xr = x + (size_t)r * L->in;
        double* yr = y + (size_t)r * L->out;
        for (int o = 0; o < L->out; o++) {
            const double* wo = L->W + (size_t)o * L->in;
            double s = 0.0;
            for (int i = 0; i < L->in; i++) s += wo[i] * xr[i];
            yr[o] = L->b[o] + s;
        }
    }
}

static double silu(double v) { return v / (1.0 + exp(-v)); }

/* GELU, tanh form: 0.5 v (1 + tanh(sqrt(2/pi) (v + 0.044715 v^3))). */
double ocf_gelu(double v)
{
    return 0.5 * v * (1.0 + tanh(sqrt(2.0 / M_PI) * (v + 0.044715 * v * v * v)));
}

/* a = LayerNorm(h) * (1 + scale) + shift over one row of n values (no affine, eps 1e-6). */
void ocf_lnmod(int n, const double* h, const double* shift, const double* scale, double* a)
{
    double mean = 0.0, var = 0.0;
    for (int i = 0; i < n; i++) mean += h[i];
    mean /= n;
    for (int i = 0; i < n; i++) var += (h[i] - mean) * (h[i] - mean);
    var /= n;
    const double inv = 1.0 / sqrt(var + 1e-6);
    for (int i = 0; i < n; i++) a[i] = (h[i] - mean) * inv * (1.0 + scale[i]) + shift[i];
}

/*
 * Scaled dot-product attention of nq queries over nk keys for one head of
 * width hd: out[f] = sum_j softmax_j(q_f . k_j / sqrt(hd)) v_j.  Rows of q,
 * k, v and out are `stride` apart (the head's columns of a wider row).
 */
void ocf_attention(int nq, int nk, int hd, const double* q, const double* k, const double* v, int stride,
                   double* out)
{
    const double scale = 1.0 / sqrt((double)hd);
    double* s = malloc(sizeof(double) * (size_t)(nk > 0 ? nk : 1));
    for (int f = 0; f < nq; f++) {
        const double* qf = q + (size_t)f * stride;
        double m = -INFINITY;
        for (int j = 0; j < nk; j++) {
            const double* kj = k + (size_t)j * stride;
            double d = 0.0;
            for (int e = 0; e < hd; e++) d += qf[e] * kj[e];
            s[j] = d * scale;
            if (s[j] > m) m = s[j];
        }
        double z = 0.0;
        for (int j = 0; j < nk; j++) {
            s[j] = exp(s[j] - m);
            z += s[j];
        }
        double* of = out + (size_t)f * stride;
        for (int e = 0; e < hd; e++) of[e] = 0.0;
        for (int j = 0; j < nk; j++) {
            const double* vj = v + (size_t)j * stride;
            const double p = s[j] / z;
            for (int e = 0; e < hd; e++) of[e] += p * vj[e];
        }
    }
    free(s);
}

/* The cosine time grid t_i = 1 - cos(pi/2 * i / n), i = 0 .. n. */
void ocf_times(int n, double* t)
{
    for (int i = 0; i <= n; i++) t[i] = 1.0 - cos(0.5 * M_PI * (double)i / (double)n);
}

/* Sinusoidal embedding of 1000 t: e[j] = cos(1000 t f_j), e[half + j] = sin(1000 t f_j),
 * f_j = 10000^(-j / half). */
void ocf_time_embedding(int t_dim, double t, double* e)
{
    const int half = t_dim / 2;
    for (int j = 0; j < half; j++) {
        const double arg = 1000.0 * t * exp(-log(10000.0) * (double)j / (double)half);
        e[j] = cos(arg);
        e[half + j] = sin(arg);
    }
}

/* x_0 of `frames` frames starting at frame index tau0 since the turn start. */
void ocf_noise(int n_mel, double temperature, uint64_t seed, uint64_t key, int64_t tau0, int frames, double* x)
{
    const uint64_t k[2] = {seed, key};
    for (int f = 0; f < frames; f++)
        for (int j = 0; j < n_mel / 2; j++) {
            const uint64_t ctr[4] = {(uint64_t)(tau0 + f), (uint64_t)j, 2, 0};
            uint64_t r[4];
            oc_philox4x64(ctr, k, r);
            double g0, g1;
            oc_box_muller(oc_u01(r[0]), oc_u01(r[1]), &g0, &g1);
            x[(size_t)f * n_mel + 2 * j] = temperature * g0;
            x[(size_t)f * n_mel + 2 * j + 1] = temperature * g1;
        }
}

/* --------------------------------------------------------------- weights */

long ocf_blob_floats(const ocf_arch* a)
{
    const long D = a->dim, M = a->n_mel, T = a->t_dim, H = a->mlp;
    long n = D * T + D + D * D + D + D * 4 * M + D;
    n += (long)a->depth * (6 * D * D + 6 * D + 3 * D * D + 3 * D + D * D + D + H * D + H + D * H + D);
    n += 2 * D * D + 2 * D + M * D + M;
    return n;
}

static ocf_lin take_lin(double** cur, int out, int in)
{
    ocf_lin L = {*cur, *cur + (size_t)out * in, out, in};
    *cur += (size_t)out * in + out;
    return L;
}

static void round_lin(ocf_lin* L)
{
    double* W = (double*)L->W;
    for (size_t i = 0; i < (size_t)L->out * L->in; i++) W[i] = (double)oc_round_bf16((float)W[i]);
}

static int valid_arch(const ocf_arch* a)
{
    return a->n_mel > 0 && a->n_mel % 2 == 0 && a->heads > 0 && a->dim % a->heads == 0 && a->depth > 0 &&
           a->mlp > 0 && a->t_dim > 0 && a->t_dim % 2 == 0 && a->n_steps > 0 && a->f_chunk > 0 &&
           a->f_call >= a->f_chunk && a->f_retained >= 0 && a->f_retained % a->f_chunk == 0 && a->f_prompt > 0;
}

/* Open a stream: weights, the time grid and the per-step modulations (they depend
 * only on t_i).  Returns NULL on a bad architecture or blob size. */
ocf_stream* ocf_open(const ocf_arch* a, int bf16, const float* blob, long blob_n, uint64_t seed, uint64_t key)
{
    if (!valid_arch(a) || blob_n != ocf_blob_floats(a)) return NULL;
    ocf_stream* s = calloc(1, sizeof(ocf_stream));
    s->a = *a;
    s->seed = seed;
    s->key = key;
    s->w = malloc(sizeof(double) * (size_t)blob_n);
    for (long i = 0; i < blob_n; i++) s->w[i] = (double)blob[i];
    const int D = a->dim, M = a->n_mel, NL = a->depth, NS = a->n_steps;
    double* cur = s->w;
    s->t1 = take_lin(&cur, D, a->t_dim);
    s->t2 = take_lin(&cur, D, D);
    s->in = take_lin(&cur, D, 4 * M);
    s->ada = malloc(sizeof(ocf_lin) * NL);
    s->qkv = malloc(sizeof(ocf_lin) * NL);
    s->o = malloc(sizeof(ocf_lin) * NL);
    s->fc1 = malloc(sizeof(ocf_lin) * NL);
    s->fc2 = malloc(sizeof(ocf_lin) * NL);
    for (int l = 0; l < NL; l++) {
        s->ada[l] = take_lin(&cur, 6 * D, D);
        s->qkv[l] = take_lin(&cur, 3 * D, D);
        s->o[l] = take_lin(&cur, D, D);
        s->fc1[l] = take_lin(&cur, a->mlp, D);
        s->fc2[l] = take_lin(&cur, D, a->mlp);
    }
    s->fada = take_lin(&cur, 2 * D, D);
    s->out = take_lin(&cur, M, D);
    if (bf16) {
        round_lin(&s->in);
        round_lin(&s->out);
        for (int l = 0; l < NL; l++) {
            round_lin(&s->qkv[l]);
            round_lin(&s->o[l]);
            round_lin(&s->fc1[l]);
            round_lin(&s->fc2[l]);
        }
    }
    s->t = malloc(sizeof(double) * (NS + 1));
    ocf_times(NS, s->t);
    s->mods = malloc(sizeof(double) * (size_t)NS * NL * 6 * D);
    s->fmods = malloc(sizeof(double) * (size_t)NS * 2 * D);
    double* e = malloc(sizeof(double) * a->t_dim);
    double* g = malloc(sizeof(double) * D);
    double* temb = malloc(sizeof(double) * D);
    for (int i = 0; i < NS; i++) {
        ocf_time_embedding(a->t_dim, s->t[i], e);
        linear(&s->t1, 1, e, g);
        for (int c = 0; c < D; c++) g[c] = silu(g[c]);
        linear(&s->t2, 1, g, temb);
        for (int c = 0; c < D; c++) g[c] = silu(temb[c]);
        for (int l = 0; l < NL; l++) linear(&s->ada[l], 1, g, s->mods + ((size_t)i * NL + l) * 6 * D);
        linear(&s->fada, 1, g, s->fmods + (size_t)i * 2 * D);
    }
    free(e);
    free(g);
    free(temb);
    s->cap = a->f_retained + a->f_prompt + a->f_chunk;
    s->K = calloc((size_t)NS * NL * 2 * s->cap * D, sizeof(double));
    s->V = calloc((size_t)NS * NL * 2 * s->cap * D, sizeof(double));
    s->spk = calloc(M, sizeof(double));
    return s;
}

void ocf_close(ocf_stream* s)
{
    if (!s) return;
    free(s->w);
    free(s->ada);
    free(s->qkv);
    free(s->o);
    free(s->fc1);
    free(s->fc2);
    free(s->t);
    free(s->mods);
    free(s->fmods);
    free(s->K);
    free(s->V);
    free(s->spk);
    free(s);
}

/* The time grid and modulations, for the pins. */
void ocf_get_times(const ocf_stream* s, double* t) { memcpy(t, s->t, sizeof(double) * (s->a.n_steps + 1)); }
void ocf_get_mods(const ocf_stream* s, int step, int layer, double* out6d)
{
    const int D = s->a.dim;
    if (layer < s->a.depth)
        memcpy(out6d, s->mods + ((size_t)step * s->a.depth + layer) * 6 * D, sizeof(double) * 6 * D);
    else
        memcpy(out6d, s->fmods + (size_t)step * 2 * D, sizeof(double) * 2 * D);
}

static double* carry_K(ocf_stream* s, int i, int l, int c)
{
    return s->K + (((size_t)i * s->a.depth + l) * 2 + c) * s->cap * s->a.dim;
}
static double* carry_V(ocf_stream* s, int i, int l, int c)
{
    return s->V + (((size_t)i * s->a.depth + l) * 2 + c) * s->cap * s->a.dim;
}

/* ------------------------------------------------------------- the solve */

/*
 * One call of n frames: integrate from the noise of its frames through the
 * n_steps Euler steps, every estimator evaluation attending to the carry of
 * its solver step (none for the prompt pass).  mu, cond: [n][n_mel] (cond
 * NULL = zeros).  keep[i][l][c] receives the keys and values of the call's
 * first `retain` frames.  mel: [n][n_mel] the final x.
 */
static void solve(ocf_stream* s, int n, const double* mu, const double* cond, int use_carry, int retain,
                  double* newK, double* newV, double* mel)
{
    const ocf_arch* a = &s->a;
    const int D = a->dim, M = a->n_mel, NL = a->depth, NS = a->n_steps, HD = D / a->heads;
    const int R = 2 * n;                 /* rows: branch c (0 conditional, 1 unconditional), frame f */
    const double w = a->cfg_rate;
    double* x = malloc(sizeof(double) * (size_t)n * M);
    double* xin = malloc(sizeof(double) * (size_t)R * 4 * M);
    double* h = malloc(sizeof(double) * (size_t)R * D);
    double* act = malloc(sizeof(double) * (size_t)R * (a->mlp > 3 * D ? a->mlp : 3 * D));
    double* qkv = malloc(sizeof(double) * (size_t)R * 3 * D);
    double* att = malloc(sizeof(double) * (size_t)R * D);
    double* y = malloc(sizeof(double) * (size_t)R * (a->mlp > D ? a->mlp : D));
    double* v = malloc(sizeof(double) * (size_t)R * M);
    const int cl = use_carry ? s->len : 0;
    const int nk = cl + n;
    double* kk = malloc(sizeof(double) * (size_t)nk * D);
    double* vv = malloc(sizeof(double) * (size_t)nk * D);

    ocf_noise(M, a->temperature, s->seed, s->key, s->pos, n, x);
    for (int i = 0; i < NS; i++) {
        for (int c = 0; c < 2; c++)
            for (int f = 0; f < n; f++) {
                double* r = xin + ((size_t)c * n + f) * 4 * M;
                for (int m = 0; m < M; m++) {
                    r[m] = x[(size_t)f * M + m];
                    r[M + m] = c == 0 ? mu[(size_t)f * M + m] : 0.0;
                    r[2 * M + m] = c == 0 ? s->spk[m] : 0.0;
                    r[3 * M + m] = (c == 0 && cond) ? cond[(size_t)f * M + m] : 0.0;
                }
            }
        linear(&s->in, R, xin, h);
        for (int l = 0; l < NL; l++) {
            const double* md = s->mods + ((size_t)i * NL + l) * 6 * D;
            const double *shift1 = md, *scale1 = md + D, *gate1 = md + 2 * D;
            const double *shift2 = md + 3 * D, *scale2 = md + 4 * D, *gate2 = md + 5 * D;
            for (int r = 0; r < R; r++) ocf_lnmod(D, h + (size_t)r * D, shift1, scale1, act + (size_t)r * D);
            linear(&s->qkv[l], R, act, qkv);
            for (int c = 0; c < 2; c++) {
                /* keys and values: the carry of (step i, block l, branch c), then the call's own frames */
                const double* CK = carry_K(s, i, l, c);
                const double* CV = carry_V(s, i, l, c);
                memcpy(kk, CK, sizeof(double) * (size_t)cl * D);
                memcpy(vv, CV, sizeof(double) * (size_t)cl * D);
                for (int f = 0; f < n; f++) {
                    const double* q = qkv + ((size_t)c * n + f) * 3 * D;
                    memcpy(kk + (size_t)(cl + f) * D, q + D, sizeof(double) * D);
                    memcpy(vv + (size_t)(cl + f) * D, q + 2 * D, sizeof(double) * D);
                }
                if (retain > 0) {
                    double* nK = newK + (((size_t)i * NL + l) * 2 + c) * (size_t)retain * D;
                    double* nV = newV + (((size_t)i * NL + l) * 2 + c) * (size_t)retain * D;
                    memcpy(nK, kk + (size_t)cl * D, sizeof(double) * (size_t)retain * D);
                    memcpy(nV, vv + (size_t)cl * D, sizeof(double) * (size_t)retain * D);
                }
                /* queries: rows (c, f), columns [0, D) of the qkv rows */
                double* qc = malloc(sizeof(double) * (size_t)n * D);
                for (int f = 0; f < n; f++) memcpy(qc + (size_t)f * D, qkv + ((size_t)c * n + f) * 3 * D, sizeof(double) * D);
#pragma omp parallel for schedule(static)
                for (int hh = 0; hh < a->heads; hh++)
                    ocf_attention(n, nk, HD, qc + hh * HD, kk + hh * HD, vv + hh * HD, D,
                                  att + (size_t)c * n * D + hh * HD);
                free(qc);
            }
            linear(&s->o[l], R, att, y);
            for (int r = 0; r < R; r++)
                for (int e = 0; e < D; e++) h[(size_t)r * D + e] += gate1[e] * y[(size_t)r * D + e];
            for (int r = 0; r < R; r++) ocf_lnmod(D, h + (size_t)r * D, shift2, scale2, act + (size_t)r * D);
            linear(&s->fc1[l], R, act, y);
            for (size_t e = 0; e < (size_t)R * a->mlp; e++) y[e] = ocf_gelu(y[e]);
            linear(&s->fc2[l], R, y, att);
            for (int r = 0; r < R; r++)
                for (int e = 0; e < D; e++) h[(size_t)r * D + e] += gate2[e] * att[(size_t)r * D + e];
        }
        const double* fm = s->fmods + (size_t)i * 2 * D;
        for (int r = 0; r < R; r++) ocf_lnmod(D, h + (size_t)r * D, fm, fm + D, act + (size_t)r * D);
        linear(&s->out, R, act, v);
        const double dt = s->t[i + 1] - s->t[i];
        for (int f = 0; f < n; f++)
            for (int m = 0; m < M; m++) {
                const double vc = v[(size_t)f * M + m], vu = v[((size_t)n + f) * M + m];
                x[(size_t)f * M + m] += dt * ((1.0 + w) * vc - w * vu);
            }
    }
    if (mel) memcpy(mel, x, sizeof(double) * (size_t)n * M);
    free(x);
    free(xin);
    free(h);
    free(act);
    free(qkv);
    free(att);
    free(y);
    free(v);
    free(kk);
    free(vv);
}

/*
 * Start a turn: the prompt pass over P frames (mu, cond: [P][n_mel]; spk:
 * [n_mel]) leaves the prompt's keys and values of every (step, block,
 * branch) as the whole carry.  mel (may be NULL) receives the prompt frames'
 * solution.  Returns 0, or -1 when P is out of range.
 */
int ocf_prompt(ocf_stream* s, int P, const double* mu, const double* cond, const double* spk, double* mel)
{
    const ocf_arch* a = &s->a;
    if (P < 1 || P > a->f_prompt) return -1;
    const int D = a->dim, NL = a->depth, NS = a->n_steps;
    memcpy(s->spk, spk, sizeof(double) * a->n_mel);
    s->pos = 0;
    s->len = 0;
    double* nK = malloc(sizeof(double) * (size_t)NS * NL * 2 * P * D);
    double* nV = malloc(sizeof(double) * (size_t)NS * NL * 2 * P * D);
    solve(s, P, mu, cond, 0, P, nK, nV, mel);
    for (int i = 0; i < NS; i++)
        for (int l = 0; l < NL; l++)
            for (int c = 0; c < 2; c++) {
                const size_t src = (((size_t)i * NL + l) * 2 + c) * (size_t)P * D;
                memcpy(carry_K(s, i, l, c), nK + src, sizeof(double) * (size_t)P * D);
                memcpy(carry_V(s, i, l, c), nV + src, sizeof(double) * (size_t)P * D);
            }
    free(nK);
    free(nV);
    s->len = P;
    s->prompt = P;
    s->pos = P;
    return 0;
}

/*
 * One chunk call of n frames (1 <= n <= f_call) with features mu [n][n_mel]:
 * mel [n][n_mel] receives the solution.  When n >= f_chunk the first f_chunk
 * frames enter the carry by Eq. carry and the stream advances f_chunk
 * frames; a shorter call is a flush and changes no state.  Returns the
 * carry's extent after the call, or -1 (no prompt yet, or n out of range).
 */
int ocf_chunk(ocf_stream* s, int n, const double* mu, double* mel)
{
    const ocf_arch* a = &s->a;
    if (s->prompt == 0 || n < 1 || n > a->f_call) return -1;
    const int D = a->dim, NL = a->depth, NS = a->n_steps;
    const int retain = n >= a->f_chunk ? a->f_chunk : 0;
    double* nK = retain ? malloc(sizeof(double) * (size_t)NS * NL * 2 * retain * D) : NULL;
    double* nV = retain ? malloc(sizeof(double) * (size_t)NS * NL * 2 * retain * D) : NULL;
    solve(s, n, mu, NULL, 1, retain, nK, nV, mel);
    if (retain) {
        const int ext = retain + s->len;                       /* extent of H = new || C */
        const int L = a->f_retained + s->prompt;
        double* H = malloc(sizeof(double) * (size_t)ext * D);
        for (int i = 0; i < NS; i++)
            for (int l = 0; l < NL; l++)
                for (int c = 0; c < 2; c++)
                    for (int kv = 0; kv < 2; kv++) {
                        double* C = kv == 0 ? carry_K(s, i, l, c) : carry_V(s, i, l, c);
                        const double* nw = (kv == 0 ? nK : nV) + (((size_t)i * NL + l) * 2 + c) * (size_t)retain * D;
                        memcpy(H, nw, sizeof(double) * (size_t)retain * D);
                        memcpy(H + (size_t)retain * D, C, sizeof(double) * (size_t)s->len * D);
                        if (ext > L) {
                            /* C[0:L] <- H[0:f_retained] || H[ext - f_prompt : ext] */
                            memcpy(C, H, sizeof(double) * (size_t)a->f_retained * D);
                            memcpy(C + (size_t)a->f_retained * D, H + (size_t)(ext - s->prompt) * D,
                                   sizeof(double) * (size_t)s->prompt * D);
                        } else {
                            memcpy(C, H, sizeof(double) * (size_t)ext * D);
                        }
                    }
        free(H);
        s->len = ext > L ? L : ext;
        s->pos += retain;
    }
    free(nK);
    free(nV);
    return s->len;
}

/* The carry of (step, block, branch): kv 0 keys, 1 values, [len][dim] in Eq. carry order.
 * Returns len. */
int ocf_carry(ocf_stream* s, int step, int layer, int branch, int kv, double* out)
{
    const double* C = kv == 0 ? carry_K(s, step, layer, branch) : carry_V(s, step, layer, branch);
    if (out) memcpy(out, C, sizeof(double) * (size_t)s->len * s->a.dim);
    return s->len;
}

int64_t ocf_position(const ocf_stream* s) { return s->pos; }
