/*
 * corun_oracle.c -- CPU oracle for the padded, fixed-shape transformer decode
 * step and the isolated single-request prefill of CoRun (arXiv 2608.14376).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * with the HIP library.
 *
 * What it computes.  CoRun does not change the model's arithmetic; it makes a
 * standard decoder step reproducible by controlling the execution shape
 * (Sec. IV, "Determinism Contract").  The determinism argument (Sec. IV,
 * "Determinism Argument") treats each request's output as a request-local
 * function d(z) of its own state z = (prefix, KV cache, sampling parameters),
 * isolated from every co-runner.  The oracle is exactly that function, written
 * out one live row at a time with no batch at all: a pre-norm grouped-query
 * decoder step (the paper names no model, so the block structure is the
 * Llama/Qwen family's; see the "readings" list in the design notes).
 *
 * Precision.  The paper fixes no precision.  The oracle keeps the model's
 * storage points -- bf16 weights, KV entries and the listed bf16 activations,
 * an fp32 residual stream -- and computes everything between two storage
 * points in fp64, with every sum taken sequentially in index order.  A product
 * of two bf16 values is exact in fp64, so each dot product is the exact sum up
 * to ~1e-16 relative.  The storage points are:
 *   - RMSNorm outputs                                  -> bf16
 *   - q, k, v after the QKV projection                  -> bf16
 *   - q, k after the rotary embedding (k is cached)     -> bf16
 *   - attention output                                 -> bf16
 *   - gate, up after their projection                   -> bf16
 *   - SwiGLU output                                     -> bf16
 *   - residual stream after each sub-layer add          -> fp32
 *   - logits                                            -> fp64 (returned)
 *
 * Threads.  OpenMP splits only independent output elements; each element's
 * sum runs in one thread in index order, so results do not depend on the
 * thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* bf16 <-> binary64.  bf16 is the upper half of an IEEE binary32: 1 sign    */
/* bit, 8 exponent bits (bias 127), 7 stored significand bits.              */
/* ------------------------------------------------------------------------ */

double orc_bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Round a binary64 value to the nearest bf16, ties to even (IEEE 754
 * roundTiesToEven), with overflow to infinity and gradual underflow.  A
 * normal bf16 has an 8-bit significand, so for |x| in [2^(e-1), 2^e) the
 * spacing of bf16 values is 2^(e-8); below 2^-126 the spacing stays 2^-133. */
uint16_t orc_f64_to_bf16(double x)
{
    if (isnan(x)) return 0x7FC0;
    if (isinf(x)) return signbit(x) ? 0xFF80 : 0x7F80;
    if (x == 0.0) return signbit(x) ? 0x8000 : 0x0000;
    int e;
    (void)frexp(x, &e);                 /* |x| in [2^(e-1), 2^e) */
    if (e < -125) e = -125;             /* subnormal range: fixed spacing */
    double spacing = ldexp(1.0, e - 8);
    double r = nearbyint(x / spacing) * spacing;   /* exact scaling; RNE */
    if (fabs(r) >= ldexp(1.0, 128)) return signbit(x) ? 0xFF80 : 0x7F80;
    float f = (float)r;                 /* exact: r has <= 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(u >> 16);
}

static double bf(uint16_t b) { return orc_bf16_to_f64(b); }
static uint16_t tobf(double x) { return orc_f64_to_bf16(x); }

/* Convert n fp32 values, given as bit patterns, to bf16 (used to pin the
 * rounding routine against an independent library, exhaustively). */
void orc_f32bits_to_bf16(const uint32_t *bits, uint16_t *out, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        float f;
        memcpy(&f, &bits[i], sizeof f);
        out[i] = orc_f64_to_bf16((double)f);
    }
}

/* ------------------------------------------------------------------------ */
/* Operators.  Each is the textbook definition.                             */
/* ------------------------------------------------------------------------ */

/* Sequential dot product of two bf16 vectors in fp64, index order. */
static double dot_bf16(const uint16_t *a, const uint16_t *b, int n)
{
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += bf(a[i]) * bf(b[i]);
    return s;
}

/* Linear layer y = W h, W in [out, in] row-major (PyTorch Linear layout),
 * no bias.  y[j] = sum_i h[i] W[j, i], fp64, not rounded. */
void orc_linear(const uint16_t *h, int in, const uint16_t *W, int out, double *y)
{
#pragma omp parallel for schedule(static)
    for (int j = 0; j < out; ++j) y[j] = dot_bf16(h, W + (int64_t)j * in, in);
}

/* RMSNorm: y_i = bf16( x_i / sqrt(mean_j x_j^2 + eps) * g_i ). */
void orc_rmsnorm(const float *x, int n, const uint16_t *g, double eps, uint16_t *y)
{
    double ss = 0.0;
    for (int i = 0; i < n; ++i) ss += (double)x[i] * (double)x[i];
    double inv = 1.0 / sqrt(ss / n + eps);
    for (int i = 0; i < n; ++i) y[i] = tobf((double)x[i] * inv * bf(g[i]));
}

/* Rotary position embedding, rotate-half pairing: dimension i < d/2 is
 * paired with i + d/2 and rotated by the angle pos * theta^(-2i/d).
 * In fp64 on one head vector; not rounded (the caller rounds). */
void orc_rope(const double *x, int d, int pos, double theta, double *y)
{
    int half = d / 2;
    for (int i = 0; i < half; ++i) {
        double w = pow(theta, -2.0 * i / d);
        double a = (double)pos * w;
        double c = cos(a), s = sin(a);
        y[i] = x[i] * c - x[i + half] * s;
        y[i + half] = x[i + half] * c + x[i] * s;
    }
}

/* Single-head scaled dot-product attention of one query over keys 0..n-1:
 * s_t = (q . k_t) / sqrt(d);  w_t = exp(s_t - max s);
 * out = sum_t w_t v_t / sum_t w_t.   K, V given as n row pointers.
 * fp64, not rounded. */
void orc_attention(const uint16_t *q, const uint16_t *const *K, const uint16_t *const *V,
                   int n, int d, double *out)
{
    double *s = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double scale = 1.0 / sqrt((double)d);
    double m = -INFINITY;
    for (int t = 0; t < n; ++t) {
        s[t] = dot_bf16(q, K[t], d) * scale;
        if (s[t] > m) m = s[t];
    }
    double l = 0.0;
    for (int t = 0; t < n; ++t) { s[t] = exp(s[t] - m); l += s[t]; }
    for (int e = 0; e < d; ++e) {
        double acc = 0.0;
        for (int t = 0; t < n; ++t) acc += s[t] * bf(V[t][e]);
        out[e] = acc / l;
    }
    free(s);
}

/* SiLU(z) = z / (1 + e^-z). */
double orc_silu(double z) { return z / (1.0 + exp(-z)); }

/* Greedy argmax: first index of the maximum (ties go to the lowest index). */
int orc_argmax_f32(const float *v, int n)
{
    int best = 0;
    for (int i = 1; i < n; ++i)
        if (v[i] > v[best]) best = i;
    return best;
}

/* ------------------------------------------------------------------------ */
/* Model description.  Weights are host bf16 arrays in Linear layout.       */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
    int32_t n_experts, top_k, expert_ffn;   /* all zero for a dense model */
    double rms_eps, rope_theta;
} orc_cfg;

typedef struct {
    const uint16_t *embed;        /* [V, H] */
    const uint16_t *final_norm;   /* [H] */
    const uint16_t *lm_head;      /* [V, H] */
    const uint16_t *const *attn_norm;     /* [L] -> [H] */
    const uint16_t *const *w_qkv;         /* [L] -> [(nq + 2 nkv) d, H]: q rows, k rows, v rows */
    const uint16_t *const *w_o;           /* [L] -> [H, nq d] */
    const uint16_t *const *mlp_norm;      /* [L] -> [H] */
    const uint16_t *const *w_gate_up;     /* [L] -> [2F, H], gate rows first */
    const uint16_t *const *w_down;        /* [L] -> [H, F] */
    const uint16_t *const *w_router;      /* [L] -> [E, H] */
    const uint16_t *const *w_exp_gate_up; /* [L] -> [E, 2Fe, H] */
    const uint16_t *const *w_exp_down;    /* [L] -> [E, H, Fe] */
} orc_weights;

enum { ORC_KV_CONTIGUOUS = 0, ORC_KV_PAGED = 1 };

/* KV cache layout (the library's contract).  Keys and values are stored by
 * token:
 *   contiguous: K, V [slot, kvh, t, d]
 *   paged:      K, V [page, kvh, t % ps, d]
 * with page = page_table[slot, t / ps]. */
typedef struct {
    int32_t layout;
    int32_t n_slots, max_seq_len;
    int32_t page_size, num_pages, max_pages_per_seq;
    uint16_t *const *k;                  /* [L] -> cache */
    uint16_t *const *v;
    const int32_t *page_table;           /* [n_slots, max_pages_per_seq], paged only */
} orc_kv;

/* Address of the key d-vector of (layer, slot, kv head, token position). */
static uint16_t *k_row(const orc_cfg *c, const orc_kv *kv, int layer, int slot, int kvh, int t)
{
    int64_t d = c->head_dim;
    if (kv->layout == ORC_KV_PAGED) {
        int32_t page = kv->page_table[(int64_t)slot * kv->max_pages_per_seq + t / kv->page_size];
        return kv->k[layer] + (((int64_t)page * c->n_kv_heads + kvh) * kv->page_size + t % kv->page_size) * d;
    }
    return kv->k[layer] + (((int64_t)slot * c->n_kv_heads + kvh) * kv->max_seq_len + t) * d;
}

/* Address of value element e of (layer, slot, kv head, token position):
 * values are stored by token, like keys. */
static uint16_t *v_elem(const orc_cfg *c, const orc_kv *kv, int layer, int slot, int kvh, int t, int e)
{
    int64_t d = c->head_dim;
    if (kv->layout == ORC_KV_PAGED) {
        int32_t page = kv->page_table[(int64_t)slot * kv->max_pages_per_seq + t / kv->page_size];
        return kv->v[layer] + (((int64_t)page * c->n_kv_heads + kvh) * kv->page_size + t % kv->page_size) * d + e;
    }
    return kv->v[layer] + (((int64_t)slot * c->n_kv_heads + kvh) * kv->max_seq_len + t) * d + e;
}

/* ------------------------------------------------------------------------ */
/* One decoder layer's pieces for a single token row.                       */
/* ------------------------------------------------------------------------ */

/* Attention sub-layer for one token at position pos: RMSNorm, QKV
 * projection, rotary embedding, KV append at pos, grouped-query attention
 * over keys 0..pos, output projection added to the fp32 residual x. */
static void attn_block(const orc_cfg *c, const orc_weights *w, const orc_kv *kv,
                       int layer, int slot, int pos, float *x)
{
    int H = c->hidden, d = c->head_dim, nq = c->n_heads, nkv = c->n_kv_heads;
    int nqkv = (nq + 2 * nkv) * d;
    int group = nq / nkv;
    uint16_t *h = malloc(sizeof(uint16_t) * H);
    double *acc = malloc(sizeof(double) * (nqkv > H ? nqkv : H));
    uint16_t *qkv = malloc(sizeof(uint16_t) * nqkv);
    double *tmp = malloc(sizeof(double) * 2 * d);
    uint16_t *o = malloc(sizeof(uint16_t) * nq * d);

    orc_rmsnorm(x, H, w->attn_norm[layer], c->rms_eps, h);
    orc_linear(h, H, w->w_qkv[layer], nqkv, acc);
    for (int j = 0; j < nqkv; ++j) qkv[j] = tobf(acc[j]);

    /* rotary embedding on the nq query heads and the nkv key heads */
    for (int hd = 0; hd < nq + nkv; ++hd) {
        uint16_t *v = qkv + hd * d;
        for (int e = 0; e < d; ++e) tmp[e] = bf(v[e]);
        orc_rope(tmp, d, pos, c->rope_theta, tmp + d);
        for (int e = 0; e < d; ++e) v[e] = tobf(tmp[d + e]);
    }
    /* append this token's k and v at position pos */
    for (int g = 0; g < nkv; ++g) {
        memcpy(k_row(c, kv, layer, slot, g, pos), qkv + (nq + g) * d, sizeof(uint16_t) * d);
        for (int e = 0; e < d; ++e) *v_elem(c, kv, layer, slot, g, pos, e) = qkv[(nq + nkv + g) * d + e];
    }
    /* each query head attends over keys 0..pos of its kv group */
    int n = pos + 1;
#pragma omp parallel for schedule(static)
    for (int hq = 0; hq < nq; ++hq) {
        int g = hq / group;
        const uint16_t **K = malloc(sizeof(*K) * n);
        const uint16_t **V = malloc(sizeof(*V) * n);
        uint16_t *vrows = malloc(sizeof(uint16_t) * (size_t)n * d);   /* value rows gathered by token */
        double *out = malloc(sizeof(double) * d);
        for (int t = 0; t < n; ++t) {
            K[t] = k_row(c, kv, layer, slot, g, t);
            for (int e = 0; e < d; ++e) vrows[(size_t)t * d + e] = *v_elem(c, kv, layer, slot, g, t, e);
            V[t] = vrows + (size_t)t * d;
        }
        orc_attention(qkv + hq * d, K, V, n, d, out);
        for (int e = 0; e < d; ++e) o[hq * d + e] = tobf(out[e]);
        free(K); free(V); free(vrows); free(out);
    }
    orc_linear(o, nq * d, w->w_o[layer], H, acc);
    for (int i = 0; i < H; ++i) x[i] = (float)((double)x[i] + acc[i]);

    free(h); free(acc); free(qkv); free(tmp); free(o);
}

/* SwiGLU feed-forward on a normed row h: g, u = bf16(W_gu h),
 * a = bf16(silu(g) * u), y = W_down a (fp64, not rounded). */
static void swiglu_mlp(const uint16_t *h, int H, int F, const uint16_t *Wgu,
                       const uint16_t *Wd, double *y)
{
    double *gu = malloc(sizeof(double) * 2 * F);
    uint16_t *a = malloc(sizeof(uint16_t) * F);
    orc_linear(h, H, Wgu, 2 * F, gu);
    for (int j = 0; j < F; ++j) {
        double g = bf(tobf(gu[j]));
        double u = bf(tobf(gu[F + j]));
        a[j] = tobf(orc_silu(g) * u);
    }
    orc_linear(a, F, Wd, H, y);
    free(gu); free(a);
}

/* Router: softmax over all experts of the fp64 router logits, the top_k
 * largest probabilities (ties go to the lower expert id), renormalised.
 * Returns the chosen experts in rank order and their weights. */
void orc_route(const double *logits, int E, int top_k, int32_t *sel, double *wsel)
{
    double m = -INFINITY;
    for (int e = 0; e < E; ++e) if (logits[e] > m) m = logits[e];
    double *p = malloc(sizeof(double) * E);
    char *used = calloc((size_t)E, 1);
    double z = 0.0;
    for (int e = 0; e < E; ++e) { p[e] = exp(logits[e] - m); z += p[e]; }
    for (int e = 0; e < E; ++e) p[e] /= z;
    double s = 0.0;
    for (int r = 0; r < top_k; ++r) {
        int best = -1;
        for (int e = 0; e < E; ++e)
            if (!used[e] && (best < 0 || p[e] > p[best])) best = e;
        used[best] = 1;
        sel[r] = best;
        wsel[r] = p[best];
        s += p[best];
    }
    for (int r = 0; r < top_k; ++r) wsel[r] /= s;
    free(p); free(used);
}

/* Routing that follows a given expert set instead of the top_k: the same
 * softmax over all experts, the chosen experts' probabilities renormalised
 * over the given set, combined in the given order.  (A top-k choice is a
 * comparison of floating-point logits; where two logits are closer than a
 * computation's error, either choice is a correct result, and a test uses
 * this to follow the choice another computation made.)  Returns -1 unless
 * the set holds top_k distinct ids in [0, E). */
int orc_route_forced(const double *logits, int E, int top_k, const int32_t *force, double *wsel)
{
    for (int r = 0; r < top_k; ++r) {
        if (force[r] < 0 || force[r] >= E) return -1;
        for (int q = 0; q < r; ++q)
            if (force[q] == force[r]) return -1;
    }
    double m = -INFINITY;
    for (int e = 0; e < E; ++e) if (logits[e] > m) m = logits[e];
    double z = 0.0;
    for (int e = 0; e < E; ++e) z += exp(logits[e] - m);
    double s = 0.0;
    for (int r = 0; r < top_k; ++r) {
        wsel[r] = exp(logits[force[r]] - m) / z;
        s += wsel[r];
    }
    for (int r = 0; r < top_k; ++r) wsel[r] /= s;
    return 0;
}

/* Per-row routing controls and records of one MoE layer (all optional):
 * force [top_k] = follow this expert set; logits_out [E] = the router
 * logits; sel_out [top_k] = the oracle's own top_k choice. */
typedef struct {
    const int32_t *force;
    double *logits_out;
    int32_t *sel_out;
} orc_route_io;

/* Feed-forward sub-layer for one row: RMSNorm, then either the dense SwiGLU
 * MLP or the routed mixture of SwiGLU experts, added to the residual x.
 * Returns -1 if a forced expert set is malformed. */
static int mlp_block(const orc_cfg *c, const orc_weights *w, int layer, float *x, orc_route_io io)
{
    int rc = 0;
    int H = c->hidden;
    uint16_t *h = malloc(sizeof(uint16_t) * H);
    double *y = malloc(sizeof(double) * H);
    orc_rmsnorm(x, H, w->mlp_norm[layer], c->rms_eps, h);
    if (c->n_experts == 0) {
        swiglu_mlp(h, H, c->ffn, w->w_gate_up[layer], w->w_down[layer], y);
        for (int i = 0; i < H; ++i) x[i] = (float)((double)x[i] + y[i]);
    } else {
        int E = c->n_experts, K = c->top_k, Fe = c->expert_ffn;
        double *rl = malloc(sizeof(double) * E);
        int32_t *sel = malloc(sizeof(int32_t) * K);
        double *ws = malloc(sizeof(double) * K);
        double *acc = calloc((size_t)H, sizeof(double));
        orc_linear(h, H, w->w_router[layer], E, rl);
        orc_route(rl, E, K, sel, ws);
        if (io.logits_out) memcpy(io.logits_out, rl, sizeof(double) * E);
        if (io.sel_out) memcpy(io.sel_out, sel, sizeof(int32_t) * K);
        if (io.force) {
            rc = orc_route_forced(rl, E, K, io.force, ws);
            memcpy(sel, io.force, sizeof(int32_t) * K);
        }
        for (int r = 0; r < K; ++r) {     /* combine in rank order */
            int e = sel[r];
            swiglu_mlp(h, H, Fe, w->w_exp_gate_up[layer] + (int64_t)e * 2 * Fe * H,
                       w->w_exp_down[layer] + (int64_t)e * H * Fe, y);
            for (int i = 0; i < H; ++i) acc[i] += ws[r] * y[i];
        }
        for (int i = 0; i < H; ++i) x[i] = (float)((double)x[i] + acc[i]);
        free(rl); free(sel); free(ws); free(acc);
    }
    free(h); free(y);
    return rc;
}

static void lm_head(const orc_cfg *c, const orc_weights *w, const float *x, double *logits)
{
    uint16_t *h = malloc(sizeof(uint16_t) * c->hidden);
    orc_rmsnorm(x, c->hidden, w->final_norm, c->rms_eps, h);
    orc_linear(h, c->hidden, w->lm_head, c->vocab, logits);
    free(h);
}

/* ------------------------------------------------------------------------ */
/* Request-local decode function d(z) (Sec. IV, "Determinism Argument"):    */
/* one token of one request at position pos (= tokens already cached),      */
/* appending its k, v at pos in every layer and returning fp64 logits.      */
/* ------------------------------------------------------------------------ */
/* As orc_decode_row, for a mixture of experts with routing controls per
 * layer (each optional): force [L][top_k] = the expert set layer l follows
 * (its own top_k where NULL), router_logits [L][E] and own_sel [L][top_k]
 * receive each layer's router logits and own top_k choice. */
int orc_decode_row_routed(const orc_cfg *c, const orc_weights *w, const orc_kv *kv, int slot, int token,
                          int pos, double *logits, const int32_t *force, double *router_logits,
                          int32_t *own_sel)
{
    if (token < 0 || token >= c->vocab || pos < 0) return -1;
    int H = c->hidden, E = c->n_experts, K = c->top_k;
    float *x = malloc(sizeof(float) * H);
    int rc = 0;
    for (int i = 0; i < H; ++i) x[i] = (float)bf(w->embed[(int64_t)token * H + i]);
    for (int l = 0; l < c->n_layers && !rc; ++l) {
        orc_route_io io = {force ? force + (int64_t)l * K : NULL,
                           router_logits ? router_logits + (int64_t)l * E : NULL,
                           own_sel ? own_sel + (int64_t)l * K : NULL};
        attn_block(c, w, kv, l, slot, pos, x);
        rc = mlp_block(c, w, l, x, io);
    }
    if (!rc) lm_head(c, w, x, logits);
    free(x);
    return rc;
}

int orc_decode_row(const orc_cfg *c, const orc_weights *w, const orc_kv *kv,
                   int slot, int token, int pos, double *logits)
{
    return orc_decode_row_routed(c, w, kv, slot, token, pos, logits, NULL, NULL, NULL);
}

/* The padded decode step at batch size B, computed row by row: each live row
 * (valid != 0) is d(z) of its own request; padding rows are skipped and get
 * next = -1 (Sec. IV, "Fixed-Shape Batched Decode": padding is masked).
 * logits: [B, V] fp64, padding rows left untouched.  The greedy choice is the
 * first maximum of the logits rounded to fp32, the precision the GPU's
 * sampler compares in (Sec. IV, "Shape-Aligned Sampling"; greedy = S with no
 * random variate). */
int orc_decode_batch(const orc_cfg *c, const orc_weights *w, const orc_kv *kv, int B,
                     const int32_t *tokens, const uint8_t *valid, const int32_t *seq_lens,
                     double *logits, int32_t *next)
{
    float *lf = malloc(sizeof(float) * c->vocab);
    int rc = 0;
    for (int b = 0; b < B; ++b) {
        next[b] = -1;
        if (!valid[b]) continue;
        double *lg = logits + (int64_t)b * c->vocab;
        rc = orc_decode_row(c, w, kv, b, tokens[b], seq_lens[b], lg);
        if (rc) break;
        for (int v = 0; v < c->vocab; ++v) lf[v] = (float)lg[v];
        next[b] = orc_argmax_f32(lf, c->vocab);
    }
    free(lf);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Isolated prefill (Sec. IV, "Isolated Prefill"; the base case of the       */
/* determinism argument): the prompt alone, all positions of a layer before  */
/* the next layer, writing KV for positions 0..Lp-1 of `slot`, and logits of  */
/* the last position only (Sec. IV, "Shape-Aligned Sampling").  Each row's   */
/* sums run in the same order as in orc_decode_row, so prefill(p ++ [t]) at  */
/* its last row equals prefill(p) followed by decode(t), bit for bit.        */
/* ------------------------------------------------------------------------ */
/* As orc_prefill, with the routing controls of orc_decode_row_routed for
 * every (layer, position): force [L][Lp][top_k], router_logits [L][Lp][E],
 * own_sel [L][Lp][top_k], each optional. */
int orc_prefill_routed(const orc_cfg *c, const orc_weights *w, const orc_kv *kv, int slot,
                       const int32_t *prompt, int Lp, double *logits, int32_t *token_out,
                       const int32_t *force, double *router_logits, int32_t *own_sel)
{
    if (Lp <= 0) return -1;
    for (int t = 0; t < Lp; ++t)
        if (prompt[t] < 0 || prompt[t] >= c->vocab) return -1;
    int H = c->hidden, E = c->n_experts, K = c->top_k;
    float *X = malloc(sizeof(float) * (int64_t)Lp * H);
    for (int t = 0; t < Lp; ++t)
        for (int i = 0; i < H; ++i)
            X[(int64_t)t * H + i] = (float)bf(w->embed[(int64_t)prompt[t] * H + i]);
    int rc = 0;
    for (int l = 0; l < c->n_layers && !rc; ++l) {
        /* positions in order: position t reads keys 0..t of this layer,
         * which positions 0..t have already written */
        for (int t = 0; t < Lp; ++t) attn_block(c, w, kv, l, slot, t, X + (int64_t)t * H);
        for (int t = 0; t < Lp && !rc; ++t) {
            int64_t at = (int64_t)l * Lp + t;
            orc_route_io io = {force ? force + at * K : NULL, router_logits ? router_logits + at * E : NULL,
                               own_sel ? own_sel + at * K : NULL};
            rc = mlp_block(c, w, l, X + (int64_t)t * H, io);
        }
    }
    if (rc) {
        free(X);
        return rc;
    }
    lm_head(c, w, X + (int64_t)(Lp - 1) * H, logits);
    float *lf = malloc(sizeof(float) * c->vocab);
    for (int v = 0; v < c->vocab; ++v) lf[v] = (float)logits[v];
    *token_out = orc_argmax_f32(lf, c->vocab);
    free(lf);
    free(X);
    return 0;
}

int orc_prefill(const orc_cfg *c, const orc_weights *w, const orc_kv *kv, int slot,
                const int32_t *prompt, int Lp, double *logits, int32_t *token_out)
{
    return orc_prefill_routed(c, w, kv, slot, prompt, Lp, logits, token_out, NULL, NULL, NULL);
}

/* ---------------------------------------------------------------------------
 * Request-bound seeded sampling (Sec. IV, "Shape-Aligned Sampling"; the
 * determinism argument's y_t = S(l_t, R(s, t)), Sec. IV "Determinism
 * Argument").  The paper fixes the properties -- the random variate is a
 * function of the request's seed s and step t only, padding consumes
 * nothing, identical logits and variate give the identical token -- but not
 * the generator or the rule.  Reading used here:
 *   R(s, t) = { u_v : v < V }, u_v from Philox4x32-10 keyed by the 64-bit
 *             seed with counter (t, v, 0, 0), t = the position of the token
 *             being sampled (a function of the request's own state);
 *   S(l, R) = argmax_v ( l_v / T + g_v ), g_v = -ln(-ln u_v)  (Gumbel-max:
 *             an exact draw from softmax(l / T)); ties to the lower index;
 *             T <= 0 is the greedy rule (no noise).
 * Decision and log-probability in fp64.
 * ------------------------------------------------------------------------- */

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011): ten rounds over four 32-bit words; each round
 * takes the two 64-bit products M0 c0 and M1 c2 and sets
 *   (c0, c1, c2, c3) <- (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)),
 * the key advancing by the Weyl constants (W0, W1) before every round but
 * the first. */
void orc_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out)
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t p0 = (uint64_t)M0 * c0, p1 = (uint64_t)M1 * c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0, n1 = (uint32_t)p1;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1, n3 = (uint32_t)p0;
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* A uniform double strictly inside (0, 1) from 52 bits of two words:
 * ((w0 >> 6) 2^26 + (w1 >> 6) + 1/2) 2^-52, in [2^-53, 1 - 2^-53] (every
 * value exactly representable: the integer part needs 53 bits). */
double orc_uniform(uint32_t w0, uint32_t w1)
{
    return ((double)(w0 >> 6) * 67108864.0 + (double)(w1 >> 6) + 0.5) * (1.0 / 4503599627370496.0);
}

/* u_v and g_v of R(s, t) for one column v. */
double orc_gumbel(uint64_t seed, int32_t t, int32_t v)
{
    const uint32_t ctr[4] = {(uint32_t)t, (uint32_t)v, 0u, 0u};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    orc_philox4x32_10(ctr, key, w);
    return -log(-log(orc_uniform(w[0], w[1])));
}

/* S(l, R(s, t)) for one row of V logits; the log-probability of the chosen
 * token under softmax(l / T) (softmax(l) when T <= 0), sums sequential in v. */
int orc_sample(const float *logits, int V, uint64_t seed, int32_t t, float temperature, int32_t *token,
               double *logprob)
{
    if (V <= 0) return -1;
    const int greedy = !(temperature > 0.0f);
    const double T = greedy ? 1.0 : (double)temperature;
    int best = 0;
    double bz = -INFINITY, M = -INFINITY;
    for (int v = 0; v < V; ++v) {
        const double x = (double)logits[v] / T;
        const double z = greedy ? x : x + orc_gumbel(seed, t, v);
        if (z > bz) {
            bz = z;
            best = v;
        }
        if (x > M) M = x;
    }
    double S = 0.0;
    for (int v = 0; v < V; ++v) S += exp((double)logits[v] / T - M);
    *token = best;
    *logprob = (double)logits[best] / T - M - log(S);
    return 0;
}

void orc_set_threads(int n)
{
#ifdef _OPENMP
    omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
