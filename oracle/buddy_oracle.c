/*
 * buddy_oracle.c -- TEST INFRASTRUCTURE ONLY: the CPU reference ("oracle")
 * of BUDDY's budget-routed decode step (arXiv 2606.09514).
 *
 * Only tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  It shares no code, header or table with the GPU
 * library.  Everything is computed in IEEE double with plain loops in the
 * order the method states it; OpenMP only splits independent output rows, so
 * results do not depend on the thread count.
 *
 * Paper passages followed (section / equation of the paper):
 *   - layer skipping, Sec. 3.1 Eq. (1): a skipped block is the identity on H;
 *   - first and last blocks always run, k = round(b L) - 2 routable blocks,
 *     Sec. 4.2.1 and Eq. (2); the start-layer ablation of Sec. 4.3 moves the
 *     router after the first S blocks, which then all run;
 *   - score fusion s' = s + omega p~ and top-k selection, Eq. (2);
 *   - two-layer MLP scorer over pooled context, Sec. 4.2.3 and App. C.1;
 *   - KV-aware planner: the first layer's KV cache plus the newest token as
 *     the router context, Sec. 4.3;
 *   - skipped layers store zero-filled K/V, Sec. 6 (limitations);
 *   - decode attention over the cache with the new token appended,
 *     App. "Background" (prefill vs decode, KV-cache equation);
 *   - the Llama-style block (Q/K/V/O projections, attention, d -> d_c -> d
 *     MLP), App. C.2.
 * Readings where the paper is silent are listed at each function.
 */
#include "buddy_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------ start layer */

int orc_start_layer(const orc_config* c)
{
    return c->start_layer > 0 ? c->start_layer : 1;
}

int orc_n_mid(const orc_config* c)
{
    return c->n_layers - 1 - orc_start_layer(c);
}

/* ---------------------------------------------------------------- storage */

static double ld(const void* p, size_t i, int dtype)
{
    if (dtype == ORC_BF16) {
        uint32_t bits = (uint32_t)((const uint16_t*)p)[i] << 16;
        float f;
        memcpy(&f, &bits, 4);
        return (double)f;
    }
    return (double)((const float*)p)[i];
}

uint16_t orc_bf16_from_double(double x)
{
    if (isnan(x)) return 0x7FC0;
    /* bf16 keeps 8 significant bits; exponent range as fp32.  Round the
     * exact value to the nearest representable value, ties to even, by
     * scaling onto an integer grid and using the current (nearest-even)
     * rounding mode of nearbyint. */
    double ax = fabs(x), r;
    if (ax == 0.0 || isinf(x)) {
        r = ax;
    } else {
        int e;
        frexp(ax, &e);                 /* ax = m 2^e, 0.5 <= m < 1 */
        int q = e - 8;                 /* quantum of the 8-bit significand */
        if (q < -133) q = -133;        /* subnormal bf16 quantum is 2^-133 */
        r = ldexp(nearbyint(ldexp(ax, -q)), q);
        if (r > 3.3895313892515355e38) r = INFINITY; /* beyond max finite */
    }
    float f = (float)r;                /* exact: r is a bf16 value */
    uint32_t bits;
    memcpy(&bits, &f, 4);
    bits >>= 16;
    if (x < 0 || (x == 0 && signbit(x))) bits |= 0x8000;
    return (uint16_t)bits;
}

static void st(void* p, size_t i, int dtype, double v)
{
    if (dtype == ORC_BF16)
        ((uint16_t*)p)[i] = orc_bf16_from_double(v);
    else
        ((float*)p)[i] = (float)v;
}


/* Routed prefill, one route per prompt: the Reuse setting of Sec. 5 keeps
 * the decode path at the prefill's decision, so the prefill itself is
 * routed.  Within a block the tokens run in order, each attending to the
 * rows its predecessors appended, which is the causal prefill of that
 * block. */
int orc_prefill_seq(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                    void* const* kc, void* const* vc, uint8_t* const* exec, int32_t len,
                    int32_t k_budget, const uint8_t* route, const float* x, double* h_out,
                    uint8_t* mask_out, float* scores_out, double* margin_out)
{
    const int L = c->n_layers, S = orc_start_layer(c), Lm = orc_n_mid(c);
    const int d = c->d_model, dt = c->dtype;
    const int nkv = c->n_kv_heads, hd = c->head_dim, T = c->max_ctx;
    if (L < 2 || Lm < 0 || len < 1 || len > T || k_budget < 0 || k_budget > Lm) return -1;
    if (!route && !dm) return -1;
    uint8_t* mask = malloc((size_t)(Lm > 0 ? Lm : 1));
    float* sc = malloc(sizeof(float) * (Lm > 0 ? Lm : 1));
    double margin = INFINITY;
    for (size_t i = 0; i < (size_t)len * d; ++i) h_out[i] = (double)x[i];

    /* the always-run leading blocks over the prompt */
    for (int l = 0; l < S; ++l)
        for (int t = 0; t < len; ++t) {
            if (exec) exec[l][t] = 1;
            orc_block_ex(c, &layers[l], kc[l], vc[l], t, h_out + (size_t)t * d,
                         exec ? exec[l] : NULL);
        }
    /* one route for the prompt: planner at the last token */
    if (route) {
        for (int i = 0; i < Lm; ++i) mask[i] = route[i] ? 1 : 0;
    } else {
        double* z = malloc(sizeof(double) * orc_context_dim(c));
        orc_router_context(c, kc[S - 1], vc[S - 1], len - 1, h_out + (size_t)(len - 1) * d, z);
        orc_dm_scores(c, dm, z, sc);
        orc_topk(sc, Lm, k_budget, mask, &margin);
        free(z);
        if (scores_out) memcpy(scores_out, sc, sizeof(float) * Lm);
        if (mask_out) memcpy(mask_out, mask, (size_t)Lm);
    }
    /* selected blocks causally over the prompt, skipped ones zero-filled */
    for (int l = S; l < L; ++l) {
        const int run = l == L - 1 || mask[l - S];
        for (int t = 0; t < len; ++t) {
            if (exec) exec[l][t] = (uint8_t)run;
            if (run) {
                orc_block_ex(c, &layers[l], kc[l], vc[l], t, h_out + (size_t)t * d,
                             exec ? exec[l] : NULL);
            } else {
                for (int g = 0; g < nkv; ++g)
                    for (int i = 0; i < hd; ++i) {
                        size_t at = ((size_t)g * T + t) * hd + i;
                        st(kc[l], at, dt, 0.0);
                        st(vc[l], at, dt, 0.0);
                    }
            }
        }
    }
    if (margin_out) *margin_out = margin;
    free(mask); free(sc);
    return 0;
}

/* ------------------------------------------------------------ prior (App. B) */

static int cmp_double(const void* a, const void* b)
{
    const double x = *(const double*)a, y = *(const double*)b;
    return (x > y) - (x < y);
}

/* Percentile at fraction q of n sorted values: the order statistic at
 * q (n - 1), interpolated linearly between its two neighbours. */
static double percentile_sorted(const double* s, int32_t n, double q)
{
    double at = q * (double)(n - 1);
    int32_t i = (int32_t)at;
    if (i >= n - 1) return s[n - 1];
    return s[i] + (at - (double)i) * (s[i + 1] - s[i]);
}

typedef struct { double v; int32_t i; } orc_keyed;

static int cmp_keyed(const void* a, const void* b)
{
    const orc_keyed* x = (const orc_keyed*)a;
    const orc_keyed* y = (const orc_keyed*)b;
    if (x->v != y->v) return (x->v > y->v) - (x->v < y->v);
    return (x->i > y->i) - (x->i < y->i);
}

void orc_prior_normalize(const double* raw, int32_t n, int32_t kind, double winsor,
                         double* out)
{
    double* x = malloc(sizeof(double) * n);
    double* s = malloc(sizeof(double) * n);
    orc_keyed* kz = malloc(sizeof(orc_keyed) * n);
    /* (i) direction: larger means more important; (ii) heavy tails */
    for (int32_t l = 0; l < n; ++l) {
        if (kind == 2) {
            x[l] = 1.0 - raw[l];                  /* cosine dissimilarity, identity */
        } else {
            double v = raw[l] > 0.0 ? raw[l] : 0.0; /* max{0, .} / clip to >= 0 */
            x[l] = log(1.0 + v);
        }
    }
    /* (iii) robust z-score with median and interquartile range */
    memcpy(s, x, sizeof(double) * n);
    qsort(s, n, sizeof(double), cmp_double);
    double med = percentile_sorted(s, n, 0.5);
    double iqr = percentile_sorted(s, n, 0.75) - percentile_sorted(s, n, 0.25);
    for (int32_t l = 0; l < n; ++l) {
        double z = (x[l] - med) / (iqr + 1e-6);
        if (winsor > 0.0) z = z < -winsor ? -winsor : (z > winsor ? winsor : z);
        kz[l].v = z;
        kz[l].i = l;
    }
    /* (iv) rank normalisation: sort, each run of equal values gets the mean
     * of the ranks it spans, u = (1 + rank) / (n + 1) */
    qsort(kz, n, sizeof(orc_keyed), cmp_keyed);
    for (int32_t a = 0; a < n;) {
        int32_t b = a;
        while (b + 1 < n && kz[b + 1].v == kz[a].v) ++b;
        double rank = 0.5 * (double)(a + b);
        for (int32_t t = a; t <= b; ++t) out[kz[t].i] = (1.0 + rank) / (double)(n + 1);
        a = b + 1;
    }
    /* Eq. 2: p~ = (p - mu(p)) / (sigma(p) + eps) with p = u */
    double mu = 0.0, var = 0.0;
    for (int32_t l = 0; l < n; ++l) mu += out[l];
    mu /= n;
    for (int32_t l = 0; l < n; ++l) var += (out[l] - mu) * (out[l] - mu);
    double sigma = sqrt(var / n);
    for (int32_t l = 0; l < n; ++l) out[l] = (out[l] - mu) / (sigma + 1e-6);
    free(x); free(s); free(kz);
}
/* ------------------------------------------------------- path grouping */

/* Batch-level path grouping (the Conclusion names grouping requests by their
 * path among the open questions of path and KV handling): the sequences of a
 * batch are ordered by route and those with identical routes form a group.
 * A route is a sequence's mask row over the routable blocks, read as run
 * (nonzero byte) or skip (zero); routes compare lexicographically in block
 * order with skip before run, and sequences with equal routes keep their
 * batch order (a stable sort).  Reading: the paper gives no order; this one
 * is fixed so that the result is unique. */
static int route_before(const uint8_t* mask, int32_t n, int32_t a, int32_t b)
{
    for (int32_t i = 0; i < n; ++i) {
        const int ra = mask[(size_t)a * n + i] != 0, rb = mask[(size_t)b * n + i] != 0;
        if (ra != rb) return ra < rb;
    }
    return a < b;
}

int32_t orc_group_by_route(const uint8_t* mask, int32_t B, int32_t n, int32_t* perm,
                           int32_t* starts)
{
    if (B < 0 || n < 1) return -1;
    /* insertion sort of the sequence indices: plain and stable */
    for (int32_t b = 0; b < B; ++b) {
        int32_t j = b;
        while (j > 0 && route_before(mask, n, b, perm[j - 1])) {
            perm[j] = perm[j - 1];
            --j;
        }
        perm[j] = b;
    }
    int32_t groups = 0;
    for (int32_t i = 0; i < B; ++i) {
        int same = i > 0;
        for (int32_t k = 0; same && k < n; ++k)
            same = (mask[(size_t)perm[i] * n + k] != 0) == (mask[(size_t)perm[i - 1] * n + k] != 0);
        if (!same) starts[groups++] = i;
    }
    starts[groups] = B;
    return groups;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* y[o] = sum_k W[row0 + o][k] x[k], o < rows; W row-major with `cols` columns. */
static void matvec(const void* W, int dtype, int64_t row0, int64_t rows,
                   int64_t cols, const double* x, double* y)
{
#pragma omp parallel for schedule(static) if (rows * cols > 65536)
    for (int64_t o = 0; o < rows; ++o) {
        double acc = 0.0;
        size_t base = (size_t)(row0 + o) * (size_t)cols;
        for (int64_t k = 0; k < cols; ++k) acc += ld(W, base + k, dtype) * x[k];
        y[o] = acc;
    }
}

/* ------------------------------------------------------------------ block */

/* RMSNorm as used by Llama-style blocks (App. C.2 names the block layout;
 * the normalisation itself follows the Llama convention). */
void orc_rmsnorm(const orc_config* c, const double* h, const void* g, double* out)
{
    int d = c->d_model;
    double ss = 0.0;
    for (int i = 0; i < d; ++i) ss += h[i] * h[i];
    double inv = 1.0 / sqrt(ss / d + c->rms_eps);
    for (int i = 0; i < d; ++i) out[i] = h[i] * inv * ld(g, i, c->dtype);
}

/* Rotary position embedding, rotate-half pairing (i, i + hd/2) with angle
 * pos * theta^(-2i/hd).  The paper only names a Llama-style block; this is
 * the Llama convention. */
void orc_rope(const orc_config* c, double* x, int32_t pos)
{
    int half = c->head_dim / 2;
    for (int i = 0; i < half; ++i) {
        double inv_freq = pow(c->rope_theta, -2.0 * i / c->head_dim);
        double ang = (double)pos * inv_freq;
        double cs = cos(ang), sn = sin(ang);
        double a = x[i], b = x[i + half];
        x[i] = a * cs - b * sn;
        x[i + half] = b * cs + a * sn;
    }
}

static double act_silu(double x) { return x / (1.0 + exp(-x)); }
static double act_gelu(double x) { return 0.5 * x * (1.0 + erf(x / sqrt(2.0))); }

void orc_block(const orc_config* c, const orc_layer* w, void* kc, void* vc,
               int32_t pos, double* h)
{
    orc_block_ex(c, w, kc, vc, pos, h, NULL);
}

void orc_block_ex(const orc_config* c, const orc_layer* w, void* kc, void* vc,
                  int32_t pos, double* h, const uint8_t* exec)
{
    const int d = c->d_model, nq = c->n_heads, nkv = c->n_kv_heads;
    const int hd = c->head_dim, f = c->d_ffn, T = c->max_ctx, dt = c->dtype;
    const int nqkv = (nq + 2 * nkv) * hd;
    double* u = malloc(sizeof(double) * d);
    double* qkv = malloc(sizeof(double) * nqkv);
    double* o = malloc(sizeof(double) * nq * hd);
    double* y = malloc(sizeof(double) * (d > 2 * f ? d : 2 * f));
    double* m = malloc(sizeof(double) * f);
    double* p = malloc(sizeof(double) * (pos + 1));

    /* attention half: u = RMSNorm(h); [q;k;v] = Wqkv u; RoPE on q and k */
    orc_rmsnorm(c, h, w->attn_norm, u);
    matvec(w->wqkv, dt, 0, nqkv, d, u, qkv);
    double* q = qkv;
    double* kn = qkv + nq * hd;
    double* vn = qkv + (nq + nkv) * hd;
    for (int hh = 0; hh < nq; ++hh) orc_rope(c, q + hh * hd, pos);
    for (int g = 0; g < nkv; ++g) orc_rope(c, kn + g * hd, pos);

    /* KV-cache update: the new row is stored at pos in storage precision */
    for (int g = 0; g < nkv; ++g)
        for (int i = 0; i < hd; ++i) {
            size_t at = ((size_t)g * T + pos) * hd + i;
            st(kc, at, dt, kn[g * hd + i]);
            st(vc, at, dt, vn[g * hd + i]);
        }

    /* decode attention of each query head over positions 0..pos of its KV
     * group g = floor(h / (nq / nkv)), scale 1/sqrt(hd), softmax, sum p V;
     * with an execution map, positions at which this block did not run are
     * left out of the softmax (weight 0) */
    const double scale = 1.0 / sqrt((double)hd);
    const int grp = nq / nkv;
    for (int hh = 0; hh < nq; ++hh) {
        int g = hh / grp;
        double mx = -INFINITY;
        for (int j = 0; j <= pos; ++j) {
            if (exec && !exec[j]) continue;
            double s = 0.0;
            for (int i = 0; i < hd; ++i)
                s += q[hh * hd + i] * ld(kc, ((size_t)g * T + j) * hd + i, dt);
            p[j] = s * scale;
            if (p[j] > mx) mx = p[j];
        }
        double den = 0.0;
        for (int j = 0; j <= pos; ++j) {
            p[j] = (exec && !exec[j]) ? 0.0 : exp(p[j] - mx);
            den += p[j];
        }
        for (int i = 0; i < hd; ++i) {
            double acc = 0.0;
            for (int j = 0; j <= pos; ++j)
                acc += p[j] * ld(vc, ((size_t)g * T + j) * hd + i, dt);
            o[hh * hd + i] = acc / den;
        }
    }

    /* h <- h + Wo o */
    matvec(w->wo, dt, 0, d, nq * hd, o, y);
    for (int i = 0; i < d; ++i) h[i] += y[i];

    /* MLP half: h <- h + Wdown (SiLU(Wgate u2) * (Wup u2)), u2 = RMSNorm(h) */
    orc_rmsnorm(c, h, w->mlp_norm, u);
    matvec(w->wgate_up, dt, 0, 2 * (int64_t)f, d, u, y);
    for (int i = 0; i < f; ++i) m[i] = act_silu(y[i]) * y[f + i];
    matvec(w->wdown, dt, 0, d, f, m, y);
    for (int i = 0; i < d; ++i) h[i] += y[i];

    free(u); free(qkv); free(o); free(y); free(m); free(p);
}

/* ----------------------------------------------------------------- router */

/* KV-aware planner (Sec. 4.3): the first layer's cache (block S-1's under
 * the start-layer ablation), with the newest token's row already appended,
 * is averaged over positions 0..pos. */
void orc_pool(const orc_config* c, const void* kc, const void* vc, int32_t pos,
              double* z)
{
    const int nkv = c->n_kv_heads, hd = c->head_dim, T = c->max_ctx;
    const int n = nkv * hd;
    for (int g = 0; g < nkv; ++g)
        for (int i = 0; i < hd; ++i) {
            double sk = 0.0, sv = 0.0;
            for (int j = 0; j <= pos; ++j) {
                size_t at = ((size_t)g * T + j) * hd + i;
                sk += ld(kc, at, c->dtype);
                sv += ld(vc, at, c->dtype);
            }
            z[g * hd + i] = sk / (pos + 1);
            z[n + g * hd + i] = sv / (pos + 1);
        }
}


/* Router context variants: the feature G_t of Sec. 4.3 is K, V or K + V of
 * the first layer's cache, pooled over the prefix and the new row (the
 * concatenation [K | V] is the default context of this implementation), and
 * the newest token's hidden state after the first block follows it (the
 * planner "pools it together with the newest token representation"). */
int orc_context_dim(const orc_config* c)
{
    const int n = c->n_kv_heads * c->head_dim;
    return (c->router_ctx == ORC_CTX_KV ? 2 * n : n) + c->d_model;
}

void orc_router_context(const orc_config* c, const void* kc, const void* vc, int32_t pos,
                        const double* h, double* z)
{
    const int n = c->n_kv_heads * c->head_dim;
    double* kv = malloc(sizeof(double) * 2 * n);
    orc_pool(c, kc, vc, pos, kv);          /* [mean K | mean V] */
    int m = 0;
    switch (c->router_ctx) {
    case ORC_CTX_K:        for (int i = 0; i < n; ++i) z[m++] = kv[i]; break;
    case ORC_CTX_V:        for (int i = 0; i < n; ++i) z[m++] = kv[n + i]; break;
    case ORC_CTX_K_PLUS_V: for (int i = 0; i < n; ++i) z[m++] = kv[i] + kv[n + i]; break;
    default:               for (int i = 0; i < 2 * n; ++i) z[m++] = kv[i]; break;
    }
    for (int i = 0; i < c->d_model; ++i) z[m++] = h[i];
    free(kv);
}

/* Decision Module scorer (Sec. 4.2.3, App. C.1): Linear - act - Linear, then
 * the prior fusion of Eq. (2).  The softmax of Eq. (2) is monotone and is not
 * needed to select the top k. */
void orc_dm_scores(const orc_config* c, const orc_dm* dm, const double* z,
                   float* scores)
{
    const int H = c->dm_hidden, Lm = orc_n_mid(c);
    const int din = orc_context_dim(c);
    double* a = malloc(sizeof(double) * H);
    double* s = malloc(sizeof(double) * Lm);
    matvec(dm->w1, c->dtype, 0, H, din, z, a);
    for (int j = 0; j < H; ++j) {
        double x = a[j] + ld(dm->b1, j, c->dtype);
        a[j] = c->dm_act == ORC_ACT_GELU_ERF ? act_gelu(x) : act_silu(x);
    }
    matvec(dm->w2, c->dtype, 0, Lm, H, a, s);
    for (int i = 0; i < Lm; ++i) {
        double v = s[i] + ld(dm->b2, i, c->dtype);
        if (dm->prior) v += dm->omega * (double)dm->prior[i];
        scores[i] = (float)v;
    }
    free(a); free(s);
}

/* Budget Predictor (Sec. 4.4): k_hat = argmax over k in {1..L-2} of the
 * policy; the softmax of the policy is monotone, so the argmax of the
 * logits is taken. */
int32_t orc_predict_budget(const orc_config* c, const orc_predictor* p, const double* z,
                           float* logits, double* margin)
{
    const int H = p->hidden, Lm = orc_n_mid(c);
    const int din = orc_context_dim(c);
    double* a = malloc(sizeof(double) * H);
    double* s = malloc(sizeof(double) * Lm);
    matvec(p->w1, c->dtype, 0, H, din, z, a);
    for (int j = 0; j < H; ++j) {
        double x = a[j] + ld(p->b1, j, c->dtype);
        a[j] = c->dm_act == ORC_ACT_GELU_ERF ? act_gelu(x) : act_silu(x);
    }
    matvec(p->w2, c->dtype, 0, Lm, H, a, s);
    int best = -1;
    float top = 0.f, second = -INFINITY;
    for (int i = 0; i < Lm; ++i) {
        float v = (float)(s[i] + ld(p->b2, i, c->dtype));
        if (logits) logits[i] = v;
        if (v != v) continue;                            /* NaN never wins */
        if (best < 0 || v > top) { second = best < 0 ? -INFINITY : top; top = v; best = i; }
        else if (v > second) second = v;
    }
    if (margin) *margin = Lm > 1 ? (double)top - (double)second : INFINITY;
    free(a); free(s);
    return (best < 0 ? 0 : best) + 1;
}

/* Deterministic ordering for the hard top-k (Eq. 2): larger score first,
 * equal scores by lower layer index, NaN after every number. */
static const float* g_cmp_scores;  /* set only under the single-threaded qsort below */

static int cmp_rank(const void* pa, const void* pb)
{
    int32_t a = *(const int32_t*)pa, b = *(const int32_t*)pb;
    float sa = g_cmp_scores[a], sb = g_cmp_scores[b];
    int na = isnan(sa), nb = isnan(sb);
    if (na != nb) return na ? 1 : -1;
    if (!na && sa != sb) return sa > sb ? -1 : 1;
    return a < b ? -1 : (a > b ? 1 : 0);
}

int orc_topk(const float* scores, int32_t n, int32_t k, uint8_t* mask,
             double* margin)
{
    if (n < 0 || k < 0 || k > n) return -1;
    int32_t* order = malloc(sizeof(int32_t) * (n > 0 ? n : 1));
    for (int32_t i = 0; i < n; ++i) order[i] = i;
#pragma omp critical(orc_topk_sort)
    {
        g_cmp_scores = scores;
        qsort(order, (size_t)n, sizeof(int32_t), cmp_rank);
    }
    for (int32_t i = 0; i < n; ++i) mask[i] = 0;
    for (int32_t r = 0; r < k; ++r) mask[order[r]] = 1;
    if (margin) {
        if (k == 0 || k == n) *margin = INFINITY;
        else {
            double m = (double)scores[order[k - 1]] - (double)scores[order[k]];
            *margin = isnan(m) ? 0.0 : m;
        }
    }
    free(order);
    return 0;
}

/* ------------------------------------------------------------- decode step */

int orc_decode_seq(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                   void* const* kc, void* const* vc, int32_t pos, int32_t k_budget,
                   const uint8_t* route, const float* x, double* h_out,
                   uint8_t* mask_out, float* scores_out, double* margin_out,
                   int32_t* n_exec_out)
{
    return orc_decode_seq_ex(c, layers, dm, kc, vc, NULL, pos, k_budget, route, x, h_out,
                             mask_out, scores_out, margin_out, n_exec_out);
}

static int decode_core(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                       const orc_predictor* pred, void* const* kc, void* const* vc,
                       uint8_t* const* exec, int32_t pos, int32_t k_budget,
                       const uint8_t* route, const float* x, double* h_out,
                       uint8_t* mask_out, float* scores_out, double* margin_out,
                       int32_t* n_exec_out, int32_t* k_out, float* logits_out,
                       double* pmargin_out)
{
    const int L = c->n_layers, S = orc_start_layer(c), Lm = orc_n_mid(c);
    const int d = c->d_model, dt = c->dtype;
    const int nkv = c->n_kv_heads, hd = c->head_dim, T = c->max_ctx;
    if (L < 2 || Lm < 0 || pos < 0 || pos >= T) return -1;
    if (pred ? (route || Lm < 1) : (k_budget < 0 || k_budget > Lm)) return -1;
    if (!route && !dm) return -1;

    double* h = malloc(sizeof(double) * d);
    uint8_t* mask = malloc((size_t)(Lm > 0 ? Lm : 1));
    float* sc = malloc(sizeof(float) * (Lm > 0 ? Lm : 1));
    double margin = INFINITY;
    for (int i = 0; i < d; ++i) h[i] = (double)x[i];

    /* the first block always runs (Sec. 4.2.1), and so do the blocks before
     * the start layer; they append the newest token's K/V, which the planner
     * then sees */
    for (int l = 0; l < S; ++l) {
        if (exec) exec[l][pos] = 1;
        orc_block_ex(c, &layers[l], kc[l], vc[l], pos, h, exec ? exec[l] : NULL);
    }

    if (route) {
        for (int i = 0; i < Lm; ++i) mask[i] = route[i] ? 1 : 0;
    } else {
        /* router context: pooled features of block S-1's cache, newest
         * hidden after block S-1 */
        double* z = malloc(sizeof(double) * orc_context_dim(c));
        orc_router_context(c, kc[S - 1], vc[S - 1], pos, h, z);
        if (pred) {   /* no budget given: the predictor's k from the same context */
            k_budget = orc_predict_budget(c, pred, z, logits_out, pmargin_out);
            if (k_out) *k_out = k_budget;
        }
        orc_dm_scores(c, dm, z, sc);
        orc_topk(sc, Lm, k_budget, mask, &margin);
        free(z);
        if (scores_out) memcpy(scores_out, sc, sizeof(float) * Lm);
        if (mask_out) memcpy(mask_out, mask, (size_t)Lm);
    }

    /* routable blocks S..L-2, Eq. (1): run when selected; when skipped, h is
     * unchanged and the layer's K/V slot at pos is zero-filled (Sec. 6) */
    int n_exec = S;
    for (int l = S; l < L - 1; ++l) {
        if (exec) exec[l][pos] = mask[l - S] ? 1 : 0;
        if (mask[l - S]) {
            orc_block_ex(c, &layers[l], kc[l], vc[l], pos, h, exec ? exec[l] : NULL);
            ++n_exec;
        } else {
            for (int g = 0; g < nkv; ++g)
                for (int i = 0; i < hd; ++i) {
                    size_t at = ((size_t)g * T + pos) * hd + i;
                    st(kc[l], at, dt, 0.0);
                    st(vc[l], at, dt, 0.0);
                }
        }
    }
    if (exec) exec[L - 1][pos] = 1;
    orc_block_ex(c, &layers[L - 1], kc[L - 1], vc[L - 1], pos, h, exec ? exec[L - 1] : NULL);
    ++n_exec;

    memcpy(h_out, h, sizeof(double) * d);
    if (margin_out) *margin_out = margin;
    if (n_exec_out) *n_exec_out = n_exec;
    free(h); free(mask); free(sc);
    return 0;
}

int orc_decode_seq_ex(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                      void* const* kc, void* const* vc, uint8_t* const* exec, int32_t pos,
                      int32_t k_budget, const uint8_t* route, const float* x, double* h_out,
                      uint8_t* mask_out, float* scores_out, double* margin_out,
                      int32_t* n_exec_out)
{
    return decode_core(c, layers, dm, NULL, kc, vc, exec, pos, k_budget, route, x, h_out,
                       mask_out, scores_out, margin_out, n_exec_out, NULL, NULL, NULL);
}

int orc_decode_seq_auto(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                        const orc_predictor* pred, void* const* kc, void* const* vc,
                        uint8_t* const* exec, int32_t pos, const float* x, double* h_out,
                        int32_t* k_out, float* logits_out, double* pmargin_out,
                        uint8_t* mask_out, float* scores_out, double* margin_out,
                        int32_t* n_exec_out)
{
    if (!pred) return -1;
    return decode_core(c, layers, dm, pred, kc, vc, exec, pos, -1, NULL, x, h_out, mask_out,
                       scores_out, margin_out, n_exec_out, k_out, logits_out, pmargin_out);
}
