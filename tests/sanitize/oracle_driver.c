/*
 * Test driver for the CPU oracle under AddressSanitizer and
 * UndefinedBehaviorSanitizer (test infrastructure only).
 *
 * Runs every oracle entry point on tiny models in both storage dtypes, with
 * each buffer allocated at exactly the size the oracle's documentation
 * gives (one allocation per layer cache and per execution map), so that a
 * read or write past any of them is reported.  Values come from a fixed
 * linear congruential sequence; no result is checked here beyond the return
 * codes and the exact-budget invariant, which the Python pins cover in
 * depth.  Exit status 0 means every call returned as expected and the
 * sanitizers reported nothing (they abort the process on a finding).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/buddy_oracle.h"

static uint64_t g_state = 0x9e3779b97f4a7c15ull;

static double rnd(void) /* uniform in [-1, 1) */
{
    g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(g_state >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

static void* alloc_fill(size_t n, int dtype, double scale, double offset)
{
    if (dtype == ORC_BF16) {
        uint16_t* p = malloc(n * sizeof(uint16_t));
        for (size_t i = 0; i < n; ++i) p[i] = orc_bf16_from_double(offset + scale * rnd());
        return p;
    }
    float* p = malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = (float)(offset + scale * rnd());
    return p;
}

static int failures = 0;
#define EXPECT(cond, what)                                              \
    do {                                                                \
        if (!(cond)) { fprintf(stderr, "FAILED: %s\n", what); ++failures; } \
    } while (0)

static void run_model(int dtype, int start_layer, int router_ctx, int act)
{
    orc_config c;
    memset(&c, 0, sizeof(c));
    c.n_layers = 6; c.d_model = 32; c.n_heads = 4; c.n_kv_heads = 2; c.head_dim = 8;
    c.d_ffn = 48; c.dm_hidden = 16; c.dm_act = act; c.dtype = dtype; c.max_ctx = 12;
    c.rms_eps = 1e-5; c.rope_theta = 1e4; c.router_ctx = router_ctx;
    c.start_layer = start_layer;
    const int L = c.n_layers, d = c.d_model, hd = c.head_dim, nq = c.n_heads;
    const int nkv = c.n_kv_heads, f = c.d_ffn, T = c.max_ctx, H = c.dm_hidden;
    const int Lm = orc_n_mid(&c), din = orc_context_dim(&c);

    orc_layer* layers = malloc(sizeof(orc_layer) * L);
    for (int l = 0; l < L; ++l) {
        layers[l].attn_norm = alloc_fill(d, dtype, 0.02, 1.0);
        layers[l].wqkv = alloc_fill((size_t)(nq + 2 * nkv) * hd * d, dtype, 0.1, 0.0);
        layers[l].wo = alloc_fill((size_t)d * nq * hd, dtype, 0.1, 0.0);
        layers[l].mlp_norm = alloc_fill(d, dtype, 0.02, 1.0);
        layers[l].wgate_up = alloc_fill((size_t)2 * f * d, dtype, 0.1, 0.0);
        layers[l].wdown = alloc_fill((size_t)d * f, dtype, 0.1, 0.0);
    }
    float* prior = malloc(sizeof(float) * (Lm > 0 ? Lm : 1));
    for (int i = 0; i < Lm; ++i) prior[i] = (float)rnd();
    orc_dm dm = {alloc_fill((size_t)H * din, dtype, 0.1, 0.0), alloc_fill(H, dtype, 0.1, 0.0),
                 alloc_fill((size_t)Lm * H, dtype, 0.1, 0.0), alloc_fill(Lm, dtype, 0.1, 0.0),
                 prior, 0.1};
    orc_predictor pred = {alloc_fill((size_t)H * din, dtype, 0.1, 0.0),
                          alloc_fill(H, dtype, 0.1, 0.0),
                          alloc_fill((size_t)Lm * H, dtype, 0.1, 0.0),
                          alloc_fill(Lm, dtype, 0.1, 0.0), H};

    const size_t es = dtype == ORC_BF16 ? 2 : 4, per = (size_t)nkv * T * hd;
    void** kc = malloc(sizeof(void*) * L);
    void** vc = malloc(sizeof(void*) * L);
    uint8_t** ex = malloc(sizeof(uint8_t*) * L);
    for (int l = 0; l < L; ++l) {
        kc[l] = calloc(per, es);
        vc[l] = calloc(per, es);
        ex[l] = calloc(T, 1);
    }
    const int P = 5;
    float* x = malloc(sizeof(float) * P * d);
    for (int i = 0; i < P * d; ++i) x[i] = (float)rnd();
    double* h = malloc(sizeof(double) * P * d);
    uint8_t* mask = malloc(Lm > 0 ? Lm : 1);
    float* scores = malloc(sizeof(float) * (Lm > 0 ? Lm : 1));
    float* logits = malloc(sizeof(float) * (Lm > 0 ? Lm : 1));
    double margin, pmargin;
    int32_t n_exec, k_hat;

    /* routed prefill of P tokens, masked and unmasked */
    for (int masked = 0; masked < 2; ++masked) {
        int rc = orc_prefill_seq(&c, layers, &dm, kc, vc, masked ? ex : NULL, P, Lm / 2, NULL,
                                 x, h, mask, scores, &margin);
        EXPECT(rc == 0, "prefill");
    }
    /* decode steps after the prompt: budgets 0..Lm, masked and unmasked,
     * a fixed route, and the budget-free step */
    float* xs = malloc(sizeof(float) * d);
    for (int i = 0; i < d; ++i) xs[i] = (float)h[(size_t)(P - 1) * d + i];
    int pos = P;
    for (int k = 0; k <= Lm && pos < T; ++k, ++pos) {
        int rc = orc_decode_seq_ex(&c, layers, &dm, kc, vc, (k & 1) ? ex : NULL, pos, k, NULL,
                                   xs, h, mask, scores, &margin, &n_exec);
        EXPECT(rc == 0 && n_exec == k + orc_start_layer(&c) + 1, "decode");
        for (int i = 0; i < d; ++i) xs[i] = (float)h[i];
    }
    if (pos < T) {
        for (int i = 0; i < Lm; ++i) mask[i] = (uint8_t)(i & 1);
        int rc = orc_decode_seq(&c, layers, NULL, kc, vc, pos++, 0, mask, xs, h, NULL, NULL,
                                &margin, &n_exec);
        EXPECT(rc == 0, "decode with a fixed route");
    }
    if (pos < T) {
        int rc = orc_decode_seq_auto(&c, layers, &dm, &pred, kc, vc, ex, pos++, xs, h, &k_hat,
                                     logits, &pmargin, mask, scores, &margin, &n_exec);
        EXPECT(rc == 0 && k_hat >= 1 && k_hat <= Lm, "budget-free decode");
    }
    /* the last row of the cache, then arguments the oracle must reject */
    {
        int rc = orc_decode_seq(&c, layers, &dm, kc, vc, T - 1, Lm, NULL, xs, h, mask, scores,
                                &margin, &n_exec);
        EXPECT(rc == 0, "decode at the last cache row");
        rc = orc_decode_seq(&c, layers, &dm, kc, vc, T, 0, NULL, xs, h, mask, scores, &margin,
                            &n_exec);
        EXPECT(rc != 0, "position past the cache rejected");
        rc = orc_decode_seq(&c, layers, &dm, kc, vc, 0, Lm + 1, NULL, xs, h, mask, scores,
                            &margin, &n_exec);
        EXPECT(rc != 0, "budget above L_mid rejected");
    }
    /* top-k edge cases */
    if (Lm > 0) {
        for (int i = 0; i < Lm; ++i) scores[i] = (i % 3 == 0) ? NAN : (float)(i / 2);
        for (int k = 0; k <= Lm; ++k) EXPECT(orc_topk(scores, Lm, k, mask, &margin) == 0, "topk");
        EXPECT(orc_topk(scores, Lm, Lm + 1, mask, &margin) != 0, "topk k > n rejected");
    }

    for (int l = 0; l < L; ++l) {
        free((void*)layers[l].attn_norm); free((void*)layers[l].wqkv); free((void*)layers[l].wo);
        free((void*)layers[l].mlp_norm); free((void*)layers[l].wgate_up);
        free((void*)layers[l].wdown);
        free(kc[l]); free(vc[l]); free(ex[l]);
    }
    free(layers); free(kc); free(vc); free(ex);
    free((void*)dm.w1); free((void*)dm.b1); free((void*)dm.w2); free((void*)dm.b2); free(prior);
    free((void*)pred.w1); free((void*)pred.b1); free((void*)pred.w2); free((void*)pred.b2);
    free(x); free(xs); free(h); free(mask); free(scores); free(logits);
}

int main(void)
{
    for (int dtype = 0; dtype < 2; ++dtype)
        for (int S = 1; S <= 3; ++S)
            for (int ctx = 0; ctx < 4; ++ctx) run_model(dtype, S, ctx, (ctx + S) & 1);

    /* App. B prior normalisation: every kind, with and without winsorising,
     * n = 1 and n with ties */
    const int n = 7;
    double raw[7] = {3.0, -1.0, 0.5, 0.5, 10.0, 0.0, 2.0};
    double* out = malloc(sizeof(double) * n);
    for (int kind = 0; kind < 3; ++kind)
        for (int w = 0; w < 2; ++w) {
            orc_prior_normalize(raw, n, kind, w ? 1.5 : 0.0, out);
            orc_prior_normalize(raw, 1, kind, w ? 1.5 : 0.0, out);
            for (int i = 0; i < n; ++i) EXPECT(isfinite(out[i]) || i >= 1, "prior finite");
        }
    free(out);

    /* batch-level path grouping: random masks with repeats, B = 1 and n = 1 */
    for (int trial = 0; trial < 20; ++trial) {
        const int32_t B = 1 + (int32_t)((rnd() + 1.0) * 40.0), n = trial % 5 == 0 ? 1 : 9;
        uint8_t* m = malloc((size_t)B * n);
        for (int32_t i = 0; i < B * n; ++i) m[i] = rnd() > 0.2 ? 1 : (rnd() > 0.5 ? 0 : 5);
        int32_t* perm = malloc(sizeof(int32_t) * B);
        int32_t* starts = malloc(sizeof(int32_t) * (B + 1));
        const int32_t g = orc_group_by_route(m, B, n, perm, starts);
        EXPECT(g >= 1 && g <= B && starts[g] == B, "path grouping");
        free(m); free(perm); free(starts);
    }
    if (failures) return 1;
    printf("oracle driver ok\n");
    return 0;
}
