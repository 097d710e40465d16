/*
 * buddy_oracle.h -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow CPU reference ("oracle") of one budget-routed decode step of
 * BUDDY (Budget-Driven Dynamic depth routing, arXiv 2606.09514).  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load
 * this library.  The GPU library never links, includes or calls it, and it
 * shares no code with the GPU library.
 *
 * Arithmetic is IEEE double throughout.  Values held in storage precision
 * (weights, the KV cache) are read by exact up-conversion; newly produced K/V
 * rows are rounded to the storage precision when stored, because the model
 * keeps its cache in that precision and later steps read the rounded values.
 * Layer scores are rounded to fp32 before the top-k decision, so both sides
 * take that integer decision on fp32 values.
 *
 * Layouts (all row-major):
 *   wqkv     [(n_heads + 2 n_kv_heads) * head_dim][d_model]  rows: q | k | v
 *   wo       [d_model][n_heads * head_dim]
 *   wgate_up [2 d_ffn][d_model]                                rows: gate | up
 *   wdown    [d_model][d_ffn]
 *   attn_norm, mlp_norm [d_model]
 *   dm w1 [dm_hidden][din], b1 [dm_hidden], w2 [L_mid][dm_hidden], b2 [L_mid]
 *      din = 2 * n_kv_heads * head_dim + d_model
 *   one sequence's cache for one layer: [n_kv_heads][max_ctx][head_dim]
 * Every weight array and the cache are in the storage dtype (fp32 or bf16).
 */
#ifndef BUDDY_ORACLE_H
#define BUDDY_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_ACT_SILU = 0, ORC_ACT_GELU_ERF = 1 };

/* Router context variants (Sec. 4.3: the features G_t in {K, V, K + V}
 * pooled from the first layer's cache, then the newest hidden state). */
enum { ORC_CTX_KV = 0, ORC_CTX_K = 1, ORC_CTX_V = 2, ORC_CTX_K_PLUS_V = 3 };

typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn;
    int32_t dm_hidden, dm_act, dtype, max_ctx;
    double rms_eps, rope_theta;
    int32_t router_ctx;   /* ORC_CTX_* */
    /* Start layer of the Decision Module (Sec. 4.3 ablation): blocks
     * 0..S-1 always run and block S-1's cache is the router context; the
     * routable blocks are S..L-2.  0 reads as 1, the paper's default. */
    int32_t start_layer;
} orc_config;

/* First routable block S and the number of routable blocks L - 1 - S. */
int orc_start_layer(const orc_config* c);
int orc_n_mid(const orc_config* c);

typedef struct {
    const void *attn_norm, *wqkv, *wo, *mlp_norm, *wgate_up, *wdown;
} orc_layer;

typedef struct {
    const void *w1, *b1, *w2, *b2;
    const float *prior;   /* normalized prior p~ [L_mid], or NULL */
    double omega;         /* prior weight; 0 disables the fusion */
} orc_dm;

/* Budget Predictor head (Sec. 4.4): a categorical policy over the actions
 * k = 1..L_mid from the router context (L_mid = orc_n_mid, L-2 by default).  The paper does not give its layers;
 * read here as the Decision Module's form, two linear layers with the
 * Decision Module's activation in between. */
typedef struct {
    const void *w1, *b1, *w2, *b2;   /* [hidden][din], [hidden], [L_mid][hidden], [L_mid] */
    int32_t hidden;
} orc_predictor;

/* bf16 bits nearest to x (round to nearest, ties to even; NaN -> quiet NaN). */
uint16_t orc_bf16_from_double(double x);

/* RMSNorm: out = h / sqrt(mean(h^2) + eps) * g (g in storage dtype). */
void orc_rmsnorm(const orc_config* c, const double* h, const void* g, double* out);

/* Rotary embedding (rotate-half pairing) of one head vector x[head_dim] at pos. */
void orc_rope(const orc_config* c, double* x, int32_t pos);

/* One decoder block (Eq. 1 with M=1) for one sequence at position pos:
 * appends K/V (rounded to storage) at pos of this layer's cache and updates h. */
void orc_block(const orc_config* c, const orc_layer* w, void* kc, void* vc,
               int32_t pos, double* h);

/* orc_block with an execution map exec[max_ctx] of this layer's cache:
 * positions j with exec[j] == 0 (the block did not run for that token) are
 * left out of the attention softmax.  exec == NULL: every position counts
 * (zero-filled slots of skipped steps are attended as ordinary entries). */
void orc_block_ex(const orc_config* c, const orc_layer* w, void* kc, void* vc,
                  int32_t pos, double* h, const uint8_t* exec);

/* Mean of the cached K and V rows at positions 0..pos (inclusive), each
 * flattened head-major to n_kv_heads*head_dim: z = [mean K | mean V]. */
void orc_pool(const orc_config* c, const void* kc, const void* vc, int32_t pos,
              double* z);

/* Length of the router context z for the configured variant. */
int orc_context_dim(const orc_config* c);

/* Router context z of one sequence: the pooled first-layer features of the
 * variant (ORC_CTX_KV: [mean K | mean V]; ORC_CTX_K: mean K; ORC_CTX_V:
 * mean V; ORC_CTX_K_PLUS_V: mean K + mean V; means over 0..pos as in
 * orc_pool), followed by the newest hidden state h[d_model]. */
void orc_router_context(const orc_config* c, const void* kc, const void* vc, int32_t pos,
                        const double* h, double* z);

/* Decision Module: s' = W2 act(W1 z + b1) + b2 + omega * prior, rounded to fp32;
 * z has orc_context_dim(c) values. */
void orc_dm_scores(const orc_config* c, const orc_dm* dm, const double* z,
                   float* scores);

/* Budget Predictor: logits = W2 act(W1 z + b1) + b2 over k = 1..L_mid, rounded
 * to fp32 (the precision the argmax is taken in); returns k_hat = 1 + argmax
 * (equal logits: the smaller k; NaN never wins).  logits[L_mid] optional;
 * *margin = best - second best logit (+inf with a single action). */
int32_t orc_predict_budget(const orc_config* c, const orc_predictor* p, const double* z,
                           float* logits, double* margin);

/* Deterministic top-k over n scores: order by (score desc, index asc, NaN last).
 * mask[i] = 1 for the first k.  *margin = s(k-th) - s(k+1-th) in that order,
 * +inf when k == 0 or k == n.  Returns 0, or -1 for k outside [0, n]. */
int orc_topk(const float* scores, int32_t n, int32_t k, uint8_t* mask,
             double* margin);

/* One full decode step for one sequence.
 *   kc[l], vc[l]: this sequence's cache of layer l ([n_kv][max_ctx][hd]).
 *   pos: cached positions before the step (the new token is written at pos).
 *   k_budget: number of routable layers to run (0..L_mid; L_mid = L-2
 *          by default, L-1-S with start layer S: blocks S..L-2).
 *   route: optional fixed mask over the L_mid routable layers (skips the
 *          Decision Module); NULL routes with the Decision Module.
 *   x: input hidden [d]; h_out: output hidden [d].
 *   mask_out[L_mid], scores_out[L_mid] (left untouched when route != NULL),
 *   margin_out, n_exec_out (blocks executed, including the S leading ones
 *   and the last):
 *   all optional.
 * Returns 0, or -1 on invalid arguments (nothing written). */
int orc_decode_seq(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                   void* const* kc, void* const* vc, int32_t pos, int32_t k_budget,
                   const uint8_t* route, const float* x, double* h_out,
                   uint8_t* mask_out, float* scores_out, double* margin_out,
                   int32_t* n_exec_out);

/* orc_decode_seq with skipped-KV masking: exec[l] is layer l's execution
 * map of this sequence ([max_ctx] bytes).  The step writes exec[l][pos] (1
 * for every block it runs, 0 for every block it skips; skipped slots are
 * still zero-filled) and each block's attention leaves out the positions at
 * which that block did not run.  exec == NULL is orc_decode_seq. */
int orc_decode_seq_ex(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                      void* const* kc, void* const* vc, uint8_t* const* exec, int32_t pos,
                      int32_t k_budget, const uint8_t* route, const float* x, double* h_out,
                      uint8_t* mask_out, float* scores_out, double* margin_out,
                      int32_t* n_exec_out);

/* orc_decode_seq_ex without a budget: the Budget Predictor picks k from the
 * same router context as the Decision Module (Sec. 4.4, b = (k + 2) / L),
 * then the step routes with it.  k_out, logits_out[L-2] and pmargin_out
 * (the predictor's best - second best logit) are optional. */
int orc_decode_seq_auto(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                        const orc_predictor* pred, void* const* kc, void* const* vc,
                        uint8_t* const* exec, int32_t pos, const float* x, double* h_out,
                        int32_t* k_out, float* logits_out, double* pmargin_out,
                        uint8_t* mask_out, float* scores_out, double* margin_out,
                        int32_t* n_exec_out);

/* Routed prefill of one sequence's prompt x[len][d] (rows 0..len-1 of the
 * cache; len <= max_ctx).  The first block runs over every token; the route
 * is decided once, from the pooled first-layer cache of the prompt and the
 * last token's hidden state after the first block (the planner at position
 * len - 1), unless `route` fixes it; then each selected block runs causally
 * over all prompt tokens and every skipped block's K/V rows 0..len-1 are
 * zero-filled (with exec maps: marked 0, selected and always-run blocks 1).
 * h_out[len][d]: every token's output of the last block.  mask_out,
 * scores_out, margin_out: as orc_decode_seq (optional).  Returns 0 or -1. */
int orc_prefill_seq(const orc_config* c, const orc_layer* layers, const orc_dm* dm,
                    void* const* kc, void* const* vc, uint8_t* const* exec, int32_t len,
                    int32_t k_budget, const uint8_t* route, const float* x, double* h_out,
                    uint8_t* mask_out, float* scores_out, double* margin_out);

/* Offline prior normalisation, App. B steps (i)-(iv) over the n routable
 * layers, then the standardisation of Eq. 2.  kind: 0 = perplexity increase
 * (PPL_skip - PPL_full), 1 = Taylor/Fisher/gradient norm, 2 = cosine
 * similarity.  winsor > 0 clips the robust z-scores to [-winsor, winsor].
 * Readings (the paper leaves them open): quartiles interpolate linearly
 * between order statistics, ranks are 0-based with tied values at their
 * mean rank, the epsilons are 1e-6 and the standard deviation is the
 * population one. */
void orc_prior_normalize(const double* raw, int32_t n, int32_t kind, double winsor,
                         double* out);

/* Number of OpenMP threads the oracle uses. */
/* Batch-level path grouping: perm [B] receives the sequences ordered by
 * route (mask [B][n], nonzero = run; lexicographic over blocks, skip before
 * run, ties in batch order); starts [B + 1] the first position of each group
 * of identical routes, then B.  Returns the number of groups (-1 on bad
 * arguments). */
int32_t orc_group_by_route(const uint8_t* mask, int32_t B, int32_t n, int32_t* perm,
                           int32_t* starts);

int orc_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
