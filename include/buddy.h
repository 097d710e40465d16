/*
 * buddy.h -- C ABI of the MI355X (gfx950) budget-routed decode step of
 * BUDDY (Budget-Driven Dynamic depth routing, arXiv 2606.09514).
 *
 * One call of buddy_decode_step advances every sequence of a batch by one
 * token:
 *   1. the first block runs for every sequence and appends its K/V row;
 *   2. the KV-aware planner (Sec. 4.3) averages the first layer's K and V
 *      cache rows 0..pos (the new row included) and joins them with the new
 *      token's hidden state after the first block:
 *          z = [mean K | mean V | h]          (din = 2 n_kv hd + d)
 *   3. the Decision Module (Sec. 4.2.3, App. C.1) scores the L-2 routable
 *      blocks, s = W2 act(W1 z + b1) + b2, and fuses the prior,
 *      s' = s + omega p~ (Eq. 2);
 *   4. a deterministic top-k keeps the k_b best blocks of sequence b
 *      (Eq. 2; ties go to the lower block index, NaN ranks last);
 *   5. each routable block runs only on the sequences that selected it
 *      (grouping by mask, App. C.1); a skipped block leaves h unchanged
 *      (Eq. 1) and gets a zero-filled K/V row at pos (Sec. 6, limitations);
 *   6. the last block runs for every sequence.
 * Start layer (the Decision Module placement ablation of Sec. 4.3):
 * with buddy_config.start_layer = S > 1, step 1 runs blocks 0..S-1, the
 * planner reads block S-1's cache and the hidden state after block S-1, and
 * the routable blocks are S..L-2.  L_mid = L - 1 - S routable blocks (L-2
 * for the default S = 1) size every mask, score and budget below.
 * The decoder block is Llama-style (App. C.2): RMSNorm, Q/K/V projection,
 * rotary embedding (rotate-half pairing, angle pos * theta^(-2i/hd)), grouped
 * query attention over the cache including the new row (App. "Background",
 * KV-cache equation), output projection, residual, RMSNorm, SwiGLU MLP,
 * residual.  Projections are bias-free.
 *
 * Conventions shared by every entry point:
 *   - Memory: every pointer marked "device" is memory the caller allocated on
 *     the current HIP device; the caller owns it and keeps it alive until the
 *     enqueued work has finished.  The library never frees caller memory.
 *     A model handle owns only its workspace.
 *   - Precision: weights and the KV cache are stored in the configured dtype
 *     (fp32 or bf16); hidden states, scores and all accumulation are fp32.
 *     New K/V rows are rounded to the storage dtype (nearest, ties to even).
 *   - Layouts are row-major.  Weight matrices are [out][in]:
 *       wqkv     [(n_heads + 2 n_kv_heads) hd][d]    rows q | k | v
 *       wo       [d][n_heads hd]
 *       wgate_up [2 d_ffn][d]                        rows gate | up
 *       wdown    [d][d_ffn]
 *       attn_norm, mlp_norm [d]
 *       Decision Module: w1 [dm_hidden][din], b1 [dm_hidden],
 *                        w2 [L_mid][dm_hidden], b2 [L_mid]  (storage dtype),
 *                        prior [L_mid] fp32 (already normalised p~) or NULL.
 *     KV cache: K and V each [n_layers][max_batch][n_kv_heads][max_ctx][hd].
 *   - Positions: pos[b] (host array) is the number of cached rows of
 *     sequence b before the step; the step writes row pos[b] of every layer
 *     and attends rows 0..pos[b].  The caller advances pos.
 *   - Streams: `stream` is a hipStream_t (NULL = the null stream).  All work
 *     is enqueued on it; outputs are valid once the stream reaches the
 *     enqueued work.  The only host wait is the optional one of the
 *     host-routed launch policy (buddy_set_launch_policy).
 *   - Errors: arguments are validated on the host before anything is
 *     enqueued; on a validation failure nothing is written and a status is
 *     returned.  BUDDY_EDEVICE reports a HIP launch error; its text is
 *     available from buddy_last_error.  Handles are not thread-safe; calls
 *     on one handle must not overlap (they share its workspace).
 */
#ifndef BUDDY_H
#define BUDDY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BUDDY_OK = 0,
    BUDDY_EINVAL = 1,       /* null pointer, bad enum, k or pos out of range */
    BUDDY_ESHAPE = 2,       /* configuration shape the kernels do not support */
    BUDDY_ECAPACITY = 3,    /* batch above max_batch */
    BUDDY_ENOMEM = 4,       /* workspace allocation failed */
    BUDDY_EDEVICE = 5,      /* HIP error (see buddy_last_error) */
    BUDDY_EUNSUPPORTED = 6  /* valid request the library does not implement  */
} buddy_status;

typedef enum { BUDDY_F32 = 0, BUDDY_BF16 = 1 } buddy_dtype;

/* Decision Module activation: SiLU (App. C.1) or exact GELU (erf form). */
typedef enum { BUDDY_ACT_SILU = 0, BUDDY_ACT_GELU_ERF = 1 } buddy_dm_act;

/* Router context (Sec. 4.3 and the feature ablation of Sec. 5): pooled
 * first-layer cache features followed by the newest token's hidden state
 * after the first block.
 *   BUDDY_CTX_KV:   [mean K | mean V | h]  (2 n_kv hd + d values)
 *   BUDDY_CTX_K:    [mean K | h]           (n_kv hd + d)
 *   BUDDY_CTX_V:    [mean V | h]           (the paper's default feature)
 *   BUDDY_CTX_K_PLUS_V: [mean K + mean V | h]
 * Means run over positions 0..pos (the new row included); the Decision
 * Module's first layer has this many inputs (w1 is [dm_hidden][din]). */
typedef enum { BUDDY_CTX_KV = 0, BUDDY_CTX_K = 1, BUDDY_CTX_V = 2, BUDDY_CTX_K_PLUS_V = 3 } buddy_router_ctx;

/* KV treatment of a skipped block.
 *   BUDDY_SKIP_KV_ZERO: the slot at the step's position is zero-filled and
 *     later steps attend to it as an ordinary entry (logit 0, value 0): the
 *     treatment the paper uses (Conclusion, limitations).
 *   BUDDY_SKIP_KV_MASK: the slot is still zero-filled, and the step also
 *     records which blocks ran in the caller's execution map (buddy_kv.exec);
 *     attention leaves out the positions at which a block did not run (the
 *     masking alternative the paper names as future work). */
typedef enum { BUDDY_SKIP_KV_ZERO = 0, BUDDY_SKIP_KV_MASK = 1 } buddy_skip_kv;

typedef struct {
    int32_t n_layers;     /* L >= 2; blocks 0 and L-1 always run          */
    int32_t d_model;      /* multiple of 8; bf16: at most 8192, a multiple
                             of 512 above 4096; fp32: at most 2048        */
    int32_t n_heads;      /* query heads, multiple of n_kv_heads           */
    int32_t n_kv_heads;   /* n_heads / n_kv_heads <= 8                     */
    int32_t head_dim;     /* 64 or 128                                     */
    int32_t d_ffn;        /* multiple of 8; bf16: at most 32768, a multiple
                             of 512 above 4096; fp32: at most 2048        */
    int32_t dm_hidden;    /* Decision Module hidden width, multiple of 8   */
    int32_t dm_act;       /* buddy_dm_act                                  */
    int32_t dtype;        /* buddy_dtype of weights and KV cache           */
    int32_t max_batch;    /* 1..256: workspace and KV cache batch capacity */
    int32_t max_ctx;      /* rows per sequence in the KV cache             */
    float rms_eps;        /* RMSNorm epsilon                               */
    float rope_theta;     /* rotary base                                   */
    int32_t router_ctx;   /* buddy_router_ctx                              */
    int32_t start_layer;  /* S: blocks 0..S-1 always run, the router reads
                             block S-1; 1 <= S <= n_layers - 1, 0 reads as
                             1 (the paper's default)                       */
} buddy_config;

typedef struct {
    const void *attn_norm, *wqkv, *wo, *mlp_norm, *wgate_up, *wdown; /* device */
} buddy_layer_weights;

typedef struct {
    const void *w1, *b1, *w2, *b2;  /* device, storage dtype              */
    const float* prior;             /* device [L_mid] fp32, or NULL       */
    float omega;                    /* prior weight of Eq. 2 (paper: 0.1) */
} buddy_dm_weights;

typedef struct {
    void* k;        /* device [L][max_batch][n_kv][max_ctx][hd], storage dtype */
    void* v;        /* same layout as k                                         */
    uint8_t* exec;  /* device [L][max_batch][max_ctx] execution map, or NULL:
                       exec[l][b][j] != 0 when block l ran for sequence b's
                       token at position j.  Read and written only with
                       BUDDY_SKIP_KV_MASK (required then); the caller fills
                       the rows of cached positions (e.g. all ones after a
                       dense prefill), each step writes every block's entry
                       at its position.  Blocks 0 and L-1 run for every
                       token, so their maps are all ones.                  */
    /* Running-sum pool (optional; both NULL or both set).  The KV-aware
     * planner's context is the mean of the first block's K and V rows
     * 0..pos (Sec. 4.3).  With these arrays the planner keeps, per sequence
     * and KV head, the fp32 sums of rows 0..pool_rows-1 and adds only the
     * rows it has not seen, instead of summing all pos + 1 rows each call:
     *   pool_sum:  device fp32 [max_batch][n_kv][2][hd], K sums then V sums
     *   pool_rows: device int32 [max_batch][n_kv], rows held in pool_sum
     * A call at position p adds rows pool_rows..p-1 (rows older than the
     * step, which the step does not rewrite) and sets pool_rows = p; row p
     * enters that call's mean without entering the sums, so repeating a step
     * at the same position stays exact.  pool_rows > p starts the sums over;
     * where pool_rows is 0 the contents of pool_sum are not read.
     * The caller zeroes pool_rows before first use and again for a slot
     * whenever it rewrites that slot's cached rows below pool_rows;
     * buddy_prefill does so itself for the slots it fills.  Sums are in a
     * different order than a fresh scan: equal up to fp32 rounding.       */
    float* pool_sum;
    int32_t* pool_rows;
} buddy_kv;

typedef struct buddy_model buddy_model;

/* Creates a model handle on the current HIP device.  `layers` holds
 * n_layers entries; the weight pointers are copied, the weights are not.
 * Allocates the handle's workspace (sized by max_batch and max_ctx).
 * Returns BUDDY_OK and *out, or an error status with *out = NULL:
 * BUDDY_ESHAPE for a shape outside the limits of the fields above (the
 * query width n_heads * head_dim within those of d_ffn, the router input
 * of at most 20480 elements), BUDDY_ECAPACITY for max_batch or max_ctx. */
buddy_status buddy_model_create(const buddy_config* cfg, const buddy_layer_weights* layers,
                                const buddy_dm_weights* dm, buddy_model** out);

/* Waits for the device, then frees the handle's workspace.  NULL is a no-op. */
void buddy_model_destroy(buddy_model* m);

/* KV-aware planner plus Decision Module (Sec. 4.3, Sec. 4.2.3, Eq. 2 fusion)
 * without routing: for b < B, pools the first layer's K/V rows 0..pos[b] of
 * kv (the newest token's row already written) with h_new[b] (device
 * [B][d] fp32) and writes s' to scores_out (device [B][L_mid] fp32).
 * pos: host [B].  B = 0 is a no-op. */
buddy_status buddy_pool_route(buddy_model* m, const buddy_kv* kv, const int32_t* pos,
                              const float* h_new, int32_t B, float* scores_out,
                              void* stream);

/* buddy_pool_route for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same planner and Decision Module scores, bit for bit, with
 * no model handle and no allocation of any kind.  The configuration and the
 * Decision Module weights come as arguments (cfg as for buddy_model_create;
 * cfg->max_batch is the batch capacity of the KV cache layout); kv, pos,
 * h_new, B, scores_out and stream as for buddy_pool_route.  Every buffer
 * the kernels need beyond the inputs and outputs (positions, pool partial
 * sums, the Decision Module's hidden activations, scores) lives in a scratch
 * array of 8 MiB that the library holds once per device for the life of the
 * process; no part of it needs to start at zero.  That limits a call to
 * pieces of 4 B bytes (three of them), 4, 4 B L_mid + 4, 4 B dm_hidden and
 * 8 B n_kv_heads head_dim splits bytes, each rounded up to 256, totalling at
 * most 8 MiB, where splits, the pool's position splits, is 1 with
 * kv->pool_sum and otherwise min(ceil(1024 / (B n_kv_heads)),
 * ceil((max pos + 1) / 64), ceil(max_ctx / 64), 64), at least 1 (e.g. a
 * Llama-3-8B shape fits any batch up to 256; a 40-KV-head, head_dim 128
 * shape fits batches up to about 190).  Beyond it the call returns
 * BUDDY_ECAPACITY and writes nothing.  Calls on one GPU
 * share its array: calls that overlap on a device (other streams or host
 * threads) race and must be ordered by the caller.  Errors as for
 * buddy_model_create and buddy_pool_route; BUDDY_EDEVICE when the scratch
 * address cannot be obtained on the current device. */
buddy_status buddy_pool_route_noalloc(const buddy_config* cfg, const buddy_dm_weights* dm,
                                      const buddy_kv* kv, const int32_t* pos, const float* h_new,
                                      int32_t B, float* scores_out, void* stream);

/* Deterministic per-row top-k (Eq. 2): mask_out[b][i] = 1 iff layer i is
 * among the k[b] largest of scores[b][0..n) under (score desc, index asc,
 * NaN last).  scores: device [B][n] fp32; k: host [B], 0 <= k[b] <= n;
 * mask_out: device [B][n] uint8; 1 <= n <= 255; B <= 65535.  Needs no
 * model handle. */
buddy_status buddy_select_topk(const float* scores, const int32_t* k, int32_t B, int32_t n,
                               uint8_t* mask_out, void* stream);

/* Batch-level path grouping (the Conclusion names grouping requests by
 * their path among its open questions): orders the B sequences of a batch
 * by route and marks the groups of identical routes, e.g. to serve each
 * group as one sub-batch with route_override.  mask: device [B][n] uint8,
 * nonzero = the block runs (as buddy_decode_step's mask_out); routes
 * compare lexicographically in block order with a skipped block before a
 * run one, and equal routes keep their batch order, so the result is
 * unique.  perm_out: device int32 [B], the sequence at each position;
 * starts_out: device int32 [B + 1], the first position of group g at
 * [g] and B after the last group; n_groups_out: device int32 [1].
 * 1 <= n <= 255, B <= 1024; B = 0 is a no-op.  Needs no model handle. */
buddy_status buddy_group_by_route(const uint8_t* mask, int32_t B, int32_t n, int32_t* perm_out,
                                  int32_t* starts_out, int32_t* n_groups_out, void* stream);

/* One budget-routed decode step for B sequences (steps 1-6 above).
 *   hidden: device [B][d] fp32; input H_0 of the new token, overwritten
 *           with the last block's output H_L (no final norm).
 *   pos:    host [B]; 0 <= pos[b] < max_ctx.
 *   k:      host [B]; 0 <= k[b] <= L_mid routable blocks to run.
 *   skip_kv: buddy_skip_kv; BUDDY_SKIP_KV_MASK needs kv->exec
 *           (BUDDY_EINVAL otherwise).
 *   route_override: device [B][L_mid] uint8 (nonzero = run) or NULL; when
 *           given, the planner and Decision Module are not run, k is
 *           ignored and scores_out is left untouched.
 *   mask_out: device [B][L_mid] uint8 or NULL: the mask that was executed.
 *   scores_out: device [B][L_mid] fp32 or NULL: s' of step 3.
 * B = 0 is a no-op; B > max_batch gives BUDDY_ECAPACITY. */
buddy_status buddy_decode_step(buddy_model* m, const buddy_kv* kv, float* hidden,
                               const int32_t* pos, const int32_t* k, int32_t B,
                               int32_t skip_kv, const uint8_t* route_override,
                               uint8_t* mask_out, float* scores_out, void* stream);

/* Budget Predictor head (Sec. 4.4): a categorical policy over k = 1..L_mid
 * from the same router context as the Decision Module, read as the Decision
 * Module's form (the paper does not give its layers): logits = w2 act(w1 z
 * + b1) + b2 with the Decision Module's activation. */
typedef struct {
    const void *w1, *b1, *w2, *b2;  /* device, storage dtype: w1 [hidden][din],
                                       b1 [hidden], w2 [L_mid][hidden], b2 [L_mid] */
    int32_t hidden;                 /* multiple of 8                          */
} buddy_predictor_weights;

/* Attaches a Budget Predictor head to the handle (the pointers are copied,
 * the weights are not; they must outlive the handle), or detaches it with
 * p == NULL.  Waits for the device, then allocates the head's workspace.
 * Errors: BUDDY_EINVAL (null pointers, hidden not a positive multiple of 8,
 * no routable block), BUDDY_ESHAPE (hidden too wide), BUDDY_ENOMEM. */
buddy_status buddy_set_budget_predictor(buddy_model* m, const buddy_predictor_weights* p);

/* Planner and Budget Predictor only (steps 3 and 4 with the predictor's
 * output layer): k_out device [B] int32 receives k_hat = 1 + argmax of the
 * logits (fp32; the smaller k on equal logits; the budget is b_hat =
 * (k_hat + 2) / L); logits_out device [B][L_mid] fp32 or NULL.  pos and h_new
 * as for buddy_pool_route.  BUDDY_EINVAL without an attached predictor. */
buddy_status buddy_predict_budget(buddy_model* m, const buddy_kv* kv, const int32_t* pos,
                                  const float* h_new, int32_t B, int32_t* k_out,
                                  float* logits_out, void* stream);

/* buddy_decode_step without budgets: each sequence's k is the Budget
 * Predictor's k_hat from the step's own router context, then the step runs
 * as buddy_decode_step with that k.  k_out: device [B] int32 or NULL.
 * BUDDY_EINVAL without an attached predictor. */
buddy_status buddy_decode_step_auto(buddy_model* m, const buddy_kv* kv, float* hidden,
                                    const int32_t* pos, int32_t B, int32_t skip_kv,
                                    int32_t* k_out, uint8_t* mask_out, float* scores_out,
                                    void* stream);

/* Routed prefill of B prompts into cache rows 0..len[b]-1 (one route per
 * prompt; the Reuse setting of Sec. 5 keeps decoding on the prefill's
 * decision, so the prefill itself is routed).  The first block (blocks
 * 0..S-1 with a start layer S) runs over
 * every prompt token; the planner and Decision Module decide the route once
 * per prompt at its last token (as a decode step at position len[b]-1
 * would), unless route_override gives it; each selected block then runs
 * causally over the prompt, and every skipped block's K/V rows 0..len[b]-1
 * are zero-filled (with BUDDY_SKIP_KV_MASK also marked in kv->exec).
 *   hidden: device [B][t_stride][d] fp32, the prompt tokens' inputs,
 *           overwritten with their last-block outputs (rows t >= len[b]
 *           untouched).
 *   len:    host [B], 1 <= len[b] <= min(t_stride, max_ctx).
 *   k:      host [B] budgets 0..L_mid (ignored with route_override).
 *   route_override, mask_out, scores_out: as buddy_decode_step.
 * Rows of all prompts together: B * t_stride <= 65535.  Grows the handle's
 * prefill workspace when needed and returns after the device has finished
 * (the host waits for the route to build the per-block token lists). */
buddy_status buddy_prefill(buddy_model* m, const buddy_kv* kv, float* hidden, int32_t t_stride,
                           const int32_t* len, const int32_t* k, int32_t B, int32_t skip_kv,
                           const uint8_t* route_override, uint8_t* mask_out, float* scores_out,
                           void* stream);

/* How buddy_decode_step launches the routable blocks.
 *   BUDDY_LAUNCH_DEVICE_ROUTED: everything is enqueued without waiting; every
 *     routable block is launched and its kernels read the routed row count
 *     on the device, so a block nobody selected costs only empty launches.
 *     The call never blocks the host (suitable for stream capture).
 *   BUDDY_LAUNCH_HOST_ROUTED: after the router, the call waits for the
 *     per-block routed counts (written by the device to mapped pinned host
 *     memory owned by the handle) and launches only the blocks some sequence
 *     runs, with grids sized to the routed rows.  The host blocks until the
 *     first block and the router have run; a device error during that wait
 *     is reported (BUDDY_EDEVICE) within about 0.1 s, and no answer within a
 *     minute also ends it with BUDDY_EDEVICE.
 *   BUDDY_LAUNCH_AUTO (default): host-routed when B <= 16 and not every
 *     sequence runs every block, device-routed otherwise, and always
 *     device-routed while the stream is being captured into a graph.
 * Under stream capture (hipStreamBeginCapture) an explicit host-routed
 * policy makes buddy_decode_step and buddy_decode_step_auto return
 * BUDDY_EINVAL with nothing enqueued, and buddy_prefill, which waits for its
 * route on the host, always returns BUDDY_EINVAL.  A captured step replays
 * with the positions and budgets it was captured with (they are kernel
 * arguments). */
typedef enum {
    BUDDY_LAUNCH_AUTO = 0,
    BUDDY_LAUNCH_DEVICE_ROUTED = 1,
    BUDDY_LAUNCH_HOST_ROUTED = 2
} buddy_launch_policy;

/* Sets the launch policy of a handle; BUDDY_EINVAL for an unknown policy. */
buddy_status buddy_set_launch_policy(buddy_model* m, int32_t policy);

/* Output tile of the prefill's tiled projections (bf16 weights, many prompt
 * tokens).
 *   BUDDY_GEMM_TILE_AUTO (default): 256 x 256 where that still gives every
 *     CU two workgroups (when the last round of such a grid would leave CUs
 *     idle, its weight rows go to a second launch of 128 x 128 tiles that
 *     fits one round); for the residual-add projections (O, down) whose
 *     256 x 256 grid is smaller, 256 x 256 with K split in two halves whose
 *     sums are added to the residual in a fixed order; else 128 x 128;
 *   BUDDY_GEMM_TILE_128, BUDDY_GEMM_TILE_256: always that tile (weight
 *     rows x token rows), K never split;
 *   BUDDY_GEMM_TILE_256_SPLIT: 256 x 256, K split for the residual-add
 *     projections.
 * The tiles without a split give the same results bit for bit; a split
 * adds the two half sums, a different rounding order. */
typedef enum {
    BUDDY_GEMM_TILE_AUTO = 0,
    BUDDY_GEMM_TILE_128 = 1,
    BUDDY_GEMM_TILE_256 = 2,
    BUDDY_GEMM_TILE_256_SPLIT = 3
} buddy_gemm_tile;

/* Sets the tile choice of a handle; BUDDY_EINVAL for an unknown value. */
buddy_status buddy_set_gemm_tile(buddy_model* m, int32_t tile);

/* Kernels of a decoder block, for buddy_set_timing_events. */
typedef enum {
    BUDDY_KERNEL_QKV = 0,        /* RMSNorm + QKV projection + rotary + KV append */
    BUDDY_KERNEL_ATTENTION = 1,  /* split-K decode attention                      */
    BUDDY_KERNEL_O_PROJ = 2,     /* output projection + residual                  */
    BUDDY_KERNEL_GATE_UP = 3,    /* RMSNorm + gate/up projection + SwiGLU         */
    BUDDY_KERNEL_DOWN = 4,       /* down projection + residual                    */
    BUDDY_KERNEL_ATTN_MERGE = 5  /* merge of the attention's position-chunk partials
                                    (no launch when one chunk covers every row:
                                    the events then mark an empty interval)      */
} buddy_kernel;

/* Measurement hook.  For the next n calls of buddy_decode_step on this
 * handle, call i times `kernel` in block `layer`: start[i] and stop[i] are
 * recorded at the dispatch begin and end of that kernel's main launch (the
 * projection itself, not the activation staging of the batched path; the
 * attention score kernel, not the chunk merge), the interval a kernel trace
 * reports.  If the block does not run, both are recorded back to back on the
 * stream at that point of the step.  start and stop are
 * arrays of n hipEvent_t handles that the caller created and keeps alive
 * until the calls have run; the handle copies the arrays.  n = 0 turns the
 * hook off.  Errors: BUDDY_EINVAL for a bad kernel, layer or n < 0, or null
 * arrays with n > 0. */
buddy_status buddy_set_timing_events(buddy_model* m, int32_t kernel, int32_t layer,
                                     void* const* start, void* const* stop, int32_t n);

/* Kinds of raw per-layer importance indicator (App. B, direction
 * unification): the skip-induced perplexity increase PPL_skip - PPL_full,
 * a Taylor / Fisher / gradient-norm score, or the cosine similarity of a
 * block's input and output. */
typedef enum {
    BUDDY_PRIOR_DELTA_PPL = 0,
    BUDDY_PRIOR_TAYLOR = 1,
    BUDDY_PRIOR_COSINE = 2
} buddy_prior_kind;

/* Offline prior normalisation (App. B, then Eq. 2), host code.  raw: host
 * [n] indicator values of the n routable layers (finite); prior_out: host
 * [n] fp32, the prior p~ for buddy_dm_weights.prior (copy it to the device).
 * Steps over the n layers: larger-is-more-important (max(0, x) for the
 * perplexity and Taylor kinds, 1 - x for cosine), log(1 + x) for the
 * perplexity and Taylor kinds, robust z = (x - median) / (IQR + 1e-6) with
 * linearly interpolated quartiles, clipped to [-winsor, winsor] when winsor
 * > 0, rank normalisation u = (1 + rank) / (n + 1) with 0-based ranks and
 * ties at their mean rank, and p~ = (u - mean u) / (population std + 1e-6).
 * Errors: BUDDY_EINVAL for null pointers, n < 1, an unknown kind, a negative
 * or non-finite winsor, or a non-finite raw value (nothing written). */
buddy_status buddy_prior_normalize(const float* raw, int32_t n, int32_t kind, float winsor,
                                   float* prior_out);

/* Budget to routable-block count, k = round(b L) - 2 (Eq. 2), halves away
 * from zero, limited to [0, L-2]; -1 when b is outside (0, 1].  This is the
 * default start layer's count; with start layer S the blocks 0..S-1 and
 * L-1 always run and k = round(b L) - (S + 1), which callers compute. */
int32_t buddy_budget_to_k(float b, int32_t n_layers);

const char* buddy_status_string(buddy_status s);

/* Text of the last HIP error seen by this handle ("" if none). */
const char* buddy_last_error(const buddy_model* m);

#ifdef __cplusplus
}
#endif
#endif
