// Host side of the C ABI declared in include/buddy.h: argument validation,
// the model handle and its workspace, and the order of kernel launches of
// one budget-routed decode step.  Every launch goes to the caller's stream;
// nothing here synchronises with the device except buddy_model_destroy.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <mutex>
#include <new>
#include <thread>

#include <vector>

#include "buddy_internal.h"

using namespace buddy;

thread_local LaunchEvents buddy::tl_launch_events = {nullptr, nullptr};
thread_local LaunchEvents buddy::tl_merge_events = {nullptr, nullptr};

struct buddy_model {
    Model M;
};

namespace {

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

buddy_status fail_device(Model& M, hipError_t e, const char* where) {
    snprintf(M.last_error, sizeof(M.last_error), "%s: %s", where, hipGetErrorString(e));
    return BUDDY_EDEVICE;
}

// Caches present; the running-sum pool arrays both given or both absent.
bool kv_ok(const buddy_kv* kv) {
    return kv && kv->k && kv->v && (kv->pool_sum == nullptr) == (kv->pool_rows == nullptr);
}

buddy_status check_config(const buddy_config* c) {
    if (!c) return BUDDY_EINVAL;
    if (c->n_layers < 2 || c->n_layers > 1024) return BUDDY_ESHAPE;
    if (c->start_layer < 0 || c->start_layer > c->n_layers - 1) return BUDDY_EINVAL;
    if (n_mid(*c) > 255) return BUDDY_ESHAPE;
    if (c->d_model <= 0 || c->d_model % 8) return BUDDY_ESHAPE;
    if (c->n_kv_heads <= 0 || c->n_heads <= 0 || c->n_heads % c->n_kv_heads) return BUDDY_ESHAPE;
    if (c->n_heads / c->n_kv_heads > kMaxGroup) return BUDDY_ESHAPE;
    if (c->head_dim != 64 && c->head_dim != 128) return BUDDY_ESHAPE;
    if (c->d_ffn <= 0 || c->d_ffn % 8) return BUDDY_ESHAPE;
    if (c->dm_hidden <= 0 || c->dm_hidden % 8) return BUDDY_ESHAPE;
    if (c->dm_act != BUDDY_ACT_SILU && c->dm_act != BUDDY_ACT_GELU_ERF) return BUDDY_EINVAL;
    if (c->dtype != BUDDY_F32 && c->dtype != BUDDY_BF16) return BUDDY_EINVAL;
    if (c->max_batch < 1 || c->max_batch > kMaxBatch) return BUDDY_ECAPACITY;
    if (c->max_ctx < 1) return BUDDY_EINVAL;
    if (c->max_ctx > (1 << 20)) return BUDDY_ECAPACITY;  // keeps attention chunks <= 256
    if (!(c->rope_theta > 0.f) || !(c->rms_eps >= 0.f)) return BUDDY_EINVAL;
    if (c->router_ctx < BUDDY_CTX_KV || c->router_ctx > BUDDY_CTX_K_PLUS_V) return BUDDY_EINVAL;
    // a GEMV wavefront holds at most 16 k-steps of a two-row unit (K = d_model)
    // and a quarter of 64 k-steps of a single row
    const int ks = 64 * (c->dtype == BUDDY_BF16 ? 8 : 4);
    if (c->d_model > 16 * ks || c->d_ffn > 64 * ks) return BUDDY_ESHAPE;
    if (c->n_heads * c->head_dim > 64 * ks) return BUDDY_ESHAPE;
    // every K the GEMVs see (d_model, d_ffn, n_heads * head_dim and the
    // router input) is a whole number of k-steps of 64 lanes x 16 bytes or at
    // most 8 k-steps; fp32 weights (small models) have rows of at most 8
    // k-steps
    const int din = pooled_dim(c->router_ctx, c->n_kv_heads, c->head_dim) + c->d_model;
    const int qdim = c->n_heads * c->head_dim;
    auto rows_ok = [ks](int K) { return K % ks == 0 || K <= 8 * ks; };
    if (c->dtype == BUDDY_BF16 &&
        !(rows_ok(c->d_model) && rows_ok(c->d_ffn) && rows_ok(qdim) && rows_ok(din)))
        return BUDDY_ESHAPE;
    if (c->dtype == BUDDY_F32 &&
        (c->d_model > 8 * ks || c->d_ffn > 8 * ks || qdim > 8 * ks || din > 8 * ks))
        return BUDDY_ESHAPE;
    // a GEMV stages an fp32 activation row in at most 80 KB of LDS, or a
    // K-sliced row of whole k-steps in two halves of at most 64 KB; the
    // router input is staged in one piece
    auto staged_ok = [ks](int K) {
        return (size_t)K * sizeof(float) <= 80 * 1024 || (K % ks == 0 && K <= 64 * ks);
    };
    if (!staged_ok(c->d_ffn) || !staged_ok(c->d_model) || !staged_ok(qdim)) return BUDDY_ESHAPE;
    if ((size_t)din * sizeof(float) > 80 * 1024) return BUDDY_ESHAPE;
    return BUDDY_OK;
}

size_t elem_size(const buddy_config& c) { return c.dtype == BUDDY_BF16 ? 2 : 4; }

// Cache base of block l (elements of the storage dtype, as bytes).
const char* layer_base(const Model& M, const void* kv, int l) {
    const buddy_config& c = M.cfg;
    const size_t per_layer = (size_t)c.max_batch * c.n_kv_heads * c.max_ctx * c.head_dim;
    return (const char*)kv + (size_t)l * per_layer * elem_size(c);
}

// Position chunks per (sequence, KV head): enough workgroups to cover the
// chip (about 2048 over the launch), chunk lengths a multiple (at least two)
// of the rows one workgroup block reads, at most kAttnMaxChunks chunks, or
// `cap` (at least 1) when that is smaller.
constexpr int kAttnMinBlocks = 2;   // workgroup blocks per chunk, at least

void attn_chunks(const Model& M, int n_rows, int max_pos, int* chunks, int* chunk_len,
                 int cap = kAttnMaxChunks) {
    const buddy_config& c = M.cfg;
    const int rows = attention_rows_per_wg(c.dtype, c.head_dim, c.n_heads / c.n_kv_heads);
    const int blocks = (max_pos + 1 + rows - 1) / rows;
    const int pairs = n_rows * c.n_kv_heads;
    // one chunk per (sequence, KV head) once that alone gives every CU a
    // workgroup: the score kernel then writes o and no merge kernel runs
    // (Llama-8B shape, B = 32: 65.5 us score + 4.8 us merge against 64.5 us)
    if (pairs >= 256) {
        *chunk_len = blocks * rows;
        *chunks = 1;
        return;
    }
    int want = (2048 + pairs - 1) / pairs;
    if (want > blocks) want = blocks;
    if (want > kAttnMaxChunks) want = kAttnMaxChunks;
    if (want > cap) want = cap;
    if (want < 1) want = 1;
    // at most kAttnMaxChunks chunks (max_ctx is bounded at create so that
    // min_chunks itself stays within it)
    const int min_chunks = (blocks + kAttnMaxChunks - 1) / kAttnMaxChunks;
    int per = (blocks + (want > min_chunks ? want : min_chunks) - 1) /
              (want > min_chunks ? want : min_chunks);
    // at least two blocks per chunk: at B = 1 (2049 rows, Llama-8B shape) 17
    // chunks instead of 33 keep the score kernel at its time (a launch of 136
    // workgroups is no slower than one of 264) and halve the merge's partials
    if (per < kAttnMinBlocks) per = kAttnMinBlocks;
    *chunk_len = per * rows;
    *chunks = (max_pos + 1 + *chunk_len - 1) / *chunk_len;
}

// Whether a projection of K inputs over `batch` rows takes the tiled GEMM.
bool uses_gemm(const Model& M, const Rows& rows, int batch, int K, int tok_T) {
    return M.cfg.dtype == BUDDY_BF16 && tok_T > 0 && rows.exact && batch >= kGemmMinRows &&
           K % 64 == 0;
}

// Whether a projection of K inputs over `batch` rows takes the MFMA path.
bool uses_mfma(const Model& M, const Rows& rows, int batch, int K, int tok_T) {
    return M.cfg.dtype == BUDDY_BF16 && batch > kGemvMaxRows && K % 128 == 0 &&
           !uses_gemm(M, rows, batch, K, tok_T);
}

// A routed projection: the GEMV for batches of up to kGemvMaxRows sequences
// (or fp32 weights), the MFMA path beyond.  The choice depends on the batch,
// not on how many sequences a block routes, so a sequence's arithmetic does
// not depend on the routes of the others or on the launch policy.
// fold: the MFMA path's residual add goes to the partial buffer for the next
// staging to add (the caller has checked that the buffer holds the rows):
// fold_part, or the handle's K-split buffer.
hipError_t launch_proj(const Model& M, int batch, int pro, int epi, GemvArgs g, hipStream_t s,
                       bool fold = false, float* fold_part = nullptr) {
    // prompt tokens of a prefill: the tiled GEMM
    if (uses_gemm(M, g.rows, batch, g.K, g.tok_T))
        return launch_gemm(pro, epi, g, M.gemm_tile, M.pf_split, s);
    if (uses_mfma(M, g.rows, batch, g.K, g.tok_T))
        return launch_mfma(pro, epi, g,
                           fold_part ? fold_part
                                     : g.rows.n_max <= M.ws.mfma_part_rows ? M.ws.mfma_part : nullptr,
                           s, fold);
    if (pro == PRO_STAGED) return hipErrorInvalidValue;   // staged inputs feed the MFMA paths only
    return launch_gemv(M.cfg.dtype, pro, epi, g, s);
}

// Activation buffers of a block's launches and the meaning of a row id: a
// sequence (decode, tok_T = 0) or a flattened prompt token (prefill).
struct BlockBufs {
    float* q; float* o; float* m;
    bf16_t* xb; int xb_ld;
    int tok_T;
    bf16_t* xb2;          // second staging buffer: the down projection's input
};

BlockBufs decode_bufs(const Model& M) {
    return BlockBufs{M.ws.q, M.ws.o, M.ws.m, M.ws.xb, M.ws.xb_ld, 0, M.ws.xb2};
}


// Timing hook: event around kernel `kind` of block l, if asked for.
bool timed(const Model& M, int kind, int l) {
    const TimingHook& t = M.timing;
    return t.n > 0 && t.next < t.n && t.kernel == kind && t.layer == l;
}

// Arms the events of the timed kernel for its main launch; at the stop mark,
// events that no launch took (no kernel of that kind ran) are recorded here.
hipError_t mark(const Model& M, int kind, int l, bool stop, hipStream_t s) {
    if (!timed(M, kind, l)) return hipSuccess;
    const TimingHook& t = M.timing;
    LaunchEvents& ev = kind == BUDDY_KERNEL_ATTN_MERGE ? tl_merge_events : tl_launch_events;
    if (!stop) {
        ev = {t.start[t.next], t.stop[t.next]};
        return hipSuccess;
    }
    if (!ev.start) return hipSuccess;
    ev = {nullptr, nullptr};
    hipError_t e = hipEventRecord(t.start[t.next], s);
    return e != hipSuccess ? e : hipEventRecord(t.stop[t.next], s);
}

// d_upto > 0: the QKV staging first adds each sequence's deferred down sums
// from the routable blocks before list index d_upto; d_out >= 0: this
// block's down projection leaves its split sums deferred, as routable block
// d_out (decode rows on the MFMA path, M.ws.down_part).  pooled: for the
// router's block, decode rows without an execution map, the attention also
// writes the planner's pool sums (its chunks as the splits) when the chunks
// fit the pool's split capacity; *pooled receives that split count, 0 if
// it did not.
buddy_status run_block(Model& M, const buddy_kv* kv, const uint8_t* exec, float* hidden, int l,
                       Rows rows, int batch, int max_pos, int pos_u, const BlockBufs& bf,
                       hipStream_t s, const int32_t* groups = nullptr, int n_groups = 0,
                       int d_upto = -1, int d_out = -1, int* pooled = nullptr) {
    const buddy_config& c = M.cfg;
    const buddy_layer_weights& w = M.layers[l];
    const int qdim = c.n_heads * c.head_dim;
    hipError_t e;

    GemvArgs g;
    memset(&g, 0, sizeof(g));
    g.rows = rows;
    g.eps = c.rms_eps;
    g.T = c.max_ctx; g.hd = c.head_dim; g.nq = c.n_heads; g.nkv = c.n_kv_heads;
    g.bcap = c.max_batch; g.pos = M.ws.pos; g.pos_u = pos_u; g.rope = M.ws.rope;
    g.kc = (void*)layer_base(M, kv->k, l);
    g.vc = (void*)layer_base(M, kv->v, l);
    g.tok_T = bf.tok_T;
    g.XB = bf.xb; g.ldxb = bf.xb_ld;

    // RMSNorm + QKV projection + rotary + KV append
    g.W = w.wqkv; g.N = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim; g.K = c.d_model;
    g.X = hidden; g.ldx = c.d_model; g.gain = w.attn_norm;
    g.Y = bf.q; g.ldy = qdim;
    const size_t down_block = (size_t)M.ws.down_splits * c.max_batch * c.d_model;
    if (d_upto > 0 && M.ws.down_part) {
        g.dpart = M.ws.down_part; g.dpart_block = down_block; g.dpart_splits = M.ws.down_splits;
        g.dpart_cap = c.max_batch; g.dinv = M.ws.inv; g.dmask = M.ws.mask; g.dLm = n_mid(c);
        g.d_upto = d_upto;
    }
    if ((e = mark(M, BUDDY_KERNEL_QKV, l, false, s)) != hipSuccess ||
        (e = launch_proj(M, batch, PRO_RMSNORM, EPI_QKV, g, s)) != hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_QKV, l, true, s)) != hipSuccess)
        return fail_device(M, e, "qkv");
    g.dpart = nullptr;

    // attention over rows 0..pos
    AttnArgs a;
    memset(&a, 0, sizeof(a));
    a.q = bf.q; a.o = bf.o; a.kc = g.kc; a.vc = g.vc;
    a.T = c.max_ctx; a.hd = c.head_dim; a.nq = c.n_heads; a.nkv = c.n_kv_heads;
    a.bcap = c.max_batch; a.pos = M.ws.pos; a.pos_u = pos_u; a.rows = rows;
    a.tok_T = bf.tok_T;
    if (bf.tok_T > 0) {
        // prompt tokens: one chunk per row (no merge; the partials are
        // sized for decode rows only)
        const int r = attention_rows_per_wg(c.dtype, c.head_dim, c.n_heads / c.n_kv_heads);
        a.chunks = 1;
        a.chunk_len = (max_pos + 1 + r - 1) / r * r;
        a.groups = groups; a.n_groups = n_groups;
        // the prefill kernel writes o straight into the O projection's
        // staging when that projection takes the tiled GEMM
        if (groups && uses_gemm(M, rows, batch, qdim, bf.tok_T)) a.xb_out = bf.xb;
    } else {
        // the router's block writing the pool's sums: no more chunks than
        // the pool has splits
        attn_chunks(M, rows.n_max, max_pos, &a.chunks, &a.chunk_len,
                    pooled && !exec ? M.ws.max_pool_splits : kAttnMaxChunks);
        // decode rows on the MFMA path: o goes straight to the O
        // projection's staging, split into bf16 high and low parts as its
        // staging would
        if (uses_mfma(M, rows, batch, qdim, 0)) a.xb_out = bf.xb;
    }
    a.part = M.ws.part; a.max_chunks = M.ws.max_chunks;
    a.exec = exec ? exec + (size_t)l * c.max_batch * c.max_ctx : nullptr;
    if (pooled) {
        *pooled = 0;
        if (bf.tok_T == 0 && !a.exec && a.chunks <= M.ws.max_pool_splits) {
            a.pool_part = M.ws.pool_part;
            a.pool_max_splits = M.ws.max_pool_splits;
            *pooled = a.chunks;
        }
    }
    if ((e = mark(M, BUDDY_KERNEL_ATTENTION, l, false, s)) != hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_ATTN_MERGE, l, false, s)) != hipSuccess ||
        (e = launch_attention(c.dtype, a, s)) != hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_ATTENTION, l, true, s)) != hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_ATTN_MERGE, l, true, s)) != hipSuccess)
        return fail_device(M, e, "attention");

    // h += Wo o.  Decode rows on the MFMA path with an MFMA gate/up behind:
    // K is split and the split sums go to the partial buffer, and the gate/up
    // staging adds them into h before its RMSNorm (no add kernel, a quarter
    // of the activation re-reads of unsplit 16-row tiles)
    const bool o_fold = bf.tok_T == 0 && a.xb_out && uses_mfma(M, rows, batch, qdim, 0) &&
                        uses_mfma(M, rows, batch, c.d_model, 0) && M.ws.mfma_part &&
                        rows.n_max <= M.ws.mfma_part_rows;
    g.W = w.wo; g.N = c.d_model; g.K = qdim; g.X = bf.o; g.ldx = qdim; g.gain = nullptr;
    g.Y = hidden; g.ldy = c.d_model;
    g.part_cap = rows.n_max;
    if ((e = mark(M, BUDDY_KERNEL_O_PROJ, l, false, s)) != hipSuccess ||
        (e = launch_proj(M, batch, a.xb_out ? PRO_STAGED : PRO_NONE, EPI_ADD, g, s, o_fold)) !=
            hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_O_PROJ, l, true, s)) != hipSuccess)
        return fail_device(M, e, "o_proj");

    // m = SiLU(Wg u2) * (Wu u2), u2 = RMSNorm(h); when both MLP projections
    // take the tiled GEMM, or both the MFMA path, m goes straight to the down
    // projection's staging (bf16 fragments in the second buffer)
    const bool m_staged = bf.xb2 && ((uses_gemm(M, rows, batch, c.d_model, bf.tok_T) &&
                                      uses_gemm(M, rows, batch, c.d_ffn, bf.tok_T)) ||
                                     (bf.tok_T == 0 && uses_mfma(M, rows, batch, c.d_model, 0) &&
                                      uses_mfma(M, rows, batch, c.d_ffn, 0)));
    g.W = w.wgate_up; g.N = 2 * c.d_ffn; g.K = c.d_model; g.X = hidden; g.ldx = c.d_model;
    g.gain = w.mlp_norm; g.f = c.d_ffn; g.Y = bf.m; g.ldy = c.d_ffn;
    g.xb_out = m_staged ? bf.xb2 : nullptr;
    if (o_fold) {
        g.addpart = M.ws.mfma_part;
        g.addpart_splits = mfma_fold_splits(c.d_model, qdim);
        g.addpart_cap = rows.n_max;
    }
    if ((e = mark(M, BUDDY_KERNEL_GATE_UP, l, false, s)) != hipSuccess ||
        (e = launch_proj(M, batch, PRO_RMSNORM, EPI_SWIGLU, g, s)) != hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_GATE_UP, l, true, s)) != hipSuccess)
        return fail_device(M, e, "gate_up");
    g.xb_out = nullptr;
    g.addpart = nullptr;

    // h += Wdown m, or (deferred) the split sums left for the sequence's
    // next block to add while staging its input
    g.W = w.wdown; g.N = c.d_model; g.K = c.d_ffn; g.X = bf.m; g.ldx = c.d_ffn;
    g.gain = nullptr; g.Y = hidden; g.ldy = c.d_model;
    if (m_staged) g.XB = bf.xb2;
    const bool defer = d_out >= 0 && M.ws.down_part && m_staged && bf.tok_T == 0;
    // a later staging adds what a deferring block leaves: never a stale buffer
    if (d_out >= 0 && !defer) return fail_device(M, hipErrorInvalidValue, "down (deferred sums)");
    float* down_fold = defer ? M.ws.down_part + (size_t)d_out * down_block : nullptr;
    g.part_cap = c.max_batch;
    if ((e = mark(M, BUDDY_KERNEL_DOWN, l, false, s)) != hipSuccess ||
        (e = launch_proj(M, batch, m_staged ? PRO_STAGED : PRO_NONE, EPI_ADD, g, s, defer, down_fold)) !=
            hipSuccess ||
        (e = mark(M, BUDDY_KERNEL_DOWN, l, true, s)) != hipSuccess)
        return fail_device(M, e, "down");
    return BUDDY_OK;
}

// Router context and the Decision Module's hidden layer for every sequence:
// split sums of the first-layer cache, then the first Decision Module GEMV,
// which folds them into z = [mean K | mean V | h] while staging its input.
// pooled > 0: that block's attention has already written the split sums
// (that many splits), and the cache is not read again.
buddy_status run_planner(Model& M, const buddy_kv* kv, const float* h, int B, int max_pos,
                         int pos_u, bool predict, hipStream_t s, int pooled = 0) {
    const buddy_config& c = M.cfg;
    hipError_t e;
    int splits = 1;
    // the router's cache: the first block's, block S-1's with a start layer
    const void* k0 = layer_base(M, kv->k, start_layer(c) - 1);
    const void* v0 = layer_base(M, kv->v, start_layer(c) - 1);
    if (pooled > 0) {
        splits = pooled;
    } else if (kv->pool_sum) {
        if ((e = launch_pool_running(M, k0, v0, kv->pool_sum, kv->pool_rows, B, pos_u, s)) !=
            hipSuccess)
            return fail_device(M, e, "pool");
    } else if ((e = launch_pool(M, k0, v0, B, max_pos, pos_u, &splits, s)) != hipSuccess) {
        return fail_device(M, e, "pool");
    }
    GemvArgs g;
    memset(&g, 0, sizeof(g));
    g.W = M.dm.w1; g.N = c.dm_hidden;
    g.K = pooled_dim(c.router_ctx, c.n_kv_heads, c.head_dim) + c.d_model;
    g.ctx = c.router_ctx;
    g.rows = Rows{M.ws.idx_all, M.ws.n_all, B, true, true};
    g.Y = M.ws.a; g.ldy = c.dm_hidden;
    g.bias = M.dm.b1; g.act = c.dm_act;
    g.hd = c.head_dim; g.nkv = c.n_kv_heads; g.pos = M.ws.pos; g.pos_u = pos_u;
    g.pool_part = M.ws.pool_part; g.pool_splits = splits;
    g.pool_max_splits = M.ws.max_pool_splits; g.h = h; g.d = c.d_model;
    // the Decision Module keeps fp32 activations at every batch size: routes
    // are decided on these scores
    if ((e = launch_gemv(c.dtype, PRO_POOL, EPI_BIAS_ACT, g, s)) != hipSuccess)
        return fail_device(M, e, "dm_hidden");
    // the Budget Predictor's first layer on the same router context
    if (predict) {
        g.W = M.pred.w1; g.N = M.pred.hidden; g.bias = M.pred.b1;
        g.Y = M.pred_a; g.ldy = M.pred.hidden;
        if ((e = launch_gemv(c.dtype, PRO_POOL, EPI_BIAS_ACT, g, s)) != hipSuccess)
            return fail_device(M, e, "predictor_hidden");
    }
    return BUDDY_OK;
}

// Per-step host values for the device: positions and budgets (kernel
// arguments), the shared position when all sequences have it, and -- only
// when they differ -- the device position array written by setup_kernel.
buddy_status prepare_step(Model& M, const int32_t* pos, const int32_t* k, int B, StepArgs* a,
                          int* pos_u, hipStream_t s) {
    memset(a, 0, sizeof(*a));
    a->B = B;
    *pos_u = pos[0];
    for (int b = 0; b < B; ++b) {
        a->pos[b] = pos[b];
        a->k[b] = k ? (uint8_t)k[b] : 0;
        if (pos[b] != pos[0]) *pos_u = -1;
    }
    if (*pos_u < 0) {
        hipError_t e = launch_setup(*a, M.ws, s);
        if (e != hipSuccess) return fail_device(M, e, "setup");
    }
    return BUDDY_OK;
}

// Host-routed launches: wait until the compaction kernel has published the
// counts of step `seq` to mapped host memory.  A device error, or no answer
// within a minute, ends the wait with BUDDY_EDEVICE.  The stream is queried
// for errors every 100 ms only: a query leaves the next kernel launch on the
// stream 15-20 us slower on the host, and that launch is the one the idle
// device waits for (a step's route takes about a millisecond).  The host
// does not spin for the whole wait: when a step follows the previous one
// back to back (the device is still running that step's blocks), its route
// comes about as long after the call as the previous step's did, so the
// thread sleeps until a margin before that time and spins from there.  A
// route already published on waking halves the next expected wait;
// otherwise the measured wait becomes the next one's expectation.  After a
// pause between steps the device has drained and the route comes at once:
// no sleep.
constexpr int64_t kRouteSpinMarginNs = 150000;
constexpr int64_t kBackToBackNs = 300000;

int64_t steady_ns() {
    return std::chrono::duration_cast<std::chrono::nanoseconds>(
               std::chrono::steady_clock::now().time_since_epoch()).count();
}

buddy_status wait_route(Model& M, int32_t seq, hipStream_t s) {
    volatile int32_t* flag = M.h_cnt + n_mid(M.cfg);
    const auto t0 = std::chrono::steady_clock::now();
    const bool back_to_back = M.step_end_ns > 0 && steady_ns() - M.step_end_ns < kBackToBackNs;
    if (back_to_back && M.route_wait_ns > 2 * kRouteSpinMarginNs && *flag != seq) {
        std::this_thread::sleep_for(std::chrono::nanoseconds(M.route_wait_ns - kRouteSpinMarginNs));
        if (*flag == seq) {
            M.route_wait_ns /= 2;   // woke late: expect less next time
            std::atomic_thread_fence(std::memory_order_acquire);
            return BUDDY_OK;
        }
    }
    auto next_check = t0 + std::chrono::milliseconds(100);
    while (*flag != seq) {
        const auto now = std::chrono::steady_clock::now();
        if (now < next_check) continue;
        next_check = now + std::chrono::milliseconds(100);
        hipError_t e = hipStreamQuery(s);
        if (e != hipSuccess && e != hipErrorNotReady) return fail_device(M, e, "route wait");
        if (now - t0 > std::chrono::seconds(60)) {
            snprintf(M.last_error, sizeof(M.last_error), "route wait: timed out");
            return BUDDY_EDEVICE;
        }
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    M.route_wait_ns = std::chrono::duration_cast<std::chrono::nanoseconds>(
                          std::chrono::steady_clock::now() - t0).count();
    return BUDDY_OK;
}

// Whether the stream is being captured into a graph.
buddy_status stream_capturing(Model& M, hipStream_t s, bool* capturing) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const hipError_t e = hipStreamIsCapturing(s, &cs);
    if (e != hipSuccess) return fail_device(M, e, "capture status");
    *capturing = cs != hipStreamCaptureStatusNone;
    return BUDDY_OK;
}

buddy_status check_step_host(const Model& M, const int32_t* pos, int B, int* max_pos) {
    *max_pos = 0;
    for (int b = 0; b < B; ++b) {
        if (pos[b] < 0 || pos[b] >= M.cfg.max_ctx) return BUDDY_EINVAL;
        if (pos[b] > *max_pos) *max_pos = pos[b];
    }
    return BUDDY_OK;
}

// Scratch of buddy_pool_route_noalloc, in place of a handle's workspace:
// one array per device (each device that loads the library holds its own
// copy at its own address until the process ends).  Host code never uses
// the array's name as an address; it takes the device address that
// hipGetSymbolAddress returns for the current device.
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices];

// Device address of `scratch` on the current device, looked up on the first
// call on that device.
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

buddy_status buddy_model_create(const buddy_config* cfg, const buddy_layer_weights* layers,
                                const buddy_dm_weights* dm, buddy_model** out) {
    if (!out) return BUDDY_EINVAL;
    *out = nullptr;
    buddy_status st = check_config(cfg);
    if (st != BUDDY_OK) return st;
    if (!layers || !dm) return BUDDY_EINVAL;
    for (int l = 0; l < cfg->n_layers; ++l) {
        const buddy_layer_weights& w = layers[l];
        if (!w.attn_norm || !w.wqkv || !w.wo || !w.mlp_norm || !w.wgate_up || !w.wdown)
            return BUDDY_EINVAL;
    }
    if (!dm->w1 || !dm->b1 || !dm->w2 || !dm->b2) return BUDDY_EINVAL;

    buddy_model* h = new (std::nothrow) buddy_model;
    if (!h) return BUDDY_ENOMEM;
    memset(&h->M, 0, sizeof(h->M));
    Model& M = h->M;
    M.cfg = *cfg;
    M.dm = *dm;
    M.layers = (buddy_layer_weights*)malloc(sizeof(buddy_layer_weights) * cfg->n_layers);
    if (!M.layers) { delete h; return BUDDY_ENOMEM; }
    memcpy(M.layers, layers, sizeof(buddy_layer_weights) * cfg->n_layers);
    (void)hipGetDevice(&M.device);

    const buddy_config& c = M.cfg;
    const size_t Bc = c.max_batch, Lm = n_mid(c), hd = c.head_dim;
    const size_t din = pooled_dim(c.router_ctx, c.n_kv_heads, hd) + c.d_model;
    const size_t qdim = (size_t)c.n_heads * hd;
    const int max_chunks = kAttnMaxChunks;
    const int max_splits = pool_max_splits(c.max_ctx);
    M.ws.max_chunks = max_chunks;
    M.ws.max_pool_splits = max_splits;
    size_t xb_ld = (size_t)c.d_model;
    if ((size_t)c.d_ffn > xb_ld) xb_ld = c.d_ffn;
    if (qdim > xb_ld) xb_ld = qdim;
    if (din > xb_ld) xb_ld = din;
    M.ws.xb_ld = (int)xb_ld;

    // K-split partials of the MFMA path (the FFN down projection), for the
    // batch or a short prompt's tokens
    size_t part_elems = 0;
    const int part_rows = Bc > kGemmMinRows ? (int)Bc : kGemmMinRows;
    if (c.dtype == BUDDY_BF16 && Bc > (size_t)kGemvMaxRows) {
        size_t splits = mfma_splits(EPI_ADD, c.d_model, c.d_ffn);
        const size_t so = mfma_fold_splits(c.d_model, (int)qdim);   // the O projection's
        if (so > splits) splits = so;
        if (splits > 1) part_elems = splits * c.d_model * part_rows;
    }
    M.ws.mfma_part_rows = part_elems ? part_rows : 0;
    // deferred down-projection sums of the routable blocks (decode on the
    // MFMA path with the down projection K-split): one buffer per block
    size_t down_elems = 0;
    M.ws.down_splits = 0;
    if (c.dtype == BUDDY_BF16 && Bc > (size_t)kGemvMaxRows && Lm > 0) {
        const int sd = mfma_splits(EPI_ADD, c.d_model, c.d_ffn);
        if (sd > 1 && mfma_fold_splits(c.d_model, c.d_ffn) == sd) {
            M.ws.down_splits = sd;
            down_elems = (size_t)Lm * sd * Bc * c.d_model;
        }
    }

    struct Piece { void** dst; size_t bytes; };
    Workspace& W = M.ws;
    Piece pieces[] = {
        {(void**)&W.pos, Bc * 4}, {(void**)&W.kb, Bc * 4}, {(void**)&W.idx_all, Bc * 4},
        {(void**)&W.n_all, 4}, {(void**)&W.idx, Lm * Bc * 4 + 4}, {(void**)&W.cnt, Lm * 4 + 4},
        {(void**)&W.mask, Bc * Lm + 1}, {(void**)&W.scores, Bc * Lm * 4 + 4},
        {(void**)&W.z, Bc * din * 4}, {(void**)&W.a, Bc * c.dm_hidden * 4},
        {(void**)&W.q, Bc * qdim * 4}, {(void**)&W.o, Bc * qdim * 4},
        {(void**)&W.m, Bc * c.d_ffn * 4},
        {(void**)&W.part, Bc * c.n_heads * max_chunks * (hd + 2) * 4},
        {(void**)&W.pool_part, Bc * c.n_kv_heads * max_splits * 2 * hd * 4},
        {(void**)&W.rope, (size_t)c.max_ctx * (hd / 2) * sizeof(float2)},
        // MFMA staging: high and low bf16 parts of every activation
        {(void**)&W.xb, 2 * ((Bc + 15) / 16 * 16) * xb_ld * sizeof(bf16_t)},
        {(void**)&W.xb2, 2 * ((Bc + 15) / 16 * 16) * xb_ld * sizeof(bf16_t)},
        {(void**)&W.mfma_part, part_elems * 4},
        {(void**)&W.inv, Lm * Bc * 4 + 4},
        {(void**)&W.down_part, down_elems * 4},
    };
    size_t total = 0;
    for (const Piece& p : pieces) total += align_up(p.bytes);
    if (hipMalloc(&M.ws_base, total) != hipSuccess) {
        free(M.layers); delete h; return BUDDY_ENOMEM;
    }
    size_t off = 0;
    for (const Piece& p : pieces) { *p.dst = (char*)M.ws_base + off; off += align_up(p.bytes); }
    if (!down_elems) W.down_part = nullptr;
    hipError_t e = hipMemset(M.ws_base, 0, total);
    // rotary table: angle pos * theta^(-2i/hd) in double, cos and sin rounded to fp32
    const size_t half = hd / 2;
    float2* rope = (float2*)malloc((size_t)c.max_ctx * half * sizeof(float2));
    if (!rope) e = hipErrorOutOfMemory;
    for (size_t i = 0; rope && i < half; ++i) {
        const double inv_freq = pow((double)c.rope_theta, -2.0 * (double)i / (double)hd);
        for (int p = 0; p < c.max_ctx; ++p) {
            const double ang = (double)p * inv_freq;
            rope[(size_t)p * half + i] = make_float2((float)cos(ang), (float)sin(ang));
        }
    }
    if (e == hipSuccess)
        e = hipMemcpy(W.rope, rope, (size_t)c.max_ctx * half * sizeof(float2), hipMemcpyHostToDevice);
    free(rope);
    if (e == hipSuccess)
        e = hipHostMalloc((void**)&M.h_cnt, (Lm + 1) * sizeof(int32_t),
                          hipHostMallocMapped | hipHostMallocCoherent);
    if (e == hipSuccess) {
        memset(M.h_cnt, 0xff, (Lm + 1) * sizeof(int32_t));
        e = hipHostGetDevicePointer((void**)&M.d_host_cnt, M.h_cnt, 0);
    }
    if (e != hipSuccess) {
        if (M.h_cnt) (void)hipHostFree(M.h_cnt);
        (void)hipFree(M.ws_base); free(M.layers); delete h; return BUDDY_EDEVICE;
    }
    *out = h;
    return BUDDY_OK;
}

void buddy_model_destroy(buddy_model* h) {
    if (!h) return;
    (void)hipDeviceSynchronize();
    (void)hipFree(h->M.ws_base);
    (void)hipFree(h->M.pred_a);
    (void)hipFree(h->M.pf_base);
    free(h->M.pf_hlists);
    (void)hipHostFree(h->M.h_cnt);
    free(h->M.layers);
    free(h->M.timing.start);
    free(h->M.timing.stop);
    delete h;
}

buddy_status buddy_pool_route(buddy_model* h, const buddy_kv* kv, const int32_t* pos,
                              const float* h_new, int32_t B, float* scores_out, void* stream) {
    if (!h || !kv_ok(kv)) return BUDDY_EINVAL;
    if (B == 0) return BUDDY_OK;
    if (B < 0) return BUDDY_EINVAL;
    Model& M = h->M;
    if (B > M.cfg.max_batch) return BUDDY_ECAPACITY;
    if (!pos || !h_new || !scores_out) return BUDDY_EINVAL;
    int max_pos;
    buddy_status st = check_step_host(M, pos, B, &max_pos);
    if (st != BUDDY_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    StepArgs a;
    int pos_u;
    if ((st = prepare_step(M, pos, nullptr, B, &a, &pos_u, s)) != BUDDY_OK) return st;
    if ((st = run_planner(M, kv, h_new, B, max_pos, pos_u, false, s)) != BUDDY_OK) return st;
    hipError_t e;
    if ((e = launch_route(M, kv->k, kv->v, nullptr, false, nullptr, nullptr, a, nullptr, nullptr,
                          scores_out, true, -1, s)) != hipSuccess)
        return fail_device(M, e, "scores");
    return BUDDY_OK;
}

buddy_status buddy_pool_route_noalloc(const buddy_config* cfg, const buddy_dm_weights* dm,
                                      const buddy_kv* kv, const int32_t* pos, const float* h_new,
                                      int32_t B, float* scores_out, void* stream) {
    buddy_status st = check_config(cfg);
    if (st != BUDDY_OK) return st;
    if (!dm || !dm->w1 || !dm->b1 || !dm->w2 || !dm->b2 || !kv_ok(kv)) return BUDDY_EINVAL;
    if (B == 0) return BUDDY_OK;
    if (B < 0) return BUDDY_EINVAL;
    if (B > cfg->max_batch) return BUDDY_ECAPACITY;
    if (!pos || !h_new || !scores_out) return BUDDY_EINVAL;
    tl_launch_events = tl_merge_events = {nullptr, nullptr};   // nothing armed by a failed earlier call
    // a model without a workspace: the planner's buffers are carved from the
    // device's scratch array, with the same split count as buddy_pool_route
    Model M;
    memset(&M, 0, sizeof(M));
    M.cfg = *cfg;
    M.dm = *dm;
    int max_pos;
    if ((st = check_step_host(M, pos, B, &max_pos)) != BUDDY_OK) return st;
    const buddy_config& c = M.cfg;
    const int max_splits = pool_max_splits(c.max_ctx);
    // the running-sum pool writes one split
    const int splits = kv->pool_sum ? 1 : pool_splits(B, c.n_kv_heads, max_pos, max_splits);
    const size_t Bs = (size_t)B;
    struct Piece { void** dst; size_t bytes; };
    Workspace& W = M.ws;
    Piece pieces[] = {
        {(void**)&W.pos, Bs * 4}, {(void**)&W.kb, Bs * 4}, {(void**)&W.idx_all, Bs * 4},
        {(void**)&W.n_all, 4}, {(void**)&W.scores, Bs * n_mid(c) * 4 + 4},
        {(void**)&W.a, Bs * c.dm_hidden * 4},
        {(void**)&W.pool_part, Bs * c.n_kv_heads * splits * 2 * c.head_dim * 4},
    };
    size_t total = 0;
    for (const Piece& q : pieces) total += align_up(q.bytes);
    if (total > kNoAllocScratchBytes) return BUDDY_ECAPACITY;
    void* base = nullptr;
    hipError_t e = scratch_address(&base);
    if (e != hipSuccess) return BUDDY_EDEVICE;
    size_t off = 0;
    for (const Piece& q : pieces) { *q.dst = (char*)base + off; off += align_up(q.bytes); }
    W.max_pool_splits = splits;          // partial stride: this call's split count
    hipStream_t s = (hipStream_t)stream;
    StepArgs a;
    int pos_u;
    if ((st = prepare_step(M, pos, nullptr, B, &a, &pos_u, s)) != BUDDY_OK) return st;
    if ((st = run_planner(M, kv, h_new, B, max_pos, pos_u, false, s)) != BUDDY_OK) return st;
    if (launch_route(M, kv->k, kv->v, nullptr, false, nullptr, nullptr, a, nullptr, nullptr,
                     scores_out, true, -1, s) != hipSuccess)
        return BUDDY_EDEVICE;
    return BUDDY_OK;
}

buddy_status buddy_predict_budget(buddy_model* h, const buddy_kv* kv, const int32_t* pos,
                                  const float* h_new, int32_t B, int32_t* k_out,
                                  float* logits_out, void* stream) {
    if (!h || !kv_ok(kv)) return BUDDY_EINVAL;
    if (B == 0) return BUDDY_OK;
    if (B < 0) return BUDDY_EINVAL;
    Model& M = h->M;
    if (B > M.cfg.max_batch) return BUDDY_ECAPACITY;
    if (!pos || !h_new || !k_out || M.pred.hidden == 0) return BUDDY_EINVAL;
    int max_pos;
    buddy_status st = check_step_host(M, pos, B, &max_pos);
    if (st != BUDDY_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    StepArgs a;
    int pos_u;
    if ((st = prepare_step(M, pos, nullptr, B, &a, &pos_u, s)) != BUDDY_OK) return st;
    if ((st = run_planner(M, kv, h_new, B, max_pos, pos_u, true, s)) != BUDDY_OK) return st;
    hipError_t e;
    if ((e = launch_route(M, kv->k, kv->v, nullptr, true, k_out, logits_out, a, nullptr, nullptr,
                          nullptr, true, -1, s)) != hipSuccess)
        return fail_device(M, e, "predictor");
    return BUDDY_OK;
}

buddy_status buddy_set_budget_predictor(buddy_model* h, const buddy_predictor_weights* p) {
    if (!h) return BUDDY_EINVAL;
    Model& M = h->M;
    if (p && (!p->w1 || !p->b1 || !p->w2 || !p->b2 || p->hidden <= 0 || p->hidden % 8 ||
              n_mid(M.cfg) < 1))
        return BUDDY_EINVAL;
    if (p && (size_t)p->hidden > (size_t)64 * 64 * (M.cfg.dtype == BUDDY_BF16 ? 8 : 4))
        return BUDDY_ESHAPE;                       // output-layer rows of at most 64 k-steps
    hipError_t e = hipDeviceSynchronize();         // no step may still read the old head
    if (e != hipSuccess) return fail_device(M, e, "set_budget_predictor");
    (void)hipFree(M.pred_a);
    M.pred_a = nullptr;
    memset(&M.pred, 0, sizeof(M.pred));
    if (!p) return BUDDY_OK;
    e = hipMalloc((void**)&M.pred_a, (size_t)M.cfg.max_batch * p->hidden * sizeof(float));
    if (e != hipSuccess) { M.pred_a = nullptr; return BUDDY_ENOMEM; }
    M.pred = *p;
    return BUDDY_OK;
}

buddy_status buddy_select_topk(const float* scores, const int32_t* k, int32_t B, int32_t n,
                               uint8_t* mask_out, void* stream) {
    if (B == 0) return BUDDY_OK;
    if (!scores || !k || !mask_out || B < 0 || B > 65535 || n < 1 || n > 255) return BUDDY_EINVAL;
    for (int b = 0; b < B; ++b)
        if (k[b] < 0 || k[b] > n) return BUDDY_EINVAL;
    hipError_t e = launch_select_topk(scores, k, B, n, mask_out, (hipStream_t)stream);
    return e == hipSuccess ? BUDDY_OK : BUDDY_EDEVICE;
}

buddy_status buddy_group_by_route(const uint8_t* mask, int32_t B, int32_t n, int32_t* perm_out,
                                  int32_t* starts_out, int32_t* n_groups_out, void* stream) {
    if (B == 0) return BUDDY_OK;
    if (!mask || !perm_out || !starts_out || !n_groups_out || B < 0 || B > kMaxGroupBatch ||
        n < 1 || n > 255)
        return BUDDY_EINVAL;
    hipError_t e = launch_group_by_route(mask, B, n, perm_out, starts_out, n_groups_out,
                                         (hipStream_t)stream);
    return e == hipSuccess ? BUDDY_OK : BUDDY_EDEVICE;
}

namespace {

// One decode step: budgets from k, or from the Budget Predictor (predict),
// or a given route.
buddy_status decode_impl(buddy_model* h, const buddy_kv* kv, float* hidden, const int32_t* pos,
                         const int32_t* k, int32_t B, int32_t skip_kv,
                         const uint8_t* route_override, bool predict, int32_t* k_out,
                         uint8_t* mask_out, float* scores_out, void* stream) {
    if (!h || !kv_ok(kv)) return BUDDY_EINVAL;
    if (skip_kv != BUDDY_SKIP_KV_ZERO && skip_kv != BUDDY_SKIP_KV_MASK) return BUDDY_EINVAL;
    if (B == 0) return BUDDY_OK;
    if (B < 0) return BUDDY_EINVAL;
    Model& M = h->M;
    const buddy_config& c = M.cfg;
    if (B > c.max_batch) return BUDDY_ECAPACITY;
    if (!hidden || !pos || (!k && !route_override && !predict)) return BUDDY_EINVAL;
    if (predict && M.pred.hidden == 0) return BUDDY_EINVAL;
    tl_launch_events = tl_merge_events = {nullptr, nullptr};   // nothing armed by a failed earlier step
    int max_pos;
    buddy_status st = check_step_host(M, pos, B, &max_pos);
    if (st != BUDDY_OK) return st;
    const int Lm = n_mid(c), S = start_layer(c);
    if (!route_override && !predict)
        for (int b = 0; b < B; ++b)
            if (k[b] < 0 || k[b] > Lm) return BUDDY_EINVAL;
    // masking needs the caller's execution map
    uint8_t* exec = skip_kv == BUDDY_SKIP_KV_MASK ? kv->exec : nullptr;
    if (skip_kv == BUDDY_SKIP_KV_MASK && !exec) return BUDDY_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    bool capturing;
    if ((st = stream_capturing(M, s, &capturing)) != BUDDY_OK) return st;
    // the host-routed policy waits for the device, which a captured stream
    // never reaches: refused before anything is enqueued
    if (choose_host_routed(M.policy, false, B, Lm, capturing) < 0) return BUDDY_EINVAL;
    StepArgs a;
    int pos_u;
    if ((st = prepare_step(M, pos, route_override || predict ? nullptr : k, B, &a, &pos_u, s)) !=
        BUDDY_OK)
        return st;
    hipError_t e;

    const Rows all{M.ws.idx_all, M.ws.n_all, B, true, true};
    // first block (blocks 0..S-1) on every sequence; block S-1 appends the
    // K/V row the planner pools, and its attention, which reads every row
    // the pool needs, writes the pool's split sums on the way (unless the
    // route is given, the caller keeps running sums, or the attention
    // leaves rows out by the execution map)
    const bool fuse_pool = !route_override && !kv->pool_sum && !exec;
    int pooled = 0;
    for (int l = 0; l < S; ++l)
        if ((st = run_block(M, kv, exec, hidden, l, all, B, max_pos, pos_u, decode_bufs(M), s, nullptr,
                            0, -1, -1, fuse_pool && l == S - 1 ? &pooled : nullptr)) != BUDDY_OK)
            return st;
    // KV-aware planner and Decision Module, unless the route is given
    if (!route_override)
        if ((st = run_planner(M, kv, hidden, B, max_pos, pos_u, predict, s, pooled)) != BUDDY_OK)
            return st;
    // Launch policy.  Device-routed: every routable block is launched and its
    // kernels read the routed row count on the device (an unused block costs
    // only empty launches).  Host-routed: the compaction kernel publishes the
    // per-block counts to mapped host memory; the host waits for them and
    // launches only the blocks some sequence runs, with exact grids.
    bool all_used = !route_override && !predict;
    for (int b = 0; all_used && b < B; ++b) all_used = k[b] == Lm;
    const int choice = choose_host_routed(M.policy, all_used, B, Lm, capturing);
    const bool host_routed = choice == 1;
    const int32_t seq = host_routed ? (M.seq = (M.seq + 1) & 0x3fffffff) : -1;
    if ((e = launch_route(M, kv->k, kv->v, exec, predict && !route_override, k_out, nullptr, a,
                          route_override, mask_out, scores_out, false, seq, s)) != hipSuccess)
        return fail_device(M, e, "route");
    if (host_routed && (st = wait_route(M, seq, s)) != BUDDY_OK) return st;
    // routable blocks S..L-2 (list i = l - S) on their compacted sub-batches.
    // On the MFMA path each one's down projection leaves its split sums to
    // the staging of the sequence's next block (no add kernel per block);
    // the sums, their order and the residual add are those of the add kernel
    const bool defer = M.ws.down_part && uses_mfma(M, all, B, c.d_model, 0) &&
                       uses_mfma(M, all, B, c.d_ffn, 0);
    for (int l = S; l < S + Lm; ++l) {
        const int i = l - S;
        int n_max = B;
        if (host_routed) {
            n_max = M.h_cnt[i];
            if (n_max == 0) {
                // a timed kernel of a block that does not run: an empty interval
                if (M.timing.n > 0 && M.timing.next < M.timing.n && M.timing.layer == l &&
                    ((e = hipEventRecord(M.timing.start[M.timing.next], s)) != hipSuccess ||
                     (e = hipEventRecord(M.timing.stop[M.timing.next], s)) != hipSuccess))
                    return fail_device(M, e, "timing events");
                continue;
            }
        }
        // every sequence routed (known on the host): the rows are the batch in order
        const Rows r{M.ws.idx + (size_t)i * c.max_batch, M.ws.cnt + i, n_max,
                     host_routed, host_routed && n_max == B};
        if ((st = run_block(M, kv, exec, hidden, l, r, B, max_pos, pos_u, decode_bufs(M), s, nullptr,
                            0, defer ? i : -1, defer ? i : -1)) != BUDDY_OK)
            return st;
    }
    // last block on every sequence (it adds what the routable blocks deferred)
    st = run_block(M, kv, exec, hidden, c.n_layers - 1, all, B, max_pos, pos_u, decode_bufs(M), s,
                   nullptr, 0, defer ? Lm : -1, -1);
    if (M.timing.n > 0 && M.timing.next < M.timing.n) ++M.timing.next;
    M.step_end_ns = steady_ns();
    return st;
}

}  // namespace

buddy_status buddy_decode_step(buddy_model* h, const buddy_kv* kv, float* hidden,
                               const int32_t* pos, const int32_t* k, int32_t B,
                               int32_t skip_kv, const uint8_t* route_override,
                               uint8_t* mask_out, float* scores_out, void* stream) {
    return decode_impl(h, kv, hidden, pos, k, B, skip_kv, route_override, false, nullptr,
                       mask_out, scores_out, stream);
}

buddy_status buddy_decode_step_auto(buddy_model* h, const buddy_kv* kv, float* hidden,
                                    const int32_t* pos, int32_t B, int32_t skip_kv,
                                    int32_t* k_out, uint8_t* mask_out, float* scores_out,
                                    void* stream) {
    return decode_impl(h, kv, hidden, pos, nullptr, B, skip_kv, nullptr, true, k_out, mask_out,
                       scores_out, stream);
}

namespace {

// Grows the prefill workspace to `rows` prompt-token rows (contents are not
// kept).  Waits for the device before freeing the old one.
buddy_status ensure_prefill_ws(Model& M, size_t rows) {
    if (rows <= M.pf_rows) return BUDDY_OK;
    const buddy_config& c = M.cfg;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail_device(M, e, "prefill workspace");
    (void)hipFree(M.pf_base);
    free(M.pf_hlists);
    M.pf_base = nullptr; M.pf_hlists = nullptr; M.pf_rows = 0;
    const size_t qdim = (size_t)c.n_heads * c.head_dim;
    const size_t L = c.n_layers, r16 = (rows + 15) / 16 * 16;
    struct Part { void** p; size_t bytes; } parts[] = {
        {(void**)&M.pf_q, rows * qdim * 4}, {(void**)&M.pf_o, rows * qdim * 4},
        {(void**)&M.pf_m, rows * (size_t)c.d_ffn * 4},
        {(void**)&M.pf_hlast, (size_t)c.max_batch * c.d_model * 4},
        // staging of the tiled GEMM (bf16) or of the MFMA path for few
        // prompt tokens (high and low parts)
        {(void**)&M.pf_xb, 2 * r16 * (size_t)M.ws.xb_ld * sizeof(bf16_t)},
        {(void**)&M.pf_xb2, 2 * r16 * (size_t)M.ws.xb_ld * sizeof(bf16_t)},
        {(void**)&M.pf_split, 2 * rows * (size_t)c.d_model * 4},
        {(void**)&M.pf_lists, L * rows * 4}, {(void**)&M.pf_len, (size_t)c.max_batch * 4},
        {(void**)&M.pf_groups, L * rows * 8},
    };
    size_t total = 0;
    for (auto& q : parts) total += (q.bytes + 255) / 256 * 256;
    if ((e = hipMalloc(&M.pf_base, total)) != hipSuccess) { M.pf_base = nullptr; return BUDDY_ENOMEM; }
    M.pf_hlists = (int32_t*)malloc(L * rows * 12);   // token lists, then group pairs
    if (!M.pf_hlists) { (void)hipFree(M.pf_base); M.pf_base = nullptr; return BUDDY_ENOMEM; }
    size_t off = 0;
    for (auto& q : parts) {
        *q.p = (char*)M.pf_base + off;
        off += (q.bytes + 255) / 256 * 256;
    }
    M.pf_rows = rows;
    return BUDDY_OK;
}

// Attention groups of a token list (tokens of one prompt contiguous and in
// order): runs of up to qt consecutive entries of one prompt, as (first
// entry, count) pairs in out; returns how many.
int token_groups(const int32_t* list, int n, int t_stride, int qt, int32_t* out) {
    int ng = 0;
    for (int i = 0; i < n;) {
        const int b = list[i] / t_stride;
        int cnt = 1;
        while (cnt < qt && i + cnt < n && list[i + cnt] / t_stride == b) ++cnt;
        out[2 * ng] = i;
        out[2 * ng + 1] = cnt;
        ++ng;
        i += cnt;
    }
    return ng;
}

}  // namespace

buddy_status buddy_prefill(buddy_model* h, const buddy_kv* kv, float* hidden, int32_t t_stride,
                           const int32_t* len, const int32_t* k, int32_t B, int32_t skip_kv,
                           const uint8_t* route_override, uint8_t* mask_out, float* scores_out,
                           void* stream) {
    if (!h || !kv_ok(kv)) return BUDDY_EINVAL;
    if (skip_kv != BUDDY_SKIP_KV_ZERO && skip_kv != BUDDY_SKIP_KV_MASK) return BUDDY_EINVAL;
    if (B == 0) return BUDDY_OK;
    if (B < 0) return BUDDY_EINVAL;
    Model& M = h->M;
    const buddy_config& c = M.cfg;
    if (B > c.max_batch) return BUDDY_ECAPACITY;
    if (!hidden || !len || (!k && !route_override) || t_stride < 1) return BUDDY_EINVAL;
    if ((size_t)B * t_stride > kMaxPrefillRows) return BUDDY_ECAPACITY;
    const int Lm = n_mid(c), S = start_layer(c);
    int max_len = 0;
    bool full = true;
    for (int b = 0; b < B; ++b) {
        if (len[b] < 1 || len[b] > t_stride || len[b] > c.max_ctx) return BUDDY_EINVAL;
        if (!route_override && (k[b] < 0 || k[b] > Lm)) return BUDDY_EINVAL;
        if (len[b] > max_len) max_len = len[b];
        full = full && len[b] == t_stride;
    }
    uint8_t* exec = skip_kv == BUDDY_SKIP_KV_MASK ? kv->exec : nullptr;
    if (skip_kv == BUDDY_SKIP_KV_MASK && !exec) return BUDDY_EINVAL;
    tl_launch_events = tl_merge_events = {nullptr, nullptr};
    buddy_status st;
    hipStream_t s = (hipStream_t)stream;
    bool capturing;
    if ((st = stream_capturing(M, s, &capturing)) != BUDDY_OK) return st;
    if (capturing) return BUDDY_EINVAL;     // the prefill waits for its route on the host
    if ((st = ensure_prefill_ws(M, (size_t)B * t_stride)) != BUDDY_OK) return st;
    hipError_t e;
    // the prompt rewrites the first block's rows of slots 0..B-1: their
    // running pool sums start over
    if (kv->pool_rows && (e = hipMemsetAsync(kv->pool_rows, 0, (size_t)B * c.n_kv_heads * 4, s)) !=
                             hipSuccess)
        return fail_device(M, e, "prefill pool");
    const size_t R = M.pf_rows;
    const BlockBufs bf{M.pf_q, M.pf_o, M.pf_m, M.pf_xb, M.ws.xb_ld, t_stride, M.pf_xb2};

    // every prompt token (list 0) for the first and last blocks; with more
    // than one token per attention group, the group pairs of list l at
    // [L R + 2 l R] (host) and [2 l R] (device)
    int32_t* hl = M.pf_hlists;
    int32_t* hg = hl + (size_t)c.n_layers * R;
    const int qt = attention_prefill_group(c.dtype, c.head_dim, c.n_heads / c.n_kv_heads);
    std::vector<int> n_g(c.n_layers, 0);
    int n_all = 0;
    for (int b = 0; b < B; ++b)
        for (int t = 0; t < len[b]; ++t) hl[n_all++] = b * t_stride + t;
    if (qt > 1) n_g[0] = token_groups(hl, n_all, t_stride, qt, hg);
    if ((e = hipMemcpyAsync(M.pf_lists, hl, (size_t)n_all * 4, hipMemcpyHostToDevice, s)) !=
            hipSuccess ||
        (qt > 1 && (e = hipMemcpyAsync(M.pf_groups, hg, (size_t)n_g[0] * 8,
                                       hipMemcpyHostToDevice, s)) != hipSuccess) ||
        (e = hipMemcpyAsync(M.pf_len, len, (size_t)B * 4, hipMemcpyHostToDevice, s)) != hipSuccess)
        return fail_device(M, e, "prefill lists");
    auto groups_of = [&](int l) { return qt > 1 ? M.pf_groups + (size_t)2 * l * R : nullptr; };
    const Rows all{M.pf_lists, nullptr, n_all, true, full};
    // blocks 0..S-1 over every token, unmasked: their map entries are
    // written with the route, and every prompt token runs them
    for (int l = 0; l < S; ++l)
        if ((st = run_block(M, kv, nullptr, hidden, l, all, n_all, max_len - 1, -1, bf, s,
                            groups_of(0), n_g[0])) != BUDDY_OK)
            return st;

    // one route per prompt: the planner and Decision Module at the last token
    std::vector<uint8_t> mask((size_t)B * (Lm > 0 ? Lm : 1));
    if (route_override) {
        if ((e = hipMemcpyAsync(mask.data(), route_override, (size_t)B * Lm, hipMemcpyDeviceToHost,
                                s)) != hipSuccess ||
            (e = hipMemcpyAsync(M.ws.mask, route_override, (size_t)B * Lm,
                                hipMemcpyDeviceToDevice, s)) != hipSuccess)
            return fail_device(M, e, "prefill route");
        if (mask_out && (e = hipMemcpyAsync(mask_out, route_override, (size_t)B * Lm,
                                            hipMemcpyDeviceToDevice, s)) != hipSuccess)
            return fail_device(M, e, "prefill route");
    } else {
        std::vector<int32_t> last(B);
        for (int b = 0; b < B; ++b) last[b] = len[b] - 1;
        StepArgs a;
        int pos_u;
        if ((st = prepare_step(M, last.data(), k, B, &a, &pos_u, s)) != BUDDY_OK) return st;
        if ((e = launch_gather_last(hidden, t_stride, c.d_model, M.pf_len, B, M.pf_hlast, s)) !=
            hipSuccess)
            return fail_device(M, e, "prefill gather");
        if ((st = run_planner(M, kv, M.pf_hlast, B, max_len - 1, pos_u, false, s)) != BUDDY_OK)
            return st;
        if ((e = launch_route(M, kv->k, kv->v, nullptr, false, nullptr, nullptr, a, nullptr,
                              mask_out, scores_out, false, -1, s)) != hipSuccess ||
            (e = hipMemcpyAsync(mask.data(), M.ws.mask, (size_t)B * Lm, hipMemcpyDeviceToHost,
                                s)) != hipSuccess)
            return fail_device(M, e, "prefill route");
    }
    // zero-filled rows (and execution-map entries) of the skipped blocks
    if ((e = launch_prefill_fill(M, kv->k, kv->v, exec, M.ws.mask, M.pf_len, B, max_len, s)) !=
        hipSuccess)
        return fail_device(M, e, "prefill fill");
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return fail_device(M, e, "prefill route");

    // token lists of the routable blocks S..L-2 (list l), then the blocks
    // over their tokens
    std::vector<int> n_l(c.n_layers, 0);
    for (int l = S; l < S + Lm; ++l) {
        int32_t* dst = hl + (size_t)l * R;
        for (int b = 0; b < B; ++b)
            if (mask[(size_t)b * Lm + (l - S)])
                for (int t = 0; t < len[b]; ++t) dst[n_l[l]++] = b * t_stride + t;
        if (qt > 1) n_g[l] = token_groups(dst, n_l[l], t_stride, qt, hg + (size_t)2 * l * R);
    }
    if (Lm > 0 && ((e = hipMemcpyAsync(M.pf_lists + S * R, hl + S * R, (size_t)Lm * R * 4,
                                       hipMemcpyHostToDevice, s)) != hipSuccess ||
                   (qt > 1 && (e = hipMemcpyAsync(M.pf_groups + 2 * S * R, hg + 2 * S * R,
                                                  (size_t)Lm * R * 8, hipMemcpyHostToDevice,
                                                  s)) != hipSuccess)))
        return fail_device(M, e, "prefill lists");
    for (int l = S; l < S + Lm; ++l) {
        if (n_l[l] == 0) continue;
        const Rows r{M.pf_lists + (size_t)l * R, nullptr, n_l[l], true, full && n_l[l] == n_all};
        if ((st = run_block(M, kv, exec, hidden, l, r, n_l[l], max_len - 1, -1, bf, s, groups_of(l),
                            n_g[l])) != BUDDY_OK)
            return st;
    }
    st = run_block(M, kv, exec, hidden, c.n_layers - 1, all, n_all, max_len - 1, -1, bf, s,
                   groups_of(0), n_g[0]);
    if (st == BUDDY_OK && (e = hipStreamSynchronize(s)) != hipSuccess)
        return fail_device(M, e, "prefill");   // the host token lists are reused next call
    return st;
}

buddy_status buddy_set_launch_policy(buddy_model* h, int32_t policy) {
    if (!h || policy < BUDDY_LAUNCH_AUTO || policy > BUDDY_LAUNCH_HOST_ROUTED) return BUDDY_EINVAL;
    h->M.policy = policy;
    return BUDDY_OK;
}

buddy_status buddy_set_gemm_tile(buddy_model* h, int32_t tile) {
    if (!h || tile < BUDDY_GEMM_TILE_AUTO || tile > BUDDY_GEMM_TILE_256_SPLIT) return BUDDY_EINVAL;
    h->M.gemm_tile = tile;
    return BUDDY_OK;
}

buddy_status buddy_set_timing_events(buddy_model* h, int32_t kernel, int32_t layer,
                                     void* const* start, void* const* stop, int32_t n) {
    if (!h || n < 0 || kernel < BUDDY_KERNEL_QKV || kernel > BUDDY_KERNEL_ATTN_MERGE)
        return BUDDY_EINVAL;
    Model& M = h->M;
    if (layer < 0 || layer >= M.cfg.n_layers) return BUDDY_EINVAL;
    if (n > 0 && (!start || !stop)) return BUDDY_EINVAL;
    free(M.timing.start);
    free(M.timing.stop);
    memset(&M.timing, 0, sizeof(M.timing));
    if (n == 0) return BUDDY_OK;
    M.timing.start = (hipEvent_t*)malloc(sizeof(hipEvent_t) * n);
    M.timing.stop = (hipEvent_t*)malloc(sizeof(hipEvent_t) * n);
    if (!M.timing.start || !M.timing.stop) {
        free(M.timing.start); free(M.timing.stop);
        memset(&M.timing, 0, sizeof(M.timing));
        return BUDDY_ENOMEM;
    }
    memcpy(M.timing.start, start, sizeof(hipEvent_t) * n);
    memcpy(M.timing.stop, stop, sizeof(hipEvent_t) * n);
    M.timing.kernel = kernel;
    M.timing.layer = layer;
    M.timing.n = n;
    return BUDDY_OK;
}

int32_t buddy_budget_to_k(float b, int32_t n_layers) {
    if (!(b > 0.f && b <= 1.f) || n_layers < 2) return -1;
    int32_t k = (int32_t)floor((double)b * n_layers + 0.5) - 2;
    if (k < 0) k = 0;
    if (k > n_layers - 2) k = n_layers - 2;
    return k;
}

const char* buddy_status_string(buddy_status s) {
    switch (s) {
        case BUDDY_OK: return "ok";
        case BUDDY_EINVAL: return "invalid argument";
        case BUDDY_ESHAPE: return "unsupported shape";
        case BUDDY_ECAPACITY: return "batch above capacity";
        case BUDDY_ENOMEM: return "out of device memory";
        case BUDDY_EDEVICE: return "HIP error";
        case BUDDY_EUNSUPPORTED: return "not implemented";
    }
    return "unknown status";
}

const char* buddy_last_error(const buddy_model* h) { return h ? h->M.last_error : ""; }

}  // extern "C"
