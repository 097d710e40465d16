// Internal declarations shared by the HIP translation units of libbuddy.
// Device helpers, the workspace layout and the launcher entry points that
// the host API (api.hip) calls.  gfx950 only: 64-lane wavefronts.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "../../include/buddy.h"

namespace buddy {

typedef uint16_t bf16_t;

constexpr int kMaxBatch = 256;     // batch capacity limit (one WG scans a column)
constexpr int kMaxPrefillRows = 65535;  // prompt-token rows of one prefill call (grid z)
constexpr int kMaxGroup = 8;       // query heads per KV head held in registers
constexpr int kWave = 64;
constexpr int kAttnMaxChunks = 256;  // position chunks per (sequence, KV head)

// ---------------------------------------------------------------- storage

__device__ __forceinline__ float bf2f(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// fp32 -> bf16, round to nearest, ties to even; NaN becomes the quiet NaN
// of its sign.  The conversion is gfx950's v_cvt_pk_bf16_f32, which gives
// the same bits as adding 0x7fff plus the lowest kept bit and truncating, on
// every non-NaN input (compared over all 2^32 inputs on the device); only
// NaN payloads differ, hence the select.
__device__ __forceinline__ bf16_t f2bf(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t rounded = __builtin_bit_cast(unsigned short, (__bf16)f);
    const uint32_t qnan = ((u >> 16) & 0x8000u) | 0x7fc0u;
    return (bf16_t)((u & 0x7fffffffu) > 0x7f800000u ? qnan : rounded);
}

// Two fp32 values as packed bf16 (a in the low half), round to nearest
// even, in one v_cvt_pk_bf16_f32; NaNs stay NaNs but keep a payload, so this
// is for MFMA operands, and f2bf for values that are stored.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

// Start layer S of the router (0 in the config reads as 1): blocks 0..S-1
// always run, blocks S..L-2 are routable (n_mid of them).
inline int start_layer(const buddy_config& c) { return c.start_layer > 0 ? c.start_layer : 1; }
inline int n_mid(const buddy_config& c) { return c.n_layers - 1 - start_layer(c); }

template <typename T> struct St;
template <> struct St<float> {
    static constexpr int V = 4;  // elements per 16-byte vector
    __device__ static float get(const float* p, size_t i) { return p[i]; }
    __device__ static void put(float* p, size_t i, float v) { p[i] = v; }
    __device__ static void vec(const float* p, float* out) {
        float4 w = *reinterpret_cast<const float4*>(p);
        out[0] = w.x; out[1] = w.y; out[2] = w.z; out[3] = w.w;
    }
};
template <> struct St<bf16_t> {
    static constexpr int V = 8;
    __device__ static float get(const bf16_t* p, size_t i) { return bf2f(p[i]); }
    __device__ static void put(bf16_t* p, size_t i, float v) { p[i] = f2bf(v); }
    __device__ static void vec(const bf16_t* p, float* out) {
        uint4 w = *reinterpret_cast<const uint4*>(p);
        out[0] = __uint_as_float(w.x << 16); out[1] = __uint_as_float(w.x & 0xffff0000u);
        out[2] = __uint_as_float(w.y << 16); out[3] = __uint_as_float(w.y & 0xffff0000u);
        out[4] = __uint_as_float(w.z << 16); out[5] = __uint_as_float(w.z & 0xffff0000u);
        out[6] = __uint_as_float(w.w << 16); out[7] = __uint_as_float(w.w & 0xffff0000u);
    }
};

// Raw 16-byte weight vectors stay packed in registers until they are used.
template <typename TW>
__device__ __forceinline__ void unpack(const uint4& w, float* out);
template <>
__device__ __forceinline__ void unpack<bf16_t>(const uint4& w, float* out) {
    out[0] = __uint_as_float(w.x << 16); out[1] = __uint_as_float(w.x & 0xffff0000u);
    out[2] = __uint_as_float(w.y << 16); out[3] = __uint_as_float(w.y & 0xffff0000u);
    out[4] = __uint_as_float(w.z << 16); out[5] = __uint_as_float(w.z & 0xffff0000u);
    out[6] = __uint_as_float(w.w << 16); out[7] = __uint_as_float(w.w & 0xffff0000u);
}
template <>
__device__ __forceinline__ void unpack<float>(const uint4& w, float* out) {
    out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
    out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
}

// ------------------------------------------------------------- reductions

// Sum over the wavefront, every lane receiving it: the butterfly of lane
// pairs 32, 16, 8, 4, 2 and 1 apart.  The first two steps take the partner
// from the gfx950 lane swaps (v_permlane32_swap / v_permlane16_swap: a lane's
// own value and its partner's in the two results), the last four from DPP
// rotations within 16-lane rows (by 8, 4, 2, 1): after the wider steps the
// lane a rotation reaches holds the same value as the partner, so every sum
// has the operands of the shuffle butterfly (bit-identical results) without
// a round trip through the LDS unit per step.
__device__ __forceinline__ float wave_sum(float v) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    constexpr int kRowRor = 0x120;   // DPP control: rotate right within each row
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 8, 0xf, 0xf, true));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 4, 0xf, 0xf, true));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 2, 0xf, 0xf, true));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 1, 0xf, 0xf, true));
    return v;
}

// Maximum over the wavefront, every lane receiving it, by the same steps.
__device__ __forceinline__ float wave_max(float v) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    constexpr int kRowRor = 0x120;
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 8, 0xf, 0xf, true)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 4, 0xf, 0xf, true)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 2, 0xf, 0xf, true)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), kRowRor + 1, 0xf, 0xf, true)));
    return v;
}

// --------------------------------------------------------------- workspace

struct Workspace {
    int32_t* pos;        // [max_batch]   positions of this step
    int32_t* kb;         // [max_batch]   budgets
    int32_t* idx_all;    // [max_batch]   identity row list for blocks 0 and L-1
    int32_t* n_all;      // [1]           = B
    int32_t* idx;        // [L-2][max_batch] per-block routed rows, ascending
    int32_t* cnt;        // [L-2]         routed row count per block
    uint8_t* mask;       // [max_batch][L-2] executed mask
    float* scores;       // [max_batch][L-2]
    float* z;            // [max_batch][din]  router context
    float* a;            // [max_batch][dm_hidden]
    float* q;            // [max_batch][n_heads hd]  rotated queries
    float* o;            // [max_batch][n_heads hd]  attention output
    float* m;            // [max_batch][d_ffn]       SwiGLU output
    float* part;         // attention partials [max_batch][n_heads][max_chunks][hd + 2]
    float* pool_part;    // pool partials [max_batch][n_kv][max_pool_splits][2 hd]
    float2* rope;        // [max_ctx][hd/2] (cos, sin) of pos * theta^(-2i/hd)
    bf16_t* xb;          // [2][round16(max_batch)][xb_ld] MFMA staging, high and low parts
    bf16_t* xb2;         // the same, for the down projection's input
    float* mfma_part;    // K-split partial sums of the MFMA path (see mfma_splits)
    int mfma_part_rows;  // routed rows the partial buffer holds (0: no buffer)
    int32_t* inv;        // [L-2][max_batch] launch row of sequence b in block i's list, or -1
    // K-split sums of each routable block's down projection, added by the
    // staging of the sequence's next block (decode on the MFMA path):
    // [L-2][splits][max_batch][d], or null
    float* down_part;
    int down_splits;
    int xb_ld;
    int max_chunks;
    int max_pool_splits;
};

// Caller-owned HIP events recorded around one kernel of one block per step.
struct TimingHook {
    int kernel, layer, n, next;
    hipEvent_t* start;
    hipEvent_t* stop;
};

// Events that the next main kernel launch (a projection, the MFMA product,
// an attention score kernel) records at its own dispatch begin and end, the
// interval a profiler's kernel trace reports; armed by the timing hook for
// one launch and cleared by that launch.
struct LaunchEvents { hipEvent_t start, stop; };
extern thread_local LaunchEvents tl_launch_events;
// The same for the attention's chunk-merge launch.
extern thread_local LaunchEvents tl_merge_events;

template <typename... KArgs, typename... Args>
inline void launch_main(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t lds,
                        hipStream_t s, Args... args) {
    LaunchEvents& ev = tl_launch_events;
    if (ev.start) {
        hipExtLaunchKernelGGL(kernel, grid, block, lds, s, ev.start, ev.stop, 0, args...);
        ev.start = ev.stop = nullptr;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
    }
}

// Largest batch for which the automatic launch policy waits for the route
// and launches only the blocks in use (at larger batches nearly every block
// is used by some sequence).
constexpr int kHostRoutedMaxBatch = 16;

// Launch policy of the routable blocks of one step: 1 host-routed (the host
// waits for the route and launches only the blocks in use), 0 device-routed,
// -1 refused.  A stream being captured into a graph never runs while the
// host waits, so AUTO then takes the device-routed launches and an explicit
// host-routed request is refused.  Lm: routable blocks (none: nothing to
// wait for); all_used: every sequence runs every routable block.
inline int choose_host_routed(int policy, bool all_used, int B, int Lm, bool capturing) {
    if (Lm <= 0 || policy == BUDDY_LAUNCH_DEVICE_ROUTED) return 0;
    if (policy == BUDDY_LAUNCH_HOST_ROUTED) return capturing ? -1 : 1;
    return !all_used && B <= kHostRoutedMaxBatch && !capturing ? 1 : 0;
}

struct Model {
    buddy_config cfg;
    TimingHook timing;
    int policy;                   // buddy_launch_policy
    int gemm_tile;                // buddy_gemm_tile
    int32_t* h_cnt;               // mapped pinned host memory: [L-2] counts, then a sequence number
    int32_t* d_host_cnt;          // device address of h_cnt
    int32_t seq;                  // sequence number of the last published route
    int64_t route_wait_ns;        // how long the host-routed wait is expected to take (0: unknown)
    int64_t step_end_ns;          // steady-clock time the last decode step's enqueue ended (0: none)
    buddy_layer_weights* layers;  // host array of device pointers
    buddy_dm_weights dm;
    buddy_predictor_weights pred;  // Budget Predictor head (pred.hidden == 0: none)
    float* pred_a;                 // [max_batch][pred.hidden] its hidden activations
    // prefill workspace, grown on demand to pf_rows prompt-token rows (one
    // allocation): queries, attention outputs, SwiGLU outputs, MFMA staging,
    // per-block token lists [L][rows], prompt lengths, last-token hidden rows
    void* pf_base; size_t pf_rows;
    float *pf_q, *pf_o, *pf_m, *pf_hlast;
    bf16_t* pf_xb, *pf_xb2;
    float* pf_split;               // split-K partial sums [2][rows][d_model]
    int32_t *pf_lists, *pf_len, *pf_groups;
    int32_t* pf_hlists;            // host copy of the token lists, then of the groups
    Workspace ws;
    void* ws_base;                // one allocation holding the workspace
    int device;
    char last_error[256];
};

// Per-step host values handed to the device through kernel arguments.
struct StepArgs {
    int32_t B;
    int32_t pos[kMaxBatch];
    uint8_t k[kMaxBatch];
};

// --------------------------------------------------------------- launchers

// Row set of one routed launch: rows i < *cnt map to sequences idx[i]; the
// grid is sized for at most n_max rows.  exact: the host knows that *cnt is
// n_max (kernels then need not read the count before starting).  identity:
// row i is sequence i (every sequence of the batch, in order), so kernels
// need not read idx either.
struct Rows {
    const int32_t* idx;
    const int32_t* cnt;
    int n_max;
    bool exact;
    bool identity;
};

__device__ __forceinline__ int row_seq(const Rows& r, int i) { return r.identity ? i : r.idx[i]; }

// Position of sequence b this step: pos_u when every sequence shares it
// (no memory read), else the published per-sequence array.
__device__ __forceinline__ int seq_pos(const int32_t* pos, int pos_u, int b) {
    return pos_u >= 0 ? pos_u : pos[b];
}

// Cache slot and position of row id b: in a decode step the row is a
// sequence at its step position; in a prefill (tok_T > 0) it is a flattened
// prompt token, slot b / tok_T at position b % tok_T.
__device__ __forceinline__ void slot_pos(int b, int tok_T, const int32_t* pos, int pos_u,
                                         int& slot, int& p) {
    if (tok_T > 0) { slot = b / tok_T; p = b - slot * tok_T; }
    else { slot = b; p = seq_pos(pos, pos_u, b); }
}

hipError_t launch_setup(const StepArgs& a, const Workspace& ws, hipStream_t s);

// Position splits per (sequence, KV head) of the pool over rows 0..max_pos:
// about four workgroups per CU to stream the first-layer cache, at least 64
// rows each, at most max_splits (few enough partials for the fold).
inline int pool_splits(int B, int nkv, int max_pos, int max_splits) {
    const int want = (1024 + B * nkv - 1) / (B * nkv);
    const int by_len = (max_pos + 1 + 63) / 64;
    int splits = want < by_len ? want : by_len;
    if (splits < 1) splits = 1;
    if (splits > max_splits) splits = max_splits;
    return splits;
}
// Most position splits per (sequence, KV head) for a cache of max_ctx rows.
inline int pool_max_splits(int max_ctx) {
    const int s = (max_ctx + 63) / 64;
    return s > 64 ? 64 : s;
}

// Split sums of the first layer's K/V rows 0..pos; returns the number of
// splits per (sequence, KV head) in *splits (the Decision Module GEMV folds
// them, PRO_POOL).
hipError_t launch_pool(const Model& M, const void* k0, const void* v0, int B, int max_pos,
                       int pos_u, int* splits, hipStream_t s);
// The same context from running sums (buddy_kv.pool_sum / pool_rows): adds
// the rows not yet summed, writes one split of partial sums (row pos
// included) for the fold.
hipError_t launch_pool_running(const Model& M, const void* k0, const void* v0, float* pool_sum,
                               int32_t* pool_rows, int B, int pos_u, hipStream_t s);

// Decision Module second layer + prior + top-k (or the override mask), then
// zero-fill of skipped K/V rows and per-block compaction.
// publish_seq >= 0: also publish the per-block counts and then publish_seq
// to the mapped host buffer (host-routed launches wait for it).  Budgets and
// positions travel in `a`.
// predict: the Budget Predictor's logits (from M.pred_a) pick each
// sequence's k instead of a.k; k_out / logits_out receive them (nullable).
hipError_t launch_route(const Model& M, const void* kc, const void* vc, uint8_t* exec, bool predict,
                        int32_t* k_out, float* logits_out, const StepArgs& a,
                        const uint8_t* route_override, uint8_t* mask_out,
                        float* scores_out, bool scores_only, int32_t publish_seq,
                        hipStream_t s);

// Prefill: zero-fills the K/V rows 0..len[b]-1 of every block sequence b
// skips (mask [B][L-2]) and, with an execution map, writes its entries for
// those rows in every block.
hipError_t launch_prefill_fill(const Model& M, void* kc, void* vc, uint8_t* exec,
                               const uint8_t* mask, const int32_t* len, int B, int max_len,
                               hipStream_t s);
// Prefill: the last prompt token's hidden row of every sequence, compacted
// to [B][d].
hipError_t launch_gather_last(const float* hidden, int t_stride, int d, const int32_t* len, int B,
                              float* out, hipStream_t s);
hipError_t launch_select_topk(const float* scores, const int32_t* k_host, int B, int n,
                              uint8_t* mask_out, hipStream_t s);
// Batch-level path grouping (buddy_group_by_route), B <= kMaxGroupBatch,
// 1 <= n <= 256.
constexpr int kMaxGroupBatch = 1024;
hipError_t launch_group_by_route(const uint8_t* mask, int B, int n, int32_t* perm, int32_t* starts,
                                 int32_t* n_groups, hipStream_t s);

enum Pro { PRO_NONE = 0, PRO_RMSNORM = 1, PRO_POOL = 2, PRO_STAGED = 3 };
// PRO_STAGED (tiled GEMM and MFMA paths): the input rows are already in XB,
// written there in fragment order by the producing kernel.
enum Epi { EPI_ADD = 0, EPI_BIAS_ACT = 1, EPI_SWIGLU = 2, EPI_QKV = 3 };

struct GemvArgs {
    const void* W; int N; int K;       // weight [N][K]
    const float* X; int ldx;           // activation rows, indexed by sequence
    const void* gain; float eps;       // PRO_RMSNORM
    Rows rows;
    float* Y; int ldy;                 // output rows, indexed by sequence
    const void* bias; int act;         // EPI_BIAS_ACT
    int f;                             // EPI_SWIGLU: rows j and f + j
    // EPI_QKV: rotary + cache append of this block (tok_T > 0: rows are
    // prompt tokens, see slot_pos)
    void* kc; void* vc; int T; int hd; int nq; int nkv; int bcap;
    const int32_t* pos; int pos_u; const float2* rope; int tok_T;
    // PRO_POOL: X is unused; row b of the input is the router context,
    // pooled first-layer features of variant ctx (buddy_router_ctx) built
    // from the pool's split partial sums, then h
    const float* pool_part; int pool_splits, pool_max_splits; const float* h; int d; int ctx;
    // MFMA path: compact activation rows, split high / low bf16 fragments
    // (xbs_index; the prefill's tiled GEMM: one bf16 fragment, xb_index)
    bf16_t* XB; int ldxb;
    // PRO_RMSNORM on the MFMA path: K-split partial sums of the preceding
    // residual-add projection, [split][row capacity][K] by launch row, that
    // the staging adds into X's rows (in split order, written back) before
    // the norm; or null
    const float* addpart; int addpart_splits; int addpart_cap;
    // PRO_RMSNORM on the MFMA path, decode rows: the deferred sums of the
    // down projections.  Routable block i's down projection leaves its split
    // sums at dpart + i dpart_block ([split][dpart_cap][K] by that block's
    // launch row); the staging adds, for each of its sequences b, those of
    // the last routable block before list index d_upto that b ran (dmask
    // [B][dLm]), at row dinv[i dpart_cap + b], into X's row (in split order,
    // written back) before the norm; or null
    const float* dpart; size_t dpart_block; int dpart_splits; int dpart_cap;
    const int32_t* dinv; const uint8_t* dmask; int dLm; int d_upto;
    // MFMA residual-add projection with fold: the row capacity of its
    // [split][row][N] partial sums
    int part_cap;
    // EPI_SWIGLU (tiled GEMM and MFMA paths): the outputs in the next
    // projection's staging order with K = f (its staged input) instead of Y:
    // xb_index bf16 for the tiled GEMM, xbs_index split for the MFMA path
    bf16_t* xb_out;
};

// Element (row i, column k) of activations in B-operand fragment order for
// a K-column input: 16 rows x 32 columns per contiguous 1 KB fragment, lane
// (i % 16) + 16 ((k / 8) % 4) holding columns 8 (k / 8) .. + 7.
__host__ __device__ inline size_t xb_index(int i, int k, int K) {
    return ((((size_t)(i >> 4) * (K >> 5) + (k >> 5)) * 64 + (i & 15) + 16 * ((k >> 3) & 3)) << 3) +
           (k & 7);
}

// Split activations of the decode MFMA path: each value as its bf16
// rounding (high part) plus the bf16 rounding of the remainder (low part),
// about 16 significant bits together, so that the bf16 products see the
// fp32 activations almost exactly (the weights are bf16 already).  Element
// (row i, column k) of part p (0 high, 1 low) for a K-column input: tile
// i / 16 and k-step k / 32 hold two contiguous 1 KB fragments, high then
// low, each in B-operand order (lane (i % 16) + 16 ((k / 8) % 4), element
// k % 8).
__host__ __device__ inline size_t xbs_index(int i, int k, int K, int part) {
    return (((((size_t)(i >> 4) * (K >> 5) + (k >> 5)) * 2 + part) * 64 + (i & 15) +
             16 * ((k >> 3) & 3)) << 3) + (k & 7);
}

// Low part of v given its high part's bits: the exact remainder rounded to
// bf16, 0 where v or its high part is not finite (they then decide alone).
__device__ __forceinline__ float split_rest(float v, uint32_t hi_bits16) {
    const float r = v - bf2f(hi_bits16);
    return (r - r) == 0.f ? r : 0.f;
}

// Stores v at high-part index `at` (xbs_index with part 0) and its low part
// one fragment (512 elements) further.
__device__ __forceinline__ void store_split(bf16_t* xb, size_t at, float v) {
    const bf16_t hi = f2bf(v);
    xb[at] = hi;
    xb[at + 512] = f2bf(split_rest(v, hi));
}

// Pooled inputs of the router context: 2 n_kv hd for [mean K | mean V],
// n_kv hd for the single-feature variants.
__host__ __device__ inline int pooled_dim(int ctx, int nkv, int hd) {
    return (ctx == BUDDY_CTX_KV ? 2 : 1) * nkv * hd;
}

// Router-context inputs k .. k+3 (k % 4 == 0, k < pooled_dim) of sequence b:
// the split sums of the pool for mean K, mean V or their sum, times 1/n.
__device__ __forceinline__ float4 pooled_feature4(const GemvArgs& g, int b, int k, float inv_n) {
    const int nh = g.nkv * g.hd;
    int kk = k, first = 0, last = 0;          // feature rows 0 (K) .. 1 (V) to add
    if (g.ctx == BUDDY_CTX_KV) { first = last = k / nh; kk = k - first * nh; }
    else if (g.ctx == BUDDY_CTX_V) { first = last = 1; }
    else if (g.ctx == BUDDY_CTX_K_PLUS_V) { last = 1; }
    const int gg = kk / g.hd, e = kk - gg * g.hd;
    const float* pp = g.pool_part + ((size_t)b * g.nkv + gg) * g.pool_max_splits * 2 * g.hd + e;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (first == last) {
        // one feature row: the splits' loads are independent, so eight at a
        // time are in flight; the sum keeps split order
        const float* p1 = pp + (size_t)first * g.hd;
#pragma unroll 8
        for (int q = 0; q < g.pool_splits; ++q) {
            const float4 t = *reinterpret_cast<const float4*>(p1 + (size_t)q * 2 * g.hd);
            v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
        }
    } else {
        // K + V: both rows of each split, in split order, four splits' loads
        // in flight at a time
#pragma unroll 4
        for (int q = 0; q < g.pool_splits; ++q) {
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const float4 t = *reinterpret_cast<const float4*>(pp + ((size_t)q * 2 + w) * g.hd);
                v.x += t.x; v.y += t.y; v.z += t.z; v.w += t.w;
            }
        }
    }
    v.x *= inv_n; v.y *= inv_n; v.z *= inv_n; v.w *= inv_n;
    return v;
}
hipError_t launch_gemv(int dtype, int pro, int epi, const GemvArgs& g, hipStream_t s);
// MFMA path (bf16 weights, K a multiple of 128): prep of the compact bf16
// rows, then the MFMA projection with the same epilogues.  part: fp32
// workspace of mfma_part_elems for the K-split projections.
// fold: for a residual-add projection, K is split per mfma_fold_splits and
// the split sums go to part by launch row ([split][n_max][N]) for the next
// staging to add (GemvArgs.addpart), instead of into Y.
hipError_t launch_mfma(int pro, int epi, const GemvArgs& g, float* part, hipStream_t s,
                       bool fold = false);
// The activation staging of the MFMA paths: routed rows as bf16 in B-operand
// fragment order (g.XB), RMSNorm / router context folded in per pro.
hipError_t launch_prep(int pro, const GemvArgs& g, hipStream_t s);
// Tiled MFMA GEMM for many rows (prompt tokens): exact row counts, bf16
// weights, K a multiple of 64.
// part: fp32 workspace of 2 x rows x N for the split-K residual-add
// projections (null: no split).
hipError_t launch_gemm(int pro, int epi, const GemvArgs& g, int tile, float* part, hipStream_t s);
constexpr int kGemmMinRows = 64;
// Routed rows above which a bf16 projection takes the MFMA path.
constexpr int kGemvMaxRows = 4;
// MFMA path: workgroups below which a launch takes smaller weight tiles per
// workgroup or splits K; the most K splits.
constexpr int kMfmaMinGrid = 384;
constexpr int kMfmaMaxSplits = 8;

// K splits of an MFMA projection of `units` output rows over K inputs
// (residual-add kinds).  A workgroup reads every routed activation row of
// its K range for its weight rows, so the activation bytes a CU fetches per
// weight byte are n / (rows per workgroup): long-K projections (K >= 2
// units, the FFN down projection) whose 64-row tiles give fewer than
// kMfmaMinGrid workgroups split K over up to kMfmaMaxSplits workgroups
// instead of shrinking the tile; a second kernel adds the split sums in a
// fixed order.  Their partial sums (splits x n x units) stay small next to
// the weights because K is long.  Fixed by the shape alone: a sequence's
// sums never depend on the batch or its routes.
inline int mfma_splits(int epi, int units, int K) {
    if (epi != EPI_ADD || K % 32 != 0 || K < 2 * units) return 1;
    const int grid = (units + 63) / 64;
    if (grid >= kMfmaMinGrid) return 1;
    const int S = K / 32;
    int splits = 1;
    for (int c = 2; c <= kMfmaMaxSplits; c *= 2) {
        if (S % (4 * c) != 0) break;
        splits = c;
        if (grid * c >= 256) break;
    }
    return splits;
}

// K splits of a residual-add MFMA projection whose split sums are added by
// the next projection's staging (no add kernel): 64-row tiles, K split until
// the grid has 256 workgroups (at most kMfmaMaxSplits, whole rounds of four
// k-steps per wavefront).  Fixed by the shape alone.
inline int mfma_fold_splits(int units, int K) {
    if (K % 32 != 0) return 1;
    const int grid = (units + 63) / 64, S = K / 32;
    int splits = 1;
    for (int c = 2; c <= kMfmaMaxSplits; c *= 2) {
        if (S % (4 * c) != 0) break;
        splits = c;
        if (grid * c >= 256) break;
    }
    return splits;
}

struct AttnArgs {
    const float* q; float* o;
    const void* kc; const void* vc;    // this block's cache base
    int T, hd, nq, nkv, bcap;
    const int32_t* pos; int pos_u;
    Rows rows;
    int chunks, chunk_len;
    float* part; int max_chunks;
    const uint8_t* exec;                // this block's execution map [bcap][T], or null
    int tok_T;                          // > 0: rows are prompt tokens (slot_pos)
    // o of launch row i in the O projection's staging order instead of fp32
    // o (decode rows: split high / low, xbs_index; prompt tokens of the
    // prefill attention kernel: bf16, xb_index, with K = nq hd); or null
    bf16_t* xb_out;
    // prompt tokens on the prefill attention kernel: groups of up to 128 / G
    // consecutive tokens of one prompt, (first row index, count) pairs; one
    // workgroup per (KV head, group) (null: one per row)
    const int32_t* groups; int n_groups;
    // decode rows of the router's block, no execution map: each workgroup
    // also writes the column sums of the K and V rows of its chunk to the
    // pool's partial sums, split c at pool_part [b][nkv][pool_max_splits]
    // [K | V][hd] (the pool kernel's layout); or null
    float* pool_part; int pool_max_splits;
};
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s);
// Cache rows one attention workgroup reads per block (chunk lengths are
// multiples of it).
int attention_rows_per_wg(int dtype, int hd, int G);
// Prompt tokens per attention workgroup of a prefill (1: no grouping).
int attention_prefill_group(int dtype, int hd, int G);

}  // namespace buddy
