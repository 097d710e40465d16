// Router-side kernels of the budget-routed decode step (gfx950).
//
//  setup_kernel   publishes the step's positions and budgets to device memory
//                 and the identity row list used by the always-run blocks.
//  pool_kernel    KV-aware planner (Sec. 4.3): sums of the first layer's K
//                 and V rows 0..pos per KV head over a few split position
//                 ranges; the Decision Module's first GEMV folds the splits
//                 into the means and joins the newest hidden state,
//                 z = [mean K | mean V | h] (PRO_POOL in k_gemv.hip).
//  pool_running_kernel  the same sums kept across steps in caller memory:
//                 only rows not yet summed are read (normally one per
//                 sequence and step).
//  route_kernel   Decision Module output layer plus prior fusion (Eq. 2),
//                 deterministic top-k by rank counting, zero-fill of the K/V
//                 row of every skipped block (Conclusion: non-executed states
//                 are zero vectors) and, with skipped-KV masking, the step's
//                 entries of the execution map; with a single sequence it
//                 also does the compaction below.
//  compact_kernel grouping by mask (App. C.1): for every routable block the
//                 ascending list of sequences that run it, their count and
//                 each sequence's row in the list (-1 if absent).
//  topk_kernel    the standalone top-k entry point.
// Partial results always travel through a kernel boundary; no kernel here
// synchronises workgroups (device-wide fences are costly across the XCDs).
#include "buddy_internal.h"

namespace buddy {

// ------------------------------------------------------------------ setup

__global__ __launch_bounds__(256) void setup_kernel(StepArgs a, Workspace ws) {
    const int t = threadIdx.x;
    if (t < a.B) {
        ws.pos[t] = a.pos[t];
        ws.kb[t] = a.k[t];
        ws.idx_all[t] = t;
    }
    if (t == 0) ws.n_all[0] = a.B;
}

hipError_t launch_setup(const StepArgs& a, const Workspace& ws, hipStream_t s) {
    setup_kernel<<<1, 256, 0, s>>>(a, ws);
    return hipGetLastError();
}

// ------------------------------------------------------------------- pool

struct PoolParams {
    const void* k0; const void* v0;  // first layer's cache base
    const int32_t* pos; int pos_u;
    float* part;
    int T, hd, nkv, splits, max_splits;
};

typedef uint32_t pool_u4 __attribute__((ext_vector_type(4)));
// 16 bytes of a cache row as fp32 (8 bf16 or 4 fp32 values), nontemporal
__device__ __forceinline__ void nt_vec(const bf16_t* q, float* out) {
    const pool_u4 w = __builtin_nontemporal_load(reinterpret_cast<const pool_u4*>(q));
    out[0] = __uint_as_float(w.x << 16); out[1] = __uint_as_float(w.x & 0xffff0000u);
    out[2] = __uint_as_float(w.y << 16); out[3] = __uint_as_float(w.y & 0xffff0000u);
    out[4] = __uint_as_float(w.z << 16); out[5] = __uint_as_float(w.z & 0xffff0000u);
    out[6] = __uint_as_float(w.w << 16); out[7] = __uint_as_float(w.w & 0xffff0000u);
}
__device__ __forceinline__ void nt_vec(const float* q, float* out) {
    const pool_u4 w = __builtin_nontemporal_load(reinterpret_cast<const pool_u4*>(q));
    out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
    out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
}

template <typename T>
__global__ __launch_bounds__(256) void pool_kernel(PoolParams p) {
    constexpr int V = St<T>::V;
    __shared__ float red[2][256 * V];   // [K|V][row slot][hd] partial sums
    const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int n = seq_pos(p.pos, p.pos_u, b) + 1;
    const int cpr = p.hd / V;           // threads per cache row
    const int rpp = 256 / cpr;          // rows per pass
    const int col = tid % cpr, slot = tid / cpr;
    const int len = (n + p.splits - 1) / p.splits;
    const int j0 = s * len, j1 = min(j0 + len, n);
    const size_t base = ((size_t)b * p.nkv + g) * p.T * p.hd;
    const T* K = (const T*)p.k0 + base;
    const T* Vc = (const T*)p.v0 + base;

    float ak[V], av[V];
#pragma unroll
    for (int e = 0; e < V; ++e) ak[e] = av[e] = 0.f;
    // the rows are read once here (this step's first-block attention has
    // already run): nontemporal 16-byte loads
#pragma unroll 4
    for (int j = j0 + slot; j < j1; j += rpp) {
        float kr[V], vr[V];
        nt_vec(K + (size_t)j * p.hd + col * V, kr);
        nt_vec(Vc + (size_t)j * p.hd + col * V, vr);
#pragma unroll
        for (int e = 0; e < V; ++e) { ak[e] += kr[e]; av[e] += vr[e]; }
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
        red[0][slot * p.hd + col * V + e] = ak[e];
        red[1][slot * p.hd + col * V + e] = av[e];
    }
    __syncthreads();
    float* part = p.part + (((size_t)b * p.nkv + g) * p.max_splits) * 2 * p.hd;
    for (int t = tid; t < 2 * p.hd; t += 256) {
        const int which = t / p.hd, e = t % p.hd;
        float acc = 0.f;
        for (int r = 0; r < rpp; ++r) acc += red[which][r * p.hd + e];
        part[(size_t)s * 2 * p.hd + t] = acc;
    }
}

hipError_t launch_pool(const Model& M, const void* k0, const void* v0, int B, int max_pos,
                       int pos_u, int* splits_out, hipStream_t s) {
    const buddy_config& c = M.cfg;
    PoolParams p;
    p.k0 = k0; p.v0 = v0; p.pos = M.ws.pos; p.pos_u = pos_u;
    p.part = M.ws.pool_part;
    p.T = c.max_ctx; p.hd = c.head_dim; p.nkv = c.n_kv_heads; p.max_splits = M.ws.max_pool_splits;
    const int splits = pool_splits(B, c.n_kv_heads, max_pos, p.max_splits);
    p.splits = splits;
    *splits_out = splits;
    dim3 grid(splits, c.n_kv_heads, B);
    if (c.dtype == BUDDY_BF16) pool_kernel<bf16_t><<<grid, 256, 0, s>>>(p);
    else pool_kernel<float><<<grid, 256, 0, s>>>(p);
    return hipGetLastError();
}

// Running sums: one workgroup per (KV head, sequence) owns its record, so
// the sums and the row count need no synchronisation between workgroups.
// Rows n0..pos-1 join the kept sums (n0 = pool_rows; a count of 0 or above
// pos starts over from empty sums); row pos joins only this call's split.
template <typename T>
__global__ __launch_bounds__(1024) void pool_running_kernel(PoolParams p, float* sum,
                                                            int32_t* rows) {
    constexpr int V = St<T>::V;
    __shared__ float red[2][16][128];   // [K|V][wavefront][hd] partial sums
    const int g = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x;
    const int pos = seq_pos(p.pos, p.pos_u, b);
    int32_t* cnt = rows + (size_t)b * p.nkv + g;
    float* rec = sum + ((size_t)b * p.nkv + g) * 2 * p.hd;
    int n0 = *cnt;
    const bool restart = n0 <= 0 || n0 > pos;   // count 0: the kept sums are not read
    if (restart) n0 = 0;
    const int cpr = p.hd / V, rpp = 1024 / cpr;
    const int col = tid % cpr, slot = tid / cpr;
    const size_t base = ((size_t)b * p.nkv + g) * p.T * p.hd;
    const T* K = (const T*)p.k0 + base;
    const T* Vc = (const T*)p.v0 + base;
    float ak[V], av[V];
#pragma unroll
    for (int e = 0; e < V; ++e) ak[e] = av[e] = 0.f;
    for (int j = n0 + slot; j < pos; j += rpp) {
        float kr[V], vr[V];
        St<T>::vec(K + (size_t)j * p.hd + col * V, kr);
        St<T>::vec(Vc + (size_t)j * p.hd + col * V, vr);
#pragma unroll
        for (int e = 0; e < V; ++e) { ak[e] += kr[e]; av[e] += vr[e]; }
    }
    // rows of one wavefront first (lanes cpr apart share a column), then
    // the 16 wavefronts through LDS
    const int lane = tid & 63, wave = tid >> 6;
    for (int o = cpr; o < kWave; o <<= 1) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
            ak[e] += __shfl_xor(ak[e], o, kWave);
            av[e] += __shfl_xor(av[e], o, kWave);
        }
    }
    if (lane < cpr) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
            red[0][wave][col * V + e] = ak[e];
            red[1][wave][col * V + e] = av[e];
        }
    }
    __syncthreads();   // every thread has also read *cnt before it is replaced
    float* part = p.part + ((size_t)b * p.nkv + g) * p.max_splits * 2 * p.hd;
    for (int t = tid; t < 2 * p.hd; t += 1024) {
        const int which = t / p.hd, e = t % p.hd;
        float acc = restart ? 0.f : rec[t];
        for (int w = 0; w < 16; ++w) acc += red[which][w][e];
        rec[t] = acc;
        part[t] = acc + St<T>::get(which ? Vc : K, (size_t)pos * p.hd + e);
    }
    if (tid == 0) *cnt = pos;
}

hipError_t launch_pool_running(const Model& M, const void* k0, const void* v0, float* pool_sum,
                               int32_t* pool_rows, int B, int pos_u, hipStream_t s) {
    const buddy_config& c = M.cfg;
    PoolParams p;
    p.k0 = k0; p.v0 = v0; p.pos = M.ws.pos; p.pos_u = pos_u;
    p.part = M.ws.pool_part;
    p.T = c.max_ctx; p.hd = c.head_dim; p.nkv = c.n_kv_heads; p.max_splits = M.ws.max_pool_splits;
    p.splits = 1;
    dim3 grid(c.n_kv_heads, B);
    if (c.dtype == BUDDY_BF16) pool_running_kernel<bf16_t><<<grid, 1024, 0, s>>>(p, pool_sum, pool_rows);
    else pool_running_kernel<float><<<grid, 1024, 0, s>>>(p, pool_sum, pool_rows);
    return hipGetLastError();
}

// ------------------------------------------------------------------ route

// Strict total order of the top-k: a number beats NaN, larger beats smaller,
// equal values go to the lower layer index.
__device__ __forceinline__ bool beats(float sj, int j, float si, int i) {
    const bool nj = isnan(sj), ni = isnan(si);
    if (nj != ni) return ni;
    if (!nj && sj != si) return sj > si;
    return j < i;
}

struct RouteParams {
    const float* a; int H;
    const void* w2; const void* b2; const float* prior; float omega;
    int Lm, B;
    int S, L;                         // start layer (routable blocks S..L-2), blocks
    const uint8_t* route_override;
    uint8_t* mask; uint8_t* mask_out;
    float* scores; float* scores_out;
    void* kc; void* vc;               // cache bases (layer 0)
    int T, hd, nkv, bcap;
    int scores_only;
    int32_t* idx; int32_t* cnt;       // compaction outputs (single-sequence launch)
    volatile int32_t* host_cnt; int32_t seq;
    uint8_t* exec;                    // execution map [L][bcap][T] (masking), or null
    // Budget Predictor: hidden activations [B][Hp] (null: budgets from the
    // step arguments), output layer, and the optional outputs
    const float* pa; int Hp; const void* pw2; const void* pb2;
    int32_t* k_out; float* logits_out;
};

// Groups by mask the routed blocks of a one-sequence batch and publishes the
// counts (shared by route_kernel at B = 1 and compact_kernel).
__device__ __forceinline__ void publish_counts(volatile int32_t* host_cnt, int Lm, int32_t seq) {
    __threadfence_system();
    host_cnt[Lm] = seq;
}

// One output layer row per wavefront: v[i] = W[i] . a + bias[i] (fp32).
template <typename T>
__device__ __forceinline__ void output_layer(const void* w, const void* bias, const float* a,
                                             int H, int Lm, int wave, int lane, float* v) {
    constexpr int V = St<T>::V;
    const int nv = H / V;              // 16-byte vectors per row
    for (int i = wave; i < Lm; i += 16) {
        float acc = 0.f;
        for (int q = lane; q < nv; q += kWave) {
            float wv[V];
            St<T>::vec((const T*)w + (size_t)i * H + q * V, wv);
#pragma unroll
            for (int e = 0; e < V; ++e) acc += wv[e] * a[q * V + e];
        }
        acc = wave_sum(acc);
        if (lane == 0) v[i] = acc + St<T>::get((const T*)bias, i);
    }
}

template <typename T>
__global__ __launch_bounds__(1024) void route_kernel(RouteParams p, StepArgs sa) {
    __shared__ float s_sc[256];
    __shared__ uint8_t s_mask[256];
    __shared__ int s_k;
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int Lm = p.Lm;

    // Budget Predictor (Sec. 4.4): k = 1 + argmax of the policy logits (the
    // softmax is monotone), smaller k on equal logits, NaN never chosen
    if (p.pa) {
        output_layer<T>(p.pw2, p.pb2, p.pa + (size_t)b * p.Hp, p.Hp, Lm, wave, lane, s_sc);
        __syncthreads();
        if (tid < Lm && p.logits_out) p.logits_out[(size_t)b * Lm + tid] = s_sc[tid];
        if (wave == 0) {
            float bv = 0.f;
            int bi = Lm;                                  // none yet
            for (int i = lane; i < Lm; i += kWave) {
                const float v = s_sc[i];
                if (v == v && (bi == Lm || v > bv)) { bv = v; bi = i; }
            }
            for (int o = kWave / 2; o > 0; o >>= 1) {
                const float ov = __shfl_xor(bv, o, kWave);
                const int oi = __shfl_xor(bi, o, kWave);
                if (oi != Lm && (bi == Lm || ov > bv || (ov == bv && oi < bi))) { bv = ov; bi = oi; }
            }
            if (lane == 0) {
                s_k = (bi == Lm ? 0 : bi) + 1;
                if (p.k_out) p.k_out[b] = s_k;
            }
        }
        __syncthreads();   // s_sc is reused for the scores below
    }
    const int kb = p.pa ? s_k : (int)sa.k[b];

    if (p.route_override) {
        if (tid < Lm) s_mask[tid] = p.route_override[(size_t)b * Lm + tid] != 0;
    } else {
        output_layer<T>(p.w2, p.b2, p.a + (size_t)b * p.H, p.H, Lm, wave, lane, s_sc);
        __syncthreads();
        if (p.prior && tid < Lm) s_sc[tid] += p.omega * p.prior[tid];
        __syncthreads();
        if (tid < Lm) {
            p.scores[(size_t)b * Lm + tid] = s_sc[tid];
            if (p.scores_out) p.scores_out[(size_t)b * Lm + tid] = s_sc[tid];
        }
        if (p.scores_only) return;
        if (tid < Lm) {
            const float si = s_sc[tid];
            int rank = 0;
            for (int j = 0; j < Lm; ++j) rank += (j != tid) && beats(s_sc[j], j, si, tid);
            s_mask[tid] = rank < kb;
        }
    }
    __syncthreads();
    if (tid < Lm) {
        p.mask[(size_t)b * Lm + tid] = s_mask[tid];
        if (p.mask_out) p.mask_out[(size_t)b * Lm + tid] = s_mask[tid];
        if (gridDim.x == 1) {   // one sequence: this workgroup is the compaction
            p.idx[(size_t)tid * p.bcap] = 0;
            p.cnt[tid] = s_mask[tid];
            if (p.host_cnt) p.host_cnt[tid] = s_mask[tid];
        }
    }
    if (gridDim.x == 1 && p.host_cnt) {
        __syncthreads();
        if (tid == 0) publish_counts(p.host_cnt, Lm, p.seq);
    }

    // with masking, every block's entry of the execution map at this step's
    // position: 1 for blocks 0..S-1, the last block and the selected ones
    const int pos = sa.pos[b];
    if (p.exec && tid < p.L)
        p.exec[((size_t)tid * p.bcap + b) * p.T + pos] =
            (tid < p.S || tid == p.L - 1) ? 1 : s_mask[tid - p.S];

    // zero-filled K/V row at this step's position for every skipped block,
    // written as 16-byte vectors
    constexpr int VZ = St<T>::V;
    const size_t layer_stride = (size_t)p.bcap * p.nkv * p.T * p.hd;
    const int per_layer = p.nkv * (p.hd / VZ);
    for (int t = tid; t < Lm * per_layer; t += 1024) {
        const int i = t / per_layer, r = t % per_layer;
        if (s_mask[i]) continue;
        const int g = r / (p.hd / VZ), e = (r % (p.hd / VZ)) * VZ;
        const size_t at = (size_t)(i + p.S) * layer_stride +
                          (((size_t)b * p.nkv + g) * p.T + pos) * p.hd + e;
        *reinterpret_cast<uint4*>((T*)p.kc + at) = make_uint4(0u, 0u, 0u, 0u);
        *reinterpret_cast<uint4*>((T*)p.vc + at) = make_uint4(0u, 0u, 0u, 0u);
    }
}

// One workgroup: each wavefront scans the mask columns of every fourth
// routable block over the batch (inv: [Lm][bcap] rows).  When host_cnt (mapped pinned host memory)
// is given, the counts are also published there, followed by the step's
// sequence number once they are visible to the host.
__global__ __launch_bounds__(256) void compact_kernel(const uint8_t* mask, int Lm, int B, int bcap,
                                                      int32_t* idx, int32_t* cnt, int32_t* inv,
                                                      volatile int32_t* host_cnt, int32_t seq) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = wave; i < Lm; i += 4) {
        int base = 0;
        for (int b0 = 0; b0 < B; b0 += kWave) {
            const int bb = b0 + lane;
            const bool sel = bb < B && mask[(size_t)bb * Lm + i];
            const uint64_t bal = __ballot(sel);
            const int before = __popcll(bal & ((1ull << lane) - 1ull));
            if (sel) idx[(size_t)i * bcap + base + before] = bb;
            if (bb < B) inv[(size_t)i * bcap + bb] = sel ? base + before : -1;
            base += __popcll(bal);
        }
        if (lane == 0) {
            cnt[i] = base;
            if (host_cnt) host_cnt[i] = base;
        }
    }
    if (host_cnt) {
        __syncthreads();
        if (tid == 0) publish_counts(host_cnt, Lm, seq);
    }
}

hipError_t launch_route(const Model& M, const void* kc, const void* vc, uint8_t* exec, bool predict,
                        int32_t* k_out, float* logits_out, const StepArgs& a,
                        const uint8_t* route_override, uint8_t* mask_out,
                        float* scores_out, bool scores_only, int32_t publish_seq,
                        hipStream_t s) {
    const buddy_config& c = M.cfg;
    const int B = a.B;
    RouteParams p;
    p.a = M.ws.a; p.H = c.dm_hidden;
    p.w2 = M.dm.w2; p.b2 = M.dm.b2; p.prior = M.dm.prior; p.omega = M.dm.omega;
    p.Lm = n_mid(c); p.B = B;
    p.S = start_layer(c); p.L = c.n_layers;
    p.route_override = route_override;
    p.mask = M.ws.mask; p.mask_out = mask_out;
    p.scores = M.ws.scores; p.scores_out = scores_out;
    p.kc = (void*)kc; p.vc = (void*)vc;
    p.T = c.max_ctx; p.hd = c.head_dim; p.nkv = c.n_kv_heads; p.bcap = c.max_batch;
    p.scores_only = scores_only ? 1 : 0;
    p.idx = M.ws.idx; p.cnt = M.ws.cnt;
    p.host_cnt = publish_seq >= 0 ? M.d_host_cnt : nullptr;
    p.seq = publish_seq;
    p.exec = exec;
    p.pa = predict ? M.pred_a : nullptr; p.Hp = M.pred.hidden;
    p.pw2 = M.pred.w2; p.pb2 = M.pred.b2;
    p.k_out = k_out; p.logits_out = logits_out;
    if (c.dtype == BUDDY_BF16) route_kernel<bf16_t><<<B, 1024, 0, s>>>(p, a);
    else route_kernel<float><<<B, 1024, 0, s>>>(p, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || scores_only || p.Lm == 0 || B == 1) return e;
    compact_kernel<<<1, 256, 0, s>>>(M.ws.mask, p.Lm, B, c.max_batch, M.ws.idx, M.ws.cnt,
                                     M.ws.inv, p.host_cnt, publish_seq);
    return hipGetLastError();
}

// ---------------------------------------------------------------- prefill

// One workgroup per (sequence, block): zero rows 0..len-1 of a skipped
// block (16-byte stores) and, with an execution map, its entries.
template <typename T>
__global__ __launch_bounds__(256) void prefill_fill_kernel(void* kc, void* vc, uint8_t* exec,
                                                           const uint8_t* mask, const int32_t* len,
                                                           int S, int L, int T_cap, int bcap,
                                                           int nkv, int hd) {
    const int b = blockIdx.y, l = blockIdx.x;      // block l of 0..L-1
    const int n = len[b];
    const int Lm = L - 1 - S;
    const bool run = l < S || l == L - 1 || mask[(size_t)b * Lm + (l - S)];
    if (exec)
        for (int t = threadIdx.x; t < n; t += 256) exec[((size_t)l * bcap + b) * T_cap + t] = run;
    if (run) return;
    constexpr int V = St<T>::V;
    const int per_row = hd / V;
    const size_t layer = (size_t)l * bcap * nkv * T_cap * hd;
    for (int t = threadIdx.x; t < nkv * n * per_row; t += 256) {
        const int g = t / (n * per_row), r = t - g * n * per_row;
        const int row = r / per_row, e = (r - row * per_row) * V;
        const size_t at = layer + (((size_t)b * nkv + g) * T_cap + row) * hd + e;
        *reinterpret_cast<uint4*>((T*)kc + at) = make_uint4(0u, 0u, 0u, 0u);
        *reinterpret_cast<uint4*>((T*)vc + at) = make_uint4(0u, 0u, 0u, 0u);
    }
}

hipError_t launch_prefill_fill(const Model& M, void* kc, void* vc, uint8_t* exec,
                               const uint8_t* mask, const int32_t* len, int B, int max_len,
                               hipStream_t s) {
    const buddy_config& c = M.cfg;
    (void)max_len;
    const dim3 grid(c.n_layers, B);
    if (c.dtype == BUDDY_BF16)
        prefill_fill_kernel<bf16_t><<<grid, 256, 0, s>>>(kc, vc, exec, mask, len, start_layer(c),
                                                         c.n_layers, c.max_ctx, c.max_batch,
                                                         c.n_kv_heads, c.head_dim);
    else
        prefill_fill_kernel<float><<<grid, 256, 0, s>>>(kc, vc, exec, mask, len, start_layer(c),
                                                        c.n_layers, c.max_ctx, c.max_batch,
                                                        c.n_kv_heads, c.head_dim);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void gather_last_kernel(const float* hidden, int t_stride, int d,
                                                          const int32_t* len, float* out) {
    const int b = blockIdx.x;
    const float* src = hidden + ((size_t)b * t_stride + len[b] - 1) * d;
    for (int i = threadIdx.x; i < d; i += 256) out[(size_t)b * d + i] = src[i];
}

hipError_t launch_gather_last(const float* hidden, int t_stride, int d, const int32_t* len, int B,
                              float* out, hipStream_t s) {
    gather_last_kernel<<<B, 256, 0, s>>>(hidden, t_stride, d, len, out);
    return hipGetLastError();
}

// ----------------------------------------------------------- select_topk

struct TopkArgs {
    int n, rows;
    uint8_t k[kMaxBatch];
};

__global__ __launch_bounds__(256) void topk_kernel(const float* scores, uint8_t* mask, TopkArgs a) {
    __shared__ float s_sc[256];
    const int r = blockIdx.x, tid = threadIdx.x;
    if (tid < a.n) s_sc[tid] = scores[(size_t)r * a.n + tid];
    __syncthreads();
    if (tid < a.n) {
        const float si = s_sc[tid];
        int rank = 0;
        for (int j = 0; j < a.n; ++j) rank += (j != tid) && beats(s_sc[j], j, si, tid);
        mask[(size_t)r * a.n + tid] = rank < (int)a.k[r];
    }
}

// ------------------------------------------------------- path grouping

// One workgroup orders the batch by route: each sequence's route (mask row,
// nonzero = run) is packed into four 64-bit words, block 0 in the top bit of
// word 0, so that comparing the words as unsigned numbers in order compares
// routes lexicographically with skip before run; a sequence's position is
// the count of (route, index) keys below its own, which is unique.  Groups
// start where the route differs from the previous position's (flags, then a
// scan in LDS).
__global__ __launch_bounds__(1024) void group_kernel(const uint8_t* mask, int B, int n, int32_t* perm,
                                                     int32_t* starts, int32_t* n_groups) {
    __shared__ uint64_t s_key[kMaxGroupBatch][4];
    __shared__ int32_t s_perm[kMaxGroupBatch];
    __shared__ int32_t s_scan[kMaxGroupBatch];
    const int t = threadIdx.x;
    if (t < B) {
        uint64_t w[4] = {0, 0, 0, 0};
        const uint8_t* row = mask + (size_t)t * n;
        for (int i = 0; i < n; ++i)
            if (row[i]) w[i >> 6] |= 1ull << (63 - (i & 63));
#pragma unroll
        for (int q = 0; q < 4; ++q) s_key[t][q] = w[q];
    }
    __syncthreads();
    if (t < B) {
        const uint64_t k0 = s_key[t][0], k1 = s_key[t][1], k2 = s_key[t][2], k3 = s_key[t][3];
        int rank = 0;
        for (int b = 0; b < B; ++b) {
            const uint64_t o0 = s_key[b][0], o1 = s_key[b][1], o2 = s_key[b][2], o3 = s_key[b][3];
            bool below;
            if (o0 != k0) below = o0 < k0;
            else if (o1 != k1) below = o1 < k1;
            else if (o2 != k2) below = o2 < k2;
            else if (o3 != k3) below = o3 < k3;
            else below = b < t;
            rank += below;
        }
        s_perm[rank] = t;
        perm[rank] = t;
    }
    __syncthreads();
    int flag = 0;
    if (t < B) {
        const int a = s_perm[t];
        flag = t == 0;
        if (t > 0) {
            const int p = s_perm[t - 1];
#pragma unroll
            for (int q = 0; q < 4; ++q) flag |= s_key[a][q] != s_key[p][q];
        }
    }
    // inclusive scan of the flags: group index + 1 at each position
    if (t < kMaxGroupBatch) s_scan[t] = flag;
    __syncthreads();
    for (int off = 1; off < kMaxGroupBatch; off <<= 1) {
        const int v = t < kMaxGroupBatch && t >= off ? s_scan[t - off] : 0;
        __syncthreads();
        if (t < kMaxGroupBatch) s_scan[t] += v;
        __syncthreads();
    }
    if (t < B && flag) starts[s_scan[t] - 1] = t;
    if (t == 0) {
        const int g = B > 0 ? s_scan[B - 1] : 0;
        starts[g] = B;
        *n_groups = g;
    }
}

hipError_t launch_group_by_route(const uint8_t* mask, int B, int n, int32_t* perm, int32_t* starts,
                                 int32_t* n_groups, hipStream_t s) {
    group_kernel<<<1, kMaxGroupBatch, 0, s>>>(mask, B, n, perm, starts, n_groups);
    return hipGetLastError();
}

hipError_t launch_select_topk(const float* scores, const int32_t* k_host, int B, int n,
                              uint8_t* mask_out, hipStream_t s) {
    for (int r0 = 0; r0 < B; r0 += kMaxBatch) {
        TopkArgs a;
        a.n = n;
        a.rows = B - r0 < kMaxBatch ? B - r0 : kMaxBatch;
        for (int r = 0; r < a.rows; ++r) a.k[r] = (uint8_t)k_host[r0 + r];
        topk_kernel<<<a.rows, 256, 0, s>>>(scores + (size_t)r0 * n, mask_out + (size_t)r0 * n, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace buddy
