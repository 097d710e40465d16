// Split-K grouped-query decode attention over the KV cache (gfx950).
//
// For a routed sequence b, KV head g and position chunk c, one workgroup
// scores the G = n_heads / n_kv_heads query heads of the group against cache
// rows j in the chunk (j <= pos[b]; the new row written by the projection
// kernel is included, as in the KV-cache equation of the paper's background
// appendix), keeps an online softmax (running max and sum, base 2) and the
// weighted sum of V rows, then writes the chunk's (max, sum, acc) partial.
// A second kernel merges the chunk partials of (b, g) in chunk order and
// writes o[b] for the group's heads (no cross-workgroup synchronisation
// inside a kernel: device-wide fences are costly across the XCDs); with a
// single chunk the first kernel writes o itself (fp32, or as bf16 straight
// into the O projection's staged input).  Zero-filled rows of skipped
// steps are ordinary cache rows here (logit 0, value 0), unless the block's
// execution map is given: then rows at which the block did not run are left
// out of the softmax (the new row at pos always counts: the block runs for
// it, and the first block's entry is written only after its attention).
// In a decode step the router's block (the first, or the one before the
// start layer) reads exactly the rows the planner pools (Sec. 4.3: the mean
// of that block's K and V rows 0..pos), so its workgroups also write the
// column sums of their chunk's K and V rows in the pool's partial-sum
// layout, and the cache is not read a second time (the pooling variants).
//
// Two score kernels:
//  attn_kernel       vector ALUs: a cache row of hd elements is read by hd/V
//                    lanes with 16-byte loads (V = 8 bf16 or 4 fp32), so a
//                    wavefront covers 64/(hd/V) rows per pass and the row dot
//                    products finish with a short DPP / shuffle tree.  Used
//                    for fp32 caches, head_dim 64 and groups of one or two.
//  attn_mfma_kernel  bf16, head_dim 128, three to eight query heads per KV
//                    head: the scores of 16 rows against the group and the
//                    P V product of those rows are MFMA products.
// The prompt tokens of a prefill (bf16, head_dim 128) take a third kernel,
// attn_prefill_kernel, with both products on the MFMA (below).
#include "buddy_internal.h"

namespace buddy {

__device__ __forceinline__ float scale_of(float m, float mn) {
    return m == -INFINITY ? 0.f : exp2f(m - mn);
}

// Sum over the 16 lanes of a DPP row (lanes 16r .. 16r+15), left in every
// lane of the row: rotations by 8, 4, 2 and 1 within the row are plain VALU
// operations, much shorter than LDS-routed shuffles.
__device__ __forceinline__ float row_sum16(float v) {
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x122, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x121, 0xF, 0xF, false));
    return v;
}

// Sum over the lpr lanes that share a cache row.
template <int LPR>
__device__ __forceinline__ float lanes_sum(float v) {
    if (LPR == 16) return row_sum16(v);
#pragma unroll
    for (int o = LPR >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// Row passes of a workgroup block, all of whose loads are issued up front:
// four for up to four query heads per KV head, two for larger groups (their
// registers hold 8 query heads and accumulators).
__host__ __device__ constexpr int attn_passes(int G) { return G <= 4 ? 4 : 2; }

// Rows of one workgroup block: passes x 4 wavefronts x (64 / (hd / V)) rows.
template <typename T>
__host__ __device__ constexpr int attn_rows_per_wg(int hd, int G) {
    return attn_passes(G) * 4 * (kWave / (hd / St<T>::V));
}

// POOL: the workgroup also sums the chunk's K and V rows per column (the
// router's pooled context, written to a.pool_part; rows past pos excluded).
template <typename T, int GM, int LPR, bool POOL = false>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    constexpr int V = St<T>::V;
    constexpr int kAttnPasses = attn_passes(GM);
    __shared__ float s_acc[4][GM][128 + 2];
    __shared__ float s_pool[POOL ? 4 : 1][2][128];
    const int i = blockIdx.z;
    if (!a.rows.exact && i >= *a.rows.cnt) return;
    const int b = row_seq(a.rows, i);
    const int g = blockIdx.y, c = blockIdx.x;
    int slot, pos;
    slot_pos(b, a.tok_T, a.pos, a.pos_u, slot, pos);
    const int G = a.nq / a.nkv;
    constexpr int lpr = LPR;           // lanes per cache row (hd / V)
    constexpr int rpw = kWave / LPR;   // rows per wavefront pass
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane % lpr, sub = lane / lpr;
    const int j0 = c * a.chunk_len;
    const int j1 = min(j0 + a.chunk_len, pos + 1);

    const size_t base = ((size_t)slot * a.nkv + g) * a.T * a.hd + col * V;
    const T* Kb = (const T*)a.kc + base;
    const T* Vb = (const T*)a.vc + base;
    const int rows_wg = kAttnPasses * 4 * rpw;
    uint4 kr[kAttnPasses], vr[kAttnPasses];
    uint8_t er[kAttnPasses];
    const uint8_t* exr = a.exec ? a.exec + (size_t)slot * a.T : nullptr;
    // every K/V row of a block is loaded before any arithmetic on it; rows
    // past the end are clamped to a valid row and masked below.  A load
    // instruction covers whole consecutive rows, read once: nontemporal.
    typedef uint32_t nt_u4 __attribute__((ext_vector_type(4)));
    auto load_block = [&](int jb) {
#pragma unroll
        for (int p = 0; p < kAttnPasses; ++p) {
            const int j = min(jb + (p * 4 + wave) * rpw + sub, max(j1 - 1, 0));
            const nt_u4 k4 = __builtin_nontemporal_load(reinterpret_cast<const nt_u4*>(Kb + (size_t)j * a.hd));
            const nt_u4 v4 = __builtin_nontemporal_load(reinterpret_cast<const nt_u4*>(Vb + (size_t)j * a.hd));
            kr[p] = make_uint4(k4.x, k4.y, k4.z, k4.w);
            vr[p] = make_uint4(v4.x, v4.y, v4.z, v4.w);
            er[p] = exr ? exr[j] : 1;
        }
    };
    load_block(j0);

    // queries of the group, pre-scaled so that exp2 of the score is the
    // softmax weight: q * log2(e) / sqrt(hd)
    const float qs = 1.4426950408889634f / sqrtf((float)a.hd);
    float qr[GM][V];
    const float* qb = a.q + (size_t)b * a.nq * a.hd + (size_t)g * G * a.hd + col * V;
#pragma unroll
    for (int h = 0; h < GM; ++h) {
#pragma unroll
        for (int e = 0; e < V; ++e) qr[h][e] = 0.f;
        if (h < G) {
#pragma unroll
            for (int e = 0; e < V; ++e) qr[h][e] = qb[(size_t)h * a.hd + e] * qs;
        }
    }

    float m[GM], l[GM], acc[GM][V];
#pragma unroll
    for (int h = 0; h < GM; ++h) {
        m[h] = -INFINITY; l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) acc[h][e] = 0.f;
    }
    float pk[V], pv[V];   // POOL: this lane's column sums of its K and V rows
#pragma unroll
    for (int e = 0; e < V; ++e) pk[e] = pv[e] = 0.f;
    for (int jb = j0; jb < j1; jb += rows_wg) {
        if (jb != j0) load_block(jb);
        // all scores of the block first: the row reductions are independent
        float sc[kAttnPasses][GM];
#pragma unroll
        for (int p = 0; p < kAttnPasses; ++p) {
            float kf[V];
            unpack<T>(kr[p], kf);
            const int jrow = jb + (p * 4 + wave) * rpw + sub;
            if constexpr (POOL) {
                // rows past the chunk were clamped to a valid row: left out
                const float w = jrow < j1 ? 1.f : 0.f;
                float vv[V];
                unpack<T>(vr[p], vv);
#pragma unroll
                for (int e = 0; e < V; ++e) { pk[e] += w * kf[e]; pv[e] += w * vv[e]; }
            }
            const bool live = jrow < j1 && (er[p] != 0 || jrow == pos);
#pragma unroll
            for (int h = 0; h < GM; ++h) {
                float d = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) d += qr[h][e] * kf[e];
                d = lanes_sum<LPR>(d);
                sc[p][h] = live ? d : -INFINITY;
            }
        }
        // one online-softmax update per block and head, branch-free: a
        // padded head (h >= G) has q = 0 and is never written, and with every
        // score of the block masked mn stays -inf and scale_of gives 0
        float vf[kAttnPasses][V];
#pragma unroll
        for (int p = 0; p < kAttnPasses; ++p) unpack<T>(vr[p], vf[p]);
#pragma unroll
        for (int h = 0; h < GM; ++h) {
            float mx = sc[0][h];
#pragma unroll
            for (int p = 1; p < kAttnPasses; ++p) mx = fmaxf(mx, sc[p][h]);
            const float mn = fmaxf(m[h], mx);
            const float al = scale_of(m[h], mn);
            l[h] *= al;
#pragma unroll
            for (int e = 0; e < V; ++e) acc[h][e] *= al;
#pragma unroll
            for (int p = 0; p < kAttnPasses; ++p) {
                const float pw = scale_of(sc[p][h], mn);
                l[h] += pw;
#pragma unroll
                for (int e = 0; e < V; ++e) acc[h][e] += pw * vf[p][e];
            }
            m[h] = mn;
        }
    }

    // merge the row slots of the wavefront (lanes with equal col)
    for (int o = lpr; o < kWave; o <<= 1) {
#pragma unroll
        for (int h = 0; h < GM; ++h) {
            {
                const float mo = __shfl_xor(m[h], o, kWave);
                const float lo = __shfl_xor(l[h], o, kWave);
                const float mn = fmaxf(m[h], mo);
                const float s1 = scale_of(m[h], mn), s2 = scale_of(mo, mn);
                l[h] = l[h] * s1 + lo * s2;
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    const float ao = __shfl_xor(acc[h][e], o, kWave);
                    acc[h][e] = acc[h][e] * s1 + ao * s2;
                }
                m[h] = mn;
            }
        }
    }
    if (sub == 0) {
#pragma unroll
        for (int h = 0; h < GM; ++h) {
            if (h < G) {
#pragma unroll
                for (int e = 0; e < V; ++e) s_acc[wave][h][col * V + e] = acc[h][e];
                if (col == 0) {
                    s_acc[wave][h][a.hd] = m[h];
                    s_acc[wave][h][a.hd + 1] = l[h];
                }
            }
        }
    }
    if constexpr (POOL) {
        // the wavefront's row slots (lanes with equal col), then per wave
        for (int o = lpr; o < kWave; o <<= 1)
#pragma unroll
            for (int e = 0; e < V; ++e) {
                pk[e] += __shfl_xor(pk[e], o, kWave);
                pv[e] += __shfl_xor(pv[e], o, kWave);
            }
        if (sub == 0)
#pragma unroll
            for (int e = 0; e < V; ++e) {
                s_pool[wave][0][col * V + e] = pk[e];
                s_pool[wave][1][col * V + e] = pv[e];
            }
    }
    __syncthreads();
    if constexpr (POOL) {
        float* pp = a.pool_part + (((size_t)b * a.nkv + g) * a.pool_max_splits + c) * 2 * a.hd;
        for (int t = tid; t < 2 * a.hd; t += 256) {
            const int which = t / a.hd, e = t - which * a.hd;
            pp[t] = (s_pool[0][which][e] + s_pool[1][which][e]) + (s_pool[2][which][e] + s_pool[3][which][e]);
        }
    }

    // merge the four wavefronts and write this chunk's partial
    const size_t pstride = (size_t)a.hd + 2;
    for (int t = tid; t < G * a.hd; t += 256) {
        const int h = t / a.hd, e = t % a.hd;
        float M = -INFINITY;
        for (int w = 0; w < 4; ++w) M = fmaxf(M, s_acc[w][h][a.hd]);
        float L = 0.f, A = 0.f;
        for (int w = 0; w < 4; ++w) {
            const float sw = scale_of(s_acc[w][h][a.hd], M);
            L += s_acc[w][h][a.hd + 1] * sw;
            A += s_acc[w][h][e] * sw;
        }
        if (a.chunks == 1) {
            const int col = (g * G + h) * a.hd + e;
            if (a.xb_out) store_split(a.xb_out, xbs_index(i, col, a.nq * a.hd, 0), A / L);
            else a.o[(size_t)b * a.nq * a.hd + col] = A / L;
        } else {
            float* pp = a.part + (((size_t)b * a.nq + g * G + h) * a.max_chunks + c) * pstride;
            pp[e] = A;
            if (e == 0) { pp[a.hd] = M; pp[a.hd + 1] = L; }
        }
    }
}

// Decode attention on MFMA: bf16 cache, head_dim 128, three to kMaxGroup
// query heads per KV head.  Each wavefront takes 16-row slabs of the chunk
// (every fourth slab) and keeps an online softmax per head:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, A = the slab's K rows (loaded
//                 to registers one slab ahead), B = the group's queries as
//                 bf16 high + low parts (heads past G are zero), so scores
//                 keep about 16 bits of the fp32 query;
//                 D: lane h + 16 r holds rows 4 r .. 4 r + 3 of head h;
//   softmax       online per head (exp2 of prescaled scores);
//   O += P V      v_mfma_f32_16x16x16_bf16 with the softmax weights in place
//                 as the A operand, split into bf16 high + low parts (two
//                 products, so P keeps about 16 bits), and V[4 rows][col] as
//                 the B operand from ds_read_b64_tr_b16: the wavefront moves
//                 its slab of V global -> LDS directly (two buffers, the next
//                 slab's loads in flight), each 256-byte row's 16-byte chunks
//                 stored at chunk ^ (row % 16); O: lane c + 16 r holds heads
//                 4 r .. 4 r + 3 of column c of each 16-column tile.
// The four wavefronts' (max, sum, O) are merged through LDS at the end.
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4
//   x32 A[i][k]: lane i + 16 (k / 8), element k % 8;  B[k][j]: lane j + 16 (k / 8)
//   x16 A[i][k]: lane i + 16 (k / 4), element k % 4;  B[k][j]: lane j + 16 (k / 4)
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) const void* attn_gptr_t;
typedef __attribute__((address_space(3))) void* attn_lptr_t;

// Eight transposing 8-byte LDS reads at per-lane addresses plus one
// immediate (the V fragments of the 8 column tiles of a 16-row slab), then a
// wait; asm so that the compiler does not first wait for the direct-to-LDS
// loads in flight into the other buffer.
template <int OFF>
__device__ __forceinline__ void read_v_tr(const uint32_t* ad, uint32_t base, s16x4_t* x) {
    i32x2_t r[8];
    asm volatile(
        "ds_read_b64_tr_b16 %0, %8 offset:%16\n\t"
        "ds_read_b64_tr_b16 %1, %9 offset:%16\n\t"
        "ds_read_b64_tr_b16 %2, %10 offset:%16\n\t"
        "ds_read_b64_tr_b16 %3, %11 offset:%16\n\t"
        "ds_read_b64_tr_b16 %4, %12 offset:%16\n\t"
        "ds_read_b64_tr_b16 %5, %13 offset:%16\n\t"
        "ds_read_b64_tr_b16 %6, %14 offset:%16\n\t"
        "ds_read_b64_tr_b16 %7, %15 offset:%16\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]),
          "=&v"(r[6]), "=&v"(r[7])
        : "v"(ad[0] + base), "v"(ad[1] + base), "v"(ad[2] + base), "v"(ad[3] + base),
          "v"(ad[4] + base), "v"(ad[5] + base), "v"(ad[6] + base), "v"(ad[7] + base), "i"(OFF)
        : "memory");
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = __builtin_bit_cast(s16x4_t, r[i]);
}

// Max and sum of a value and its copy 16 (or 32) lanes away, by the gfx950
// lane swaps: with both operands the same register, v_permlane16_swap
// (v_permlane32_swap) leaves each lane's own value in one result and its
// partner's in the other, so their max or sum is the pair's -- the same
// operands as a cross-lane shuffle (so the same result bit for bit), without
// its round trip through the LDS unit.
__device__ __forceinline__ float max_xor16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// s_waitcnt with at most n vector-memory operations outstanding (the other
// counters left at their maxima).
__device__ __forceinline__ constexpr int vmcnt_at_most(int n) {
    return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);
}

// Three workgroups per CU: 138 registers (accumulators in VGPRs) and at most
// 49 KB of LDS each.
// Cache policy of a load: nontemporal (the NT bit of the instruction).  The
// slab's V rows arrive as whole 256-byte rows, 1 KB per instruction, and are
// read once: loading them nontemporal made the Llama-8B B = 32 launch 6 %
// faster; K, fetched 64 bytes of a row per instruction, stays cached (its
// nontemporal loads were slower).
constexpr int kCpolNontemporal = 2;

// POOL (no execution map): the workgroup also sums the chunk's K and V rows
// per column, the router's pooled context (a.pool_part).  The V sums come
// from the P V product itself: a query head past G has q = 0, so its scores
// are 0 and its softmax weights exactly 1 on every row of the chunk, and its
// row of O accumulates the plain sum of the V rows.  The K sums are vector
// adds of the K fragments already in registers.
// (The pooling variant runs only for the router's block, one launch per
// step; its 32 K sums per lane would spill within three waves' registers,
// so it takes two.)
template <int GM, bool MASKED, bool POOL = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(POOL ? 2 : 3))) void attn_mfma_kernel(AttnArgs a) {
    static_assert(!(POOL && MASKED), "the pooled sums take every row of the chunk");
    static_assert(GM < 16, "a padded query head carries the V sums");
    constexpr int HD = 128, KS = HD / 32;
    constexpr int kSlab = 16 * HD * 2;        // bytes of a 16-row V slab
    __shared__ __attribute__((aligned(16))) char s_v[4][2][kSlab];   // [wave][buffer]
    __shared__ float s_acc[4][GM][HD + 2];
    const int i = blockIdx.z;
    if (!a.rows.exact && i >= *a.rows.cnt) return;
    const int b = row_seq(a.rows, i);
    const int g = blockIdx.y, c = blockIdx.x;
    int slot, pos;
    slot_pos(b, a.tok_T, a.pos, a.pos_u, slot, pos);
    const int G = a.nq / a.nkv;
    const int tid = threadIdx.x, lane = tid & 63;
    const int li = lane & 15, lg = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j0 = c * a.chunk_len;
    const int j1 = min(j0 + a.chunk_len, pos + 1);
    const size_t base = ((size_t)slot * a.nkv + g) * a.T * HD;
    const bf16_t* Kb = (const bf16_t*)a.kc + base;
    const bf16_t* Vb = (const bf16_t*)a.vc + base;

    // B operand of the scores: queries of the group, scaled so that exp2 of
    // a score is the softmax weight, as bf16 high + low parts
    bf16x8_t qh[KS], ql[KS];
    {
        const float qs = 1.4426950408889634f / sqrtf((float)HD);
        const float* qp = a.q + ((size_t)b * a.nq + g * G + min(li, G - 1)) * HD + 8 * lg;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const float4 x0 = *reinterpret_cast<const float4*>(qp + 32 * s);
            const float4 x1 = *reinterpret_cast<const float4*>(qp + 32 * s + 4);
            const float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float v0 = li < G ? xv[e] * qs : 0.f, v1 = li < G ? xv[e + 1] * qs : 0.f;
                const uint32_t hp = pack_bf16x2(v0, v1);
                const float r0 = v0 - __uint_as_float(hp << 16), r1 = v1 - __uint_as_float(hp & 0xffff0000u);
                hi[e / 2] = hp;
                lo[e / 2] = pack_bf16x2(r0, r1);
            }
            qh[s] = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
            ql[s] = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
        }
    }

    // V addresses of ds_read_b64_tr_b16 in a slab (B operand: lane c + 16 r
    // holds V[4 r .. 4 r + 3][c]): source lane s = lane % 16 addresses row
    // 4 r + s / 4, columns 16 dt + 4 (s % 4) .. + 3, stored in chunk
    // (column / 8) ^ row
    const uint32_t lds_w = (uint32_t)(uintptr_t)(attn_lptr_t)&s_v[wave][0][0];
    uint32_t vad[8];
    {
        const int rr = 4 * lg + (li >> 2), cin = 4 * (li & 3);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const int col = 16 * dt + cin;
            vad[dt] = lds_w + rr * 256 + (((col >> 3) ^ rr) * 16) + (col & 7) * 2;
        }
    }

    float mrun = -INFINITY;     // running max of head li (same in its four lanes)
    float lrun = 0.f;           // running sum over this lane's rows of that head
    f32x4_t o[8];               // O[4 lg + e][16 dt + li]
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

    // a slab: its K fragments to registers (rows clamped to a valid row,
    // masked below), with a map its map entries, then its V rows global ->
    // LDS buffer `buf` (lane L of load ld lands at row 4 ld + L / 16, stored
    // chunk L % 16, which holds source chunk (L % 16) ^ row).  The next
    // slab's loads are issued once the current scores have used the K
    // registers.  Without a map the K loads are asm, outside the compiler's
    // load tracking, which with direct-to-LDS loads pending would wait for
    // every load before the scores; the waits below cover them (in this
    // issue order the scores need all but the slab's last 4 loads, its V,
    // done).  With a map, and in the pooling variant, every register load
    // is the compiler's, and so are their waits: the asm loads are sound
    // only while the compiler keeps their results in place until the wait,
    // and with the pooling variant's 32 more live registers it copied the
    // next slab's K registers at the loop's back edge, before the wait.
    bf16x8_t kf[KS];
    uint8_t en[4];
    // POOL: sums of this lane's K rows (row li of each slab), columns
    // 32 s + 8 lg + e
    float ks[KS][8];
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) ks[s][e] = 0.f;
    auto load_slab = [&](int jb, int buf) {
        const int jr = min(jb + li, j1 - 1);
        const bf16_t* kp = Kb + (size_t)jr * HD + 8 * lg;
        if constexpr (MASKED || POOL) {
#pragma unroll
            for (int s = 0; s < KS; ++s) kf[s] = *reinterpret_cast<const bf16x8_t*>(kp + 32 * s);
            if constexpr (MASKED) {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    en[v] = a.exec[(size_t)slot * a.T + min(jb + 4 * lg + v, j1 - 1)];
            }
        } else {
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                typedef uint32_t u4 __attribute__((ext_vector_type(4)));
                u4 r;
                asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(kp + 32 * s) : "memory");
                kf[s] = __builtin_bit_cast(bf16x8_t, r);
            }
        }
#pragma unroll
        for (int ld = 0; ld < 4; ++ld) {
            const int rl = 4 * ld + lg;
            const size_t src = (size_t)min(jb + rl, j1 - 1) * HD + ((li ^ rl) * 8);
            __builtin_amdgcn_global_load_lds((attn_gptr_t)(Vb + src),
                                             (attn_lptr_t)(&s_v[wave][buf][ld * 1024]), 16, 0,
                                             kCpolNontemporal);
        }
    };
    int buf = 0;
    if (j0 + 16 * wave < j1) load_slab(j0 + 16 * wave, 0);
    for (int jb = j0 + 16 * wave; jb < j1; jb += 64, buf ^= 1) {
        __builtin_amdgcn_s_waitcnt(vmcnt_at_most(4));
        __builtin_amdgcn_sched_barrier(0);   // nothing reads K before the wait
        uint8_t ex[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) ex[v] = MASKED ? en[v] : 1;
        f32x4_t d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], qh[s], d, 0, 0, 0);
            d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], ql[s], d, 0, 0, 0);
        }
        if constexpr (POOL) {
            // row jb + li (clamped past the chunk's end: left out)
            const uint32_t keep = jb + li < j1 ? ~0u : 0u;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const uint4 w = __builtin_bit_cast(uint4, kf[s]);
                const uint32_t x[4] = {w.x & keep, w.y & keep, w.z & keep, w.w & keep};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    ks[s][2 * e] += __uint_as_float(x[e] << 16);
                    ks[s][2 * e + 1] += __uint_as_float(x[e] & 0xffff0000u);
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);   // the K registers are free only now
        const bool more = jb + 64 < j1;
        if (more) load_slab(jb + 64, buf ^ 1);
        // rows of this lane: jb + 4 lg + v; head li
        float sc[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int jrow = jb + 4 * lg + v;
            sc[v] = jrow < j1 && (ex[v] != 0 || jrow == pos) ? d[v] : -INFINITY;
        }
        float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
        mx = max_xor32(max_xor16(mx));
        const float mn = fmaxf(mrun, mx);
        const float al = scale_of(mrun, mn);
        float p[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) p[v] = scale_of(sc[v], mn);
        lrun = lrun * al + ((p[0] + p[1]) + (p[2] + p[3]));
        mrun = mn;
        // A operand (head li, rows 4 lg .. 4 lg + 3) as bf16 high + low parts
        const uint32_t h01 = pack_bf16x2(p[0], p[1]), h23 = pack_bf16x2(p[2], p[3]);
        const s16x4_t ph = __builtin_bit_cast(s16x4_t, make_uint2(h01, h23));
        const s16x4_t pl = __builtin_bit_cast(s16x4_t, make_uint2(
            pack_bf16x2(p[0] - __uint_as_float(h01 << 16), p[1] - __uint_as_float(h01 & 0xffff0000u)),
            pack_bf16x2(p[2] - __uint_as_float(h23 << 16), p[3] - __uint_as_float(h23 & 0xffff0000u))));
        // rescale O (lane c + 16 r holds heads 4 r .. 4 r + 3) unless no
        // head's running max moved; a multiply by 1 would change nothing
        if (__any(al != 1.f)) {
            float ar[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) ar[e] = __shfl(al, 4 * lg + e, kWave);
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
#pragma unroll
                for (int e = 0; e < 4; ++e) o[dt][e] *= ar[e];
        }
        // this slab's V is in LDS once its four loads are done (the next
        // slab's K and V loads, 8, and with a map its 4 map loads, may still
        // be in flight)
        if (more) __builtin_amdgcn_s_waitcnt(vmcnt_at_most(8));
        else __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));
        s16x4_t vf[8];
        if (buf == 0) read_v_tr<0>(vad, 0, vf);
        else read_v_tr<kSlab>(vad, 0, vf);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ph, vf[dt], o[dt], 0, 0, 0);
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl, vf[dt], o[dt], 0, 0, 0);
        }
    }

    // per wave: total of each head's running sum over its four lanes
    lrun = sum_xor32(sum_xor16(lrun));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int hh = 4 * lg + e;
        if (hh < GM) {
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) s_acc[wave][hh][16 * dt + li] = o[dt][e];
        }
    }
    if (lane < GM) {
        s_acc[wave][lane][HD] = mrun;
        s_acc[wave][lane][HD + 1] = lrun;
    }
    // POOL: the wave's K sums (over the 16 lanes of a row group) and V sums
    // (O's row of head G) in its own V buffers, idle now: its last slab's
    // loads and LDS reads are done
    float* s_pool = reinterpret_cast<float*>(&s_v[wave][0][0]);
    if constexpr (POOL) {
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int e = 0; e < 8; ++e) ks[s][e] = row_sum16(ks[s][e]);
        if (li == 0)
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int e = 0; e < 8; ++e) s_pool[32 * s + 8 * lg + e] = ks[s][e];
        if (lg == (G >> 2)) {
            const int eg = G & 3;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                s_pool[HD + 16 * dt + li] = eg == 0 ? o[dt][0] : eg == 1 ? o[dt][1] : eg == 2 ? o[dt][2] : o[dt][3];
        }
    }
    __syncthreads();
    if constexpr (POOL) {
        float* pp = a.pool_part + (((size_t)b * a.nkv + g) * a.pool_max_splits + c) * 2 * HD;
        const float* p0 = reinterpret_cast<const float*>(&s_v[0][0][0]);
        const float* p1 = reinterpret_cast<const float*>(&s_v[1][0][0]);
        const float* p2 = reinterpret_cast<const float*>(&s_v[2][0][0]);
        const float* p3 = reinterpret_cast<const float*>(&s_v[3][0][0]);
        pp[tid] = (p0[tid] + p1[tid]) + (p2[tid] + p3[tid]);   // 256 threads = 2 HD sums
    }

    // merge the four wavefronts and write this chunk's partial
    const size_t pstride = (size_t)HD + 2;
    for (int t = tid; t < G * HD; t += 256) {
        const int h = t / HD, e = t % HD;
        float M = -INFINITY;
        for (int w = 0; w < 4; ++w) M = fmaxf(M, s_acc[w][h][HD]);
        float L = 0.f, A = 0.f;
        for (int w = 0; w < 4; ++w) {
            const float sw = scale_of(s_acc[w][h][HD], M);
            L += s_acc[w][h][HD + 1] * sw;
            A += s_acc[w][h][e] * sw;
        }
        if (a.chunks == 1) {
            const int col = (g * G + h) * HD + e;
            if (a.xb_out) store_split(a.xb_out, xbs_index(i, col, a.nq * HD, 0), A / L);
            else a.o[(size_t)b * a.nq * HD + col] = A / L;
        } else {
            float* pp = a.part + (((size_t)b * a.nq + g * G + h) * a.max_chunks + c) * pstride;
            pp[e] = A;
            if (e == 0) { pp[HD] = M; pp[HD + 1] = L; }
        }
    }
}

// ------------------------------------------------------ prefill attention

// Causal attention of the prompt tokens of a prefill (bf16 cache, head_dim
// 128): one workgroup per (KV head, group of up to 128 / G consecutive
// tokens of one prompt); its 128 query rows are (token, head) pairs, 16 per
// wavefront, eight wavefronts sharing every K/V tile.  K and V tiles of 64
// rows pass through LDS (four buffers, the next three tiles' direct-to-LDS
// loads in flight while the current one is used; one workgroup per CU),
// each row's 16-byte chunks stored at chunk ^ (row % 16) so that both reads
// below are free of bank conflicts.  Per tile and wavefront:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, A = K rows from LDS, B = the
//                 queries (held as bf16 high and low parts, as in the decode
//                 kernel); D: lane q + 16 r holds rows 4 r .. 4 r + 3 of q;
//   softmax       online per query row (exp2 of prescaled scores), causal
//                 through each row's own position;
//   O += P V      v_mfma_f32_16x16x16_bf16: the A operand (4 consecutive
//                 rows per lane) is the softmax of S^T in place, the B
//                 operand V[4 rows][d] comes from ds_read_b64_tr_b16, whose
//                 16-lane groups return element l % 4 of the 8-byte block
//                 addressed by lane l / 4 + 4 e (checked on the device).

constexpr int kPfRows = 64;                      // K/V rows per tile
constexpr int kPfTile = kPfRows * 128 * 2;       // bytes of a K or V tile
constexpr int kPfWaves = 8;                      // wavefronts (16 query rows each)
constexpr int kPfBufs = 4;                       // tiles in LDS: three loading ahead

// Four 16-byte LDS reads at per-lane addresses plus one immediate, then a
// wait; asm so that the compiler does not wait for the direct-to-LDS loads
// into the other buffer first.
template <int OFF>
__device__ __forceinline__ void pf_read_k(const uint32_t* ad, uint32_t base, bf16x8_t* x) {
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    u4 r0, r1, r2, r3;
    asm volatile(
        "ds_read_b128 %0, %4 offset:%8\n\t"
        "ds_read_b128 %1, %5 offset:%8\n\t"
        "ds_read_b128 %2, %6 offset:%8\n\t"
        "ds_read_b128 %3, %7 offset:%8\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r0), "=&v"(r1), "=&v"(r2), "=&v"(r3)
        : "v"(ad[0] + base), "v"(ad[1] + base), "v"(ad[2] + base), "v"(ad[3] + base), "i"(OFF)
        : "memory");
    x[0] = __builtin_bit_cast(bf16x8_t, r0);
    x[1] = __builtin_bit_cast(bf16x8_t, r1);
    x[2] = __builtin_bit_cast(bf16x8_t, r2);
    x[3] = __builtin_bit_cast(bf16x8_t, r3);
}
__global__ __launch_bounds__(64 * kPfWaves) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_prefill_kernel(AttnArgs a) {
    constexpr int HD = 128;
    __shared__ __attribute__((aligned(16))) char s_kv[kPfBufs][2][kPfTile];   // [buffer][K | V]
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = blockIdx.y;
    const int gi = a.n_groups - 1 - blockIdx.z;            // the longest groups first
    const int first = a.groups[2 * gi], count = a.groups[2 * gi + 1];
    const int G = a.nq / a.nkv;
    int slot, pos0;
    slot_pos(row_seq(a.rows, first), a.tok_T, a.pos, a.pos_u, slot, pos0);
    const int pos_last = pos0 + count - 1;
    const int ntiles = pos_last / kPfRows + 1;

    // this lane's query row (S^T column, softmax row): 16 wave + lane % 16
    const int qr = 16 * wave + (lane & 15);
    const int qt = qr / G, hq = qr - qt * G;
    const bool q_ok = qt < count;
    const int q_pos = pos0 + qt;
    bf16x8_t qh[4], ql[4];
    {
        const int bq = row_seq(a.rows, first + min(qt, count - 1));
        const float qs = 1.4426950408889634f / sqrtf((float)HD);
        const float* qp = a.q + ((size_t)bq * a.nq + g * G + hq) * HD + 8 * (lane >> 4);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const float4 x0 = *reinterpret_cast<const float4*>(qp + 32 * s);
            const float4 x1 = *reinterpret_cast<const float4*>(qp + 32 * s + 4);
            const float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const float v0 = q_ok ? xv[e] * qs : 0.f, v1 = q_ok ? xv[e + 1] * qs : 0.f;
                const uint32_t hp = pack_bf16x2(v0, v1);
                const float r0 = v0 - __uint_as_float(hp << 16), r1 = v1 - __uint_as_float(hp & 0xffff0000u);
                hi[e / 2] = hp;
                lo[e / 2] = pack_bf16x2(r0, r1);
            }
            qh[s] = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
            ql[s] = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
        }
    }

    // Tile loads: wavefront w moves rows 8 w .. 8 w + 7 of K and of V, four
    // rows (1 KB) per load; lane L lands at 16 L of the load's block, i.e. row
    // L / 16 of it and stored chunk L % 16, which holds source chunk
    // (L % 16) ^ (row % 16).  Rows past the last position repeat it (masked).
    const size_t cbase = ((size_t)slot * a.nkv + g) * a.T * HD;
    const bf16_t* Kg = (const bf16_t*)a.kc + cbase;
    const bf16_t* Vg = (const bf16_t*)a.vc + cbase;
    constexpr int kWaveRows = kPfRows / kPfWaves;                   // 8 rows of each
    auto issue = [&](int kt, int buf) {
#pragma unroll
        for (int ld = 0; ld < kWaveRows / 4; ++ld) {
            const int rl = kWaveRows * wave + 4 * ld + (lane >> 4);   // row within the tile
            const int row = min(kt * kPfRows + rl, pos_last);
            const size_t src = (size_t)row * HD + (((lane & 15) ^ (rl & 15)) * 8);
            const int dst = (kWaveRows * wave + 4 * ld) * 256;
            __builtin_amdgcn_global_load_lds((attn_gptr_t)(Kg + src), (attn_lptr_t)(s_kv[buf][0] + dst),
                                             16, 0, 0);
            __builtin_amdgcn_global_load_lds((attn_gptr_t)(Vg + src), (attn_lptr_t)(s_kv[buf][1] + dst),
                                             16, 0, 0);
        }
    };

    // K fragment addresses (A operand: lane i + 16 dg holds row 16 t + i,
    // d = 32 s + 8 dg .. + 7): stored chunk (4 s + dg) ^ i; the tile t of 16
    // rows is an immediate 4 KB t.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(attn_lptr_t)&s_kv[0][0][0];
    const int li = lane & 15, lg = lane >> 4;
    uint32_t kad[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) kad[s] = lds0 + li * 256 + (((4 * s + lg) ^ li) * 16);
    // V addresses for ds_read_b64_tr_b16 (B operand: lane d + 16 r holds
    // V[4 r .. 4 r + 3][d] of a 16-row tile): source lane s = lane % 16
    // addresses row 4 r + s / 4, columns 16 dt + 4 (s % 4) .. + 3.
    uint32_t vad[8];
    {
        const int rr = 4 * lg + (li >> 2);                          // row within a 16-row tile
        const int cin = 4 * (li & 3);                                // column within the 16-column tile
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
            const int col = 16 * dt + cin;
            vad[dt] = lds0 + kPfTile + rr * 256 + (((col >> 3) ^ rr) * 16) + (col & 7) * 2;
        }
    }

    float m_run = -INFINITY, l_run = 0.f;                           // query row lane % 16
    f32x4_t o[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

    // Tile kt sits in buffer kt % 4, its loads issued three tiles ahead: at
    // tile kt, wait until only the loads of the tiles after it that have been
    // issued (kt + 1 and kt + 2, those that exist; kWaveRows / 2 loads each)
    // are in flight, barrier (everyone's loads of tile kt have landed, and
    // everyone has read tile kt - 1's buffer), refill that buffer with tile
    // kt + 3.
    constexpr int kTileLoads = kWaveRows / 2;                      // K and V loads per wavefront
    for (int j = 0; j < kPfBufs - 1 && j < ntiles; ++j) issue(j, j);
    for (int kt = 0; kt < ntiles; ++kt) {
        const int buf = kt % kPfBufs;
        const int later = min(ntiles - 1, kt + kPfBufs - 2) - kt;      // tiles issued after kt
        if (later >= 2) __builtin_amdgcn_s_waitcnt(vmcnt_at_most(2 * kTileLoads));
        else if (later == 1) __builtin_amdgcn_s_waitcnt(vmcnt_at_most(kTileLoads));
        else __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));
        asm volatile("s_barrier" ::: "memory");
        if (kt + kPfBufs - 1 < ntiles) issue(kt + kPfBufs - 1, (kt + kPfBufs - 1) % kPfBufs);
        const uint32_t bb = buf * 2 * kPfTile;

        // S^T for the 4 row tiles of the K tile
        f32x4_t st[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            bf16x8_t kf[4];
            switch (t) {
                case 0: pf_read_k<0>(kad, bb, kf); break;
                case 1: pf_read_k<4096>(kad, bb, kf); break;
                case 2: pf_read_k<8192>(kad, bb, kf); break;
                default: pf_read_k<12288>(kad, bb, kf); break;
            }
            f32x4_t d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], qh[s], d, 0, 0, 0);
                d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], ql[s], d, 0, 0, 0);
            }
            st[t] = d;
        }
        // causal mask and online softmax of query row lane % 16
        const int r0 = kt * kPfRows + 4 * lg;
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = r0 + 16 * t + e;
                st[t][e] = q_ok && row <= q_pos ? st[t][e] : -INFINITY;
                mx = fmaxf(mx, st[t][e]);
            }
        mx = max_xor32(max_xor16(mx));
        const float mn = fmaxf(m_run, mx);
        const float al = scale_of(m_run, mn);
        float ls = 0.f;
        s16x4_t pa[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            float p[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                p[e] = scale_of(st[t][e], mn);
                ls += p[e];
            }
            pa[t] = __builtin_bit_cast(s16x4_t, make_uint2(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])));
        }
        ls = sum_xor32(sum_xor16(ls));
        l_run = l_run * al + ls;
        m_run = mn;
        // rescale O: lane d + 16 r holds query rows 4 r .. 4 r + 3
        float ar[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) ar[e] = __shfl(al, 4 * lg + e, kWave);
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
#pragma unroll
            for (int e = 0; e < 4; ++e) o[dt][e] *= ar[e];
        // O += P V, 16 rows at a time
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            s16x4_t vf[8];
            switch (t) {
                case 0: read_v_tr<0>(vad, bb, vf); break;
                case 1: read_v_tr<4096>(vad, bb, vf); break;
                case 2: read_v_tr<8192>(vad, bb, vf); break;
                default: read_v_tr<12288>(vad, bb, vf); break;
            }
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa[t], vf[dt], o[dt], 0, 0, 0);
        }
    }

    // O / l, query rows 4 r + e of this lane
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float le = __shfl(l_run, 4 * lg + e, kWave);
        const int r = 16 * wave + 4 * lg + e;
        const int t = r / G, h = r - t * G;
        if (t >= count) continue;
        const float inv = 1.f / le;
        if (a.xb_out) {   // bf16, straight into the O projection's staging
            const int k0 = (g * G + h) * HD + li;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt)
                a.xb_out[xb_index(first + t, k0 + 16 * dt, a.nq * HD)] = f2bf(o[dt][e] * inv);
        } else {
            float* op = a.o + ((size_t)row_seq(a.rows, first + t) * a.nq + g * G + h) * HD + li;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) op[16 * dt] = o[dt][e] * inv;
        }
    }
}


// Merge of the chunk partials of one (routed sequence, query head): the
// chunk maxima and sums go through LDS once, then every thread folds one
// output element over the chunks in chunk order with coalesced reads.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
    __shared__ float s_w[kAttnMaxChunks];
    __shared__ float s_red[4];
    const int i = blockIdx.y;
    if (!a.rows.exact && i >= *a.rows.cnt) return;
    const int b = row_seq(a.rows, i);
    const int head = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t pstride = (size_t)a.hd + 2;
    const float* pp = a.part + ((size_t)b * a.nq + head) * a.max_chunks * pstride;
    // each chunk's max and sum, both loaded before the first reduction
    const float mc = tid < a.chunks ? pp[tid * pstride + a.hd] : -INFINITY;
    const float lc = tid < a.chunks ? pp[tid * pstride + a.hd + 1] : 0.f;
    float M = wave_max(mc);
    if (lane == 0) s_red[wave] = M;
    __syncthreads();
    M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
    const float wc = scale_of(mc, M);
    if (tid < a.chunks) s_w[tid] = wc;
    float L = tid < a.chunks ? lc * wc : 0.f;
    L = wave_sum(L);
    __syncthreads();                      // s_red reads above are done
    if (lane == 0) s_red[wave] = L;
    __syncthreads();
    L = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
    for (int e = tid; e < a.hd; e += 256) {
        float A = 0.f;
#pragma unroll 8
        for (int q = 0; q < a.chunks; ++q) A += pp[q * pstride + e] * s_w[q];
        const int col = head * a.hd + e;
        if (a.xb_out) store_split(a.xb_out, xbs_index(i, col, a.nq * a.hd, 0), A / L);
        else a.o[(size_t)b * a.nq * a.hd + col] = A / L;
    }
}

static bool attn_uses_mfma(int dtype, int hd, int G) { return dtype == BUDDY_BF16 && hd == 128 && G >= 3 && G <= kMaxGroup; }

int attention_prefill_group(int dtype, int hd, int G) {
    return dtype == BUDDY_BF16 && hd == 128 && G <= kMaxGroup ? 16 * kPfWaves / G : 1;
}

int attention_rows_per_wg(int dtype, int hd, int G) {
    if (attn_uses_mfma(dtype, hd, G)) return 64;
    // G rounded up to the register class the launcher picks
    const int gm = G <= 1 ? 1 : G <= 2 ? 2 : G <= 4 ? 4 : 8;
    return dtype == BUDDY_BF16 ? attn_rows_per_wg<bf16_t>(hd, gm) : attn_rows_per_wg<float>(hd, gm);
}

// The vector score kernel for a cache dtype, head_dim and group size.
template <bool POOL>
static void launch_vector_attention(int dtype, int G, dim3 grid, const AttnArgs& a, hipStream_t s) {
    if (dtype == BUDDY_BF16) {
        if (a.hd == 128) {
            if (G == 1) launch_main(attn_kernel<bf16_t, 1, 16, POOL>, grid, dim3(256), 0, s, a);
            else launch_main(attn_kernel<bf16_t, 2, 16, POOL>, grid, dim3(256), 0, s, a);
        } else {
            if (G <= 2) launch_main(attn_kernel<bf16_t, 2, 8, POOL>, grid, dim3(256), 0, s, a);
            else launch_main(attn_kernel<bf16_t, 8, 8, POOL>, grid, dim3(256), 0, s, a);
        }
    } else {
        if (a.hd == 128) {
            if (G <= 2) launch_main(attn_kernel<float, 2, 32, POOL>, grid, dim3(256), 0, s, a);
            else launch_main(attn_kernel<float, 8, 32, POOL>, grid, dim3(256), 0, s, a);
        } else {
            if (G <= 2) launch_main(attn_kernel<float, 2, 16, POOL>, grid, dim3(256), 0, s, a);
            else launch_main(attn_kernel<float, 8, 16, POOL>, grid, dim3(256), 0, s, a);
        }
    }
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
    dim3 grid(a.chunks, a.nkv, a.rows.n_max);
    const int G = a.nq / a.nkv;   // query heads per KV head, held in registers
    // lanes per cache row: hd / 8 (bf16) or hd / 4 (fp32); head_dim is 64 or 128
    if (a.groups) {               // prompt-token groups (one chunk)
        if (attention_prefill_group(dtype, a.hd, G) < 2 || a.chunks != 1) return hipErrorInvalidValue;
        launch_main(attn_prefill_kernel, dim3(1, a.nkv, a.n_groups), dim3(64 * kPfWaves), 0, s, a);
        return hipGetLastError();
    }
    if (a.pool_part && (a.exec || a.tok_T > 0)) return hipErrorInvalidValue;
    if (attn_uses_mfma(dtype, a.hd, G)) {
        if (a.pool_part) {
            if (G <= 4) launch_main(attn_mfma_kernel<4, false, true>, grid, dim3(256), 0, s, a);
            else launch_main(attn_mfma_kernel<kMaxGroup, false, true>, grid, dim3(256), 0, s, a);
        } else if (a.exec) {
            if (G <= 4) launch_main(attn_mfma_kernel<4, true>, grid, dim3(256), 0, s, a);
            else launch_main(attn_mfma_kernel<kMaxGroup, true>, grid, dim3(256), 0, s, a);
        } else {
            if (G <= 4) launch_main(attn_mfma_kernel<4, false>, grid, dim3(256), 0, s, a);
            else launch_main(attn_mfma_kernel<kMaxGroup, false>, grid, dim3(256), 0, s, a);
        }
    } else if (a.pool_part) {
        launch_vector_attention<true>(dtype, G, grid, a, s);
    } else {
        launch_vector_attention<false>(dtype, G, grid, a, s);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.chunks == 1) return hipSuccess;   // the score kernel wrote o
    LaunchEvents& ev = tl_merge_events;
    if (ev.start) {
        hipExtLaunchKernelGGL(attn_combine_kernel, dim3(a.nq, a.rows.n_max), dim3(256), 0, s,
                              ev.start, ev.stop, 0, a);
        ev.start = ev.stop = nullptr;
    } else {
        attn_combine_kernel<<<dim3(a.nq, a.rows.n_max), 256, 0, s>>>(a);
    }
    return hipGetLastError();
}

}  // namespace buddy
