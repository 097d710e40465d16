// MFMA path of the routed projections (gfx950, bf16 weights), used for
// batches of more than four sequences: the projection is then a real dense
// contraction over the routed rows.
//
//  prep_kernel  writes the routed rows in MFMA operand order (row i of the
//               launch is sequence idx[i]) as bf16 high and low parts
//               (xbs_index): RMSNorm and gain folded in (PRO_RMSNORM), the
//               router context built from the pool's split sums (PRO_POOL), or
//               a plain conversion (PRO_NONE).  Inputs staged by their
//               producer (PRO_STAGED: the attention output, the SwiGLU output)
//               skip it.
//  mfma_kernel  Y = W XB^T with v_mfma_f32_16x16x32_bf16 (fp32 accumulate),
//               each activation fragment as its high part times W plus its
//               low part times W, so the fp32 activations enter with about 16
//               significant bits instead of bf16's 8.
//               A workgroup owns RT 16-row weight tiles (16 RT rows, or 8 RT
//               two-row units) and all routed rows; its four wavefronts take
//               a quarter of K each (of the workgroup's K range when K is
//               split over gridDim.y workgroups), their sums are reduced
//               through LDS one epilogue group at a time, and the fused
//               epilogues of the GEMV path run on the finished sums, or the
//               sums go to a partial buffer when K is split.
//  split_add_kernel  adds the K-split partial sums in split order to the
//               residual rows.
//
// Operand layouts of v_mfma_f32_16x16x32_bf16 (checked on the device):
//   A[i][k] (16 x 32): lane i + 16 (k / 8), element k % 8
//   B[k][j] (32 x 16): lane j + 16 (k / 8), element k % 8
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4
// One 16-byte load per lane fetches an A tile segment from the row-major
// weights (16 rows x 64 bytes).  The activations are small and re-read by
// every workgroup, so they are stored in B-operand order: the B tiles of
// column tile c and k-step s are 2 KB at ((c * K/32 + s) * 128 + lane) * 8
// elements, the high part's 1 KB then the low part's, one contiguous load
// per wavefront each.
#include <atomic>

#include "buddy_internal.h"
#include "epilogue.h"

namespace buddy {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kMfmaMaxTiles = 8;   // 16-row column tiles of routed rows per pass


// ----------------------------------------------------------------- prep

// Threads of a staging workgroup (one routed row): 512, so that a 4096-wide
// row takes one pass of 8 elements per thread, its loads (the row and any
// split sums) all in flight at once.
constexpr int kPrepThreads = 512;

template <int PRO>
__global__ __launch_bounds__(kPrepThreads) void prep_kernel(GemvArgs g, int n_host) {
    __shared__ float s_ss[kPrepThreads / 64];
    const int i = blockIdx.x;
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    if (i >= n) return;
    const int b = row_seq(g.rows, i);
    const int K = g.K, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float inv = 1.f;
    if (PRO == PRO_RMSNORM) {
        // each thread owns the same 8-element groups here and in the staging
        // below, so it reads back its own residual writes
        float* x = const_cast<float*>(g.X) + (size_t)b * g.ldx;   // written only with split sums
        // split sums to add: the preceding projection's of this block (by
        // launch row), or the down projection's of the last routable block
        // this sequence ran (deferred)
        const float* ap = g.addpart;
        int an = g.addpart_splits, acap = g.addpart_cap, arow = i;
        if (g.dpart) {
            int last = -1;
            for (int q = g.d_upto - 1; q >= 0; --q)
                if (g.dmask[(size_t)b * g.dLm + q]) { last = q; break; }
            if (last >= 0) {
                ap = g.dpart + (size_t)last * g.dpart_block;
                an = g.dpart_splits; acap = g.dpart_cap;
                arow = g.dinv[(size_t)last * g.dpart_cap + b];
            }
        }
        float ss = 0.f;
        for (int k = tid * 8; k < K; k += kPrepThreads * 8) {
            float4 v0 = *reinterpret_cast<const float4*>(x + k);
            float4 v1 = *reinterpret_cast<const float4*>(x + k + 4);
            if (ap) {
                // K-split sums in split order, then the residual add (as the
                // split-add kernel does it)
                float4 a0 = make_float4(0.f, 0.f, 0.f, 0.f), a1 = a0;
                for (int q = 0; q < an; ++q) {
                    const float* pp = ap + ((size_t)q * acap + arow) * K + k;
                    const float4 t0 = *reinterpret_cast<const float4*>(pp);
                    const float4 t1 = *reinterpret_cast<const float4*>(pp + 4);
                    a0.x += t0.x; a0.y += t0.y; a0.z += t0.z; a0.w += t0.w;
                    a1.x += t1.x; a1.y += t1.y; a1.z += t1.z; a1.w += t1.w;
                }
                v0.x += a0.x; v0.y += a0.y; v0.z += a0.z; v0.w += a0.w;
                v1.x += a1.x; v1.y += a1.y; v1.z += a1.z; v1.w += a1.w;
                *reinterpret_cast<float4*>(x + k) = v0;
                *reinterpret_cast<float4*>(x + k + 4) = v1;
            }
            ss += v0.x * v0.x + v0.y * v0.y + v0.z * v0.z + v0.w * v0.w;
            ss += v1.x * v1.x + v1.y * v1.y + v1.z * v1.z + v1.w * v1.w;
        }
        ss = wave_sum(ss);
        if (lane == 0) s_ss[wave] = ss;
        __syncthreads();
        const float ss_all = ((s_ss[0] + s_ss[1]) + (s_ss[2] + s_ss[3])) +
                             ((s_ss[4] + s_ss[5]) + (s_ss[6] + s_ss[7]));
        inv = 1.0f / sqrtf(ss_all / (float)K + g.eps);
    }
    const float inv_n = PRO == PRO_POOL ? 1.0f / (float)(seq_pos(g.pos, g.pos_u, b) + 1) : 0.f;
    const int zdim = pooled_dim(g.ctx, g.nkv, g.hd);
    for (int k = tid * 8; k < K; k += kPrepThreads * 8) {
        float v[8];
        if (PRO == PRO_POOL && k < zdim) {
            const float4 t0 = pooled_feature4(g, b, k, inv_n), t1 = pooled_feature4(g, b, k + 4, inv_n);
            v[0] = t0.x; v[1] = t0.y; v[2] = t0.z; v[3] = t0.w;
            v[4] = t1.x; v[5] = t1.y; v[6] = t1.z; v[7] = t1.w;
        } else {
            const float* x = PRO == PRO_POOL ? g.h + (size_t)b * g.d + (k - zdim)
                                             : g.X + (size_t)b * g.ldx + k;
            const float4 t0 = *reinterpret_cast<const float4*>(x);
            const float4 t1 = *reinterpret_cast<const float4*>(x + 4);
            v[0] = t0.x; v[1] = t0.y; v[2] = t0.z; v[3] = t0.w;
            v[4] = t1.x; v[5] = t1.y; v[6] = t1.z; v[7] = t1.w;
        }
        if (PRO == PRO_RMSNORM) {
            float gv[8];
            St<bf16_t>::vec((const bf16_t*)g.gain + k, gv);
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] *= inv * gv[q];
        }
        // high parts, then the low parts from the exact remainders
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            hi[q] = pack_bf16x2(v[2 * q], v[2 * q + 1]);
            lo[q] = pack_bf16x2(split_rest(v[2 * q], hi[q] & 0xffffu),
                                split_rest(v[2 * q + 1], hi[q] >> 16));
        }
        const size_t at = xbs_index(i, k, K, 0);
        *reinterpret_cast<uint4*>(g.XB + at) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        *reinterpret_cast<uint4*>(g.XB + at + 512) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    }
}

// ----------------------------------------------------------------- MFMA

// Partial sums of K split `ks`, weight tile t of a unit (0, or 1 for the
// second row of the two-row kinds), unit u, routed row j: index
// ((ks GT + t) units + u) n_cap + j, n_cap = the launch's row capacity.
__device__ __forceinline__ size_t part_index(int ks, int GT, int t, int units, int u, int n_cap, int j) {
    return ((size_t)(ks * GT + t) * units + u) * n_cap + j;
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const void* mfma_gptr_t;
typedef __attribute__((address_space(3))) void* mfma_lptr_t;

// s_waitcnt with at most n vector-memory operations outstanding
__device__ __forceinline__ constexpr int mfma_vmcnt(int n) {
    return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8);
}

// Bytes of LDS: the weight rounds (4 wavefronts x 2 buffers x RT tiles x 16
// rows x 64 KR bytes), reused for the K-slice reduction afterwards.
__host__ __device__ constexpr int mfma_lds_bytes(int rt, int nt, int gt, int kr = 2) {
    return 4 * 2 * rt * 1024 * kr > 4 * gt * 16 * nt * 16 * 4 ? 4 * 2 * rt * 1024 * kr
                                                               : 4 * gt * 16 * nt * 16 * 4;
}

// Weight stream: a round is KR k-steps, 64 KR bytes of each of the
// wavefront's 16 RT rows (KR = 2: one cache line of each row; KR = 4: two,
// which the small grids stream markedly faster -- the longer run of each
// row per round suits the DRAM pages better).  The rows move global -> LDS
// directly with 1 KB loads of whole lines (1024 / (64 KR) rows each),
// nontemporal (read once per launch), into one of two buffers while the
// other is used; each row's 16-byte chunk c is stored at c ^ (row % (4 KR)),
// so that the fragment reads (16 rows, one chunk each) spread over the banks.
// The activation fragments of a round (1 KB contiguous each) are asm
// register loads issued at the round's start, outside the compiler's load
// tracking: the waits are explicit (the round's weights, issued a round
// earlier, and activations are in once no more than the next round's RT KR
// weight loads are pending).  The k-steps enter the accumulators in the
// same order for either round length, so the sums are identical bit for bit.
// KR = 4 needs a multiple of four k-steps per wavefront (no partial round).
template <int EPI, int NT, int RT, int KR = 2>
__global__ __launch_bounds__(256) void mfma_kernel(GemvArgs g, int units, int n_host, float* part,
                                                   int fold) {
    static_assert(KR == 2 || KR == 4, "rounds of two or four k-steps");
    constexpr bool kPaired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    constexpr int GT = kPaired ? 2 : 1;       // weight tiles per epilogue group
    constexpr int NG = RT / GT;               // epilogue groups (16 units or rows each)
    constexpr int kRow = 64 * KR;             // bytes of a weight row per round
    constexpr int kCpr = kRow / 16;           // its 16-byte chunks (8 or 16)
    constexpr int kRpi = 64 / kCpr;           // rows of one 1 KB load (8 or 4)
    constexpr int kIpt = 16 / kRpi;           // loads per 16-row tile (2 or 4)
    constexpr int kBuf = RT * 16 * kRow;      // bytes of one wavefront's round
    extern __shared__ __attribute__((aligned(16))) char s_lds[];   // mfma_lds_bytes(RT, NT, GT, KR)
    auto s_red = reinterpret_cast<float (*)[GT][16][NT * 16]>(s_lds);
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    if (n <= 0) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int K = g.K;
    const int S = K >> 5;                     // k-steps of a row
    const int sw = S / (4 * gridDim.y);       // k-steps of a wavefront (exact)
    const int kw = (blockIdx.y * 4 + wave) * sw;   // its first k-step
    // rounds; with KR = 2 the last is half when sw is odd
    const int nr = (sw + KR - 1) / KR;
    const int u0 = blockIdx.x * 16 * NG;      // first unit (two-row kinds) or row

    // weight rows of this lane's direct loads: tile t, load h covers rows
    // kRpi h + lane / kCpr of the tile; past the end the last valid unit is
    // read and its sums are discarded
    const bf16_t* Ar[RT][kIpt];
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
        for (int h = 0; h < kIpt; ++h) {
            const int u = min(u0 + 16 * q + kRpi * h + lane / kCpr, units - 1);
            int r0 = u, r1 = u;
            if (kPaired) unit_rows<EPI>(g, u, r0, r1);
            Ar[q][h] = (const bf16_t*)g.W + (size_t)r0 * K + kw * 32;
            if (kPaired) Ar[NG + q][h] = (const bf16_t*)g.W + (size_t)r1 * K + kw * 32;
        }
    // this lane's 16-byte chunk of a row: stored position lane % kCpr of
    // tile row kRpi h + lane / kCpr holds source chunk position ^ row; a
    // half round (KR = 2, 64 bytes per row) loads chunks 0..3 and fills the
    // rest with copies
    int csrc[kIpt];
#pragma unroll
    for (int h = 0; h < kIpt; ++h) csrc[h] = (lane % kCpr) ^ ((kRpi * h + lane / kCpr) % kCpr);
    const uint32_t lds_w = (uint32_t)(uintptr_t)(mfma_lptr_t)(s_lds + wave * 2 * kBuf);
    auto issue_a = [&](int r, int buf) {
        const bool part_round = KR == 2 && 2 * r + 1 >= sw;
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int h = 0; h < kIpt; ++h) {
                const int c = part_round ? (csrc[h] & 3) : csrc[h];
                __builtin_amdgcn_global_load_lds((mfma_gptr_t)(Ar[t][h] + 32 * KR * r + 8 * c),
                                                 (mfma_lptr_t)(s_lds + wave * 2 * kBuf + buf * kBuf +
                                                               (16 * t + kRpi * h) * kRow),
                                                 16, 0, 2 /* nontemporal */);
            }
    };
    // fragment (tile t, k-step u of the round): row 16 t + lane % 16, chunk
    // 4 u + lane / 16, stored at that chunk ^ (row % kCpr)
    uint32_t ad[RT][KR];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int u = 0; u < KR; ++u) {
            const int i = lane & 15;
            ad[t][u] = lds_w + (16 * t + i) * kRow + (((4 * u + (lane >> 4)) ^ (i % kCpr)) * 16);
        }

    for (int j0 = 0; j0 < n; j0 += NT * 16) {   // column groups of NT tiles
        // tiles past the last one re-read the last tile and their sums are
        // discarded: the load rounds stay branch-free
        const int nct = min(NT, (n - j0 + 15) / 16);
        const bf16_t* Bp[NT];
#pragma unroll
        for (int c = 0; c < NT; ++c)
            Bp[c] = g.XB + (((size_t)((j0 >> 4) + min(c, nct - 1)) * S + kw) * 128 + lane) * 8;

        f32x4_t acc[RT][NT];
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int c = 0; c < NT; ++c) acc[t][c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

        if (j0 > 0) __syncthreads();   // the previous group's epilogue is done with the LDS
        issue_a(0, 0);
        for (int r = 0; r < nr; ++r) {
            const int buf = r & 1;
            const bool half = KR == 2 && 2 * r + 1 >= sw;
            u32x4_t bv[KR][2][NT];   // [k-step u][high, low][column tile]
#pragma unroll
            for (int u = 0; u < KR; ++u)
#pragma unroll
                for (int c = 0; c < NT; ++c) {
                    const bf16_t* bp = Bp[c] + 1024 * (KR * r + (half ? 0 : u));
                    // reads data no kernel writes while this one runs: no memory clobber
                    asm volatile("global_load_dwordx4 %0, %2, off\n\t"
                                 "global_load_dwordx4 %1, %2, off offset:1024"
                                 : "=&v"(bv[u][0][c]), "=&v"(bv[u][1][c]) : "v"(bp));
                }
            if (r + 1 < nr) {
                issue_a(r + 1, buf ^ 1);
                __builtin_amdgcn_s_waitcnt(mfma_vmcnt(kIpt * RT));
            } else {
                __builtin_amdgcn_s_waitcnt(mfma_vmcnt(0));
            }
            __builtin_amdgcn_sched_barrier(0);   // nothing reads bv or the LDS round before the wait
            u32x4_t a[RT][KR];
#pragma unroll
            for (int t = 0; t < RT; ++t) {
                if constexpr (KR == 2) {
                    asm volatile(
                        "ds_read_b128 %0, %2\n\t"
                        "ds_read_b128 %1, %3\n\t"
                        "s_waitcnt lgkmcnt(0)"
                        : "=&v"(a[t][0]), "=&v"(a[t][1])
                        : "v"(ad[t][0] + buf * kBuf), "v"(ad[t][1] + buf * kBuf)
                        : "memory");
                } else {
                    asm volatile(
                        "ds_read_b128 %0, %4\n\t"
                        "ds_read_b128 %1, %5\n\t"
                        "ds_read_b128 %2, %6\n\t"
                        "ds_read_b128 %3, %7\n\t"
                        "s_waitcnt lgkmcnt(0)"
                        : "=&v"(a[t][0]), "=&v"(a[t][1]), "=&v"(a[t][2]), "=&v"(a[t][3])
                        : "v"(ad[t][0] + buf * kBuf), "v"(ad[t][1] + buf * kBuf),
                          "v"(ad[t][2] + buf * kBuf), "v"(ad[t][3] + buf * kBuf)
                        : "memory");
                }
            }
            // a half round's second k-step multiplies zeros (adds exactly 0):
            // the MFMAs stay unconditional
            if constexpr (KR == 2) {
                const uint32_t keep = half ? 0u : ~0u;
#pragma unroll
                for (int c = 0; c < NT; ++c) {
                    bv[1][0][c] &= keep;
                    bv[1][1][c] &= keep;
                }
            }
#pragma unroll
            for (int u = 0; u < KR; ++u)
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int t = 0; t < RT; ++t)
#pragma unroll
                        for (int c = 0; c < NT; ++c)
                            acc[t][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8_t, a[t][u]),
                                __builtin_bit_cast(bf16x8_t, bv[u][p][c]), acc[t][c], 0, 0, 0);
        }

        // per epilogue group: reduce the four K-slices through LDS, then the
        // epilogue on the finished sums (wavefront order fixed: deterministic)
        const int ncols = min(NT * 16, n - j0);
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            __syncthreads();   // the previous group's epilogue is done with s_red
#pragma unroll
            for (int t = 0; t < GT; ++t)
#pragma unroll
                for (int c = 0; c < NT; ++c)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        s_red[wave][t][4 * (lane >> 4) + v][c * 16 + (lane & 15)] = acc[q + t * NG][c][v];
            __syncthreads();
            if (part && fold) {   // K split, by launch row: [split][part_cap][units]
                for (int p = tid; p < 16 * ncols; p += 256) {
                    const int il = p & 15, j = p >> 4;
                    const int uu = u0 + 16 * q + il;
                    if (uu >= units) continue;
                    part[((size_t)blockIdx.y * g.part_cap + j0 + j) * units + uu] =
                        (s_red[0][0][il][j] + s_red[1][0][il][j]) +
                        (s_red[2][0][il][j] + s_red[3][0][il][j]);
                }
                continue;
            }
            if (part) {   // K split: the workgroup's sums, row j fastest
                for (int p = tid; p < 16 * ncols; p += 256) {
                    const int il = p / ncols, j = p - il * ncols;
                    const int uu = u0 + 16 * q + il;
                    if (uu >= units) continue;
#pragma unroll
                    for (int t = 0; t < GT; ++t)
                        part[part_index(blockIdx.y, GT, t, units, uu, g.rows.n_max, j0 + j)] =
                            (s_red[0][t][il][j] + s_red[1][t][il][j]) +
                            (s_red[2][t][il][j] + s_red[3][t][il][j]);
                }
                continue;
            }
            for (int p = tid; p < 16 * ncols; p += 256) {
                const int il = p / ncols, j = p - il * ncols;
                const int uu = u0 + 16 * q + il;
                if (uu >= units) continue;
                const int b = row_seq(g.rows, j0 + j);
                const float v0 = (s_red[0][0][il][j] + s_red[1][0][il][j]) +
                                 (s_red[2][0][il][j] + s_red[3][0][il][j]);
                if (kPaired) {
                    const float v1 = (s_red[0][GT - 1][il][j] + s_red[1][GT - 1][il][j]) +
                                     (s_red[2][GT - 1][il][j] + s_red[3][GT - 1][il][j]);
                    if (EPI == EPI_SWIGLU && g.xb_out) {   // the down projection's staged input
                        store_split(g.xb_out, xbs_index(j0 + j, uu, g.f, 0), swiglu(v0, v1));
                        continue;
                    }
                    int r0, r1;
                    unit_rows<EPI>(g, uu, r0, r1);
                    epilogue<bf16_t, EPI>(g, b, uu, r0, r1, v0, v1);
                } else {
                    epilogue1<bf16_t, EPI>(g, b, uu, v0);
                }
            }
        }
    }
}

// Sum of the K-split partials in split order, then the residual add.  A
// workgroup takes 64 rows x 16 routed rows: every partial of a thread is
// loaded before the first add, the routed row runs fastest in the reads,
// and a transpose through LDS lets the writes run along the output rows.
template <int SPLITS>
__global__ __launch_bounds__(256) void split_add_kernel(GemvArgs g, int units, int n_host,
                                                        const float* part) {
    __shared__ float s_v[16][65];
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    const int u0 = blockIdx.x * 64, j0 = blockIdx.y * 16;
    if (j0 >= n) return;
    const int tid = threadIdx.x, n_cap = g.rows.n_max;
    const int jl = tid & 15, j = min(j0 + jl, n - 1);
    float v[4][SPLITS];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int u = min(u0 + (tid >> 4) + 16 * r, units - 1);
#pragma unroll
        for (int ks = 0; ks < SPLITS; ++ks) v[r][ks] = part[part_index(ks, 1, 0, units, u, n_cap, j)];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int ks = 0; ks < SPLITS; ++ks) acc += v[r][ks];
        s_v[jl][(tid >> 4) + 16 * r] = acc;
    }
    __syncthreads();
    const int ul = tid & 63, u = u0 + ul;
    if (u >= units) return;
    for (int jj = tid >> 6; jj < 16 && j0 + jj < n; jj += 4)
        epilogue1<bf16_t, EPI_ADD>(g, row_seq(g.rows, j0 + jj), u, s_v[jj][ul]);
}

// One instantiation's launch; LDS beyond the 64 KB default (eight weight
// tiles per workgroup, or four-k-step rounds) is allowed once per device.
template <int EPI, int NT, int RT, int KR>
static hipError_t launch_tiles(dim3 grid, const GemvArgs& g, int units, int n_host, float* part,
                               int fold, hipStream_t s) {
    constexpr int kGT = EPI == EPI_SWIGLU || EPI == EPI_QKV ? 2 : 1;
    constexpr int lds = mfma_lds_bytes(RT, NT, kGT, KR);
    static_assert(lds <= 160 * 1024, "LDS of one CU");
    if constexpr (lds > 64 * 1024) {
        static std::atomic<uint64_t> attr_set{0};
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        const uint64_t bit = 1ull << (dev & 63);
        if (!(attr_set.load(std::memory_order_relaxed) & bit)) {
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(&mfma_kernel<EPI, NT, RT, KR>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, lds);
            if (e != hipSuccess) return e;
            attr_set.fetch_or(bit, std::memory_order_relaxed);
        }
    }
    launch_main(mfma_kernel<EPI, NT, RT, KR>, grid, dim3(256), (uint32_t)lds, s, g, units, n_host,
                part, fold);
    return hipGetLastError();
}

// The launch of a tile configuration with rounds of KR k-steps.
template <int EPI, int RT, int KR>
static hipError_t launch_mfma_rounds(const GemvArgs& g, int units, int n_host, int splits, float* part,
                                     hipStream_t s, int fold) {
    constexpr int per = 16 * (EPI == EPI_SWIGLU || EPI == EPI_QKV ? RT / 2 : RT);
    const dim3 grid((units + per - 1) / per, splits);
    const int tiles = (g.rows.n_max + 15) / 16;
    hipError_t e;
    if (tiles <= 1) e = launch_tiles<EPI, 1, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if (tiles <= 2) e = launch_tiles<EPI, 2, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if (tiles <= 3) e = launch_tiles<EPI, 3, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if (tiles <= 4) e = launch_tiles<EPI, 4, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if (tiles <= 5) e = launch_tiles<EPI, 5, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if (tiles <= 6) e = launch_tiles<EPI, 6, RT, KR>(grid, g, units, n_host, part, fold, s);
    else if constexpr (RT <= 2 && KR == 2) {
        if (tiles <= 7) e = launch_tiles<EPI, 7, RT, KR>(grid, g, units, n_host, part, fold, s);
        else e = launch_tiles<EPI, kMfmaMaxTiles, RT, KR>(grid, g, units, n_host, part, fold, s);
    } else {
        return hipErrorInvalidValue;   // four or eight weight tiles, or long rounds: at most six column tiles
    }
    if (e != hipSuccess || splits == 1 || fold) return e;
    if constexpr (EPI == EPI_ADD) {
        const dim3 sg((units + 63) / 64, (g.rows.n_max + 15) / 16);
        if (splits == 2) split_add_kernel<2><<<sg, 256, 0, s>>>(g, units, n_host, part);
        else if (splits == 4) split_add_kernel<4><<<sg, 256, 0, s>>>(g, units, n_host, part);
        else split_add_kernel<kMfmaMaxSplits><<<sg, 256, 0, s>>>(g, units, n_host, part);
        return hipGetLastError();
    }
    return hipErrorInvalidValue;   // only the residual-add kinds split K
}

// Rounds of four k-steps (two cache lines of each weight row) where the
// tile keeps the LDS of a workgroup within 64 KB (at most two weight tiles),
// the batch within four column tiles (beyond, the round's activation
// registers push the compiler into spilling, and a spill of an untracked
// load's registers before its wait would read data not yet arrived), and
// every wavefront's k-steps split into whole rounds.
inline bool mfma_long_rounds(int rt, int K, int splits, int n_max) {
    return rt <= 2 && (n_max + 15) / 16 <= 4 && (K / 32) % (16 * splits) == 0;
}

template <int EPI, int RT>
static hipError_t launch_mfma_nt(const GemvArgs& g, int units, int n_host, int splits, float* part,
                                 hipStream_t s, int fold = 0) {
    if constexpr (RT <= 2) {
        if (mfma_long_rounds(RT, g.K, splits, g.rows.n_max))
            return launch_mfma_rounds<EPI, RT, 4>(g, units, n_host, splits, part, s, fold);
    }
    return launch_mfma_rounds<EPI, RT, 2>(g, units, n_host, splits, part, s, fold);
}

// A K-split launch takes 128-row tiles (the same splits) where 64-row tiles
// would need a second round of workgroups on part of the chip and 128-row
// ones still give 128 workgroups: the busiest CU then moves one workgroup's
// bytes, not two (13B MHA shape, B = 96: O and down projections).
static bool split_rows128(int units, int splits) {
    return (units + 63) / 64 * splits > 256 && (units + 127) / 128 * splits >= 128;
}

// Weight tiles per workgroup (up to six column tiles of routed rows; beyond,
// the registers of four or eight tiles would halve the occupancy): for the
// two-row kinds eight (gate/up) or four when that grid still has 192 to 256
// (eight) or at least 192 (four) workgroups, since every workgroup re-reads
// all routed rows; for the others the largest that keeps kMfmaMinGrid
// workgroups.  K split per mfma_splits, with 64-row (or, beyond six column
// tiles, 32-row) tiles, or 128-row ones per split_rows128.

template <int EPI>
static hipError_t launch_mfma_epi(const GemvArgs& g, int units, int n_host, float* part, hipStream_t s,
                                  bool fold = false) {
    const bool wide = g.rows.n_max <= 16 * 6;
    if constexpr (EPI == EPI_ADD) {
        if (fold) {   // split sums for the next staging to add
            const int splits = mfma_fold_splits(units, g.K);
            if (wide && split_rows128(units, splits))
                return launch_mfma_nt<EPI, 8>(g, units, n_host, splits, part, s, 1);
            if (wide) return launch_mfma_nt<EPI, 4>(g, units, n_host, splits, part, s, 1);
            return launch_mfma_nt<EPI, 2>(g, units, n_host, splits, part, s, 1);
        }
    }
    const int splits = part ? mfma_splits(EPI, units, g.K) : 1;
    if (splits > 1) {
        if constexpr (EPI == EPI_ADD) {
            if (wide && split_rows128(units, splits))
                return launch_mfma_nt<EPI, 8>(g, units, n_host, splits, part, s);
        }
        if (wide) return launch_mfma_nt<EPI, 4>(g, units, n_host, splits, part, s);
        return launch_mfma_nt<EPI, 2>(g, units, n_host, splits, part, s);
    }
    if constexpr (EPI == EPI_SWIGLU) {
        // a grid that fits the chip in one round of workgroups (one per CU):
        // eight weight tiles per workgroup halve the activation re-reads
        // against four (Llama-8B shape B = 32: 47.3 -> 44.0 us; 13B MHA shape
        // B = 96: 97.9 -> 77.6 us; a second round of workgroups, Qwen-7B B = 64,
        // 82 -> 94 us)
        const int wg8 = (units + 63) / 64;
        if (wide && wg8 >= 192 && wg8 <= 256) return launch_mfma_nt<EPI, 8>(g, units, n_host, 1, nullptr, s);
    }
    if constexpr (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
        // four tiles once they still give 192 workgroups: with many routed
        // rows the activation re-reads outweigh the weights (13B MHA shape,
        // B = 96: QKV 78.1 -> 61.8 us)
        if (wide && units / 32 >= 192) return launch_mfma_nt<EPI, 4>(g, units, n_host, 1, nullptr, s);
        return launch_mfma_nt<EPI, 2>(g, units, n_host, 1, nullptr, s);
    } else {
        if (wide && units / 64 >= kMfmaMinGrid) return launch_mfma_nt<EPI, 4>(g, units, n_host, 1, nullptr, s);
        if (units / 32 >= kMfmaMinGrid) return launch_mfma_nt<EPI, 2>(g, units, n_host, 1, nullptr, s);
        return launch_mfma_nt<EPI, 1>(g, units, n_host, 1, nullptr, s);
    }
}

hipError_t launch_prep(int pro, const GemvArgs& g, hipStream_t s) {
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    if (pro == PRO_RMSNORM) prep_kernel<PRO_RMSNORM><<<g.rows.n_max, kPrepThreads, 0, s>>>(g, n_host);
    else if (pro == PRO_POOL) prep_kernel<PRO_POOL><<<g.rows.n_max, kPrepThreads, 0, s>>>(g, n_host);
    else prep_kernel<PRO_NONE><<<g.rows.n_max, kPrepThreads, 0, s>>>(g, n_host);
    return hipGetLastError();
}

hipError_t launch_mfma(int pro, int epi, const GemvArgs& g, float* part, hipStream_t s, bool fold) {
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    if (pro != PRO_STAGED) {
        hipError_t e = launch_prep(pro, g, s);
        if (e != hipSuccess) return e;
    }
    if (epi == EPI_QKV) return launch_mfma_epi<EPI_QKV>(g, (g.nq + 2 * g.nkv) * (g.hd / 2), n_host, part, s);
    if (epi == EPI_SWIGLU) return launch_mfma_epi<EPI_SWIGLU>(g, g.f, n_host, part, s);
    if (epi == EPI_BIAS_ACT) return launch_mfma_epi<EPI_BIAS_ACT>(g, g.N, n_host, part, s);
    if (fold && (!part || pro != PRO_STAGED)) return hipErrorInvalidValue;
    return launch_mfma_epi<EPI_ADD>(g, g.N, n_host, part, s, fold);
}

}  // namespace buddy
