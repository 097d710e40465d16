// MFMA path of the routed projections (gfx950, bf16 weights), used for
// batches of more than four sequences: the projection is then a real dense
// contraction over the routed rows.
//
//  prep_kernel  writes the routed rows as bf16 in MFMA operand order (row i
//               of the launch is sequence idx[i]): RMSNorm and gain folded in
//               (PRO_RMSNORM), the router context built from the pool's split
//               sums (PRO_POOL), or a plain conversion (PRO_NONE).
//  mfma_kernel  Y = W XB^T with v_mfma_f32_16x16x32_bf16 (fp32 accumulate).
//               A workgroup owns RT 16-row weight tiles (16 RT rows, or 8 RT
//               two-row units) and all routed rows; its four wavefronts take
//               a quarter of K each, their sums are reduced through LDS one
//               epilogue group at a time, and the fused epilogues of the GEMV
//               path run on the finished sums.
//
// Operand layouts of v_mfma_f32_16x16x32_bf16 (checked on the device):
//   A[i][k] (16 x 32): lane i + 16 (k / 8), element k % 8
//   B[k][j] (32 x 16): lane j + 16 (k / 8), element k % 8
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4
// One 16-byte load per lane fetches an A tile segment from the row-major
// weights (16 rows x 64 bytes).  The activations are small and re-read by
// every workgroup, so they are stored in B-operand order: the B tile of
// column tile c and k-step s is 1 KB at ((c * K/32 + s) * 64 + lane) * 8
// elements, one contiguous load per wavefront.
#include "buddy_internal.h"
#include "epilogue.h"

namespace buddy {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kMfmaMaxTiles = 8;   // 16-row column tiles of routed rows per pass


// ----------------------------------------------------------------- prep

template <int PRO>
__global__ __launch_bounds__(256) void prep_kernel(GemvArgs g, int n_host) {
    __shared__ float s_ss[4];
    const int i = blockIdx.x;
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    if (i >= n) return;
    const int b = row_seq(g.rows, i);
    const int K = g.K, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float inv = 1.f;
    if (PRO == PRO_RMSNORM) {
        const float* x = g.X + (size_t)b * g.ldx;
        float ss = 0.f;
        for (int k = tid * 4; k < K; k += 1024) {
            const float4 v = *reinterpret_cast<const float4*>(x + k);
            ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        }
        ss = wave_sum(ss);
        if (lane == 0) s_ss[wave] = ss;
        __syncthreads();
        inv = 1.0f / sqrtf((s_ss[0] + s_ss[1] + s_ss[2] + s_ss[3]) / (float)K + g.eps);
    }
    const float inv_n = PRO == PRO_POOL ? 1.0f / (float)(seq_pos(g.pos, g.pos_u, b) + 1) : 0.f;
    const int zdim = pooled_dim(g.ctx, g.nkv, g.hd);
    for (int k = tid * 8; k < K; k += 256 * 8) {
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
        uint4 o;
        o.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
        o.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
        o.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
        o.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
        // B-operand order: tile i / 16, k-step k / 32, lane (i % 16) + 16 (k / 8 % 4)
        const size_t frag = ((size_t)(i >> 4) * (K >> 5) + (k >> 5)) * 64 + (i & 15) + 16 * ((k >> 3) & 3);
        *reinterpret_cast<uint4*>(g.XB + frag * 8) = o;
    }
}

// ----------------------------------------------------------------- MFMA

// k-steps per load round: all loads of a round are issued before its MFMAs
__host__ __device__ constexpr int mfma_round(int rt, int nt) {
    return 16 / (rt + nt) < 1 ? 1 : 16 / (rt + nt) > 8 ? 8 : 16 / (rt + nt);
}

template <int EPI, int NT, int RT>
__global__ __launch_bounds__(256) void mfma_kernel(GemvArgs g, int units, int n_host) {
    constexpr bool kPaired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    constexpr int GT = kPaired ? 2 : 1;       // weight tiles per epilogue group
    constexpr int NG = RT / GT;               // epilogue groups (16 units or rows each)
    constexpr int U = mfma_round(RT, NT);
    __shared__ float s_red[4][GT][16][NT * 16];
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    if (n <= 0) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int K = g.K;
    const int S = K >> 5;                     // k-steps of a row
    const int sw = S >> 2;                    // k-steps of a wavefront (K % 128 == 0)
    const int u0 = blockIdx.x * 16 * NG;      // first unit (two-row kinds) or row

    // A rows of this lane (lane % 16 within each tile); past the end the
    // last valid unit is read and its sums are discarded
    const bf16_t* Ap[RT];
#pragma unroll
    for (int q = 0; q < NG; ++q) {
        const int u = min(u0 + 16 * q + (lane & 15), units - 1);
        int r0 = u, r1 = u;
        if (kPaired) unit_rows<EPI>(g, u, r0, r1);
        Ap[q] = (const bf16_t*)g.W + (size_t)r0 * K + wave * (K >> 2) + 8 * (lane >> 4);
        if (kPaired) Ap[NG + q] = (const bf16_t*)g.W + (size_t)r1 * K + wave * (K >> 2) + 8 * (lane >> 4);
    }

    for (int j0 = 0; j0 < n; j0 += NT * 16) {   // column groups of NT tiles
        // tiles past the last one re-read the last tile and their sums are
        // discarded: the load rounds stay branch-free
        const int nct = min(NT, (n - j0 + 15) / 16);
        const bf16_t* Bp[NT];
#pragma unroll
        for (int c = 0; c < NT; ++c)
            Bp[c] = g.XB + (((size_t)((j0 >> 4) + min(c, nct - 1)) * S + wave * sw) * 64 + lane) * 8;

        f32x4_t acc[RT][NT];
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int c = 0; c < NT; ++c) acc[t][c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

        int s = 0;
        for (; s + U <= sw; s += U) {
            bf16x8_t a[U][RT], bv[U][NT];
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int t = 0; t < RT; ++t)
                    a[u][t] = *reinterpret_cast<const bf16x8_t*>(Ap[t] + 32 * (s + u));
#pragma unroll
                for (int c = 0; c < NT; ++c)
                    bv[u][c] = *reinterpret_cast<const bf16x8_t*>(Bp[c] + 512 * (s + u));
            }
            __builtin_amdgcn_sched_barrier(0);   // keep every load of the round ahead
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int c = 0; c < NT; ++c)
                        acc[t][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][t], bv[u][c],
                                                                            acc[t][c], 0, 0, 0);
        }
        for (; s < sw; ++s) {
            bf16x8_t a[RT], bv[NT];
#pragma unroll
            for (int t = 0; t < RT; ++t) a[t] = *reinterpret_cast<const bf16x8_t*>(Ap[t] + 32 * s);
#pragma unroll
            for (int c = 0; c < NT; ++c) bv[c] = *reinterpret_cast<const bf16x8_t*>(Bp[c] + 512 * s);
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int c = 0; c < NT; ++c)
                    acc[t][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], bv[c], acc[t][c], 0, 0, 0);
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

// Workgroups below which a launch takes smaller weight tiles per workgroup
constexpr int kMfmaMinGrid = 384;

template <int EPI, int RT>
static hipError_t launch_mfma_nt(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    constexpr int per = 16 * (EPI == EPI_SWIGLU || EPI == EPI_QKV ? RT / 2 : RT);
    const int grid = (units + per - 1) / per;
    const int tiles = (g.rows.n_max + 15) / 16;
    if (tiles <= 1) launch_main(mfma_kernel<EPI, 1, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if (tiles <= 2) launch_main(mfma_kernel<EPI, 2, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if (tiles <= 3) launch_main(mfma_kernel<EPI, 3, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if (tiles <= 4) launch_main(mfma_kernel<EPI, 4, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if (tiles <= 5) launch_main(mfma_kernel<EPI, 5, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if (tiles <= 6) launch_main(mfma_kernel<EPI, 6, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    else if constexpr (RT <= 2) {
        if (tiles <= 7) launch_main(mfma_kernel<EPI, 7, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
        else launch_main(mfma_kernel<EPI, kMfmaMaxTiles, RT>, dim3(grid), dim3(256), 0, s, g, units, n_host);
    }
    return hipGetLastError();
}

// Largest weight tile per workgroup that still gives kMfmaMinGrid workgroups
// (four tiles only up to six column tiles: beyond, their registers would
// halve the occupancy)
template <int EPI>
static hipError_t launch_mfma_epi(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    const bool wide = g.rows.n_max <= 16 * 6;
    if constexpr (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
        if (wide && units / 32 >= kMfmaMinGrid) return launch_mfma_nt<EPI, 4>(g, units, n_host, s);
        return launch_mfma_nt<EPI, 2>(g, units, n_host, s);
    } else {
        if (wide && units / 64 >= kMfmaMinGrid) return launch_mfma_nt<EPI, 4>(g, units, n_host, s);
        if (units / 32 >= kMfmaMinGrid) return launch_mfma_nt<EPI, 2>(g, units, n_host, s);
        return launch_mfma_nt<EPI, 1>(g, units, n_host, s);
    }
}

hipError_t launch_prep(int pro, const GemvArgs& g, hipStream_t s) {
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    if (pro == PRO_RMSNORM) prep_kernel<PRO_RMSNORM><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    else if (pro == PRO_POOL) prep_kernel<PRO_POOL><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    else prep_kernel<PRO_NONE><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    return hipGetLastError();
}

hipError_t launch_mfma(int pro, int epi, const GemvArgs& g, hipStream_t s) {
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    hipError_t e = launch_prep(pro, g, s);
    if (e != hipSuccess) return e;
    if (epi == EPI_QKV) return launch_mfma_epi<EPI_QKV>(g, (g.nq + 2 * g.nkv) * (g.hd / 2), n_host, s);
    if (epi == EPI_SWIGLU) return launch_mfma_epi<EPI_SWIGLU>(g, g.f, n_host, s);
    if (epi == EPI_BIAS_ACT) return launch_mfma_epi<EPI_BIAS_ACT>(g, g.N, n_host, s);
    return launch_mfma_epi<EPI_ADD>(g, g.N, n_host, s);
}

}  // namespace buddy
