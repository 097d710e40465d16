// MFMA path of the routed projections (gfx950, bf16 weights), used when a
// launch has more routed rows than the GEMV stages in one pass: the
// projection is then a real dense contraction over the routed rows.
//
//  prep_kernel  writes the routed rows as compact bf16 rows XB[i] (row i of
//               the launch is sequence idx[i]): RMSNorm and gain folded in
//               (PRO_RMSNORM), the router context built from the pool's split
//               sums (PRO_POOL), or a plain conversion (PRO_NONE).
//  mfma_kernel  Y = W XB^T with v_mfma_f32_16x16x32_bf16 (fp32 accumulate).
//               A workgroup owns 16 weight rows (or 16 two-row units) and all
//               routed rows; its four wavefronts take a quarter of K each and
//               are reduced through LDS, then the same fused epilogues as the
//               GEMV path run on the finished sums.
//
// Operand layouts of v_mfma_f32_16x16x32_bf16 (checked on the device):
//   A[i][k] (16 x 32): lane i + 16 (k / 8), element k % 8
//   B[k][j] (32 x 16): lane j + 16 (k / 8), element k % 8
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4
// so one 16-byte load per lane fetches an A tile row segment from the
// row-major weights and a B tile from a compact activation row.
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
    bf16_t* out = g.XB + (size_t)i * g.ldxb;
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
    const int zdim = 2 * g.nkv * g.hd;
    for (int k = tid * 8; k < K; k += 256 * 8) {
        float v[8];
        if (PRO == PRO_POOL && k < zdim) {
            const int which = k / (g.nkv * g.hd), gg = (k / g.hd) % g.nkv, e = k % g.hd;
            const float* pp = g.pool_part +
                (((size_t)b * g.nkv + gg) * g.pool_max_splits) * 2 * g.hd + which * g.hd + e;
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = 0.f;
            for (int s = 0; s < g.pool_splits; ++s) {
                const float4 t0 = *reinterpret_cast<const float4*>(pp + (size_t)s * 2 * g.hd);
                const float4 t1 = *reinterpret_cast<const float4*>(pp + (size_t)s * 2 * g.hd + 4);
                v[0] += t0.x; v[1] += t0.y; v[2] += t0.z; v[3] += t0.w;
                v[4] += t1.x; v[5] += t1.y; v[6] += t1.z; v[7] += t1.w;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] *= inv_n;
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
        *reinterpret_cast<uint4*>(out + k) = o;
    }
}

// ----------------------------------------------------------------- MFMA

template <int EPI, int NT>
__global__ __launch_bounds__(256) void mfma_kernel(GemvArgs g, int units, int n_host) {
    constexpr bool kPaired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    constexpr int RT = kPaired ? 2 : 1;       // weight row tiles per wavefront
    __shared__ float s_red[4][RT][16][NT * 16];
    const int n = n_host >= 0 ? n_host : *g.rows.cnt;
    if (n <= 0) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int K = g.K;
    const int ks = K / 4;                     // this wavefront's K-slice (K % 128 == 0)
    const int kbeg = wave * ks + 8 * (lane >> 4);
    const int t0 = blockIdx.x * 16;           // first unit (two-row kinds) or row

    // A rows of this lane (lane % 16 within the tile); past the end the last
    // valid unit is read and its results are discarded
    const int u = min(t0 + (lane & 15), units - 1);
    int arow[RT];
    if (kPaired) {
        int r0, r1;
        unit_rows<EPI>(g, u, r0, r1);
        arow[0] = r0;
        arow[RT - 1] = r1;
    } else {
        arow[0] = u;
    }
    const bf16_t* Ap[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) Ap[t] = (const bf16_t*)g.W + (size_t)arow[t] * K + kbeg;

    for (int j0 = 0; j0 < n; j0 += NT * 16) {   // column groups of NT tiles
        const int nct = min(NT, (n - j0 + 15) / 16);
        const bf16_t* Bp[NT];
#pragma unroll
        for (int c = 0; c < NT; ++c)
            Bp[c] = g.XB + (size_t)(j0 + min(c, nct - 1) * 16 + (lane & 15)) * g.ldxb + kbeg;

        f32x4_t acc[RT][NT];
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int c = 0; c < NT; ++c) acc[t][c] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

#pragma unroll 2
        for (int k = 0; k < ks; k += 32) {
            bf16x8_t a[RT], bv[NT];
#pragma unroll
            for (int t = 0; t < RT; ++t) a[t] = *reinterpret_cast<const bf16x8_t*>(Ap[t] + k);
#pragma unroll
            for (int c = 0; c < NT; ++c)
                if (c < nct) bv[c] = *reinterpret_cast<const bf16x8_t*>(Bp[c] + k);
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int c = 0; c < NT; ++c)
                    if (c < nct)
                        acc[t][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], bv[c], acc[t][c],
                                                                            0, 0, 0);
        }

        // reduce the four K-slices through LDS
        if (j0 > 0) __syncthreads();   // the previous group's epilogue is done with s_red
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    s_red[wave][t][4 * (lane >> 4) + v][c * 16 + (lane & 15)] = acc[t][c][v];
        __syncthreads();

        const int ncols = min(NT * 16, n - j0);
        for (int p = tid; p < 16 * ncols; p += 256) {
            const int il = p / ncols, j = p - il * ncols;
            const int uu = t0 + il;
            if (uu >= units) continue;
            const int b = row_seq(g.rows, j0 + j);
            const float v0 = (s_red[0][0][il][j] + s_red[1][0][il][j]) +
                             (s_red[2][0][il][j] + s_red[3][0][il][j]);
            if (kPaired) {
                const float v1 = (s_red[0][RT - 1][il][j] + s_red[1][RT - 1][il][j]) +
                                 (s_red[2][RT - 1][il][j] + s_red[3][RT - 1][il][j]);
                int r0, r1;
                unit_rows<EPI>(g, uu, r0, r1);
                epilogue<bf16_t, EPI>(g, b, uu, r0, r1, v0, v1);
            } else {
                epilogue1<bf16_t, EPI>(g, b, uu, v0);
            }
        }
    }
}

template <int EPI>
static hipError_t launch_mfma_epi(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    const int grid = (units + 15) / 16;
    const int tiles = (g.rows.n_max + 15) / 16;
    if (tiles <= 1) mfma_kernel<EPI, 1><<<grid, 256, 0, s>>>(g, units, n_host);
    else if (tiles <= 2) mfma_kernel<EPI, 2><<<grid, 256, 0, s>>>(g, units, n_host);
    else if (tiles <= 4) mfma_kernel<EPI, 4><<<grid, 256, 0, s>>>(g, units, n_host);
    else mfma_kernel<EPI, kMfmaMaxTiles><<<grid, 256, 0, s>>>(g, units, n_host);
    return hipGetLastError();
}

hipError_t launch_mfma(int pro, int epi, const GemvArgs& g, hipStream_t s) {
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    if (pro == PRO_RMSNORM) prep_kernel<PRO_RMSNORM><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    else if (pro == PRO_POOL) prep_kernel<PRO_POOL><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    else prep_kernel<PRO_NONE><<<g.rows.n_max, 256, 0, s>>>(g, n_host);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (epi == EPI_QKV) return launch_mfma_epi<EPI_QKV>(g, (g.nq + 2 * g.nkv) * (g.hd / 2), n_host, s);
    if (epi == EPI_SWIGLU) return launch_mfma_epi<EPI_SWIGLU>(g, g.f, n_host, s);
    if (epi == EPI_BIAS_ACT) return launch_mfma_epi<EPI_BIAS_ACT>(g, g.N, n_host, s);
    return launch_mfma_epi<EPI_ADD>(g, g.N, n_host, s);
}

}  // namespace buddy
