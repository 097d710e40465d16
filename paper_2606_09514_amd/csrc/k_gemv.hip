// Weight-streaming GEMV for the routed blocks and the Decision Module's first
// layer (gfx950).
//
// Y[b] (op)= W x_b for the routed rows b = idx[i], i < cnt, with W [N][K]
// row-major in the storage dtype and x_b fp32.  Each 64-lane wavefront owns a
// "unit" of two weight rows and streams them once with 16-byte loads per lane
// while the activation rows of the workgroup sit in LDS, so every weight byte
// is read from HBM once per launch whatever the number of routed rows.
//
// Prologues:  PRO_NONE    x = X[b]
//             PRO_RMSNORM x = X[b] / sqrt(mean(X[b]^2) + eps) * gain
// Epilogues:  EPI_ADD      Y[b][r] += acc              (residual of Eq. 1)
//             EPI_BIAS_ACT Y[b][r] = act(acc + bias)  (Decision Module layer 1)
//             EPI_SWIGLU   unit j = rows (j, f + j): Y[b][j] = SiLU(g) * u
//             EPI_QKV      unit = rows (i, i + hd/2) of one head: rotary
//                          embedding at pos[b] for q and k heads, q to Y,
//                          k and v appended to the cache rounded to storage.
#include "buddy_internal.h"

namespace buddy {

constexpr int kGemvLds = 80 * 1024;  // dynamic LDS cap of one GEMV workgroup

template <int EPI>
__device__ __forceinline__ void unit_rows(const GemvArgs& g, int u, int& r0, int& r1) {
    if (EPI == EPI_SWIGLU) { r0 = u; r1 = g.f + u; }
    else if (EPI == EPI_QKV) {
        const int half = g.hd >> 1;
        const int hg = u / half, i = u - hg * half;
        r0 = hg * g.hd + i; r1 = r0 + half;
    } else { r0 = 2 * u; r1 = 2 * u + 1; }
}

__device__ __forceinline__ float act_fn(float x, int act) {
    if (act == BUDDY_ACT_GELU_ERF) return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
    return x / (1.0f + expf(-x));
}

template <typename TW, int EPI>
__device__ __forceinline__ void epilogue(const GemvArgs& g, int b, int u, int r0, int r1,
                                         float v0, float v1) {
    if (EPI == EPI_ADD) {
        float* y = g.Y + (size_t)b * g.ldy;
        y[r0] += v0;
        y[r1] += v1;
    } else if (EPI == EPI_BIAS_ACT) {
        float* y = g.Y + (size_t)b * g.ldy;
        const TW* bias = (const TW*)g.bias;
        y[r0] = act_fn(v0 + St<TW>::get(bias, r0), g.act);
        y[r1] = act_fn(v1 + St<TW>::get(bias, r1), g.act);
    } else if (EPI == EPI_SWIGLU) {
        g.Y[(size_t)b * g.ldy + u] = v0 / (1.0f + expf(-v0)) * v1;
    } else {  // EPI_QKV
        const int half = g.hd >> 1;
        const int hg = u / half, i = u - hg * half;
        const int pos = g.pos[b];
        if (hg < g.nq + g.nkv) {
            double sn, cs;
            sincos((double)pos * g.inv_freq[i], &sn, &cs);
            const float c = (float)cs, s = (float)sn;
            const float a0 = v0 * c - v1 * s;
            const float a1 = v1 * c + v0 * s;
            v0 = a0; v1 = a1;
        }
        if (hg < g.nq) {
            float* y = g.Y + (size_t)b * g.ldy + (size_t)hg * g.hd;
            y[i] = v0;
            y[i + half] = v1;
        } else {
            const bool is_k = hg < g.nq + g.nkv;
            const int kvh = is_k ? hg - g.nq : hg - g.nq - g.nkv;
            TW* dst = (TW*)(is_k ? g.kc : g.vc) +
                      (((size_t)b * g.nkv + kvh) * g.T + pos) * g.hd;
            St<TW>::put(dst, i, v0);
            St<TW>::put(dst, i + half, v1);
        }
    }
}

template <typename TW, int NR, int PRO, int EPI>
__global__ __launch_bounds__(256) void gemv_kernel(GemvArgs g, int units) {
    extern __shared__ float xs[];   // [NR][K] activation rows of the current group
    __shared__ float s_red[4][NR];
    __shared__ float s_inv[NR];
    const int n = *g.rows.cnt;
    if (n <= 0) return;
    constexpr int V = St<TW>::V;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int K = g.K;
    const TW* W = (const TW*)g.W;

    for (int i0 = 0; i0 < n; i0 += NR) {
        const int nr = min(NR, n - i0);
        __syncthreads();  // the previous group's readers are done with xs
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            float ss = 0.f;
            if (r < nr) {
                const float* xr = g.X + (size_t)g.rows.idx[i0 + r] * g.ldx;
                for (int k = tid * 4; k < K; k += 1024) {
                    const float4 v = *reinterpret_cast<const float4*>(xr + k);
                    *reinterpret_cast<float4*>(xs + r * K + k) = v;
                    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
                }
            } else {
                for (int k = tid * 4; k < K; k += 1024)
                    *reinterpret_cast<float4*>(xs + r * K + k) = make_float4(0.f, 0.f, 0.f, 0.f);
            }
            if (PRO == PRO_RMSNORM) {
                ss = wave_sum(ss);
                if (lane == 0) s_red[wave][r] = ss;
            }
        }
        if (PRO == PRO_RMSNORM) {
            __syncthreads();
            if (tid < NR) {
                const float t = s_red[0][tid] + s_red[1][tid] + s_red[2][tid] + s_red[3][tid];
                s_inv[tid] = 1.0f / sqrtf(t / (float)K + g.eps);
            }
            __syncthreads();
            const TW* gain = (const TW*)g.gain;
            for (int r = 0; r < nr; ++r)
                for (int k = tid; k < K; k += 256) xs[r * K + k] *= s_inv[r] * St<TW>::get(gain, k);
        }
        __syncthreads();

        for (int u = blockIdx.x * 4 + wave; u < units; u += gridDim.x * 4) {
            int r0, r1;
            unit_rows<EPI>(g, u, r0, r1);
            const TW* w0 = W + (size_t)r0 * K;
            const TW* w1 = W + (size_t)r1 * K;
            float acc0[NR], acc1[NR];
#pragma unroll
            for (int r = 0; r < NR; ++r) acc0[r] = acc1[r] = 0.f;
#pragma unroll 4
            for (int k = lane * V; k < K; k += kWave * V) {
                float a[V], c[V];
                St<TW>::vec(w0 + k, a);
                St<TW>::vec(w1 + k, c);
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    const float* x = xs + r * K + k;
#pragma unroll
                    for (int e = 0; e < V; ++e) {
                        acc0[r] += a[e] * x[e];
                        acc1[r] += c[e] * x[e];
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                acc0[r] = wave_sum(acc0[r]);
                acc1[r] = wave_sum(acc1[r]);
            }
            if (lane < nr) {
                // lane r finishes routed row r of the group
#pragma unroll
                for (int r = 0; r < NR; ++r)
                    if (r == lane) epilogue<TW, EPI>(g, g.rows.idx[i0 + r], u, r0, r1, acc0[r], acc1[r]);
            }
        }
    }
}

template <typename TW, int NR, int PRO, int EPI>
static hipError_t launch_one(const GemvArgs& g, int units, hipStream_t s) {
    const size_t lds = (size_t)NR * g.K * sizeof(float);
    static bool attr_set = false;
    if (lds > 64 * 1024 && !attr_set) {
        // dynamic LDS above the 64 KB default; the dispatcher never asks
        // for more than kGemvLds
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<TW, NR, PRO, EPI>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kGemvLds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    int grid = (units + 3) / 4;
    if (grid > 2048) grid = 2048;
    gemv_kernel<TW, NR, PRO, EPI><<<grid, 256, lds, s>>>(g, units);
    return hipGetLastError();
}

template <typename TW, int PRO, int EPI>
static hipError_t dispatch_nr(const GemvArgs& g, int units, hipStream_t s) {
    // rows staged per pass: as many as fit in kGemvLds, at most 4
    const size_t row_bytes = (size_t)g.K * sizeof(float);
    const int fit = (int)(kGemvLds / row_bytes);
    int nr = g.rows.n_max < fit ? g.rows.n_max : fit;
    if (nr >= 4) return launch_one<TW, 4, PRO, EPI>(g, units, s);
    if (nr >= 2) return launch_one<TW, 2, PRO, EPI>(g, units, s);
    return launch_one<TW, 1, PRO, EPI>(g, units, s);
}

template <typename TW>
static hipError_t dispatch_epi(int pro, int epi, const GemvArgs& g, hipStream_t s) {
    if (epi == EPI_QKV) {
        const int units = (g.nq + 2 * g.nkv) * (g.hd / 2);
        return dispatch_nr<TW, PRO_RMSNORM, EPI_QKV>(g, units, s);
    }
    if (epi == EPI_SWIGLU) return dispatch_nr<TW, PRO_RMSNORM, EPI_SWIGLU>(g, g.f, s);
    if (epi == EPI_BIAS_ACT) return dispatch_nr<TW, PRO_NONE, EPI_BIAS_ACT>(g, g.N / 2, s);
    if (pro == PRO_RMSNORM) return dispatch_nr<TW, PRO_RMSNORM, EPI_ADD>(g, g.N / 2, s);
    return dispatch_nr<TW, PRO_NONE, EPI_ADD>(g, g.N / 2, s);
}

hipError_t launch_gemv(int dtype, int pro, int epi, const GemvArgs& g, hipStream_t s) {
    if (dtype == BUDDY_BF16) return dispatch_epi<bf16_t>(pro, epi, g, s);
    return dispatch_epi<float>(pro, epi, g, s);
}

}  // namespace buddy
