// Epilogues shared by the GEMV (k_gemv.hip) and MFMA (k_mfma.hip) paths of
// the routed projections: weight-row pairing of the two-row kinds and what is
// done with a finished sum (residual add, bias + activation, SwiGLU, rotary
// embedding with KV append).
#pragma once

#include "buddy_internal.h"

namespace buddy {

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

// SwiGLU of a gate sum v0 and an up sum v1: SiLU(v0) v1.
__device__ __forceinline__ float swiglu(float v0, float v1) { return v0 / (1.0f + expf(-v0)) * v1; }

// Epilogue of one finished row for the single-row kinds.
template <typename TW, int EPI>
__device__ __forceinline__ void epilogue1(const GemvArgs& g, int b, int row, float v) {
    float* y = g.Y + (size_t)b * g.ldy;
    if (EPI == EPI_ADD) y[row] += v;
    else y[row] = act_fn(v + St<TW>::get((const TW*)g.bias, row), g.act);
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
        g.Y[(size_t)b * g.ldy + u] = swiglu(v0, v1);
    } else {  // EPI_QKV
        const int half = g.hd >> 1;
        const int hg = u / half, i = u - hg * half;
        int slot, pos;
        slot_pos(b, g.tok_T, g.pos, g.pos_u, slot, pos);
        if (hg < g.nq + g.nkv) {
            const float2 cs = g.rope[(size_t)pos * half + i];
            const float a0 = v0 * cs.x - v1 * cs.y;
            const float a1 = v1 * cs.x + v0 * cs.y;
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
                      (((size_t)slot * g.nkv + kvh) * g.T + pos) * g.hd;
            St<TW>::put(dst, i, v0);
            St<TW>::put(dst, i + half, v1);
        }
    }
}

}  // namespace buddy
