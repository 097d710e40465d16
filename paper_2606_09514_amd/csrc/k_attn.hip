// Split-K grouped-query decode attention over the KV cache (gfx950).
//
// For a routed sequence b, KV head g and position chunk c, one workgroup
// scores the G = n_heads / n_kv_heads query heads of the group against cache
// rows j in the chunk (j <= pos[b]; the new row written by the projection
// kernel is included, as in the KV-cache equation of the paper's background
// appendix), keeps an online softmax (running max and sum, base 2) and the
// weighted sum of V rows, then writes the chunk's (max, sum, acc) partial.
// The workgroup that finishes last for (b, g) merges the chunk partials in
// chunk order and writes o[b] for the group's heads.  Zero-filled rows of
// skipped steps are ordinary cache rows here (logit 0, value 0).
//
// Lane layout: a cache row of hd elements is read by hd/V lanes with 16-byte
// loads (V = 8 bf16 or 4 fp32), so a wavefront covers 64/(hd/V) rows per
// pass and the row dot products finish with a short xor-shuffle tree.
#include "buddy_internal.h"

namespace buddy {

__device__ __forceinline__ float scale_of(float m, float mn) {
    return m == -INFINITY ? 0.f : exp2f(m - mn);
}

template <typename T>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
    constexpr int V = St<T>::V;
    __shared__ float s_acc[4][kMaxGroup][256 + 2];
    const int i = blockIdx.z;
    const int n = *a.rows.cnt;
    if (i >= n) return;
    const int b = a.rows.idx[i];
    const int g = blockIdx.y, c = blockIdx.x;
    const int pos = a.pos[b];
    const int G = a.nq / a.nkv;
    const int lpr = a.hd / V;          // lanes per cache row
    const int rpw = kWave / lpr;       // rows per wavefront pass
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane % lpr, sub = lane / lpr;
    const int j0 = c * a.chunk_len;
    const int j1 = min(j0 + a.chunk_len, pos + 1);

    // queries of the group, pre-scaled so that exp2 of the score is the
    // softmax weight: q * log2(e) / sqrt(hd)
    const float qs = 1.4426950408889634f / sqrtf((float)a.hd);
    float qr[kMaxGroup][V];
    const float* qb = a.q + (size_t)b * a.nq * a.hd + (size_t)g * G * a.hd + col * V;
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
#pragma unroll
        for (int e = 0; e < V; ++e) qr[h][e] = 0.f;
        if (h < G) {
#pragma unroll
            for (int e = 0; e < V; ++e) qr[h][e] = qb[(size_t)h * a.hd + e] * qs;
        }
    }

    float m[kMaxGroup], l[kMaxGroup], acc[kMaxGroup][V];
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
        m[h] = -INFINITY; l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < V; ++e) acc[h][e] = 0.f;
    }

    const size_t base = ((size_t)b * a.nkv + g) * a.T * a.hd + col * V;
    const T* Kb = (const T*)a.kc + base;
    const T* Vb = (const T*)a.vc + base;
    for (int j = j0 + wave * rpw + sub; j < j1; j += 4 * rpw) {
        float kr[V], vr[V];
        St<T>::vec(Kb + (size_t)j * a.hd, kr);
        St<T>::vec(Vb + (size_t)j * a.hd, vr);
#pragma unroll
        for (int h = 0; h < kMaxGroup; ++h) {
            if (h < G) {
                float sc = 0.f;
#pragma unroll
                for (int e = 0; e < V; ++e) sc += qr[h][e] * kr[e];
                for (int o = lpr >> 1; o > 0; o >>= 1) sc += __shfl_xor(sc, o, kWave);
                const float mn = fmaxf(m[h], sc);
                const float al = scale_of(m[h], mn);
                const float p = exp2f(sc - mn);
                l[h] = l[h] * al + p;
#pragma unroll
                for (int e = 0; e < V; ++e) acc[h][e] = acc[h][e] * al + p * vr[e];
                m[h] = mn;
            }
        }
    }

    // merge the row slots of the wavefront (lanes with equal col)
    for (int o = lpr; o < kWave; o <<= 1) {
#pragma unroll
        for (int h = 0; h < kMaxGroup; ++h) {
            if (h < G) {
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
        for (int h = 0; h < kMaxGroup; ++h) {
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
    __syncthreads();

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
        float* pp = a.part + (((size_t)b * a.nq + g * G + h) * a.max_chunks + c) * pstride;
        pp[e] = A;
        if (e == 0) { pp[a.hd] = M; pp[a.hd + 1] = L; }
    }

    if (arrive_last(&a.counters[b * a.nkv + g], a.chunks)) {
        for (int t = tid; t < G * a.hd; t += 256) {
            const int h = t / a.hd, e = t % a.hd;
            const float* pp = a.part + (((size_t)b * a.nq + g * G + h) * a.max_chunks) * pstride;
            float M = -INFINITY;
            for (int q = 0; q < a.chunks; ++q) M = fmaxf(M, pp[q * pstride + a.hd]);
            float L = 0.f, A = 0.f;
            for (int q = 0; q < a.chunks; ++q) {
                const float sw = scale_of(pp[q * pstride + a.hd], M);
                L += pp[q * pstride + a.hd + 1] * sw;
                A += pp[q * pstride + e] * sw;
            }
            a.o[(size_t)b * a.nq * a.hd + (size_t)(g * G + h) * a.hd + e] = A / L;
        }
    }
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
    dim3 grid(a.chunks, a.nkv, a.rows.n_max);
    if (dtype == BUDDY_BF16) attn_kernel<bf16_t><<<grid, 256, 0, s>>>(a);
    else attn_kernel<float><<<grid, 256, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace buddy
