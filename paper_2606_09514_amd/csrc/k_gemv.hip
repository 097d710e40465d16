// Weight-streaming GEMV for the routed blocks and the Decision Module's first
// layer (gfx950).
//
// Y[b] (op)= W x_b for the routed rows b = idx[i], i < cnt, with W [N][K]
// row-major in the storage dtype and x_b fp32.  Each 64-lane wavefront owns
// one weight row (or a K-slice of it), issues all of its 16-byte loads at
// once and keeps them in registers while the activation rows of the
// workgroup pass through LDS, so every weight byte is read from HBM once per
// launch whatever the number of routed rows.  Latency is hidden by the many
// resident wavefronts rather than by software pipelining.
//
// Prologues:  PRO_NONE    x = X[b]
//             PRO_RMSNORM x = X[b] / sqrt(mean(X[b]^2) + eps) * gain
//             PRO_POOL    x = [sum K / n | sum V / n | h_b], folding the split
//                         sums of the first-layer pool (router context)
// Epilogues:  EPI_ADD      Y[b][r] += acc              (residual of Eq. 1)
//             EPI_BIAS_ACT Y[b][r] = act(acc + bias)  (Decision Module layer 1)
//             EPI_SWIGLU   unit j = rows (j, f + j): Y[b][j] = SiLU(g) * u
//             EPI_QKV      unit = rows (i, i + hd/2) of one head: rotary
//                          embedding at pos[b] for q and k heads, q to Y,
//                          k and v appended to the cache rounded to storage.
#include <atomic>
#include <cstdint>
#include <type_traits>

#include "buddy_internal.h"
#include "epilogue.h"

namespace buddy {

constexpr int kGemvLds = 80 * 1024;  // dynamic LDS cap of one GEMV workgroup

// Dot product of one packed 16-byte weight vector with the matching
// activations x[0..V) (16-byte aligned in LDS).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float dot16(const u32x4_t& w, const float* x, bf16_t) {
    const float4 a = *reinterpret_cast<const float4*>(x);
    const float4 b = *reinterpret_cast<const float4*>(x + 4);
    float s = __uint_as_float(w.x << 16) * a.x;
    s += __uint_as_float(w.x & 0xffff0000u) * a.y;
    s += __uint_as_float(w.y << 16) * a.z;
    s += __uint_as_float(w.y & 0xffff0000u) * a.w;
    s += __uint_as_float(w.z << 16) * b.x;
    s += __uint_as_float(w.z & 0xffff0000u) * b.y;
    s += __uint_as_float(w.w << 16) * b.z;
    s += __uint_as_float(w.w & 0xffff0000u) * b.w;
    return s;
}
__device__ __forceinline__ float dot16(const u32x4_t& w, const float* x, float) {
    const float4 a = *reinterpret_cast<const float4*>(x);
    float s = __uint_as_float(w.x) * a.x;
    s += __uint_as_float(w.y) * a.y;
    s += __uint_as_float(w.z) * a.z;
    s += __uint_as_float(w.w) * a.w;
    return s;
}

// Weight row of wavefront slot `slot` (0..P-1, P wavefronts per workgroup)
// in workgroup `blk`, or -1.
//   EPI_ADD, EPI_BIAS_ACT: P/S rows per workgroup, each split over S K-slices.
//   EPI_SWIGLU, EPI_QKV: P/2 units per workgroup; slot s < P/2 holds the
//   first row of unit s, slot P/2 + s its second row.
template <int EPI, int S, int P>
__device__ __forceinline__ int slot_row(const GemvArgs& g, int blk, int slot, int units) {
    if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
        const int u = blk * (P / 2) + slot % (P / 2);
        if (u >= units) return -1;
        int r0, r1;
        unit_rows<EPI>(g, u, r0, r1);
        return slot < P / 2 ? r0 : r1;
    }
    const int row = blk * (P / S) + slot / S;
    return row < g.N ? row : -1;
}

// GEMV with every weight load of a wavefront issued up front.  Wavefront w of
// a workgroup of P wavefronts owns one weight row (slot w / S) and the
// K-slice w % S of it: nsteps k-steps of 64 lanes x 16 bytes are split into S
// slices of spw steps.  The weights stay in registers while the routed
// activation rows pass through LDS NR at a time, so each weight byte is read
// once per launch; wide workgroups share one staging of the activations.
// When the host knows the routed row count (n_host >= 0) the weight loads
// start before anything else; otherwise the device count is read first and
// an empty launch returns without touching the weights.  PRO_RMSNORM stages
// gain * x and applies 1/rms(x) to the finished sums.  NP = 2 (K-sliced rows
// too long for one staging in LDS): the activation rows pass through LDS in
// two halves, the first for the wavefronts of slices 0 .. S/2 - 1, the
// second for the others.
template <typename TW, int NR, int PRO, int EPI, int S, int ML, int P, bool TAIL, bool MULTI,
          int NP = 1>
__global__ __launch_bounds__(64 * P) void gemv_kernel(GemvArgs g, int units, int nsteps, int spw,
                                                    int n_host, int rb) {
    static_assert(NP == 1 || (NP == 2 && S % 2 == 0 && !TAIL && PRO != PRO_POOL),
                  "two staging passes split the K-slices of whole k-steps");
    extern __shared__ float xs[];   // [NR][Kp] staged activation rows (Kp = K when NP = 1)
    __shared__ float s_ss[P][NR];
    __shared__ float s_part[P][NR];
    constexpr int V = St<TW>::V;
    constexpr int KS = kWave * V;   // elements per k-step
    constexpr int NT = 64 * P;      // threads per workgroup
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wavefront
    const int K = g.K;
    const int slice = wave % S;
    int n = n_host;
    if (n < 0) {
        n = *g.rows.cnt;
        if (n <= 0) return;
    }
    // MULTI: this workgroup's slice of rb routed rows (grid.y slices)
    const int rbase = MULTI ? (int)blockIdx.y * rb : 0;
    if (MULTI && rbase >= n) return;
    const int row = slot_row<EPI, S, P>(g, blockIdx.x, wave, units);
    const int st0 = slice * spw;
    const int nl = row < 0 ? 0 : max(0, min(spw, nsteps - st0));

    // all weight loads of this wavefront: one base address plus constant
    // offsets; only a K that is not a whole number of k-steps (TAIL) needs
    // clamped addresses for the partial last step.  The weights are read
    // once per launch in whole 1 KB pieces, so they are loaded nontemporal
    // (not kept in the caches): the gate/up GEMV at the Llama-8B shape runs
    // in 37 us instead of 41 us.
    u32x4_t w[ML];
    const TW* wr = (const TW*)g.W + (size_t)max(row, 0) * K + st0 * KS + lane * V;
#pragma unroll
    for (int q = 0; q < ML; ++q) {
        if (q < nl) {
            if (TAIL) {
                const int k = min((st0 + q) * KS + lane * V, K - V) - st0 * KS - lane * V;
                w[q] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(wr + k));
            } else {
                w[q] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(wr + q * KS));
            }
        }
    }

    // MULTI = false: the host guarantees n <= NR, and the single pass keeps
    // the weight registers out of a loop (half the VGPRs, twice the waves)
    const int nloc = MULTI ? min(rb, n - rbase) : n;
    const int groups = MULTI ? (nloc + NR - 1) / NR : 1;
    // k-steps and elements of one staging pass
    const int spp = NP == 1 ? nsteps : (S / NP) * spw;
    const int Kp = NP == 1 ? K : spp * KS;
    for (int gi = 0; gi < groups; ++gi) {
        const int i0 = rbase + gi * NR;
        const int nr = min(NR, rbase + nloc - i0);
        if (MULTI) __syncthreads();  // the previous group is done with xs and s_part
        const TW* gain = (const TW*)g.gain;
        float ssr[NR], acc[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) ssr[r] = acc[r] = 0.f;
#pragma unroll
        for (int pass = 0; pass < NP; ++pass) {
            const int kb = pass * Kp, ke = NP == 1 ? K : min(K, kb + Kp);
            if (pass > 0) __syncthreads();   // the previous pass is done with xs
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                float ss = 0.f;
                if (PRO == PRO_POOL && r < nr) {
                    // router context of sequence b: means of the pool's split sums,
                    // then the newest hidden state
                    const int b = row_seq(g.rows, i0 + r);
                    const int zdim = pooled_dim(g.ctx, g.nkv, g.hd);
                    const float inv_n = 1.0f / (float)(seq_pos(g.pos, g.pos_u, b) + 1);
                    for (int k = tid * 4; k < K; k += NT * 4) {
                        float4 v;
                        if (k < zdim) {
                            v = pooled_feature4(g, b, k, inv_n);
                        } else {
                            v = *reinterpret_cast<const float4*>(g.h + (size_t)b * g.d + (k - zdim));
                        }
                        *reinterpret_cast<float4*>(xs + r * Kp + k) = v;
                    }
                } else if (r < nr) {
                    const float* xr = g.X + (size_t)row_seq(g.rows, i0 + r) * g.ldx;
                    for (int k = kb + tid * V; k < ke; k += NT * V) {
                        float v[V];
#pragma unroll
                        for (int e = 0; e < V; e += 4) {
                            const float4 t = *reinterpret_cast<const float4*>(xr + k + e);
                            v[e] = t.x; v[e + 1] = t.y; v[e + 2] = t.z; v[e + 3] = t.w;
                        }
                        if (PRO == PRO_RMSNORM) {
                            float gv[V];
                            St<TW>::vec(gain + k, gv);
#pragma unroll
                            for (int e = 0; e < V; ++e) { ss += v[e] * v[e]; v[e] *= gv[e]; }
                        }
#pragma unroll
                        for (int e = 0; e < V; e += 4)
                            *reinterpret_cast<float4*>(xs + r * Kp + (k - kb) + e) =
                                make_float4(v[e], v[e + 1], v[e + 2], v[e + 3]);
                    }
                } else {
                    for (int k = kb + tid * 4; k < ke; k += NT * 4)
                        *reinterpret_cast<float4*>(xs + r * Kp + (k - kb)) = make_float4(0.f, 0.f, 0.f, 0.f);
                }
                ssr[r] += ss;
                if (PRO == PRO_RMSNORM && pass == NP - 1) {
                    const float t = wave_sum(ssr[r]);
                    if (lane == 0) s_ss[wave][r] = t;
                }
            }
            __syncthreads();

            // this pass's K-slices: the wavefronts whose slice it staged
            if (NP == 1 || slice / (S / NP) == pass) {
                const float* xw = xs + (st0 - pass * spp) * KS + lane * V;
#pragma unroll
                for (int q = 0; q < ML; ++q) {
                    if (q < nl && (!TAIL || (st0 + q) * KS + lane * V < K)) {
#pragma unroll
                        for (int r = 0; r < NR; ++r) acc[r] += dot16(w[q], xw + r * Kp + q * KS, TW());
                    }
                }
            }
        }   // staging passes
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const float v = wave_sum(acc[r]);
            if (lane == 0) s_part[wave][r] = v;
        }
        __syncthreads();

        float inv[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            inv[r] = 1.f;
            if (PRO == PRO_RMSNORM) {
                float t = 0.f;
                for (int q = 0; q < P; ++q) t += s_ss[q][r];
                inv[r] = 1.0f / sqrtf(t / (float)K + g.eps);
            }
        }
        // epilogues: one (unit or row, routed row) pair per thread
        if (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
            constexpr int UPB = P / 2;
            if (tid < UPB * nr) {
                const int uu = tid / nr, r = tid - uu * nr;
                const int u = blockIdx.x * UPB + uu;
                if (u < units) {
                    float sc = 1.f;
#pragma unroll
                    for (int q = 0; q < NR; ++q) if (q == r) sc = inv[q];
                    int r0, r1;
                    unit_rows<EPI>(g, u, r0, r1);
                    epilogue<TW, EPI>(g, row_seq(g.rows, i0 + r), u, r0, r1, s_part[uu][r] * sc,
                                      s_part[UPB + uu][r] * sc);
                }
            }
        } else {
            constexpr int RPB = P / S;
            if (tid < RPB * nr) {
                const int sl = tid / nr, r = tid - sl * nr;
                const int rw = blockIdx.x * RPB + sl;
                if (rw < g.N) {
                    float v = 0.f, sc = 1.f;
#pragma unroll
                    for (int q = 0; q < S; ++q) v += s_part[sl * S + q][r];
#pragma unroll
                    for (int q = 0; q < NR; ++q) if (q == r) sc = inv[q];
                    epilogue1<TW, EPI>(g, row_seq(g.rows, i0 + r), rw, v * sc);
                }
            }
        }
    }
}

template <typename TW, int NR, int PRO, int EPI, int S, int ML, int P, bool TAIL, bool MULTI,
          int NP = 1>
static hipError_t launch_one(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    constexpr int KS0 = kWave * St<TW>::V;
    const int nsteps0 = (g.K + KS0 - 1) / KS0;
    const int kp = NP == 1 ? g.K : (S / NP) * ((nsteps0 + S - 1) / S) * KS0;
    const size_t lds = (size_t)NR * kp * sizeof(float);
    // devices (one bit each, current device) on which this instantiation
    // may take more than the 64 KB default of dynamic LDS
    static std::atomic<uint64_t> attr_set{0};
    if (lds > 64 * 1024) {
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        const uint64_t bit = 1ull << (dev & 63);
        if (!(attr_set.load(std::memory_order_relaxed) & bit)) {
            // the dispatcher never asks for more than kGemvLds
            e = hipFuncSetAttribute(
                reinterpret_cast<const void*>(&gemv_kernel<TW, NR, PRO, EPI, S, ML, P, TAIL, MULTI, NP>),
                hipFuncAttributeMaxDynamicSharedMemorySize, kGemvLds);
            if (e != hipSuccess) return e;
            attr_set.fetch_or(bit, std::memory_order_relaxed);
        }
    }
    constexpr int KS = kWave * St<TW>::V;
    const int nsteps = (g.K + KS - 1) / KS;
    const int spw = (nsteps + S - 1) / S;
    const int per_wg = (EPI == EPI_SWIGLU || EPI == EPI_QKV) ? P / 2 : P / S;
    const int items = (EPI == EPI_SWIGLU || EPI == EPI_QKV) ? units : g.N;
    const int grid = (items + per_wg - 1) / per_wg;
    // MULTI: the batch's staging groups split into slices over grid.y, so
    // that the launch has about 512 workgroups (each slice loads its weight
    // rows again, mostly from L2): at B = 32 on the Llama-8B shape the
    // Decision Module layer's 128 column workgroups left half the CUs idle
    // (92 us, 52 us with four slices)
    int rb = 0, gy = 1;
    if (MULTI) {
        const int ng = (g.rows.n_max + NR - 1) / NR;   // staging groups of the batch
        int slices = (512 + grid - 1) / grid;
        if (slices > ng) slices = ng;
        rb = (ng + slices - 1) / slices * NR;
        gy = (g.rows.n_max + rb - 1) / rb;
    }
    launch_main(gemv_kernel<TW, NR, PRO, EPI, S, ML, P, TAIL, MULTI, NP>, dim3(grid, gy), dim3(64 * P),
                (uint32_t)lds, s, g, units, nsteps, spw, n_host, rb);
    return hipGetLastError();
}

// K-slices per weight row and loads per lane: 8 loads per lane where the row
// (or a half or quarter of it) allows, else 16.  Two-row units keep S = 1
// (their K is d_model).  Eight wavefronts per workgroup share one staging of
// the activations.
// Shape classes (k-steps of 64 lanes x 16 bytes per weight row):
//   <= 8 steps: one wavefront per row, 8 loads per lane, 8 wavefronts per
//   workgroup (16 for plain rows without a prologue, 12 for QKV units);
//   two-row units with <= 16 steps: 16 loads per lane; single rows with
//   <= 32 (<= 64) steps: quarter rows of <= 8 (16) loads per lane, 16
//   wavefronts per workgroup so four rows share one activation staging.
template <typename TW, int NR, int PRO, int EPI, bool TAIL, bool MULTI>
static hipError_t dispatch_s(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    constexpr int KS = kWave * St<TW>::V;
    const int nsteps = (g.K + KS - 1) / KS;
    if (nsteps <= 8) {
        // workgroup widths that keep the Llama-8B grids whole multiples of
        // the 256 CUs at B = 1: plain rows (the attention output projection)
        // 16 rows per workgroup, 256 workgroups (9.5 -> 8.9 us against 8);
        // QKV units six per workgroup, 512 workgroups (12.2 -> 11.8 us; with
        // 16 wavefronts, 384 workgroups: 12.8 us); SwiGLU units keep four
        // (3584 workgroups; seven per workgroup, 2048: 37 -> 70 us)
        if (EPI == EPI_ADD && PRO == PRO_NONE)
            return launch_one<TW, NR, PRO, EPI, 1, 8, 16, TAIL, MULTI>(g, units, n_host, s);
        if (EPI == EPI_QKV)
            return launch_one<TW, NR, PRO, EPI, 1, 8, 12, TAIL, MULTI>(g, units, n_host, s);
        return launch_one<TW, NR, PRO, EPI, 1, 8, 8, TAIL, MULTI>(g, units, n_host, s);
    }
    if constexpr (std::is_same<TW, float>::value) {
        return hipErrorInvalidValue;   // fp32 rows are at most 8 k-steps (checked at create)
    } else {
        if (EPI == EPI_SWIGLU || EPI == EPI_QKV)
            return launch_one<TW, NR, PRO, EPI, 1, 16, 8, TAIL, MULTI>(g, units, n_host, s);
        if (nsteps <= 32) return launch_one<TW, NR, PRO, EPI, 4, 8, 16, TAIL, MULTI>(g, units, n_host, s);
        return launch_one<TW, NR, PRO, EPI, 4, 16, 16, TAIL, MULTI>(g, units, n_host, s);
    }
}

// A K that is not a whole number of k-steps (TAIL) only occurs for small
// models; MULTI passes are built for one or four staged rows.
template <typename TW, int NR, int PRO, int EPI>
static hipError_t dispatch_tail(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    constexpr int KS = kWave * St<TW>::V;
    constexpr bool kMultiOk = NR != 2;
    const bool multi = g.rows.n_max > NR;
    if constexpr (!kMultiOk) {
        if (multi) return dispatch_tail<TW, 1, PRO, EPI>(g, units, n_host, s);
    }
    if (g.K % KS) {
        // partial last k-step: only rows of at most 8 k-steps (checked at create)
        if (g.K > 8 * KS) return hipErrorInvalidValue;
        if (multi) return launch_one<TW, NR, PRO, EPI, 1, 8, 8, true, kMultiOk>(g, units, n_host, s);
        return launch_one<TW, NR, PRO, EPI, 1, 8, 8, true, false>(g, units, n_host, s);
    }
    if (multi) return dispatch_s<TW, NR, PRO, EPI, false, kMultiOk>(g, units, n_host, s);
    return dispatch_s<TW, NR, PRO, EPI, false, false>(g, units, n_host, s);
}

// Rows longer than one staging in kGemvLds (bf16 K-sliced rows of 41 to 64
// k-steps: the FFN down projection of d_ffn up to 32768) pass through LDS in
// two halves of at most 32 k-steps (64 KB), one routed row at a time.
template <typename TW, int PRO, int EPI>
static hipError_t dispatch_halves(const GemvArgs& g, int units, int n_host, hipStream_t s) {
    if constexpr (std::is_same<TW, float>::value || PRO == PRO_POOL || EPI == EPI_SWIGLU ||
                  EPI == EPI_QKV) {
        return hipErrorInvalidValue;   // K of at most d_model or the router input (checked at create)
    } else {
        constexpr int KS = kWave * St<TW>::V;
        if (g.K % KS || g.K > 64 * KS) return hipErrorInvalidValue;
        if (g.rows.n_max > 1) return launch_one<TW, 1, PRO, EPI, 4, 16, 16, false, true, 2>(g, units, n_host, s);
        return launch_one<TW, 1, PRO, EPI, 4, 16, 16, false, false, 2>(g, units, n_host, s);
    }
}

template <typename TW, int PRO, int EPI>
static hipError_t dispatch_nr(const GemvArgs& g, int units, hipStream_t s) {
    // rows staged per pass: as many as fit in kGemvLds, at most 4
    const size_t row_bytes = (size_t)g.K * sizeof(float);
    const int fit = (int)(kGemvLds / row_bytes);
    const int nr = g.rows.n_max < fit ? g.rows.n_max : fit;
    const int n_host = g.rows.exact ? g.rows.n_max : -1;
    if (fit == 0) return dispatch_halves<TW, PRO, EPI>(g, units, n_host, s);
    if (nr >= 4) return dispatch_tail<TW, 4, PRO, EPI>(g, units, n_host, s);
    if (nr >= 2) return dispatch_tail<TW, 2, PRO, EPI>(g, units, n_host, s);
    return dispatch_tail<TW, 1, PRO, EPI>(g, units, n_host, s);
}

template <typename TW>
static hipError_t dispatch_epi(int pro, int epi, const GemvArgs& g, hipStream_t s) {
    if (epi == EPI_QKV) {
        const int units = (g.nq + 2 * g.nkv) * (g.hd / 2);
        return dispatch_nr<TW, PRO_RMSNORM, EPI_QKV>(g, units, s);
    }
    if (epi == EPI_SWIGLU) return dispatch_nr<TW, PRO_RMSNORM, EPI_SWIGLU>(g, g.f, s);
    if (epi == EPI_BIAS_ACT) return dispatch_nr<TW, PRO_POOL, EPI_BIAS_ACT>(g, g.N, s);
    if (pro == PRO_RMSNORM) return dispatch_nr<TW, PRO_RMSNORM, EPI_ADD>(g, g.N, s);
    return dispatch_nr<TW, PRO_NONE, EPI_ADD>(g, g.N, s);
}

hipError_t launch_gemv(int dtype, int pro, int epi, const GemvArgs& g, hipStream_t s) {
    if (dtype == BUDDY_BF16) return dispatch_epi<bf16_t>(pro, epi, g, s);
    return dispatch_epi<float>(pro, epi, g, s);
}

}  // namespace buddy
