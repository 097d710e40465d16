// Tiled MFMA GEMM for projections over many rows (the prompt tokens of a
// routed prefill): Y = W X^T with v_mfma_f32_16x16x32_bf16, fp32 accumulate,
// and the fused epilogues of the decode paths.
//
// A workgroup computes a 128-weight-row x 128-row tile (for the two-row
// kinds: 64 units, their first rows in tile rows 0..63 and their second rows
// in 64..127), stepping K by 64.  Both operands pass through LDS in MFMA
// fragment order, so each wavefront reads a fragment as one conflict-free
// 16-byte read per lane:
//   A fragment (row tile rt, k-step s): 1 KB at (rt * 2 + s) KB, lane
//     i + 16 q holding tile row 16 rt + i, k = 32 s + 8 q .. + 7;
//   B fragment (column tile ct, k-step s): 1 KB at (ct * 2 + s) KB, copied
//     as is from the activations, which the staging kernel already wrote in
//     B-operand order (16 rows x 32 k per contiguous KB).
// The next K step's tiles travel straight from memory to the idle LDS
// buffer (global_load_lds) while the current one is multiplied (two
// buffers, one barrier per step).  Wavefront w takes
// tile rows of half w / 2 (for two-row kinds: its 32 units' first and second
// rows) and tile columns of half w % 2: 4 x 4 accumulator tiles.
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4.
#include "buddy_internal.h"
#include "epilogue.h"

namespace buddy {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kTileM = 128, kTileN = 128, kTileK = 64;

typedef __attribute__((address_space(1))) const void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// Two workgroups per CU (64 KB of LDS each): registers for two wavefronts
// per SIMD.
template <int EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_kernel(GemvArgs g, int units, int n) {
    constexpr bool kPaired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    // two buffers as separate arrays, so that the compiler can tell the loads
    // into one from the reads of the other and keep the loads in flight
    __shared__ uint4 s_a0[kTileM * kTileK / 8], s_a1[kTileM * kTileK / 8];   // 16 A fragments
    __shared__ uint4 s_b0[kTileN * kTileK / 8], s_b1[kTileN * kTileK / 8];   // 16 B fragments
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int K = g.K, S = K >> 5, nk = K / kTileK;
    const int u0 = blockIdx.x * (kPaired ? kTileM / 2 : kTileM);   // first unit or row
    const int t0 = blockIdx.y * kTileN;                             // first row (token)
    const int last_tile = (n - 1) >> 4;                             // last 16-row column tile

    // Direct global -> LDS loads (each lane's 16 bytes land at the wave's LDS
    // base + 16 lane): wavefront w loads the A fragments of row tiles 2w and
    // 2w + 1 and the B fragments of column tiles 2w and 2w + 1, both k-steps.
    // A fragment lane i + 16 q: tile row 16 rt + i, k = 32 s + 8 q.
    const bf16_t* arow[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int r = 16 * (2 * wave + t) + (lane & 15);
        int row;
        if (kPaired) {
            const int u = min(u0 + (r & 63), units - 1);
            int r0, r1;
            unit_rows<EPI>(g, u, r0, r1);
            row = r < 64 ? r0 : r1;
        } else {
            row = min(u0 + r, units - 1);
        }
        arow[t] = (const bf16_t*)g.W + (size_t)row * K + 8 * (lane >> 4);
    }
    const bf16_t* bfrag[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int c = min((t0 >> 4) + 2 * wave + t, last_tile);   // repeats of the last tile are discarded
        bfrag[t] = g.XB + ((size_t)c * S * 64 + lane) * 8;
    }
    auto issue = [&](int kb, uint4* sa, uint4* sb) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                __builtin_amdgcn_global_load_lds((gptr_t)(arow[t] + kb * kTileK + 32 * s),
                                                 (lptr_t)&sa[((2 * wave + t) * 2 + s) * 64], 16, 0, 0);
                __builtin_amdgcn_global_load_lds((gptr_t)(bfrag[t] + (size_t)(2 * kb + s) * 512),
                                                 (lptr_t)&sb[((2 * wave + t) * 2 + s) * 64], 16, 0, 0);
            }
    };

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    // this wavefront's row tiles: its units' first rows then second rows, or 4 row tiles
    int rts[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) rts[i] = kPaired ? (i < 2 ? 2 * wm + i : 4 + 2 * wm + (i - 2)) : 4 * wm + i;

    auto compute = [&](const uint4* sa, const uint4* sb) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            bf16x8_t a[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a[i] = __builtin_bit_cast(bf16x8_t, sa[(rts[i] * 2 + s) * 64 + lane]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bv[j] = __builtin_bit_cast(bf16x8_t, sb[((4 * wn + j) * 2 + s) * 64 + lane]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bv[j], acc[i][j], 0, 0, 0);
        }
    };

    // Two K steps per trip, one per buffer.  At each step: this step's tiles
    // have landed (own loads, then everyone's at the barrier) and every
    // wavefront is done reading the other buffer, which then receives the
    // next step's tiles while this one is multiplied.
    issue(0, s_a0, s_b0);
    for (int kb = 0; kb < nk; kb += 2) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (kb + 1 < nk) issue(kb + 1, s_a1, s_b1);
        compute(s_a0, s_b0);
        if (kb + 1 >= nk) break;
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (kb + 2 < nk) issue(kb + 2, s_a0, s_b0);
        compute(s_a1, s_b1);
    }

    // epilogue from the accumulators: rows 4 (lane / 16) + e of each tile
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int col = t0 + 64 * wn + 16 * j + (lane & 15);
        if (col >= n) continue;
        const int b = row_seq(g.rows, col);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (kPaired) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int u = u0 + 32 * wm + 16 * i + 4 * (lane >> 4) + e;
                    if (u >= units) continue;
                    int r0, r1;
                    unit_rows<EPI>(g, u, r0, r1);
                    epilogue<bf16_t, EPI>(g, b, u, r0, r1, acc[i][j][e], acc[2 + i][j][e]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = u0 + 64 * wm + 16 * i + 4 * (lane >> 4) + e;
                    if (r < units) epilogue1<bf16_t, EPI>(g, b, r, acc[i][j][e]);
                }
            }
        }
    }
}

template <int EPI>
static hipError_t launch_gemm_epi(const GemvArgs& g, int units, hipStream_t s) {
    constexpr int per = EPI == EPI_SWIGLU || EPI == EPI_QKV ? kTileM / 2 : kTileM;
    const int n = g.rows.n_max;
    const dim3 grid((units + per - 1) / per, (n + kTileN - 1) / kTileN);
    launch_main(gemm_kernel<EPI>, grid, dim3(256), 0, s, g, units, n);
    return hipGetLastError();
}

hipError_t launch_gemm(int pro, int epi, const GemvArgs& g, hipStream_t s) {
    hipError_t e = launch_prep(pro, g, s);
    if (e != hipSuccess) return e;
    if (epi == EPI_QKV) return launch_gemm_epi<EPI_QKV>(g, (g.nq + 2 * g.nkv) * (g.hd / 2), s);
    if (epi == EPI_SWIGLU) return launch_gemm_epi<EPI_SWIGLU>(g, g.f, s);
    if (epi == EPI_BIAS_ACT) return launch_gemm_epi<EPI_BIAS_ACT>(g, g.N, s);
    return launch_gemm_epi<EPI_ADD>(g, g.N, s);
}

}  // namespace buddy
