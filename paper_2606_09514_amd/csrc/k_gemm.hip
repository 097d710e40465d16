// Tiled MFMA GEMM for projections over many rows (the prompt tokens of a
// routed prefill): Y = W X^T with v_mfma_f32_16x16x32_bf16, fp32 accumulate,
// and the fused epilogues of the decode paths.
//
// A workgroup of WM x WN wavefronts computes a (16 WM TI weight rows) x
// (16 WN TJ rows) tile, each wavefront TI x TJ accumulator tiles of 16 x 16,
// stepping K by 32.  For the two-row kinds (SwiGLU, QKV) the weight rows of
// a tile are 8 WM TI units: their first rows in the upper half of the row
// tiles and their second rows in the lower half, and each wavefront holds
// the first and second rows of the same units.  Two shapes:
//   128 x 128 (2 x 2 wavefronts of 64 x 64), two workgroups per CU;
//   256 x 256 (2 x 4 wavefronts of 128 x 64), one workgroup per CU, which
//     halves the bytes each CU fetches per flop (the loads through the
//     texture path, not the MFMA, bound the smaller tile).
// Both operands pass through LDS in MFMA fragment order, so each wavefront
// reads a fragment as one conflict-free 16-byte read per lane:
//   A fragment (row tile rt): 1 KB at rt KB of the step's buffer, lane
//     i + 16 q holding tile row 16 rt + i, k = 8 q .. + 7 of the step;
//   B fragment (column tile ct): 1 KB after the A fragments, copied as is
//     from the activations, which the staging kernel already wrote in
//     B-operand order (16 rows x 32 k per contiguous KB).
// Tiles travel straight from memory to LDS (global_load_lds) three K steps
// ahead of the multiply (four buffers, one barrier per step); each row
// tile's MFMAs start as soon as its own fragment read has landed.
//   D[i][j] (16 x 16): lane j + 16 (i / 4), element i % 4.
#include "buddy_internal.h"
#include "epilogue.h"

namespace buddy {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(1))) const void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

constexpr int kTileK = 32;
constexpr int kFragBytes = 1024;                 // one 16 x 32 bf16 fragment
constexpr int kBufs = 4;                         // K steps in LDS, three ahead

// s_waitcnt operand: at most n vector-memory operations outstanding, other
// counters unconstrained (gfx9 encoding: vmcnt low bits 3:0 and high bits
// 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int vmcnt_at_most(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Fragment reads from LDS: 16 bytes at address a (or b) plus immediate
// offsets, issued without a wait.  Written as asm so that the compiler, which
// cannot tell the direct-to-LDS loads into the other buffers from these
// reads, does not make them wait for every load in flight.  LDS reads return
// in issue order, so after a step's reads (the B fragments, then the A
// fragments in row-tile order) lgkmcnt(n) means that all but the last n have
// landed, and the MFMAs of row tile i can start once TI - 1 - i reads remain
// (lds_wait): the first MFMAs wait for 4 + 1 reads, not for all of them.
// Other counted operations the compiler issues only make such a wait longer.
// Until its wait, the compiler believes a read's registers written: the wait
// takes them as operands it modifies, so that nothing reads them earlier.
template <int O0, int O1, int O2, int O3>
__device__ __forceinline__ void lds_issue4(uint32_t a, u32x4_t* x) {
    asm volatile(
        "ds_read_b128 %0, %4 offset:%5\n\t"
        "ds_read_b128 %1, %4 offset:%6\n\t"
        "ds_read_b128 %2, %4 offset:%7\n\t"
        "ds_read_b128 %3, %4 offset:%8"
        : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3])
        : "v"(a), "i"(O0), "i"(O1), "i"(O2), "i"(O3)
        : "memory");
}
// B fragments at b + 0, 1, 2, 3 KB, then A fragments at a + O0 .. O3
template <int O0, int O1, int O2, int O3>
__device__ __forceinline__ void lds_issue8(uint32_t a, uint32_t b, u32x4_t* x, u32x4_t* y) {
    asm volatile(
        "ds_read_b128 %4, %9 offset:0\n\t"
        "ds_read_b128 %5, %9 offset:1024\n\t"
        "ds_read_b128 %6, %9 offset:2048\n\t"
        "ds_read_b128 %7, %9 offset:3072\n\t"
        "ds_read_b128 %0, %8 offset:%10\n\t"
        "ds_read_b128 %1, %8 offset:%11\n\t"
        "ds_read_b128 %2, %8 offset:%12\n\t"
        "ds_read_b128 %3, %8 offset:%13"
        : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3]), "=&v"(y[0]), "=&v"(y[1]),
          "=&v"(y[2]), "=&v"(y[3])
        : "v"(a), "v"(b), "i"(O0), "i"(O1), "i"(O2), "i"(O3)
        : "memory");
}
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t& r) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(r) : "i"(N));
}
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t& r, u32x4_t* y) {
    asm volatile("s_waitcnt lgkmcnt(%5)"
                 : "+v"(r), "+v"(y[0]), "+v"(y[1]), "+v"(y[2]), "+v"(y[3])
                 : "i"(N));
}

// One K step's MFMAs, row tile I onwards: each row tile after its own read
// (and, for the first, the B fragments') has landed.
template <int I, int TI, int TJ>
__device__ __forceinline__ void mfma_rows(f32x4_t (&acc)[TI][TJ], u32x4_t* a, u32x4_t* bv) {
    if constexpr (I == 0)
        lds_wait<TI - 1>(a[0], bv);
    else
        lds_wait<TI - 1 - I>(a[I]);
#pragma unroll
    for (int j = 0; j < TJ; ++j)
        acc[I][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8_t, a[I]), __builtin_bit_cast(bf16x8_t, bv[j]), acc[I][j], 0,
            0, 0);
    // keep the next row tile's wait behind these MFMAs (the scheduler would
    // otherwise gather the waits ahead of them)
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (I + 1 < TI) mfma_rows<I + 1>(acc, a, bv);
}

template <int WM, int WN, int TI, int TJ>
struct GemmShape {
    static constexpr int kWaves = WM * WN, kThreads = 64 * kWaves;
    static constexpr int kRowTiles = WM * TI, kColTiles = WN * TJ;
    static constexpr int kRows = 16 * kRowTiles, kCols = 16 * kColTiles;
    static constexpr int kBufBytes = (kRowTiles + kColTiles) * kFragBytes;
    // fragments each wavefront loads per K step
    static constexpr int kALoads = kRowTiles / kWaves, kBLoads = kColTiles / kWaves;
    static_assert(kRowTiles % kWaves == 0 && kColTiles % kWaves == 0, "even load split");
    static_assert(kBufs * kBufBytes <= 128 * 1024, "LDS");
    static_assert(TJ == 4 && (TI == 4 || TI == 8), "wavefront tile");
};

template <int EPI, int WM, int WN, int TI, int TJ>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_kernel(GemvArgs g, int units, int n, float* part, int ubase) {
    using Sh = GemmShape<WM, WN, TI, TJ>;
    constexpr bool kPaired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    __shared__ __attribute__((aligned(16))) char s_buf[kBufs * Sh::kBufBytes];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave % WN;
    // split K (part != null): workgroup z takes K steps [z nk, (z + 1) nk)
    // and writes its fp32 sums to part[z][row][unit] for a separate add
    const int K = g.K, S = K >> 5, nk = K / kTileK / gridDim.z, k0 = blockIdx.z * nk;
    const int u0 = ubase + blockIdx.x * (kPaired ? Sh::kRows / 2 : Sh::kRows);   // first unit or row
    const int t0 = blockIdx.y * Sh::kCols;                               // first row (token)
    const int last_tile = (n - 1) >> 4;                                   // last 16-row column tile

    // Direct global -> LDS loads (each lane's 16 bytes land at the wave's LDS
    // base + 16 lane): wavefront w loads row tiles kALoads w .. and column
    // tiles kBLoads w .. of every step.
    // A fragment lane i + 16 q: tile row 16 rt + i, k = 8 q of the step.
    const bf16_t* arow[Sh::kALoads];
#pragma unroll
    for (int t = 0; t < Sh::kALoads; ++t) {
        const int r = 16 * (Sh::kALoads * wave + t) + (lane & 15);
        int row;
        if (kPaired) {
            const int half = Sh::kRows / 2;
            const int u = min(u0 + (r % half), units - 1);
            int r0, r1;
            unit_rows<EPI>(g, u, r0, r1);
            row = r < half ? r0 : r1;
        } else {
            row = min(u0 + r, units - 1);
        }
        arow[t] = (const bf16_t*)g.W + (size_t)row * K + 8 * (lane >> 4);
    }
    const bf16_t* bfrag[Sh::kBLoads];
#pragma unroll
    for (int t = 0; t < Sh::kBLoads; ++t) {
        const int c = min((t0 >> 4) + Sh::kBLoads * wave + t, last_tile);   // repeats of the last tile are discarded
        bfrag[t] = g.XB + ((size_t)c * S * 64 + lane) * 8;
    }
    // one load per fragment; steps past the end reload the last one into a
    // buffer that is not read again
    auto issue = [&](int kb) {
        const int kc = k0 + min(kb, nk - 1);
        char* base = s_buf + (kb % kBufs) * Sh::kBufBytes;
#pragma unroll
        for (int t = 0; t < Sh::kALoads; ++t)
            __builtin_amdgcn_global_load_lds((gptr_t)(arow[t] + kc * kTileK),
                                             (lptr_t)(base + (Sh::kALoads * wave + t) * kFragBytes),
                                             16, 0, 0);
#pragma unroll
        for (int t = 0; t < Sh::kBLoads; ++t)
            __builtin_amdgcn_global_load_lds(
                (gptr_t)(bfrag[t] + (size_t)kc * 512),
                (lptr_t)(base + (Sh::kRowTiles + Sh::kBLoads * wave + t) * kFragBytes), 16, 0, 0);
    };
    constexpr int kLoads = Sh::kALoads + Sh::kBLoads;   // per wavefront and step

    f32x4_t acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    // this wavefront's fragments within a buffer.  Row tiles: paired, its
    // units' first rows (TI/2 tiles from wm TI/2) and second rows (the same
    // TI/2 tiles of the lower half); otherwise TI tiles from wm TI.  Column
    // tiles: TJ from wn TJ.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lptr_t)s_buf;
    const uint32_t a_off = lds0 + lane * 16 + (kPaired ? wm * TI / 2 : wm * TI) * kFragBytes;
    const uint32_t b_off = lds0 + lane * 16 + (Sh::kRowTiles + wn * TJ) * kFragBytes;
    constexpr int kSecond = kPaired ? Sh::kRowTiles / 2 - TI / 2 : 0;   // gap to the second rows
    constexpr int F = kFragBytes;

    // At step kb: wait until only the loads of steps kb + 1 and kb + 2 are
    // outstanding, barrier (every wavefront's loads of step kb have landed
    // and every wavefront has read step kb - 1's buffer), refill that buffer
    // with step kb + 3, multiply step kb.
    issue(0);
    issue(1);
    issue(2);
    for (int kb = 0; kb < nk; ++kb) {
        __builtin_amdgcn_s_waitcnt(vmcnt_at_most(2 * kLoads));
        // a plain barrier: __syncthreads() would also wait for every load in
        // flight (its fence covers the direct-to-LDS writes)
        asm volatile("s_barrier" ::: "memory");
        issue(kb + 3);
        const uint32_t sb = (kb % kBufs) * Sh::kBufBytes;
        u32x4_t a[TI], bv[TJ];
        if constexpr (TI == 4) {
            lds_issue8<0, F, (2 + kSecond) * F, (3 + kSecond) * F>(a_off + sb, b_off + sb, a, bv);
        } else {
            lds_issue8<0, F, 2 * F, 3 * F>(a_off + sb, b_off + sb, a, bv);
            lds_issue4<(4 + kSecond) * F, (5 + kSecond) * F, (6 + kSecond) * F, (7 + kSecond) * F>(
                a_off + sb, a + 4);
        }
        mfma_rows<0>(acc, a, bv);
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));   // the reloads past the end

    if (part) {   // split K (single-row kinds): 4 consecutive units per lane, one 16-byte store
        float* pz = part + (size_t)blockIdx.z * n * units;
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            const int col = t0 + 16 * (wn * TJ + j) + (lane & 15);
            if (col >= n) continue;
#pragma unroll
            for (int i = 0; i < TI; ++i) {
                const int r = u0 + 16 * (wm * TI + i) + 4 * (lane >> 4);
                if (r < units)
                    *reinterpret_cast<float4*>(pz + (size_t)col * units + r) =
                        make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
            }
        }
        return;
    }

    // epilogue from the accumulators: rows 4 (lane / 16) + e of each tile
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
        const int col = t0 + 16 * (wn * TJ + j) + (lane & 15);
        if (col >= n) continue;
        const int b = row_seq(g.rows, col);
        if (EPI == EPI_SWIGLU && g.xb_out) {
            // SiLU(gate) * up of 4 consecutive units as bf16 into the next
            // projection's staging: one 8-byte store (f % 8 == 0)
#pragma unroll
            for (int i = 0; i < TI / 2; ++i) {
                const int ub = u0 + 16 * (wm * TI / 2 + i) + 4 * (lane >> 4);
                if (ub >= units) continue;
                float m[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) m[e] = swiglu(acc[i][j][e], acc[TI / 2 + i][j][e]);
                *reinterpret_cast<uint2*>(g.xb_out + xb_index(col, ub, units)) =
                    make_uint2(pack_bf16x2(m[0], m[1]), pack_bf16x2(m[2], m[3]));
            }
            continue;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (kPaired) {
#pragma unroll
                for (int i = 0; i < TI / 2; ++i) {
                    const int u = u0 + 16 * (wm * TI / 2 + i) + 4 * (lane >> 4) + e;
                    if (u >= units) continue;
                    int r0, r1;
                    unit_rows<EPI>(g, u, r0, r1);
                    epilogue<bf16_t, EPI>(g, b, u, r0, r1, acc[i][j][e], acc[TI / 2 + i][j][e]);
                }
            } else {
#pragma unroll
                for (int i = 0; i < TI; ++i) {
                    const int r = u0 + 16 * (wm * TI + i) + 4 * (lane >> 4) + e;
                    if (r < units) epilogue1<bf16_t, EPI>(g, b, r, acc[i][j][e]);
                }
            }
        }
    }
}

// ----------------------------------------------------------- staging

// Activation staging for the tiled GEMM: the rows of a 16-row column tile
// as bf16 in B-operand fragment order, with the RMSNorm folded in
// (PRO_RMSNORM) or a plain conversion (PRO_NONE).  One workgroup of 16
// wavefronts per tile (and, for PRO_NONE, per chunk of kPrepChunk columns):
// wavefront w converts row w of the tile into LDS (rows padded by 16 bytes,
// so the fragment reads below are conflict-free), then every thread writes
// whole 16-byte pieces of the tile's fragments, consecutive threads to
// consecutive addresses.  For the RMSNorm the row's sum of squares comes
// first, over all of K.
constexpr int kPrepChunk = 2048;                 // columns per LDS pass
constexpr int kPrepPitch = kPrepChunk * 2 + 16;  // bytes per LDS row

template <int PRO>
__global__ __launch_bounds__(1024) void prep_tile_kernel(GemvArgs g, int n) {
    __shared__ __attribute__((aligned(16))) char s_rows[16 * kPrepPitch];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = blockIdx.x, K = g.K, S = K >> 5;
    const int i = 16 * tile + w;                      // this wavefront's row (list index)
    const bool live = i < n;
    const float* x = g.X + (size_t)(live ? row_seq(g.rows, i) : 0) * g.ldx;
    float inv = 1.f;
    if (PRO == PRO_RMSNORM) {
        float ss = 0.f;
        if (live)
            for (int k = 4 * lane; k < K; k += 256) {
                const float4 v = *reinterpret_cast<const float4*>(x + k);
                ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
            }
        ss = wave_sum(ss);
        inv = 1.0f / sqrtf(ss / (float)K + g.eps);
    }
    const int c_first = PRO == PRO_RMSNORM ? 0 : blockIdx.y * kPrepChunk;
    const int c_end = PRO == PRO_RMSNORM ? K : min(K, c_first + kPrepChunk);
    for (int c0 = c_first; c0 < c_end; c0 += kPrepChunk) {
        const int kc = min(kPrepChunk, K - c0);
        char* row = s_rows + w * kPrepPitch;
        for (int k = 4 * lane; k < kc; k += 256) {
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (live) {
                v = *reinterpret_cast<const float4*>(x + c0 + k);
                if (PRO == PRO_RMSNORM) {
                    const bf16_t* gp = (const bf16_t*)g.gain + c0 + k;
                    v.x *= inv * bf2f(gp[0]); v.y *= inv * bf2f(gp[1]);
                    v.z *= inv * bf2f(gp[2]); v.w *= inv * bf2f(gp[3]);
                }
            }
            *reinterpret_cast<uint2*>(row + 2 * k) =
                make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
        }
        __syncthreads();
        // fragment (k-step s, lane L): row L % 16, columns 32 s + 8 (L / 16) .. + 7
        const int nfrag = (kc >> 5) * 64;
        for (int f = tid; f < nfrag; f += 1024) {
            const int sl = f >> 6, L = f & 63;
            const uint4 v = *reinterpret_cast<const uint4*>(s_rows + (L & 15) * kPrepPitch +
                                                           2 * (32 * sl + 8 * (L >> 4)));
            const size_t frag = ((size_t)tile * S + (c0 >> 5) + sl) * 64 + L;
            *reinterpret_cast<uint4*>(g.XB + frag * 8) = v;
        }
        __syncthreads();
    }
}

static hipError_t launch_prep_tiles(int pro, const GemvArgs& g, hipStream_t s) {
    const int n = g.rows.n_max, tiles = (n + 15) / 16;
    if (pro == PRO_RMSNORM) {
        prep_tile_kernel<PRO_RMSNORM><<<dim3(tiles, 1), 1024, 0, s>>>(g, n);
    } else if (pro == PRO_NONE) {
        const int chunks = (g.K + kPrepChunk - 1) / kPrepChunk;
        prep_tile_kernel<PRO_NONE><<<dim3(tiles, chunks), 1024, 0, s>>>(g, n);
    } else {
        return launch_prep(pro, g, s);
    }
    return hipGetLastError();
}

constexpr int kCUs = 256;   // compute units of the MI355X: one round of 256 x 256 tiles

// units (weight rows, or row pairs for the two-row kinds) per row tile
template <int EPI, int WM, int WN, int TI, int TJ>
constexpr int tile_units() {
    return EPI == EPI_SWIGLU || EPI == EPI_QKV ? GemmShape<WM, WN, TI, TJ>::kRows / 2
                                               : GemmShape<WM, WN, TI, TJ>::kRows;
}

template <int EPI, int WM, int WN, int TI, int TJ>
static dim3 gemm_grid(int units, int n) {
    constexpr int per = tile_units<EPI, WM, WN, TI, TJ>();
    return dim3((units + per - 1) / per, (n + GemmShape<WM, WN, TI, TJ>::kCols - 1) /
                                             GemmShape<WM, WN, TI, TJ>::kCols);
}

// Units [ubase, uend) of the projection (uend = -1: to the last one).
template <int EPI, int WM, int WN, int TI, int TJ>
static void gemm_launch(const GemvArgs& g, int units, int n, hipStream_t s, float* part = nullptr,
                        int splits = 1, int ubase = 0, int uend = -1) {
    dim3 grid = gemm_grid<EPI, WM, WN, TI, TJ>((uend < 0 ? units : uend) - ubase, n);
    grid.z = splits;
    launch_main(gemm_kernel<EPI, WM, WN, TI, TJ>, grid, dim3(GemmShape<WM, WN, TI, TJ>::kThreads),
                0, s, g, units, n, part, ubase);
}

// The last round of a 256 x 256 grid that does not fill the CUs: the units
// of the row tiles that fill whole rounds stay on 256 x 256 tiles, and the
// rest go to a second launch of 128 x 128 tiles when those take one round
// of two workgroups per CU (half the flops of a large round, at about 0.8
// of the large tile's rate per flop measured on the MI355X: some 0.6 of its
// time) instead of a partly idle round of the large one.  Returns the
// first unit of the 128 x 128 launch, or units for none.  The outputs are
// the same bit for bit: every output sums its K steps in the same order in
// either tile.
template <int EPI>
static int gemm_tail_units(int units, int n) {
    const dim3 big = gemm_grid<EPI, 2, 4, 8, 4>(units, n);
    const int tiles = big.x * big.y, whole = tiles / kCUs * kCUs;
    if (whole == tiles || whole == 0) return units;
    const int ubig = whole / big.y * tile_units<EPI, 2, 4, 8, 4>();
    const dim3 small = gemm_grid<EPI, 2, 2, 4, 4>(units - ubig, n);
    return small.x * small.y <= 2 * kCUs ? ubig : units;
}

// Residual add of the split-K partial sums: Y[row] += part[0] + part[1]
// (fixed order), four units per thread.
__global__ __launch_bounds__(256) void splitk_add_kernel(GemvArgs g, int units, int n,
                                                         const float* part) {
    const int q = units >> 2;
    for (size_t t = (size_t)blockIdx.x * 256 + threadIdx.x; t < (size_t)n * q;
         t += (size_t)gridDim.x * 256) {
        const int col = (int)(t / q), r = 4 * (int)(t - (size_t)col * q);
        const float4 a = *reinterpret_cast<const float4*>(part + (size_t)col * units + r);
        const float4 b = *reinterpret_cast<const float4*>(part + ((size_t)n + col) * units + r);
        float* y = g.Y + (size_t)row_seq(g.rows, col) * g.ldy + r;
        float4 v = *reinterpret_cast<float4*>(y);
        v.x += a.x + b.x; v.y += a.y + b.y; v.z += a.z + b.z; v.w += a.w + b.w;
        *reinterpret_cast<float4*>(y) = v;
    }
}

// Tile choice (automatic): 256 x 256 where it still gives the CUs two
// rounds of workgroups, else 128 x 128 (two per CU).  A 256 x 128 tile with
// one wavefront per SIMD was slower than 128 x 128 on the 4096-row
// projections (measured).
template <int EPI>
static hipError_t launch_gemm_epi(const GemvArgs& g, int units, int tile, float* part,
                                  hipStream_t s) {
    const int n = g.rows.n_max;
    const dim3 big = gemm_grid<EPI, 2, 4, 8, 4>(units, n);
    // split K in two for residual-add projections whose 256 x 256 grid would
    // leave CUs idle but fills them when doubled (O and down at prefill sizes)
    const bool split_ok = EPI == EPI_ADD && part && (g.K / kTileK) % 2 == 0 && units % 4 == 0;
    const bool split = split_ok && (tile == BUDDY_GEMM_TILE_256_SPLIT ||
                                    (tile == BUDDY_GEMM_TILE_AUTO && big.x * big.y < 2 * kCUs &&
                                     2 * big.x * big.y >= kCUs));
    if (split) {
        gemm_launch<EPI, 2, 4, 8, 4>(g, units, n, s, part, 2);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const size_t work = (size_t)n * (units / 4);
        const int grid = (int)((work + 255) / 256 < 4096 ? (work + 255) / 256 : 4096);
        splitk_add_kernel<<<grid, 256, 0, s>>>(g, units, n, part);
    } else if (tile == BUDDY_GEMM_TILE_256 || tile == BUDDY_GEMM_TILE_256_SPLIT) {
        gemm_launch<EPI, 2, 4, 8, 4>(g, units, n, s);
    } else if (tile == BUDDY_GEMM_TILE_AUTO && big.x * big.y >= 2 * kCUs) {
        const int ubig = gemm_tail_units<EPI>(units, n);
        gemm_launch<EPI, 2, 4, 8, 4>(g, units, n, s, nullptr, 1, 0, ubig);
        if (ubig < units) gemm_launch<EPI, 2, 2, 4, 4>(g, units, n, s, nullptr, 1, ubig);
    } else {
        gemm_launch<EPI, 2, 2, 4, 4>(g, units, n, s);
    }
    return hipGetLastError();
}

hipError_t launch_gemm(int pro, int epi, const GemvArgs& g, int tile, float* part, hipStream_t s) {
    if (pro != PRO_STAGED) {
        hipError_t e = launch_prep_tiles(pro, g, s);
        if (e != hipSuccess) return e;
    }
    if (epi == EPI_QKV)
        return launch_gemm_epi<EPI_QKV>(g, (g.nq + 2 * g.nkv) * (g.hd / 2), tile, nullptr, s);
    if (epi == EPI_SWIGLU) return launch_gemm_epi<EPI_SWIGLU>(g, g.f, tile, nullptr, s);
    if (epi == EPI_BIAS_ACT) return launch_gemm_epi<EPI_BIAS_ACT>(g, g.N, tile, nullptr, s);
    return launch_gemm_epi<EPI_ADD>(g, g.N, tile, part, s);
}

}  // namespace buddy
