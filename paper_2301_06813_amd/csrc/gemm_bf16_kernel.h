// gemm_bf16_kernel.h -- bf16 MFMA GEMM for the local matmul of an SBP linear
// layer on CDNA4 (gfx950).
//
// Computes C[i][j] = sum_k A(i,k) B(k,j) for an m x n output over a reduction
// of length k, with fp32 accumulation, where each operand is a strided view
// read in place:
//   A_KMAJ:  A(i,k) = A[i*lda + k]   else  A(i,k) = A[k*lda + i]
//   B_KMAJ:  B(k,j) = B[j*ldb + k]   else  B(k,j) = B[k*ldb + j]
// The three local products of an SBP linear (AutoDDL Sec. 4.2 local matmul
// and its backward) are the orientations
//   forward       Y  = X  W     A k-major,  B n-major
//   backward-data dX = dY W^T   A k-major,  B k-major
//   backward-wt   dW = X^T dY   A m-major,  B n-major.
//
// Design (one workgroup = 4 waves of 64 lanes = 256 threads):
//   * Output tile BM x BN, reduction step BK = 64; each wave owns a
//     (BM/2) x (BN/2) quarter computed with v_mfma_f32_32x32x16_bf16.
//   * Both operand tiles live in LDS "k-contiguous": one 128-byte row of 64
//     bf16 reduction values per output row/column, cut into eight 16-byte
//     chunks whose position is XOR-swizzled by the row index, so that the
//     16-byte MFMA fragment reads and the tile writes are free of bank
//     conflicts.
//   * k-major operands are loaded as 16-byte vectors along k. m/n-major
//     operands are loaded as 16-byte vectors along m/n, KB rows at a time,
//     and transposed in registers (16-bit lane packing) before the LDS
//     write, so both orientations share one LDS layout and one inner loop.
//   * Register prefetch + two LDS buffers: the global loads of step t+1 are
//     in flight while step t runs on the MFMA units; one barrier per step.
//   * Split reduction (splits > 1): each workgroup reduces one k-range and
//     writes its fp32 partial tile to slice `split` of a workspace laid out
//     like the output; a second kernel (split_reduce_kernel) adds the slices
//     in split order -- deterministic -- and writes the output. Kernel
//     boundaries order the two, so no device-scope fences or atomics are
//     needed (on gfx950 such fences write back and invalidate the XCD's L2).
//   * Workgroup -> tile order is XCD-aware: consecutive workgroup ids go to
//     different XCDs, so ids are remapped to give each XCD a contiguous run
//     of tiles (shared A rows / B columns stay in that XCD's L2).
//   * Edges: any m, n, k (including k = 0, which writes zeros) and any
//     element alignment. Vector loads are used only where the whole 16-byte
//     vector is inside the operand and the operand's base and leading
//     dimension keep it 16-byte aligned (a uniform per-launch flag); other
//     vectors are assembled from masked element loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm.h"

namespace sbpk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 64;          // reduction step (elements)
constexpr int NT = 256;         // threads per workgroup
constexpr int ROWB = BK * 2;    // bytes per LDS row

struct GemmArgs {
    const uint16_t *A;
    const uint16_t *B;
    void *C;
    int64_t lda, ldb, ldc;
    int32_t m, n, k;
    int32_t tiles_m, tiles_n;
    int32_t splits;             // reduction splits (>= 1)
    int32_t kchunk;             // reduction elements per split (a multiple of 64)
    float *ws;                  // split partials: splits slices of m x n floats,
                                // row stride partial_ld(n)
    int32_t vec_a, vec_b;       // operand base and ld allow aligned 16-byte loads
    int32_t vec_c4, vec_c8;     // C's base and ldc allow aligned 16-byte stores of
                                // 4 fp32 / 8 bf16 elements
    int32_t accumulate;         // fp32 C: add the product to C's contents
    // Batched products (the attention core): nbatch = batches x heads
    // independent m x n x k products; product z = b * heads + h reads A at
    // A + b sa_b + h sa_h (elements), likewise B, and writes C at
    // C + b sc_b + h sc_h. nbatch = 1 for a single product. Batched launches
    // never split the reduction.
    int32_t nbatch, heads;
    int64_t sa_b, sa_h, sb_b, sb_h, sc_b, sc_h;
};

// Arguments of the pipelined kernel's shifted form, for operands that start
// inside a 16-byte block (a shard view at an element offset that is not a
// multiple of 8) or whose contiguous extent is not a multiple of 8: A and B
// point at the 16-byte boundary at or below the view, and the kernel works
// in an index space shifted by the view's offset within that block --
// output rows by sm (an m-major A), output columns by sn (an n-major B), the
// reduction by sk (both operands k-major, with the same offset). Kernel row
// i is output row i - sm, and so on; reduction index kk is valid for
// sk <= kk < sk + k. kmask: the first and last reduction chunks hold
// elements outside that range (an offset, or k not a multiple of 8), which
// the kernel zeroes in LDS before those steps. The unshifted kernels take
// plain GemmArgs, and the accessors below give them zero shifts.
struct GemmArgsShift : GemmArgs {
    int32_t sm, sn, sk, kmask;
};
__device__ __forceinline__ int shift_m(const GemmArgs &) { return 0; }
__device__ __forceinline__ int shift_n(const GemmArgs &) { return 0; }
__device__ __forceinline__ int shift_k(const GemmArgs &) { return 0; }
__device__ __forceinline__ int kmask_of(const GemmArgs &) { return 0; }
__device__ __forceinline__ int shift_m(const GemmArgsShift &g) { return g.sm; }
__device__ __forceinline__ int shift_n(const GemmArgsShift &g) { return g.sn; }
__device__ __forceinline__ int shift_k(const GemmArgsShift &g) { return g.sk; }
__device__ __forceinline__ int kmask_of(const GemmArgsShift &g) { return g.kmask; }

// Operand and output bases of batch item z (uniform per work item).
template <bool OUT_F32>
__device__ __forceinline__ void batch_bases(const GemmArgs &g, int z, const uint16_t **A,
                                            const uint16_t **B, void **C) {
    *A = g.A;
    *B = g.B;
    *C = g.C;
    if (g.nbatch > 1) {
        const int64_t zb = z / g.heads, zh = z % g.heads;
        *A += zb * g.sa_b + zh * g.sa_h;
        *B += zb * g.sb_b + zh * g.sb_h;
        *C = static_cast<char *>(g.C) + (zb * g.sc_b + zh * g.sc_h) * (OUT_F32 ? 4 : 2);
    }
}

// Byte offset of 16-byte chunk c (0..7) of LDS row `row`.
__device__ __forceinline__ uint32_t lds_off(int row, int c) {
    int sw = (row & 7) ^ ((row >> 3) & 7);
    return (uint32_t)(row * ROWB + ((c ^ sw) << 4));
}

// Eight consecutive bf16 of a row starting at p; `valid` of them are inside
// the operand (<= 0: none). Whole in-bounds vectors use one 16-byte load when
// the operand's base and leading dimension make it 16-byte aligned (vec).
__device__ __forceinline__ u32x4 load8(const uint16_t *p, int valid, bool vec) {
    if (vec && valid >= 8) {
        return *reinterpret_cast<const u32x4 *>(p);
    }
    uint32_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = (i < valid) ? (uint32_t)p[i] : 0u;
    u32x4 v;
    v[0] = e[0] | (e[1] << 16);
    v[1] = e[2] | (e[3] << 16);
    v[2] = e[4] | (e[5] << 16);
    v[3] = e[6] | (e[7] << 16);
    return v;
}

__device__ __forceinline__ uint32_t half16(const u32x4 &v, int c) {
    uint32_t w = v[c >> 1];
    return (c & 1) ? (w >> 16) : (w & 0xffffu);
}

// --------------------------------------------------------------------------
// Operand tile loaders. A tile covers BMN rows of the output dimension
// (m for A, n for B) and BK reduction values, starting at (mn0, k0).
// mn_lim / k_lim are the exclusive bounds of the operand.
// --------------------------------------------------------------------------

// Storage contiguous along k: element (mn, k) at base[mn*ld + k].
template <int BMN>
struct KMajorTile {
    static constexpr int NV = BMN * BK / 8 / NT;   // 16-byte vectors per thread
    u32x4 v[NV];

    // Whole tile inside the operand and 16-byte aligned: plain vector loads.
    __device__ __forceinline__ void load_full(const uint16_t *base, int64_t ld, int mn0, int k0,
                                              int tid) {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            int q = i * NT + tid;
            const uint16_t *p = base + (int64_t)(mn0 + (q >> 3)) * ld + (k0 + (q & 7) * 8);
            v[i] = *reinterpret_cast<const u32x4 *>(p);
        }
    }

    // Edge or unaligned tile: masked loads, zero outside the operand.
    __device__ __forceinline__ void load_edge(const uint16_t *base, int64_t ld, int mn0, int mn_lim,
                                           int k0, int k_lim, int tid, bool vec) {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            int q = i * NT + tid;
            int row = q >> 3;
            int kc = q & 7;
            int mn = mn0 + row;
            int kk = k0 + kc * 8;
            int valid = (mn < mn_lim) ? (k_lim - kk) : 0;
            const uint16_t *p = base + (int64_t)(mn < mn_lim ? mn : 0) * ld + (valid > 0 ? kk : 0);
            v[i] = load8(p, valid, vec);
        }
    }

    __device__ __forceinline__ void store(char *lds, int tid) const {
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            int q = i * NT + tid;
            int row = q >> 3;
            int kc = q & 7;
            *reinterpret_cast<u32x4 *>(lds + lds_off(row, kc)) = v[i];
        }
    }
};

// Storage contiguous along m/n: element (mn, k) at base[k*ld + mn].
// Each thread owns a KB x 8 block (KB reduction rows x 8 output indices),
// loaded as KB 16-byte row vectors and written to LDS transposed.
template <int BMN>
struct MNMajorTile {
    static constexpr int KB = BMN * BK / 8 / NT;   // 8, 4 or 2
    static constexpr int NMB = BMN / 8;            // 8-wide blocks per k-row
    static_assert(KB == 8 || KB == 4 || KB == 2, "unsupported tile");
    u32x4 v[KB];

    __device__ __forceinline__ void load_full(const uint16_t *base, int64_t ld, int mn0, int k0,
                                              int tid) {
        const int mnb = tid % NMB;
        const int kb = tid / NMB;
        const uint16_t *p = base + (int64_t)(k0 + kb * KB) * ld + (mn0 + mnb * 8);
#pragma unroll
        for (int r = 0; r < KB; ++r) v[r] = *reinterpret_cast<const u32x4 *>(p + (int64_t)r * ld);
    }

    __device__ __forceinline__ void load_edge(const uint16_t *base, int64_t ld, int mn0, int mn_lim,
                                           int k0, int k_lim, int tid, bool vec) {
        int mnb = tid % NMB;
        int kb = tid / NMB;
        int mn = mn0 + mnb * 8;
#pragma unroll
        for (int r = 0; r < KB; ++r) {
            int kk = k0 + kb * KB + r;
            int valid = (kk < k_lim) ? (mn_lim - mn) : 0;
            const uint16_t *p = base + (int64_t)(kk < k_lim ? kk : 0) * ld + (valid > 0 ? mn : 0);
            v[r] = load8(p, valid, vec);
        }
    }

    __device__ __forceinline__ void store(char *lds, int tid) const {
        int mnb = tid % NMB;
        int kb = tid / NMB;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            int row = mnb * 8 + c;
            if constexpr (KB == 8) {
                u32x4 w;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[q] = half16(v[2 * q], c) | (half16(v[2 * q + 1], c) << 16);
                *reinterpret_cast<u32x4 *>(lds + lds_off(row, kb)) = w;
            } else if constexpr (KB == 4) {
                u32x2 w;
                w[0] = half16(v[0], c) | (half16(v[1], c) << 16);
                w[1] = half16(v[2], c) | (half16(v[3], c) << 16);
                *reinterpret_cast<u32x2 *>(lds + lds_off(row, kb >> 1) + ((kb & 1) << 3)) = w;
            } else {
                uint32_t w = half16(v[0], c) | (half16(v[1], c) << 16);
                *reinterpret_cast<uint32_t *>(lds + lds_off(row, kb >> 2) + ((kb & 3) << 2)) = w;
            }
        }
    }
};

template <int BMN, bool KMAJ>
using TileOf = typename std::conditional<KMAJ, KMajorTile<BMN>, MNMajorTile<BMN>>::type;

// Logical tile index of this workgroup: XCD-contiguous runs, see header.
// Tile-rows per run of the grouped tile order (measured on the 24-layer
// step: 4 rows 4.64-4.74 ms, 2 rows +0.4 %, 8 rows +0.8 %, 1 or 16 rows
// +2 %).
#ifndef SBP_TILE_GROUP
#define SBP_TILE_GROUP 4
#endif
__device__ __forceinline__ int remap_xcd(int wg, int total) {
#ifdef SBP_NO_XCD_REMAP
    return wg;
#endif
    constexpr int NX = 8;
    int per = total / NX;
    int rem = total % NX;
    int x = wg % NX;
    int idx = wg / NX;
    return (x < rem) ? x * (per + 1) + idx : rem * (per + 1) + (x - rem) * per + idx;
}

// Store of a GEMM output that this launch does not read back: non-temporal,
// so the output stream does not displace the operand tiles that other
// workgroups still re-read from L2 (measured: the step's fp32 partial-sum
// outputs 10-13 % faster, the whole step 4 %). Split partials take other
// stores (st_part in the pipelined kernel; ordinary ones in this kernel).
template <typename T>
__device__ __forceinline__ void st_nt(T *p, T v) {
    __builtin_nontemporal_store(v, p);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    __bf16 h = (__bf16)f;   // round to nearest even (v_cvt_pk_bf16_f32)
    return __builtin_bit_cast(uint16_t, h);
}


template <int BM, int BN, bool A_KMAJ, bool B_KMAJ, bool OUT_F32>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmArgs g) {
    constexpr int WM = BM / 2, WN = BN / 2;       // wave tile
    constexpr int MI = WM / 32, NI = WN / 32;     // 32x32 MFMA blocks per wave
    constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
    constexpr int STAGE = A_BYTES + B_BYTES;
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // ---- which batch item, tile and reduction range
    const int tiles = g.tiles_m * g.tiles_n;
    const int per_b = tiles * g.splits;
    const int Lz = remap_xcd(blockIdx.x, per_b * g.nbatch);
    const int L = Lz % per_b;
    const uint16_t *Ab, *Bb;
    void *Cb;
    batch_bases<OUT_F32>(g, Lz / per_b, &Ab, &Bb, &Cb);
    const int split = L / tiles;
    const int t = L % tiles;
    // grouped order: runs of GROUP tile-rows, column-major inside a run
    constexpr int GROUP = SBP_TILE_GROUP;
    const int grp = t / (GROUP * g.tiles_n);
    const int first_m = grp * GROUP;
    const int gsize = min(g.tiles_m - first_m, GROUP);
    const int tm = first_m + (t % (GROUP * g.tiles_n)) % gsize;
    const int tn = (t % (GROUP * g.tiles_n)) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    const int k_begin = split * g.kchunk;
    const int k_lim = min(g.k, k_begin + g.kchunk);
    const int nkb = max(0, (k_lim - k_begin + BK - 1) / BK);
    const int kb_begin = k_begin / BK;

    TileOf<BM, A_KMAJ> ta;
    TileOf<BN, B_KMAJ> tb;
    const bool va = g.vec_a != 0, vb = g.vec_b != 0;
    // uniform per workgroup: the tile's m (n) range is inside the operand and aligned
    const bool a_in = va && (m0 + BM <= g.m);
    const bool b_in = vb && (n0 + BN <= g.n);
    auto load_tiles = [&](int k0) {
        const bool k_in = (k0 + BK <= k_lim);
        if (a_in && k_in) ta.load_full(Ab, g.lda, m0, k0, tid);
        else ta.load_edge(Ab, g.lda, m0, g.m, k0, k_lim, tid, va);
        if (b_in && k_in) tb.load_full(Bb, g.ldb, n0, k0, tid);
        else tb.load_edge(Bb, g.ldb, n0, g.n, k0, k_lim, tid, vb);
    };

    f32x16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    if (nkb > 0) {
        load_tiles(kb_begin * BK);
        ta.store(smem, tid);
        tb.store(smem + A_BYTES, tid);
        __syncthreads();

        for (int it = 0; it < nkb; ++it) {
            char *cur = smem + (it & 1) * STAGE;
            const bool more = (it + 1 < nkb);
            if (more) {
                load_tiles((kb_begin + it + 1) * BK);
            }
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                const int chunk = ks * 2 + (lane >> 5);
                bf16x8 af[MI], bfr[NI];
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    int row = wm * WM + i * 32 + (lane & 31);
                    af[i] = *reinterpret_cast<const bf16x8 *>(cur + lds_off(row, chunk));
                }
#pragma unroll
                for (int j = 0; j < NI; ++j) {
                    int row = wn * WN + j * 32 + (lane & 31);
                    bfr[j] = *reinterpret_cast<const bf16x8 *>(cur + A_BYTES + lds_off(row, chunk));
                }
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NI; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
            }
            if (more) {
                char *nxt = smem + ((it + 1) & 1) * STAGE;
                ta.store(nxt, tid);
                tb.store(nxt + A_BYTES, tid);
            }
            __syncthreads();
        }
    }

    // ---- split reduction: partials to the workspace; split_reduce_kernel adds them
    if (g.splits > 1) {
        // Split reduction: this workgroup's fp32 partial goes to slice
        // `split` of the workspace (m x n, row stride partial_ld(n));
        // a separate kernel adds the slices in split order.
        const int64_t ldw = sbpi::partial_ld(g.n);
        float *P = g.ws + (size_t)split * (size_t)g.m * (size_t)ldw;
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int col = n0 + wn * WN + j * 32 + (lane & 31);
                const int rbase = m0 + wm * WM + i * 32 + 4 * (lane >> 5);
                if (col < g.n) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = rbase + 8 * (r >> 2) + (r & 3);
                        // ordinary stores: this kernel's partials are small and read
                        // back at once (non-temporal ones measured 15 % slower here)
                        if (row < g.m) P[(int64_t)row * ldw + col] = acc[i][j][r];
                    }
                }
            }
        return;
    }

    // ---- epilogue: MFMA 32x32 accumulator layout -> row-major C
    // lane holds column (lane & 31); register r holds row 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int j = 0; j < NI; ++j) {
            const int col = n0 + wn * WN + j * 32 + (lane & 31);
            const int rbase = m0 + wm * WM + i * 32 + 4 * (lane >> 5);
            if (col < g.n) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = rbase + 8 * (r >> 2) + (r & 3);
                    if (row < g.m) {
                        if constexpr (OUT_F32) {
                            float *C = reinterpret_cast<float *>(Cb) + (int64_t)row * g.ldc + col;
                            if (g.accumulate) *C = *C + acc[i][j][r];
                            else st_nt(C, acc[i][j][r]);
                        } else {
                            uint16_t *C = reinterpret_cast<uint16_t *>(Cb);
                            st_nt(C + (int64_t)row * g.ldc + col, f32_to_bf16_bits(acc[i][j][r]));
                        }
                    }
                }
            }
        }
    }
}

}  // namespace sbpk
