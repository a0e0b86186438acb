// gemm_bf16_dma.h -- pipelined bf16 MFMA GEMM with direct global->LDS loads
// (CDNA4 / gfx950). Same contract and operand orientations as
// gemm_bf16_kernel.h; used when every operand is 16-byte aligned with a
// leading dimension and a contiguous extent that are multiples of 8
// elements, so each 16-byte chunk of an operand is either wholly inside or
// wholly outside it.
//
// Design:
//   * Workgroups of 4 waves (2 x 2) or 8 waves (2 x 4, two per SIMD, for
//     the 256 x 256 tile, whose 128 fp32 accumulator registers per wave
//     leave room for two waves per SIMD).
//   * Operand tiles move HBM -> LDS with buffer loads that write LDS
//     directly (16 bytes per lane, lane l's bytes at base + 16 l); no
//     registers are spent on staging, so NS pipeline stages (2-4, as LDS
//     allows) are in flight: the loads of step t + NS - 1 are issued while
//     step t computes, hiding HBM latency behind NS - 1 steps of MFMA work.
//     Chunks outside the operand get an out-of-range offset and read as 0.
//   * The reduction step BKD is a template parameter (64 for every instance;
//     32 is supported for deeper pipelines but its row swizzle is not yet free
//     of bank conflicts on gfx950).
//   * k-major operand tiles keep their storage order in LDS: one row of BKD
//     reduction values per output row, 16-byte chunks XOR-swizzled by row;
//     fragments are read with ds_read_b128.
//   * m/n-major operand tiles also keep their storage order: one row of BMN
//     values per reduction index, chunks XOR-swizzled by 4 (row % 4); MFMA
//     fragments (8 consecutive reduction values of one output index per
//     lane) are read with two ds_read_b64_tr_b16, the LDS transpose read: in
//     each 16-lane group, lane t receives element t % 4 of the 4-element
//     rows addressed by lanes 4 j + t / 4, j = 0..3.
//   * v_mfma_f32_32x32x16_bf16, fp32 accumulators; split reduction, XCD-aware
//     tile order and epilogue as in gemm_bf16_kernel.h.
#pragma once

#include "gemm_bf16_kernel.h"

namespace sbpk {

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
#define SBP_LDS __attribute__((address_space(3)))

constexpr int OOB = (int)0x80000000;   // buffer offset that reads as zero

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer descriptor of a raw byte range starting at `base` (wave-uniform):
// stride 0, 2^31 - 1 bytes addressable, 32-bit data format, so an offset of
// 2^31 is out of range and reads as zero.
__device__ __forceinline__ i32x4 make_rsrc(const void *base) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xffffu));
    r[2] = 0x7fffffff;
    r[3] = 0x00020000;
    return r;
}

// One 16-byte-per-lane buffer load that writes LDS directly: lane l's bytes
// land at lds + 16 l. Issued as inline assembly (M0 set in the same
// statement) so that the compiler does not drain every outstanding load at
// the next barrier; completion is awaited explicitly with wait_vm<N>().
__device__ __forceinline__ void dma16(i32x4 r, char *lds, int voff) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(SBP_LDS void *)lds);
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(voff), "s"(r)
                 : "memory", "m0");
}

// ---------------------------------------------------------------- k-major
// LDS: BMN rows x RB bytes (RB = 2 BK: 64 reduction values in 8 chunks of
// 16 B, or 32 in 4). Chunk c of row r sits at r*RB + 16*(c ^ f(r)); f makes
// the 16-byte fragment reads of 8 consecutive rows (32 banks) and of 16
// (64 banks) hit distinct banks.
template <int BMN, int NW, int BK_>
struct KTileDma {
    static constexpr int RB = BK_ * 2;            // bytes per row
    static constexpr int CPR = BK_ / 8;           // chunks per row
    static constexpr int RPS = 1024 / RB;         // rows per 1 KB segment
    static constexpr int SEGS = BMN * RB / 1024;
    static constexpr int PER_WAVE = SEGS / NW;    // segments each wave loads
    static_assert(SEGS % NW == 0, "tile too small for the wave count");

    __device__ __forceinline__ static int swz(int row) {
        return CPR == 8 ? ((row & 7) ^ ((row >> 3) & 7)) : (((row >> 1) ^ (row >> 3)) & 3);
    }
    __device__ __forceinline__ static int off(int row, int c) {
        return row * RB + ((c ^ swz(row)) << 4);
    }

    // Issue the loads of one stage: rows [mn0, mn0+BMN) x reduction [k0, k0+BK_).
    __device__ __forceinline__ static void issue(const uint16_t *base, int64_t ld, int mn0,
                                                 int mn_lim, int k0, int k_lim, char *lds,
                                                 int wave, int lane) {
        const i32x4 r = make_rsrc(base + (int64_t)mn0 * ld + k0);
#pragma unroll
        for (int i = 0; i < PER_WAVE; ++i) {
            const int s = i * NW + wave;
            const int row = s * RPS + lane / CPR;
            const int c = (lane % CPR) ^ swz(row);
            const bool ok = (mn0 + row < mn_lim) && (k0 + c * 8 + 8 <= k_lim);
            const int voff = ok ? (int)((row * ld + c * 8) * 2) : OOB;
            dma16(r, lds + s * 1024, voff);
        }
    }

    // Fragment for rows [r0, r0+32) and reduction [16 ks, 16 ks + 16).
    __device__ __forceinline__ static bf16x8 frag(const char *lds, int r0, int ks, int lane) {
        const int row = r0 + (lane & 31);
        const int chunk = ks * 2 + (lane >> 5);
        return *reinterpret_cast<const bf16x8 *>(lds + off(row, chunk));
    }
};

// ---------------------------------------------------------------- m/n-major
// LDS: BK rows (reduction index) x BMN values; chunk c of row r at
// r*RB + 16*(c ^ (4*(r%4) % CPR)) with RB = 2*BMN bytes, CPR chunks per row.
template <int BMN, int NW, int BK_>
struct MNTileDma {
    static constexpr int RB = BMN * 2;            // bytes per row
    static constexpr int CPR = BMN / 8;           // chunks per row
    static constexpr int SEGS = BMN * BK_ * 2 / 1024;   // 1 KB segments in the BK_-row tile
    static constexpr int PER_WAVE = SEGS / NW;
    static_assert(SEGS % NW == 0, "tile too small for the wave count");

    __device__ __forceinline__ static int swz(int row) {
        return CPR >= 16 ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
    }

    __device__ __forceinline__ static void issue(const uint16_t *base, int64_t ld, int mn0,
                                                 int mn_lim, int k0, int k_lim, char *lds,
                                                 int wave, int lane) {
        const i32x4 r = make_rsrc(base + (int64_t)k0 * ld + mn0);
#pragma unroll
        for (int i = 0; i < PER_WAVE; ++i) {
            const int s = i * NW + wave;
            const int byte = s * 1024 + lane * 16;
            const int row = byte / RB;
            const int phys = (byte % RB) >> 4;
            const int c = phys ^ swz(row);
            const bool ok = (k0 + row < k_lim) && (mn0 + c * 8 + 8 <= mn_lim);
            const int voff = ok ? (int)((row * ld + c * 8) * 2) : OOB;
            dma16(r, lds + s * 1024, voff);
        }
    }

    // Fragment for output indices [c0, c0+32) and reduction [16 ks, 16 ks + 16):
    // lane L gets reduction 16 ks + 8 (L/32) + 0..7 of output index c0 + L%32.
    __device__ __forceinline__ static bf16x8 frag(const char *lds, int c0, int ks, int lane) {
        const int g = lane >> 4, t = lane & 15;
        const int mn = c0 + 16 * (g & 1) + 4 * (t & 3);
        const int rowb = ks * 16 + (g >> 1) * 8 + (t >> 2);
        s16x4 h[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int row = rowb + hh * 4;
            const int off = row * RB + (((mn >> 3) ^ swz(row)) << 4) + ((mn & 7) << 1);
            h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SBP_LDS s16x4 *)(lds + off));
        }
        s16x4 a = h[0], b = h[1];
        s16x8 v8 = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        return __builtin_bit_cast(bf16x8, v8);
    }
};

template <int BMN, int NW, int BK_, bool KMAJ>
using DmaTileOf =
    typename std::conditional<KMAJ, KTileDma<BMN, NW, BK_>, MNTileDma<BMN, NW, BK_>>::type;

template <int N>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int BM, int BN, int BKD, int NS>
struct DmaStage {
    static constexpr int A_BYTES = BM * BKD * 2, B_BYTES = BN * BKD * 2;   // one stage
    static constexpr int BYTES = A_BYTES + B_BYTES;
};

// One work item (an output tile and a reduction split) of a product, by the
// whole workgroup: WGM x WGN waves (2 x 2, or 2 x 4 for the 256 x 256 tile:
// 8 waves, two per SIMD, each owning 128 x 64 outputs). L is the item's
// logical index in [0, tiles * splits).
template <int BM, int BN, int BKD, int NS, int WGM, int WGN, bool A_KMAJ, bool B_KMAJ,
          bool OUT_F32>
__device__ __forceinline__ void dma_tile_body(const GemmArgs &g, const int L, char *smem) {
    constexpr int NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int MI = WM / 32, NI = WN / 32;
    constexpr int A_BYTES = DmaStage<BM, BN, BKD, NS>::A_BYTES;
    constexpr int STAGE = DmaStage<BM, BN, BKD, NS>::BYTES;
    constexpr int LOADS = STAGE / 1024 / NW;                         // dma per thread per stage

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;

    const int tiles = g.tiles_m * g.tiles_n;
    const int split = L / tiles;
    const int t = L % tiles;
    constexpr int GROUP = SBP_TILE_GROUP;
    const int grp = t / (GROUP * g.tiles_n);
    const int first_m = grp * GROUP;
    const int gsize = min(g.tiles_m - first_m, GROUP);
    const int tm = first_m + (t % (GROUP * g.tiles_n)) % gsize;
    const int tn = (t % (GROUP * g.tiles_n)) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    // this split's reduction range [k_begin, k_lim)
    const int k_begin = split * g.kchunk;
    const int k_lim = min(g.k, k_begin + g.kchunk);
    const int nkb = max(0, (k_lim - k_begin + BKD - 1) / BKD);

    using TA = DmaTileOf<BM, NW, BKD, A_KMAJ>;
    using TB = DmaTileOf<BN, NW, BKD, B_KMAJ>;

    auto issue = [&](int kb, int stage) {
        char *base = smem + stage * STAGE;
        const int k0 = k_begin + kb * BKD;
        TA::issue(g.A, g.lda, m0, g.m, k0, k_lim, base, wave, lane);
        TB::issue(g.B, g.ldb, n0, g.n, k0, k_lim, base + A_BYTES, wave, lane);
    };

    f32x16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // prologue: stages 0 .. NS-2 in flight
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < nkb) issue(s, s);

    for (int it = 0; it < nkb; ++it) {
        // wait for this thread's loads of step `it`; later steps may stay in flight
        const int ahead = min(NS - 2, nkb - 1 - it);
        if (ahead >= 2) wait_vm<2 * LOADS>();
        else if (ahead == 1) wait_vm<LOADS>();
        else wait_vm<0>();
        __syncthreads();
        if (it + NS - 1 < nkb) issue(it + NS - 1, (it + NS - 1) % NS);

        const char *cur = smem + (it % NS) * STAGE;
#pragma unroll
        for (int ks = 0; ks < BKD / 16; ++ks) {
            bf16x8 af[MI], bfr[NI];
#pragma unroll
            for (int i = 0; i < MI; ++i)
                af[i] = TA::frag(cur, wm * WM + i * 32, ks, lane);
#pragma unroll
            for (int j = 0; j < NI; ++j)
                bfr[j] = TB::frag(cur + A_BYTES, wn * WN + j * 32, ks, lane);
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    }

    if (g.splits > 1) {
        // Split reduction: this workgroup's fp32 partial goes to slice
        // `split` of the workspace, laid out like the output (m x n, ld n);
        // a separate kernel adds the slices in split order.
        float *P = g.ws + (size_t)split * (size_t)g.m * (size_t)g.n;
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
                        if (row < g.m) P[(int64_t)row * g.n + col] = acc[i][j][r];
                    }
                }
            }
        return;
    }

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
                            float *C = reinterpret_cast<float *>(g.C);
                            C[(int64_t)row * g.ldc + col] = acc[i][j][r];
                        } else {
                            uint16_t *C = reinterpret_cast<uint16_t *>(g.C);
                            C[(int64_t)row * g.ldc + col] = f32_to_bf16_bits(acc[i][j][r]);
                        }
                    }
                }
            }
        }
    }
}


template <int BM, int BN, int BKD, int NS, int WGM, int WGN, bool A_KMAJ, bool B_KMAJ,
          bool OUT_F32>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_bf16_dma_kernel(GemmArgs g) {
    __shared__ __attribute__((aligned(1024))) char smem[NS * DmaStage<BM, BN, BKD, NS>::BYTES];
    const int total = g.tiles_m * g.tiles_n * g.splits;
    dma_tile_body<BM, BN, BKD, NS, WGM, WGN, A_KMAJ, B_KMAJ, OUT_F32>(
        g, remap_xcd(blockIdx.x, total), smem);
}

// The two backward products of one linear in one launch: gd is the
// backward-data product (both operands k-major), gw the backward-weight
// product (both m/n-major). They are independent (each reads only dY and one
// of X, W), so their work items share the grid; the product whose work
// items are longer is dispatched first (data_first) so that the short items
// of the other fill the machine behind them.
template <int BM, int BN, int BKD, int NS, int WGM, int WGN, bool OUTD_F32, bool OUTW_F32>
__global__ __launch_bounds__(64 * WGM * WGN, 1) void gemm_bf16_dma_bwd_kernel(GemmArgs gd,
                                                                             GemmArgs gw,
                                                                             int data_first) {
    __shared__ __attribute__((aligned(1024))) char smem[NS * DmaStage<BM, BN, BKD, NS>::BYTES];
    const int wd = gd.tiles_m * gd.tiles_n * gd.splits;
    const int ww = gw.tiles_m * gw.tiles_n * gw.splits;
    const int b = blockIdx.x;
    const bool is_data = data_first ? (b < wd) : (b >= ww);
    if (is_data) {
        const int local = data_first ? b : b - ww;
        dma_tile_body<BM, BN, BKD, NS, WGM, WGN, true, true, OUTD_F32>(gd, remap_xcd(local, wd),
                                                                      smem);
    } else {
        const int local = data_first ? b - wd : b;
        dma_tile_body<BM, BN, BKD, NS, WGM, WGN, false, false, OUTW_F32>(gw, remap_xcd(local, ww),
                                                                        smem);
    }
}

}  // namespace sbpk
