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
//   * The reduction step BKD is a template parameter: 64; 32 for deeper
//     pipelines (more stages in the same LDS); or 128, with two reduction
//     groups, for half the barriers per flop and 256-byte k-major rows.
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

#include <type_traits>

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
// 16 B, 32 in 4, or 128 in 16). Chunk c of row r sits at r*RB + 16*(c ^
// f(r)); f makes the 16-byte fragment reads of 8 consecutive rows (32 banks)
// and of 16 (64 banks) hit distinct banks: with 64-byte rows, 16 aligned
// rows cover the 16 bank quads once as 4 (r % 4) + (c ^ (r / 4 % 4)); with
// 256-byte rows (one row spans all 64 banks) f(r) = r % 16.
template <int BMN, int NW, int BK_>
struct KTileDma {
    static constexpr int RB = BK_ * 2;            // bytes per row
    static constexpr int CPR = BK_ / 8;           // chunks per row
    static constexpr int RPS = 1024 / RB;         // rows per 1 KB segment
    static constexpr int SEGS = BMN * RB / 1024;
    static constexpr int PER_WAVE = SEGS / NW;    // segments each wave loads
    static_assert(SEGS % NW == 0, "tile too small for the wave count");

    __device__ __forceinline__ static int swz(int row) {
        if constexpr (CPR == 16) return row & 15;
        return CPR == 8 ? ((row & 7) ^ ((row >> 3) & 7)) : ((row >> 2) & 3);
    }
    __device__ __forceinline__ static int off(int row, int c) {
        return row * RB + ((c ^ swz(row)) << 4);
    }

    // Issue the loads of one stage: rows [mn0, mn0+BMN) x reduction [k0, k0+BK_).
    // PART (shifted index spaces): a chunk that starts inside the operand is
    // read whole -- its 16 bytes lie in one 16-byte block of a row that holds
    // operand elements, so the read stays inside that row's memory -- and
    // its elements past the limit are zeroed in LDS (zero_outside); else a
    // chunk is read only if it lies wholly inside.
    template <bool PART>
    __device__ __forceinline__ static void issue(const uint16_t *base, int64_t ld, int mn0,
                                                 int mn_lim, int k0, int k_lim, char *lds,
                                                 int wave, int lane) {
        const i32x4 r = make_rsrc(base + (int64_t)mn0 * ld + k0);
#pragma unroll
        for (int i = 0; i < PER_WAVE; ++i) {
            const int s = i * NW + wave;
            const int row = s * RPS + lane / CPR;
            const int c = (lane % CPR) ^ swz(row);
            const bool ok = (mn0 + row < mn_lim) &&
                            (PART ? k0 + c * 8 < k_lim : k0 + c * 8 + 8 <= k_lim);
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

    // In the stage holding reduction indices [k0, k0 + BK_): zeroes every
    // element whose index lies outside [lo, hi) in the chunks that hold lo
    // and hi (the only chunks read whole that can contain such elements),
    // by nt threads.
    __device__ static void zero_outside(char *lds, int k0, int lo, int hi, int tid, int nt) {
        for (int q = tid; q < BMN * 2; q += nt) {
            const int row = q >> 1;
            const int kc = ((q & 1) ? hi : lo) & ~7;   // first index of the chunk
            const int c = (kc - k0) >> 3;
            if (kc < k0 || c >= CPR) continue;
            uint16_t *p = reinterpret_cast<uint16_t *>(lds + off(row, c));
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (kc + e < lo || kc + e >= hi) p[e] = 0;
        }
    }
};

// ---------------------------------------------------------------- m/n-major
// LDS: BK rows (reduction index) x BMN values; chunk c of row r at
// r*RB + 16*(c ^ f(r)) with RB = 2*BMN bytes, CPR chunks per row. A transpose
// read of one half-wave touches 4 consecutive rows and 4 consecutive chunks
// (64 bytes of each row); f spreads those 4 rows over the 64 banks: rows of
// 256 or 512 bytes all start on bank 0, so f(r) = 4 (r % 4); rows of 128 or
// 384 bytes start on banks 0 and 32 alternately, so f(r) = 4 ((r / 2) % 2)
// (which keeps the 24 chunks of a 384-byte row inside the row).
template <int BMN, int NW, int BK_>
struct MNTileDma {
    static constexpr int RB = BMN * 2;            // bytes per row
    static constexpr int CPR = BMN / 8;           // chunks per row
    static constexpr int SEGS = BMN * BK_ * 2 / 1024;   // 1 KB segments in the BK_-row tile
    static constexpr int PER_WAVE = SEGS / NW;
    static_assert(SEGS % NW == 0, "tile too small for the wave count");

    static_assert(CPR == 8 || CPR == 16 || CPR == 24 || CPR == 32, "unsupported tile width");
    __device__ __forceinline__ static int swz(int row) {
        return (CPR == 16 || CPR == 32) ? 4 * (row & 3) : 4 * ((row >> 1) & 1);
    }

    // PART: as for KTileDma (a chunk past mn_lim holds only outputs that are
    // never stored).
    template <bool PART>
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
            const bool ok = (k0 + row < k_lim) &&
                            (PART ? mn0 + c * 8 < mn_lim : mn0 + c * 8 + 8 <= mn_lim);
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
    static_assert(N >= 0 && N <= 63, "vmcnt holds 6 bits");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `ahead` of this thread's stages (LOADS loads each) are
// still in flight; `ahead` <= K.
template <int K, int LOADS>
__device__ __forceinline__ void wait_stages(int ahead) {
    if constexpr (K <= 0) {
        wait_vm<0>();
    } else {
        if (ahead >= K) wait_vm<K * LOADS>();
        else wait_stages<K - 1, LOADS>(ahead);
    }
}

template <int BM, int BN, int BKD, int NS>
struct DmaStage {
    static constexpr int A_BYTES = BM * BKD * 2, B_BYTES = BN * BKD * 2;   // one stage
    static constexpr int BYTES = A_BYTES + B_BYTES;
};

// Launch bound of an instance: the minimum number of waves per SIMD the
// compiler budgets registers for. A four-wave workgroup puts one wave on each
// SIMD, so for those this is the number of workgroups per compute unit that
// the LDS pipeline allows (160 KB per CU; e.g. two 128 x 128 two-stage
// workgroups, not one). Eight-wave (two-group) workgroups get 1: no register
// limit. (Budgeting the two-stage 128 x 128 two-group instance for two
// workgroups per CU, 128 registers, made its reduction steps no faster than
// the four-wave instance's at two per CU, with a higher fixed cost.)
template <int BM, int BN, int BKD, int NS, int NWAVES, int KG>
struct Occupancy {
    static constexpr int BY_LDS = 163840 / (NS * DmaStage<BM, BN, BKD, NS>::BYTES);
    static constexpr int BY_WAVES = 16 / NWAVES;
    static constexpr int V0 = BY_LDS < BY_WAVES ? BY_LDS : BY_WAVES;
    static constexpr int VALUE = (KG > 1 || V0 < 1) ? 1 : V0;
};

// Output rows of the staged epilogue are padded by 8 floats where the LDS
// allows: the two half-waves of a 32 x 32 MFMA block write rows 4 apart, and
// 4 (BN + 8) = 32 mod 64 floats puts them on disjoint LDS banks (unpadded, the
// two halves share banks: a 2-way conflict on those writes).
template <int BN, int BM = 0, int BYTES = 1 << 30>
struct StageRow {
    // floats per staged output row: padded when the padded tile fits
    static constexpr int LD = (BM * (BN + 8) * 4 <= BYTES) ? BN + 8 : BN;
};

// Stores of split partials (the fp32 slices that the split reduction reads
// after this launch): buffer stores at device scope (sc1), which write
// through the XCD's L2 instead of leaving dirty lines there. Measured on the
// 24-layer step (same box, alternating runs): 1.0-1.3 % faster than
// non-temporal stores; plain or sc0 stores 1.4 % and sc1 with nt 1.5 %
// slower than sc1, sc0 with sc1 the same. (Final outputs stay
// non-temporal: sc1 for them made the step 3.6 % slower.) `idx` is the
// element index from the slice base; a slice is below 2^31 bytes (the
// workspace bound of every plan).
#ifndef SBP_PART_CPOL
#define SBP_PART_CPOL 16   // sc1
#endif
__device__ __forceinline__ __amdgpu_buffer_rsrc_t part_rsrc(const void *slice) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(slice), (short)0, 0x7fffffff,
                                             0x00020000);
}
__device__ __forceinline__ void st_part(__amdgpu_buffer_rsrc_t r, int64_t idx, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, (int)(idx * 4), 0,
                                          SBP_PART_CPOL);
}
__device__ __forceinline__ void st_part(__amdgpu_buffer_rsrc_t r, int64_t idx, f32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)(idx * 4), 0,
                                           SBP_PART_CPOL);
}

// Stores the BM x BN fp32 tile staged in LDS (`tile`, row stride
// LD floats) to rows [m0, m0 + BM) x columns [n0, n0 + BN) of C
// (ld `ldc`, clipped to [0, m) x [0, n); m0 and n0 may be negative in a
// shifted index space), by all NT_ threads: each thread moves whole
// 16-byte chunks along a row -- 4 floats, or 8 values rounded to bf16 -- so a
// wave writes whole contiguous row segments. `vec`: C's base and ldc allow
// aligned 16-byte stores; otherwise (and at the right edge) elements are
// stored one by one. PART: C is a split partial slice (st_part).
template <int BM, int BN, int LD, int NT_, bool F32, bool ACC = false, bool SHIFT = false,
          bool PART = false>
__device__ __forceinline__ void store_staged(const float *tile, void *C, int64_t ldc, int m,
                                             int n, int m0, int n0, bool vec, int tid) {
    static_assert(F32 || !ACC, "accumulation needs an fp32 output");
    constexpr int EPC = F32 ? 4 : 8;             // output elements per 16-byte chunk
    constexpr int CPR = BN / EPC;                // chunks per tile row
    constexpr int ITER = BM * CPR / NT_;
    static_assert((BM * CPR) % NT_ == 0, "tile not divisible among threads");
#pragma unroll 4
    for (int it = 0; it < ITER; ++it) {
        const int q = it * NT_ + tid;
        const int r = q / CPR, c = (q % CPR) * EPC;
        const int row = m0 + r, col = n0 + c;
        if (SHIFT ? ((unsigned)row >= (unsigned)m || col >= n || col + EPC <= 0)
                  : (row >= m || col >= n))
            continue;
        const float *src = tile + r * LD + c;
        if constexpr (F32) {
            f32x4 v = *reinterpret_cast<const f32x4 *>(src);
            float *dst = reinterpret_cast<float *>(C) + (int64_t)row * ldc + col;
            if (vec && (!SHIFT || col >= 0) && col + 4 <= n) {
                if constexpr (ACC) {
                    v += *reinterpret_cast<const f32x4 *>(dst);
                    *reinterpret_cast<f32x4 *>(dst) = v;
                } else if constexpr (PART) {
                    st_part(part_rsrc(C), (int64_t)row * ldc + col, v);
                } else {
                    st_nt(reinterpret_cast<f32x4 *>(dst), v);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (SHIFT ? (unsigned)(col + e) < (unsigned)n : col + e < n) {
                        if constexpr (ACC) dst[e] = dst[e] + v[e];
                        else if constexpr (PART) st_part(part_rsrc(C), (int64_t)row * ldc + col + e, v[e]);
                        else st_nt(dst + e, v[e]);
                    }
            }
        } else {
            const f32x4 a = *reinterpret_cast<const f32x4 *>(src);
            const f32x4 b = *reinterpret_cast<const f32x4 *>(src + 4);
            uint16_t *dst = reinterpret_cast<uint16_t *>(C) + (int64_t)row * ldc + col;
            if (vec && (!SHIFT || col >= 0) && col + 8 <= n) {
                u32x4 w;
                w[0] = (uint32_t)f32_to_bf16_bits(a[0]) | ((uint32_t)f32_to_bf16_bits(a[1]) << 16);
                w[1] = (uint32_t)f32_to_bf16_bits(a[2]) | ((uint32_t)f32_to_bf16_bits(a[3]) << 16);
                w[2] = (uint32_t)f32_to_bf16_bits(b[0]) | ((uint32_t)f32_to_bf16_bits(b[1]) << 16);
                w[3] = (uint32_t)f32_to_bf16_bits(b[2]) | ((uint32_t)f32_to_bf16_bits(b[3]) << 16);
                st_nt(reinterpret_cast<u32x4 *>(dst), w);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (SHIFT ? (unsigned)(col + e) < (unsigned)n : col + e < n)
                        st_nt(dst + e, f32_to_bf16_bits(e < 4 ? a[e] : b[e - 4]));
            }
        }
    }
}

// Epilogue variants of the tile body.
enum : int {
    EPI_DIRECT = 0,   // each lane stores its MFMA elements (4-byte / 2-byte stores)
    EPI_STAGED = 1,   // tile staged in LDS, stored as 16-byte row chunks by all threads
    EPI_ROWQ = 2      // MFMA operands swapped so that each lane holds 4 consecutive
                      // outputs of one row: 16-byte (fp32) / 8-byte (bf16) stores
                      // straight from registers, no LDS and no wait
};

// One work item (an output tile and a reduction split) of a product, by the
// whole workgroup of KG x WGM x WGN waves. The WGM x WGN waves of a
// reduction group own (BM / WGM) x (BN / WGN) outputs each; with KG = 2 the
// two groups take alternate halves of every 64-wide reduction step (so each
// SIMD holds two waves, one of each group, and one's MFMAs run while the
// other waits on LDS), and their fp32 sums are added through LDS at the end.
// L is the item's logical index in [0, tiles * splits). On return from the
// staged and row-quad epilogues every wave is done reading the pipeline's
// LDS, so the next item may refill it; after the direct epilogue the caller
// must synchronise the workgroup first.
template <int BM, int BN, int BKD, int NS, int WGM, int WGN, int KG, int EPI, bool A_KMAJ,
          bool B_KMAJ, bool OUT_F32, bool SHIFT, class Args>
__device__ __forceinline__ void dma_tile_body(const Args &g, const int L, char *smem) {
    constexpr int NSW = WGM * WGN;                // waves per reduction group
    constexpr int NW = NSW * KG;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int MI = WM / 32, NI = WN / 32;
    constexpr int KSG = BKD / 16 / KG;            // 16-wide sub-steps per group and step
    constexpr int A_BYTES = DmaStage<BM, BN, BKD, NS>::A_BYTES;
    constexpr int STAGE = DmaStage<BM, BN, BKD, NS>::BYTES;
    constexpr int LOADS = STAGE / 1024 / NW;                         // dma per thread per stage
    constexpr bool SWAP = EPI == EPI_ROWQ;
    static_assert(KG == 1 || KG == 2, "one or two reduction groups");
    static_assert(BKD % (16 * KG) == 0, "reduction step not divisible among groups");
    constexpr int SLD = StageRow<BN, BM, NS * STAGE>::LD;
    static_assert(EPI != EPI_STAGED || BM * SLD * 4 <= NS * STAGE,
                  "staged output tile does not fit the pipeline's LDS");
    static_assert(KG == 1 || NSW * MI * NI * 64 * 64 <= NS * STAGE,
                  "group partial sums do not fit the pipeline's LDS");
    static_assert(KG == 1 || EPI != EPI_DIRECT, "two reduction groups need a summing epilogue");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // wave < NW; with one group the compiler must see kg = 0 to keep the
    // fragment addresses compile-time offsets
    const int kg = KG == 1 ? 0 : wave / NSW;
    const int sw = KG == 1 ? wave : wave % NSW;
    const int wm = sw / WGN, wn = sw % WGN;

    const int tiles = g.tiles_m * g.tiles_n;
    // batch item (the attention core's batched products; 0 otherwise)
    const int per_b = tiles * g.splits;
    const uint16_t *Ab, *Bb;
    void *Cb;
    batch_bases<OUT_F32>(g, L / per_b, &Ab, &Bb, &Cb);
    const int Lb = L % per_b;
    const int split = Lb / tiles;
    const int t = Lb % tiles;
    constexpr int GROUP = SBP_TILE_GROUP;
    const int grp = t / (GROUP * g.tiles_n);
    const int first_m = grp * GROUP;
    const int gsize = min(g.tiles_m - first_m, GROUP);
    const int tm = first_m + (t % (GROUP * g.tiles_n)) % gsize;
    const int tn = (t % (GROUP * g.tiles_n)) / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    // this split's reduction range [k_begin, k_lim) in the kernel's index
    // space (the last split also takes the up to 7 extra elements of a
    // reduction offset)
    const int k_end = g.k + shift_k(g);
    const int k_begin = split * g.kchunk;
    const int k_lim =
        SHIFT && split == g.splits - 1 ? k_end : min(k_end, k_begin + g.kchunk);
    const int nkb = max(0, (k_lim - k_begin + BKD - 1) / BKD);

    using TA = DmaTileOf<BM, NW, BKD, A_KMAJ>;
    using TB = DmaTileOf<BN, NW, BKD, B_KMAJ>;

    auto issue = [&](int kb, int stage) {
        char *base = smem + stage * STAGE;
        const int k0 = k_begin + kb * BKD;
        TA::template issue<SHIFT>(Ab, g.lda, m0, g.m + shift_m(g), k0, k_lim, base, wave, lane);
        TB::template issue<SHIFT>(Bb, g.ldb, n0, g.n + shift_n(g), k0, k_lim, base + A_BYTES, wave,
                                  lane);
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
        wait_stages<NS - 2, LOADS>(min(NS - 2, nkb - 1 - it));
        __syncthreads();
        if (it + NS - 1 < nkb) issue(it + NS - 1, (it + NS - 1) % NS);

        const char *cur = smem + (it % NS) * STAGE;
        if constexpr (SHIFT) {
            if (kmask_of(g) && (it == 0 || it == nkb - 1)) {
                // a boundary step: zero the k-major tiles' elements outside
                // the reduction (at most two partial chunks per row), then
                // let every wave see them
                const int k0 = k_begin + it * BKD;
                if constexpr (A_KMAJ)
                    TA::zero_outside(const_cast<char *>(cur), k0, shift_k(g), k_end, tid,
                                     64 * NW);
                if constexpr (B_KMAJ)
                    TB::zero_outside(const_cast<char *>(cur) + A_BYTES, k0, shift_k(g), k_end,
                                     tid, 64 * NW);
                __syncthreads();
            }
        }
#pragma unroll
        for (int kk = 0; kk < KSG; ++kk) {
            const int ks = kg * KSG + kk;
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
                    acc[i][j] = SWAP ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i],
                                                                               acc[i][j], 0, 0, 0)
                                     : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j],
                                                                               acc[i][j], 0, 0, 0);
        }
    }

    // Split reduction: this workgroup's fp32 partial goes to slice `split`
    // of the workspace (m x n, row stride partial_ld(n)); a separate kernel
    // adds the slices in split order.
    const bool partial = g.splits > 1;
    const int ldw = (int)sbpi::partial_ld(g.n);
    float *const ws_out = g.ws + (size_t)split * (size_t)g.m * (size_t)ldw;
    const bool ws_vec = shift_n(g) % 4 == 0;
    // the tile's first output row and column (SHIFT: kernel index minus the
    // shift; may be negative, and bounds are then checked as unsigned)
    const int om0 = m0 - shift_m(g), on0 = n0 - shift_n(g);
    // output index in range: [0, lim) when shifted, else below lim
    auto inb = [](int i, int lim) { return SHIFT ? (unsigned)i < (unsigned)lim : i < lim; };

    if constexpr (EPI != EPI_DIRECT) __syncthreads();   // every wave is done with the pipeline's LDS

    if constexpr (KG == 2 && EPI == EPI_ROWQ) {
        // group 1 hands its sums to group 0 through LDS (lane-contiguous
        // 16-byte slots, conflict free); group 0 stores the total
        f32x4 *slot = reinterpret_cast<f32x4 *>(smem) + sw * (MI * NI * 4 * 64) + lane;
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                   acc[i][j][4 * q + 3]};
                        slot[((i * NI + j) * 4 + q) * 64] = v;
                    }
        }
        __syncthreads();
        if (kg == 0) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const f32x4 v = slot[((i * NI + j) * 4 + q) * 64];
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += v[e];
                    }
        }
        __syncthreads();   // the slots are free again
        if (kg == 1) return;
    }

    if constexpr (EPI == EPI_ROWQ) {
        // lane owns row r = lane % 32 of each 32 x 32 block and, for register
        // quad q, columns 8 q + 4 (lane / 32) + 0..3
        // part_tag: out is a split partial slice (st_part)
        auto store_all = [&](auto f32_tag, auto acc_tag, void *out, int64_t ldo, bool vec,
                             auto part_tag) {
            constexpr bool F32 = decltype(f32_tag)::value;
            constexpr bool ACC = decltype(acc_tag)::value;
            constexpr bool PART = decltype(part_tag)::value;
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                const int row = om0 + wm * WM + i * 32 + (lane & 31);
                if (!inb(row, g.m)) continue;
#pragma unroll
                for (int j = 0; j < NI; ++j) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int col = on0 + wn * WN + j * 32 + 8 * q + 4 * (lane >> 5);
                        if (col >= g.n || (SHIFT && col + 4 <= 0)) continue;
                        if constexpr (F32) {
                            float *dst = reinterpret_cast<float *>(out) + (int64_t)row * ldo + col;
                            if (vec && (!SHIFT || col >= 0) && col + 4 <= g.n) {
                                f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1],
                                           acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                                if constexpr (ACC) {
                                    v += *reinterpret_cast<const f32x4 *>(dst);
                                    *reinterpret_cast<f32x4 *>(dst) = v;
                                } else if constexpr (PART) {
                                    st_part(part_rsrc(out), (int64_t)row * ldo + col, v);
                                } else {
                                    st_nt(reinterpret_cast<f32x4 *>(dst), v);
                                }
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (inb(col + e, g.n)) {
                                        if constexpr (ACC)
                                            dst[e] = dst[e] + acc[i][j][4 * q + e];
                                        else if constexpr (PART)
                                            st_part(part_rsrc(out), (int64_t)row * ldo + col + e,
                                                    acc[i][j][4 * q + e]);
                                        else
                                            st_nt(dst + e, acc[i][j][4 * q + e]);
                                    }
                            }
                        } else {
                            uint16_t *dst =
                                reinterpret_cast<uint16_t *>(out) + (int64_t)row * ldo + col;
                            if (vec && (!SHIFT || col >= 0) && col + 4 <= g.n) {
                                u32x2 w;
                                w[0] = (uint32_t)f32_to_bf16_bits(acc[i][j][4 * q]) |
                                       ((uint32_t)f32_to_bf16_bits(acc[i][j][4 * q + 1]) << 16);
                                w[1] = (uint32_t)f32_to_bf16_bits(acc[i][j][4 * q + 2]) |
                                       ((uint32_t)f32_to_bf16_bits(acc[i][j][4 * q + 3]) << 16);
                                st_nt(reinterpret_cast<u32x2 *>(dst), w);
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (inb(col + e, g.n))
                                        st_nt(dst + e, f32_to_bf16_bits(acc[i][j][4 * q + e]));
                            }
                        }
                    }
                }
            }
        };
        if (partial)
            store_all(std::true_type{}, std::false_type{}, ws_out, (int64_t)ldw, ws_vec,
                      std::true_type{});
        else if (OUT_F32 && g.accumulate)
            store_all(std::integral_constant<bool, OUT_F32>{}, std::integral_constant<bool, OUT_F32>{},
                      Cb, g.ldc, (bool)g.vec_c4, std::false_type{});
        else
            store_all(std::integral_constant<bool, OUT_F32>{}, std::false_type{}, Cb, g.ldc,
                      (bool)g.vec_c4, std::false_type{});
        return;
    }

    if constexpr (EPI == EPI_STAGED) {
        constexpr int LD = SLD;
        float *tile = reinterpret_cast<float *>(smem);
        // element (r, c) of 32 x 32 block (i, j) of this wave, MFMA layout:
        // c = lane % 32, r = 8 (q / 4) + 4 (lane / 32) + q % 4 for register q
        const int cbase = wn * WN + (lane & 31);
        const int rbase = wm * WM + 4 * (lane >> 5);
        if (kg == KG - 1) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int q = 0; q < 16; ++q)
                        tile[(rbase + i * 32 + 8 * (q >> 2) + (q & 3)) * LD + cbase + j * 32] =
                            acc[i][j][q];
        }
        if constexpr (KG == 2) {
            __syncthreads();
            if (kg == 0) {
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NI; ++j)
#pragma unroll
                        for (int q = 0; q < 16; ++q) {
                            float *e = &tile[(rbase + i * 32 + 8 * (q >> 2) + (q & 3)) * LD +
                                             cbase + j * 32];
                            *e = acc[i][j][q] + *e;
                        }
            }
        }
        __syncthreads();
        if (partial)
            store_staged<BM, BN, LD, 64 * NW, true, false, SHIFT, true>(tile, ws_out, ldw, g.m, g.n,
                                                                  om0, on0, ws_vec, tid);
        else if (OUT_F32 && g.accumulate)
            store_staged<BM, BN, LD, 64 * NW, OUT_F32, OUT_F32, SHIFT>(
                tile, Cb, g.ldc, g.m, g.n, om0, on0, g.vec_c4, tid);
        else
            store_staged<BM, BN, LD, 64 * NW, OUT_F32, false, SHIFT>(
                tile, Cb, g.ldc, g.m, g.n, om0, on0, OUT_F32 ? g.vec_c4 : g.vec_c8, tid);
        __syncthreads();   // the staged tile is free again
        return;
    }

    // part_tag: out is a split partial slice (st_part)
    auto store_all = [&](auto f32_tag, auto acc_tag, void *out, int64_t ldo, auto part_tag) {
        constexpr bool F32 = decltype(f32_tag)::value;
        constexpr bool ACC = decltype(acc_tag)::value;
        constexpr bool PART = decltype(part_tag)::value;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int col = on0 + wn * WN + j * 32 + (lane & 31);
                const int rbase = om0 + wm * WM + i * 32 + 4 * (lane >> 5);
                if (inb(col, g.n)) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = rbase + 8 * (r >> 2) + (r & 3);
                        if (inb(row, g.m)) {
                            if constexpr (F32 && ACC) {
                                float *d = reinterpret_cast<float *>(out) + (int64_t)row * ldo + col;
                                *d = *d + acc[i][j][r];
                            } else if constexpr (F32 && PART)
                                st_part(part_rsrc(out), (int64_t)row * ldo + col, acc[i][j][r]);
                            else if constexpr (F32)
                                st_nt(reinterpret_cast<float *>(out) + (int64_t)row * ldo + col,
                                      acc[i][j][r]);
                            else
                                st_nt(reinterpret_cast<uint16_t *>(out) + (int64_t)row * ldo + col,
                                      f32_to_bf16_bits(acc[i][j][r]));
                        }
                    }
                }
            }
        }
    };
    if (partial)
        store_all(std::true_type{}, std::false_type{}, ws_out, (int64_t)ldw, std::true_type{});
    else if (OUT_F32 && g.accumulate)
        store_all(std::integral_constant<bool, OUT_F32>{}, std::integral_constant<bool, OUT_F32>{},
                  Cb, g.ldc, std::false_type{});
    else
        store_all(std::integral_constant<bool, OUT_F32>{}, std::false_type{}, Cb, g.ldc,
                  std::false_type{});
}


// A grid of `gridDim.x` workgroups works through the product's
// tiles * splits items: workgroup b takes items b, b + G, b + 2G, ...
// (G = gridDim.x, a multiple of 8 when smaller than the item count, so that
// every item of one workgroup maps to the same XCD under remap_xcd). With a
// grid smaller than the item count, one item's output stores drain while
// the next item's operand loads are in flight.
template <bool SHIFT>
using ArgsOf = typename std::conditional<SHIFT, GemmArgsShift, GemmArgs>::type;

template <int BM, int BN, int BKD, int NS, int WGM, int WGN, int KG, int EPI, bool A_KMAJ,
          bool B_KMAJ, bool OUT_F32, bool SHIFT = false>
__global__ __launch_bounds__(64 * WGM * WGN * KG,
                             (Occupancy<BM, BN, BKD, NS, WGM * WGN * KG, KG>::VALUE))
void gemm_bf16_dma_kernel(ArgsOf<SHIFT> g) {
    __shared__ __attribute__((aligned(1024))) char smem[NS * DmaStage<BM, BN, BKD, NS>::BYTES];
    const int total = g.tiles_m * g.tiles_n * g.splits * g.nbatch;
    for (int v = blockIdx.x; v < total; v += gridDim.x) {
        // a later item refills the pipeline's LDS: every wave must be done
        // reading it (the direct epilogue does not end with a barrier)
        if (EPI == EPI_DIRECT && v != (int)blockIdx.x) __syncthreads();
        dma_tile_body<BM, BN, BKD, NS, WGM, WGN, KG, EPI, A_KMAJ, B_KMAJ, OUT_F32, SHIFT>(
            g, remap_xcd(v, total), smem);
    }
}

// The two backward products of one linear in one launch: gd is the
// backward-data product (both operands k-major), gw the backward-weight
// product (both m/n-major). They are independent (each reads only dY and one
// of X, W), so their work items share the grid; the product whose work
// items are longer is dispatched first (data_first) so that the short items
// of the other fill the machine behind them.
template <int BM, int BN, int BKD, int NS, int WGM, int WGN, int KG, int EPI, bool OUTD_F32,
          bool OUTW_F32, bool SHIFT = false>
__global__ __launch_bounds__(64 * WGM * WGN * KG,
                             (Occupancy<BM, BN, BKD, NS, WGM * WGN * KG, KG>::VALUE))
void gemm_bf16_dma_bwd_kernel(ArgsOf<SHIFT> gd, ArgsOf<SHIFT> gw, int data_first) {
    __shared__ __attribute__((aligned(1024))) char smem[NS * DmaStage<BM, BN, BKD, NS>::BYTES];
    const int wd = gd.tiles_m * gd.tiles_n * gd.splits * gd.nbatch;
    const int ww = gw.tiles_m * gw.tiles_n * gw.splits * gw.nbatch;
    const int b = blockIdx.x;
    const bool is_data = data_first ? (b < wd) : (b >= ww);
    if (is_data) {
        const int local = data_first ? b : b - ww;
        dma_tile_body<BM, BN, BKD, NS, WGM, WGN, KG, EPI, true, true, OUTD_F32, SHIFT>(
            gd, remap_xcd(local, wd), smem);
    } else {
        const int local = data_first ? b - wd : b;
        dma_tile_body<BM, BN, BKD, NS, WGM, WGN, KG, EPI, false, false, OUTW_F32, SHIFT>(
            gw, remap_xcd(local, ww), smem);
    }
}

}  // namespace sbpk
