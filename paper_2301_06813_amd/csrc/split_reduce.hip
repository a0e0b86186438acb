// split_reduce.hip -- second half of the split reduction.
//
// A GEMM launched with S > 1 reduction splits leaves S fp32 partial
// products in a workspace, slice s holding the m x n output of split s
// (row-major, row stride partial_ld(n): n rounded up to a multiple of 4).
// This kernel adds the slices in split order 0, 1, ..., S-1 -- the same
// order whatever the schedule, so results are deterministic -- and writes
// the output as fp32 (or adds the sum to the fp32 output's contents), or as
// bf16 rounded to nearest even. Each thread owns 4 consecutive columns of
// one row: one 16-byte load per slice (the padded stride keeps every group
// aligned, also where n is not a multiple of 4: measured 13.6 -> 10.4 us on
// a 256 x 125 x 4096 product split 8 ways, whose element-wise loads of
// 125-wide slices waited on memory once per element), and one vector store
// (or element stores at a ragged edge or an unaligned output) that is
// contiguous across the threads of a wave.
#include "gemm.h"
#include "profile.h"

namespace sbpk {

typedef float f32x4v __attribute__((ext_vector_type(4)));

// Sums the S slices of one product's 4-column group gidx (row gidx /
// groups_per_row) in split order and stores it; out-of-range ids do nothing.
// The slices' loads are issued four at a time before they are added (still
// in split order), so a thread waits for one memory latency per four slices
// rather than per slice. vec: C's base and ldc allow one 16-byte (fp32) or
// 8-byte (bf16) store per group.
template <bool OUT_F32>
__device__ __forceinline__ void reduce_group(const float *ws, int m, int n, int S, void *C,
                                             int64_t ldc, bool vec, bool acc, int64_t gidx) {
    const int groups_per_row = (n + 3) / 4;
    if (gidx >= (int64_t)m * groups_per_row) return;
    const int row = (int)(gidx / groups_per_row);
    const int col = (int)(gidx % groups_per_row) * 4;
    const int64_t ldw = sbpi::partial_ld(n);
    const size_t slice = (size_t)m * (size_t)ldw;
    const float *p = ws + (size_t)row * ldw + col;
    auto ld = [&](int s) {
        return __builtin_nontemporal_load(reinterpret_cast<const f32x4v *>(p + s * slice));
    };
    f32x4v v = {0.f, 0.f, 0.f, 0.f};
    int s = 0;
    for (; s + 4 <= S; s += 4) {
        const f32x4v x0 = ld(s), x1 = ld(s + 1), x2 = ld(s + 2), x3 = ld(s + 3);
        v += x0;
        v += x1;
        v += x2;
        v += x3;
    }
    for (; s < S; ++s) v += ld(s);
    if (vec && col + 4 <= n) {
        if constexpr (OUT_F32) {
            f32x4v *dst =
                reinterpret_cast<f32x4v *>(reinterpret_cast<float *>(C) + (int64_t)row * ldc + col);
            if (acc) *dst = *dst + v;
            else __builtin_nontemporal_store(v, dst);   // not read back by this kernel
        } else {
            typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
            u32x2v w;
            w[0] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[0]) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[1]) << 16);
            w[1] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[2]) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)v[3]) << 16);
            __builtin_nontemporal_store(
                w, reinterpret_cast<u32x2v *>(reinterpret_cast<uint16_t *>(C) +
                                              (int64_t)row * ldc + col));
        }
        return;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (col + e >= n) break;
        if constexpr (OUT_F32) {
            float *dst = reinterpret_cast<float *>(C) + (int64_t)row * ldc + col + e;
            if (acc) *dst = *dst + v[e];
            else __builtin_nontemporal_store(v[e], dst);
        } else {
            __bf16 h = (__bf16)v[e];
            __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, h),
                                        reinterpret_cast<uint16_t *>(C) + (int64_t)row * ldc +
                                            col + e);
        }
    }
}

template <bool OUT_F32>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *ws, int m, int n, int S,
                                                           void *C, int64_t ldc, int vec,
                                                           int acc) {
    reduce_group<OUT_F32>(ws, m, n, S, C, ldc, vec != 0, OUT_F32 && acc != 0,
                          (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// The split reductions of the two backward products of one linear in one
// launch: blocks [0, blocks_d) reduce the backward-data product, the rest the
// backward-weight product.
struct ReduceJob {
    const float *ws;
    int m, n, S;
    void *C;
    int64_t ldc;
    int vec;
    int acc;   // fp32 output: add to C's contents
};

template <bool OD, bool OW>
__global__ __launch_bounds__(256) void split_reduce_pair_kernel(ReduceJob d, ReduceJob w,
                                                                int blocks_d) {
    const int b = blockIdx.x;
    if (b < blocks_d)
        reduce_group<OD>(d.ws, d.m, d.n, d.S, d.C, d.ldc, d.vec != 0, OD && d.acc != 0,
                         (int64_t)b * blockDim.x + threadIdx.x);
    else
        reduce_group<OW>(w.ws, w.m, w.n, w.S, w.C, w.ldc, w.vec != 0, OW && w.acc != 0,
                         (int64_t)(b - blocks_d) * blockDim.x + threadIdx.x);
}

}  // namespace sbpk

namespace sbpi {

// Whether every 4-column group of C can be stored with one aligned vector
// store: 16 bytes for fp32, 8 for bf16.
static int reduce_vec(const Gemm &g) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(g.C);
    const uintptr_t align = g.out_dtype == DT_F32 ? 16 : 8;
    return (a % align == 0 && g.ldc % 4 == 0) ? 1 : 0;
}

hipError_t launch_split_reduce(const Gemm &g, int splits, const float *ws, hipStream_t s) {
    const int64_t groups = g.m * ((g.n + 3) / 4);
    const unsigned blocks = (unsigned)((groups + 255) / 256);
    const int vec = reduce_vec(g);
    if (g.out_dtype == DT_F32)
        return launch_kernel(sbpk::split_reduce_kernel<true>, "split_reduce_kernel<true>",
                             dim3(blocks), dim3(256), s, ws, (int)g.m, (int)g.n, splits, g.C,
                             g.ldc, vec, g.accumulate);
    return launch_kernel(sbpk::split_reduce_kernel<false>, "split_reduce_kernel<false>",
                         dim3(blocks), dim3(256), s, ws, (int)g.m, (int)g.n, splits, g.C, g.ldc,
                         vec, 0);
}

static unsigned reduce_blocks(const Gemm &g) {
    const int64_t groups = g.m * ((g.n + 3) / 4);
    return (unsigned)((groups + 255) / 256);
}

hipError_t launch_split_reduce_pair(const Gemm &gd, int sd, const float *wsd, const Gemm &gw,
                                    int sw, const float *wsw, hipStream_t s) {
    const sbpk::ReduceJob d{wsd, (int)gd.m, (int)gd.n, sd, gd.C, gd.ldc, reduce_vec(gd),
                            gd.accumulate};
    const sbpk::ReduceJob w{wsw, (int)gw.m, (int)gw.n, sw, gw.C, gw.ldc, reduce_vec(gw),
                            gw.accumulate};
    const unsigned bd = reduce_blocks(gd), bw = reduce_blocks(gw);
    const bool od = gd.out_dtype == DT_F32, ow = gw.out_dtype == DT_F32;
#define SBP_PAIR(OD_, OW_, NAME)                                                             \
    if (od == OD_ && ow == OW_)                                                              \
        return launch_kernel(sbpk::split_reduce_pair_kernel<OD_, OW_>, NAME, dim3(bd + bw),  \
                             dim3(256), s, d, w, (int)bd);
    SBP_PAIR(true, true, "split_reduce_pair_kernel<true, true>")
    SBP_PAIR(true, false, "split_reduce_pair_kernel<true, false>")
    SBP_PAIR(false, true, "split_reduce_pair_kernel<false, true>")
    SBP_PAIR(false, false, "split_reduce_pair_kernel<false, false>")
#undef SBP_PAIR
    return hipErrorInvalidValue;
}

}  // namespace sbpi
