// gemm.h -- internal interface between the C-ABI host code and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sbpi {

// Operand orientation of the three local products (see gemm_bf16_kernel.h):
//   FWD         A k-major, B n-major     (Y  = X  W)
//   BWD_DATA    A k-major, B k-major     (dX = dY W^T)
//   BWD_WEIGHT  A m-major, B n-major     (dW = X^T dY)
enum Orient { OR_FWD = 0, OR_BWD_DATA = 1, OR_BWD_WEIGHT = 2 };

// dtype codes match sbp_dtype_t
enum { DT_BF16 = 0, DT_F32 = 1 };

struct Gemm {
    int orient;
    int in_dtype;
    int out_dtype;
    const void *A;
    int64_t lda;
    const void *B;
    int64_t ldb;
    void *C;
    int64_t ldc;
    int64_t m, n, k;
    int accumulate = 0;    // fp32 output only: C += product instead of C = product
    // fp32 elements of caller workspace this product may use for split
    // partials (0: the reduction is never split)
    size_t ws_floats = 0;
    // batched products (attention core): batches x heads independent
    // products; element strides between consecutive batches / heads of A, B, C
    int64_t batches = 1, heads = 1;
    int64_t sa_b = 0, sa_h = 0, sb_b = 0, sb_h = 0, sc_b = 0, sc_h = 0;
    int64_t nbatch() const { return batches * heads; }
};

struct Plan {
    int bm, bn;            // output tile
    int splits;            // reduction splits actually launched
    int kblk_per_split;    // 64-wide reduction blocks per split
    bool dma;              // pipelined direct-to-LDS kernel (else the generic kernel)
    int ns = 0;            // pipelined kernel: stages (0 = the tile's default)
    int kg = 1;            // pipelined kernel: reduction groups of waves (1 or 2)
    int epi = 0;           // pipelined kernel: epilogue (sbpk::EPI_DIRECT / _STAGED / _ROWQ)
    int occ = 0;           // persistent workgroups per compute unit (0: one per work item)
    int bk = 64;           // pipelined kernel: reduction elements per stage (64 or 32)
    bool shift = false;    // pipelined kernel in the shifted index space (see dma_mode)
};

// Compute units of the current device (cached per device).
int device_cus();

// Whether the pipelined direct-to-LDS kernel can run this product: leading
// dimensions multiples of 8 elements (so every row of an operand sits at the
// same offset within a 16-byte block), an offset along the reduction only
// where both operands are k-major and share it, tile offsets that fit
// 31-bit buffer offsets; batched products need aligned operands.
bool dma_eligible(const Gemm &g);
// 0: the generic kernel; 1: the pipelined kernel (operands 16-byte aligned,
// contiguous extents multiples of 8); 2: the pipelined kernel's shifted
// form (dma_eligible, but not 1), which only the instances of
// SBP_DMA_SHIFT_INSTANCES have.
int dma_mode(const Gemm &g);
// Offset in elements of a bf16 pointer within its 16-byte block.
int block_offset(const void *p);

// Row stride (floats) of a split reduction's partial slices for an m x n
// output: n rounded up to a multiple of 4, so that every 4-column group of a
// slice is one aligned 16-byte load in the reduction (the padding columns
// are never written or stored).
__host__ __device__ inline int64_t partial_ld(int64_t n) { return (n + 3) & ~int64_t(3); }

// Workspace of the split reduction: `splits` slices of m x partial_ld(n)
// fp32 partials.
// Plans never use more than WS_FLOATS_PREFERRED floats, however large the
// caller's workspace, so that a workspace of that size always gets the
// library's preferred plan (the value of SBP_WORKSPACE_BYTES / 4).
constexpr size_t WS_FLOATS_PREFERRED = size_t(16) << 20;   // 64 MiB

// bf16 planning: heuristic choice of tile and splits (an override may be set
// per thread through sbp_set_plan_override). The partials of a split plan
// always fit g.ws_floats; with no workspace the reduction is not split.
Plan plan_bf16(const Gemm &g);
bool tile_supported(int bm, int bn, bool dma);
void set_override(int bm, int bn, int splits, int kernel);   // bm = 0 clears
void set_override_occ(int occ);                              // 0: one workgroup per item
void set_override_orients(int mask);   // bit o: the override applies to orientation o
void set_bwd_override(int mode, int splits_w);   // 0 default, 1 separate, 2 grouped
bool override_supported(int bm, int bn, int kernel);
int kernel_code(const Plan &p);   // kernel code of a plan, as sbp_plan reports it

// Workspace floats a plan's partials take (0 without splits).
size_t plan_ws_floats(const Gemm &g, const Plan &p);

// GEMM of plan p; with p.splits > 1 it writes partials to ws and then runs
// the split reduction into g.C.
hipError_t launch_bf16(const Gemm &g, const Plan &p, float *ws, hipStream_t s);
// Adds the splits' partials (in split order) and stores them into g.C, or
// adds the sum to g.C's contents when g.accumulate.
hipError_t launch_split_reduce(const Gemm &g, int splits, const float *ws, hipStream_t s);
// Both split reductions of a grouped backward launch, in one launch.
hipError_t launch_split_reduce_pair(const Gemm &gd, int sd, const float *wsd, const Gemm &gw,
                                    int sw, const float *wsw, hipStream_t s);

// Backward-data (gd) and backward-weight (gw) products of one linear. If
// plan_bf16_bwd returns true, *pd and *pw share a pipelined tile and
// launch_bf16_bwd_group runs both in one grid (then the split reductions);
// otherwise the two products run as separate launches of their own plans.
// Both products share one workspace of gd.ws_floats floats (gw.ws_floats
// must be equal): a grouped plan's partials of both fit it together.
bool plan_bf16_bwd(const Gemm &gd, const Gemm &gw, Plan *pd, Plan *pw);
hipError_t launch_bf16_bwd_group(const Gemm &gd, const Plan &pd, const Gemm &gw,
                                 const Plan &pw, float *ws, hipStream_t s);
hipError_t launch_f32(const Gemm &g, hipStream_t s);

// The library's static scratch on the current device (its address there,
// looked up once per device) and its size in floats (WS_FLOATS_PREFERRED).
hipError_t static_scratch(float **ptr, size_t *floats);

}  // namespace sbpi
