// Building blocks of the wide-layer matrix-core kernels (gemm_wide.hip for
// the forward, gemm_wide_bwd.hip for the gradients): 256 x 256 output tiles
// on 512-thread workgroups, 32-deep reduction chunks staged in LDS in a ring
// of four stages, v_mfma_f32_16x16x32_bf16 on 128 x 64 blocks per wavefront.
//
// A staged operand tile of one chunk holds 256 rows of the output dimension
// by 32 reduction elements (bf16, 16 KB) in one of two layouts:
//  * N ("normal"): row-major [256][32], for operands whose rows run along
//    the reduction in memory (A rows in the forward, G rows in dA).  Rows
//    are 64 bytes; their four 16-byte granules are XOR-swizzled by bits 1..2
//    of the row, so that the fragment reads (16 rows of one granule) are
//    free of bank conflicts.
//  * T ("transposed"): [32][256], reduction-major, for operands whose
//    reduction runs down the rows of a row-major matrix (A and G in dW).
//    Rows are 512 bytes of 32 16-byte units; unit u of reduction row k sits
//    at u ^ 2 ((k & 3) + 4 ((k >> 3) & 3)).  A fragment is read with two
//    ds_read_b64_tr_b16: in each group of 16 lanes, the lane that gives the
//    address of row k0 + t / 4, columns c0 + 4 (t % 4) .. + 3 receives
//    column c0 + t of rows k0 .. k0 + 3; the swizzle spreads the 16 rows one
//    such read touches over distinct banks.
#pragma once

#include "internal.h"

namespace gnn {
namespace wide {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kTile = 256;        // output tile edge
constexpr int kBK = 32;           // reduction chunk
constexpr int kStages = 4;        // LDS ring
constexpr int kXcds = 8;
constexpr int kTileElems = kTile * kBK;  // one operand tile of one chunk, bf16 elements

// s_waitcnt immediate: vmcnt(vm) expcnt(7, no wait) lgkmcnt(lgkm)
constexpr int waitcnt(int vm, int lgkm) { return (vm & 15) | ((vm >> 4) << 14) | 0x70 | ((lgkm & 15) << 8); }

// N layout: element (row r, reduction k) of a staged tile
__device__ __forceinline__ int sw_idx(int r, int k) { return r * kBK + ((((k >> 3) ^ ((r >> 1) & 3))) << 3) + (k & 7); }

// T layout: physical 16-byte unit of logical unit u in reduction row k, and
// the element index of (reduction k, column c)
__device__ __forceinline__ int t_unit(int k, int u) { return u ^ (((k & 3) | ((k >> 1) & 12)) << 1); }
__device__ __forceinline__ int t_idx(int k, int c) { return k * kTile + (t_unit(k, c >> 3) << 3) + (c & 7); }

// MFMA operand fragment of 16 tile rows starting at r0: lane l holds row
// r0 + l % 16, reduction elements 8 (l / 16) .. + 7.
__device__ __forceinline__ bf16x8 frag_n(const uint16_t *S, int r0, int lane) {
    return *reinterpret_cast<const bf16x8 *>(S + sw_idx(r0 + (lane & 15), (lane >> 4) * 8));
}
__device__ __forceinline__ bf16x8 frag_t(const uint16_t *S, int r0, int lane) {
    const int k = (lane >> 4) * 8 + ((lane >> 2) & 3), c = r0 + 4 * (lane & 3);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(S + t_idx(k, c)));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(S + t_idx(k + 4, c)));
    const i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
}
template <bool T> __device__ __forceinline__ bf16x8 frag(const uint16_t *S, int r0, int lane) {
    if constexpr (T) return frag_t(S, r0, lane);
    else return frag_n(S, r0, lane);
}

// Wait for this wavefront's outstanding copies and LDS accesses as WAIT
// says, then meet the other wavefronts.  The scheduling barriers keep the
// compiler from moving LDS accesses across.
template <int WAIT> __device__ __forceinline__ void chunk_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(WAIT);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
    return static_cast<uint32_t>(f32_to_bf16(x)) | (static_cast<uint32_t>(f32_to_bf16(y)) << 16);
}

}  // namespace wide
}  // namespace gnn
