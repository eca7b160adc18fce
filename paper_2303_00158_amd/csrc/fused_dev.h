// Pieces shared by the fused layer kernels (fused_layer.hip: one layer per
// launch; fused_two.hip: both layers of a two-layer model per launch): the
// workgroup shape, bf16 weight fragments for the matrix cores, feature
// chunks of bf16 rows and the softmax cross-entropy epilogue of the last
// layer.
#pragma once

#include "internal.h"

namespace gnn {
namespace fl {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kLogitLd = 65;  // row stride of the staged logits (fp32)
constexpr int kNbr = 16;      // neighbour loads in flight per aggregation item

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Kernel arguments are read with scalar loads, which the compiler otherwise
// places next to their first use: several dependent round trips to the
// argument buffer before the first vector load.  Naming every field in an
// empty asm statement at entry makes all of them one batch of loads.
template <class T> __device__ __forceinline__ void in_sgpr(const T &v) { asm volatile("" ::"s"(v)); }

// A 16-byte MFMA operand fragment of bf16 W^T: elements k .. k+7 of the row
// starting at element `row`.  W16 (K a multiple of 8, W^T 16-byte aligned):
// one 16-byte load, indices past K read the row's last eight elements;
// otherwise two 8-byte halves (K is a multiple of 4), indices past K read
// the last four.  Those values are not zeroed: they meet A entries that are
// zero (the A tile's padding), so a finite weight there contributes exactly
// 0.  A wavefront's fragment is then 16 rows x 64 contiguous bytes.  Offsets
// are 32-bit (W^T is far below 4 GiB) and the loads are unconditional and
// branch-free: they are the first thing a wavefront issues, and a branch
// around them would make the compiler wait for all of them at its join.
template <bool W16>
__device__ __forceinline__ bf16x8 load_wfrag(const uint16_t *wt, uint32_t row, uint32_t K, uint32_t k) {
    const char *base = reinterpret_cast<const char *>(wt);
    if constexpr (W16) {
        return *reinterpret_cast<const bf16x8 *>(base + 2u * (row + min(k, K - 8)));
    } else {
        const uint32_t last = K - 4;
        const uint2 lo = *reinterpret_cast<const uint2 *>(base + 2u * (row + min(k, last)));
        const uint2 hi = *reinterpret_cast<const uint2 *>(base + 2u * (row + min(k + 4u, last)));
        return __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
    }
}

// Features e0 .. e0 + CW - 1 (CW = 4 or 8 bf16, one 8- or 16-byte access) of
// a row, as floats.
template <int CW> struct Chunk;
template <> struct Chunk<4> {
    using raw = uint2;
    float v[4];
    __device__ __forceinline__ static raw load(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ __forceinline__ void set(raw u) {
        v[0] = __uint_as_float(u.x << 16);
        v[1] = __uint_as_float(u.x & 0xffff0000u);
        v[2] = __uint_as_float(u.y << 16);
        v[3] = __uint_as_float(u.y & 0xffff0000u);
    }
    __device__ __forceinline__ raw bf16() const {
        return make_uint2(static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                          static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16));
    }
    __device__ __forceinline__ static void store(uint16_t *p, raw u) { *reinterpret_cast<uint2 *>(p) = u; }
    __device__ __forceinline__ static raw zero() { return make_uint2(0u, 0u); }
};
template <> struct Chunk<8> {
    using raw = uint4;
    float v[8];
    __device__ __forceinline__ static raw load(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }
    __device__ __forceinline__ void set(raw u) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ __forceinline__ raw bf16() const {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = static_cast<uint32_t>(f32_to_bf16(v[2 * i])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * i + 1])) << 16);
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
    __device__ __forceinline__ static void store(uint16_t *p, raw u) { *reinterpret_cast<uint4 *>(p) = u; }
    __device__ __forceinline__ static raw zero() { return make_uint4(0u, 0u, 0u, 0u); }
};

// Softmax cross-entropy of one staged logit row zr (n_out values, the
// last layer's output Z = H W + b; Section II-B's loss), by the TPR threads
// j = 0 .. TPR-1 of a group inside one wavefront: the row's loss
// log(sum exp z) - z_y, the gradient (softmax - onehot(y)) / b of the mean
// loss, and the logits themselves.  Every thread of the group runs the
// shuffles; only `live` groups (a target row of the mini-batch) store.
// g_bf (optional, LDS): the row's gradient rounded to bf16 (as floats), the
// left operand of dA = G W^T; columns n_out .. gpad - 1, and every column of
// a row that is not live, are zero.
template <int TPR>
__device__ __forceinline__ void softmax_ce_row(const float *zr, int j, bool live, int64_t row, int64_t y,
                                               int64_t n_out, int64_t b, float *logits, float *g, float *row_loss,
                                               float *g_bf = nullptr, int gpad = 0) {
    float mx = -INFINITY;
    for (int n = j; n < n_out; n += TPR) mx = fmaxf(mx, zr[n]);
#pragma unroll
    for (int o = TPR / 2; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    float s = 0.f;
    for (int n = j; n < n_out; n += TPR) s += expf(zr[n] - mx);
#pragma unroll
    for (int o = TPR / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (live) {
        const float lse = mx + logf(s);
        const float inv_b = 1.f / static_cast<float>(b);
        float *lg = logits + row * n_out;
        for (int n = j; n < n_out; n += TPR) {
            const float p = expf(zr[n] - lse);
            const float gn = (p - (n == y ? 1.f : 0.f)) * inv_b;
            g[row * n_out + n] = gn;
            lg[n] = zr[n];
            if (g_bf) g_bf[n] = bf16_to_f32(f32_to_bf16(gn));
        }
        if (j == 0) row_loss[row] = lse - zr[y];
    }
    if (g_bf)
        for (int n = live ? static_cast<int>(n_out) + j : j; n < gpad; n += TPR) g_bf[n] = 0.f;
}

}  // namespace fl
}  // namespace gnn
