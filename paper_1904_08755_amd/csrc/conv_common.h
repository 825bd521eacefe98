// Device helpers shared by the convolution kernels (conv.hip, conv_bf16.hip).
#pragma once

#include "gsc_internal.h"

namespace gsc {

constexpr int kMaxKConv = 1024;   // offsets per convolution call

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef short shortx4 __attribute__((ext_vector_type(4)));

struct WSel {
    int16_t w[kMaxKConv];
    __device__ __forceinline__ int operator()(int k) const { return w[k]; }
};
struct WIdentity {
    __device__ __forceinline__ int operator()(int k) const { return k; }
};

// Per-output-channel affine map and activation applied to a convolution's
// fp32 sums before they are stored: y[c] = act(sum[c] * scale[c] + shift[c])
// (batch normalisation in its inference form followed by a ReLU: non-spatial
// functions of Sec. 4.5 fused into the kernel that produces the rows).
struct Epilogue {
    const float* scale = nullptr;   // null: 1
    const float* shift = nullptr;   // null: 0
    int relu = 0;
    bool on() const { return scale || shift || relu; }
};

// NaN propagates through the ReLU (a NaN sum is not clipped to 0)
__device__ __forceinline__ float epi_apply(float v, float sc, float sh, int relu) {
    v = fmaf(v, sc, sh);
    return relu && v < 0.f ? 0.f : v;
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void store_out(float* y, float v) { *y = v; }
__device__ __forceinline__ void store_out(uint16_t* y, float v) { *y = f32_to_bf16_rne(v); }

// B operand element: forward uses W[w] (ca x cb), the input gradient W[w]^T.
template <typename TIn, bool WT>
__device__ __forceinline__ TIn w_at(const TIn* W, int w, int brow, int col, int ca, int cb) {
    if (WT) return W[((int64_t)w * cb + col) * ca + brow];
    return W[((int64_t)w * ca + brow) * cb + col];
}

// offset and pair range of a work item
__device__ __forceinline__ bool dw_item(const int64_t* ibase, const int64_t* chunk, const int64_t* seg, int K,
                                        int64_t item, int* k_out, int64_t* p_begin, int64_t* p_end) {
    if (item >= ibase[K]) return false;
    int lo = 0, hi = K - 1;   // last k with ibase[k] <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (ibase[mid] <= item) lo = mid; else hi = mid - 1;
    }
    *k_out = lo;
    *p_begin = seg[lo] + (item - ibase[lo]) * chunk[lo];
    *p_end = min(seg[lo + 1], *p_begin + chunk[lo]);
    return true;
}

}  // namespace gsc
