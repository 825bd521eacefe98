// Host-side interface of the bfloat16 large-channel convolution engine
// (conv_bf16.hip), used by the C entry points in conv.hip.
#pragma once

#include "conv_common.h"

namespace gsc {

// Output-stationary forward / input-gradient kernel for bf16 with reduction
// width ca and output width cb (ca in {32, 64, 128, 256}, cb in {64, 128,
// 256}, K <= 64).
bool conv_bf16_supported(int ca, int cb, int K);

// Y (n_y x cb) = sum over the map of X[gat] * B_sel(k), B_w[k][col] =
// Bt[w][col][k] (Bt: K x cb x ca).  perm (nullable) maps output positions to
// rows.  Asynchronous.
template <typename Sel>
int conv_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const int32_t* gat, const int32_t* sca,
              const int64_t* gidx, const int32_t* perm, int K, int64_t n_y, void* Y, Sel sel, hipStream_t s);

// Bt[w][col][k] = W[w][k][col] for K matrices of rows x cols bf16; sets
// *zero_counter (nullable, device memory) to 0 on the way.
size_t transpose_ws_bytes(int K, int rows, int cols);
int transpose_w_bf16(const void* W, int K, int rows, int cols, void* Bt, hipStream_t s,
                     unsigned* zero_counter = nullptr);

// Weight-gradient partials for bf16 with ci, co multiples of 128.
bool dw_bf16_supported(int ci, int co);
int dw_bf16(int ci, int co, const void* X, int64_t n_in, const void* dY, int64_t n_out, const int32_t* in_idx,
            const int32_t* out_idx, const int64_t* seg, const int64_t* ibase, const int64_t* chunk, int K,
            int64_t items, float* part, hipStream_t s);

}  // namespace gsc
