// Host-side interface of the block convolution engines (conv_blk.hip): the
// forward and input-gradient convolutions over a block plan (plan.hip), with
// each 16-row block's sums held in registers.
#pragma once

#include "conv_common.h"

namespace gsc {

// A block plan: perm[i] = output row at position i; block b covers positions
// 16b..16b+15, its offsets are the set bits of bmask[b], and its items
// (one per offset, in increasing offset order) start at ibase[b]; item t
// holds the 16 input rows items[16t .. 16t+15] (-1 = none).
struct BlockPlan {
    const int32_t* perm;
    const uint32_t* bmask;
    const int64_t* ibase;
    const int32_t* items;
};

// fp32 engine: reduction width ca and output width cb in {16, 32, 64}, with
// the K weight matrices held in LDS (K * ca * cb * 4 bytes within the
// engine's LDS budget).
bool blk_f32_supported(int ca, int cb, int K);

// Y (n_y x cb) = sum over the plan's items of X[item rows] * B_k with
// B_k = W[k] (ca x cb) when !wt, or B_k = W[sel(k)]^T (W: K x cb x ca) when
// wt; with accum, Y += that sum instead.  Asynchronous.
// A forward call (!wt) may carry an epilogue, applied to the sums (with
// accum: to Y plus the sums) before they are stored.
int conv_blk_f32(int ca, int cb, const float* X, int64_t n_x, const float* W, bool wt, const WSel& sel, int K,
                 const BlockPlan& plan, int64_t n_y, float* Y, hipStream_t s, const Epilogue& ep = Epilogue{},
                 bool accum = false);

// bf16 engine for wide layers: reduction width ca and output width cb in
// {64, 128, 256}, K <= 32.  Y (n_y x cb, bf16) = sum over the plan's items
// of X[item rows] * B_k, B_k[ch][col] = Bt[sel(k)][col][ch] (Bt: K x cb x ca
// bf16: the transposed weights for the forward pass, W itself for the input
// gradient).  The forward call (Sel = WIdentity) may carry an epilogue,
// applied to the fp32 sums before they are rounded.  Asynchronous.
bool blk_bf16_supported(int ca, int cb, int K);
// The engine addresses X with 32-bit byte offsets: n_x * ca below 2^30.
bool blk_bf16_fits(int64_t n_x, int ca);
template <typename Sel>
int conv_blk_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const Sel& sel, int K,
                  const BlockPlan& plan, int64_t n_y, void* Y, hipStream_t s, const Epilogue& ep = Epilogue{});

// The bf16 tile engine (conv_tile.hip): the same product as conv_blk_bf16
// for ca, cb in {64, 128, 256}, K <= 29, a tile of 16 blocks by all cb
// columns per workgroup, persistent workgroups.  nb = number of plan blocks;
// counter (nullable): 4 bytes of device memory the call uses to hand out
// tiles (large ones first; without it the tiles go out in a fixed order),
// set to 0 by the call unless counter_ready (an earlier launch on the stream
// did).  n_x * ca below 2^30.  Asynchronous.
bool tile_bf16_supported(int ca, int cb, int K);
template <typename Sel>
int conv_tile_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const Sel& sel, int K,
                   const BlockPlan& plan, int64_t nb, int64_t n_y, void* Y, unsigned* counter, hipStream_t s,
                   const Epilogue& ep, bool counter_ready = false);

// Weight gradient of a wide bf16 layer (conv_tile.hip), ci, co in {128,
// 256): the partial sum of each work item (dw_item) over its pairs, written
// to part[item] (ci x co float32); grid = items.  Asynchronous.
bool dw_tile_bf16_supported(int ci, int co);
int dw_tile_bf16(int ci, int co, const void* X, int64_t n_in, const void* dY, int64_t n_out, const int32_t* in_idx,
                 const int32_t* out_idx, const int64_t* seg, const int64_t* ibase, const int64_t* chunk, int K,
                 int64_t items, float* part, hipStream_t s);

// Y (n x c, float32 or bf16 by dtype) = the epilogue applied in place (the
// row-form paths, whose sums are complete only in Y).  Asynchronous.
int affine_act(int dtype, void* Y, int64_t n, int c, const Epilogue& ep, hipStream_t s);

}  // namespace gsc
