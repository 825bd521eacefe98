// Sparse convolution engine: forward (a4), transposed forward (a5, the same
// kernel on the role-reversed map), input gradient (a6) and weight gradient
// (a7).
//
// Forward / input gradient: output-stationary.  A workgroup owns a tile of
// 128 consecutive output rows and up to 64 output columns, accumulated in
// LDS.  For each offset it finds the pairs whose output row lies in the tile
// through the kernel map's 64-row group index (pairs of one offset are sorted
// by output row, so they are contiguous), gathers the input rows 16 pairs at
// a time as the A operand of an MFMA tile, multiplies by the offset's weight
// and adds the 16 result rows into the LDS tile.  Each output row is written
// to HBM once, with no global atomics and no zero-fill pass.
//
// Weight gradient: split-K over the pairs of each offset.  A workgroup
// reduces a chunk of one offset's pairs into a 64 x 64 fp32 tile (MFMA with
// the pair index as the reduction dimension) and stores it as a partial; a
// second kernel adds the partials of each offset in a fixed order.
#include <climits>
#include <vector>

#include "conv_common.h"
#include "conv_bf16.h"
#include "conv_blk.h"

namespace gsc {

constexpr int kThreads = 256;
constexpr int kTileRows = 128;
constexpr int kTileGroups = kTileRows / GSC_GROUP_ROWS;
constexpr int kColSlice = 64;
constexpr int kAccStride = kColSlice + 1;
constexpr int kDwTile = 64;

// ---------------------------------------------------------------------------
// output-stationary gather -> MFMA -> LDS accumulate
//   Y[sca[p]] += X[gat[p]] * B_w  for every pair p of segment k, w = sel(k)
//   X: n_x x ca, Y: n_y x cb, B_w = W[w] (ca x cb) or W[w]^T.
// ---------------------------------------------------------------------------
template <typename TIn, typename TOut, bool WT, typename Sel>
__global__ void __launch_bounds__(kThreads)
k_conv_os(const TIn* __restrict__ X, int64_t n_x, const TIn* __restrict__ W, const int32_t* __restrict__ gat,
          const int32_t* __restrict__ sca, const int64_t* __restrict__ gidx, const int32_t* __restrict__ perm, int K,
          int64_t G, int ca, int cb, int64_t n_y, TOut* __restrict__ Y, Sel sel) {
    __shared__ float acc[kTileRows * kAccStride];
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t tile = tile_unit(blockIdx.x, gridDim.x, perm != nullptr);
    const int64_t row0 = tile * kTileRows;
    const int col0 = blockIdx.y * kColSlice;
    const int ncols = min(kColSlice, cb - col0);
    const int nnb = (ncols + 15) >> 4;

    for (int i = tid; i < kTileRows * kAccStride; i += kThreads) acc[i] = 0.f;
    __syncthreads();

    const int64_t g0 = tile * kTileGroups;
    const int64_t g1 = min(g0 + kTileGroups, G);
    int item = 0;
    for (int k = 0; k < K; ++k) {
        const int64_t lo = gidx[(int64_t)k * G + g0];
        const int64_t hi = gidx[(int64_t)k * G + g1];
        const int64_t np = hi - lo;
        for (int64_t pb = 0; pb < np; pb += 16, ++item) {
            if ((item & 3) != wave) continue;
            const int w = sel(k);
            const int64_t p = lo + pb + r16;
            const bool in_grp = pb + r16 < np;
            int32_t gr = in_grp ? gat[p] : 0;
            int32_t sr = in_grp ? sca[p] : 0;
            const bool pv = in_grp && gr >= 0 && gr < n_x && sr >= row0 && sr < row0 + kTileRows;
            floatx4 d[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) d[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
            if constexpr (sizeof(TIn) == 4) {
                // fp32: v_mfma_f32_16x16x4_f32, A[row][kk] = X[gat][kb + kk], lane = (row, kk)
                for (int kb = 0; kb < ca; kb += 4) {
                    const int ch = kb + q;
                    const float a = (pv && ch < ca) ? to_f32(X[(int64_t)gr * ca + ch]) : 0.f;
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        if (nb < nnb) {
                            const int col = col0 + nb * 16 + r16;
                            const float b = (ch < ca && col < cb) ? to_f32(w_at<TIn, WT>(W, w, ch, col, ca, cb)) : 0.f;
                            d[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, d[nb], 0, 0, 0);
                        }
                    }
                }
            } else {
                // bf16: v_mfma_f32_16x16x16_bf16, lane = (row, 4 consecutive kk)
                for (int kb = 0; kb < ca; kb += 16) {
                    shortx4 a;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int ch = kb + 4 * q + e;
                        a[e] = (pv && ch < ca) ? (short)X[(int64_t)gr * ca + ch] : (short)0;
                    }
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb) {
                        if (nb < nnb) {
                            const int col = col0 + nb * 16 + r16;
                            shortx4 b;
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const int brow = kb + 4 * q + e;
                                b[e] = (brow < ca && col < cb) ? (short)w_at<TIn, WT>(W, w, brow, col, ca, cb)
                                                               : (short)0;
                            }
                            d[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, d[nb], 0, 0, 0);
                        }
                    }
                }
            }
            // D row 4q + j of block nb belongs to pair row 4q + j, column r16
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int prow = 4 * q + j;
                const int32_t srow = __shfl(sr, prow, 64);
                const int valid_row = __shfl((int)pv, prow, 64);
                if (valid_row) {
                    float* a_row = acc + (int)(srow - row0) * kAccStride;
#pragma unroll
                    for (int nb = 0; nb < 4; ++nb)
                        if (nb < nnb && nb * 16 + r16 < ncols) atomicAdd(a_row + nb * 16 + r16, d[nb][j]);
                }
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < kTileRows * ncols; i += kThreads) {
        const int r = i / ncols, c = i - r * ncols;
        const int64_t pos = row0 + r;
        if (pos < n_y) {
            const int64_t row = perm ? (int64_t)perm[pos] : pos;
            store_out(Y + row * cb + col0 + c, acc[r * kAccStride + c]);
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 specialisation for reduction width CA and output width CB (multiples of
// 16, <= 64).  Differences from the generic kernel:
//   * the (offset, 16-pair group) items of a tile are split into four
//     contiguous ranges, one per wave, so a wave meets few distinct offsets and
//     keeps the offset's B fragments (CA/4 x CB/16 floats per lane) in
//     registers across its groups;
//   * lane (r16, q) gathers channels [q*CA/4, (q+1)*CA/4) of pair r16's row with
//     16-byte loads; MFMA step s then reduces over channels {q*CA/4 + s}, and B
//     uses the same channel permutation;
//   * the next group's row gather is issued before the current group's MFMAs.
// ---------------------------------------------------------------------------
template <int CA>
struct RowFrag {
    float v[CA / 4];
};

// Branch-free row fragment load: the address is always valid (row is
// clamped by the caller) and invalid pairs are zeroed with a select, so the
// loads of a batch are issued back to back with no wait between them.
template <int CA>
__device__ __forceinline__ void load_row_frag(const float* __restrict__ X, int64_t row, int q, bool ok,
                                              RowFrag<CA>& a) {
    constexpr int KS = CA / 4;
    const float4* src = reinterpret_cast<const float4*>(X + row * CA + q * KS);
#pragma unroll
    for (int i = 0; i < KS / 4; ++i) {
        const float4 t = src[i];
        a.v[4 * i + 0] = ok ? t.x : 0.f;
        a.v[4 * i + 1] = ok ? t.y : 0.f;
        a.v[4 * i + 2] = ok ? t.z : 0.f;
        a.v[4 * i + 3] = ok ? t.w : 0.f;
    }
}

constexpr int kMaxKLds = 256;   // offsets whose tile table fits in LDS (specialised kernels)
constexpr int kItemBatch = 4;   // items per wave in flight

// Per-tile offset table in LDS: pairs of offset k in this tile start at
// s_lo[k] (global pair index), there are s_np[k] of them, and its 16-pair
// items are numbered from s_ib[k]; s_ib[K] = items of the tile.
struct TileTable {
    int64_t lo[kMaxKLds];
    int32_t np[kMaxKLds];
    int32_t ib[kMaxKLds + 1];
};

__device__ __forceinline__ void build_tile_table(TileTable& t, const int64_t* __restrict__ gidx, int K, int64_t G,
                                                 int64_t g0, int64_t g1) {
    for (int k = threadIdx.x; k < K; k += kThreads) {
        const int64_t lo = gidx[(int64_t)k * G + g0];
        t.lo[k] = lo;
        t.np[k] = (int32_t)(gidx[(int64_t)k * G + g1] - lo);
    }
    __syncthreads();
    if (threadIdx.x < 64) {   // wave 0: exclusive scan of item counts
        int carry = 0;
        for (int k0 = 0; k0 < K; k0 += 64) {
            const int k = k0 + threadIdx.x;
            const int v = k < K ? (t.np[k] + 15) >> 4 : 0;
            int inc = v;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int u = __shfl_up(inc, d, 64);
                if ((int)threadIdx.x >= d) inc += u;
            }
            if (k < K) t.ib[k] = carry + inc - v;
            carry += __shfl(inc, 63, 64);
        }
        if (threadIdx.x == 0) t.ib[K] = carry;
    }
    __syncthreads();
}

// Wave-per-group fp32 kernel.  Each wave owns one 64-row group of output
// rows (the kernel map's group granularity) and accumulates it in a private
// LDS region with plain read-modify-write: no LDS atomics, no workgroup
// barriers, deterministic order.  The wave's per-offset table (first pair,
// pair count, first item) is held one offset per lane (K <= 64).
constexpr int kWaveKMax = 64;

template <int CA, int CB, bool WT, typename Sel>
__global__ void __launch_bounds__(kThreads)
k_conv_f32(const float* __restrict__ X, int64_t n_x, const float* __restrict__ W, const int32_t* __restrict__ gat,
           const int32_t* __restrict__ sca, const int64_t* __restrict__ gidx, const int32_t* __restrict__ perm, int K,
           int64_t G, int64_t n_y, float* __restrict__ Y, Sel sel) {
    constexpr int KS = CA / 4;
    constexpr int NNB = CB / 16;
    constexpr int AS = CB + 1;
    constexpr int RG = GSC_GROUP_ROWS;
    constexpr int B = CA * CB <= 1024 ? kItemBatch : kItemBatch / 2;   // bound the register footprint
    __shared__ float acc_all[kThreads / 64][RG * AS];
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t g = tile_unit(blockIdx.x, gridDim.x, perm != nullptr) * (kThreads / 64) + wave;
    if (g >= G) return;                        // no barrier below, so a wave may leave early
    float* acc = acc_all[wave];
    const int64_t row0 = g * RG;
    for (int i = lane; i < RG * AS; i += 64) acc[i] = 0.f;
    wave_lds_sync();

    // per-offset table, one offset per lane
    int64_t lo = 0;
    int np = 0;
    if (lane < K) {
        lo = gidx[(int64_t)lane * G + g];
        np = (int)(gidx[(int64_t)lane * G + g + 1] - lo);
    }
    const int nit = (np + 15) >> 4;
    int incl = nit;                            // inclusive scan of items over lanes
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int u = __shfl_up(incl, d, 64);
        if (lane >= d) incl += u;
    }
    const int excl = incl - nit;
    const int total = __shfl(incl, 63, 64);

    // pair indices of the batch starting at item0; every address is valid
    // (lanes past the end of a group re-read its last pair, items past the
    // end repeat the last item) and the invalid ones are masked
    auto fetch_idx = [&](int item0, int (&kb)[B], int32_t (&gr)[B], int32_t (&sr)[B], bool (&ok)[B]) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int item = min(item0 + b, total - 1);
            const int k = __popcll(__ballot(incl <= item));     // offset of the item
            kb[b] = k;
            const int64_t klo = __shfl(lo, k, 64);
            const int knp = __shfl(np, k, 64);
            const int pb = (item - __shfl(excl, k, 64)) * 16 + r16;
            const int64_t p = klo + min(pb, knp - 1);
            gr[b] = gat[p];
            sr[b] = sca[p];
            ok[b] = item0 + b < total && pb < knp;
        }
    };
    int kb[B], kbn[B];
    int32_t gr[B], sr[B], grn[B], srn[B];
    bool ok[B], okn[B];
    if (total > 0) fetch_idx(0, kb, gr, sr, ok);
    for (int item0 = 0; item0 < total; item0 += B) {
        // 1. rows and weights of the batch
        RowFrag<CA> a[B];
        float bfr[B][KS][NNB];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            ok[b] = ok[b] && gr[b] >= 0 && gr[b] < n_x && sr[b] >= row0 && sr[b] < row0 + RG;
            load_row_frag<CA>(X, ok[b] ? gr[b] : 0, q, ok[b], a[b]);
            const int w = sel(kb[b]);
            if constexpr (WT) {
                // W[w]^T: lane (r16, q) needs W[w][col][q*KS .. q*KS + KS), contiguous
#pragma unroll
                for (int nb = 0; nb < NNB; ++nb) {
                    const float4* src =
                        reinterpret_cast<const float4*>(W + ((int64_t)w * CB + nb * 16 + r16) * CA + q * KS);
#pragma unroll
                    for (int i = 0; i < KS / 4; ++i) {
                        const float4 t = src[i];
                        bfr[b][4 * i + 0][nb] = t.x;
                        bfr[b][4 * i + 1][nb] = t.y;
                        bfr[b][4 * i + 2][nb] = t.z;
                        bfr[b][4 * i + 3][nb] = t.w;
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < KS; ++s)
#pragma unroll
                    for (int nb = 0; nb < NNB; ++nb)
                        bfr[b][s][nb] = W[((int64_t)w * CA + q * KS + s) * CB + nb * 16 + r16];
            }
        }
        // 2. next batch's indices in flight during this batch's MFMAs
        if (item0 + B < total) fetch_idx(item0 + B, kbn, grn, srn, okn);
        // 3. group row of each MFMA output row (pair row 4q + j), -1 if none
        int lrow[B][4];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int mine = ok[b] ? (int)(sr[b] - row0) : -1;
#pragma unroll
            for (int j = 0; j < 4; ++j) lrow[b][j] = __shfl(mine, 4 * q + j, 64);
        }
        // 4. MFMA, then add the 16 result rows into the wave's rows (distinct
        //    within an item; items of the wave are applied in order)
#pragma unroll
        for (int b = 0; b < B; ++b) {
            floatx4 d[NNB];
#pragma unroll
            for (int nb = 0; nb < NNB; ++nb) d[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int nb = 0; nb < NNB; ++nb)
                    d[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[b].v[s], bfr[b][s][nb], d[nb], 0, 0, 0);
            wave_lds_sync();   // rows updated by other lanes for earlier items
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (lrow[b][j] >= 0) {
                    float* arow = acc + lrow[b][j] * AS;
#pragma unroll
                    for (int nb = 0; nb < NNB; ++nb) arow[nb * 16 + r16] += d[nb][j];
                }
            }
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            kb[b] = kbn[b];
            gr[b] = grn[b];
            sr[b] = srn[b];
            ok[b] = okn[b];
        }
    }
    wave_lds_sync();
    // 5. the group's rows, written once
    for (int i = lane; i < RG * CB; i += 64) {
        const int r = i / CB, cc = i - r * CB;
        const int64_t pos = row0 + r;
        if (pos < n_y) {
            const int64_t row = perm ? (int64_t)perm[pos] : pos;
            Y[row * CB + cc] = acc[r * AS + cc];
        }
    }
}

// ---------------------------------------------------------------------------
// weight gradient
// ---------------------------------------------------------------------------
// Work items of the weight gradient: offset k's pairs are split into chunks
// of `ch` pairs (the last one shorter); ibase[k] = first item of offset k,
// ibase[K] = total.  Equal chunks keep the work items balanced whatever the
// offsets' sizes (the centre offset of a submanifold map has one pair per
// row, the others far fewer).
// counter (nullable) is set to 0 on the way (the input gradient's tile
// counter, when that pass runs after this kernel).
__global__ void k_dw_items(const int64_t* seg, int K, int64_t ch, int64_t* ibase, int64_t* chunk,
                           unsigned* counter) {
    // one wave: 64 offsets per round, their item counts scanned with shuffles
    if (blockIdx.x != 0 || threadIdx.x >= 64) return;
    const int lane = threadIdx.x;
    if (counter && lane == 0) *counter = 0u;
    int64_t carry = 0;
    for (int k0 = 0; k0 < K; k0 += 64) {
        const int k = k0 + lane;
        const int64_t n = k < K ? seg[k + 1] - seg[k] : 0;
        const int64_t c = n > 0 ? (n + ch - 1) / ch : 0;
        int64_t inc = c;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t u = __shfl_up(inc, d, 64);
            if (lane >= d) inc += u;
        }
        if (k < K) {
            ibase[k] = carry + inc - c;
            chunk[k] = ch;
        }
        carry += __shfl(inc, 63, 64);
    }
    if (lane == 0) ibase[K] = carry;
}

// Per-wave partial tiles are summed in wave order (deterministic), then stored.
template <int R, int C>
__device__ __forceinline__ void dw_store_partial(float* sh, const floatx4 (&d)[4][4], int na, int nbk, int wave,
                                                 int q, int r16, int rows, int cols, float* __restrict__ out,
                                                 int64_t ld) {
    constexpr int S = C + 1;
    float* mine = sh + wave * R * S;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            if (a < na && b < nbk)
#pragma unroll
                for (int j = 0; j < 4; ++j) mine[(16 * a + 4 * q + j) * S + 16 * b + r16] = d[a][b][j];
    __syncthreads();
    for (int i = threadIdx.x; i < rows * cols; i += kThreads) {
        const int r = i / cols, c = i - r * cols;
        float v = sh[r * S + c];
        for (int w = 1; w < kThreads / 64; ++w) v += sh[w * R * S + r * S + c];
        out[r * ld + c] = v;
    }
}

// Generic weight-gradient partial (any dtype, any width): a 64 x 64 tile of
// X[in]^T dY[out] over one chunk of one offset's pairs.
template <typename TIn>
__global__ void __launch_bounds__(kThreads)
k_dw_partial(const TIn* __restrict__ X, int64_t n_in, const TIn* __restrict__ dY, int64_t n_out,
             const int32_t* __restrict__ in_idx, const int32_t* __restrict__ out_idx, const int64_t* __restrict__ seg,
             const int64_t* __restrict__ ibase, const int64_t* __restrict__ chunk, int K, int ci, int co,
             float* __restrict__ part) {
    __shared__ float sh[4 * kDwTile * (kDwTile + 1)];
    int k;
    int64_t p_begin, p_end;
    // the grid covers an upper bound of the items; order the real ones XCD-wise
    if ((int64_t)blockIdx.x >= ibase[K]) return;
    const int64_t item = xcd_unit(blockIdx.x, ibase[K]);
    if (!dw_item(ibase, chunk, seg, K, item, &k, &p_begin, &p_end)) return;
    const int ntj = (co + kDwTile - 1) / kDwTile;
    const int ci0 = (blockIdx.y / ntj) * kDwTile, co0 = (blockIdx.y % ntj) * kDwTile;
    const int na = (min(kDwTile, ci - ci0) + 15) >> 4, nbk = (min(kDwTile, co - co0) + 15) >> 4;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, q = lane >> 4;

    floatx4 d[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) d[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    if constexpr (sizeof(TIn) == 4) {
        // 4 pairs per MFMA step (reduction index kk = q); waves interleave steps
        for (int64_t p0 = p_begin + 4 * wave; p0 < p_end; p0 += 16) {
            const int64_t p = p0 + q;
            int32_t g = p < p_end ? in_idx[p] : -1;
            int32_t s = p < p_end ? out_idx[p] : -1;
            const bool v = g >= 0 && g < n_in && s >= 0 && s < n_out;
            float xa[4], yb[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int c = ci0 + 16 * a + r16;
                xa[a] = (v && a < na && c < ci) ? to_f32(X[(int64_t)g * ci + c]) : 0.f;
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int c = co0 + 16 * b + r16;
                yb[b] = (v && b < nbk && c < co) ? to_f32(dY[(int64_t)s * co + c]) : 0.f;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    if (a < na && b < nbk) d[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[a], yb[b], d[a][b], 0, 0, 0);
        }
    } else {
        // 16 pairs per MFMA step: lane (r16, q) supplies pairs 4q .. 4q+3
        for (int64_t p0 = p_begin + 16 * wave; p0 < p_end; p0 += 64) {
            int32_t g[4], s[4];
            bool v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t p = p0 + 4 * q + e;
                g[e] = p < p_end ? in_idx[p] : -1;
                s[e] = p < p_end ? out_idx[p] : -1;
                v[e] = g[e] >= 0 && g[e] < n_in && s[e] >= 0 && s[e] < n_out;
            }
            shortx4 xa[4], yb[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int c = ci0 + 16 * a + r16;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    xa[a][e] = (v[e] && a < na && c < ci) ? (short)X[(int64_t)g[e] * ci + c] : (short)0;
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int c = co0 + 16 * b + r16;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    yb[b][e] = (v[e] && b < nbk && c < co) ? (short)dY[(int64_t)s[e] * co + c] : (short)0;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    if (a < na && b < nbk)
                        d[a][b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(xa[a], yb[b], d[a][b], 0, 0, 0);
        }
    }
    // D[m][n]: m = 4q + j (input channel), n = r16 (output channel)
    const int rows = min(kDwTile, ci - ci0), cols = min(kDwTile, co - co0);
    dw_store_partial<kDwTile, kDwTile>(sh, d, na, nbk, wave, q, r16, rows, cols,
                                       part + (item * ci + ci0) * (int64_t)co + co0, co);
}

// fp32 weight gradient for CI x CO <= 64 x 64 (multiples of 16).  Each wave
// stages 32 pairs at a time in a private LDS buffer: lane l loads half a row
// of X[in_idx] and of dY[out_idx] for pair l % 32 with 16-byte loads (all
// addresses valid: pairs past the chunk are clamped and their dY half-rows
// zeroed by a select), then eight 16x16x4 MFMA steps reduce the 32 pairs,
// reading A = X rows and B = dY rows from LDS.
constexpr int kDwStage = 32;

// Row halves of the 32-pair sub-chunk at p0: lane (pr, half) loads half of
// X[in_idx[p0 + pr]] and of dY[out_idx[p0 + pr]].  Every address is valid
// (pairs past the chunk are clamped) and their dY half-rows are zeroed.
template <int CI, int CO>
struct DwRows {
    float4 x[CI / 8];
    float4 y[CO / 8];
};

template <int CI, int CO>
__device__ __forceinline__ DwRows<CI, CO> dw_fetch(const float* __restrict__ X, const float* __restrict__ dY,
                                                   const int32_t* __restrict__ in_idx,
                                                   const int32_t* __restrict__ out_idx, int64_t n_in, int64_t n_out,
                                                   int64_t p0, int64_t p_end, int pr, int half) {
    DwRows<CI, CO> r;
    const int64_t p = min(p0 + pr, p_end - 1);
    int32_t g = in_idx[p], sidx = out_idx[p];
    const bool v = p0 + pr < p_end && g >= 0 && g < n_in && sidx >= 0 && sidx < n_out;
    g = v ? g : 0;
    sidx = v ? sidx : 0;
    const float4* xr = reinterpret_cast<const float4*>(X + (int64_t)g * CI + half * (CI / 2));
    const float4* yr = reinterpret_cast<const float4*>(dY + (int64_t)sidx * CO + half * (CO / 2));
#pragma unroll
    for (int i = 0; i < CI / 8; ++i) r.x[i] = xr[i];
#pragma unroll
    for (int i = 0; i < CO / 8; ++i) {
        const float4 t = yr[i];
        r.y[i] = v ? t : float4{0.f, 0.f, 0.f, 0.f};
    }
    return r;
}

template <int CI, int CO>
__global__ void __launch_bounds__(kThreads)
k_dw_f32(const float* __restrict__ X, int64_t n_in, const float* __restrict__ dY, int64_t n_out,
         const int32_t* __restrict__ in_idx, const int32_t* __restrict__ out_idx, const int64_t* __restrict__ seg,
         const int64_t* __restrict__ ibase, const int64_t* __restrict__ chunk, int K, float* __restrict__ part) {
    constexpr int NA = CI / 16, NB = CO / 16;
    constexpr int XS = CI + 4, YS = CO + 4;            // row strides (16-byte aligned rows)
    constexpr int STAGE = kDwStage * (XS + YS);
    constexpr int RED = CI * (CO + 1);
    constexpr int SH = (STAGE > RED ? STAGE : RED) * (kThreads / 64);
    __shared__ __attribute__((aligned(16))) float sh[SH];
    int k;
    int64_t p_begin, p_end;
    // the grid covers an upper bound of the items; order the real ones XCD-wise
    if ((int64_t)blockIdx.x >= ibase[K]) return;
    const int64_t item = xcd_unit(blockIdx.x, ibase[K]);
    if (!dw_item(ibase, chunk, seg, K, item, &k, &p_begin, &p_end)) return;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, q = lane >> 4;
    float* xs = sh + wave * STAGE;
    float* ys = xs + kDwStage * XS;
    floatx4 d[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) d[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int pr = lane % kDwStage, half = lane / kDwStage;
    constexpr int64_t kStep = kDwStage * (kThreads / 64);
    int64_t p0 = p_begin + kDwStage * wave;
    for (; p0 < p_end; p0 += kStep) {
        const DwRows<CI, CO> rows = dw_fetch<CI, CO>(X, dY, in_idx, out_idx, n_in, n_out, p0, p_end, pr, half);
        float4* xw = reinterpret_cast<float4*>(xs + pr * XS + half * (CI / 2));
        float4* yw = reinterpret_cast<float4*>(ys + pr * YS + half * (CO / 2));
#pragma unroll
        for (int i = 0; i < CI / 8; ++i) xw[i] = rows.x[i];
#pragma unroll
        for (int i = 0; i < CO / 8; ++i) yw[i] = rows.y[i];
        wave_lds_sync();   // lanes read rows other lanes of the wave staged
#pragma unroll
        for (int t = 0; t < kDwStage / 4; ++t) {
            const int row = 4 * t + q;
            float xa[NA], yb[NB];
#pragma unroll
            for (int a = 0; a < NA; ++a) xa[a] = xs[row * XS + 16 * a + r16];
#pragma unroll
            for (int b = 0; b < NB; ++b) yb[b] = ys[row * YS + 16 * b + r16];
#pragma unroll
            for (int a = 0; a < NA; ++a)
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    d[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[a], yb[b], d[a][b], 0, 0, 0);
        }
        wave_lds_sync();   // the next stage overwrites rows other lanes just read
    }
    __syncthreads();   // staging buffers are reused for the partial sums
    dw_store_partial<CI, CO>(sh, d, NA, NB, wave, q, r16, CI, CO, part + item * CI * (int64_t)CO, CO);
}

// dW[k] = sum of offset k's partials in a fixed order.  A block covers 64 V
// elements of one offset (V = 4: a 16-byte load per lane, for wide layers
// with ci * co a multiple of 4 and dW 16-byte aligned); wave w adds partials
// w, w + 4, w + 8, ... with eight loads in flight, and the four wave sums are
// combined in wave order.
template <int V>
__global__ void __launch_bounds__(kThreads) k_dw_reduce(const float* __restrict__ part, const int64_t* __restrict__ ibase,
                                                        int ci, int co, float* __restrict__ dW) {
    typedef float vec __attribute__((ext_vector_type(V)));
    __shared__ vec sh[4][64];
    const int k = blockIdx.y;
    const int64_t cc = (int64_t)ci * co;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t e = ((int64_t)blockIdx.x * 64 + lane) * V;
    const int64_t ee = e < cc ? e : 0;
    const int64_t i0 = ibase[k], i1 = ibase[k + 1];
    vec acc8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc8[u] = vec(0.f);
    for (int64_t it = i0 + wave; it < i1; it += 32) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t i = it + 4 * u;
            const vec v = *reinterpret_cast<const vec*>(part + (i < i1 ? i : i0) * cc + ee);
            acc8[u] += i < i1 ? v : vec(0.f);   // a select, not a branch: all eight loads stay in flight
        }
    }
    vec v = vec(0.f);
#pragma unroll
    for (int u = 0; u < 8; ++u) v += acc8[u];
    sh[wave][lane] = v;
    __syncthreads();
    if (wave == 0 && e < cc)
        *reinterpret_cast<vec*>(dW + (int64_t)k * cc + e) = ((sh[0][lane] + sh[1][lane]) + sh[2][lane]) + sh[3][lane];
}

static int dw_tiles(int ci, int co) { return ((ci + kDwTile - 1) / kDwTile) * ((co + kDwTile - 1) / kDwTile); }

// pairs per dW work item: 1024 for one output tile, more for wide layers so
// that the number of partial tiles stays moderate
static int64_t dw_chunk(int ci, int co) {
    const int t = dw_tiles(ci, co);
    return t <= 1 ? 1024 : (t <= 4 ? 2048 : (t <= 16 ? 4096 : 8192));
}

// upper bound of the work items for at most n_pairs pairs
static int64_t dw_items_bound(int64_t n_pairs, int K, int64_t ch) { return (n_pairs + ch - 1) / ch + K; }

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

static bool dw_f32_specialised(int ci, int co) {
    return (ci == 16 || ci == 32 || ci == 64) && (co == 16 || co == 32 || co == 64);
}

template <int CA, int CB, bool WT, typename Sel>
static void launch_f32(const void* X, int64_t n_x, const void* W, const int32_t* gat, const int32_t* sca,
                       const int64_t* gidx, const int32_t* perm, int K, int64_t G, int64_t n_y, void* Y, Sel sel,
                       hipStream_t s) {
    const int64_t blocks = (G + kThreads / 64 - 1) / (kThreads / 64);
    hipLaunchKernelGGL((k_conv_f32<CA, CB, WT, Sel>), dim3((unsigned)blocks), dim3(kThreads), 0, s,
                       reinterpret_cast<const float*>(X), n_x, reinterpret_cast<const float*>(W), gat, sca, gidx,
                       perm, K, G, n_y, reinterpret_cast<float*>(Y), sel);
}

// fp32 shapes with a specialised kernel
template <bool WT, typename Sel>
static bool try_f32(int ca, int cb, const void* X, int64_t n_x, const void* W, const int32_t* gat,
                    const int32_t* sca, const int64_t* gidx, const int32_t* perm, int K, int64_t G, int64_t n_y,
                    void* Y, Sel sel, hipStream_t s) {
#define GSC_F32_CASE(A, B)                                                                     \
    if (ca == A && cb == B) {                                                                  \
        launch_f32<A, B, WT, Sel>(X, n_x, W, gat, sca, gidx, perm, K, G, n_y, Y, sel, s);      \
        return true;                                                                           \
    }
    GSC_F32_CASE(16, 16) GSC_F32_CASE(16, 32) GSC_F32_CASE(32, 16) GSC_F32_CASE(32, 32)
    GSC_F32_CASE(32, 64) GSC_F32_CASE(64, 32) GSC_F32_CASE(64, 64) GSC_F32_CASE(16, 64) GSC_F32_CASE(64, 16)
#undef GSC_F32_CASE
    return false;
}

template <typename TIn, typename TOut, bool WT, typename Sel>
static int launch_os(const void* X, int64_t n_x, const void* W, const int32_t* gat, const int32_t* sca,
                     const int64_t* gidx, const int32_t* perm, int K, int ca, int cb, int64_t n_y, void* Y, Sel sel,
                     hipStream_t s) {
    if (n_y == 0) return GSC_OK;
    const int64_t tiles = (n_y + kTileRows - 1) / kTileRows;
    const int64_t G = (n_y + GSC_GROUP_ROWS - 1) / GSC_GROUP_ROWS;
    if constexpr (sizeof(TIn) == 4) {
        if (K <= kWaveKMax && try_f32<WT, Sel>(ca, cb, X, n_x, W, gat, sca, gidx, perm, K, G, n_y, Y, sel, s)) {
            GSC_LAUNCH_CHECK();
            return GSC_OK;
        }
    }
    dim3 grid((unsigned)tiles, (unsigned)((cb + kColSlice - 1) / kColSlice));
    hipLaunchKernelGGL((k_conv_os<TIn, TOut, WT, Sel>), grid, dim3(kThreads), 0, s, reinterpret_cast<const TIn*>(X),
                       n_x, reinterpret_cast<const TIn*>(W), gat, sca, gidx, perm, K, G, ca, cb, n_y,
                       reinterpret_cast<TOut*>(Y), sel);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

// The epilogue as a pass of its own over complete rows (row-form forward).
template <typename T>
__global__ void k_affine_act(T* __restrict__ y, int64_t n, int c, Epilogue ep) {
    const int64_t total = n * c;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int col = (int)(i % c);
        const float sc = ep.scale ? ep.scale[col] : 1.f;
        const float sh = ep.shift ? ep.shift[col] : 0.f;
        store_out(&y[i], epi_apply(to_f32(y[i]), sc, sh, ep.relu));
    }
}

int affine_act(int dtype, void* Y, int64_t n, int c, const Epilogue& ep, hipStream_t s) {
    const int64_t total = n * c;
    if (total == 0) return GSC_OK;
    const unsigned grid = (unsigned)((total + 255) / 256 < 8192 ? (total + 255) / 256 : 8192);
    if (dtype == GSC_BF16)
        hipLaunchKernelGGL(k_affine_act<uint16_t>, dim3(grid), dim3(256), 0, s, reinterpret_cast<uint16_t*>(Y), n, c,
                           ep);
    else
        hipLaunchKernelGGL(k_affine_act<float>, dim3(grid), dim3(256), 0, s, reinterpret_cast<float*>(Y), n, c, ep);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

// Backward of the epilogue y = act(z * scale + shift) (Sec. 4.5, the
// non-spatial functions after a convolution; the chain rule per element):
// g = dy where the ReLU passed (y > 0; everywhere without it), dz = g * scale,
// and per channel dscale = sum over rows of g * z, dshift = sum of g, with z
// recovered from y as (y - shift) / scale on the rows where g counts.  Rows
// are split into kAbChunks chunks at most; a block sums its chunk per channel
// (lane l of a channel takes rows l, l + L, ...; the L lanes are added in
// lane order), the chunk sums go to part, and a second kernel adds them in
// chunk order (so the sums are deterministic).
constexpr int kAbThreads = 256;
constexpr int64_t kAbChunks = 1024;

static int64_t ab_chunks(int64_t n) {
    const int64_t c = (n + 63) / 64;
    return c < 1 ? 1 : (c > kAbChunks ? kAbChunks : c);
}

template <typename T>
__global__ void __launch_bounds__(kAbThreads) k_affine_act_bwd(const T* __restrict__ y, const T* __restrict__ dy,
                                                               int64_t n, int c, Epilogue ep, T* __restrict__ dz,
                                                               float* __restrict__ part_s, float* __restrict__ part_t) {
    __shared__ float ss[kAbThreads], st[kAbThreads];
    const int64_t chunks = gridDim.x;
    const int64_t r0 = n * blockIdx.x / chunks, r1 = n * (blockIdx.x + 1) / chunks;
    const int L = c < kAbThreads ? kAbThreads / c : 1;   // lanes per channel
    const int t = threadIdx.x;
    for (int cb = 0; cb < c; cb += kAbThreads) {   // channels cb .. cb + (L > 1 ? c : 256) - 1
        const int lane = t / (L > 1 ? c : kAbThreads);
        const int ch = cb + t % (L > 1 ? c : kAbThreads);
        float gs = 0.f, gt = 0.f;
        if (lane < L && ch < c) {
            const float sc = ep.scale ? ep.scale[ch] : 1.f;
            const float sh = ep.shift ? ep.shift[ch] : 0.f;
            for (int64_t r = r0 + lane; r < r1; r += L) {
                const int64_t i = r * c + ch;
                const float yv = to_f32(y[i]);
                const float g = ep.relu && !(yv > 0.f) ? 0.f : to_f32(dy[i]);
                store_out(&dz[i], g * sc);
                if (part_s && g != 0.f) {
                    gs += g * ((yv - sh) / sc);
                    gt += g;
                }
            }
        }
        if (part_s) {
            __syncthreads();   // the previous channel group's sums are read
            ss[t] = gs;
            st[t] = gt;
            __syncthreads();
            const int span = L > 1 ? c : kAbThreads;
            if (t < span && cb + t < c) {
                float a = 0.f, b = 0.f;
                for (int l = 0; l < L; ++l) {
                    a += ss[l * span + t];
                    b += st[l * span + t];
                }
                part_s[(int64_t)blockIdx.x * c + cb + t] = a;
                part_t[(int64_t)blockIdx.x * c + cb + t] = b;
            }
        }
    }
}

__global__ void k_affine_act_bwd_sum(const float* __restrict__ part_s, const float* __restrict__ part_t,
                                     int64_t chunks, int c, float* __restrict__ dscale, float* __restrict__ dshift) {
    const int ch = blockIdx.x * blockDim.x + threadIdx.x;
    if (ch >= c) return;
    double a = 0.0, b = 0.0;
    for (int64_t k = 0; k < chunks; ++k) {
        a += part_s[k * c + ch];
        b += part_t[k * c + ch];
    }
    if (dscale) dscale[ch] = (float)a;
    if (dshift) dshift[ch] = (float)b;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

static bool fwd_uses_bf16_engine(int32_t dtype, int32_t c_in, int32_t c_out, int32_t K) {
    return dtype == GSC_BF16 && conv_bf16_supported(c_in, c_out, K);
}

// Workspace of the forward pass: the bf16 engines' transposed weights, then
// (tile engine) the tile counter.
static size_t fwd_counter_offset(int32_t c_in, int32_t c_out, int32_t K) {
    return (transpose_ws_bytes(K, c_in, c_out) + 255) & ~(size_t)255;
}

size_t gsc_conv_fwd_ws_bytes(int32_t dtype, int32_t c_in, int32_t c_out, int32_t K) {
    if (c_in < 1 || c_out < 1 || K < 1) return 0;
    return fwd_uses_bf16_engine(dtype, c_in, c_out, K) ? fwd_counter_offset(c_in, c_out, K) + 256 : 0;
}

// The plan (perm, bmask, ibase, items) is all given or all null (checked
// when there are output rows; with none the plan is not read).
static int plan_args(const char* who, int64_t n, const int32_t* perm, const uint32_t* bmask, const int64_t* ibase,
                     const int32_t* items, bool* given) {
    *given = false;
    if (n == 0) return GSC_OK;
    const int nn = (perm != nullptr) + (bmask != nullptr) + (ibase != nullptr) + (items != nullptr);
    if (nn != 0 && nn != 4) return fail(GSC_EINVAL, "%s: the block plan needs perm, bmask, ibase and items", who);
    *given = nn == 4;
    return GSC_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// The fp32 engine over a plan of one or more ranges of offsets (see
// gsc_conv_plan): one launch per range, each adding its sums to the rows
// written by the ranges before it; the epilogue goes with the last.
static int blk_f32_ranges(int ca, int cb, const float* X, int64_t n_x, const float* W, bool wt, const WSel& sel,
                          int K, const BlockPlan& plan, int64_t n_y, float* Y, hipStream_t s, const Epilogue& ep) {
    const int R = plan_ranges(K), S = plan_range_size(K);
    if (R == 1) return conv_blk_f32(ca, cb, X, n_x, W, wt, sel, K, plan, n_y, Y, s, ep);
    const int64_t nb = gsc_plan_blocks(n_y);
    for (int r = 0; r < R; ++r) {
        const int k0 = r * S, kr = K - k0 < S ? K - k0 : S;
        const BlockPlan pr{plan.perm + (int64_t)r * n_y, plan.bmask + (int64_t)r * nb,
                           plan.ibase + (int64_t)r * (nb + 1), plan.items + (int64_t)k0 * nb * 16};
        WSel sr{};
        for (int k = 0; k < kr && wt; ++k) sr.w[k] = sel.w[k0 + k];
        const float* Wr = wt ? W : W + (int64_t)k0 * ca * cb;   // forward: the range's own matrices
        const int rc = conv_blk_f32(ca, cb, X, n_x, Wr, wt, sr, kr, pr, n_y, Y, s, r == R - 1 ? ep : Epilogue{},
                                    r > 0);
        if (rc) return rc;
    }
    return GSC_OK;
}

int32_t gsc_conv_block_engine(int32_t dtype, int32_t c_red, int32_t c_out, int32_t K) {
    if (dtype == GSC_F32)
        return K >= 1 && K <= kPlanMaxKAll && blk_f32_supported(c_red, c_out, plan_range_size(K)) ? 1 : 0;
    if (dtype == GSC_BF16) return blk_bf16_supported(c_red, c_out, K) ? 1 : 0;
    return 0;
}

static int conv_fwd(int32_t dtype, const void* X, int64_t n_in, int32_t c_in, const void* W, int32_t c_out,
                    int32_t K, const int32_t* in_idx, const int32_t* out_idx, const int64_t* gidx, int64_t n_pairs,
                    const int32_t* perm, const uint32_t* bmask, const int64_t* ibase, const int32_t* items,
                    const Epilogue& ep, void* Y, int64_t n_out, void* ws, size_t ws_bytes, hipStream_t s) {
    if (dtype != GSC_F32 && dtype != GSC_BF16) return fail(GSC_EINVAL, "conv_fwd: unknown dtype %d", dtype);
    if (n_in < 0 || n_out < 0 || n_in > INT32_MAX || n_out > INT32_MAX)
        return fail(GSC_EINVAL, "conv_fwd: bad row counts n_in=%lld n_out=%lld", (long long)n_in, (long long)n_out);
    if (c_in < 1 || c_out < 1) return fail(GSC_EINVAL, "conv_fwd: channels must be >= 1");
    if (K < 1 || K > kMaxKConv) return fail(GSC_EINVAL, "conv_fwd: K=%d outside [1,%d]", K, kMaxKConv);
    if (n_pairs < 0) return fail(GSC_EINVAL, "conv_fwd: n_pairs < 0");
    if (n_out > 0 && (!Y || !gidx || !W)) return fail(GSC_EINVAL, "conv_fwd: null Y/gidx/W");
    if (n_pairs > 0 && (!X || !in_idx || !out_idx)) return fail(GSC_EINVAL, "conv_fwd: null X/in_idx/out_idx");
    const size_t need = gsc_conv_fwd_ws_bytes(dtype, c_in, c_out, K);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(GSC_ESHORT, "conv_fwd: ws needs %zu bytes, got %zu", need, ws ? ws_bytes : (size_t)0);
    bool planned = false;
    int rc = plan_args("conv_fwd", n_out, perm, bmask, ibase, items, &planned);
    if (rc) return rc;
    if (planned && gsc_conv_block_engine(dtype, c_in, c_out, K) && aligned16(X) && aligned16(W) &&
        (dtype != GSC_BF16 || blk_bf16_fits(n_in, c_in))) {
        if (n_in > 0 && !X) return fail(GSC_EINVAL, "conv_fwd: X is null");
        const BlockPlan plan{perm, bmask, ibase, items};
        if (dtype == GSC_BF16) {   // B_k = W[k]: the engine reads its columns, so the transposed copy
            const bool tile = n_in > 0 && tile_bf16_supported(c_in, c_out, K);
            unsigned* counter = reinterpret_cast<unsigned*>(reinterpret_cast<char*>(ws) +
                                                            fwd_counter_offset(c_in, c_out, K));
            rc = transpose_w_bf16(W, K, c_in, c_out, ws, s, tile ? counter : nullptr);   // also zeroes the counter
            if (rc) return rc;
            if (tile)
                return conv_tile_bf16<WIdentity>(c_in, c_out, X, n_in, ws, WIdentity{}, K, plan,
                                                 (n_out + kPlanBlockRows - 1) / kPlanBlockRows, n_out, Y, counter, s,
                                                 ep, /*counter_ready=*/true);
            return conv_blk_bf16<WIdentity>(c_in, c_out, X, n_in, ws, WIdentity{}, K, plan, n_out, Y, s, ep);
        }
        static const WSel kNoSel{};
        return blk_f32_ranges(c_in, c_out, reinterpret_cast<const float*>(X), n_in, reinterpret_cast<const float*>(W),
                              false, kNoSel, K, plan, n_out, reinterpret_cast<float*>(Y), s, ep);
    }
    // row form: the sums are complete only once the call's kernels are done,
    // so the epilogue is a pass of its own over Y
    if (dtype == GSC_F32) {
        rc = launch_os<float, float, false>(X, n_in, W, in_idx, out_idx, gidx, nullptr, K, c_in, c_out, n_out, Y,
                                            WIdentity{}, s);
    } else if (fwd_uses_bf16_engine(dtype, c_in, c_out, K)) {
        if (n_out == 0) return GSC_OK;
        rc = transpose_w_bf16(W, K, c_in, c_out, ws, s);
        if (rc) return rc;
        rc = conv_bf16<WIdentity>(c_in, c_out, X, n_in, ws, in_idx, out_idx, gidx, nullptr, K, n_out, Y, WIdentity{},
                                  s);
    } else {
        rc = launch_os<uint16_t, uint16_t, false>(X, n_in, W, in_idx, out_idx, gidx, nullptr, K, c_in, c_out, n_out,
                                                  Y, WIdentity{}, s);
    }
    if (rc || !ep.on()) return rc;
    return affine_act(dtype, Y, n_out, c_out, ep, s);
}

int gsc_sparse_conv_fwd(int32_t dtype, const void* X, int64_t n_in, int32_t c_in, const void* W, int32_t c_out,
                        int32_t K, const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                        const int64_t* gidx, int64_t n_pairs, const int32_t* perm, const uint32_t* bmask,
                        const int64_t* ibase, const int32_t* items, void* Y, int64_t n_out, void* ws,
                        size_t ws_bytes, void* stream) {
    (void)seg;
    clear_error();
    return conv_fwd(dtype, X, n_in, c_in, W, c_out, K, in_idx, out_idx, gidx, n_pairs, perm, bmask, ibase, items,
                    Epilogue{}, Y, n_out, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

int gsc_sparse_conv_fwd_affine(int32_t dtype, const void* X, int64_t n_in, int32_t c_in, const void* W,
                               int32_t c_out, int32_t K, const int32_t* in_idx, const int32_t* out_idx,
                               const int64_t* seg, const int64_t* gidx, int64_t n_pairs, const int32_t* perm,
                               const uint32_t* bmask, const int64_t* ibase, const int32_t* items, const float* scale,
                               const float* shift, int32_t act, void* Y, int64_t n_out, void* ws, size_t ws_bytes,
                               void* stream) {
    (void)seg;
    clear_error();
    if (act != GSC_ACT_NONE && act != GSC_ACT_RELU) return fail(GSC_EINVAL, "conv_fwd_affine: unknown act %d", act);
    Epilogue ep;
    ep.scale = scale;
    ep.shift = shift;
    ep.relu = act == GSC_ACT_RELU;
    return conv_fwd(dtype, X, n_in, c_in, W, c_out, K, in_idx, out_idx, gidx, n_pairs, perm, bmask, ibase, items, ep,
                    Y, n_out, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

// Workspace of the backward pass: the weight gradient's chunk tables and
// partial sums, then the tile counter of the input gradient's tile engine.
static size_t bwd_counter_offset(int64_t n_pairs, int32_t c_in, int32_t c_out, int32_t K) {
    const int64_t items = dw_items_bound(n_pairs, K, dw_chunk(c_in, c_out));
    return 2 * al256((size_t)(K + 1) * sizeof(int64_t)) + al256((size_t)items * c_in * c_out * sizeof(float));
}

size_t gsc_conv_bwd_ws_bytes(int64_t n_pairs, int32_t c_in, int32_t c_out, int32_t K) {
    if (n_pairs < 0 || c_in < 1 || c_out < 1 || K < 1) return 0;
    return bwd_counter_offset(n_pairs, c_in, c_out, K) + 256;
}

int gsc_sparse_conv_bwd(int32_t dtype, const void* X, const void* W, const void* dY, int64_t n_in, int32_t c_in,
                        int32_t c_out, int32_t K, const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                        int64_t n_pairs, const int32_t* t_in_idx, const int32_t* t_out_idx, const int64_t* t_seg,
                        const int64_t* t_gidx, int64_t t_n_pairs, const int32_t* t_wsel, const int32_t* t_perm,
                        const uint32_t* t_bmask, const int64_t* t_ibase, const int32_t* t_items, void* dX, float* dW,
                        int64_t n_out, void* ws, size_t ws_bytes, void* stream) {
    (void)t_seg;
    clear_error();
    if (dtype != GSC_F32 && dtype != GSC_BF16) return fail(GSC_EINVAL, "conv_bwd: unknown dtype %d", dtype);
    if (n_in < 0 || n_out < 0 || n_in > INT32_MAX || n_out > INT32_MAX)
        return fail(GSC_EINVAL, "conv_bwd: bad row counts");
    if (c_in < 1 || c_out < 1) return fail(GSC_EINVAL, "conv_bwd: channels must be >= 1");
    if (K < 1 || K > kMaxKConv) return fail(GSC_EINVAL, "conv_bwd: K=%d outside [1,%d]", K, kMaxKConv);
    if (!W) return fail(GSC_EINVAL, "conv_bwd: W is null");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (dW) {
        if (n_pairs < 0) return fail(GSC_EINVAL, "conv_bwd: n_pairs < 0");
        if (!seg || !ws) return fail(GSC_EINVAL, "conv_bwd: null seg/ws");
        if (n_pairs > 0 && (!X || !dY || !in_idx || !out_idx)) return fail(GSC_EINVAL, "conv_bwd: null X/dY/idx");
        const size_t need = gsc_conv_bwd_ws_bytes(n_pairs, c_in, c_out, K);
        if (ws_bytes < need) return fail(GSC_ESHORT, "conv_bwd: ws needs %zu bytes, got %zu", need, ws_bytes);
    }
    // the weight gradient's work items (at the start of ws)
    const int64_t dw_ch = dw_chunk(c_in, c_out);
    int64_t* dw_ibase = ws ? reinterpret_cast<int64_t*>(ws) : nullptr;
    int64_t* dw_chunks =
        ws ? reinterpret_cast<int64_t*>(reinterpret_cast<char*>(ws) + al256((size_t)(K + 1) * sizeof(int64_t)))
           : nullptr;
    bool dw_items_done = false;
    if (dX) {
        if (t_n_pairs < 0) return fail(GSC_EINVAL, "conv_bwd: t_n_pairs < 0");
        if (n_in > 0 && (!t_gidx || !t_wsel)) return fail(GSC_EINVAL, "conv_bwd: null t_gidx/t_wsel");
        if (t_n_pairs > 0 && (!dY || !t_in_idx || !t_out_idx))
            return fail(GSC_EINVAL, "conv_bwd: null dY/t_in_idx/t_out_idx");
        // the role-reversed map's offsets pair one to one with the forward map's
        WSel sel;
        std::vector<uint8_t> seen((size_t)K, 0);
        for (int k = 0; k < K; ++k) {
            if (t_wsel[k] < 0 || t_wsel[k] >= K)
                return fail(GSC_EINVAL, "conv_bwd: t_wsel[%d]=%d outside [0,%d)", k, t_wsel[k], K);
            if (seen[t_wsel[k]]++)
                return fail(GSC_EINVAL, "conv_bwd: t_wsel is not a permutation (%d appears twice)", t_wsel[k]);
            sel.w[k] = (int16_t)t_wsel[k];
        }
        bool planned = false;
        int rc = plan_args("conv_bwd", n_in, t_perm, t_bmask, t_ibase, t_items, &planned);
        if (rc) return rc;
        if (planned && gsc_conv_block_engine(dtype, c_out, c_in, K) && aligned16(dY) && aligned16(W) &&
            (dtype != GSC_BF16 || blk_bf16_fits(n_out, c_out))) {
            const BlockPlan plan{t_perm, t_bmask, t_ibase, t_items};
            if (dtype == GSC_BF16 && n_out > 0 && tile_bf16_supported(c_out, c_in, K)) {
                // B_k[ch][col] = W[sel(k)][col][ch]: W is already the engine's layout.  The tile
                // counter sits after the weight gradient's part of ws, when ws is given in full.
                unsigned* counter = nullptr;
                if (ws && n_pairs >= 0 && ws_bytes >= gsc_conv_bwd_ws_bytes(n_pairs, c_in, c_out, K))
                    counter = reinterpret_cast<unsigned*>(reinterpret_cast<char*>(ws) +
                                                          bwd_counter_offset(n_pairs, c_in, c_out, K));
                if (counter && dW) {   // one small launch: the weight gradient's items and the tile counter
                    hipLaunchKernelGGL(k_dw_items, dim3(1), dim3(64), 0, s, seg, K, dw_ch, dw_ibase, dw_chunks,
                                       counter);
                    GSC_LAUNCH_CHECK();
                    dw_items_done = true;
                }
                rc = conv_tile_bf16<WSel>(c_out, c_in, dY, n_out, W, sel, K, plan,
                                          (n_in + kPlanBlockRows - 1) / kPlanBlockRows, n_in, dX, counter, s,
                                          Epilogue{}, /*counter_ready=*/dw_items_done);
            } else if (dtype == GSC_BF16)   // B_k[ch][col] = W[sel(k)][col][ch]: W is already the engine's layout
                rc = conv_blk_bf16<WSel>(c_out, c_in, dY, n_out, W, sel, K, plan, n_in, dX, s);
            else
                rc = blk_f32_ranges(c_out, c_in, reinterpret_cast<const float*>(dY), n_out,
                                    reinterpret_cast<const float*>(W), true, sel, K, plan, n_in,
                                    reinterpret_cast<float*>(dX), s, Epilogue{});
        }
        else if (dtype == GSC_F32)
            rc = launch_os<float, float, true>(dY, n_out, W, t_in_idx, t_out_idx, t_gidx, nullptr, K, c_out, c_in,
                                               n_in, dX, sel, s);
        else if (conv_bf16_supported(c_out, c_in, K))   // W[w] (c_in x c_out) is already the B layout of dY W^T
            rc = conv_bf16<WSel>(c_out, c_in, dY, n_out, W, t_in_idx, t_out_idx, t_gidx, nullptr, K, n_in, dX, sel,
                                 s);
        else
            rc = launch_os<uint16_t, uint16_t, true>(dY, n_out, W, t_in_idx, t_out_idx, t_gidx, nullptr, K, c_out,
                                                     c_in, n_in, dX, sel, s);
        if (rc) return rc;
    }
    if (dW) {
        const int64_t ch = dw_ch;
        const int64_t items = dw_items_bound(n_pairs, K, ch);
        char* w = reinterpret_cast<char*>(ws);
        int64_t* ibase = dw_ibase;
        int64_t* chunk = dw_chunks;
        float* part = reinterpret_cast<float*>(w + 2 * al256((size_t)(K + 1) * sizeof(int64_t)));
        if (!dw_items_done) {
            hipLaunchKernelGGL(k_dw_items, dim3(1), dim3(64), 0, s, seg, K, ch, ibase, chunk, nullptr);
            GSC_LAUNCH_CHECK();
        }
        if (dtype == GSC_F32 && dw_f32_specialised(c_in, c_out)) {
            auto X32 = reinterpret_cast<const float*>(X);
            auto dY32 = reinterpret_cast<const float*>(dY);
#define GSC_DW_CASE(A, B)                                                                              \
    if (c_in == A && c_out == B)                                                                       \
        hipLaunchKernelGGL((k_dw_f32<A, B>), dim3((unsigned)items), dim3(kThreads), 0, s, X32, n_in, dY32, \
                           n_out, in_idx, out_idx, seg, ibase, chunk, K, part);
            GSC_DW_CASE(16, 16) GSC_DW_CASE(16, 32) GSC_DW_CASE(16, 64) GSC_DW_CASE(32, 16) GSC_DW_CASE(32, 32)
            GSC_DW_CASE(32, 64) GSC_DW_CASE(64, 16) GSC_DW_CASE(64, 32) GSC_DW_CASE(64, 64)
#undef GSC_DW_CASE
        } else if (dtype == GSC_BF16 && dw_tile_bf16_supported(c_in, c_out) && blk_bf16_fits(n_in, c_in) &&
                   blk_bf16_fits(n_out, c_out)) {
            int rc = dw_tile_bf16(c_in, c_out, X, n_in, dY, n_out, in_idx, out_idx, seg, ibase, chunk, K, items, part,
                                  s);
            if (rc) return rc;
        } else if (dtype == GSC_BF16 && dw_bf16_supported(c_in, c_out)) {
            int rc = dw_bf16(c_in, c_out, X, n_in, dY, n_out, in_idx, out_idx, seg, ibase, chunk, K, items, part, s);
            if (rc) return rc;
        } else {
            const unsigned tiles = (unsigned)dw_tiles(c_in, c_out);
            if (dtype == GSC_F32)
                hipLaunchKernelGGL(k_dw_partial<float>, dim3((unsigned)items, tiles), dim3(kThreads), 0, s,
                                   reinterpret_cast<const float*>(X), n_in, reinterpret_cast<const float*>(dY), n_out,
                                   in_idx, out_idx, seg, ibase, chunk, K, c_in, c_out, part);
            else
                hipLaunchKernelGGL(k_dw_partial<uint16_t>, dim3((unsigned)items, tiles), dim3(kThreads), 0, s,
                                   reinterpret_cast<const uint16_t*>(X), n_in, reinterpret_cast<const uint16_t*>(dY),
                                   n_out, in_idx, out_idx, seg, ibase, chunk, K, c_in, c_out, part);
        }
        GSC_LAUNCH_CHECK();
        const int64_t cc = (int64_t)c_in * c_out;
        // 16-byte lanes where that still leaves thousands of blocks (wide layers)
        if (cc % 4 == 0 && cc >= 16384 && reinterpret_cast<uintptr_t>(dW) % 16 == 0)
            hipLaunchKernelGGL(k_dw_reduce<4>, dim3((unsigned)((cc + 255) / 256), (unsigned)K), dim3(kThreads), 0, s,
                               part, ibase, c_in, c_out, dW);
        else
            hipLaunchKernelGGL(k_dw_reduce<1>, dim3((unsigned)((cc + 63) / 64), (unsigned)K), dim3(kThreads), 0, s,
                               part, ibase, c_in, c_out, dW);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

// Workspace of gsc_sparse_conv_bwd_fwdmap: the weight gradient's part (as
// gsc_sparse_conv_bwd's, with its tile counter), the dX map (dense form,
// pairs, segments, group index) and the transposition's scratch, then, when a
// block engine takes the input gradient, the dX map's plan and its scratch.
struct FwdmapWs {
    size_t dw, dense, t_in, t_out, t_seg, t_gidx, tr, perm, bmask, ibase, items, plan, total;
};

static FwdmapWs fwdmap_layout(int32_t dtype, int64_t n_in, int64_t cap, int32_t c_in, int32_t c_out, int32_t K) {
    FwdmapWs L{};
    const int64_t G = gsc_kmap_groups(n_in);
    size_t o = 0;
    auto take = [&](size_t b) {
        const size_t at = o;
        o += al256(b);
        return at;
    };
    L.dw = take(gsc_conv_bwd_ws_bytes(cap, c_in, c_out, K));
    L.dense = take((size_t)K * n_in * sizeof(int32_t));
    L.t_in = take((size_t)cap * sizeof(int32_t));
    L.t_out = take((size_t)cap * sizeof(int32_t));
    L.t_seg = take((size_t)(K + 1) * sizeof(int64_t));
    L.t_gidx = take((size_t)(K * G + 1) * sizeof(int64_t));
    L.tr = take(gsc_kernel_map_transpose_ws_bytes(n_in, K));
    if (gsc_conv_block_engine(dtype, c_out, c_in, K)) {
        const int64_t R = gsc_plan_ranges(K), nb = gsc_plan_blocks(n_in);
        L.perm = take((size_t)R * n_in * sizeof(int32_t));
        L.bmask = take((size_t)R * nb * sizeof(uint32_t));
        L.ibase = take((size_t)R * (nb + 1) * sizeof(int64_t));
        L.items = take((size_t)K * nb * 16 * sizeof(int32_t));
        L.plan = take(gsc_conv_plan_ws_bytes(n_in, K));
    } else {
        L.perm = L.bmask = L.ibase = L.items = L.plan = SIZE_MAX;
    }
    L.total = o;
    return L;
}

size_t gsc_conv_bwd_fwdmap_ws_bytes(int32_t dtype, int64_t n_in, int64_t cap_pairs, int32_t c_in, int32_t c_out,
                                    int32_t K) {
    if ((dtype != GSC_F32 && dtype != GSC_BF16) || n_in < 0 || cap_pairs < 0 || c_in < 1 || c_out < 1 || K < 1 ||
        K > kMaxKConv)
        return 0;
    return fwdmap_layout(dtype, n_in, cap_pairs, c_in, c_out, K).total;
}

int gsc_sparse_conv_bwd_fwdmap(int32_t dtype, const void* X, const void* W, const void* dY, int64_t n_in,
                               int32_t c_in, int32_t c_out, int32_t K, const int32_t* in_idx, const int32_t* out_idx,
                               const int64_t* seg, int64_t cap_pairs, int32_t transpose, void* dX, float* dW,
                               int64_t n_out, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (dtype != GSC_F32 && dtype != GSC_BF16) return fail(GSC_EINVAL, "conv_bwd_fwdmap: unknown dtype %d", dtype);
    if (K < 1 || K > kMaxKConv) return fail(GSC_EINVAL, "conv_bwd_fwdmap: K=%d outside [1,%d]", K, kMaxKConv);
    if (n_in < 0 || n_out < 0 || n_in > INT32_MAX || n_out > INT32_MAX || cap_pairs < 0 || c_in < 1 || c_out < 1)
        return fail(GSC_EINVAL, "conv_bwd_fwdmap: bad sizes");
    if (!seg || !ws) return fail(GSC_EINVAL, "conv_bwd_fwdmap: null seg/ws");
    const size_t need = gsc_conv_bwd_fwdmap_ws_bytes(dtype, n_in, cap_pairs, c_in, c_out, K);
    if (ws_bytes < need) return fail(GSC_ESHORT, "conv_bwd_fwdmap: ws needs %zu bytes, got %zu", need, ws_bytes);
    // a: the pairs' rows of X, b: their rows of Y (the transposed convolution ran the map with roles exchanged)
    const int32_t* a = transpose ? out_idx : in_idx;
    const int32_t* b = transpose ? in_idx : out_idx;
    const FwdmapWs L = fwdmap_layout(dtype, n_in, cap_pairs, c_in, c_out, K);
    char* w = reinterpret_cast<char*>(ws);
    int32_t* t_in = reinterpret_cast<int32_t*>(w + L.t_in);
    int32_t* t_out = reinterpret_cast<int32_t*>(w + L.t_out);
    int64_t* t_seg = reinterpret_cast<int64_t*>(w + L.t_seg);
    int64_t* t_gidx = reinterpret_cast<int64_t*>(w + L.t_gidx);
    int32_t* dense = reinterpret_cast<int32_t*>(w + L.dense);
    const bool planned = L.plan != SIZE_MAX;
    int32_t* perm = planned ? reinterpret_cast<int32_t*>(w + L.perm) : nullptr;
    uint32_t* bmask = planned ? reinterpret_cast<uint32_t*>(w + L.bmask) : nullptr;
    int64_t* ibase = planned ? reinterpret_cast<int64_t*>(w + L.ibase) : nullptr;
    int32_t* items = planned ? reinterpret_cast<int32_t*>(w + L.items) : nullptr;
    int rc;
    if (dX) {
        // the dX map: the same pairs listed by their row of X (and its plan)
        rc = gsc_kernel_map_transpose(a, b, seg, K, cap_pairs, n_in, t_in, t_out, t_seg, t_gidx, dense, w + L.tr,
                                      gsc_kernel_map_transpose_ws_bytes(n_in, K), stream);
        if (rc) return rc;
        if (planned) {
            rc = gsc_conv_plan(dense, n_in, K, perm, bmask, ibase, items, (int64_t)K * gsc_plan_blocks(n_in),
                               w + L.plan, gsc_conv_plan_ws_bytes(n_in, K), stream);
            if (rc) return rc;
        }
    }
    std::vector<int32_t> ident((size_t)K);
    for (int k = 0; k < K; ++k) ident[k] = k;   // segment k of the dX map holds offset k's pairs
    return gsc_sparse_conv_bwd(dtype, X, W, dY, n_in, c_in, c_out, K, a, b, seg, cap_pairs, t_in, t_out, t_seg,
                               t_gidx, cap_pairs, ident.data(), perm, bmask, ibase, items, dX, dW, n_out, w + L.dw,
                               gsc_conv_bwd_ws_bytes(cap_pairs, c_in, c_out, K), stream);
}

size_t gsc_affine_act_bwd_ws_bytes(int64_t n, int32_t c) {
    if (n < 0 || c < 1) return 0;
    return 2 * al256((size_t)ab_chunks(n) * c * sizeof(float));
}

int gsc_affine_act_bwd(int32_t dtype, const void* Y, const void* dY, int64_t n, int32_t c, const float* scale,
                       const float* shift, int32_t act, void* dZ, float* dscale, float* dshift, void* ws,
                       size_t ws_bytes, void* stream) {
    clear_error();
    if (dtype != GSC_F32 && dtype != GSC_BF16) return fail(GSC_EINVAL, "affine_act_bwd: unknown dtype %d", dtype);
    if (act != GSC_ACT_NONE && act != GSC_ACT_RELU) return fail(GSC_EINVAL, "affine_act_bwd: unknown act %d", act);
    if (n < 0 || c < 1) return fail(GSC_EINVAL, "affine_act_bwd: bad sizes n=%lld c=%d", (long long)n, c);
    if (n > 0 && (!Y || !dY || !dZ)) return fail(GSC_EINVAL, "affine_act_bwd: null Y/dY/dZ");
    const bool sums = dscale || dshift;
    if (sums) {
        const size_t need = gsc_affine_act_bwd_ws_bytes(n, c);
        if (!ws || ws_bytes < need)
            return fail(GSC_ESHORT, "affine_act_bwd: ws needs %zu bytes, got %zu", need, ws ? ws_bytes : (size_t)0);
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    Epilogue ep;
    ep.scale = scale;
    ep.shift = shift;
    ep.relu = act == GSC_ACT_RELU;
    const int64_t chunks = ab_chunks(n);
    float* part_s = sums ? reinterpret_cast<float*>(ws) : nullptr;
    float* part_t = sums ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                                    al256((size_t)chunks * c * sizeof(float)))
                         : nullptr;
    if (dtype == GSC_BF16)
        hipLaunchKernelGGL(k_affine_act_bwd<uint16_t>, dim3((unsigned)chunks), dim3(kAbThreads), 0, s,
                           reinterpret_cast<const uint16_t*>(Y), reinterpret_cast<const uint16_t*>(dY), n, c, ep,
                           reinterpret_cast<uint16_t*>(dZ), part_s, part_t);
    else
        hipLaunchKernelGGL(k_affine_act_bwd<float>, dim3((unsigned)chunks), dim3(kAbThreads), 0, s,
                           reinterpret_cast<const float*>(Y), reinterpret_cast<const float*>(dY), n, c, ep,
                           reinterpret_cast<float*>(dZ), part_s, part_t);
    GSC_LAUNCH_CHECK();
    if (sums) {
        hipLaunchKernelGGL(k_affine_act_bwd_sum, dim3((unsigned)((c + 255) / 256)), dim3(256), 0, s, part_s, part_t,
                           chunks, c, dscale, dshift);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

}  // extern "C"
