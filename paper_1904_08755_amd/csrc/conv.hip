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

#include "gsc_internal.h"

namespace gsc {

constexpr int kThreads = 256;
constexpr int kTileRows = 128;
constexpr int kTileGroups = kTileRows / GSC_GROUP_ROWS;
constexpr int kColSlice = 64;
constexpr int kAccStride = kColSlice + 1;
constexpr int kMaxKConv = 1024;
constexpr int kDwTile = 64;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef short shortx4 __attribute__((ext_vector_type(4)));

struct WSel {
    int16_t w[kMaxKConv];
    __device__ __forceinline__ int operator()(int k) const { return w[k]; }
};
struct WIdentity {
    __device__ __forceinline__ int operator()(int k) const { return k; }
};

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

// ---------------------------------------------------------------------------
// output-stationary gather -> MFMA -> LDS accumulate
//   Y[sca[p]] += X[gat[p]] * B_w  for every pair p of segment k, w = sel(k)
//   X: n_x x ca, Y: n_y x cb, B_w = W[w] (ca x cb) or W[w]^T.
// ---------------------------------------------------------------------------
template <typename TIn, typename TOut, bool WT, typename Sel>
__global__ void __launch_bounds__(kThreads)
k_conv_os(const TIn* __restrict__ X, int64_t n_x, const TIn* __restrict__ W, const int32_t* __restrict__ gat,
          const int32_t* __restrict__ sca, const int64_t* __restrict__ gidx, int K, int64_t G, int ca, int cb,
          int64_t n_y, TOut* __restrict__ Y, Sel sel) {
    __shared__ float acc[kTileRows * kAccStride];
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.x * kTileRows;
    const int col0 = blockIdx.y * kColSlice;
    const int ncols = min(kColSlice, cb - col0);
    const int nnb = (ncols + 15) >> 4;

    for (int i = tid; i < kTileRows * kAccStride; i += kThreads) acc[i] = 0.f;
    __syncthreads();

    const int64_t g0 = (int64_t)blockIdx.x * kTileGroups;
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
        const int64_t row = row0 + r;
        if (row < n_y) store_out(Y + row * cb + col0 + c, acc[r * kAccStride + c]);
    }
}

// ---------------------------------------------------------------------------
// weight gradient
// ---------------------------------------------------------------------------
// item bases: ibase[k] = sum over k' < k of ceil(|M_k'| / CH); ibase[K] = total
__global__ void k_dw_items(const int64_t* seg, int K, int64_t CH, int64_t* ibase) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    int64_t t = 0;
    for (int k = 0; k < K; ++k) {
        ibase[k] = t;
        const int64_t n = seg[k + 1] - seg[k];
        t += n > 0 ? (n + CH - 1) / CH : 0;
    }
    ibase[K] = t;
}

template <typename TIn>
__global__ void __launch_bounds__(kThreads)
k_dw_partial(const TIn* __restrict__ X, int64_t n_in, const TIn* __restrict__ dY, int64_t n_out,
             const int32_t* __restrict__ in_idx, const int32_t* __restrict__ out_idx, const int64_t* __restrict__ seg,
             const int64_t* __restrict__ ibase, int K, int64_t CH, int ci, int co, float* __restrict__ part) {
    __shared__ float acc[kDwTile * (kDwTile + 1)];
    const int64_t item = blockIdx.x;
    if (item >= ibase[K]) return;
    int lo = 0, hi = K - 1;   // last k with ibase[k] <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (ibase[mid] <= item) lo = mid; else hi = mid - 1;
    }
    const int k = lo;
    const int64_t p_begin = seg[k] + (item - ibase[k]) * CH;
    const int64_t p_end = min(seg[k + 1], p_begin + CH);
    const int ntj = (co + kDwTile - 1) / kDwTile;
    const int ci0 = (blockIdx.y / ntj) * kDwTile, co0 = (blockIdx.y % ntj) * kDwTile;
    const int na = (min(kDwTile, ci - ci0) + 15) >> 4, nbk = (min(kDwTile, co - co0) + 15) >> 4;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, q = lane >> 4;

    for (int i = tid; i < kDwTile * (kDwTile + 1); i += kThreads) acc[i] = 0.f;
    __syncthreads();

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
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            if (a < na && b < nbk)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    atomicAdd(&acc[(16 * a + 4 * q + j) * (kDwTile + 1) + 16 * b + r16], d[a][b][j]);
    __syncthreads();
    const int rows = min(kDwTile, ci - ci0), cols = min(kDwTile, co - co0);
    for (int i = tid; i < rows * cols; i += kThreads) {
        const int r = i / cols, c = i - r * cols;
        part[(item * ci + ci0 + r) * (int64_t)co + co0 + c] = acc[r * (kDwTile + 1) + c];
    }
}

__global__ void __launch_bounds__(kThreads) k_dw_reduce(const float* __restrict__ part, const int64_t* __restrict__ ibase,
                                                        int ci, int co, float* __restrict__ dW) {
    const int k = blockIdx.y;
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t cc = (int64_t)ci * co;
    if (e >= cc) return;
    float s = 0.f;
    for (int64_t it = ibase[k]; it < ibase[k + 1]; ++it) s += part[it * cc + e];
    dW[(int64_t)k * cc + e] = s;
}

// chunk of pairs per dW work item: about 1024 work items in total
static int64_t dw_chunk(int64_t n_pairs, int ci, int co) {
    const int64_t tiles = (int64_t)((ci + kDwTile - 1) / kDwTile) * ((co + kDwTile - 1) / kDwTile);
    int64_t ch = 256;
    while (ch < (int64_t)1 << 16 && (n_pairs * tiles) / ch > 1024) ch <<= 1;
    return ch;
}

static int64_t dw_items_max(int64_t n_pairs, int32_t K, int64_t ch) { return (n_pairs + ch - 1) / ch + K; }

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

template <typename TIn, typename TOut, bool WT, typename Sel>
static int launch_os(const void* X, int64_t n_x, const void* W, const int32_t* gat, const int32_t* sca,
                     const int64_t* gidx, int K, int ca, int cb, int64_t n_y, void* Y, Sel sel, hipStream_t s) {
    if (n_y == 0) return GSC_OK;
    const int64_t tiles = (n_y + kTileRows - 1) / kTileRows;
    const int64_t G = (n_y + GSC_GROUP_ROWS - 1) / GSC_GROUP_ROWS;
    dim3 grid((unsigned)tiles, (unsigned)((cb + kColSlice - 1) / kColSlice));
    hipLaunchKernelGGL((k_conv_os<TIn, TOut, WT, Sel>), grid, dim3(kThreads), 0, s, reinterpret_cast<const TIn*>(X),
                       n_x, reinterpret_cast<const TIn*>(W), gat, sca, gidx, K, G, ca, cb, n_y,
                       reinterpret_cast<TOut*>(Y), sel);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

int gsc_sparse_conv_fwd(int32_t dtype, const void* X, int64_t n_in, int32_t c_in, const void* W, int32_t c_out,
                        int32_t K, const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                        const int64_t* gidx, int64_t n_pairs, void* Y, int64_t n_out, void* stream) {
    (void)seg;
    clear_error();
    if (dtype != GSC_F32 && dtype != GSC_BF16) return fail(GSC_EINVAL, "conv_fwd: unknown dtype %d", dtype);
    if (n_in < 0 || n_out < 0 || n_in > INT32_MAX || n_out > INT32_MAX)
        return fail(GSC_EINVAL, "conv_fwd: bad row counts n_in=%lld n_out=%lld", (long long)n_in, (long long)n_out);
    if (c_in < 1 || c_out < 1) return fail(GSC_EINVAL, "conv_fwd: channels must be >= 1");
    if (K < 1 || K > kMaxKConv) return fail(GSC_EINVAL, "conv_fwd: K=%d outside [1,%d]", K, kMaxKConv);
    if (n_pairs < 0) return fail(GSC_EINVAL, "conv_fwd: n_pairs < 0");
    if (n_out > 0 && (!Y || !gidx || !W)) return fail(GSC_EINVAL, "conv_fwd: null Y/gidx/W");
    if (n_pairs > 0 && (!X || !in_idx || !out_idx)) return fail(GSC_EINVAL, "conv_fwd: null X/in_idx/out_idx");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (dtype == GSC_F32)
        return launch_os<float, float, false>(X, n_in, W, in_idx, out_idx, gidx, K, c_in, c_out, n_out, Y,
                                              WIdentity{}, s);
    return launch_os<uint16_t, uint16_t, false>(X, n_in, W, in_idx, out_idx, gidx, K, c_in, c_out, n_out, Y,
                                                WIdentity{}, s);
}

size_t gsc_conv_bwd_ws_bytes(int64_t n_pairs, int32_t c_in, int32_t c_out, int32_t K) {
    if (n_pairs < 0 || c_in < 1 || c_out < 1 || K < 1) return 0;
    const int64_t ch = dw_chunk(n_pairs, c_in, c_out);
    return al256((size_t)(K + 1) * sizeof(int64_t)) +
           al256((size_t)dw_items_max(n_pairs, K, ch) * c_in * c_out * sizeof(float)) + 256;
}

int gsc_sparse_conv_bwd(int32_t dtype, const void* X, const void* W, const void* dY, int64_t n_in, int32_t c_in,
                        int32_t c_out, int32_t K, const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                        int64_t n_pairs, const int32_t* t_in_idx, const int32_t* t_out_idx, const int64_t* t_seg,
                        const int64_t* t_gidx, int64_t t_n_pairs, const int32_t* t_wsel, void* dX, float* dW,
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
    if (dX) {
        if (t_n_pairs < 0) return fail(GSC_EINVAL, "conv_bwd: t_n_pairs < 0");
        if (n_in > 0 && (!t_gidx || !t_wsel)) return fail(GSC_EINVAL, "conv_bwd: null t_gidx/t_wsel");
        if (t_n_pairs > 0 && (!dY || !t_in_idx || !t_out_idx))
            return fail(GSC_EINVAL, "conv_bwd: null dY/t_in_idx/t_out_idx");
        WSel sel;
        for (int k = 0; k < K; ++k) {
            if (t_wsel[k] < 0 || t_wsel[k] >= K)
                return fail(GSC_EINVAL, "conv_bwd: t_wsel[%d]=%d outside [0,%d)", k, t_wsel[k], K);
            sel.w[k] = (int16_t)t_wsel[k];
        }
        int rc = dtype == GSC_F32
                     ? launch_os<float, float, true>(dY, n_out, W, t_in_idx, t_out_idx, t_gidx, K, c_out, c_in, n_in,
                                                     dX, sel, s)
                     : launch_os<uint16_t, uint16_t, true>(dY, n_out, W, t_in_idx, t_out_idx, t_gidx, K, c_out, c_in,
                                                           n_in, dX, sel, s);
        if (rc) return rc;
    }
    if (dW) {
        if (n_pairs < 0) return fail(GSC_EINVAL, "conv_bwd: n_pairs < 0");
        if (!seg || !ws) return fail(GSC_EINVAL, "conv_bwd: null seg/ws");
        if (n_pairs > 0 && (!X || !dY || !in_idx || !out_idx)) return fail(GSC_EINVAL, "conv_bwd: null X/dY/idx");
        const size_t need = gsc_conv_bwd_ws_bytes(n_pairs, c_in, c_out, K);
        if (ws_bytes < need) return fail(GSC_ESHORT, "conv_bwd: ws needs %zu bytes, got %zu", need, ws_bytes);
        const int64_t ch = dw_chunk(n_pairs, c_in, c_out);
        const int64_t items = dw_items_max(n_pairs, K, ch);
        char* w = reinterpret_cast<char*>(ws);
        int64_t* ibase = reinterpret_cast<int64_t*>(w);
        float* part = reinterpret_cast<float*>(w + al256((size_t)(K + 1) * sizeof(int64_t)));
        hipLaunchKernelGGL(k_dw_items, dim3(1), dim3(64), 0, s, seg, K, ch, ibase);
        GSC_LAUNCH_CHECK();
        const unsigned tiles = (unsigned)(((c_in + kDwTile - 1) / kDwTile) * ((c_out + kDwTile - 1) / kDwTile));
        if (dtype == GSC_F32)
            hipLaunchKernelGGL(k_dw_partial<float>, dim3((unsigned)items, tiles), dim3(kThreads), 0, s,
                               reinterpret_cast<const float*>(X), n_in, reinterpret_cast<const float*>(dY), n_out,
                               in_idx, out_idx, seg, ibase, K, ch, c_in, c_out, part);
        else
            hipLaunchKernelGGL(k_dw_partial<uint16_t>, dim3((unsigned)items, tiles), dim3(kThreads), 0, s,
                               reinterpret_cast<const uint16_t*>(X), n_in, reinterpret_cast<const uint16_t*>(dY),
                               n_out, in_idx, out_idx, seg, ibase, K, ch, c_in, c_out, part);
        GSC_LAUNCH_CHECK();
        const int64_t cc = (int64_t)c_in * c_out;
        hipLaunchKernelGGL(k_dw_reduce, dim3((unsigned)((cc + kThreads - 1) / kThreads), (unsigned)K), dim3(kThreads),
                           0, s, part, ibase, c_in, c_out, dW);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

}  // extern "C"
