// Tile plan of a kernel map for the convolution kernels.
//
// The output-stationary convolution kernels process a tile of consecutive
// output positions at a time, and every offset present in a tile costs a
// pass over that offset's weight matrix.  In the natural row order almost
// every offset occurs in every tile (a tile is a short run of voxels, and
// their neighbours point every way), so for wide layers the kernels would
// read each weight matrix once per tile.  The plan orders the output rows by
// their neighbour mask (bit k set when the row has a pair at offset k), so
// rows with the same neighbourhood shape (say, voxels of one flat surface)
// share tiles and a tile touches few offsets.
//
// The result is the same kernel map over output positions: perm[i] is the
// output row at position i, and (p_in, p_pos, p_seg, p_gidx) list every pair
// of the original map as (input row, position), grouped by offset in the
// original offset order, increasing position within an offset, with the
// 64-position group index p_gidx.  Steps:
//   masks:  one wave per 64-row group of the map: neighbour mask of every row
//           (LDS OR of the offsets' bits) and a dense table nbr[k][row] of the
//           input row of each pair;
//   sort:   stable LSD radix sort of (mask, row) by mask, 10-bit digits;
//   count:  per 64-position group a wave ballot of every offset's bit;
//   scan:   the counts give p_gidx (and p_seg);
//   fill:   each (position, offset) pair is placed at its group start plus
//           its rank among the wave's set bits.
// Everything is deterministic and runs without a host round trip.
#include <climits>

#include "gsc_internal.h"

namespace gsc {

constexpr int kPlanThreads = 256;
constexpr int kRsBits = 10;                       // radix digit width
constexpr int kRsBins = 1 << kRsBits;
constexpr int kRsPer = 16;                        // keys per thread and block
constexpr int kRsTile = kPlanThreads * kRsPer;    // keys per block

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

template <typename KeyT>
__device__ __forceinline__ KeyT key_bit(int k) {
    return (KeyT)1 << k;
}

// ---------------------------------------------------------------------------
// masks + dense neighbour table
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ void __launch_bounds__(kPlanThreads) k_plan_masks(const int32_t* __restrict__ in_idx,
                                                             const int32_t* __restrict__ out_idx,
                                                             const int64_t* __restrict__ gidx, int K, int64_t G,
                                                             int64_t n_out, KeyT* __restrict__ keys,
                                                             int32_t* __restrict__ nbr) {
    __shared__ KeyT sm[kPlanThreads / 64][64];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * (kPlanThreads / 64) + wave;
    if (g >= G) return;   // no block barrier below
    sm[wave][lane] = 0;
    int64_t lo = 0;
    int n = 0;
    if (lane < K) {
        lo = gidx[(int64_t)lane * G + g];
        n = (int)(gidx[(int64_t)lane * G + g + 1] - lo);
    }
    wave_lds_sync();
    const int64_t row0 = g * 64;
    constexpr int B = 8;   // offsets whose pairs are loaded together
    for (int k0 = 0; k0 < K; k0 += B) {
        int32_t o[B], r[B];
        bool v[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int k = min(k0 + b, K - 1);
            const int64_t klo = __shfl(lo, k, 64);
            const int kn = __shfl(n, k, 64);
            v[b] = k0 + b < K && lane < kn;
            if (v[b]) {
                o[b] = out_idx[klo + lane];
                r[b] = in_idx[klo + lane];
            }
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            if (v[b]) {
                const int64_t rel = (int64_t)o[b] - row0;
                if (rel >= 0 && rel < 64) atomicOr(&sm[wave][rel], key_bit<KeyT>(k0 + b));
                if (o[b] >= 0 && o[b] < n_out) nbr[(int64_t)(k0 + b) * n_out + o[b]] = r[b];
            }
        }
    }
    wave_lds_sync();
    if (row0 + lane < n_out) keys[row0 + lane] = sm[wave][lane];
}

// ---------------------------------------------------------------------------
// stable LSD radix sort of (key, value) by key
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ void __launch_bounds__(kPlanThreads) k_rs_hist(const KeyT* __restrict__ keys, int64_t n, int shift,
                                                          int32_t* __restrict__ hist, int64_t nb) {
    __shared__ int32_t h[kRsBins];
    for (int i = threadIdx.x; i < kRsBins; i += kPlanThreads) h[i] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
#pragma unroll
    for (int i = 0; i < kRsPer; ++i) {
        const int64_t idx = base + (int64_t)i * kPlanThreads + threadIdx.x;
        if (idx < n) atomicAdd(&h[(int)((keys[idx] >> shift) & (kRsBins - 1))], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kRsBins; i += kPlanThreads) hist[(int64_t)i * nb + blockIdx.x] = h[i];
}

// Block b places its keys in rounds of 256 (in index order: stable).  All of
// the block's keys are loaded first (16 per thread, in flight together).
// Within a wave, lanes with equal digits are found with kRsBits ballots; the
// wave's count of each digit goes to LDS, and a key's position is the block's
// running start of its digit + the counts of lower waves in this round + its
// rank in its wave.  vals_in == NULL means value = index.
template <typename KeyT>
__global__ void __launch_bounds__(kPlanThreads) k_rs_scatter(const KeyT* __restrict__ kin,
                                                             const int32_t* __restrict__ vin, int64_t n, int shift,
                                                             const int64_t* __restrict__ hoff, int64_t nb,
                                                             KeyT* __restrict__ kout, int32_t* __restrict__ vout) {
    constexpr int W = kPlanThreads / 64;
    __shared__ int64_t start[kRsBins];
    __shared__ int32_t wcnt[W][kRsBins];
    const int tid = threadIdx.x, wave = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
    KeyT key[kRsPer];
    int32_t val[kRsPer];
#pragma unroll
    for (int r = 0; r < kRsPer; ++r) {
        const int64_t idx = base + (int64_t)r * kPlanThreads + tid;
        const bool valid = idx < n;
        key[r] = valid ? kin[idx] : (KeyT)0;
        val[r] = valid ? (vin ? vin[idx] : (int32_t)idx) : 0;
    }
    for (int i = tid; i < kRsBins; i += kPlanThreads) start[i] = hoff[(int64_t)i * nb + blockIdx.x];
    for (int i = tid; i < W * kRsBins; i += kPlanThreads) (&wcnt[0][0])[i] = 0;
    const unsigned long long below = lanemask_lt();
#pragma unroll
    for (int rnd = 0; rnd < kRsPer; ++rnd) {
        const int64_t idx = base + (int64_t)rnd * kPlanThreads + tid;
        const bool valid = idx < n;
        const int d = (int)((key[rnd] >> shift) & (kRsBins - 1));
        unsigned long long peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < kRsBits; ++b) {
            const bool bit = (d >> b) & 1;
            const unsigned long long m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const int rank = __popcll(peers & below);
        __syncthreads();   // wcnt is clear, start holds this round's bases
        if (valid && rank == 0) wcnt[wave][d] = __popcll(peers);
        __syncthreads();
        int64_t pos = 0;
        if (valid) {
            pos = start[d] + rank;
            for (int w = 0; w < wave; ++w) pos += wcnt[w][d];
        }
        __syncthreads();   // every lane has read start and wcnt
        if (valid) {
            if (pos < n) {   // always true for consistent histograms; keeps a bad input from writing outside
                kout[pos] = key[rnd];
                vout[pos] = val[rnd];
            }
            if (rank == 0) {   // the lowest wave holding digit d advances start[d] by the round's count
                int32_t t = 0;
                bool first = true;
                for (int w = 0; w < W; ++w) {
                    t += wcnt[w][d];
                    if (w < wave) first = first && wcnt[w][d] == 0;
                }
                if (first) start[d] += t;
            }
        }
        __syncthreads();   // start updated by the first holders of each digit
        if (valid && rank == 0) wcnt[wave][d] = 0;
    }
}

// ---------------------------------------------------------------------------
// plan map: counts per (offset, 64-position group), then the fill
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ void __launch_bounds__(kPlanThreads) k_plan_count(const KeyT* __restrict__ keys, int64_t n, int K,
                                                             int64_t G, int32_t* __restrict__ cnt) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * (kPlanThreads / 64) + wave;
    if (g >= G) return;
    const int64_t i = g * 64 + lane;
    const KeyT key = i < n ? keys[i] : (KeyT)0;
    int mine = 0;
    for (int k = 0; k < K; ++k) {
        const int c = __popcll(__ballot((key >> k) & 1));
        if (lane == k) mine = c;
    }
    if (lane < K) cnt[(int64_t)lane * G + g] = mine;
}

template <typename KeyT>
__global__ void __launch_bounds__(kPlanThreads) k_plan_fill(const KeyT* __restrict__ keys,
                                                            const int32_t* __restrict__ perm,
                                                            const int32_t* __restrict__ nbr,
                                                            const int64_t* __restrict__ pgidx, int64_t n, int K,
                                                            int64_t G, int64_t cap, int32_t* __restrict__ p_in,
                                                            int32_t* __restrict__ p_pos) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t g = (int64_t)blockIdx.x * (kPlanThreads / 64) + wave;
    if (g >= G) return;
    const int64_t i = g * 64 + lane;
    const bool valid = i < n;
    const KeyT key = valid ? keys[i] : (KeyT)0;
    const int64_t row = valid ? perm[i] : 0;
    const int64_t st = lane < K ? pgidx[(int64_t)lane * G + g] : 0;
    const unsigned long long below = lanemask_lt();
    constexpr int B = 8;
    for (int k0 = 0; k0 < K; k0 += B) {
        int32_t r[B];
        int64_t pos[B];
        bool v[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int k = min(k0 + b, K - 1);
            v[b] = k0 + b < K && ((key >> k) & 1);
            const unsigned long long m = __ballot(v[b]);
            pos[b] = __shfl(st, k, 64) + __popcll(m & below);
            if (v[b]) r[b] = nbr[(int64_t)k * n + row];
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            if (v[b] && pos[b] < cap) {
                p_in[pos[b]] = r[b];
                p_pos[pos[b]] = (int32_t)i;
            }
        }
    }
}

template <typename KeyT>
static int plan_enqueue(const int32_t* in_idx, const int32_t* out_idx, const int64_t* gidx, int64_t n, int K,
                        int64_t cap, int32_t* perm, int32_t* p_in, int32_t* p_pos, int64_t* p_seg, int64_t* p_gidx,
                        void* ws, hipStream_t s) {
    const int64_t G = (n + 63) / 64;
    const int64_t nb = (n + kRsTile - 1) / kRsTile;
    char* w = reinterpret_cast<char*>(ws);
    KeyT* ka = reinterpret_cast<KeyT*>(w);
    w += al256((size_t)n * sizeof(KeyT));
    KeyT* kb = reinterpret_cast<KeyT*>(w);
    w += al256((size_t)n * sizeof(KeyT));
    int32_t* va = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)n * sizeof(int32_t));
    int32_t* vb = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)n * sizeof(int32_t));
    int32_t* hist = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)kRsBins * nb * sizeof(int32_t));
    int64_t* hoff = reinterpret_cast<int64_t*>(w);
    w += al256((size_t)(kRsBins * nb + 1) * sizeof(int64_t));
    int32_t* nbr = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)K * n * sizeof(int32_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)K * G * sizeof(int32_t));
    void* scan_ws = w;

    const unsigned gblocks = (unsigned)((G + kPlanThreads / 64 - 1) / (kPlanThreads / 64));
    if (n > 0) {
        hipLaunchKernelGGL((k_plan_masks<KeyT>), dim3(gblocks), dim3(kPlanThreads), 0, s, in_idx, out_idx, gidx, K,
                           G, n, ka, nbr);
        GSC_LAUNCH_CHECK();
        const int passes = (K + kRsBits - 1) / kRsBits;
        const KeyT* kin = ka;
        const int32_t* vin = nullptr;
        for (int p = 0; p < passes; ++p) {
            KeyT* kout = (p & 1) ? ka : kb;
            int32_t* vout = (p == passes - 1) ? perm : ((p & 1) ? va : vb);
            hipLaunchKernelGGL((k_rs_hist<KeyT>), dim3((unsigned)nb), dim3(kPlanThreads), 0, s, kin, n, p * kRsBits,
                               hist, nb);
            GSC_LAUNCH_CHECK();
            int rc = scan_counts(hist, kRsBins * nb, hoff, nullptr, scan_ws, s);
            if (rc) return rc;
            hipLaunchKernelGGL((k_rs_scatter<KeyT>), dim3((unsigned)nb), dim3(kPlanThreads), 0, s, kin, vin, n,
                               p * kRsBits, hoff, nb, kout, vout);
            GSC_LAUNCH_CHECK();
            kin = kout;
            vin = vout;
        }
        hipLaunchKernelGGL((k_plan_count<KeyT>), dim3(gblocks), dim3(kPlanThreads), 0, s, kin, n, K, G, cnt);
        GSC_LAUNCH_CHECK();
        int rc = scan_counts(cnt, K * G, p_gidx, nullptr, scan_ws, s);
        if (rc) return rc;
        rc = seg_from_gidx(p_gidx, K, G, p_seg, s);
        if (rc) return rc;
        hipLaunchKernelGGL((k_plan_fill<KeyT>), dim3(gblocks), dim3(kPlanThreads), 0, s, kin, perm, nbr, p_gidx, n, K,
                           G, cap, p_in, p_pos);
        GSC_LAUNCH_CHECK();
    } else {
        hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(256), 0, s, p_seg, (int64_t)K + 1);
        GSC_LAUNCH_CHECK();
        hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(256), 0, s, p_gidx, (int64_t)1);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

size_t gsc_conv_plan_ws_bytes(int64_t n_out, int32_t K) {
    if (n_out < 0 || K < 1 || K > kPlanMaxK) return 0;
    const int64_t G = (n_out + 63) / 64;
    const int64_t nb = (n_out + kRsTile - 1) / kRsTile;
    size_t b = 2 * al256((size_t)n_out * sizeof(uint64_t));
    b += 2 * al256((size_t)n_out * sizeof(int32_t));
    b += al256((size_t)kRsBins * nb * sizeof(int32_t));
    b += al256((size_t)(kRsBins * nb + 1) * sizeof(int64_t));
    b += al256((size_t)K * n_out * sizeof(int32_t));
    b += al256((size_t)K * G * sizeof(int32_t));
    const int64_t m = kRsBins * nb > K * G ? kRsBins * nb : K * G;
    b += scan_ws_bytes(m);
    return b + 256;
}

int gsc_conv_plan(const int32_t* in_idx, const int32_t* out_idx, const int64_t* gidx, int64_t n_out, int32_t K,
                  int64_t cap_pairs, int32_t* perm, int32_t* p_in, int32_t* p_pos, int64_t* p_seg, int64_t* p_gidx,
                  void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (K < 1 || K > kPlanMaxK) return fail(GSC_EINVAL, "conv_plan: K=%d outside [1,%d]", K, kPlanMaxK);
    if (n_out < 0 || n_out > INT32_MAX) return fail(GSC_EINVAL, "conv_plan: n_out=%lld invalid", (long long)n_out);
    if (cap_pairs < 0) return fail(GSC_EINVAL, "conv_plan: cap_pairs < 0");
    if (!p_seg || !p_gidx || !ws) return fail(GSC_EINVAL, "conv_plan: null p_seg/p_gidx/ws");
    if (n_out > 0 && (!gidx || !perm)) return fail(GSC_EINVAL, "conv_plan: null gidx/perm");
    if (cap_pairs > 0 && (!in_idx || !out_idx || !p_in || !p_pos))
        return fail(GSC_EINVAL, "conv_plan: null in_idx/out_idx/p_in/p_pos");
    const size_t need = gsc_conv_plan_ws_bytes(n_out, K);
    if (ws_bytes < need) return fail(GSC_ESHORT, "conv_plan: ws needs %zu bytes, got %zu", need, ws_bytes);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (K <= 32)
        return plan_enqueue<uint32_t>(in_idx, out_idx, gidx, n_out, K, cap_pairs, perm, p_in, p_pos, p_seg, p_gidx,
                                      ws, s);
    return plan_enqueue<unsigned long long>(in_idx, out_idx, gidx, n_out, K, cap_pairs, perm, p_in, p_pos, p_seg,
                                            p_gidx, ws, s);
}

}  // extern "C"
