// Block plan of a kernel map for the convolution kernels.
//
// The block convolution engines compute 16 output rows at a time (one MFMA
// row block) and keep the block's sums in registers: for every offset that
// any of the 16 rows has, they gather the 16 input rows (a zero row where a
// row has no pair at that offset) and multiply by that offset's weights.  The
// cost of a block is therefore the number of distinct offsets among its rows.
// In the natural row order a block's rows point every way and almost all
// offsets occur; the plan orders the output rows by neighbour mask (bit k set
// when the row has a pair at offset k), so rows with the same neighbourhood
// shape share blocks, and the blocks' offset sets shrink to about those of
// single rows.
//
// Output, for n_out rows, nb = ceil(n_out / 16) blocks:
//   perm[i]      output row at position i (i < n_out);
//   bmask[b]     union of the masks of block b's rows (positions 16b..16b+15);
//   ibase[b]     first item of block b (exclusive scan of popcount(bmask));
//                ibase[nb] = number of items;
//   items[16*t + r]  for item t = ibase[b] + j, the j-th offset k of bmask[b]
//                in increasing order: the input row paired with position
//                16b + r at offset k, or -1 if there is none.
// Input: the map's dense form nbr[k][j] (input row or -1), which the kernel
// map writes as it probes.  Steps:
//   masks:  every row's mask from its column of nbr;
//   sort:   stable LSD radix sort of (mask, row) by mask, 10-bit digits;
//   count:  block unions and item counts; a scan gives ibase;
//   fill:   one lane per position writes its entry of each of its block's
//           items.
// Everything is deterministic and runs without a host round trip.
#include <climits>

#include "gsc_internal.h"

namespace gsc {

constexpr int kPlanThreads = 256;
constexpr int kRsBits = 10;                       // radix digit width
constexpr int kRsBins = 1 << kRsBits;
constexpr int kRsThreads = 1024;                  // radix sort block
constexpr int kRsPer = 4;                         // keys per thread and block
constexpr int kRsTile = kRsThreads * kRsPer;      // keys per block

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------
// masks from the dense map
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kPlanThreads) k_plan_masks(const int32_t* __restrict__ nbr, int64_t n, int K,
                                                             uint32_t* __restrict__ keys) {
    const int64_t j = (int64_t)blockIdx.x * kPlanThreads + threadIdx.x;
    if (j >= n) return;
    uint32_t m = 0;
    constexpr int B = 8;   // table entries loaded together
    for (int k0 = 0; k0 < K; k0 += B) {
        int32_t r[B];
#pragma unroll
        for (int b = 0; b < B; ++b) r[b] = k0 + b < K ? nbr[(int64_t)(k0 + b) * n + j] : -1;
#pragma unroll
        for (int b = 0; b < B; ++b) m |= (uint32_t)(r[b] >= 0) << ((k0 + b) & 31);
    }
    keys[j] = m;
}

// ---------------------------------------------------------------------------
// stable LSD radix sort of (key, value) by key
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ void __launch_bounds__(kRsThreads) k_rs_hist(const KeyT* __restrict__ keys, int64_t n, int shift,
                                                        int32_t* __restrict__ hist, int64_t nb) {
    __shared__ int32_t h[kRsBins];
    for (int i = threadIdx.x; i < kRsBins; i += kRsThreads) h[i] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
    KeyT key[kRsPer];
#pragma unroll
    for (int i = 0; i < kRsPer; ++i) {
        const int64_t idx = base + (int64_t)i * kRsThreads + threadIdx.x;
        key[i] = idx < n ? keys[idx] : (KeyT)0;
    }
#pragma unroll
    for (int i = 0; i < kRsPer; ++i)
        if (base + (int64_t)i * kRsThreads + threadIdx.x < n) atomicAdd(&h[(int)((key[i] >> shift) & (kRsBins - 1))], 1);
    __syncthreads();
    for (int i = threadIdx.x; i < kRsBins; i += kRsThreads) hist[(int64_t)i * nb + blockIdx.x] = h[i];
}

// Block b places its keys in rounds of kRsThreads (in index order: stable).
// All of the block's keys are loaded first (kRsPer per thread, in flight
// together).  Within a wave, lanes with equal digits are found with kRsBits
// ballots; the wave's count of each digit goes to LDS, and a key's position
// is the block's running start of its digit + the counts of lower waves in
// this round + its rank in its wave.  vals_in == NULL means value = index.
template <typename KeyT>
__global__ void __launch_bounds__(kRsThreads) k_rs_scatter(const KeyT* __restrict__ kin,
                                                           const int32_t* __restrict__ vin, int64_t n, int shift,
                                                           const int64_t* __restrict__ hoff, int64_t nb,
                                                           KeyT* __restrict__ kout, int32_t* __restrict__ vout) {
    constexpr int W = kRsThreads / 64;
    __shared__ int64_t start[kRsBins];
    __shared__ int32_t wcnt[W][kRsBins];
    const int tid = threadIdx.x, wave = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
    KeyT key[kRsPer];
    int32_t val[kRsPer];
#pragma unroll
    for (int r = 0; r < kRsPer; ++r) {
        const int64_t idx = base + (int64_t)r * kRsThreads + tid;
        const bool valid = idx < n;
        key[r] = valid ? kin[idx] : (KeyT)0;
        val[r] = valid ? (vin ? vin[idx] : (int32_t)idx) : 0;
    }
    for (int i = tid; i < kRsBins; i += kRsThreads) start[i] = hoff[(int64_t)i * nb + blockIdx.x];
    for (int i = tid; i < W * kRsBins; i += kRsThreads) (&wcnt[0][0])[i] = 0;
    const unsigned long long below = lanemask_lt();
#pragma unroll
    for (int rnd = 0; rnd < kRsPer; ++rnd) {
        const int64_t idx = base + (int64_t)rnd * kRsThreads + tid;
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
// blocks: union masks and item counts, then the items
// ---------------------------------------------------------------------------
// OR of a value over the 16 lanes of its block (lanes 16j..16j+15).
__device__ __forceinline__ uint32_t block_or16(uint32_t v) {
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) v |= (uint32_t)__shfl_xor((int)v, d, 64);
    return v;
}

__global__ void __launch_bounds__(kPlanThreads) k_blk_count(const uint32_t* __restrict__ keys, int64_t n, int64_t nb,
                                                            uint32_t* __restrict__ bmask, int32_t* __restrict__ cnt) {
    const int64_t i = (int64_t)blockIdx.x * kPlanThreads + threadIdx.x;
    const uint32_t u = block_or16(i < n ? keys[i] : 0u);
    const int64_t b = i >> 4;
    if ((threadIdx.x & 15) == 0 && b < nb) {
        bmask[b] = u;
        cnt[b] = __popc(u);
    }
}

__global__ void __launch_bounds__(kPlanThreads) k_blk_fill(const uint32_t* __restrict__ keys,
                                                           const int32_t* __restrict__ perm,
                                                           const int32_t* __restrict__ nbr,
                                                           const int64_t* __restrict__ ibase, int64_t n, int64_t nb,
                                                           int32_t* __restrict__ items) {
    const int64_t i = (int64_t)blockIdx.x * kPlanThreads + threadIdx.x;
    const int64_t b = i >> 4;
    const int r = threadIdx.x & 15;
    const bool valid = i < n;
    const uint32_t key = valid ? keys[i] : 0u;
    const uint32_t u = block_or16(key);
    if (b >= nb) return;   // whole blocks of 16 lanes leave together
    const int64_t row = valid ? perm[i] : 0;
    const int64_t base = ibase[b];
    uint32_t m = u;
    for (int j = 0; m != 0; ++j) {
        const int k = __ffs(m) - 1;
        m &= m - 1;
        items[(base + j) * 16 + r] = ((key >> k) & 1u) ? nbr[(int64_t)k * n + row] : -1;
    }
}

static int plan_enqueue(const int32_t* nbr, int64_t n, int K, int32_t* perm, uint32_t* bmask, int64_t* ibase,
                        int32_t* items, void* ws, hipStream_t s) {
    const int64_t nb = (n + 15) / 16;
    const int64_t nrs = (n + kRsTile - 1) / kRsTile;
    char* w = reinterpret_cast<char*>(ws);
    uint32_t* ka = reinterpret_cast<uint32_t*>(w);
    w += al256((size_t)n * sizeof(uint32_t));
    uint32_t* kb = reinterpret_cast<uint32_t*>(w);
    w += al256((size_t)n * sizeof(uint32_t));
    int32_t* va = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)n * sizeof(int32_t));
    int32_t* vb = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)n * sizeof(int32_t));
    int32_t* hist = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)kRsBins * nrs * sizeof(int32_t));
    int64_t* hoff = reinterpret_cast<int64_t*>(w);
    w += al256((size_t)(kRsBins * nrs + 1) * sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)nb * sizeof(int32_t));
    void* scan_ws = w;

    if (n == 0) {
        hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(256), 0, s, ibase, (int64_t)1);
        GSC_LAUNCH_CHECK();
        return GSC_OK;
    }
    const unsigned pblocks = (unsigned)((n + kPlanThreads - 1) / kPlanThreads);
    hipLaunchKernelGGL(k_plan_masks, dim3(pblocks), dim3(kPlanThreads), 0, s, nbr, n, K, ka);
    GSC_LAUNCH_CHECK();
    const int passes = (K + kRsBits - 1) / kRsBits;
    const uint32_t* kin = ka;
    const int32_t* vin = nullptr;
    for (int p = 0; p < passes; ++p) {
        uint32_t* kout = (p & 1) ? ka : kb;
        int32_t* vout = (p == passes - 1) ? perm : ((p & 1) ? va : vb);
        hipLaunchKernelGGL((k_rs_hist<uint32_t>), dim3((unsigned)nrs), dim3(kRsThreads), 0, s, kin, n,
                           p * kRsBits, hist, nrs);
        GSC_LAUNCH_CHECK();
        int rc = scan_counts(hist, kRsBins * nrs, hoff, nullptr, scan_ws, s);
        if (rc) return rc;
        hipLaunchKernelGGL((k_rs_scatter<uint32_t>), dim3((unsigned)nrs), dim3(kRsThreads), 0, s, kin, vin, n,
                           p * kRsBits, hoff, nrs, kout, vout);
        GSC_LAUNCH_CHECK();
        kin = kout;
        vin = vout;
    }
    hipLaunchKernelGGL(k_blk_count, dim3(pblocks), dim3(kPlanThreads), 0, s, kin, n, nb, bmask, cnt);
    GSC_LAUNCH_CHECK();
    int rc = scan_counts(cnt, nb, ibase, nullptr, scan_ws, s);
    if (rc) return rc;
    hipLaunchKernelGGL(k_blk_fill, dim3(pblocks), dim3(kPlanThreads), 0, s, kin, perm, nbr, ibase, n, nb, items);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

int64_t gsc_plan_blocks(int64_t n_out) { return n_out <= 0 ? 0 : (n_out + 15) / 16; }

size_t gsc_conv_plan_ws_bytes(int64_t n_out, int32_t K) {
    if (n_out < 0 || K < 1 || K > kPlanMaxK) return 0;
    const int64_t nb = (n_out + 15) / 16;
    const int64_t nrs = (n_out + kRsTile - 1) / kRsTile;
    size_t b = 4 * al256((size_t)n_out * sizeof(uint32_t));
    b += al256((size_t)kRsBins * nrs * sizeof(int32_t));
    b += al256((size_t)(kRsBins * nrs + 1) * sizeof(int64_t));
    b += al256((size_t)nb * sizeof(int32_t));
    const int64_t m = kRsBins * nrs > nb ? kRsBins * nrs : nb;
    b += scan_ws_bytes(m);
    return b + 256;
}

int gsc_conv_plan(const int32_t* nbr, int64_t n_out, int32_t K, int32_t* perm, uint32_t* bmask, int64_t* ibase,
                  int32_t* items, int64_t cap_items, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (K < 1 || K > kPlanMaxK) return fail(GSC_EINVAL, "conv_plan: K=%d outside [1,%d]", K, kPlanMaxK);
    if (n_out < 0 || n_out > INT32_MAX) return fail(GSC_EINVAL, "conv_plan: n_out=%lld invalid", (long long)n_out);
    if (!ibase || !ws) return fail(GSC_EINVAL, "conv_plan: null ibase/ws");
    if (n_out > 0 && (!nbr || !perm || !bmask || !items))
        return fail(GSC_EINVAL, "conv_plan: null nbr/perm/bmask/items");
    const int64_t need_items = (int64_t)K * gsc_plan_blocks(n_out);
    if (cap_items < need_items)
        return fail(GSC_ESHORT, "conv_plan: cap_items=%lld, need K*ceil(n_out/16) = %lld", (long long)cap_items,
                    (long long)need_items);
    const size_t need = gsc_conv_plan_ws_bytes(n_out, K);
    if (ws_bytes < need) return fail(GSC_ESHORT, "conv_plan: ws needs %zu bytes, got %zu", need, ws_bytes);
    return plan_enqueue(nbr, n_out, K, perm, bmask, ibase, items, ws, reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"
