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
// single rows.  The sort key puts the mask's popcount, capped to the bits
// that the last 10-bit digit leaves free, above the mask: rows are grouped
// by neighbour count first, so a run of blocks (the tile engine's tile of
// 16) also has fewer distinct offsets, and the plan's positions come in
// rough order of cost (which the tile engine uses to hand out its largest
// tiles first).
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
//   sort:   stable LSD radix sort of (key, row) by key = (min(popcount of
//           the mask, cap) << K) | mask, 10-bit digits, one kernel per digit
//           (cap: plan_key_cap);
//   count:  block unions and item counts; a scan gives ibase;
//   fill:   one lane per position writes its entry of each of its block's
//           items.
// Everything is deterministic and runs without a host round trip.
#include <algorithm>
#include <climits>
#include <cstdlib>

#include "gsc_internal.h"

namespace gsc {

constexpr int kPlanThreads = 256;
constexpr int kRsBits = 10;                       // radix digit width
constexpr int kRsBins = 1 << kRsBits;
constexpr int kRsThreads = 1024;                  // radix sort block
constexpr int kRsPer = 2;                         // keys per thread and block (2048-key tiles: more tiles in flight)
constexpr int kRsTile = kRsThreads * kRsPer;      // keys per block

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

// The popcount field of the sort key: as many bits as the last 10-bit digit
// of the K-bit mask leaves free (at most 6, and within a 32-bit key); its
// largest value, 0 when there is no room.  K = 27: 3 bits, counts capped at 7.
__host__ __device__ inline int plan_key_pbits(int K) {
    const int spare = (K + kRsBits - 1) / kRsBits * kRsBits - K;
    const int a = spare < 32 - K ? spare : 32 - K;
    return a < 6 ? a : 6;
}
__host__ __device__ inline uint32_t plan_key_cap(int K) { return (1u << plan_key_pbits(K)) - 1u; }

// Offsets of plan range r of a K-offset map planned in ranges of S offsets
// (the last one may be shorter), and their mask bits.
__host__ __device__ inline int range_k0(int r, int S) { return r * S; }
__host__ __device__ inline int range_len(int r, int S, int K) { return K - r * S < S ? K - r * S : S; }
__host__ __device__ inline uint32_t range_kmask(int kr) { return kr >= 32 ? ~0u : (1u << kr) - 1u; }

// ---------------------------------------------------------------------------
// masks from the dense map
// ---------------------------------------------------------------------------
// Range r = blockIdx.y of the plan: keys[r * n + j] for its offsets.  (Also
// clears the sort's counters and first look-back entries, zero[0, nzero),
// which the histogram kernel after it starts to fill.)
__global__ void __launch_bounds__(kPlanThreads) k_plan_masks(const int32_t* __restrict__ nbr, int64_t n, int Kall,
                                                             int S, uint32_t* __restrict__ keys,
                                                             uint32_t* __restrict__ zero, int64_t nzero,
                                                             uint32_t* __restrict__ lb_status) {
    const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;   // block number over all ranges
    if (lb_status && lin == 0 && threadIdx.x == 0) *lb_status = 0u;     // the plan call's first kernel
    for (int64_t i = lin * kPlanThreads + threadIdx.x; i < nzero; i += (int64_t)gridDim.x * gridDim.y * kPlanThreads)
        zero[i] = 0;
    const int rg = blockIdx.y;
    const int K = range_len(rg, S, Kall);
    const uint32_t cap = plan_key_cap(K);
    nbr += (int64_t)range_k0(rg, S) * n;
    keys += (int64_t)rg * n;
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
    const uint32_t c = min((uint32_t)__popc(m), cap);
    keys[j] = cap ? m | (c << K) : m;   // cap > 0 only where K + its bits <= 32
}

// ---------------------------------------------------------------------------
// stable LSD radix sort of (key, value) by key, one kernel per pass
// ---------------------------------------------------------------------------
// The digit counts of every pass over all keys come first (one histogram
// kernel); each tile of a pass scans its pass's counts to know where each
// digit's range starts.  A pass kernel
// takes tiles of kRsTile keys in ticket order (an atomic counter, so every
// tile a block waits for is already running), publishes its tile's count of
// each digit and looks back over the earlier tiles' published counts to find
// how many keys with that digit precede the tile (the decoupled look-back
// of Merrill and Garland's single-pass prefix scan: a tile's entry holds
// either its own count or, once known, its inclusive prefix).  The keys are then placed stably: in rounds of kRsThreads keys in
// index order, lanes with equal digits found with kRsBits ballots.
constexpr int kRsMaxPasses = 4;                   // keys of up to 40 bits
constexpr uint32_t kStAgg = 1u << 30;             // entry holds the tile's own count
constexpr uint32_t kStIncl = 1u << 31;            // entry holds the inclusive prefix
constexpr uint32_t kStCount = kStAgg - 1;
constexpr int64_t kRsMaxKeys = kStCount;          // counts must fit below the flag bits
constexpr int kSpinMax = 1 << 22;                 // bound on polls of one entry (not reached in practice)

// Range r = blockIdx.y: its keys at keys + r * n, its counts at
// ghist + r * kRsMaxPasses * kRsBins.
__global__ void __launch_bounds__(kRsThreads) k_rs_ghist(const uint32_t* __restrict__ keys, int64_t n, int passes,
                                                         uint32_t* __restrict__ ghist) {
    __shared__ int32_t h[kRsMaxPasses][kRsBins];
    keys += (int64_t)blockIdx.y * n;
    ghist += (int64_t)blockIdx.y * kRsMaxPasses * kRsBins;
    for (int i = threadIdx.x; i < kRsMaxPasses * kRsBins; i += kRsThreads) (&h[0][0])[i] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kRsTile;
    uint32_t key[kRsPer];
#pragma unroll
    for (int i = 0; i < kRsPer; ++i) {
        const int64_t idx = base + (int64_t)i * kRsThreads + threadIdx.x;
        key[i] = idx < n ? keys[idx] : 0u;
    }
#pragma unroll
    for (int i = 0; i < kRsPer; ++i) {
        if (base + (int64_t)i * kRsThreads + threadIdx.x < n)
            for (int p = 0; p < passes; ++p) atomicAdd(&h[p][(key[i] >> (p * kRsBits)) & (kRsBins - 1)], 1);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < passes * kRsBins; i += kRsThreads) {
        const int32_t c = (&h[0][0])[i];
        if (c) atomicAdd(&ghist[i], (uint32_t)c);
    }
}

// Tiles of all ranges share the ticket: ticket T is tile T % nrs of range
// T / nrs, which looks back over its own range's tiles only (all of them
// took smaller tickets).  Range r's keys and values are at r * n, its look-
// back entries at r * nrs * kRsBins, its digit counts at r * kRsMaxPasses *
// kRsBins (ghist points at the pass's row of range 0).
__global__ void __launch_bounds__(kRsThreads) k_rs_pass(const uint32_t* __restrict__ kin,
                                                        const int32_t* __restrict__ vin, int64_t n, int64_t nrs,
                                                        int R, int shift, const uint32_t* __restrict__ ghist,
                                                        uint32_t* __restrict__ status,
                                                        uint32_t* __restrict__ status_next,
                                                        uint32_t* __restrict__ ticket, uint32_t* __restrict__ kout,
                                                        int32_t* __restrict__ vout, int spin_max,
                                                        uint32_t* __restrict__ lb_status) {
    constexpr int W = kRsThreads / 64;
    static_assert(kRsThreads == kRsBins, "one thread per digit in the look-back");
    __shared__ int64_t start[kRsBins];
    __shared__ int32_t hist[kRsBins];
    __shared__ int32_t wcnt[W][kRsBins];
    __shared__ int64_t tile_sh;
    __shared__ int64_t wsum[W];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    if (tid == 0) tile_sh = atomicAdd(ticket, 1u);
    hist[tid] = 0;
    for (int i = tid; i < W * kRsBins; i += kRsThreads) (&wcnt[0][0])[i] = 0;
    // the pass's digit counts: range 0's load while the ticket is out (a
    // single-range plan waits for nothing more); a tile of another range
    // loads its own once the ticket has told it its range
    int64_t dc = ghist[tid];
    int64_t rg = 0;   // the tile's range
    if (R > 1) {      // uniform
        __syncthreads();
        rg = (int64_t)tile_sh / nrs;
        if (rg != 0) dc = ghist[rg * kRsMaxPasses * kRsBins + tid];
    }
    kin += rg * n;
    vout += rg * n;
    kout += rg * n;
    if (vin) vin += rg * n;
    status += rg * nrs * kRsBins;
    status_next += rg * nrs * kRsBins;
    // where digit tid's keys start in this pass's output (the keys of smaller
    // digits): every tile scans the pass's digit counts itself
    int64_t dinc = dc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t u = __shfl_up(dinc, o, 64);
        if (lane >= o) dinc += u;
    }
    if (lane == 63) wsum[wave] = dinc;
    __syncthreads();
    int64_t dbase = dinc - dc;
    for (int i = 0; i < wave; ++i) dbase += wsum[i];
    const int64_t t = tile_sh - rg * nrs;   // (visible: a barrier has passed since thread 0 set it)
    const int64_t base = t * kRsTile;
    status_next[t * kRsBins + tid] = 0;   // the next pass's entry of this tile (that array is idle now)
    uint32_t key[kRsPer];
    int32_t val[kRsPer];
#pragma unroll
    for (int r = 0; r < kRsPer; ++r) {
        const int64_t idx = base + (int64_t)r * kRsThreads + tid;
        const bool valid = idx < n;
        key[r] = valid ? kin[idx] : 0u;
        val[r] = valid ? (vin ? vin[idx] : (int32_t)idx) : 0;
    }
#pragma unroll
    for (int r = 0; r < kRsPer; ++r)
        if (base + (int64_t)r * kRsThreads + tid < n) atomicAdd(&hist[(key[r] >> shift) & (kRsBins - 1)], 1);
    __syncthreads();
    {   // publish this tile's count of digit tid, then look back for the keys before the tile
        // (the entries are the only data exchanged, so relaxed atomics at
        // agent scope suffice: they go to L2 and every poll sees the latest)
        const uint32_t c = (uint32_t)hist[tid];
        uint32_t* mine = status + t * kRsBins + tid;
        uint32_t before = 0;
        __hip_atomic_store(mine, (t == 0 ? kStIncl : kStAgg) | c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (t > 0) {
            constexpr int LW = 4;   // predecessors' entries loaded together (wider batches read more entries past the first inclusive one, and measured slower)
            bool done = false;
            for (int64_t j0 = t - 1; !done && j0 >= 0; j0 -= LW) {
                uint32_t v[LW];
#pragma unroll
                for (int i = 0; i < LW; ++i)
                    v[i] = j0 - i >= 0 ? __hip_atomic_load(status + (j0 - i) * kRsBins + tid, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT)
                                       : kStIncl;
#pragma unroll
                for (int i = 0; i < LW; ++i) {
                    if (done) break;
                    uint32_t x = spin_max < 0 ? 0u : v[i];   // spin_max < 0: give up at once (tests only)
                    for (int spin = 0; x == 0 && spin < spin_max; ++spin) {   // not published yet: it will be
                        __builtin_amdgcn_s_sleep(1);
                        x = __hip_atomic_load(status + (j0 - i) * kRsBins + tid, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
                    }
                    if (x == 0) {   // gave up: the prefix is wrong, and the plan call's status says so
                        __hip_atomic_fetch_or(lb_status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        done = true;
                        break;
                    }
                    before += x & kStCount;
                    done = (x & kStIncl) != 0;
                }
            }
            __hip_atomic_store(mine, kStIncl | (before + c), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        start[tid] = dbase + before;
    }
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
            if (pos >= 0 && pos < n) {   // always true for consistent counts; keeps a bad input from writing outside
                kout[pos] = key[rnd];
                vout[pos] = val[rnd];
            }
            if (rank == 0) {   // the lowest wave holding digit d advances start[d] by the round's count
                int32_t c = 0;
                bool first = true;
                for (int w = 0; w < W; ++w) {
                    c += wcnt[w][d];
                    if (w < wave) first = first && wcnt[w][d] == 0;
                }
                if (first) start[d] += c;
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

// Range r = blockIdx.y (its keys at r * n, its blocks at r * nb).  (The
// sorted keys are masked to the range's offsets and the rows clamped to
// [0, n): after a look-back that gave up they need not be what the sort
// meant, and the plan must still stay inside its arrays.)
__global__ void __launch_bounds__(kPlanThreads) k_blk_count(const uint32_t* __restrict__ keys, int Kall, int S,
                                                            int64_t n, int64_t nb, uint32_t* __restrict__ bmask,
                                                            int32_t* __restrict__ cnt) {
    const int rg = blockIdx.y;
    const uint32_t kmask = range_kmask(range_len(rg, S, Kall));
    keys += (int64_t)rg * n;
    bmask += (int64_t)rg * nb;
    cnt += (int64_t)rg * nb;
    const int64_t i = (int64_t)blockIdx.x * kPlanThreads + threadIdx.x;
    const uint32_t u = block_or16(i < n ? keys[i] & kmask : 0u);
    const int64_t b = i >> 4;
    if ((threadIdx.x & 15) == 0 && b < nb) {
        bmask[b] = u;
        cnt[b] = __popc(u);
    }
}

// Range r = blockIdx.y: keys and perm at r * n, the range's offsets' dense
// rows from nbr + k0 * n, ibase at r * (nb + 1), items from items + 16 k0 nb.
__global__ void __launch_bounds__(kPlanThreads) k_blk_fill(const uint32_t* __restrict__ keys, int Kall, int S,
                                                           const int32_t* __restrict__ perm,
                                                           const int32_t* __restrict__ nbr,
                                                           const int64_t* __restrict__ ibase, int64_t n, int64_t nb,
                                                           int32_t* __restrict__ items) {
    const int rg = blockIdx.y;
    const int k0 = range_k0(rg, S);
    const uint32_t kmask = range_kmask(range_len(rg, S, Kall));
    keys += (int64_t)rg * n;
    perm += (int64_t)rg * n;
    nbr += (int64_t)k0 * n;
    ibase += (int64_t)rg * (nb + 1);
    items += (int64_t)k0 * nb * 16;
    const int64_t i = (int64_t)blockIdx.x * kPlanThreads + threadIdx.x;
    const int64_t b = i >> 4;
    const int r = threadIdx.x & 15;
    const bool valid = i < n;
    const uint32_t key = valid ? keys[i] & kmask : 0u;
    const uint32_t u = block_or16(key);
    if (b >= nb) return;   // whole blocks of 16 lanes leave together
    const int32_t pr = valid ? perm[i] : 0;
    const int64_t row = pr >= 0 && pr < n ? pr : 0;
    const int64_t base = ibase[b];
    uint32_t m = u;
    // four of the block's offsets per round, their table entries loaded together
    for (int j = 0; m != 0; j += 4) {
        int kk[4];
        int32_t v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            kk[t] = m ? __ffs(m) - 1 : -1;
            m &= m - 1;
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = kk[t] >= 0 && ((key >> kk[t]) & 1u) ? nbr[(int64_t)kk[t] * n + row] : -1;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (kk[t] >= 0) items[(base + j + t) * 16 + r] = v[t];
    }
}

// Sets each range's ibase[0] = 0 (ibase[r]: nb = 0) and clears the
// look-back status (a plan over no rows).
__global__ void k_plan_empty(int64_t* ibase, int R, uint32_t* lb_status) {
    if (blockIdx.x == 0 && (int)threadIdx.x < R) {
        ibase[threadIdx.x] = 0;
        if (lb_status && threadIdx.x == 0) *lb_status = 0u;
    }
}

// The workspace of a plan over n rows in R ranges: keys and values twice,
// the zeroed counters (digit counts per range and pass, tickets, the first
// pass's look-back entries), the second look-back array, block item counts,
// the scan's scratch.
struct PlanWs {
    uint32_t *ka, *kb;
    int32_t *va, *vb;
    uint32_t *ghist, *ticket, *st0, *st1;
    int64_t nzero;
    int32_t* cnt;
    void* scan_ws;
    size_t bytes;   // up to here
};

static PlanWs plan_ws_layout(void* ws, int64_t n, int R) {
    const int64_t nb = (n + 15) / 16;
    const int64_t nrs = (n + kRsTile - 1) / kRsTile;
    PlanWs L{};
    char* base = reinterpret_cast<char*>(ws);
    size_t o = 0;
    auto take = [&](size_t bytes) {
        char* p = base ? base + o : nullptr;
        o += al256(bytes);
        return p;
    };
    L.ka = reinterpret_cast<uint32_t*>(take((size_t)R * n * sizeof(uint32_t)));
    L.kb = reinterpret_cast<uint32_t*>(take((size_t)R * n * sizeof(uint32_t)));
    L.va = reinterpret_cast<int32_t*>(take((size_t)R * n * sizeof(int32_t)));
    L.vb = reinterpret_cast<int32_t*>(take((size_t)R * n * sizeof(int32_t)));
    L.nzero = (int64_t)R * kRsMaxPasses * kRsBins + kRsMaxPasses + (int64_t)R * nrs * kRsBins;
    L.ghist = reinterpret_cast<uint32_t*>(take((size_t)L.nzero * sizeof(uint32_t)));
    L.ticket = L.ghist ? L.ghist + (int64_t)R * kRsMaxPasses * kRsBins : nullptr;
    L.st0 = L.ticket ? L.ticket + kRsMaxPasses : nullptr;
    L.st1 = reinterpret_cast<uint32_t*>(take((size_t)R * nrs * kRsBins * sizeof(uint32_t)));
    L.cnt = reinterpret_cast<int32_t*>(take((size_t)R * nb * sizeof(int32_t)));
    L.scan_ws = take(scan_ws_bytes(nb));
    L.bytes = o;
    return L;
}

// All ranges of a plan (R ranges of S offsets, the last one K - (R-1) S)
// go through one launch per step: the kernels take the range from the
// grid's second dimension (the radix passes from the tile's ticket), so a
// map with more than 32 offsets costs the launches of one plan.  The item
// counts are scanned per range (ibase restarts at 0 in every range).
// lb_status: the plan call's look-back status word, cleared by the first
// kernel and set by a pass that gave up.
static int plan_enqueue(const int32_t* nbr, int64_t n, int K, int R, int S, int32_t* perm, uint32_t* bmask,
                        int64_t* ibase, int32_t* items, void* ws, uint32_t* lb_status, int spin_max, hipStream_t s) {
    const int64_t nb = (n + 15) / 16;
    const int64_t nrs = (n + kRsTile - 1) / kRsTile;
    // as many passes as for the widest range's mask alone (the popcount field fills spare bits)
    const int passes = (S + plan_key_pbits(S) + kRsBits - 1) / kRsBits;
    const PlanWs L = plan_ws_layout(ws, n, R);
    if (n == 0) {
        hipLaunchKernelGGL(k_plan_empty, dim3(1), dim3(64), 0, s, ibase, R, lb_status);
        GSC_LAUNCH_CHECK();
        return GSC_OK;
    }
    const unsigned pblocks = (unsigned)((n + kPlanThreads - 1) / kPlanThreads);
    hipLaunchKernelGGL(k_plan_masks, dim3(pblocks, (unsigned)R), dim3(kPlanThreads), 0, s, nbr, n, K, S, L.ka, L.ghist,
                       L.nzero, lb_status);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_rs_ghist, dim3((unsigned)nrs, (unsigned)R), dim3(kRsThreads), 0, s, L.ka, n, passes, L.ghist);
    GSC_LAUNCH_CHECK();
    const uint32_t* kin = L.ka;
    const int32_t* vin = nullptr;
    for (int p = 0; p < passes; ++p) {
        uint32_t* kout = (p & 1) ? L.ka : L.kb;
        int32_t* vout = (p == passes - 1) ? perm : ((p & 1) ? L.va : L.vb);
        uint32_t* st = (p & 1) ? L.st1 : L.st0;
        uint32_t* st_next = (p & 1) ? L.st0 : L.st1;
        hipLaunchKernelGGL(k_rs_pass, dim3((unsigned)(nrs * R)), dim3(kRsThreads), 0, s, kin, vin, n, nrs, R,
                           p * kRsBits, L.ghist + (int64_t)p * kRsBins, st, st_next, L.ticket + p, kout, vout,
                           spin_max, lb_status);
        GSC_LAUNCH_CHECK();
        kin = kout;
        vin = vout;
    }
    hipLaunchKernelGGL(k_blk_count, dim3(pblocks, (unsigned)R), dim3(kPlanThreads), 0, s, kin, K, S, n, nb, bmask,
                       L.cnt);
    GSC_LAUNCH_CHECK();
    for (int r = 0; r < R; ++r) {
        const int rc = scan_counts(L.cnt + (int64_t)r * nb, nb, ibase + (int64_t)r * (nb + 1), nullptr, L.scan_ws, s);
        if (rc) return rc;
    }
    hipLaunchKernelGGL(k_blk_fill, dim3(pblocks, (unsigned)R), dim3(kPlanThreads), 0, s, kin, K, S, perm, nbr, ibase,
                       n, nb, items);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

// The look-back status word sits in the last 256 bytes of the plan's ws.
static uint32_t* plan_status_word(void* ws, int64_t n_out, int K) {
    return reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + gsc_conv_plan_ws_bytes(n_out, K) - 256);
}

// Polls of one look-back entry before a pass gives up: kSpinMax, or the value
// of the environment variable GSC_PLAN_SPIN_LIMIT (a test hook: a negative
// value gives up at the first poll, so the failure path can be exercised
// while every kernel still ends normally).
static int lookback_spin_limit() {
    const char* e = getenv("GSC_PLAN_SPIN_LIMIT");
    if (!e || !*e) return kSpinMax;
    const long v = strtol(e, nullptr, 10);
    return v < -1 ? -1 : (v > kSpinMax ? kSpinMax : (int)v);
}

}  // namespace gsc

using namespace gsc;

extern "C" {

int64_t gsc_plan_blocks(int64_t n_out) { return n_out <= 0 ? 0 : (n_out + 15) / 16; }

int32_t gsc_plan_ranges(int32_t K) { return K < 1 || K > kPlanMaxKAll ? 0 : plan_ranges(K); }

size_t gsc_conv_plan_ws_bytes(int64_t n_out, int32_t K) {
    if (n_out < 0 || n_out > kRsMaxKeys || K < 1 || K > kPlanMaxKAll) return 0;
    return plan_ws_layout(nullptr, n_out, plan_ranges(K)).bytes + 256;
}

int gsc_conv_plan(const int32_t* nbr, int64_t n_out, int32_t K, int32_t* perm, uint32_t* bmask, int64_t* ibase,
                  int32_t* items, int64_t cap_items, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (K < 1 || K > kPlanMaxKAll) return fail(GSC_EINVAL, "conv_plan: K=%d outside [1,%d]", K, kPlanMaxKAll);
    if (n_out < 0 || n_out > kRsMaxKeys)
        return fail(GSC_EINVAL, "conv_plan: n_out=%lld outside [0, %lld]", (long long)n_out, (long long)kRsMaxKeys);
    if (!ibase || !ws) return fail(GSC_EINVAL, "conv_plan: null ibase/ws");
    if (n_out > 0 && (!nbr || !perm || !bmask || !items))
        return fail(GSC_EINVAL, "conv_plan: null nbr/perm/bmask/items");
    const int64_t need_items = (int64_t)K * gsc_plan_blocks(n_out);
    if (cap_items < need_items)
        return fail(GSC_ESHORT, "conv_plan: cap_items=%lld, need K*ceil(n_out/16) = %lld", (long long)cap_items,
                    (long long)need_items);
    const size_t need = gsc_conv_plan_ws_bytes(n_out, K);
    if (ws_bytes < need) return fail(GSC_ESHORT, "conv_plan: ws needs %zu bytes, got %zu", need, ws_bytes);
    // every range of offsets in the same launches
    return plan_enqueue(nbr, n_out, K, plan_ranges(K), plan_range_size(K), perm, bmask, ibase, items, ws,
                        plan_status_word(ws, n_out, K), lookback_spin_limit(), reinterpret_cast<hipStream_t>(stream));
}

int gsc_conv_plan_status(const void* ws, size_t ws_bytes, int64_t n_out, int32_t K, void* stream) {
    clear_error();
    const size_t need = gsc_conv_plan_ws_bytes(n_out, K);
    if (!ws || need == 0) return fail(GSC_EINVAL, "conv_plan_status: null ws or bad n_out/K");
    if (ws_bytes < need) return fail(GSC_ESHORT, "conv_plan_status: ws needs %zu bytes, got %zu", need, ws_bytes);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    uint32_t word = 0;
    if (hipMemcpyAsync(&word, plan_status_word(const_cast<void*>(ws), n_out, K), sizeof(word), hipMemcpyDeviceToHost,
                       s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return fail(GSC_EHIP, "conv_plan_status: %s", hipGetErrorString(hipGetLastError()));
    if (word != 0)
        return fail(GSC_ETIMEOUT, "conv_plan: a radix pass gave up waiting for an earlier tile's count; the plan "
                                  "is not valid");
    return GSC_OK;
}

}  // extern "C"
