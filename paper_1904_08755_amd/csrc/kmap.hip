// Kernel map (a3): for every offset o_k and output row j, the input row of
// u_j + ts (.) o_k, if present.  Two passes over (output row, offset):
//   count: one lane per output row probes the table for every offset; the
//          input row found (or -1) goes to a dense offset-major neighbour
//          table nbr[k][j], and per offset a wave64 ballot of hits gives the
//          pair count of every 64-row group;
//   scan:  exclusive scan of the (offset-major, group-minor) counts gives the
//          start of each group's pairs (the group index gidx) and the total;
//   fill:  each hit is placed at its group start plus its rank among the
//          wave's hits (popcount of the lower-lane mask), its input row read
//          from the neighbour table.
// Pairs of one offset therefore come out sorted by output row, and the
// result does not depend on scheduling.
//
// A map of a coordinate set onto itself (the stride-1 layers of Sec. 3.1:
// the output coordinates are the rows the table was built from, in the same
// order) over a region closed under negation, listed so that
// o_{K-1-k} = -o_k with the origin in the middle, is symmetric: (i, j) is a
// pair at offset k exactly when (j, i) is one at offset K-1-k, and the middle
// offset pairs every row with itself.  Whenever the region is listed so and
// the output has as many rows as the table, the count pass probes only the
// offsets up to the middle one: each hit also writes its mirrored entry of
// the neighbour table (set to -1 beforehand), and a second pass counts the
// mirrored offsets' pairs per group from the table.  The middle offset
// checks the premise: output row j must find table row j.  If one row does
// not (other coordinates, another order, rows rewritten since the build),
// the second pass probes the mirrored offsets itself instead, overwriting
// their entries, so the result equals the full probe in every case.
#include <algorithm>
#include <climits>
#include <mutex>
#include <vector>

#include "gsc_internal.h"

namespace gsc {

constexpr int kThreads = 256;
constexpr int kOffArgMax = 768;   // K * D offsets passed by value in the kernel arguments

// Offsets of the region, either by value in the kernel arguments (no host
// to device copy, so the map can be enqueued asynchronously) or in device
// memory (large regions, synchronous mode only).
struct OffsArg {
    int32_t v[kOffArgMax];
    __device__ __forceinline__ const int32_t* at(int64_t i) const { return v + i; }
};
struct OffsPtr {
    const int32_t* p;
    __device__ __forceinline__ const int32_t* at(int64_t i) const { return p + i; }
};

__device__ __forceinline__ bool header_ok(const TableHeader* h, int ncol) {
    return h->magic == kTableMagic && h->ncol == ncol && h->status == 0;
}

// Probes issued together per lane in the count pass: 4 (186 VGPRs at 16 halve
// the resident waves; 8 and 16 measured slower on a 300k-row map), or 16
// when every row's wave is resident at once even at that size (a 120k-row
// map: 53 -> 45 us).  Wide keys take one at a time, so that their path needs
// no more registers than the others.
constexpr int kBatch = 4;
constexpr int kBatchSmall = 16;
template <typename KeyT, int NB>
constexpr int batch_of() { return sizeof(KeyT) > 8 ? 1 : NB; }

// Key arithmetic in KeyT (uint32_t when the table's keys fit in 32 bits, the
// usual case, uint64_t up to 62 bits, else the 128-bit wide key).  The packed
// key is linear in the coordinate: key(u + o) = base(u) + delta(o), exact (mod
// 2^bits) whenever every column of u + o lies in the table's box, so a probe
// is a range check per column and one add.
template <typename KeyT>
struct KeyOps;

template <>
struct KeyOps<uint32_t> {
    static __device__ __forceinline__ uint32_t hash(uint32_t k) { return fmix32(k); }
    static __device__ __forceinline__ bool eq(const Slot& e, uint32_t k) { return e.key == (unsigned long long)k; }
};
template <>
struct KeyOps<unsigned long long> {
    static __device__ __forceinline__ uint32_t hash(unsigned long long k) { return hash_key(k); }
    static __device__ __forceinline__ bool eq(const Slot& e, unsigned long long k) { return e.key == k; }
};
template <>
struct KeyOps<u128> {
    static __device__ __forceinline__ uint32_t hash(u128 k) { return hash_key_wide(k); }
    static __device__ __forceinline__ bool eq(const Slot& e, u128 k) { return e.key == wide_lo(k) && e.hi == wide_hi(k); }
};

// Count pass.  Each lane owns one output row.  Offsets are probed NB at a
// time; every load is issued unconditionally (a lane whose query is out of
// the box reads slot 0 and ignores it) so the NB loads are in flight
// together, and collision chains are followed in rounds.  A probe reads the
// whole 16-byte slot, so a hit also yields the input row, which goes to
// nbr[k * n_out + j] (-1 for a miss); hits are counted per 64-row group with
// a wave ballot.
template <typename KeyT, int NBT, typename Offs>
__device__ __forceinline__ void count_rows(const TableHeader* h, const Slot* __restrict__ slots,
                                           const int32_t* __restrict__ out_coords, int64_t n_out, int ncol,
                                           const Offs& offs, int K, int k_begin, int k_end, int mirror_end,
                                           int mid, int64_t G, int32_t* __restrict__ cnt,
                                           int32_t* __restrict__ nbr, bool ok, int64_t j,
                                           int32_t* __restrict__ not_self) {
    const bool valid = ok && j < n_out;
    const int D = ncol - 1;
    const unsigned long long mask = ok ? (unsigned long long)h->capacity - 1 : 0;
    const int nblk = h->nblk;
    KeyT clear = ~(KeyT)0;
    int bsh[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        bsh[i] = h->blk_shift[i];
        if (i < nblk) clear &= ~((KeyT)1 << bsh[i]);
    }
    int32_t rel[kMaxCols], span[kMaxCols], shc[kMaxCols];
    KeyT base = 0;
    bool in_b = valid;
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c) {
        if (c < ncol) {
            const int32_t lo = h->lo[c];
            shc[c] = h->shift[c];
            span[c] = h->hi[c] - lo;
            rel[c] = (valid ? out_coords[j * ncol + c] : lo) - lo;
            base += (KeyT)(uint32_t)rel[c] << shc[c];    // (KeyT)(int) sign-extends for 64-bit keys below
        }
    }
    if (sizeof(KeyT) >= 8) {   // redo with sign extension: rel may be negative when u is outside the box
        base = 0;
#pragma unroll
        for (int c = 0; c < kMaxCols; ++c)
            if (c < ncol) base += (KeyT)(long long)rel[c] << shc[c];
    }
    in_b = in_b && (uint32_t)rel[0] <= (uint32_t)span[0];
    const int64_t g = j >> 6;
    const bool writer = __lane_id() == 0 && g < G;
    constexpr int NB = batch_of<KeyT, NBT>();
    for (int k0 = k_begin; k0 < k_end; k0 += NB) {
        KeyT key[NB];
        unsigned long long pos[NB];
        bool pend[NB], hit[NB];
        int32_t row[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int k = min(k0 + b, k_end - 1);
            const int32_t* o = offs.at((int64_t)k * D);
            bool in = in_b && k0 + b < k_end;
            KeyT delta = 0;
#pragma unroll
            for (int c = 1; c < kMaxCols; ++c) {
                if (c < ncol) {
                    in = in && (uint32_t)(rel[c] + o[c - 1]) <= (uint32_t)span[c];
                    delta += (KeyT)(long long)o[c - 1] << shc[c];
                }
            }
            const KeyT kk = base + delta;
            KeyT local = 0;
#pragma unroll
            for (int i = 0; i < 3; ++i)
                if (i < nblk) local |= ((kk >> bsh[i]) & 1) << i;
            const unsigned long long hs =
                (((unsigned long long)KeyOps<KeyT>::hash(kk & clear) << nblk) | (unsigned long long)local) & mask;
            key[b] = kk;
            pos[b] = in ? hs : 0;
            pend[b] = in;
            hit[b] = false;
            row[b] = -1;
        }
        for (unsigned long long round = 0; round <= mask; ++round) {
            Slot e[NB];
            if (round == 0) {
#pragma unroll
                for (int b = 0; b < NB; ++b) e[b] = slots[pos[b]];   // unconditional: all in flight
            } else {   // collision chains: few probes still pending
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    e[b].key = kEmptyKey;
                    e[b].val = -1;
                    e[b].hi = kHiUnset;
                    if (pend[b]) e[b] = slots[pos[b]];
                }
            }
            bool any = false;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const bool h1 = pend[b] && KeyOps<KeyT>::eq(e[b], key[b]);
                const bool stop = h1 || e[b].key == kEmptyKey;
                hit[b] = hit[b] || h1;
                row[b] = h1 ? e[b].val : row[b];
                pend[b] = pend[b] && !stop;
                pos[b] = pend[b] ? ((pos[b] + 1) & mask) : pos[b];
                any = any || pend[b];
            }
            if (!__any(any)) break;
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int k = k0 + b;
            if (k < k_end) {
                const unsigned long long m = __ballot(hit[b]);
                if (writer) cnt[(int64_t)k * G + g] = __popcll(m);
                if (j < n_out) nbr[(int64_t)k * n_out + j] = hit[b] ? row[b] : -1;
                // the mirrored pair (j, row) at offset K-1-k
                if (k < mirror_end && hit[b] && row[b] >= 0 && row[b] < n_out)
                    nbr[(int64_t)(K - 1 - k) * n_out + row[b]] = (int32_t)j;
                // the middle offset of a self map pairs every row with itself
                if (k == mid) {
                    const unsigned long long bad = __ballot(j < n_out && !(hit[b] && row[b] == j));
                    if (bad && __lane_id() == 0) atomicOr(not_self, 1);
                }
            }
        }
    }
}

// Whether a map onto out_coords over a symmetric listing (sym) may be a map
// of the table's coordinate set onto itself: the table is valid and has as
// many rows as the output.  The count pass checks the rest (row j finds row j).
__device__ __forceinline__ bool self_candidate(const TableHeader* h, int ncol, int64_t n_out, int sym) {
    return sym && header_ok(h, ncol) && h->n == n_out;
}

template <typename Offs, int NB>
__global__ void __launch_bounds__(kThreads) k_kmap_count(const void* table, const int32_t* __restrict__ out_coords,
                                                         int64_t n_out, int ncol, Offs offs, int K, int sym, int64_t G,
                                                         int32_t* __restrict__ cnt, int32_t* __restrict__ nbr,
                                                         int64_t* err, int32_t* not_self) {
    const TableHeader* h = reinterpret_cast<const TableHeader*>(table);
    const Slot* __restrict__ slots = table_slots(table);
    const bool ok = header_ok(h, ncol);
    if (blockIdx.x == 0 && threadIdx.x == 0) *err = ok ? 0 : 1;
    const bool self = self_candidate(h, ncol, n_out, sym);
    const int k_end = self ? (K + 1) / 2 : K;        // up to and including the middle offset
    const int mirror_end = self ? (K - 1) / 2 : 0;   // offsets whose hits are mirrored
    const int mid = self ? (K - 1) / 2 : -1;
    const int64_t j = xcd_unit(blockIdx.x, gridDim.x) * kThreads + threadIdx.x;
    if (h->total_bits <= 32)   // uniform: all lanes take the same path
        count_rows<uint32_t, NB>(h, slots, out_coords, n_out, ncol, offs, K, 0, k_end, mirror_end, mid, G, cnt, nbr, ok,
                             j, not_self);
    else if (h->total_bits <= kNarrowKeyBits)
        count_rows<unsigned long long, NB>(h, slots, out_coords, n_out, ncol, offs, K, 0, k_end, mirror_end, mid, G, cnt,
                                       nbr, ok, j, not_self);
    else
        count_rows<u128, NB>(h, slots, out_coords, n_out, ncol, offs, K, 0, k_end, mirror_end, mid, G, cnt, nbr, ok, j,
                         not_self);
}

// Symmetric listing: clear the self-map check, and if the map may be a self
// map, start the mirrored offsets' rows of the neighbour table empty.
__global__ void __launch_bounds__(kThreads) k_kmap_self_init(const void* table, int64_t n_out, int ncol, int K,
                                                             int sym, int32_t* __restrict__ nbr,
                                                             int32_t* __restrict__ not_self) {
    const TableHeader* h = reinterpret_cast<const TableHeader*>(table);
    if (blockIdx.x == 0 && threadIdx.x == 0) *not_self = 0;
    if (!self_candidate(h, ncol, n_out, sym)) return;
    const int64_t first = (int64_t)((K + 1) / 2) * n_out, n = (int64_t)(K / 2) * n_out;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        nbr[first + i] = -1;
}

// Symmetric listing, second pass over the offsets after the middle one: for a
// self map (the count pass found every row at its own index) their pair
// counts per 64-row group come from the mirrored entries of the neighbour
// table; otherwise every row probes them itself.
template <typename Offs, int NB>
__global__ void __launch_bounds__(kThreads) k_kmap_mirror_count(const void* table,
                                                                const int32_t* __restrict__ out_coords, int64_t n_out,
                                                                int ncol, Offs offs, int K, int sym, int64_t G,
                                                                int32_t* __restrict__ nbr, int32_t* __restrict__ cnt,
                                                                int32_t* not_self) {
    const TableHeader* h = reinterpret_cast<const TableHeader*>(table);
    if (!self_candidate(h, ncol, n_out, sym)) return;
    const int64_t j = xcd_unit(blockIdx.x, gridDim.x) * kThreads + threadIdx.x;
    if (*not_self) {
        const Slot* __restrict__ slots = table_slots(table);
        if (h->total_bits <= 32)
            count_rows<uint32_t, NB>(h, slots, out_coords, n_out, ncol, offs, K, (K + 1) / 2, K, 0, -1, G, cnt, nbr, true,
                                 j, not_self);
        else if (h->total_bits <= kNarrowKeyBits)
            count_rows<unsigned long long, NB>(h, slots, out_coords, n_out, ncol, offs, K, (K + 1) / 2, K, 0, -1, G, cnt,
                                           nbr, true, j, not_self);
        else
            count_rows<u128, NB>(h, slots, out_coords, n_out, ncol, offs, K, (K + 1) / 2, K, 0, -1, G, cnt, nbr, true, j,
                             not_self);
        return;
    }
    const int64_t g = j >> 6;
    const bool writer = __lane_id() == 0 && g < G;
    constexpr int B = 8;
    for (int k0 = (K + 1) / 2; k0 < K; k0 += B) {
        int32_t r[B];
#pragma unroll
        for (int b = 0; b < B; ++b) r[b] = j < n_out && k0 + b < K ? nbr[(int64_t)(k0 + b) * n_out + j] : -1;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const unsigned long long m = __ballot(r[b] >= 0);
            if (writer && k0 + b < K) cnt[(int64_t)(k0 + b) * G + g] = __popcll(m);
        }
    }
}

// Fill pass: lane j reads its row of the neighbour table offset by offset;
// each hit goes to its group start plus its rank among the wave's hits.
__global__ void __launch_bounds__(kThreads) k_kmap_fill(int64_t n_out, int K, int64_t G,
                                                        const int32_t* __restrict__ nbr,
                                                        const int64_t* __restrict__ gidx, int32_t* __restrict__ in_idx,
                                                        int32_t* __restrict__ out_idx, int64_t cap) {
    const int64_t j = xcd_unit(blockIdx.x, gridDim.x) * kThreads + threadIdx.x;
    const bool valid = j < n_out;
    const int64_t g = j >> 6;
    const unsigned long long below = lanemask_lt();
    constexpr int B = 8;   // offsets whose table entries (and group starts) are loaded together
    for (int k0 = 0; k0 < K; k0 += B) {
        int32_t r[B];
        int64_t gs[B];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            r[b] = valid && k0 + b < K ? nbr[(int64_t)(k0 + b) * n_out + j] : -1;
            gs[b] = g < G && k0 + b < K ? gidx[(int64_t)(k0 + b) * G + g] : 0;
        }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const bool hit = r[b] >= 0;
            const unsigned long long m = __ballot(hit);
            if (hit) {
                const int64_t pos = gs[b] + __popcll(m & below);
                if (pos < cap) {
                    in_idx[pos] = r[b];
                    out_idx[pos] = (int32_t)j;
                }
            }
        }
    }
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------
// Role reversal of a map without the coordinate table (Sec. 4.2: the pairs of
// the transposed convolution are those of the forward one with input and
// output exchanged).  A map lists each input row at most once per offset (its
// output coordinate is the input's minus the scaled offset), so the reversed
// map's dense form is a scatter of the pairs; the count, scan and fill passes
// of the kernel map then list the pairs by the former input row.
// ---------------------------------------------------------------------------
__global__ void k_fill_neg1(int32_t* __restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = -1;
}

// nbr[k * n_rev + in_idx[p]] = out_idx[p] for the pairs p < seg[K] (offset k
// of pair p found by a search of seg); a row outside [0, n_rev) is skipped
// (the caller's map is checked: err[0] is set).
__global__ void __launch_bounds__(kThreads) k_map_scatter(const int32_t* __restrict__ in_idx,
                                                          const int32_t* __restrict__ out_idx,
                                                          const int64_t* __restrict__ seg, int K, int64_t cap,
                                                          int64_t n_rev, int32_t* __restrict__ nbr,
                                                          int32_t* __restrict__ err) {
    const int64_t total = seg[K] < cap ? seg[K] : cap;
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < total; p += (int64_t)gridDim.x * kThreads) {
        int lo = 0, hi = K;   // the k with seg[k] <= p < seg[k + 1]
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (seg[mid] <= p) lo = mid;
            else hi = mid;
        }
        const int32_t r = in_idx[p];
        if (r >= 0 && r < n_rev) nbr[(int64_t)lo * n_rev + r] = out_idx[p];
        else atomicOr(err, 1);
    }
}

// cnt[k * G + g] = entries >= 0 of nbr[k * n][64 g .. 64 g + 63].
__global__ void __launch_bounds__(kThreads) k_nbr_count(const int32_t* __restrict__ nbr, int64_t n, int K, int64_t G,
                                                        int32_t* __restrict__ cnt) {
    const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t g = j >> 6;
    const bool valid = j < n;
    for (int k = 0; k < K; ++k) {
        const unsigned long long m = __ballot(valid && nbr[(int64_t)k * n + j] >= 0);
        if ((threadIdx.x & 63) == 0 && g < G) cnt[(int64_t)k * G + g] = (int32_t)__popcll(m);
    }
}

template <typename Offs>
static int kmap_enqueue(const void* in_table, const int32_t* out_coords, int64_t n_out, int ncol, Offs offs, int K,
                        int sym, int64_t G, int32_t* in_idx, int32_t* out_idx, int64_t cap_pairs, int64_t* seg,
                        int64_t* gidx, int64_t* n_pairs, int64_t* res, int32_t* cnt, int32_t* nbr, void* scan_ws,
                        hipStream_t s) {
    int32_t* not_self = reinterpret_cast<int32_t*>(res + 2);
    const unsigned nblk = (unsigned)((n_out + kThreads - 1) / kThreads);
    if (nblk > 0) {
        if (sym && K > 1) {   // whether the map is a self map is read from the table on the device
            const int64_t n_init = (int64_t)(K / 2) * n_out;
            const int64_t gi = (n_init + kThreads - 1) / kThreads;
            hipLaunchKernelGGL(k_kmap_self_init, dim3((unsigned)(gi < 4096 ? (gi > 0 ? gi : 1) : 4096)), dim3(kThreads), 0,
                               s, in_table, n_out, ncol, K, sym, nbr, not_self);
            GSC_LAUNCH_CHECK();
        }
        // the wide batch while every row's wave fits at once (two waves per SIMD)
        const bool small = n_out <= (int64_t)device_cus() * 4 * 2 * 64;
        if (small)
            hipLaunchKernelGGL((k_kmap_count<Offs, kBatchSmall>), dim3(nblk), dim3(kThreads), 0, s, in_table,
                               out_coords, n_out, ncol, offs, K, sym, G, cnt, nbr, res + 1, not_self);
        else
            hipLaunchKernelGGL((k_kmap_count<Offs, kBatch>), dim3(nblk), dim3(kThreads), 0, s, in_table, out_coords,
                               n_out, ncol, offs, K, sym, G, cnt, nbr, res + 1, not_self);
        GSC_LAUNCH_CHECK();
        if (sym && K > 1) {
            if (small)
                hipLaunchKernelGGL((k_kmap_mirror_count<Offs, kBatchSmall>), dim3(nblk), dim3(kThreads), 0, s,
                                   in_table, out_coords, n_out, ncol, offs, K, sym, G, nbr, cnt, not_self);
            else
                hipLaunchKernelGGL((k_kmap_mirror_count<Offs, kBatch>), dim3(nblk), dim3(kThreads), 0, s, in_table,
                                   out_coords, n_out, ncol, offs, K, sym, G, nbr, cnt, not_self);
            GSC_LAUNCH_CHECK();
        }
    }
    // the scan also writes seg[k] = gidx[k * G] (a launch of its own without groups)
    int rc = G > 0 ? scan_counts(cnt, K * G, gidx, res, scan_ws, s, seg, G)
                   : scan_counts(cnt, 0, gidx, res, scan_ws, s);
    if (rc) return rc;
    if (G == 0) {
        rc = seg_from_gidx(gidx, K, G, seg, s);
        if (rc) return rc;
    }
    int64_t bound = cap_pairs;
    if (n_pairs) {
        int64_t hres[2];
        GSC_HIP(hipMemcpyAsync(hres, res, sizeof(hres), hipMemcpyDeviceToHost, s));
        GSC_HIP(hipStreamSynchronize(s));
        // the count kernel (launched when n_out > 0) writes the header check
        if (nblk > 0 && hres[1])
            return fail(GSC_EINVAL, "kernel_map: in_table is not a valid table of %d-column rows", ncol);
        *n_pairs = hres[0];
        if (hres[0] > cap_pairs)
            return fail(GSC_ESHORT, "kernel_map: %lld pairs exceed cap_pairs=%lld", (long long)hres[0],
                        (long long)cap_pairs);
        bound = hres[0];
    }
    if (nblk > 0 && bound > 0) {
        hipLaunchKernelGGL(k_kmap_fill, dim3(nblk), dim3(kThreads), 0, s, n_out, K, G, nbr, gidx, in_idx, out_idx,
                           cap_pairs);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

// Host-side checks and the offsets scaled by the tensor stride (by value in
// `arg` when K * D <= kOffArgMax, always in `offs`); sym = the listing is
// symmetric (K odd, o_{K-1-k} = -o_k, the origin in the middle).
static int kmap_prepare(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D,
                        const int32_t* offsets, int32_t K, const int32_t* tensor_stride, int32_t* in_idx,
                        int32_t* out_idx, int64_t cap_pairs, int64_t* seg, int64_t* gidx, int64_t* n_pairs,
                        OffsArg& arg, std::vector<int32_t>& offs, int& sym) {
    if (D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "kernel_map: D=%d outside [1,%d]", D, kMaxCols - 1);
    if (K < 1) return fail(GSC_EINVAL, "kernel_map: K=%d must be >= 1", K);
    if (n_out < 0 || n_out > INT32_MAX) return fail(GSC_EINVAL, "kernel_map: n_out=%lld invalid", (long long)n_out);
    if (!in_table || !offsets || !seg || !gidx) return fail(GSC_EINVAL, "kernel_map: null in_table/offsets/seg/gidx");
    if (n_out > 0 && !out_coords) return fail(GSC_EINVAL, "kernel_map: out_coords is null");
    if (cap_pairs < 0) return fail(GSC_EINVAL, "kernel_map: cap_pairs < 0");
    if (cap_pairs > 0 && (!in_idx || !out_idx)) return fail(GSC_EINVAL, "kernel_map: null in_idx/out_idx");
    const bool by_value = (int64_t)K * D <= kOffArgMax;
    if (!n_pairs) {   // asynchronous mode
        if (cap_pairs < (int64_t)K * n_out)
            return fail(GSC_ESHORT, "kernel_map: asynchronous mode needs cap_pairs >= K*n_out = %lld",
                        (long long)K * n_out);
        if (!by_value)
            return fail(GSC_EINVAL, "kernel_map: asynchronous mode needs K*D <= %d (got %d)", kOffArgMax, K * D);
    }
    offs.assign((size_t)K * D, 0);
    sym = K % 2 == 1 ? 1 : 0;
    for (int k = 0; k < K && sym; ++k)
        for (int d = 0; d < D; ++d) {
            const int32_t a = offsets[(size_t)k * D + d], b = offsets[(size_t)(K - 1 - k) * D + d];
            if ((int64_t)a != -(int64_t)b) sym = 0;
        }
    for (int k = 0; k < K; ++k)
        for (int d = 0; d < D; ++d) {
            const int64_t ts = tensor_stride ? tensor_stride[d] : 1;
            if (ts < 1) return fail(GSC_EINVAL, "kernel_map: tensor_stride[%d]=%lld must be >= 1", d, (long long)ts);
            const int64_t v = ts * (int64_t)offsets[(size_t)k * D + d];
            if (v < -(1ll << 30) || v > (1ll << 30))
                return fail(GSC_ERANGE, "kernel_map: scaled offset %lld out of range", (long long)v);
            offs[(size_t)k * D + d] = (int32_t)v;
            if (by_value) arg.v[(size_t)k * D + d] = (int32_t)v;
        }
    return GSC_OK;
}

// Scratch of the allocation-free kernel map: a device array of fixed size in
// the library's code object.  Each GPU holds its own copy at its own address,
// taken once per device with hipGetSymbolAddress (the array's name is not a
// device address in host code).  Calls on one GPU share it, so calls that
// overlap on one GPU race.
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

static int noalloc_scratch(char** out) {
    int dev = -1;
    GSC_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(GSC_EINVAL, "kernel_map_noalloc: device %d unsupported", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        GSC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(GSC_EHIP, "kernel_map_noalloc: no address for the scratch array on device %d", dev);
        g_scratch_ptr[dev] = p;
    }
    *out = reinterpret_cast<char*>(g_scratch_ptr[dev]);
    return GSC_OK;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

int64_t gsc_kmap_groups(int64_t n_out) { return n_out <= 0 ? 0 : (n_out + 63) / 64; }

size_t gsc_kmap_ws_bytes(int64_t n_out, int32_t K, int32_t D) {
    if (n_out < 0 || K < 1 || D < 1) return 0;
    const int64_t G = gsc_kmap_groups(n_out);
    size_t b = align256((size_t)K * D * sizeof(int32_t));      // offsets (scaled)
    b += align256(3 * sizeof(int64_t));                         // total, error flag, self-map check
    b += align256((size_t)K * G * sizeof(int32_t));             // counts
    b += align256((size_t)K * n_out * sizeof(int32_t));         // neighbour table
    b += scan_ws_bytes(K * G);
    return b + 256;
}

int gsc_kernel_map(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D, const int32_t* offsets,
                   int32_t K, const int32_t* tensor_stride, int32_t* in_idx, int32_t* out_idx, int64_t cap_pairs,
                   int64_t* seg, int64_t* gidx, int32_t* nbr_out, int64_t* n_pairs, void* ws, size_t ws_bytes,
                   void* stream) {
    clear_error();
    if (!ws) return fail(GSC_EINVAL, "kernel_map: null ws");
    if (ws_bytes < gsc_kmap_ws_bytes(n_out, K, D))
        return fail(GSC_ESHORT, "kernel_map: ws needs %zu bytes, got %zu", gsc_kmap_ws_bytes(n_out, K, D), ws_bytes);
    OffsArg arg;
    std::vector<int32_t> offs;
    int sym = 0;
    int rc = kmap_prepare(in_table, out_coords, n_out, D, offsets, K, tensor_stride, in_idx, out_idx, cap_pairs, seg,
                          gidx, n_pairs, arg, offs, sym);
    if (rc) return rc;
    const bool by_value = (int64_t)K * D <= kOffArgMax;

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int ncol = D + 1;
    const int64_t G = gsc_kmap_groups(n_out);
    char* w = reinterpret_cast<char*>(ws);
    int32_t* d_offs = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * D * sizeof(int32_t));
    int64_t* res = reinterpret_cast<int64_t*>(w);   // res[0] = total, res[1] = header error, res[2] = self check
    w += align256(3 * sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * G * sizeof(int32_t));
    int32_t* nbr = nbr_out ? nbr_out : reinterpret_cast<int32_t*>(w);   // the caller's dense map, if asked for
    w += align256((size_t)K * n_out * sizeof(int32_t));
    void* scan_ws = w;
    if (by_value)
        return kmap_enqueue(in_table, out_coords, n_out, ncol, arg, K, sym, G, in_idx, out_idx, cap_pairs, seg, gidx,
                            n_pairs, res, cnt, nbr, scan_ws, s);
    // synchronous mode: the copy below completes before this call returns
    GSC_HIP(hipMemcpyAsync(d_offs, offs.data(), offs.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
    return kmap_enqueue(in_table, out_coords, n_out, ncol, OffsPtr{d_offs}, K, sym, G, in_idx, out_idx, cap_pairs,
                        seg, gidx, n_pairs, res, cnt, nbr, scan_ws, s);
}

size_t gsc_kernel_map_noalloc_bytes(int64_t n_out, int32_t K) {
    if (n_out < 0 || K < 1) return 0;
    const int64_t G = gsc_kmap_groups(n_out);
    return align256(3 * sizeof(int64_t)) + align256((size_t)K * G * sizeof(int32_t)) + scan_ws_bytes(K * G);
}

int gsc_kernel_map_noalloc(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D,
                           const int32_t* offsets, int32_t K, const int32_t* tensor_stride, int32_t* in_idx,
                           int32_t* out_idx, int64_t cap_pairs, int64_t* seg, int64_t* gidx, int32_t* nbr,
                           void* stream) {
    clear_error();
    if (!nbr) return fail(GSC_EINVAL, "kernel_map_noalloc: the dense form nbr is required");
    const size_t need = gsc_kernel_map_noalloc_bytes(n_out, K);
    if (n_out >= 0 && K >= 1 && need > kNoAllocScratchBytes)
        return fail(GSC_ERANGE, "kernel_map_noalloc: needs %zu bytes of scratch, the library holds %zu per GPU "
                    "(n_out=%lld, K=%d); use gsc_kernel_map with a workspace", need, kNoAllocScratchBytes,
                    (long long)n_out, K);
    OffsArg arg;
    std::vector<int32_t> offs;
    int sym = 0;
    int rc = kmap_prepare(in_table, out_coords, n_out, D, offsets, K, tensor_stride, in_idx, out_idx, cap_pairs, seg,
                          gidx, nullptr, arg, offs, sym);
    if (rc) return rc;
    char* w = nullptr;
    rc = noalloc_scratch(&w);
    if (rc) return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t G = gsc_kmap_groups(n_out);
    int64_t* res = reinterpret_cast<int64_t*>(w);
    w += align256(3 * sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * G * sizeof(int32_t));
    return kmap_enqueue(in_table, out_coords, n_out, D + 1, arg, K, sym, G, in_idx, out_idx, cap_pairs, seg, gidx,
                        nullptr, res, cnt, nbr, w, s);
}

size_t gsc_kernel_map_transpose_ws_bytes(int64_t n_rev, int32_t K) {
    if (n_rev < 0 || K < 1) return 0;
    const int64_t G = gsc_kmap_groups(n_rev);
    return align256(sizeof(int64_t)) + align256((size_t)K * G * sizeof(int32_t)) + scan_ws_bytes(K * G) + 256;
}

int gsc_kernel_map_transpose(const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg, int32_t K,
                             int64_t cap_pairs, int64_t n_rev, int32_t* t_in_idx, int32_t* t_out_idx, int64_t* t_seg,
                             int64_t* t_gidx, int32_t* t_nbr, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (K < 1 || cap_pairs < 0 || n_rev < 0 || n_rev > INT32_MAX)
        return fail(GSC_EINVAL, "kernel_map_transpose: bad K=%d, cap_pairs=%lld or n_rev=%lld", K,
                    (long long)cap_pairs, (long long)n_rev);
    if (!seg || !t_seg || !t_gidx || !t_nbr || !ws)
        return fail(GSC_EINVAL, "kernel_map_transpose: null seg/t_seg/t_gidx/t_nbr/ws");
    if (cap_pairs > 0 && (!in_idx || !out_idx || !t_in_idx || !t_out_idx))
        return fail(GSC_EINVAL, "kernel_map_transpose: null pair arrays");
    const size_t need = gsc_kernel_map_transpose_ws_bytes(n_rev, K);
    if (ws_bytes < need)
        return fail(GSC_ESHORT, "kernel_map_transpose: ws needs %zu bytes, got %zu", need, ws_bytes);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t G = gsc_kmap_groups(n_rev);
    char* w = reinterpret_cast<char*>(ws);
    int32_t* err = reinterpret_cast<int32_t*>(w);
    w += align256(sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * G * sizeof(int32_t));
    const int64_t n_dense = (int64_t)K * n_rev;
    hipLaunchKernelGGL(k_fill_neg1, dim3((unsigned)std::min<int64_t>((n_dense + kThreads - 1) / kThreads + 1, 4096)),
                       dim3(kThreads), 0, s, t_nbr, n_dense);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_zero_i64, dim3(1), dim3(64), 0, s, reinterpret_cast<int64_t*>(err), (int64_t)1);
    GSC_LAUNCH_CHECK();
    if (cap_pairs > 0) {
        hipLaunchKernelGGL(k_map_scatter, dim3((unsigned)std::min<int64_t>((cap_pairs + kThreads - 1) / kThreads, 8192)),
                           dim3(kThreads), 0, s, in_idx, out_idx, seg, K, cap_pairs, n_rev, t_nbr, err);
        GSC_LAUNCH_CHECK();
    }
    const unsigned nblk = (unsigned)((n_rev + kThreads - 1) / kThreads);
    if (nblk > 0) {
        hipLaunchKernelGGL(k_nbr_count, dim3(nblk), dim3(kThreads), 0, s, t_nbr, n_rev, K, G, cnt);
        GSC_LAUNCH_CHECK();
    }
    int rc = G > 0 ? scan_counts(cnt, K * G, t_gidx, nullptr, w, s, t_seg, G)
                   : scan_counts(cnt, 0, t_gidx, nullptr, w, s);
    if (rc) return rc;
    if (G == 0) {
        rc = seg_from_gidx(t_gidx, K, G, t_seg, s);
        if (rc) return rc;
    }
    if (nblk > 0 && cap_pairs > 0) {
        hipLaunchKernelGGL(k_kmap_fill, dim3(nblk), dim3(kThreads), 0, s, n_rev, K, G, t_nbr, t_gidx, t_in_idx,
                           t_out_idx, cap_pairs);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

int gsc_kernel_map_transpose_status(const void* ws, void* stream) {
    clear_error();
    if (!ws) return fail(GSC_EINVAL, "kernel_map_transpose_status: null ws");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    int32_t e = 0;
    GSC_HIP(hipMemcpyAsync(&e, ws, sizeof(e), hipMemcpyDeviceToHost, s));
    GSC_HIP(hipStreamSynchronize(s));
    return e ? fail(GSC_EINVAL, "kernel_map_transpose: a pair's input row lies outside [0, n_rev)") : GSC_OK;
}

}  // extern "C"
