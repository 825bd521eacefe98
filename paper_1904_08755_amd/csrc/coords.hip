// Coordinate hash table (a1) and output coordinates of a strided
// convolution (a2).
//
// The table is open addressing with linear probing over 16-byte slots in
// HBM.  A coordinate row (b, x_1..x_D) is packed into a key relative to the
// bounding box of the rows (computed on the device, so the build needs no
// host round trip before the insert), batch column in the high bits, so the
// numeric order of keys is the lexicographic order of rows.
#include <climits>

#include <cstddef>
#include <cstring>

#include "gsc_internal.h"

namespace gsc {

constexpr int kThreads = 256;

struct StrideArg {
    int32_t s[kMaxCols];   // s[0] = 1 (batch), s[c] = stride of spatial column c
    int32_t on;            // 0: identity transform
};

__device__ __forceinline__ void load_row(const int32_t* coords, int64_t r, int ncol, const StrideArg& st,
                                         int64_t* v) {
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c) {
        int64_t x = c < ncol ? coords[r * ncol + c] : 0;
        if (st.on && c > 0 && c < ncol) x = floor_mul(x, st.s[c]);
        v[c] = x;
    }
}

__global__ void __launch_bounds__(kThreads) k_table_init(TableHeader* h, Slot* slots, int64_t cap, int ncol,
                                                         int64_t n, int32_t init_val) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cap; i += stride) {
        Slot e;
        e.key = kEmptyKey;
        e.val = init_val;
        e.hi = kHiUnset;
        slots[i] = e;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        h->magic = kTableMagic;
        h->ncol = ncol;
        h->capacity = cap;
        h->n = n;
        h->status = 0;
        h->total_bits = 0;
        for (int c = 0; c < kMaxCols; ++c) {
            h->lo[c] = INT_MAX;
            h->hi[c] = INT_MIN;
            h->shift[c] = 0;
            h->bits[c] = 0;
        }
        h->nblk = 0;
        for (int i = 0; i < 3; ++i) h->blk_shift[i] = 0;
        for (int c = 0; c < kMaxCols; ++c) h->vary[c] = 0;
    }
}

// Bounding box of the (optionally strided) rows: per-thread min/max, wave
// shuffles, then LDS across the block's waves, so the header sees one atomic
// per column per block.
__global__ void __launch_bounds__(kThreads) k_bbox(const int32_t* coords, int64_t n, int ncol, StrideArg st,
                                                   TableHeader* h) {
    __shared__ int sh_lo[kThreads / 64][kMaxCols], sh_hi[kThreads / 64][kMaxCols], sh_or[kThreads / 64][kMaxCols];
    int64_t lo[kMaxCols], hi[kMaxCols], v0[kMaxCols];
    int vary[kMaxCols];
    for (int c = 0; c < kMaxCols; ++c) {
        lo[c] = INT_MAX;
        hi[c] = INT_MIN;
        vary[c] = 0;
    }
    load_row(coords, 0, ncol, st, v0);   // n > 0 here
    bool out_of_range = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    // kBboxRows rows per thread and round, all loaded before any is used
    constexpr int kBboxRows = 4;
    for (int64_t r0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r0 < n; r0 += kBboxRows * stride) {
        int32_t raw[kBboxRows][kMaxCols];
#pragma unroll
        for (int i = 0; i < kBboxRows; ++i) {
            const int64_t r = r0 + i * stride;
            const int64_t rr = r < n ? r : r0;   // a row past the end repeats the first one
#pragma unroll
            for (int c = 0; c < kMaxCols; ++c) raw[i][c] = c < ncol ? coords[rr * ncol + c] : 0;
        }
#pragma unroll
        for (int i = 0; i < kBboxRows; ++i) {
#pragma unroll
            for (int c = 0; c < kMaxCols; ++c) {
                if (c >= ncol) break;
                int64_t x = raw[i][c];
                if (st.on && c > 0) x = floor_mul(x, st.s[c]);
                out_of_range |= x < INT_MIN || x > INT_MAX;   // strided value left int32
                lo[c] = x < lo[c] ? x : lo[c];
                hi[c] = x > hi[c] ? x : hi[c];
                vary[c] |= (int)(x ^ v0[c]);
            }
        }
    }
    if (out_of_range) atomicOr(&h->status, ST_RANGE);
    const int w = threadIdx.x >> 6;
    for (int c = 0; c < ncol; ++c) {
        int a = (int)max(lo[c], (int64_t)INT_MIN), b = (int)min(hi[c], (int64_t)INT_MAX), o = vary[c];
        for (int d = 32; d > 0; d >>= 1) {
            int ta = __shfl_xor(a, d, 64), tb = __shfl_xor(b, d, 64), to = __shfl_xor(o, d, 64);
            a = ta < a ? ta : a;
            b = tb > b ? tb : b;
            o |= to;
        }
        if (__lane_id() == 0) {
            sh_lo[w][c] = a;
            sh_hi[w][c] = b;
            sh_or[w][c] = o;
        }
    }
    __syncthreads();
    if (threadIdx.x < ncol) {
        const int c = threadIdx.x;
        int a = sh_lo[0][c], b = sh_hi[0][c], o = sh_or[0][c];
        for (int i = 1; i < kThreads / 64; ++i) {
            a = sh_lo[i][c] < a ? sh_lo[i][c] : a;
            b = sh_hi[i][c] > b ? sh_hi[i][c] : b;
            o |= sh_or[i][c];
        }
        atomicMin(&h->lo[c], a);
        atomicMax(&h->hi[c], b);
        if (o) atomicOr(&h->vary[c], o);
    }
}

// The packed key's layout from the bounding box: bit widths and shifts per
// column, and the blocked columns of the slot hash (see home_slot).
struct KeyLayout {
    int32_t shift[kMaxCols], bits[kMaxCols];
    int32_t total_bits, nblk, blk_shift[3];
};

__device__ void key_layout(const TableHeader* h, int ncol, KeyLayout* kl) {
    int total = 0;
    for (int c = 0; c < kMaxCols; ++c) {
        int b = 0;
        if (c < ncol) {
            const int64_t range = (int64_t)h->hi[c] - (int64_t)h->lo[c];
            if (range > 0) b = 64 - __clzll((unsigned long long)range);
            if (h->lo[c] > h->hi[c]) b = 0;   // no rows
        }
        kl->bits[c] = b;
        total += b;
    }
    int sh = 0;
    for (int c = kMaxCols - 1; c >= 0; --c) {
        kl->shift[c] = c < ncol ? sh : 0;
        if (c < ncol) sh += kl->bits[c];
    }
    kl->total_bits = total;
    int nb = 0;
    for (int i = 0; i < 3; ++i) kl->blk_shift[i] = 0;
    for (int c = 1; c < ncol && nb < 3; ++c) {
        const int t = h->vary[c] ? __ffs(h->vary[c]) - 1 : -1;   // lowest varying bit
        if (t >= 0 && t < kl->bits[c]) kl->blk_shift[nb++] = kl->shift[c] + t;
    }
    kl->nblk = nb;
}

// the layout into the header (ST_RANGE when the key needs more than kMaxKeyBits)
__device__ void store_key_layout(TableHeader* h, int ncol, const KeyLayout& kl) {
    for (int c = 0; c < ncol; ++c) {
        h->shift[c] = kl.shift[c];
        h->bits[c] = kl.bits[c];
    }
    h->total_bits = kl.total_bits;
    if (kl.total_bits > kMaxKeyBits) atomicOr(&h->status, ST_RANGE);
    for (int i = 0; i < 3; ++i) h->blk_shift[i] = kl.blk_shift[i];
    h->nblk = kl.nblk;
}

// one thread: the key layout of a table with no rows to insert
__global__ void k_plan(TableHeader* h) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    KeyLayout kl;
    key_layout(h, h->ncol, &kl);
    store_key_layout(h, h->ncol, kl);
}

// The insert kernels work the key layout out from the bounding box
// themselves (thread 0 of every block, into LDS), so no launch of its own
// sits between the box and the inserts; block 0 also stores it in the header
// for the kernels after them.  Returns the view a query needs and whether
// the key fits (all blocks compute the same).
__device__ __forceinline__ bool block_key_view(TableHeader* h, int ncol, KeyLayout* kl_s, TableView* tv) {
    if (threadIdx.x == 0) {
        key_layout(h, ncol, kl_s);
        if (blockIdx.x == 0) store_key_layout(h, ncol, *kl_s);
    }
    __syncthreads();
    tv->sh.mask = (unsigned long long)h->capacity - 1;
    tv->sh.nblk = kl_s->nblk;
    for (int i = 0; i < 3; ++i) tv->sh.blk_shift[i] = kl_s->blk_shift[i];
    tv->ncol = ncol;
    for (int c = 0; c < kMaxCols; ++c) {
        tv->lo[c] = c < ncol ? h->lo[c] : 0;
        tv->hi[c] = c < ncol ? h->hi[c] : 0;
        tv->shift[c] = kl_s->shift[c];
    }
    return kl_s->total_bits <= kMaxKeyBits;
}

// Wide keys: the CAS claims a slot by the key's low 62 bits and the claiming
// thread then writes the high bits into Slot::hi.  A thread that meets the
// same low bits reads Slot::hi, and while it is still unset it polls the same
// slot again: the writer has claimed it and stores right after.  The claim's
// store comes before any comparison in every round, so a writer in the same
// wave has stored before its neighbours look.  The probing ends when the key
// is placed or found or the table has been walked through; a slot whose high
// bits stay unset past kWidePolls polls ends it with ST_FULL.
constexpr int kWidePolls = 1 << 22;

// One round of a wide find-or-insert at slot s: returns 1 placed (this thread
// claimed the slot), 2 found (the slot holds the key), 3 retry the same slot,
// 0 move on.
__device__ __forceinline__ int wide_round(Slot* slots, unsigned long long s, unsigned long long lo, int32_t hi) {
    const unsigned long long prev = atomicCAS(&slots[s].key, kEmptyKey, lo);
    const bool won = prev == kEmptyKey;
    if (won) __hip_atomic_store(&slots[s].hi, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    if (won) return 1;
    if (prev != lo) return 0;
    const int32_t h2 = __hip_atomic_load(&slots[s].hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return h2 == kHiUnset ? 3 : (h2 == hi ? 2 : 0);
}

// a row of a table with wide keys (k_insert)
__device__ void insert_wide(const TableView& tv, const int64_t* v, int64_t r, TableHeader* h, Slot* slots) {
    u128 key;
    if (!pack_key_wide(tv, v, &key)) {   // cannot happen: the box holds every row
        atomicOr(&h->status, ST_RANGE);
        return;
    }
    const unsigned long long lo = wide_lo(key), mask = tv.sh.mask;
    const int32_t hi = wide_hi(key);
    unsigned long long s = home_slot_wide(tv.sh, key);
    int polls = 0;
    for (unsigned long long i = 0; i <= mask;) {
        const int res = wide_round(slots, s, lo, hi);
        if (res == 1) {
            slots[s].val = (int32_t)r;
            return;
        }
        if (res == 2) {
            atomicOr(&h->status, ST_DUP);
            return;
        }
        if (res == 3) {
            if (++polls > kWidePolls) break;
            continue;
        }
        s = (s + 1) & mask;
        ++i;
    }
    atomicOr(&h->status, ST_FULL);
}

__global__ void __launch_bounds__(kThreads) k_insert(const int32_t* coords, int64_t n, TableHeader* h,
                                                     Slot* slots) {
    __shared__ KeyLayout kl_s;
    const int ncol = h->ncol;
    TableView tv;
    const bool fits = block_key_view(h, ncol, &kl_s, &tv);
    const int64_t r = xcd_unit(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    if (r >= n || !fits) return;
    if (h->status & ST_RANGE) return;   // set by the box: a row outside int32
    const unsigned long long mask = tv.sh.mask;
    int64_t v[kMaxCols];
    StrideArg none{};
    load_row(coords, r, ncol, none, v);
    if (kl_s.total_bits > kNarrowKeyBits) {   // uniform
        insert_wide(tv, v, r, h, slots);
        return;
    }
    unsigned long long key;
    if (!pack_key(tv, v, &key)) {  // cannot happen: the box holds every row
        atomicOr(&h->status, ST_RANGE);
        return;
    }
    unsigned long long s = home_slot(tv.sh, key);
    for (unsigned long long i = 0; i <= mask; ++i) {
        unsigned long long prev = atomicCAS(&slots[s].key, kEmptyKey, key);
        if (prev == kEmptyKey) {
            slots[s].val = (int32_t)r;
            return;
        }
        if (prev == key) {
            atomicOr(&h->status, ST_DUP);
            return;
        }
        s = (s + 1) & mask;
    }
    atomicOr(&h->status, ST_FULL);
}

// strided: find-or-insert the strided key, keep the smallest input row that
// produces it; remember the slot of every row.
// Rows of one wave are consecutive, so rows with the same (strided) key are
// often neighbouring lanes: only the first lane of each run of equal keys
// inserts (its row is the run's smallest) and the others take its slot by a
// shuffle, which spares the contended atomics on the shared slot.
__global__ void __launch_bounds__(kThreads) k_insert_min(const int32_t* coords, int64_t n, StrideArg st,
                                                         TableHeader* h, Slot* slots, int64_t* slot_of) {
    __shared__ KeyLayout kl_s;
    const int ncol = h->ncol;
    TableView tv;
    const bool fits = block_key_view(h, ncol, &kl_s, &tv);
    const int64_t r = xcd_unit(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    const bool valid = r < n;
    if (!fits || (h->status & ST_RANGE)) {   // uniform (the box's flag is set before this kernel)
        if (valid) slot_of[r] = 0;
        return;
    }
    const unsigned long long mask = tv.sh.mask;
    const bool wide = kl_s.total_bits > kNarrowKeyBits;   // uniform
    unsigned long long key = 0;   // a narrow key, or a wide key's low 62 bits
    int32_t khi = 0;              // a wide key's high bits
    u128 wkey = 0;
    bool ok = false;
    if (valid) {
        int64_t v[kMaxCols];
        load_row(coords, r, ncol, st, v);
        if (wide) {
            ok = pack_key_wide(tv, v, &wkey);
            key = wide_lo(wkey);
            khi = wide_hi(wkey);
        } else {
            ok = pack_key(tv, v, &key);
        }
        if (!ok) {
            atomicOr(&h->status, ST_RANGE);
            slot_of[r] = 0;
        }
    }
    const int lane = __lane_id();
    const unsigned long long pkey = __shfl_up(key, 1, 64);
    const int32_t phi = __shfl_up(khi, 1, 64);
    const bool pok = __shfl_up((int)ok, 1, 64) != 0;
    const bool follower = ok && lane > 0 && pok && pkey == key && phi == khi;
    const unsigned long long leaders = __ballot(ok && !follower);
    unsigned long long s = 0;
    if (ok && !follower) {
        bool placed = false;
        if (wide) {   // see insert_wide
            s = home_slot_wide(tv.sh, wkey);
            int polls = 0;
            for (unsigned long long i = 0; i <= mask;) {
                const int res = wide_round(slots, s, key, khi);
                if (res == 1 || res == 2) {
                    atomicMin(&slots[s].val, (int32_t)r);
                    placed = true;
                    break;
                }
                if (res == 3) {
                    if (++polls > kWidePolls) break;
                    continue;
                }
                s = (s + 1) & mask;
                ++i;
            }
        } else {
            s = home_slot(tv.sh, key);
            for (unsigned long long i = 0; i <= mask; ++i) {
                const unsigned long long prev = atomicCAS(&slots[s].key, kEmptyKey, key);
                if (prev == kEmptyKey || prev == key) {
                    atomicMin(&slots[s].val, (int32_t)r);
                    placed = true;
                    break;
                }
                s = (s + 1) & mask;
            }
        }
        if (!placed) {
            atomicOr(&h->status, ST_FULL);
            s = 0;
        }
    }
    // a follower's run starts at the highest leader lane at or below it
    const unsigned long long upto = lane == 63 ? ~0ull : ((2ull << lane) - 1ull);
    const unsigned long long lm = leaders & upto;
    const int ld = lm ? 63 - __clzll(lm) : lane;
    const unsigned long long ls = __shfl(s, ld, 64);
    if (ok) slot_of[r] = (int64_t)(follower ? ls : s);
}

// mark representatives (slot holds this row) and count them per 64-row group
__global__ void __launch_bounds__(kThreads) k_rep_count(int64_t n, const TableHeader* h, const Slot* slots,
                                                        int64_t* slot_of, int32_t* cnt) {
    const int64_t r = xcd_unit(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    bool rep = false;
    if (r < n && h->status == 0) {
        const int64_t s = slot_of[r];
        rep = slots[s].val == (int32_t)r;
        if (rep) slot_of[r] = ~s;   // negative: representative
    }
    const unsigned long long m = __ballot(rep);
    const int64_t g = r >> 6;
    if (__lane_id() == 0 && g * 64 < n) cnt[g] = __popcll(m);
}

__global__ void __launch_bounds__(kThreads) k_rep_write(const int32_t* coords, int64_t n, StrideArg st,
                                                        TableHeader* h, Slot* slots, const int64_t* slot_of,
                                                        const int64_t* off, int32_t* out_coords, int32_t* rep_row) {
    const int64_t r = xcd_unit(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
    bool rep = false;
    int64_t s = 0;
    if (r < n && h->status == 0) {
        s = slot_of[r];
        rep = s < 0;
        s = ~s;
    }
    const unsigned long long m = __ballot(rep);
    if (!rep) return;
    const int64_t row = off[r >> 6] + __popcll(m & lanemask_lt());
    const int ncol = h->ncol;
    int64_t v[kMaxCols];
    load_row(coords, r, ncol, st, v);
    for (int c = 0; c < ncol; ++c) out_coords[row * ncol + c] = (int32_t)v[c];
    slots[s].val = (int32_t)row;
    if (rep_row) rep_row[row] = (int32_t)r;
}

// ---------------------------------------------------------------------------
// Sparse tensor quantization (Sec. 4.1, Alg. 1): integer rows (b, floor(p/v))
// deduplicated through the table exactly as strided output coordinates are
// (first point of a voxel is its representative, rows in the order of their
// representatives), then labels merged per voxel.
// ---------------------------------------------------------------------------
struct VoxelArg {
    float v[kMaxCols - 1];   // voxel size per spatial axis
};

// qc[r] = (batch[r] or 0, floor(p_d / v_d)), the floor of the exact quotient
// of the stored float32 values.  A coordinate outside +-2^30 sets the range
// status.
__global__ void __launch_bounds__(kThreads) k_quantize(const float* __restrict__ points,
                                                       const int32_t* __restrict__ batch, int64_t n, int D, VoxelArg va,
                                                       int32_t* __restrict__ qc, TableHeader* h) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n) return;
    const int ncol = D + 1;
    qc[r * ncol] = batch ? batch[r] : 0;
    bool bad = false;
    for (int d = 0; d < D; ++d) {
        // floor of the exact quotient p / v of the stored float32 values.  The
        // quotient rounded to double is at least floor(p / v) (every integer
        // below 2^53 is a double) and at most floor(p / v) + 1; the fma
        // residual p - f v is rounded once, so its sign is that of the exact
        // residual, and a negative one means f overshoots by one.
        const double p = (double)points[r * D + d], v = (double)va.v[d];
        double f = floor(p / v);
        if (fma(-f, v, p) < 0.0) f -= 1.0;
        bad |= !(f >= -1073741824.0 && f <= 1073741824.0);   // also NaN
        qc[r * ncol + 1 + d] = bad ? 0 : (int32_t)f;
    }
    if (bad) atomicOr(&h->status, ST_RANGE);
}

// per voxel: the row of every point (inverse) and the min / max label of its points
__global__ void __launch_bounds__(kThreads) k_quant_labels(int64_t n, const TableHeader* h, const Slot* slots,
                                                           const int64_t* __restrict__ slot_of,
                                                           const int32_t* __restrict__ labels,
                                                           int32_t* __restrict__ inverse, int32_t* __restrict__ lmin,
                                                           int32_t* __restrict__ lmax) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n || h->status != 0) return;
    int64_t sl = slot_of[r];
    if (sl < 0) sl = ~sl;   // a representative
    const int32_t o = slots[sl].val;
    if (o < 0 || o >= n) return;
    if (inverse) inverse[r] = o;
    if (labels) {
        atomicMin(&lmin[o], labels[r]);
        atomicMax(&lmax[o], labels[r]);
    }
}

__global__ void __launch_bounds__(kThreads) k_fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// voxel label: the points' common label, else ignore_label (f of Alg. 1)
__global__ void __launch_bounds__(kThreads) k_quant_final(int64_t cap, const TableHeader* h,
                                                          const int32_t* __restrict__ lmin,
                                                          const int32_t* __restrict__ lmax, int32_t ignore_label,
                                                          int32_t* __restrict__ out_labels) {
    const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (o >= cap || o >= h->n || h->status != 0) return;
    out_labels[o] = lmin[o] == lmax[o] ? lmin[o] : ignore_label;
}

static unsigned grid_for(int64_t n, int per = kThreads) {
    int64_t g = (n + per - 1) / per;
    if (g < 1) g = 1;
    return (unsigned)g;
}

static unsigned grid_capped(int64_t n, int64_t cap = 2048) {
    int64_t g = (n + kThreads - 1) / kThreads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

static int read_status(const void* table, hipStream_t s, TableHeader* out) {
    GSC_HIP(hipMemcpyAsync(out, table, sizeof(TableHeader), hipMemcpyDeviceToHost, s));
    GSC_HIP(hipStreamSynchronize(s));
    return GSC_OK;
}

static int status_to_code(const TableHeader& h, const char* what) {
    if (h.status & ST_RANGE)
        return fail(GSC_ERANGE, "%s: coordinates need more than %d key bits (box needs %d)", what, kMaxKeyBits,
                    h.total_bits);
    if (h.status & ST_DUP) return fail(GSC_EDUP, "%s: a coordinate row occurs more than once", what);
    if (h.status & ST_FULL) return fail(GSC_EFULL, "%s: hash table full", what);
    return GSC_OK;
}

}  // namespace gsc

using namespace gsc;

extern "C" {

size_t gsc_table_bytes(int64_t n) {
    if (n < 0) return 0;
    return kHeaderBytes + (size_t)table_capacity(n) * sizeof(Slot);
}

static int build_enqueue(const int32_t* coords, int64_t n, int32_t D, void* table, size_t table_bytes,
                         hipStream_t s, const char* what) {
    if (D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "%s: D=%d outside [1,%d]", what, D, kMaxCols - 1);
    if (n < 0 || n > INT32_MAX) return fail(GSC_EINVAL, "%s: n=%lld outside [0, 2^31)", what, (long long)n);
    if (!table) return fail(GSC_EINVAL, "%s: table is null", what);
    if (n > 0 && !coords) return fail(GSC_EINVAL, "%s: coords is null", what);
    if (table_bytes < gsc_table_bytes(n))
        return fail(GSC_ESHORT, "%s: table needs %zu bytes, got %zu", what, gsc_table_bytes(n), table_bytes);
    const int ncol = D + 1;
    const int64_t cap = table_capacity(n);
    TableHeader* h = reinterpret_cast<TableHeader*>(table);
    Slot* slots = table_slots(table);
    hipLaunchKernelGGL(k_table_init, dim3(grid_capped(cap)), dim3(kThreads), 0, s, h, slots, cap, ncol, n, -1);
    GSC_LAUNCH_CHECK();
    StrideArg none{};
    if (n > 0) {
        hipLaunchKernelGGL(k_bbox, dim3(grid_capped(n, 256)), dim3(kThreads), 0, s, coords, n, ncol, none, h);
        GSC_LAUNCH_CHECK();
    }
    if (n > 0)   // the inserts work out (and store) the key layout themselves
        hipLaunchKernelGGL(k_insert, dim3(grid_for(n)), dim3(kThreads), 0, s, coords, n, h, slots);
    else
        hipLaunchKernelGGL(k_plan, dim3(1), dim3(64), 0, s, h);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

int gsc_coords_build(const int32_t* coords, int64_t n, int32_t D, void* table, size_t table_bytes, void* stream) {
    clear_error();
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    int rc = build_enqueue(coords, n, D, table, table_bytes, s, "coords_build");
    if (rc) return rc;
    TableHeader hh;
    rc = read_status(table, s, &hh);
    if (rc) return rc;
    return status_to_code(hh, "coords_build");
}

int gsc_coords_build_async(const int32_t* coords, int64_t n, int32_t D, void* table, size_t table_bytes,
                           void* stream) {
    clear_error();
    return build_enqueue(coords, n, D, table, table_bytes, reinterpret_cast<hipStream_t>(stream),
                         "coords_build_async");
}

int gsc_table_status(const void* table, void* stream) {
    clear_error();
    if (!table) return fail(GSC_EINVAL, "table_status: table is null");
    TableHeader hh;
    int rc = read_status(table, reinterpret_cast<hipStream_t>(stream), &hh);
    if (rc) return rc;
    if (hh.magic != kTableMagic) return fail(GSC_EINVAL, "table_status: not a table built by gsc_coords_build");
    return status_to_code(hh, "table");
}

size_t gsc_stride_ws_bytes(int64_t n_in) {
    if (n_in < 0) return 0;
    const int64_t groups = (n_in + 63) / 64;
    size_t b = (size_t)n_in * sizeof(int64_t);            // slot of each row
    b = (b + 255) & ~(size_t)255;
    b += (size_t)groups * sizeof(int32_t);                // counts
    b = (b + 255) & ~(size_t)255;
    b += (size_t)(groups + 1) * sizeof(int64_t);          // offsets
    b = (b + 255) & ~(size_t)255;
    b += scan_ws_bytes(groups);
    return b + 256;
}

// The kernels of gsc_coords_stride; the output count ends in the header (n).
static int stride_enqueue(const int32_t* in_coords, int64_t n_in, int32_t D, const int32_t* stride,
                          int32_t* out_coords, void* out_table, size_t out_table_bytes, void* ws, size_t ws_bytes,
                          hipStream_t s, const char* what) {
    if (D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "%s: D=%d outside [1,%d]", what, D, kMaxCols - 1);
    if (n_in < 0 || n_in > INT32_MAX) return fail(GSC_EINVAL, "%s: n_in=%lld invalid", what, (long long)n_in);
    if (!stride || !out_table) return fail(GSC_EINVAL, "%s: null stride/out_table", what);
    if (n_in > 0 && (!in_coords || !out_coords || !ws)) return fail(GSC_EINVAL, "%s: null in_coords/out_coords/ws", what);
    StrideArg st{};
    st.on = 1;
    st.s[0] = 1;
    for (int d = 0; d < D; ++d) {
        if (stride[d] < 1) return fail(GSC_EINVAL, "%s: stride[%d]=%d must be >= 1", what, d, stride[d]);
        st.s[d + 1] = stride[d];
    }
    if (out_table_bytes < gsc_table_bytes(n_in))
        return fail(GSC_ESHORT, "%s: out_table needs %zu bytes, got %zu", what, gsc_table_bytes(n_in), out_table_bytes);
    if (n_in > 0 && ws_bytes < gsc_stride_ws_bytes(n_in))
        return fail(GSC_ESHORT, "%s: ws needs %zu bytes, got %zu", what, gsc_stride_ws_bytes(n_in), ws_bytes);
    const int ncol = D + 1;
    const int64_t cap = table_capacity(n_in);
    TableHeader* h = reinterpret_cast<TableHeader*>(out_table);
    Slot* slots = table_slots(out_table);
    hipLaunchKernelGGL(k_table_init, dim3(grid_capped(cap)), dim3(kThreads), 0, s, h, slots, cap, ncol,
                       (int64_t)0, (int32_t)INT_MAX);
    GSC_LAUNCH_CHECK();
    if (n_in == 0) {
        hipLaunchKernelGGL(k_plan, dim3(1), dim3(64), 0, s, h);
        GSC_LAUNCH_CHECK();
        return GSC_OK;
    }
    const int64_t groups = (n_in + 63) / 64;
    char* w = reinterpret_cast<char*>(ws);
    int64_t* slot_of = reinterpret_cast<int64_t*>(w);
    w += ((size_t)n_in * sizeof(int64_t) + 255) & ~(size_t)255;
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += ((size_t)groups * sizeof(int32_t) + 255) & ~(size_t)255;
    int64_t* off = reinterpret_cast<int64_t*>(w);
    w += ((size_t)(groups + 1) * sizeof(int64_t) + 255) & ~(size_t)255;
    void* scan_ws = w;

    hipLaunchKernelGGL(k_bbox, dim3(grid_capped(n_in, 256)), dim3(kThreads), 0, s, in_coords, n_in, ncol, st, h);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_insert_min, dim3(grid_for(n_in)), dim3(kThreads), 0, s, in_coords, n_in, st, h, slots,
                       slot_of);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_rep_count, dim3(grid_for(n_in)), dim3(kThreads), 0, s, n_in, h, slots, slot_of, cnt);
    GSC_LAUNCH_CHECK();
    int rc = scan_counts(cnt, groups, off, &h->n, scan_ws, s);   // header n = number of output rows
    if (rc) return rc;
    hipLaunchKernelGGL(k_rep_write, dim3(grid_for(n_in)), dim3(kThreads), 0, s, in_coords, n_in, st, h, slots,
                       slot_of, off, out_coords, (int32_t*)nullptr);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

int gsc_coords_stride(const int32_t* in_coords, int64_t n_in, int32_t D, const int32_t* stride,
                      int32_t* out_coords, int64_t* n_out, void* out_table, size_t out_table_bytes, void* ws,
                      size_t ws_bytes, void* stream) {
    clear_error();
    if (!n_out) return fail(GSC_EINVAL, "coords_stride: null n_out");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    int rc = stride_enqueue(in_coords, n_in, D, stride, out_coords, out_table, out_table_bytes, ws, ws_bytes, s,
                            "coords_stride");
    if (rc) return rc;
    TableHeader hh;
    rc = read_status(out_table, s, &hh);
    if (rc) return rc;
    rc = status_to_code(hh, "coords_stride");
    if (rc) return rc;
    *n_out = hh.n;
    return GSC_OK;
}

// The header's n, status and total_bits, contiguous: what the asynchronous
// form copies to the host.
static_assert(offsetof(TableHeader, status) == offsetof(TableHeader, n) + 8 &&
                  offsetof(TableHeader, total_bits) == offsetof(TableHeader, n) + 12,
              "header layout of the stride result");

int gsc_coords_stride_async(const int32_t* in_coords, int64_t n_in, int32_t D, const int32_t* stride,
                            int32_t* out_coords, int64_t* result, void* out_table, size_t out_table_bytes, void* ws,
                            size_t ws_bytes, void* stream) {
    clear_error();
    if (!result) return fail(GSC_EINVAL, "coords_stride_async: null result");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    int rc = stride_enqueue(in_coords, n_in, D, stride, out_coords, out_table, out_table_bytes, ws, ws_bytes, s,
                            "coords_stride_async");
    if (rc) return rc;
    GSC_HIP(hipMemcpyAsync(result, &reinterpret_cast<TableHeader*>(out_table)->n, 16, hipMemcpyDeviceToHost, s));
    return GSC_OK;
}

int gsc_coords_stride_result(const int64_t* result, int64_t* n_out) {
    clear_error();
    if (!result || !n_out) return fail(GSC_EINVAL, "coords_stride_result: null result/n_out");
    TableHeader hh{};
    hh.n = result[0];
    std::memcpy(&hh.status, reinterpret_cast<const char*>(result) + 8, 4);
    std::memcpy(&hh.total_bits, reinterpret_cast<const char*>(result) + 12, 4);
    const int rc = status_to_code(hh, "coords_stride");
    if (rc) return rc;
    *n_out = hh.n;
    return GSC_OK;
}

size_t gsc_quantize_ws_bytes(int64_t n, int32_t D) {
    if (n < 0 || D < 1 || D + 1 > kMaxCols) return 0;
    const int64_t groups = (n + 63) / 64;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    size_t b = al((size_t)n * (D + 1) * sizeof(int32_t));   // integer rows
    b += al((size_t)n * sizeof(int64_t));                    // slot of each row
    b += al((size_t)groups * sizeof(int32_t));               // counts
    b += al((size_t)(groups + 1) * sizeof(int64_t));         // offsets
    b += 2 * al((size_t)n * sizeof(int32_t));                // label min / max per voxel
    b += scan_ws_bytes(groups);
    return b + 256;
}

int gsc_quantize(const float* points, const int32_t* batch, int64_t n, int32_t D, const float* voxel,
                 const int32_t* labels, int32_t ignore_label, int32_t* out_coords, int64_t* n_out, int32_t* rep,
                 int32_t* out_labels, int32_t* inverse, void* out_table, size_t out_table_bytes, void* ws,
                 size_t ws_bytes, void* stream) {
    clear_error();
    if (D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "quantize: D=%d outside [1,%d]", D, kMaxCols - 1);
    if (n < 0 || n > INT32_MAX) return fail(GSC_EINVAL, "quantize: n=%lld invalid", (long long)n);
    if (!voxel || !n_out || !out_table) return fail(GSC_EINVAL, "quantize: null voxel/n_out/out_table");
    if (n > 0 && (!points || !out_coords || !rep || !ws))
        return fail(GSC_EINVAL, "quantize: null points/out_coords/rep/ws");
    if (n > 0 && out_labels && !labels) return fail(GSC_EINVAL, "quantize: out_labels without labels");
    VoxelArg va{};
    for (int d = 0; d < D; ++d) {
        if (!(voxel[d] > 0.f) || voxel[d] == INFINITY)
            return fail(GSC_EINVAL, "quantize: voxel[%d]=%g must be positive and finite", d, (double)voxel[d]);
        va.v[d] = voxel[d];
    }
    if (out_table_bytes < gsc_table_bytes(n))
        return fail(GSC_ESHORT, "quantize: out_table needs %zu bytes, got %zu", gsc_table_bytes(n), out_table_bytes);
    if (n > 0 && ws_bytes < gsc_quantize_ws_bytes(n, D))
        return fail(GSC_ESHORT, "quantize: ws needs %zu bytes, got %zu", gsc_quantize_ws_bytes(n, D), ws_bytes);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int ncol = D + 1;
    const int64_t cap = table_capacity(n);
    TableHeader* h = reinterpret_cast<TableHeader*>(out_table);
    Slot* slots = table_slots(out_table);
    hipLaunchKernelGGL(k_table_init, dim3(grid_capped(cap)), dim3(kThreads), 0, s, h, slots, cap, ncol, (int64_t)0,
                       (int32_t)INT_MAX);
    GSC_LAUNCH_CHECK();
    if (n == 0) {
        hipLaunchKernelGGL(k_plan, dim3(1), dim3(64), 0, s, h);
        GSC_LAUNCH_CHECK();
        GSC_HIP(hipStreamSynchronize(s));
        *n_out = 0;
        return GSC_OK;
    }
    const int64_t groups = (n + 63) / 64;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    char* w = reinterpret_cast<char*>(ws);
    int32_t* qc = reinterpret_cast<int32_t*>(w);
    w += al((size_t)n * ncol * sizeof(int32_t));
    int64_t* slot_of = reinterpret_cast<int64_t*>(w);
    w += al((size_t)n * sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += al((size_t)groups * sizeof(int32_t));
    int64_t* off = reinterpret_cast<int64_t*>(w);
    w += al((size_t)(groups + 1) * sizeof(int64_t));
    int32_t* lmin = reinterpret_cast<int32_t*>(w);
    w += al((size_t)n * sizeof(int32_t));
    int32_t* lmax = reinterpret_cast<int32_t*>(w);
    w += al((size_t)n * sizeof(int32_t));
    void* scan_ws = w;

    StrideArg none{};
    hipLaunchKernelGGL(k_quantize, dim3(grid_for(n)), dim3(kThreads), 0, s, points, batch, n, (int)D, va, qc, h);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_bbox, dim3(grid_capped(n, 256)), dim3(kThreads), 0, s, qc, n, ncol, none, h);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_insert_min, dim3(grid_for(n)), dim3(kThreads), 0, s, qc, n, none, h, slots, slot_of);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_rep_count, dim3(grid_for(n)), dim3(kThreads), 0, s, n, h, slots, slot_of, cnt);
    GSC_LAUNCH_CHECK();
    int rc = scan_counts(cnt, groups, off, &h->n, scan_ws, s);   // header n = number of voxels
    if (rc) return rc;
    hipLaunchKernelGGL(k_rep_write, dim3(grid_for(n)), dim3(kThreads), 0, s, qc, n, none, h, slots, slot_of, off,
                       out_coords, rep);
    GSC_LAUNCH_CHECK();
    if (labels) {
        hipLaunchKernelGGL(k_fill_i32, dim3(grid_capped(n)), dim3(kThreads), 0, s, lmin, n, (int32_t)INT_MAX);
        GSC_LAUNCH_CHECK();
        hipLaunchKernelGGL(k_fill_i32, dim3(grid_capped(n)), dim3(kThreads), 0, s, lmax, n, (int32_t)INT_MIN);
        GSC_LAUNCH_CHECK();
    }
    if (labels || inverse) {
        hipLaunchKernelGGL(k_quant_labels, dim3(grid_for(n)), dim3(kThreads), 0, s, n, h, slots, slot_of, labels,
                           inverse, lmin, lmax);
        GSC_LAUNCH_CHECK();
    }
    if (labels && out_labels) {
        hipLaunchKernelGGL(k_quant_final, dim3(grid_for(n)), dim3(kThreads), 0, s, n, h, lmin, lmax, ignore_label,
                           out_labels);
        GSC_LAUNCH_CHECK();
    }
    TableHeader hh;
    rc = read_status(out_table, s, &hh);
    if (rc) return rc;
    rc = status_to_code(hh, "quantize");
    if (rc) return rc;
    *n_out = hh.n;
    return GSC_OK;
}

}  // extern "C"
