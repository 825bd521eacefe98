// Internal definitions shared by the HIP sources of libgsc.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>
#include <cstddef>

#include "../../include/gsc.h"

namespace gsc {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

#define GSC_HIP(call)                                                                  \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess)                                                          \
            return ::gsc::fail(GSC_EHIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
    } while (0)

#define GSC_LAUNCH_CHECK()                                                             \
    do {                                                                               \
        hipError_t e_ = hipGetLastError();                                             \
        if (e_ != hipSuccess)                                                          \
            return ::gsc::fail(GSC_EHIP, "kernel launch failed: %s", hipGetErrorString(e_)); \
    } while (0)

// ---------------------------------------------------------------------------
// coordinate hash table (lives in caller memory)
// ---------------------------------------------------------------------------
constexpr int kMaxCols = 8;                       // 1 batch column + up to 7 spatial
constexpr unsigned long long kEmptyKey = ~0ull;    // Slot::key holds <= 62 key bits
constexpr uint32_t kTableMagic = 0x54435347u;      // "GSCT"
constexpr size_t kHeaderBytes = 256;
// A packed key of up to kNarrowKeyBits bits lives in Slot::key alone; a wider
// one (up to kMaxKeyBits) keeps its low 62 bits there and the rest in
// Slot::hi, which the inserting thread writes right after claiming the slot
// (kHiUnset until then).
constexpr int kNarrowKeyBits = 62;
constexpr int kMaxKeyBits = 92;
constexpr int32_t kHiUnset = -1;
typedef unsigned __int128 u128;

enum : int { ST_DUP = 1, ST_FULL = 2, ST_RANGE = 4 };

struct TableHeader {
    uint32_t magic;
    int32_t ncol;          // 1 + D
    int64_t capacity;      // slots, power of two
    int64_t n;             // number of keys
    int32_t status;        // ST_* bits set on the device
    int32_t total_bits;
    int32_t lo[kMaxCols];  // bounding box, inclusive
    int32_t hi[kMaxCols];
    int32_t shift[kMaxCols];
    int32_t bits[kMaxCols];
    int32_t vary[kMaxCols];  // OR over rows of (row XOR first row): the bits that vary per column
    int32_t nblk;            // spatial columns whose lowest varying key bit selects the slot in a line
    int32_t blk_shift[3];    // that key bit, per blocked column
};
static_assert(sizeof(TableHeader) <= kHeaderBytes, "header too large");

struct alignas(16) Slot {
    unsigned long long key;
    int32_t val;
    int32_t hi;   // key bits 62 and up of a wide key
};
static_assert(sizeof(Slot) == 16, "slot must be 16 bytes");

// capacity: a power of two >= 4n (load factor <= 1/4) and >= 64.  The
// environment variable GSC_TABLE_CAP_LIMIT (a test hook) caps it at the
// largest power of two >= 64 not above its value, so that a table too small
// for its rows, and the EFULL it reports, can be exercised; every insert and
// query still stops after one pass over the slots.
inline int64_t table_capacity(int64_t n) {
    int64_t cap = 64;
    while (cap < 4 * n) cap <<= 1;
    if (const char* e = getenv("GSC_TABLE_CAP_LIMIT")) {
        const long long lim = strtoll(e, nullptr, 10);
        while (cap > 64 && cap > lim) cap >>= 1;
    }
    return cap;
}

inline __host__ __device__ Slot* table_slots(void* t) {
    return reinterpret_cast<Slot*>(reinterpret_cast<char*>(t) + kHeaderBytes);
}
inline __host__ __device__ const Slot* table_slots(const void* t) {
    return reinterpret_cast<const Slot*>(reinterpret_cast<const char*>(t) + kHeaderBytes);
}

// 32-bit finaliser of MurmurHash3 (Appleby): a bijective avalanche mix.
__device__ __forceinline__ uint32_t fmix32(uint32_t h) {
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

// Hash of a (<= 62-bit) key: fold the high word in with a multiply, then mix.
__device__ __forceinline__ uint32_t hash_key(unsigned long long k) {
    return fmix32((uint32_t)k ^ ((uint32_t)(k >> 32) * 0x9e3779b1u));
}

// Hash of a wide key: its high word folded into the low one, then hash_key.
__device__ __forceinline__ uint32_t hash_key_wide(u128 k) {
    return hash_key((unsigned long long)k ^ ((unsigned long long)(k >> 64) * 0x9e3779b97f4a7c15ull));
}
__device__ __forceinline__ unsigned long long wide_lo(u128 k) {
    return (unsigned long long)k & ((1ull << kNarrowKeyBits) - 1ull);
}
__device__ __forceinline__ int32_t wide_hi(u128 k) { return (int32_t)(uint32_t)(k >> kNarrowKeyBits); }

// Home slot of a key.  The lowest varying bit of each of the first (up to)
// three spatial columns (bit 0 for unit tensor stride, bit 1 for coordinates
// that are all even, ...) selects the slot inside an aligned group of 2^nblk
// slots and the rest of the key is hashed to pick the group, so the 2 x 2 x 2
// block of coordinates around a point shares one 128-byte line of the table
// and a 3 x 3 x 3 neighbourhood touches about 8 lines instead of 27.
struct SlotHash {
    unsigned long long mask;   // capacity - 1
    int nblk;
    int blk_shift[3];
};

__device__ __forceinline__ SlotHash slot_hash(const TableHeader* h) {
    SlotHash sh;
    sh.mask = (unsigned long long)h->capacity - 1;
    sh.nblk = h->nblk;
    for (int i = 0; i < 3; ++i) sh.blk_shift[i] = h->blk_shift[i];
    return sh;
}

__device__ __forceinline__ unsigned long long home_slot(const SlotHash& sh, unsigned long long key) {
    unsigned long long local = 0, bkey = key;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        if (i < sh.nblk) {
            local |= ((key >> sh.blk_shift[i]) & 1ull) << i;
            bkey &= ~(1ull << sh.blk_shift[i]);
        }
    }
    return (((unsigned long long)hash_key(bkey) << sh.nblk) | local) & sh.mask;
}

// the same for a wide key (blocked bits, then hash_key_wide of the rest)
__device__ __forceinline__ unsigned long long home_slot_wide(const SlotHash& sh, u128 key) {
    unsigned long long local = 0;
    u128 bkey = key;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        if (i < sh.nblk) {
            local |= (unsigned long long)((key >> sh.blk_shift[i]) & 1u) << i;
            bkey &= ~((u128)1 << sh.blk_shift[i]);
        }
    }
    return (((unsigned long long)hash_key_wide(bkey) << sh.nblk) | local) & sh.mask;
}

// Register copy of the fields a query needs: loaded once per thread, so that
// stores made between queries (which may alias the table for the compiler)
// do not force the header to be read again.
struct TableView {
    SlotHash sh;
    int ncol;
    int32_t lo[kMaxCols], hi[kMaxCols], shift[kMaxCols];
};

__device__ __forceinline__ TableView table_view(const TableHeader* h, int ncol) {
    TableView t;
    t.sh = slot_hash(h);
    t.ncol = ncol;
    for (int c = 0; c < kMaxCols; ++c) {
        t.lo[c] = c < ncol ? h->lo[c] : 0;
        t.hi[c] = c < ncol ? h->hi[c] : 0;
        t.shift[c] = c < ncol ? h->shift[c] : 0;
    }
    return t;
}

// Pack a coordinate (already offset, in 64-bit) into a key; false if it lies
// outside the table's bounding box (such a coordinate cannot be in the table,
// so a query for it is a miss, never an alias of another key).  Unrolled
// over kMaxCols with a guard, so the arrays stay in registers.
__device__ __forceinline__ bool pack_key(const TableView& t, const int64_t* v, unsigned long long* key) {
    unsigned long long k = 0;
    bool in = true;
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c) {
        if (c < t.ncol) {
            in = in && v[c] >= t.lo[c] && v[c] <= t.hi[c];
            k |= (unsigned long long)(v[c] - t.lo[c]) << t.shift[c];
        }
    }
    *key = k;
    return in;
}

// the same for a wide key
__device__ __forceinline__ bool pack_key_wide(const TableView& t, const int64_t* v, u128* key) {
    u128 k = 0;
    bool in = true;
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c) {
        if (c < t.ncol) {
            in = in && v[c] >= t.lo[c] && v[c] <= t.hi[c];
            k |= (u128)(unsigned long long)(v[c] - t.lo[c]) << t.shift[c];
        }
    }
    *key = k;
    return in;
}

// floor(a / s) * s for s > 0
__device__ __forceinline__ int64_t floor_mul(int64_t a, int64_t s) {
    int64_t q = a / s;
    if ((a % s) != 0 && a < 0) q -= 1;
    return q * s;
}

// ---------------------------------------------------------------------------
// device-wide exclusive scan of int32 counts into int64 offsets:
// out[i] = sum(cnt[0..i)), out[m] = total; optionally also *total_out, and
// every_out[i / every] = out[i] for the multiples i of every (every > 0
// dividing m: a kernel map's segment table seg[k] = gidx[k * G]).
// ---------------------------------------------------------------------------
size_t scan_ws_bytes(int64_t m);
// compute units of the current device (cached per device; 256 if the query fails)
int device_cus();

int scan_counts(const int32_t* cnt, int64_t m, int64_t* out, int64_t* total_out, void* ws,
                hipStream_t s, int64_t* every_out = nullptr, int64_t every = 0);

// Largest offset count of one range of a block plan (neighbour masks are
// 32-bit).  A map with more offsets is planned in ranges of consecutive
// offsets (at most kPlanMaxRanges, of plan_range_size(K) offsets each but the
// last), each range a plan of its own over the same rows.
constexpr int kPlanMaxK = 32;
constexpr int kPlanMaxRanges = 4;
constexpr int kPlanMaxKAll = kPlanMaxK * kPlanMaxRanges;
inline int plan_ranges(int K) { return (K + kPlanMaxK - 1) / kPlanMaxK; }
inline int plan_range_size(int K) {
    const int R = plan_ranges(K);
    return (K + R - 1) / R;
}

// Rows of a block of the block plan (one MFMA row block).
constexpr int kPlanBlockRows = 16;

// p[i] = 0 for i < n.
__global__ void k_zero_i64(int64_t* p, int64_t n);

// seg[k] = gidx[k * G] for k <= K (offset starts from a group index).
int seg_from_gidx(const int64_t* gidx, int K, int64_t G, int64_t* seg, hipStream_t s);

// ---------------------------------------------------------------------------
// XCD-aware block order.  The eight XCDs of the MI355X receive workgroups
// round-robin (workgroup b runs on XCD b % 8) and each XCD has its own L2.
// Work unit t = xcd_unit(b, n) gives XCD x a contiguous range of units, so
// neighbouring units (which gather mostly the same rows) share an L2.  It is
// a bijection of [0, n).
// ---------------------------------------------------------------------------
constexpr int kNumXcd = 8;

__device__ __forceinline__ int64_t xcd_unit(int64_t b, int64_t n) {
    const int64_t q = n / kNumXcd, r = n % kNumXcd;
    const int64_t x = b % kNumXcd, i = b / kNumXcd;
    return x * q + (x < r ? x : r) + i;
}

// Work unit of a block for output tiles: tiles in the natural row order go
// to XCDs in contiguous ranges (neighbouring tiles gather mostly the same
// rows, which then share an L2); tiles of a plan (rows ordered by neighbour
// mask, so their cost varies along the order) go round-robin, which spreads
// cheap and expensive tiles evenly over the XCDs.
__device__ __forceinline__ int64_t tile_unit(int64_t b, int64_t n, bool planned) {
    return planned ? b : xcd_unit(b, n);
}

// ---------------------------------------------------------------------------
// wave helpers (wave64)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Order the LDS accesses of one wave: a lane may read what another lane of
// the same wave wrote just before.  The LDS executes a wave's operations in
// order; this keeps the compiler from moving accesses across the point.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ unsigned long long lanemask_lt() {
    const int l = __lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

}  // namespace gsc
