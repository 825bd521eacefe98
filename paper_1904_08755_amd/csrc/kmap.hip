// Kernel map (a3): for every offset o_k and output row j, the input row of
// u_j + ts (.) o_k, if present.  Two passes over (output row, offset):
//   count: one lane per output row; per offset a wave64 ballot of hits gives
//          the pair count of every 64-row group;
//   scan:  exclusive scan of the (offset-major, group-minor) counts gives the
//          start of each group's pairs (the group index gidx) and the total;
//   fill:  the same probes again; a hit is written at its group start plus
//          its rank among the wave's hits (popcount of the lower-lane mask).
// Pairs of one offset therefore come out sorted by output row, and the
// result does not depend on scheduling.
#include <climits>
#include <vector>

#include "gsc_internal.h"

namespace gsc {

constexpr int kThreads = 256;

__device__ __forceinline__ bool header_ok(const TableHeader* h, int ncol) {
    return h->magic == kTableMagic && h->ncol == ncol && h->status == 0;
}

__device__ __forceinline__ int32_t probe(const TableHeader* h, const Slot* slots, unsigned long long mask, int ncol,
                                         const int64_t* u, const int32_t* off) {
    int64_t q[kMaxCols];
    q[0] = u[0];
    for (int c = 1; c < ncol; ++c) q[c] = u[c] + off[c - 1];
    unsigned long long key;
    if (!pack_key(h, ncol, q, &key)) return -1;
    return table_find(slots, mask, key);
}

__global__ void __launch_bounds__(kThreads) k_kmap_count(const void* table, const int32_t* out_coords, int64_t n_out,
                                                         int ncol, const int32_t* offs, int K, int64_t G,
                                                         int32_t* cnt, int64_t* err) {
    const TableHeader* h = reinterpret_cast<const TableHeader*>(table);
    const Slot* slots = table_slots(table);
    const bool ok = header_ok(h, ncol);
    if (!ok && blockIdx.x == 0 && threadIdx.x == 0) *err = 1;
    const unsigned long long mask = ok ? (unsigned long long)h->capacity - 1 : 0;
    const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool valid = ok && j < n_out;
    int64_t u[kMaxCols];
    for (int c = 0; c < ncol; ++c) u[c] = valid ? out_coords[j * ncol + c] : 0;
    const int64_t g = j >> 6;
    const bool writer = __lane_id() == 0 && g < G;
    const int D = ncol - 1;
    for (int k = 0; k < K; ++k) {
        const bool hit = valid && probe(h, slots, mask, ncol, u, offs + (int64_t)k * D) >= 0;
        const unsigned long long m = __ballot(hit);
        if (writer) cnt[(int64_t)k * G + g] = __popcll(m);
    }
}

__global__ void __launch_bounds__(kThreads) k_kmap_fill(const void* table, const int32_t* out_coords, int64_t n_out,
                                                        int ncol, const int32_t* offs, int K, int64_t G,
                                                        const int64_t* gidx, int32_t* in_idx, int32_t* out_idx) {
    const TableHeader* h = reinterpret_cast<const TableHeader*>(table);
    const Slot* slots = table_slots(table);
    if (!header_ok(h, ncol)) return;
    const unsigned long long mask = (unsigned long long)h->capacity - 1;
    const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool valid = j < n_out;
    int64_t u[kMaxCols];
    for (int c = 0; c < ncol; ++c) u[c] = valid ? out_coords[j * ncol + c] : 0;
    const int64_t g = j >> 6;
    const int D = ncol - 1;
    const unsigned long long below = lanemask_lt();
    for (int k = 0; k < K; ++k) {
        const int32_t r = valid ? probe(h, slots, mask, ncol, u, offs + (int64_t)k * D) : -1;
        const unsigned long long m = __ballot(r >= 0);
        if (r >= 0) {
            const int64_t pos = gidx[(int64_t)k * G + g] + __popcll(m & below);
            in_idx[pos] = r;
            out_idx[pos] = (int32_t)j;
        }
    }
}

__global__ void k_seg_from_gidx(const int64_t* gidx, int K, int64_t G, int64_t* seg) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k <= K) seg[k] = gidx[(int64_t)k * G];
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace gsc

using namespace gsc;

extern "C" {

int64_t gsc_kmap_groups(int64_t n_out) { return n_out <= 0 ? 0 : (n_out + 63) / 64; }

size_t gsc_kmap_ws_bytes(int64_t n_out, int32_t K, int32_t D) {
    if (n_out < 0 || K < 1 || D < 1) return 0;
    const int64_t G = gsc_kmap_groups(n_out);
    size_t b = align256((size_t)K * D * sizeof(int32_t));      // offsets (scaled)
    b += align256(2 * sizeof(int64_t));                         // total, error flag
    b += align256((size_t)K * G * sizeof(int32_t));             // counts
    b += scan_ws_bytes(K * G);
    return b + 256;
}

int gsc_kernel_map(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D, const int32_t* offsets,
                   int32_t K, const int32_t* tensor_stride, int32_t* in_idx, int32_t* out_idx, int64_t cap_pairs,
                   int64_t* seg, int64_t* gidx, int64_t* n_pairs, void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "kernel_map: D=%d outside [1,%d]", D, kMaxCols - 1);
    if (K < 1) return fail(GSC_EINVAL, "kernel_map: K=%d must be >= 1", K);
    if (n_out < 0 || n_out > INT32_MAX) return fail(GSC_EINVAL, "kernel_map: n_out=%lld invalid", (long long)n_out);
    if (!in_table || !offsets || !seg || !gidx || !n_pairs || !ws)
        return fail(GSC_EINVAL, "kernel_map: null in_table/offsets/seg/gidx/n_pairs/ws");
    if (n_out > 0 && !out_coords) return fail(GSC_EINVAL, "kernel_map: out_coords is null");
    if (cap_pairs < 0) return fail(GSC_EINVAL, "kernel_map: cap_pairs < 0");
    if (cap_pairs > 0 && (!in_idx || !out_idx)) return fail(GSC_EINVAL, "kernel_map: null in_idx/out_idx");
    if (ws_bytes < gsc_kmap_ws_bytes(n_out, K, D))
        return fail(GSC_ESHORT, "kernel_map: ws needs %zu bytes, got %zu", gsc_kmap_ws_bytes(n_out, K, D), ws_bytes);
    std::vector<int32_t> offs((size_t)K * D);
    for (int k = 0; k < K; ++k)
        for (int d = 0; d < D; ++d) {
            const int64_t ts = tensor_stride ? tensor_stride[d] : 1;
            if (ts < 1) return fail(GSC_EINVAL, "kernel_map: tensor_stride[%d]=%lld must be >= 1", d, (long long)ts);
            const int64_t v = ts * (int64_t)offsets[(size_t)k * D + d];
            if (v < -(1ll << 30) || v > (1ll << 30))
                return fail(GSC_ERANGE, "kernel_map: scaled offset %lld out of range", (long long)v);
            offs[(size_t)k * D + d] = (int32_t)v;
        }

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int ncol = D + 1;
    const int64_t G = gsc_kmap_groups(n_out);
    char* w = reinterpret_cast<char*>(ws);
    int32_t* d_offs = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * D * sizeof(int32_t));
    int64_t* res = reinterpret_cast<int64_t*>(w);   // res[0] = total, res[1] = header error
    w += align256(2 * sizeof(int64_t));
    int32_t* cnt = reinterpret_cast<int32_t*>(w);
    w += align256((size_t)K * G * sizeof(int32_t));
    void* scan_ws = w;

    GSC_HIP(hipMemcpyAsync(d_offs, offs.data(), offs.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
    GSC_HIP(hipMemsetAsync(res, 0, 2 * sizeof(int64_t), s));
    const unsigned nblk = (unsigned)((n_out + kThreads - 1) / kThreads);
    if (nblk > 0) {
        hipLaunchKernelGGL(k_kmap_count, dim3(nblk), dim3(kThreads), 0, s, in_table, out_coords, n_out, ncol, d_offs,
                           K, G, cnt, res + 1);
        GSC_LAUNCH_CHECK();
    }
    int rc = scan_counts(cnt, K * G, gidx, res, scan_ws, s);
    if (rc) return rc;
    hipLaunchKernelGGL(k_seg_from_gidx, dim3((unsigned)((K + 1 + 255) / 256)), dim3(256), 0, s, gidx, K, G, seg);
    GSC_LAUNCH_CHECK();
    int64_t hres[2];
    GSC_HIP(hipMemcpyAsync(hres, res, sizeof(hres), hipMemcpyDeviceToHost, s));
    GSC_HIP(hipStreamSynchronize(s));
    if (hres[1]) return fail(GSC_EINVAL, "kernel_map: in_table is not a valid table of %d-column rows", ncol);
    *n_pairs = hres[0];
    if (hres[0] > cap_pairs)
        return fail(GSC_ESHORT, "kernel_map: %lld pairs exceed cap_pairs=%lld", (long long)hres[0],
                    (long long)cap_pairs);
    if (nblk > 0 && hres[0] > 0) {
        hipLaunchKernelGGL(k_kmap_fill, dim3(nblk), dim3(kThreads), 0, s, in_table, out_coords, n_out, ncol, d_offs,
                           K, G, gidx, in_idx, out_idx);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

}  // extern "C"
