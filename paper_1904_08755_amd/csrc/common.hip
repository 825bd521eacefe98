// Error plumbing and the device-wide exclusive scan used by the coordinate
// and kernel-map stages.
#include <cstdarg>
#include <cstdio>

#include "gsc_internal.h"

namespace gsc {

static thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = '\0'; }

// ---------------------------------------------------------------------------
// scan: 256 threads x 8 elements per block
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 256;
constexpr int kScanPer = 8;
constexpr int kScanTile = kScanThreads * kScanPer;

// inclusive wave scan (wave64) of a 64-bit value
__device__ __forceinline__ int64_t wave_inclusive(int64_t v) {
    const int l = __lane_id();
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int64_t t = __shfl_up(v, d, 64);
        if (l >= d) v += t;
    }
    return v;
}

// exclusive block scan of one value per thread; returns the block total in *tot
__device__ __forceinline__ int64_t block_exclusive(int64_t v, int64_t* sh, int64_t* tot) {
    const int w = threadIdx.x >> 6, l = __lane_id();
    int64_t inc = wave_inclusive(v);
    if (l == 63) sh[w] = inc;
    __syncthreads();
    int64_t base = 0, all = 0;
    for (int i = 0; i < kScanThreads / 64; ++i) {
        if (i < w) base += sh[i];
        all += sh[i];
    }
    __syncthreads();
    *tot = all;
    return base + inc - v;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_reduce(const int32_t* cnt, int64_t m, int64_t* part) {
    __shared__ int64_t sh[kScanThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i)
        if (base + i < m) s += cnt[base + i];
    int64_t tot;
    block_exclusive(s, sh, &tot);
    if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

// single block: exclusive scan of the per-tile partials, in place
__global__ void __launch_bounds__(kScanThreads) k_scan_partials(int64_t* part, int64_t nb, int64_t* out_total_a,
                                                                int64_t* out_total_b) {
    __shared__ int64_t sh[kScanThreads / 64];
    int64_t carry = 0;
    for (int64_t b0 = 0; b0 < nb; b0 += kScanThreads) {
        const int64_t i = b0 + threadIdx.x;
        int64_t v = i < nb ? part[i] : 0;
        int64_t tot;
        int64_t ex = block_exclusive(v, sh, &tot);
        if (i < nb) part[i] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) {
        if (out_total_a) *out_total_a = carry;
        if (out_total_b) *out_total_b = carry;
    }
}

__global__ void __launch_bounds__(kScanThreads) k_scan_down(const int32_t* cnt, int64_t m, const int64_t* part,
                                                            int64_t* out) {
    __shared__ int64_t sh[kScanThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
    int64_t v[kScanPer];
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        v[i] = base + i < m ? cnt[base + i] : 0;
        s += v[i];
    }
    int64_t tot;
    int64_t run = part[blockIdx.x] + block_exclusive(s, sh, &tot);
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        if (base + i < m) out[base + i] = run;
        run += v[i];
    }
}

size_t scan_ws_bytes(int64_t m) {
    const int64_t nb = (m + kScanTile - 1) / kScanTile;
    return (size_t)((nb > 0 ? nb : 1) * sizeof(int64_t) + 256);
}

int scan_counts(const int32_t* cnt, int64_t m, int64_t* out, int64_t* total_out, void* ws, hipStream_t s) {
    int64_t* part = reinterpret_cast<int64_t*>(ws);
    const int64_t nb = (m + kScanTile - 1) / kScanTile;
    if (nb > 0) {
        hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, s, cnt, m, part);
        GSC_LAUNCH_CHECK();
    }
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kScanThreads), 0, s, part, nb, out + m, total_out);
    GSC_LAUNCH_CHECK();
    if (nb > 0) {
        hipLaunchKernelGGL(k_scan_down, dim3((unsigned)nb), dim3(kScanThreads), 0, s, cnt, m, part, out);
        GSC_LAUNCH_CHECK();
    }
    return GSC_OK;
}

}  // namespace gsc

extern "C" {

const char* gsc_last_error(void) { return gsc::g_err; }

int gsc_abi_version(void) { return 1; }

}  // extern "C"
