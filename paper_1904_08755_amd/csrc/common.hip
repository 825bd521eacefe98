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

// Single-block scan of up to kScanSingleMax counts (one tile: 1024 threads x
// 8 contiguous counts each), for small scans where a launch matters more
// than the bandwidth.
constexpr int kScanSingleThreads = 1024;
constexpr int kScanSingleE = 8;
constexpr int64_t kScanSingleMax = (int64_t)kScanSingleThreads * kScanSingleE;

__global__ void __launch_bounds__(kScanSingleThreads) k_scan_single(const int32_t* __restrict__ cnt, int64_t m,
                                                                    int64_t* __restrict__ out,
                                                                    int64_t* __restrict__ total_out,
                                                                    int64_t* __restrict__ every_out, int64_t every) {
    __shared__ int64_t sh[kScanSingleThreads / 64];
    const int t = threadIdx.x, w = t >> 6, l = __lane_id();
    const int64_t b = (int64_t)t * kScanSingleE;
    int32_t v[kScanSingleE];
#pragma unroll
    for (int i = 0; i < kScanSingleE; ++i) v[i] = b + i < m ? cnt[b + i] : 0;
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanSingleE; ++i) s += v[i];
    const int64_t inc = wave_inclusive(s);
    if (l == 63) sh[w] = inc;
    __syncthreads();
    int64_t base = 0, all = 0;
    for (int i = 0; i < kScanSingleThreads / 64; ++i) {
        if (i < w) base += sh[i];
        all += sh[i];
    }
    int64_t run = base + inc - s;
    int64_t nxt = every_out ? (b + every - 1) / every * every : -1;   // next index to copy to every_out
#pragma unroll
    for (int i = 0; i < kScanSingleE; ++i) {
        if (b + i < m) {
            out[b + i] = run;
            if (b + i == nxt) {
                every_out[nxt / every] = run;
                nxt += every;
            }
        }
        run += v[i];
    }
    if (t == 0) {
        out[m] = all;
        if (total_out) *total_out = all;
        if (every_out) every_out[m / every] = all;
    }
}

// Second pass of the two-kernel scan: block b adds up the tile sums of the
// blocks before it (a block-wide reduction over at most nb values, read from
// L2), then scans its own tile.  The last block also writes the total.
__global__ void __launch_bounds__(kScanThreads) k_scan_down2(const int32_t* __restrict__ cnt, int64_t m,
                                                             const int64_t* __restrict__ part, int64_t nb,
                                                             int64_t* __restrict__ out, int64_t* __restrict__ total_out,
                                                             int64_t* __restrict__ every_out, int64_t every) {
    __shared__ int64_t sh[kScanThreads / 64];
    __shared__ int64_t carry_sh;
    const int w = threadIdx.x >> 6, l = __lane_id();
    int64_t c = 0;
    for (int64_t i = threadIdx.x; i < (int64_t)blockIdx.x; i += kScanThreads) c += part[i];
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) c += __shfl_xor(c, d, 64);
    if (l == 0) sh[w] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int i = 0; i < kScanThreads / 64; ++i) t += sh[i];
        carry_sh = t;
    }
    __syncthreads();
    const int64_t carry = carry_sh;
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
    int64_t v[kScanPer];
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        v[i] = base + i < m ? cnt[base + i] : 0;
        s += v[i];
    }
    int64_t tot;
    int64_t run = carry + block_exclusive(s, sh, &tot);
    int64_t nxt = every_out ? (base + every - 1) / every * every : -1;   // next index to copy to every_out
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        if (base + i < m) {
            out[base + i] = run;
            if (base + i == nxt) {
                every_out[nxt / every] = run;
                nxt += every;
            }
        }
        run += v[i];
    }
    if (blockIdx.x == nb - 1 && threadIdx.x == 0) {
        out[m] = carry + tot;
        if (total_out) *total_out = carry + tot;
        if (every_out) every_out[m / every] = carry + tot;
    }
}

__global__ void k_zero_i64(int64_t* p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = 0;
}

__global__ void k_seg_from_gidx(const int64_t* gidx, int K, int64_t G, int64_t* seg) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k <= K) seg[k] = gidx[(int64_t)k * G];
}

int seg_from_gidx(const int64_t* gidx, int K, int64_t G, int64_t* seg, hipStream_t s) {
    hipLaunchKernelGGL(k_seg_from_gidx, dim3((unsigned)((K + 1 + 255) / 256)), dim3(256), 0, s, gidx, K, G, seg);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

int device_cus() {
    static int cus[64] = {0};   // per device, read once (a benign race: every writer stores the same value)
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cus[dev] = n;
    }
    return cus[dev];
}

size_t scan_ws_bytes(int64_t m) {
    const int64_t nb = (m + kScanTile - 1) / kScanTile;
    return (size_t)((nb > 0 ? nb : 1) * sizeof(int64_t) + 256);
}

int scan_counts(const int32_t* cnt, int64_t m, int64_t* out, int64_t* total_out, void* ws, hipStream_t s,
                int64_t* every_out, int64_t every) {
    if (every_out && (every <= 0 || m % every != 0)) return fail(GSC_EINVAL, "scan: bad every=%lld", (long long)every);
    if (m <= kScanSingleMax) {
        hipLaunchKernelGGL(k_scan_single, dim3(1), dim3(kScanSingleThreads), 0, s, cnt, m, out, total_out, every_out,
                           every);
        GSC_LAUNCH_CHECK();
        return GSC_OK;
    }
    int64_t* part = reinterpret_cast<int64_t*>(ws);
    const int64_t nb = (m + kScanTile - 1) / kScanTile;
    hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, s, cnt, m, part);
    GSC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_scan_down2, dim3((unsigned)nb), dim3(kScanThreads), 0, s, cnt, m, part, nb, out, total_out,
                       every_out, every);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

}  // namespace gsc

extern "C" {

const char* gsc_last_error(void) { return gsc::g_err; }

int gsc_abi_version(void) { return 1; }

}  // extern "C"
