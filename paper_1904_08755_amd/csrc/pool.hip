// Pooling over a kernel map (Sec. 4.3 max pooling, Alg. 3; Sec. 4.4 average
// and sum pooling, Alg. 4) and global pooling, fp32.
//
// The paper sorts the pairs by output row and reduces segments (max) or
// multiplies by the map's sparse 0/1 matrix (average, sum).  Here the map's
// dense form nbr[k][j] (the input row paired with output j at offset k, or
// -1, as the kernel map writes it) already lists every output's inputs in
// offset order, so the forward pass is output-stationary with no sort: one
// lane per (output row, channel), consecutive lanes on consecutive channels
// of a row (coalesced feature rows, the row's neighbour entries shared; four
// channels per lane when C is a multiple of 4).  The
// backward pass is input-stationary over the role-reversed map's dense form,
// so every input gradient is a sum in a fixed order (no atomics).
//
// Global pooling maps every row of batch b to output b: per-chunk partial
// reductions in LDS, then one ordered pass over the chunks.
#include <cfloat>

#include "gsc_internal.h"

namespace gsc {

namespace {

constexpr int kPoolThreads = 256;
constexpr int kPoolBatch = 8;            // neighbour entries loaded together per lane
constexpr int kGlobalChunk = 256;        // rows per partial of global pooling
constexpr int kGlobalMaxBatch = 32;      // batch indices of global pooling
constexpr int kGlobalChan = 256;         // channels per partial pass (one per thread)

unsigned blocks_for(int64_t n, int64_t per = kPoolThreads) {
    const int64_t g = (n + per - 1) / per;
    return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

// Forward: lane (j, c).  Inputs of output j are visited in offset order; max
// keeps the first input attaining the maximum (strict comparison).
__global__ void __launch_bounds__(kPoolThreads) k_pool_fwd(int mode, const float* __restrict__ X, int64_t n_in, int C,
                                                           const int32_t* __restrict__ nbr, int K, int64_t n_out,
                                                           float* __restrict__ Y, int32_t* __restrict__ arg,
                                                           int32_t* __restrict__ cnt) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_out * C) return;
    const int64_t j = t / C;
    const int c = (int)(t - j * C);
    float acc = 0.f;
    int32_t best = -1;
    int32_t n = 0;
    for (int k0 = 0; k0 < K; k0 += kPoolBatch) {
        int32_t r[kPoolBatch];
        float v[kPoolBatch];
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) r[b] = k0 + b < K ? nbr[(int64_t)(k0 + b) * n_out + j] : -1;
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            const bool ok = r[b] >= 0 && r[b] < n_in;
            v[b] = ok ? X[(int64_t)r[b] * C + c] : 0.f;
        }
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            if (!(r[b] >= 0 && r[b] < n_in)) continue;
            ++n;
            if (mode == GSC_POOL_MAX) {
                if (best < 0 || v[b] > acc) {
                    acc = v[b];
                    best = r[b];
                }
            } else {
                acc += v[b];
            }
        }
    }
    if (mode == GSC_POOL_AVG && n > 0) acc = acc / (float)n;
    Y[t] = acc;
    if (arg) arg[t] = best;
    if (cnt && c == 0) cnt[j] = n;
}

// The same with four channels per lane (C a multiple of 4, 16-byte aligned
// rows): one float4 gather per (output, offset), so a 32-channel row takes 8
// lanes and a wave covers 8 outputs.
__global__ void __launch_bounds__(kPoolThreads) k_pool_fwd4(int mode, const float* __restrict__ X, int64_t n_in, int C,
                                                            const int32_t* __restrict__ nbr, int K, int64_t n_out,
                                                            float* __restrict__ Y, int32_t* __restrict__ arg,
                                                            int32_t* __restrict__ cnt) {
    const int nq = C >> 2;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_out * nq) return;
    const int64_t j = t / nq;
    const int q = (int)(t - j * nq);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    int4 best = make_int4(-1, -1, -1, -1);
    int32_t n = 0;
    for (int k0 = 0; k0 < K; k0 += kPoolBatch) {
        int32_t r[kPoolBatch];
        float4 v[kPoolBatch];
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) r[b] = k0 + b < K ? nbr[(int64_t)(k0 + b) * n_out + j] : -1;
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            const bool ok = r[b] >= 0 && r[b] < n_in;
            v[b] = ok ? reinterpret_cast<const float4*>(X + (int64_t)r[b] * C)[q] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            if (!(r[b] >= 0 && r[b] < n_in)) continue;
            ++n;
            if (mode == GSC_POOL_MAX) {
                if (best.x < 0 || v[b].x > acc.x) { acc.x = v[b].x; best.x = r[b]; }
                if (best.y < 0 || v[b].y > acc.y) { acc.y = v[b].y; best.y = r[b]; }
                if (best.z < 0 || v[b].z > acc.z) { acc.z = v[b].z; best.z = r[b]; }
                if (best.w < 0 || v[b].w > acc.w) { acc.w = v[b].w; best.w = r[b]; }
            } else {
                acc.x += v[b].x;
                acc.y += v[b].y;
                acc.z += v[b].z;
                acc.w += v[b].w;
            }
        }
    }
    if (mode == GSC_POOL_AVG && n > 0) {
        const float fn = (float)n;
        acc = make_float4(acc.x / fn, acc.y / fn, acc.z / fn, acc.w / fn);
    }
    reinterpret_cast<float4*>(Y)[t] = acc;
    if (arg) reinterpret_cast<int4*>(arg)[t] = best;
    if (cnt && q == 0) cnt[j] = n;
}

// Backward: lane (i, c); nbrT[k][i] = the output that input i feeds at offset k.
__global__ void __launch_bounds__(kPoolThreads) k_pool_bwd(int mode, const float* __restrict__ dY, int64_t n_out,
                                                           int C, const int32_t* __restrict__ nbrT, int K,
                                                           int64_t n_in, const int32_t* __restrict__ arg,
                                                           const int32_t* __restrict__ cnt, float* __restrict__ dX) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_in * C) return;
    const int64_t i = t / C;
    const int c = (int)(t - i * C);
    float acc = 0.f;
    for (int k0 = 0; k0 < K; k0 += kPoolBatch) {
        int32_t o[kPoolBatch];
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) o[b] = k0 + b < K ? nbrT[(int64_t)(k0 + b) * n_in + i] : -1;
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            if (!(o[b] >= 0 && o[b] < n_out)) continue;
            const int64_t e = (int64_t)o[b] * C + c;
            if (mode == GSC_POOL_MAX) {
                if (arg[e] == (int32_t)i) acc += dY[e];
            } else if (mode == GSC_POOL_AVG) {
                const int32_t n = cnt[o[b]];
                if (n > 0) acc += dY[e] / (float)n;
            } else {
                acc += dY[e];
            }
        }
    }
    dX[t] = acc;
}

// Global pooling, pass 1: partial[chunk][b][c] over rows of one chunk (in row
// order), channels [c0, c0 + kGlobalChan) of this launch, one per thread.
__global__ void __launch_bounds__(kGlobalChan) k_gpool_partial(int mode, const float* __restrict__ X, int64_t n,
                                                               int C, int c0, const int32_t* __restrict__ coords,
                                                               int ncol, int n_batch, float* __restrict__ pval,
                                                               int32_t* __restrict__ parg, int32_t* __restrict__ pcnt) {
    __shared__ int32_t bat[kGlobalChunk];
    const int64_t r0 = (int64_t)blockIdx.x * kGlobalChunk;
    const int nr = (int)min((int64_t)kGlobalChunk, n - r0);
    for (int i = threadIdx.x; i < nr; i += blockDim.x) bat[i] = coords[(r0 + i) * ncol];
    __syncthreads();
    const int c = c0 + (int)threadIdx.x;
    float val[kGlobalMaxBatch];
    int32_t best[kGlobalMaxBatch];
#pragma unroll
    for (int b = 0; b < kGlobalMaxBatch; ++b) {
        val[b] = 0.f;
        best[b] = -1;
    }
    if (c < C) {
        for (int i = 0; i < nr; ++i) {
            const int b = bat[i];
            if (b < 0 || b >= n_batch) continue;
            const float v = X[(r0 + i) * C + c];
#pragma unroll
            for (int bb = 0; bb < kGlobalMaxBatch; ++bb) {
                if (bb != b) continue;
                if (mode == GSC_POOL_MAX) {
                    if (best[bb] < 0 || v > val[bb]) {
                        val[bb] = v;
                        best[bb] = (int32_t)(r0 + i);
                    }
                } else {
                    val[bb] += v;
                    best[bb] = 0;
                }
            }
        }
#pragma unroll
        for (int b = 0; b < kGlobalMaxBatch; ++b) {
            if (b >= n_batch) break;
            const int64_t e = ((int64_t)blockIdx.x * n_batch + b) * C + c;
            pval[e] = val[b];
            parg[e] = best[b];
        }
    }
    if (c0 == 0 && threadIdx.x < n_batch) {   // rows of each batch index in this chunk
        int32_t m = 0;
        for (int i = 0; i < nr; ++i) m += bat[i] == (int)threadIdx.x;
        pcnt[(int64_t)blockIdx.x * n_batch + threadIdx.x] = m;
    }
}

// Global pooling, pass 2: lane (b, c) combines the chunks in order.
__global__ void __launch_bounds__(kPoolThreads) k_gpool_final(int mode, int64_t nchunk, int C, int n_batch,
                                                              const float* __restrict__ pval,
                                                              const int32_t* __restrict__ parg,
                                                              const int32_t* __restrict__ pcnt, float* __restrict__ Y,
                                                              int32_t* __restrict__ arg, int32_t* __restrict__ cnt) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_batch * C) return;
    const int b = (int)(t / C), c = (int)(t - (int64_t)b * C);
    float acc = 0.f;
    int32_t best = -1;
    int64_t n = 0;
    for (int64_t q = 0; q < nchunk; ++q) {
        const int64_t e = (q * n_batch + b) * C + c;
        n += pcnt[q * n_batch + b];
        const int32_t a = parg[e];
        if (a < 0) continue;   // no row of b in this chunk
        const float v = pval[e];
        if (mode == GSC_POOL_MAX) {
            if (best < 0 || v > acc) {
                acc = v;
                best = a;
            }
        } else {
            acc += v;
        }
    }
    if (mode == GSC_POOL_AVG && n > 0) acc = acc / (float)n;
    Y[t] = acc;
    if (arg) arg[t] = mode == GSC_POOL_MAX ? best : -1;
    if (cnt && c == 0) cnt[b] = (int32_t)n;
}

// Global pooling backward: lane (i, c).
__global__ void __launch_bounds__(kPoolThreads) k_gpool_bwd(int mode, const float* __restrict__ dY, int n_batch, int C,
                                                            const int32_t* __restrict__ coords, int ncol, int64_t n,
                                                            const int32_t* __restrict__ arg,
                                                            const int32_t* __restrict__ cnt, float* __restrict__ dX) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n * C) return;
    const int64_t i = t / C;
    const int c = (int)(t - i * C);
    const int b = coords[i * ncol];
    float g = 0.f;
    if (b >= 0 && b < n_batch) {
        const int64_t e = (int64_t)b * C + c;
        if (mode == GSC_POOL_MAX)
            g = arg[e] == (int32_t)i ? dY[e] : 0.f;
        else if (mode == GSC_POOL_AVG)
            g = cnt[b] > 0 ? dY[e] / (float)cnt[b] : 0.f;
        else
            g = dY[e];
    }
    dX[t] = g;
}

// Backward with four channels per lane.
__global__ void __launch_bounds__(kPoolThreads) k_pool_bwd4(int mode, const float* __restrict__ dY, int64_t n_out,
                                                            int C, const int32_t* __restrict__ nbrT, int K,
                                                            int64_t n_in, const int32_t* __restrict__ arg,
                                                            const int32_t* __restrict__ cnt, float* __restrict__ dX) {
    const int nq = C >> 2;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_in * nq) return;
    const int64_t i = t / nq;
    const int q = (int)(t - i * nq);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k0 = 0; k0 < K; k0 += kPoolBatch) {
        int32_t o[kPoolBatch];
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) o[b] = k0 + b < K ? nbrT[(int64_t)(k0 + b) * n_in + i] : -1;
#pragma unroll
        for (int b = 0; b < kPoolBatch; ++b) {
            if (!(o[b] >= 0 && o[b] < n_out)) continue;
            const int64_t e = (int64_t)o[b] * nq + q;
            const float4 g = reinterpret_cast<const float4*>(dY)[e];
            if (mode == GSC_POOL_MAX) {
                const int4 a = reinterpret_cast<const int4*>(arg)[e];
                const int32_t ii = (int32_t)i;
                acc.x += a.x == ii ? g.x : 0.f;
                acc.y += a.y == ii ? g.y : 0.f;
                acc.z += a.z == ii ? g.z : 0.f;
                acc.w += a.w == ii ? g.w : 0.f;
            } else if (mode == GSC_POOL_AVG) {
                const int32_t n = cnt[o[b]];
                if (n > 0) {
                    const float fn = (float)n;
                    acc.x += g.x / fn;
                    acc.y += g.y / fn;
                    acc.z += g.z / fn;
                    acc.w += g.w / fn;
                }
            } else {
                acc.x += g.x;
                acc.y += g.y;
                acc.z += g.z;
                acc.w += g.w;
            }
        }
    }
    reinterpret_cast<float4*>(dX)[t] = acc;
}

static bool aligned16(const void* p) { return p == nullptr || ((uintptr_t)p & 15) == 0; }

static size_t al256(size_t b) { return (b + 255) & ~(size_t)255; }

static bool mode_ok(int mode) { return mode == GSC_POOL_MAX || mode == GSC_POOL_AVG || mode == GSC_POOL_SUM; }

}  // namespace gsc

using namespace gsc;

extern "C" {

int gsc_sparse_pool_fwd(int32_t mode, const float* X, int64_t n_in, int32_t C, const int32_t* nbr, int32_t K,
                        int64_t n_out, float* Y, int32_t* arg, int32_t* cnt, void* stream) {
    clear_error();
    if (!mode_ok(mode)) return fail(GSC_EINVAL, "pool_fwd: mode=%d", mode);
    if (C < 1 || K < 1 || n_in < 0 || n_out < 0) return fail(GSC_EINVAL, "pool_fwd: bad sizes");
    if (n_out * (int64_t)C > ((int64_t)1 << 40)) return fail(GSC_EINVAL, "pool_fwd: output too large");
    if (n_out == 0) return GSC_OK;
    if (!nbr || !Y || (n_in > 0 && !X)) return fail(GSC_EINVAL, "pool_fwd: null X/nbr/Y");
    if (mode == GSC_POOL_MAX && !arg) return fail(GSC_EINVAL, "pool_fwd: max pooling needs arg");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (C % 4 == 0 && aligned16(X) && aligned16(Y) && aligned16(arg))
        hipLaunchKernelGGL(k_pool_fwd4, dim3(blocks_for(n_out * (C / 4))), dim3(kPoolThreads), 0, s, (int)mode, X,
                           n_in, (int)C, nbr, (int)K, n_out, Y, arg, cnt);
    else
        hipLaunchKernelGGL(k_pool_fwd, dim3(blocks_for(n_out * C)), dim3(kPoolThreads), 0, s, (int)mode, X, n_in,
                           (int)C, nbr, (int)K, n_out, Y, arg, cnt);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

int gsc_sparse_pool_bwd(int32_t mode, const float* dY, int64_t n_out, int32_t C, const int32_t* nbrT, int32_t K,
                        int64_t n_in, const int32_t* arg, const int32_t* cnt, float* dX, void* stream) {
    clear_error();
    if (!mode_ok(mode)) return fail(GSC_EINVAL, "pool_bwd: mode=%d", mode);
    if (C < 1 || K < 1 || n_in < 0 || n_out < 0) return fail(GSC_EINVAL, "pool_bwd: bad sizes");
    if (n_in == 0) return GSC_OK;
    if (!nbrT || !dX || (n_out > 0 && !dY)) return fail(GSC_EINVAL, "pool_bwd: null dY/nbrT/dX");
    if (mode == GSC_POOL_MAX && !arg) return fail(GSC_EINVAL, "pool_bwd: max pooling needs arg");
    if (mode == GSC_POOL_AVG && !cnt) return fail(GSC_EINVAL, "pool_bwd: average pooling needs cnt");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (C % 4 == 0 && aligned16(dY) && aligned16(dX) && aligned16(arg))
        hipLaunchKernelGGL(k_pool_bwd4, dim3(blocks_for(n_in * (C / 4))), dim3(kPoolThreads), 0, s, (int)mode, dY,
                           n_out, (int)C, nbrT, (int)K, n_in, arg, cnt, dX);
    else
        hipLaunchKernelGGL(k_pool_bwd, dim3(blocks_for(n_in * C)), dim3(kPoolThreads), 0, s, (int)mode, dY, n_out,
                           (int)C, nbrT, (int)K, n_in, arg, cnt, dX);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

size_t gsc_global_pool_ws_bytes(int64_t n, int32_t C, int32_t n_batch) {
    if (n < 0 || C < 1 || n_batch < 1) return 0;
    const int64_t nchunk = (n + kGlobalChunk - 1) / kGlobalChunk;
    const int64_t e = nchunk * n_batch * C;
    return al256((size_t)e * sizeof(float)) + al256((size_t)e * sizeof(int32_t)) +
           al256((size_t)nchunk * n_batch * sizeof(int32_t)) + 256;
}

int gsc_global_pool_fwd(int32_t mode, const float* X, int64_t n, int32_t C, const int32_t* coords, int32_t D,
                        int32_t n_batch, float* Y, int32_t* arg, int32_t* cnt, void* ws, size_t ws_bytes,
                        void* stream) {
    clear_error();
    if (!mode_ok(mode)) return fail(GSC_EINVAL, "global_pool_fwd: mode=%d", mode);
    if (C < 1 || n < 0 || D < 1 || D + 1 > kMaxCols) return fail(GSC_EINVAL, "global_pool_fwd: bad sizes");
    if (n_batch < 1 || n_batch > kGlobalMaxBatch)
        return fail(GSC_EINVAL, "global_pool_fwd: n_batch=%d outside [1,%d]", n_batch, kGlobalMaxBatch);
    if (!Y || !ws || (n > 0 && (!X || !coords))) return fail(GSC_EINVAL, "global_pool_fwd: null pointer");
    if (mode == GSC_POOL_MAX && !arg) return fail(GSC_EINVAL, "global_pool_fwd: max pooling needs arg");
    const size_t need = gsc_global_pool_ws_bytes(n, C, n_batch);
    if (ws_bytes < need) return fail(GSC_ESHORT, "global_pool_fwd: ws needs %zu bytes, got %zu", need, ws_bytes);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t nchunk = (n + kGlobalChunk - 1) / kGlobalChunk;
    const int64_t e = nchunk * n_batch * C;
    char* w = reinterpret_cast<char*>(ws);
    float* pval = reinterpret_cast<float*>(w);
    w += al256((size_t)e * sizeof(float));
    int32_t* parg = reinterpret_cast<int32_t*>(w);
    w += al256((size_t)e * sizeof(int32_t));
    int32_t* pcnt = reinterpret_cast<int32_t*>(w);
    for (int c0 = 0; c0 < C && nchunk > 0; c0 += kGlobalChan) {
        hipLaunchKernelGGL(k_gpool_partial, dim3((unsigned)nchunk), dim3(kGlobalChan), 0, s, (int)mode, X, n, (int)C, c0,
                           coords, (int)(D + 1), (int)n_batch, pval, parg, pcnt);
        GSC_LAUNCH_CHECK();
    }
    hipLaunchKernelGGL(k_gpool_final, dim3(blocks_for((int64_t)n_batch * C)), dim3(kPoolThreads), 0, s, (int)mode,
                       nchunk, (int)C, (int)n_batch, pval, parg, pcnt, Y, arg, cnt);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

int gsc_global_pool_bwd(int32_t mode, const float* dY, int32_t n_batch, int32_t C, const int32_t* coords, int32_t D,
                        int64_t n, const int32_t* arg, const int32_t* cnt, float* dX, void* stream) {
    clear_error();
    if (!mode_ok(mode)) return fail(GSC_EINVAL, "global_pool_bwd: mode=%d", mode);
    if (C < 1 || n < 0 || D < 1 || D + 1 > kMaxCols || n_batch < 1)
        return fail(GSC_EINVAL, "global_pool_bwd: bad sizes");
    if (n == 0) return GSC_OK;
    if (!dY || !coords || !dX) return fail(GSC_EINVAL, "global_pool_bwd: null pointer");
    if (mode == GSC_POOL_MAX && !arg) return fail(GSC_EINVAL, "global_pool_bwd: max pooling needs arg");
    if (mode == GSC_POOL_AVG && !cnt) return fail(GSC_EINVAL, "global_pool_bwd: average pooling needs cnt");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_gpool_bwd, dim3(blocks_for(n * C)), dim3(kPoolThreads), 0, s, (int)mode, dY, (int)n_batch,
                       (int)C, coords, (int)(D + 1), n, arg, cnt, dX);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

}  // extern "C"
