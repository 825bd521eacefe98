// Large-channel bfloat16 convolution engine (inputs and weights in bfloat16,
// accumulation in fp32): forward / transposed forward / input gradient
// (Alg. 2 and its chain rule) and the weight gradient, on the 16 x 16 x 32
// bf16 MFMA of CDNA4.
//
// Forward and input gradient (k_conv_bf16): output-stationary, like the fp32
// engine, but sized for wide channels.  A workgroup of four waves owns a tile
// of T output rows (T * C_out fp32 = 128 KiB of LDS) and every wave owns a
// quarter of the columns.  The tile's work is a list of items (16 pairs of
// one offset, pairs of one offset being sorted by output row); all four
// waves walk the same list.  For an item a wave gathers the 16 input rows as
// the MFMA A operand straight from global memory (per MFMA step the four
// lane groups of a row load 64 contiguous bytes), multiplies them by its column slice of the
// offset's weight (held in registers for as long as the offset lasts) and
// adds the 16 result rows into the LDS tile.  The tile is rounded to bf16 and
// written once.
//
// The B operand has to hold 8 consecutive reduction channels of one output
// column per lane, so the kernel reads the weights as Bt[w][col][k]
// (C_out x C_in per offset): the input gradient uses W[w] itself (W[w] is
// C_in x C_out, i.e. already column-major for dX = dY W^T), the forward a
// transposed copy made by k_transpose_w.
//
// Weight gradient (k_dw_bf16): split-K over the pairs of each offset.  The
// reduction runs over pairs, so a workgroup stages 32 pairs' rows of X and
// dY in LDS transposed (channel-major) and every lane then reads its 8
// consecutive pairs of one channel with one 16-byte LDS load.
#include "conv_common.h"
#include "conv_bf16.h"

namespace gsc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16_rne(lo) | ((uint32_t)f32_to_bf16_rne(hi) << 16);
}

constexpr int kBfThreads = 256;
constexpr int kBfWaves = kBfThreads / 64;
constexpr int kBfAccFloats = 32768;   // LDS accumulator: T rows x C_out columns of fp32

template <int CA, int CB>
struct BfShape {
    static constexpr int T = kBfAccFloats / CB;      // output rows per tile (128 for C_out = 256)
    static constexpr int TG = T / GSC_GROUP_ROWS;    // kernel-map groups per tile
    static constexpr int AS = CB + 4;                // LDS row stride (floats)
    static constexpr int CW = CB / kBfWaves;         // columns per wave
    static constexpr int NB = CW / 16;               // 16-column MFMA blocks per wave
    static constexpr int KS = CA / 32;               // MFMA steps over the reduction
    static_assert(CA % 32 == 0 && CB % 64 == 0 && NB >= 1, "unsupported shape");
};

// Bt[w][col][k] = W[w][k][col] for a K x rows x cols stack of bf16 matrices:
// a workgroup moves one 64 x 64 tile of one matrix through LDS.  V16: rows
// and cols multiples of 8 and both matrices 16-byte aligned, so the tile is
// read and written 16 bytes (8 elements) per lane; otherwise one element per
// lane.  The padded LDS rows keep the column reads on distinct banks.
// counter (nullable) is set to 0 on the way: the tile engine launched after
// it hands out its tiles with it.
constexpr int kTrTile = 64;
template <bool V16>
__global__ void __launch_bounds__(256) k_transpose_w(const uint16_t* __restrict__ W, int rows, int cols,
                                                     uint16_t* __restrict__ Bt, unsigned* __restrict__ counter) {
    constexpr int P = V16 ? 8 : 2;   // row padding (elements)
    __shared__ __attribute__((aligned(16))) uint16_t tile[kTrTile][kTrTile + P];
    if (counter && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) *counter = 0u;
    const int64_t w = blockIdx.z;
    const int r0 = blockIdx.y * kTrTile, c0 = blockIdx.x * kTrTile;
    const uint16_t* src = W + w * (int64_t)rows * cols;
    uint16_t* dst = Bt + w * (int64_t)rows * cols;
    if constexpr (V16) {
        typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
        for (int i = 0; i < 2; ++i) {   // 512 chunks of 8 elements: row j / 8, columns 8 (j % 8) ..
            const int j = threadIdx.x + 256 * i, r = j >> 3, c = (j & 7) * 8;
            if (r0 + r < rows && c0 + c < cols)
                *reinterpret_cast<u32x4*>(&tile[r][c]) =
                    *reinterpret_cast<const u32x4*>(src + (int64_t)(r0 + r) * cols + c0 + c);
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 2; ++i) {   // output row (column of W) j / 8, elements 8 (j % 8) ..
            const int j = threadIdx.x + 256 * i, c = j >> 3, r = (j & 7) * 8;
            if (c0 + c < cols && r0 + r < rows) {
                uint32_t u[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    u[e] = (uint32_t)tile[r + 2 * e][c] | ((uint32_t)tile[r + 2 * e + 1][c] << 16);
                *reinterpret_cast<u32x4*>(dst + (int64_t)(c0 + c) * rows + r0 + r) = u32x4{u[0], u[1], u[2], u[3]};
            }
        }
    } else {
        const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < kTrTile / 4; ++i) {
            const int r = q + 4 * i;
            if (r0 + r < rows && c0 + lane < cols) tile[r][lane] = src[(int64_t)(r0 + r) * cols + c0 + lane];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kTrTile / 4; ++i) {
            const int c = q + 4 * i;
            if (c0 + c < cols && r0 + lane < rows) dst[(int64_t)(c0 + c) * rows + r0 + lane] = tile[lane][c];
        }
    }
}

// Y[sca[p]] += X[gat[p]] * B_w for the pairs p of every offset, B_w[k][col] =
// Bt[w][col][k], w = sel(offset).  gidx is the map's 64-row group index over
// n_y output positions; when perm is given, position i is output row perm[i].
template <int CA, int CB, typename Sel>
__global__ void __launch_bounds__(kBfThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_conv_bf16(const uint16_t* __restrict__ X, int64_t n_x, const uint16_t* __restrict__ Bt,
            const int32_t* __restrict__ gat, const int32_t* __restrict__ sca, const int64_t* __restrict__ gidx,
            const int32_t* __restrict__ perm, int K, int64_t G, int64_t n_y, uint16_t* __restrict__ Y, Sel sel) {
    using S = BfShape<CA, CB>;
    __shared__ __attribute__((aligned(16))) float acc[S::T * S::AS];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, q = lane >> 4;
    const int64_t tile = tile_unit(blockIdx.x, gridDim.x, perm != nullptr);
    const int64_t g0 = tile * S::TG;
    const int64_t g1 = min(g0 + (int64_t)S::TG, G);
    const int64_t row0 = g0 * GSC_GROUP_ROWS;
    {
        float4* a4 = reinterpret_cast<float4*>(acc);
        for (int i = tid; i < S::T * S::AS / 4; i += kBfThreads) a4[i] = float4{0.f, 0.f, 0.f, 0.f};
    }

    // lane k < K: first pair and pair count of offset k in this tile; items
    // (16 pairs of one offset) are numbered offset by offset
    int64_t lo = 0;
    int np = 0;
    if (lane < K) {
        lo = gidx[(int64_t)lane * G + g0];
        np = (int)(gidx[(int64_t)lane * G + g1] - lo);
    }
    const int nit = (np + 15) >> 4;
    int incl = nit;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int u = __shfl_up(incl, d, 64);
        if (lane >= d) incl += u;
    }
    const int excl = incl - nit;
    const int total = __shfl(incl, 63, 64);
    __syncthreads();   // the tile is zero

    const int colw = wave * S::CW;
    // item -> its offset and the pair of this lane's row (clamped: every
    // address stays valid; lanes past the offset's last pair are masked)
    auto locate = [&](int item, int& k, int32_t& gr, int32_t& sr, bool& ok) {
        k = __popcll(__ballot(incl <= item));
        const int64_t klo = __shfl(lo, k, 64);
        const int knp = __shfl(np, k, 64);
        const int pb = (item - __shfl(excl, k, 64)) * 16 + r16;
        const int64_t p = klo + min(pb, knp - 1);
        gr = gat[p];
        sr = sca[p];
        ok = pb < knp;
    };
    // MFMA step s reduces over channels [32 s, 32 s + 32); lane group q holds
    // channels 32 s + 8 q .. + 8 of its row (A) or column (B), so the four
    // lane groups of a row read 64 contiguous bytes per load
    auto load_a = [&](int32_t gr, bool ok, uint4 (&a)[S::KS]) {
        const uint4* src = reinterpret_cast<const uint4*>(X + (int64_t)(ok ? gr : 0) * CA + 8 * q);
#pragma unroll
        for (int s = 0; s < S::KS; ++s) a[s] = src[4 * s];
    };
    auto load_b = [&](int w, uint4 (&b)[S::NB][S::KS]) {
#pragma unroll
        for (int nb = 0; nb < S::NB; ++nb) {
            const uint4* src =
                reinterpret_cast<const uint4*>(Bt + ((int64_t)w * CB + colw + nb * 16 + r16) * CA + 8 * q);
#pragma unroll
            for (int s = 0; s < S::KS; ++s) b[nb][s] = src[4 * s];
        }
    };

    if (total > 0) {
        int k_c, k_n = 0;
        int32_t gr_c, sr_c, gr_n = 0, sr_n = 0;
        bool ok_c, ok_n = false;
        locate(0, k_c, gr_c, sr_c, ok_c);
        if (total > 1) locate(1, k_n, gr_n, sr_n, ok_n);
        uint4 bc[S::NB][S::KS], bn[S::NB][S::KS];
        uint4 ac[S::KS], an[S::KS];
        load_b(sel(k_c), bc);
        ok_c = ok_c && gr_c >= 0 && gr_c < n_x;
        load_a(gr_c, ok_c, ac);
        for (int it = 0; it < total; ++it) {
            const bool has_n = it + 1 < total;
            const bool new_b = has_n && k_n != k_c;
            // 1. the next item's rows (its indices arrived during this one's
            //    predecessor) and, when its offset differs, its weights
            if (has_n) {
                ok_n = ok_n && gr_n >= 0 && gr_n < n_x;
                load_a(gr_n, ok_n, an);
            }
            if (new_b) load_b(sel(k_n), bn);
            // 2. indices of the item after next
            int k_nn = 0;
            int32_t gr_nn = 0, sr_nn = 0;
            bool ok_nn = false;
            if (it + 2 < total) locate(it + 2, k_nn, gr_nn, sr_nn, ok_nn);
            // 3. 16 rows x CW columns of this item
            floatx4 d[S::NB];
#pragma unroll
            for (int nb = 0; nb < S::NB; ++nb) d[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < S::KS; ++s)
#pragma unroll
                for (int nb = 0; nb < S::NB; ++nb)
                    d[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ac[s]), as_bf16x8(bc[nb][s]), d[nb],
                                                                    0, 0, 0);
            // 4. add into the tile: D row 4q + j is the item's pair row 4q + j
            const int64_t rel = (int64_t)sr_c - row0;
            const int mine = (ok_c && rel >= 0 && rel < S::T) ? (int)rel : -1;
            int lrow[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) lrow[j] = __shfl(mine, 4 * q + j, 64);
            wave_lds_sync();   // rows this wave updated for earlier items
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (lrow[j] >= 0) {
                    float* arow = acc + lrow[j] * S::AS + colw + r16;
#pragma unroll
                    for (int nb = 0; nb < S::NB; ++nb) arow[nb * 16] += d[nb][j];
                }
            }
            // 5. rotate the pipeline
#pragma unroll
            for (int s = 0; s < S::KS; ++s) ac[s] = an[s];
            if (new_b) {
#pragma unroll
                for (int nb = 0; nb < S::NB; ++nb)
#pragma unroll
                    for (int s = 0; s < S::KS; ++s) bc[nb][s] = bn[nb][s];
            }
            k_c = k_n;
            gr_c = gr_n;
            sr_c = sr_n;
            ok_c = ok_n;
            k_n = k_nn;
            gr_n = gr_nn;
            sr_n = sr_nn;
            ok_n = ok_nn;
        }
    }
    __syncthreads();
    // the tile's rows, rounded to bf16 and written once (8 columns per lane)
    constexpr int C8 = CB / 8;
    for (int i = tid; i < S::T * C8; i += kBfThreads) {
        const int r = i / C8, c8 = (i - r * C8) * 8;
        const int64_t pos = row0 + r;
        if (pos < n_y) {
            const int64_t row = perm ? (int64_t)perm[pos] : pos;
            const float4* a = reinterpret_cast<const float4*>(acc + r * S::AS + c8);
            const float4 v0 = a[0], v1 = a[1];
            uint4 o;
            o.x = pack_bf16x2(v0.x, v0.y);
            o.y = pack_bf16x2(v0.z, v0.w);
            o.z = pack_bf16x2(v1.x, v1.y);
            o.w = pack_bf16x2(v1.z, v1.w);
            *reinterpret_cast<uint4*>(Y + row * CB + c8) = o;
        }
    }
}

// ---------------------------------------------------------------------------
// k_conv_bf16_dma: the same computation for reduction width CA and output
// width CB in {128, 256}, with the gathered rows brought into LDS by the load
// units themselves (global_load_lds_dwordx4: each lane's 16 bytes land at
// consecutive LDS addresses), so no register ever waits on a gather.
//
// Per item (16 pairs of one offset) the pipeline runs stages ahead:
//   idx:  a dword DMA per wave copies the item's 16 input rows (gat) and 16
//         output positions (sca) into the wave's index ring, 6 items ahead;
//   rows: 3 items ahead, each wave reads 4 input-row indices from its index
//         ring and DMAs those 4 rows (CA bf16 each) into the shared row ring,
//         16-byte chunks XOR-swizzled by row so the MFMA operand reads spread
//         over the LDS banks;
//   operands: one item ahead, the rows are read from the ring into registers,
//         so an item's MFMAs run while the next item's loads are issued and
//         its operands read.
// The weight slice of the next offset is loaded into the second register
// buffer at the first item of the current offset (offsets alternate between
// the two buffers, so no copies).  Vector-memory waits are explicit: every
// item issues the same loads in the same order, so the number of newer loads
// still allowed in flight is known.  Item bookkeeping is scalar (iterators
// over the tile's offsets), and every LDS read of DMA-filled memory, as well
// as the accumulator read-add-write, is one asm block with one wait.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// s_waitcnt on the vector-memory counter only (vmcnt[3:0] in bits 3:0,
// vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt at their maxima).  Followed by
// a compiler barrier so LDS reads of the data stay after it.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N <= 63, "vmcnt has 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
    asm volatile("" ::: "memory");
}

// Workgroup barrier without the release fence of __syncthreads: that fence
// would wait for every LDS-DMA load in flight (they count as LDS stores).
// Cross-wave LDS hand-offs in the pipeline are covered by the explicit
// vector-memory waits before it; the empty asm keeps the compiler from
// moving LDS accesses across.
__device__ __forceinline__ void barrier_no_fence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// wait until at most min(63, BASE + STEP * m) newer vector loads are in
// flight, m in [0, 4] (the number of weight-slice loads in the window)
template <int BASE, int STEP>
__device__ __forceinline__ void wait_vm_window(int m) {
    constexpr int c0 = BASE, c1 = BASE + STEP < 63 ? BASE + STEP : 63;
    constexpr int c2 = BASE + 2 * STEP < 63 ? BASE + 2 * STEP : 63;
    constexpr int c3 = BASE + 3 * STEP < 63 ? BASE + 3 * STEP : 63;
    constexpr int c4 = BASE + 4 * STEP < 63 ? BASE + 4 * STEP : 63;
    m = __builtin_amdgcn_readfirstlane(m);
    if (m <= 0) wait_vm<c0>();
    else if (m == 1) wait_vm<c1>();
    else if (m == 2) wait_vm<c2>();
    else if (m == 3) wait_vm<c3>();
    else wait_vm<c4>();
}

// wait until at most n newer vector loads are in flight (n clamped to
// [0, 63]; a runtime value, so the immediate is picked by a switch)
__device__ __forceinline__ void wait_vm_dyn(int n) {
    n = __builtin_amdgcn_readfirstlane(n);
    n = n < 0 ? 0 : (n > 63 ? 63 : n);
    switch (n) {
#define GSC_WV(c) case c: wait_vm<c>(); break;
#define GSC_WV8(c) GSC_WV(c) GSC_WV(c + 1) GSC_WV(c + 2) GSC_WV(c + 3) GSC_WV(c + 4) GSC_WV(c + 5) GSC_WV(c + 6) GSC_WV(c + 7)
        GSC_WV8(0) GSC_WV8(8) GSC_WV8(16) GSC_WV8(24) GSC_WV8(32) GSC_WV8(40) GSC_WV8(48) GSC_WV8(56)
#undef GSC_WV8
#undef GSC_WV
        default: wait_vm<0>();
    }
}

// LDS reads of memory the DMA loads fill.  The compiler cannot tell which
// in-flight DMA an LDS read depends on and would wait for all of them before
// every read; these reads are issued from inline asm instead (each call
// waits for its own LDS results), and the pipeline's explicit vector-memory
// waits order them after the DMA they depend on.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_off(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ int32_t lds_read_i32(const void* p) {
    int32_t v;
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(lds_off(p)) : "memory");
    return v;
}

constexpr int kRowRing = 3;   // items of gathered rows in LDS
constexpr int kIdxRing = 8;   // items of indices per wave (the index copy runs 5 items ahead)

template <int CA, int CB>
struct DmaShape {
    static constexpr int T = 128;                 // output positions per tile
    static constexpr int TG = T / GSC_GROUP_ROWS;
    static constexpr int NC = CA / 8;             // 16-byte chunks per row
    static constexpr int CW = CB / kBfWaves;      // columns per wave
    static constexpr int NB = CW / 16;
    static constexpr int KS = CA / 32;
    static constexpr int DPW = CA / 128;          // row DMAs (1 KiB each) per wave per item
    static constexpr int SLOT = 16 * CA * 2;      // bytes of one item's rows
    static constexpr int BL = NB * KS;            // weight loads per wave per offset
    static_assert((CA == 128 || CA == 256) && (CB == 128 || CB == 256), "unsupported shape");
};

// Iterator over the items of a tile (offset by offset, 16 pairs each); all
// fields are wave-uniform.  Past the last item it stays on the last item, so
// the loads issued for items past the end repeat it and keep the pattern of
// loads per item fixed.
struct ItemIter {
    unsigned long long om;   // nonempty offsets after the current one
    int k;                   // current offset
    int knp;                 // its pairs in the tile
    int t;                   // item within the offset
    int64_t klo;             // its first pair
    __device__ __forceinline__ int64_t p0() const { return klo + 16 * t; }
    __device__ __forceinline__ int cnt() const { return min(16, knp - 16 * t); }
};

// asm LDS reads of one item's A operands (KS x 16 bytes) and of the output
// position of the lane's pair, with a single wait
template <int KS>
__device__ __forceinline__ void lds_read_item(const uint32_t (&ad)[KS], uint32_t pos_ad, u32x4 (&a)[KS],
                                              int32_t& pos);

template <>
__device__ __forceinline__ void lds_read_item<4>(const uint32_t (&ad)[4], uint32_t pos_ad, u32x4 (&a)[4],
                                                 int32_t& pos) {
    asm volatile(
        "ds_read_b128 %0, %5\n\tds_read_b128 %1, %6\n\tds_read_b128 %2, %7\n\tds_read_b128 %3, %8\n\t"
        "ds_read_b32 %4, %9\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3]), "=&v"(pos)
        : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(pos_ad)
        : "memory");
}

template <>
__device__ __forceinline__ void lds_read_item<8>(const uint32_t (&ad)[8], uint32_t pos_ad, u32x4 (&a)[8],
                                                 int32_t& pos) {
    asm volatile(
        "ds_read_b128 %0, %9\n\tds_read_b128 %1, %10\n\tds_read_b128 %2, %11\n\tds_read_b128 %3, %12\n\t"
        "ds_read_b128 %4, %13\n\tds_read_b128 %5, %14\n\tds_read_b128 %6, %15\n\tds_read_b128 %7, %16\n\t"
        "ds_read_b32 %8, %17\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3]), "=&v"(a[4]), "=&v"(a[5]), "=&v"(a[6]), "=&v"(a[7]),
          "=&v"(pos)
        : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]), "v"(ad[6]), "v"(ad[7]), "v"(pos_ad)
        : "memory");
}

// read-add-write of NB x 4 accumulator floats (one asm wait for the reads)
template <int NB>
__device__ __forceinline__ void lds_accumulate(const uint32_t (&ad)[NB], const floatx4 (&d)[NB]);

template <>
__device__ __forceinline__ void lds_accumulate<2>(const uint32_t (&ad)[2], const floatx4 (&d)[2]) {
    floatx4 v0, v1;
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v0), "=&v"(v1)
                 : "v"(ad[0]), "v"(ad[1])
                 : "memory");
    v0 += d[0];
    v1 += d[1];
    asm volatile("ds_write_b128 %0, %2\n\tds_write_b128 %1, %3" : : "v"(ad[0]), "v"(ad[1]), "v"(v0), "v"(v1) : "memory");
}

template <>
__device__ __forceinline__ void lds_accumulate<4>(const uint32_t (&ad)[4], const floatx4 (&d)[4]) {
    floatx4 v0, v1, v2, v3;
    asm volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v0), "=&v"(v1), "=&v"(v2), "=&v"(v3)
        : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3])
        : "memory");
    v0 += d[0];
    v1 += d[1];
    v2 += d[2];
    v3 += d[3];
    asm volatile("ds_write_b128 %0, %4\n\tds_write_b128 %1, %5\n\tds_write_b128 %2, %6\n\tds_write_b128 %3, %7"
                 :
                 : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(v0), "v"(v1), "v"(v2), "v"(v3)
                 : "memory");
}

template <int CA, int CB, typename Sel>
__global__ void __launch_bounds__(kBfThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_conv_bf16_dma(const uint16_t* __restrict__ X, int64_t n_x, const uint16_t* __restrict__ Bt,
                const int32_t* __restrict__ gat, const int32_t* __restrict__ sca, const int64_t* __restrict__ gidx,
                const int32_t* __restrict__ perm, int K, int64_t G, int64_t n_y, uint16_t* __restrict__ Y, Sel sel) {
    using S = DmaShape<CA, CB>;
    __shared__ __attribute__((aligned(16))) float acc[S::T * CB];
    __shared__ __attribute__((aligned(16))) char rows[kRowRing * S::SLOT];
    __shared__ __attribute__((aligned(16))) int32_t idxr[kBfWaves][kIdxRing][32];
    __shared__ int32_t prow[S::T];   // output row of each position of the tile
    const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, q = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t tile = tile_unit(blockIdx.x, gridDim.x, perm != nullptr);
    const int64_t g0 = tile * S::TG;
    const int64_t g1 = min(g0 + (int64_t)S::TG, G);
    const int64_t row0 = g0 * GSC_GROUP_ROWS;
    if (tid < S::T) {
        const int64_t pos = row0 + tid;
        prow[tid] = pos < n_y ? (perm ? perm[pos] : (int32_t)pos) : 0;
    }
    {
        float4* a4 = reinterpret_cast<float4*>(acc);
        for (int i = tid; i < S::T * CB / 4; i += kBfThreads) a4[i] = float4{0.f, 0.f, 0.f, 0.f};
    }
    int64_t lo = 0;
    int np = 0;
    if (lane < K) {
        lo = gidx[(int64_t)lane * G + g0];
        np = (int)(gidx[(int64_t)lane * G + g1] - lo);
    }
    const int wsel_lane = lane < K ? sel(lane) : 0;   // weight of offset k, held by lane k
    const unsigned long long om0 = __ballot(lane < K && np > 0);
    __syncthreads();   // the tile is zero
    if (om0 != 0) {
        const int colw = wave * S::CW;
        auto iter_begin = [&](ItemIter& it) {
            it.k = __builtin_ctzll(om0);
            it.om = om0 & (om0 - 1);
            it.klo = __shfl(lo, it.k, 64);
            it.knp = __shfl(np, it.k, 64);
            it.t = 0;
        };
        auto iter_next = [&](ItemIter& it) {
            if (16 * (it.t + 1) < it.knp) {
                ++it.t;
            } else if (it.om) {
                it.k = __builtin_ctzll(it.om);
                it.om &= it.om - 1;
                it.klo = __shfl(lo, it.k, 64);
                it.knp = __shfl(np, it.k, 64);
                it.t = 0;
            }
        };
        // idx stage: lanes 0..15 copy the item's input rows, 16..31 its positions
        auto issue_idx = [&](const ItemIter& it, int slot) {
            if (lane < 32) {
                const int e = min(lane & 15, it.cnt() - 1);
                const int32_t* src = (lane < 16 ? gat : sca) + it.p0() + e;
                __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)&idxr[wave][slot][0], 4, 0, 0);
            }
        };
        // rows stage: this wave's 4 rows (4 wave .. 4 wave + 3) of the item
        // whose indices are in idx slot islot, into row slot rslot
        auto issue_rows = [&](int islot, int rslot) {
            const int32_t* ix = &idxr[wave][islot][0];
            char* slot = rows + rslot * S::SLOT;
            int32_t rr[S::DPW];
            if constexpr (S::DPW == 1) {
                rr[0] = lds_read_i32(ix + (64 * wave + lane) / S::NC);
            } else {
                const uint32_t a0 = lds_off(ix + (64 * (2 * wave) + lane) / S::NC);
                const uint32_t a1 = lds_off(ix + (64 * (2 * wave + 1) + lane) / S::NC);
                asm volatile("ds_read_b32 %0, %2\n\tds_read_b32 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                             : "=&v"(rr[0]), "=&v"(rr[1])
                             : "v"(a0), "v"(a1)
                             : "memory");
            }
#pragma unroll
            for (int h = 0; h < S::DPW; ++h) {
                const int i = wave * S::DPW + h;         // 1 KiB block of the slot
                const int P = 64 * i + lane;             // 16-byte chunk of the slot
                const int r = P / S::NC, cs = P % S::NC;
                const int c = cs ^ (r & (S::NC - 1));
                const int32_t row = (rr[h] >= 0 && rr[h] < n_x) ? rr[h] : 0;
                const uint16_t* src = X + (int64_t)row * CA + c * 8;
                __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)(slot + i * 1024), 16, 0, 0);
            }
        };
        // weight slice of offset w: NB x KS 16-byte loads per lane
        auto load_b = [&](int w, uint4 (&b)[S::NB][S::KS]) {
#pragma unroll
            for (int nb = 0; nb < S::NB; ++nb) {
                const uint4* src =
                    reinterpret_cast<const uint4*>(Bt + ((int64_t)w * CB + colw + nb * 16 + r16) * CA + 8 * q);
#pragma unroll
                for (int s = 0; s < S::KS; ++s) b[nb][s] = src[4 * s];
            }
        };
        // A operands of the item in row slot rslot (rows XOR-swizzled) and the
        // position of this lane's pair from idx slot islot
        auto read_item = [&](int rslot, int islot, u32x4 (&a)[S::KS], int32_t& pos) {
            const char* slot = rows + rslot * S::SLOT;
            uint32_t ad[S::KS];
#pragma unroll
            for (int s = 0; s < S::KS; ++s)
                ad[s] = lds_off(slot + r16 * (S::NC * 16) + (((4 * s + q) ^ (r16 & (S::NC - 1))) * 16));
            lds_read_item<S::KS>(ad, lds_off(&idxr[wave][islot][16 + r16]), a, pos);
        };

        ItemIter ii, ir, ic;   // next item to copy indices of, to copy rows of, to compute
        iter_begin(ii);
        iter_begin(ir);
        iter_begin(ic);
        uint4 b0[S::NB][S::KS], b1[S::NB][S::KS];
        load_b(__shfl(wsel_lane, ic.k, 64), b0);   // oldest load of all
        // Steady state, iteration j issues idx(j + 6), then rows(j + 3) once
        // idx(j + 3) has landed, then the next offset's weights if item j
        // starts an offset.  The prologue issues what iterations -6 .. -1
        // would have, in the same order.
        int ji = 0, jr = 0;   // items whose indices / rows have been issued
        for (; ji < 4; ++ji) {
            issue_idx(ii, ji % kIdxRing);
            iter_next(ii);
        }
        wait_vm<3>();                       // idx(0): idx(1..3) may be in flight
        issue_rows(jr % kIdxRing, jr % kRowRing);
        iter_next(ir);
        ++jr;
        issue_idx(ii, ji % kIdxRing);
        iter_next(ii);
        ++ji;
        wait_vm<3 + S::DPW>();              // idx(1): idx(2..4), rows(0)
        issue_rows(jr % kIdxRing, jr % kRowRing);
        iter_next(ir);
        ++jr;
        issue_idx(ii, ji % kIdxRing);
        iter_next(ii);
        ++ji;
        wait_vm<3 + 2 * S::DPW>();          // idx(2): idx(3..5), rows(0..1)
        issue_rows(jr % kIdxRing, jr % kRowRing);
        iter_next(ir);
        ++jr;
        wait_vm<2 + 2 * S::DPW>();          // rows(0): idx(4..5), rows(1..2)
        barrier_no_fence();
        u32x4 a_cur[S::KS], a_nxt[S::KS];
        int32_t pos_cur, pos_nxt;
        read_item(0, 0, a_cur, pos_cur);

        unsigned hist = 0;     // bit t: weights were loaded t iterations ago (bit 0: this one)
        bool t_load = false;   // weight loads issued at the start of the current iteration
        int j = 0;
        auto step = [&](uint4 (&bc)[S::NB][S::KS]) {
            // 1. item j on the matrix cores (its operands are in registers)
            floatx4 d[S::NB];
#pragma unroll
            for (int nb = 0; nb < S::NB; ++nb) d[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < S::KS; ++s)
#pragma unroll
                for (int nb = 0; nb < S::NB; ++nb)
                    d[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(bc[nb][s]),
                                                                    __builtin_bit_cast(bf16x8, a_cur[s]), d[nb], 0,
                                                                    0, 0);
            // 2. loads for the items ahead (a weight slice, if any, was issued
            //    at the start of this iteration, before the MFMAs)
            hist = ((hist << 1) | (t_load ? 1u : 0u)) & 15u;
            t_load = false;
            barrier_no_fence();   // every wave has read item j's rows: its row slot is free
            issue_idx(ii, ji % kIdxRing);
            iter_next(ii);
            ++ji;
            // idx(j + 3) has landed: after it came rows(j..j + 2), idx(j + 4..j + 6) and the
            // weight slices of iterations j - 2..j
            wait_vm_window<3 + 3 * S::DPW, S::BL>(__popc(hist & 7u));
            issue_rows(jr % kIdxRing, jr % kRowRing);
            iter_next(ir);
            ++jr;
            // rows(j + 1) have landed: after them came idx(j + 5..j + 6), rows(j + 2..j + 3)
            // and the weight slices of iterations j - 1..j
            wait_vm_window<2 + 2 * S::DPW, S::BL>(__popc(hist & 3u));
            barrier_no_fence();   // ... for every wave
            // 3. operands of item j + 1 (past the last item: a repeat, unused)
            read_item((j + 1) % kRowRing, (j + 1) % kIdxRing, a_nxt, pos_nxt);
            // 4. add item j into the tile: lane (p, q) holds output columns
            //    4 q .. 4 q + 3 of each 16-column block for pair p
            const int64_t rel = (int64_t)pos_cur - row0;
            if (r16 < ic.cnt() && rel >= 0 && rel < S::T) {
                const float* arow = acc + rel * CB;
                const int sw = ((int)rel & 15) << 2;   // 4-column groups XOR row: an item's rows spread over banks
                uint32_t ad[S::NB];
#pragma unroll
                for (int nb = 0; nb < S::NB; ++nb) ad[nb] = lds_off(arow + ((colw + nb * 16 + 4 * q) ^ sw));
                lds_accumulate<S::NB>(ad, d);
            }
#pragma unroll
            for (int s = 0; s < S::KS; ++s) a_cur[s] = a_nxt[s];
            pos_cur = pos_nxt;
            iter_next(ic);
            ++j;
        };
        // Offsets alternate between the two weight buffers: before the items
        // of an offset, the next offset's slice is loaded into the other
        // buffer (it is first used one offset later).  The item loops are
        // do-while loops, so the compiler can count the loads issued after a
        // slice load on every path to its first use.
        while (true) {
            bool more = ic.om != 0;
            int n = (ic.knp + 15) >> 4;
            if (more) {
                load_b(__builtin_amdgcn_readfirstlane(__shfl(wsel_lane, __builtin_ctzll(ic.om), 64)), b1);
                t_load = true;
            }
            int t = 0;
            do {
                step(b0);
            } while (++t < n);
            if (!more) break;
            more = ic.om != 0;
            n = (ic.knp + 15) >> 4;
            if (more) {
                load_b(__builtin_amdgcn_readfirstlane(__shfl(wsel_lane, __builtin_ctzll(ic.om), 64)), b0);
                t_load = true;
            }
            t = 0;
            do {
                step(b1);
            } while (++t < n);
            if (!more) break;
        }
        wait_vm<0>();   // loads issued for items past the end
    }
    __syncthreads();
    constexpr int C8 = CB / 8;
    for (int i = tid; i < S::T * C8; i += kBfThreads) {
        const int r = i / C8, c8 = (i - r * C8) * 8;
        if (row0 + r < n_y) {
            const int64_t row = prow[r];
            const int sw = (r & 15) << 2;
            const float4 v0 = *reinterpret_cast<const float4*>(acc + r * CB + (c8 ^ sw));
            const float4 v1 = *reinterpret_cast<const float4*>(acc + r * CB + ((c8 + 4) ^ sw));
            uint4 o;
            o.x = pack_bf16x2(v0.x, v0.y);
            o.y = pack_bf16x2(v0.z, v0.w);
            o.z = pack_bf16x2(v1.x, v1.y);
            o.w = pack_bf16x2(v1.z, v1.w);
            *reinterpret_cast<uint4*>(Y + row * CB + c8) = o;
        }
    }
}

// ---------------------------------------------------------------------------
// weight gradient: partial[item][CI][CO] = X[in]^T dY[out] over one chunk of
// one offset's pairs, for one 128 x 128 tile of dW (grid.y = tile).
// ---------------------------------------------------------------------------
constexpr int kDwbTile = 128;
constexpr int kDwbPairs = 32;                 // pairs per stage (one MFMA reduction step)
constexpr int kDwbPS = kDwbPairs + 8;         // LDS stride of a channel row (bf16 elements)

template <int CI, int CO>
__global__ void __launch_bounds__(kBfThreads)
k_dw_bf16(const uint16_t* __restrict__ X, int64_t n_in, const uint16_t* __restrict__ dY, int64_t n_out,
          const int32_t* __restrict__ in_idx, const int32_t* __restrict__ out_idx, const int64_t* __restrict__ seg,
          const int64_t* __restrict__ ibase, const int64_t* __restrict__ chunk, int K, float* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint16_t xt[kDwbTile * kDwbPS];
    __shared__ __attribute__((aligned(16))) uint16_t yt[kDwbTile * kDwbPS];
    if ((int64_t)blockIdx.x >= ibase[K]) return;
    const int64_t item = xcd_unit(blockIdx.x, ibase[K]);
    int k;
    int64_t p_begin, p_end;
    if (!dw_item(ibase, chunk, seg, K, item, &k, &p_begin, &p_end)) return;
    constexpr int NTO = CO / kDwbTile;
    const int ci0 = (blockIdx.y / NTO) * kDwbTile, co0 = (blockIdx.y % NTO) * kDwbTile;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, q = lane >> 4;
    const int wi = wave >> 1, wo = wave & 1;   // 64 x 64 sub-tile of the wave

    // staging map: thread -> pairs (2 pp2, 2 pp2 + 1), channels [8 cc, 8 cc + 8)
    const int pp2 = tid & 15, cc = tid >> 4;
    auto fetch = [&](int64_t p0, uint4 (&xr)[2], uint4 (&yr)[2]) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int64_t p = p0 + 2 * pp2 + h;
            const int64_t pc = p < p_end ? p : p_end - 1;
            int32_t g = in_idx[pc], s = out_idx[pc];
            const bool v = p < p_end && g >= 0 && g < n_in && s >= 0 && s < n_out;
            g = v ? g : 0;
            s = v ? s : 0;
            xr[h] = *reinterpret_cast<const uint4*>(X + (int64_t)g * CI + ci0 + 8 * cc);
            const uint4 t = *reinterpret_cast<const uint4*>(dY + (int64_t)s * CO + co0 + 8 * cc);
            yr[h] = v ? t : uint4{0u, 0u, 0u, 0u};   // a masked pair adds nothing
        }
    };
    auto stage = [&](const uint4 (&xr)[2], const uint4 (&yr)[2]) {
        const uint32_t* x0 = reinterpret_cast<const uint32_t*>(&xr[0]);
        const uint32_t* x1 = reinterpret_cast<const uint32_t*>(&xr[1]);
        const uint32_t* y0 = reinterpret_cast<const uint32_t*>(&yr[0]);
        const uint32_t* y1 = reinterpret_cast<const uint32_t*>(&yr[1]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int sh = (e & 1) * 16;
            const uint32_t xv = ((x0[e >> 1] >> sh) & 0xffffu) | (((x1[e >> 1] >> sh) & 0xffffu) << 16);
            const uint32_t yv = ((y0[e >> 1] >> sh) & 0xffffu) | (((y1[e >> 1] >> sh) & 0xffffu) << 16);
            *reinterpret_cast<uint32_t*>(xt + (8 * cc + e) * kDwbPS + 2 * pp2) = xv;
            *reinterpret_cast<uint32_t*>(yt + (8 * cc + e) * kDwbPS + 2 * pp2) = yv;
        }
    };

    floatx4 d[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) d[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    uint4 xr[2], yr[2];
    fetch(p_begin, xr, yr);
    for (int64_t p0 = p_begin; p0 < p_end; p0 += kDwbPairs) {
        __syncthreads();   // the previous stage has been read
        stage(xr, yr);
        __syncthreads();
        if (p0 + kDwbPairs < p_end) fetch(p0 + kDwbPairs, xr, yr);   // in flight during the MFMAs
        uint4 av[4], bv[4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
            av[a] = *reinterpret_cast<const uint4*>(xt + (wi * 64 + a * 16 + r16) * kDwbPS + 8 * q);
#pragma unroll
        for (int b = 0; b < 4; ++b)
            bv[b] = *reinterpret_cast<const uint4*>(yt + (wo * 64 + b * 16 + r16) * kDwbPS + 8 * q);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b)
                d[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av[a]), as_bf16x8(bv[b]), d[a][b], 0, 0, 0);
    }
    // D[a][b] row 4q + j = input channel, column r16 = output channel
    float* out = part + (item * CI + ci0 + wi * 64) * (int64_t)CO + co0 + wo * 64;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int b = 0; b < 4; ++b) out[(int64_t)(a * 16 + 4 * q + j) * CO + b * 16 + r16] = d[a][b][j];
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
bool conv_bf16_supported(int ca, int cb, int K) {
    const bool a = ca == 32 || ca == 64 || ca == 128 || ca == 256;
    const bool b = cb == 64 || cb == 128 || cb == 256;
    return a && b && K <= 64;
}

size_t transpose_ws_bytes(int K, int rows, int cols) { return (size_t)K * rows * cols * sizeof(uint16_t); }

int transpose_w_bf16(const void* W, int K, int rows, int cols, void* Bt, hipStream_t s, unsigned* zero_counter) {
    if (K <= 0 || rows <= 0 || cols <= 0) return GSC_OK;
    const dim3 grid((unsigned)((cols + kTrTile - 1) / kTrTile), (unsigned)((rows + kTrTile - 1) / kTrTile),
                    (unsigned)K);
    const bool v16 = rows % 8 == 0 && cols % 8 == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(Bt) % 16 == 0;
    if (v16)
        hipLaunchKernelGGL(k_transpose_w<true>, grid, dim3(256), 0, s, reinterpret_cast<const uint16_t*>(W), rows,
                           cols, reinterpret_cast<uint16_t*>(Bt), zero_counter);
    else
        hipLaunchKernelGGL(k_transpose_w<false>, grid, dim3(256), 0, s, reinterpret_cast<const uint16_t*>(W), rows,
                           cols, reinterpret_cast<uint16_t*>(Bt), zero_counter);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

template <int CA, int CB, typename Sel>
static void launch_bf16(const void* X, int64_t n_x, const void* Bt, const int32_t* gat, const int32_t* sca,
                        const int64_t* gidx, const int32_t* perm, int K, int64_t G, int64_t n_y, void* Y, Sel sel,
                        hipStream_t s) {
    using S = BfShape<CA, CB>;
    const int64_t tiles = (G + S::TG - 1) / S::TG;
    hipLaunchKernelGGL((k_conv_bf16<CA, CB, Sel>), dim3((unsigned)tiles), dim3(kBfThreads), 0, s,
                       reinterpret_cast<const uint16_t*>(X), n_x, reinterpret_cast<const uint16_t*>(Bt), gat, sca,
                       gidx, perm, K, G, n_y, reinterpret_cast<uint16_t*>(Y), sel);
}

template <int CA, int CB, typename Sel>
static void launch_bf16_dma(const void* X, int64_t n_x, const void* Bt, const int32_t* gat, const int32_t* sca,
                            const int64_t* gidx, const int32_t* perm, int K, int64_t G, int64_t n_y, void* Y, Sel sel,
                            hipStream_t s) {
    using S = DmaShape<CA, CB>;
    const int64_t tiles = (G + S::TG - 1) / S::TG;
    hipLaunchKernelGGL((k_conv_bf16_dma<CA, CB, Sel>), dim3((unsigned)tiles), dim3(kBfThreads), 0, s,
                       reinterpret_cast<const uint16_t*>(X), n_x, reinterpret_cast<const uint16_t*>(Bt), gat, sca,
                       gidx, perm, K, G, n_y, reinterpret_cast<uint16_t*>(Y), sel);
}

template <typename Sel>
int conv_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const int32_t* gat, const int32_t* sca,
              const int64_t* gidx, const int32_t* perm, int K, int64_t n_y, void* Y, Sel sel, hipStream_t s) {
    if (n_y == 0) return GSC_OK;
    const int64_t G = (n_y + GSC_GROUP_ROWS - 1) / GSC_GROUP_ROWS;
#define GSC_BFD_CASE(A, B)                                                                  \
    if (ca == A && cb == B) {                                                               \
        launch_bf16_dma<A, B, Sel>(X, n_x, Bt, gat, sca, gidx, perm, K, G, n_y, Y, sel, s); \
        GSC_LAUNCH_CHECK();                                                                 \
        return GSC_OK;                                                                      \
    }
    GSC_BFD_CASE(128, 128) GSC_BFD_CASE(256, 128) GSC_BFD_CASE(128, 256) GSC_BFD_CASE(256, 256)
#undef GSC_BFD_CASE
#define GSC_BF_CASE(A, B)                                                                   \
    if (ca == A && cb == B) {                                                               \
        launch_bf16<A, B, Sel>(X, n_x, Bt, gat, sca, gidx, perm, K, G, n_y, Y, sel, s);     \
        GSC_LAUNCH_CHECK();                                                                 \
        return GSC_OK;                                                                      \
    }
    GSC_BF_CASE(32, 64) GSC_BF_CASE(64, 64) GSC_BF_CASE(128, 64) GSC_BF_CASE(256, 64)
    GSC_BF_CASE(32, 128) GSC_BF_CASE(64, 128) GSC_BF_CASE(128, 128) GSC_BF_CASE(256, 128)
    GSC_BF_CASE(32, 256) GSC_BF_CASE(64, 256) GSC_BF_CASE(128, 256) GSC_BF_CASE(256, 256)
#undef GSC_BF_CASE
    return fail(GSC_EINVAL, "conv_bf16: unsupported channels %d -> %d", ca, cb);
}

template int conv_bf16<WIdentity>(int, int, const void*, int64_t, const void*, const int32_t*, const int32_t*,
                                  const int64_t*, const int32_t*, int, int64_t, void*, WIdentity, hipStream_t);
template int conv_bf16<WSel>(int, int, const void*, int64_t, const void*, const int32_t*, const int32_t*,
                             const int64_t*, const int32_t*, int, int64_t, void*, WSel, hipStream_t);

bool dw_bf16_supported(int ci, int co) { return (ci == 128 || ci == 256) && (co == 128 || co == 256); }

int dw_bf16(int ci, int co, const void* X, int64_t n_in, const void* dY, int64_t n_out, const int32_t* in_idx,
            const int32_t* out_idx, const int64_t* seg, const int64_t* ibase, const int64_t* chunk, int K,
            int64_t items, float* part, hipStream_t s) {
    const unsigned tiles = (unsigned)((ci / kDwbTile) * (co / kDwbTile));
#define GSC_DWB_CASE(A, B)                                                                                  \
    if (ci == A && co == B) {                                                                               \
        hipLaunchKernelGGL((k_dw_bf16<A, B>), dim3((unsigned)items, tiles), dim3(kBfThreads), 0, s,          \
                           reinterpret_cast<const uint16_t*>(X), n_in, reinterpret_cast<const uint16_t*>(dY), n_out, \
                           in_idx, out_idx, seg, ibase, chunk, K, part);                                    \
        GSC_LAUNCH_CHECK();                                                                                 \
        return GSC_OK;                                                                                      \
    }
    GSC_DWB_CASE(128, 128) GSC_DWB_CASE(128, 256) GSC_DWB_CASE(256, 128) GSC_DWB_CASE(256, 256)
#undef GSC_DWB_CASE
    return fail(GSC_EINVAL, "dw_bf16: unsupported channels %d x %d", ci, co);
}

}  // namespace gsc
