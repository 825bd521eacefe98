// Block convolution engines: the sum of Eq. 3 (Alg. 2's per-offset products,
// regrouped by output row block) over a block plan.
//
// A 16-row block of output positions is computed by one wave: for each
// offset in the block's union mask (in increasing offset order) the wave
// gathers the block's 16 input rows of that offset (zero rows where a row has
// no pair there) and accumulates their product with the offset's weight
// matrix into the block's sums, which stay in registers until the block is
// written, once, to its rows.  There is no scatter, no atomic and no partial
// buffer; a row's value is the sum of its offsets' products in increasing
// offset order whatever the position order, so results do not depend on the
// plan's row order.
//
// fp32 engine (reduction width CA, output width CB <= 64): all K weight
// matrices live in LDS in MFMA fragment order for the whole launch (one
// workgroup per CU, every wave of it walking its own blocks), so weights cost
// no global traffic per item.  A wave's items stream through a software
// pipeline of S slots: an item's 16 row indices are loaded S-1 items ahead,
// its rows (and its positions' output rows) RD items ahead, and its MFMAs
// (v_mfma_f32_16x16x4f32) run last.  (Deeper pipelines measured no faster:
// with 16 waves per CU the loads are not what the engine waits for.)  The loop body is unrolled over the slots, so each slot keeps its
// registers (no copies of loads in flight).
#include <type_traits>
#include <utility>

#include "conv_blk.h"

namespace gsc {

constexpr int kBlkLdsBytes = 144 * 1024;   // weight storage of the fp32 engine

// s_waitcnt operand for vmcnt(0) with expcnt and lgkmcnt left free (gfx9
// encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int kWaitVm0 = (7 << 4) | (15 << 8);
constexpr int kWaitLgkm0 = 0x3f | (7 << 4) | (3 << 14);   // lgkmcnt(0), vmcnt and expcnt left free

template <int CA, int CB>
struct BlkF32 {
    static constexpr int KS = CA / 4;        // MFMA steps (4 channels each)
    static constexpr int NNB = CB / 16;      // 16-column output blocks
    static constexpr int WF = KS * NNB;      // weight floats per lane per offset
    static constexpr int WG4 = WF / 4;       // ... as float4 groups
    static constexpr int RV = KS / 4;        // float4 row loads per lane
    // 16 waves per CU (128 VGPRs each) for 16- and 32-wide rows, 8 (256 VGPRs) for 64-wide ones
    static constexpr int THREADS = (CA == 64 || CB == 64) ? 512 : 1024;
    static constexpr int WAVES = THREADS / 64;
    static constexpr int S = 3;              // pipeline slots (items in flight)
    static constexpr int ID = S - 1;         // row indices are loaded ID items ahead
    static constexpr int RD = 1;             // rows are loaded RD items ahead
};

// One pipeline item: offset k (-1: a block with no offsets), block b (-1: a
// dummy), and whether it is the block's last item.
struct BlkItem {
    int k;
    int32_t b;
    bool last;
};

// f(0) || f(1) || ... || f(N-1) with compile-time arguments (stops at the
// first true).
template <typename F, size_t... I>
__device__ __forceinline__ bool run_steps(F& f, std::index_sequence<I...>) {
    return (f(std::integral_constant<int, (int)I>{}) || ...);
}

__device__ __forceinline__ int readlane_i32(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ int64_t readlane_i64(int64_t v, int l) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <int CA, int CB, bool WT, bool EP, bool ACC>
__global__ void __launch_bounds__((BlkF32<CA, CB>::THREADS))
k_conv_blk_f32(const float* __restrict__ X, int64_t n_x, const float* __restrict__ W, int K, WSel sel,
               const int32_t* __restrict__ perm, const uint32_t* __restrict__ bmask,
               const int64_t* __restrict__ ibase, const int32_t* __restrict__ items, int64_t nb, int64_t n_y,
               Epilogue ep, float* __restrict__ Y) {
    using C = BlkF32<CA, CB>;
    __shared__ float wl[kBlkLdsBytes / 4];
    // Weights in fragment order: lane (c, q) of offset k needs, for MFMA step
    // s and column block j, B_k[q*KS + s][16j + c]; flat f = s*NNB + j is
    // component f%4 of float4 group f/4 at ((k*WG4 + f/4)*64 + lane).  The
    // source is read in its own order as float4s, kFillBatch per thread in
    // flight before any is stored (the fill is latency-bound otherwise).
    {
        constexpr int kFillBatch = 8;
        const int per4 = CA * CB / 4;
        const int total4 = K * per4;
        const float4* W4 = reinterpret_cast<const float4*>(W);
        for (int e0 = threadIdx.x; e0 < total4; e0 += C::THREADS * kFillBatch) {
            float4 v[kFillBatch];
#pragma unroll
            for (int u = 0; u < kFillBatch; ++u) {
                const int e = e0 + u * C::THREADS;
                const int k = e / per4;
                const int src = WT ? sel(e < total4 ? k : 0) * per4 + (e - k * per4) : e;
                v[u] = W4[e < total4 ? src : 0];
            }
#pragma unroll
            for (int u = 0; u < kFillBatch; ++u) {
                const int e = e0 + u * C::THREADS;
                if (e >= total4) break;
                const int k = e / per4;
                const int rem = 4 * (e - k * per4);
                const float* vv = reinterpret_cast<const float*>(&v[u]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    int ch, col;
                    if constexpr (WT) {   // W[sel(k)] is cb x ca: B_k[ch][col] = W[sel(k)][col][ch]
                        col = (rem + i) / CA;
                        ch = (rem + i) - col * CA;
                    } else {
                        ch = (rem + i) / CB;
                        col = (rem + i) - ch * CB;
                    }
                    const int q = ch / C::KS, s = ch - q * C::KS;
                    const int f = s * C::NNB + (col >> 4);
                    wl[((k * C::WG4 + (f >> 2)) * 64 + (col & 15) + 16 * q) * 4 + (f & 3)] = vv[i];
                }
            }
        }
    }
    __syncthreads();

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform: block walk in SGPRs
    const int lane = threadIdx.x & 63;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t NW = (int64_t)gridDim.x * C::WAVES;
    const int64_t gw = (int64_t)blockIdx.x * C::WAVES + wave;
    const float4* wq = reinterpret_cast<const float4*>(wl) + lane;
    // epilogue coefficients of the lane's output columns 16j + r16
    float esc[C::NNB], esh[C::NNB];
#pragma unroll
    for (int j = 0; j < C::NNB; ++j) {
        esc[j] = EP && ep.scale ? ep.scale[16 * j + r16] : 1.f;
        esh[j] = EP && ep.shift ? ep.shift[16 * j + r16] : 0.f;
    }

    for (int64_t c0 = gw; c0 < nb; c0 += 64 * NW) {
        // this chunk: the wave's blocks c0 + l*NW, one per lane l
        const int64_t bl = c0 + (int64_t)lane * NW;
        const bool bv = bl < nb;
        const uint32_t lm = bv ? bmask[bl] : 0u;
        const int64_t lb = bv ? ibase[bl] : 0;
        const int nit = bv ? max(__popc(lm), 1) : 0;   // a block with no offsets still writes zeros
        int incl = nit;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int u = __shfl_up(incl, d, 64);
            if (lane >= d) incl += u;
        }
        const int T = readlane_i32(incl, 63);
        // the chunk's block table has arrived: without this wait the loop
        // would wait for every load in flight each time it reads the table
        __builtin_amdgcn_s_waitcnt(kWaitVm0);

        // decoder of the next item (wave-uniform state); past the chunk's T
        // items it yields dummies, so every pipeline step issues the same
        // loads (a load skipped on some path would make the compiler wait
        // for every load in flight before the MFMAs)
        int dslot = -1, dcount = 0;
        uint32_t drem = 0;
        int64_t dgi = 0;
        int32_t dblk = 0;
        auto decode = [&](BlkItem& m) -> int64_t {   // returns the item's index (0 if none)
            if (dcount >= T) {
                m = BlkItem{-1, -1, false};
                return 0;
            }
            ++dcount;
            if (drem == 0) {
                ++dslot;
                const uint32_t mm = (uint32_t)readlane_i32((int)lm, dslot);
                dgi = readlane_i64(lb, dslot);
                dblk = (int32_t)(c0 + (int64_t)dslot * NW);
                if (mm == 0) {
                    m = BlkItem{-1, dblk, true};
                    return 0;
                }
                drem = mm;
            }
            m.k = __ffs(drem) - 1;
            drem &= drem - 1;
            m.b = dblk;
            m.last = drem == 0;
            return dgi++;
        };

        constexpr int S = C::S;
        BlkItem mt[S];
        int32_t idxr[S], pmr[S];   // raw loads; validity is applied where they are used
        bool okr[S];
        float4 rv[S][C::RV];
        floatx4 acc[C::NNB];
#pragma unroll
        for (int j = 0; j < C::NNB; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < S; ++i) {
            mt[i] = BlkItem{-1, -1, false};
            idxr[i] = -1;
        }

        auto issue_idx = [&](auto P) {
            constexpr int p = decltype(P)::value;
            const int64_t gi = decode(mt[p]);
            idxr[p] = items[gi * 16 + r16];
        };
        auto issue_rows = [&](auto P) {
            constexpr int p = decltype(P)::value;
            const int32_t id = mt[p].k >= 0 ? idxr[p] : -1;
            okr[p] = id >= 0 && id < n_x;
            const float4* src = reinterpret_cast<const float4*>(X + (int64_t)(okr[p] ? id : 0) * CA + q * C::KS);
#pragma unroll
            for (int v = 0; v < C::RV; ++v) rv[p][v] = src[v];
            int64_t pos = (int64_t)mt[p].b * 16 + r16;
            pos = pos < 0 ? 0 : (pos < n_y ? pos : n_y - 1);
            pmr[p] = perm[pos];
        };
        auto compute = [&](auto P) {
            constexpr int p = decltype(P)::value;
            const int k = mt[p].k;
            if (k >= 0) {
                float4 wf[C::WG4];
#pragma unroll
                for (int g = 0; g < C::WG4; ++g) wf[g] = wq[(k * C::WG4 + g) * 64];
                const float* w = reinterpret_cast<const float*>(wf);
                const float* ar = reinterpret_cast<const float*>(rv[p]);
                float a[C::KS];
#pragma unroll
                for (int s = 0; s < C::KS; ++s) a[s] = okr[p] ? ar[s] : 0.f;
#pragma unroll
                for (int s = 0; s < C::KS; ++s)
#pragma unroll
                    for (int j = 0; j < C::NNB; ++j)
                        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], w[s * C::NNB + j], acc[j], 0, 0, 0);
            }
            if (mt[p].last) {
                // lane (c, q) holds rows 4q+i, column 16j + c of the block
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int32_t row = __shfl(pmr[p], 4 * q + i, 64);
                    const int64_t pos = (int64_t)mt[p].b * 16 + 4 * q + i;
                    if (pos < n_y && row >= 0 && row < n_y) {
                        float* yr = Y + (int64_t)row * CB + r16;
                        float prev[C::NNB];   // the earlier offset ranges' sums (ACC)
#pragma unroll
                        for (int j = 0; j < C::NNB; ++j) prev[j] = ACC ? yr[16 * j] : 0.f;
#pragma unroll
                        for (int j = 0; j < C::NNB; ++j) {
                            const float v = acc[j][i] + prev[j];
                            yr[16 * j] = EP ? epi_apply(v, esc[j], esh[j], ep.relu) : v;
                        }
                    }
                }
#pragma unroll
                for (int j = 0; j < C::NNB; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
            }
        };

        // Item i uses slot i mod S.  At u + p (u a multiple of S) the wave
        // loads item c + ID's row indices, item c + RD's rows and computes
        // item c = u + p - ID.  The chunk has T >= 1 items (its lane 0 holds
        // a block); before item 0 the slots hold dummies, so every step issues
        // the same loads and none is issued outside the loop.
        int u = 0;
        auto step = [&](auto P) -> bool {
            constexpr int p = decltype(P)::value;
            const int c = u + p - C::ID;
            issue_idx(std::integral_constant<int, p>{});
            issue_rows(std::integral_constant<int, (p + S - C::ID + C::RD) % S>{});
            if (c >= 0) compute(std::integral_constant<int, (p + S - C::ID) % S>{});
            return c + 1 >= T;
        };
        for (;; u += S)
            if (run_steps(step, std::make_index_sequence<S>{})) break;
    }
}

// Y = 0 (an input with no rows contributes nothing).
__global__ void k_zero_f32(float* __restrict__ y, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = 0.f;
}

// ---------------------------------------------------------------------------
// bf16 engine for wide layers (reduction width CA in {64, 128, 256}, output
// width CB in {64, 128, 256}): v_mfma_f32_16x16x32_bf16, fp32 sums, bf16
// output (nearest even).
//
// A workgroup of four waves owns a tile of kBfT blocks (128 positions); wave
// w owns output columns [w*CB/4, (w+1)*CB/4) of all of them and keeps their
// sums in registers.  The tile is computed group by group: a group is one
// offset of the union of the tile's masks and one 64-channel part of the
// reduction, and it applies that part of the offset's weights to every
// block having the offset (the mask-sorted order makes that most of the
// tile's blocks).  The schedule is a software pipeline over groups, written
// out statically (blocks in a static loop, groups unrolled over the three
// stages), so every iteration issues the same loads and the compiler's
// waits cover exactly the data an MFMA needs:
//   group g + 2: wave w loads the rows of blocks 2w and 2w + 1 (eight rows
//                of 128 bytes per load) and its own weight fragments into
//                registers, through buffer loads: a block without the
//                offset, or an item without a row, reads out of range and
//                so gets zeros;
//   group g + 1: the rows go to the LDS slab of that group (two slabs);
//   group g:     the MFMAs, rows read from LDS, weights from registers.
// One barrier per group hands a slab over.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBfT = 8;                              // blocks per tile
constexpr int kBfThreads = 256;
constexpr int kBfIdxInts = kBfT * kPlanMaxK * 16;    // the tile's items, at most
constexpr int kBufFlags = 0x00020000;                // buffer descriptor word 3: 32-bit data format
constexpr uint32_t kBufNone = 0x80000000u;           // an offset past any row buffer the engine takes

template <int CA, int CB>
struct BlkBf16 {
    static constexpr int NC = CB / 4;                // output columns per wave
    static constexpr int NB = NC / 16;               // 16-column blocks per wave
    static constexpr int CAH = 64;                   // channels per part
    static constexpr int H = CA / CAH;               // parts of the reduction
    static constexpr int KH = CAH / 32;              // MFMA steps per part
    static constexpr int RW = KH * NB;               // weight fragments (16 bytes per lane) per group
    static constexpr int WB = kBfT / 4;              // blocks whose rows one wave loads
    static constexpr int RL = 2 * WB;                // row loads (eight rows each) per wave and group
    static_assert(RW <= kBfT && RL <= kBfT, "a group's loads are spread over its block iterations");
};

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

// two fp32 values -> packed bf16 pair (lo, hi), nearest even
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// value of lane l ^ 1 (DPP quad_perm 1, 0, 3, 2)
__device__ __forceinline__ float xor1(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xb1, 0xf, 0xf, false));
}

// One group of the walk (wave-uniform): offset k, part h, blocks having k.
struct BfGroup {
    int k, h;
    uint32_t bk;
    bool valid;
};

template <int CA, int CB, typename Sel, bool EP>
__global__ void __launch_bounds__(kBfThreads, 2)
k_conv_blk_bf16(const uint16_t* __restrict__ X, int64_t n_x, const uint16_t* __restrict__ Bt, int K, Sel sel,
                const int32_t* __restrict__ perm, const uint32_t* __restrict__ bmask,
                const int64_t* __restrict__ ibase, const int32_t* __restrict__ items, int64_t nb, int64_t n_y,
                int cb_full, int64_t ntiles, Epilogue ep, uint16_t* __restrict__ Y) {
    using C = BlkBf16<CA, CB>;
    __shared__ __attribute__((aligned(16))) uint8_t slab[2][kBfT][16 * 128];   // [group parity][block][row][128 B]
    __shared__ int32_t idx_s[kBfIdxInts];
    __shared__ int32_t perm_s[kBfT * 16];
    // Workgroup -> (tile, column slice): the slices of one tile are 8
    // workgroups apart, so they run on the same XCD (workgroup i runs on XCD
    // i mod 8) at about the same time and share the tile's rows in its L2.
    const int nslice = cb_full / CB;
    const int64_t rest = blockIdx.x >> 3;
    const int slice = (int)(rest % nslice);
    const int64_t tile = (rest / nslice) * 8 + (blockIdx.x & 7);
    if (tile >= ntiles) return;
    const int col0 = slice * CB;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t b0 = tile * kBfT;
    const int nbt = (int)min((int64_t)kBfT, nb - b0);

    // the tile's blocks (wave-uniform) and the offset -> weight map per lane
    uint32_t bm[kBfT];
    int32_t ibl[kBfT];
    const int64_t ib0 = ibase[b0];
    uint32_t U = 0;
#pragma unroll
    for (int b = 0; b < kBfT; ++b) {
        bm[b] = b < nbt ? bmask[b0 + b] : 0u;
        ibl[b] = b < nbt ? (int32_t)(ibase[b0 + b] - ib0) : 0;
        U |= bm[b];
    }
    // the blocks whose rows this wave loads
    uint32_t bmw[C::WB];
    int32_t iblw[C::WB];
#pragma unroll
    for (int j = 0; j < C::WB; ++j) {
        bmw[j] = 0u;
        iblw[j] = 0;
#pragma unroll
        for (int b = j; b < kBfT; b += C::WB)
            if (b == C::WB * wave + j) {
                bmw[j] = bm[b];
                iblw[j] = ibl[b];
            }
    }
    const int n_items = (int)(ibase[b0 + nbt] - ib0);
    const int sel_lane = lane < K ? sel(lane) : 0;
    for (int i = tid; i < n_items * 16; i += kBfThreads) idx_s[i] = items[ib0 * 16 + i];
    for (int i = tid; i < kBfT * 16; i += kBfThreads) {
        const int64_t pos = b0 * 16 + i;
        perm_s[i] = pos < n_y ? perm[pos] : -1;
    }
    __syncthreads();   // items and output rows staged

    // X as a buffer of n_x * CA * 2 bytes (below 2^31), so that kBufNone reads zeros
    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void*)X, (short)0, (int)(n_x * CA * 2), kBufFlags);
    const __amdgpu_buffer_rsrc_t wr =
        __builtin_amdgcn_make_buffer_rsrc((void*)Bt, (short)0, (int)((int64_t)K * cb_full * CA * 2), kBufFlags);

    auto blocks_with = [&](int k) {
        uint32_t m = 0;
#pragma unroll
        for (int b = 0; b < kBfT; ++b) m |= ((bm[b] >> k) & 1u) << b;
        return m;
    };
    auto next_of = [&](BfGroup g) {
        if (!g.valid) return g;
        if (g.h + 1 < C::H) {
            ++g.h;
            return g;
        }
        const uint32_t kr = g.k < 31 ? U & ~((2u << g.k) - 1u) : 0u;
        if (!kr) {
            g.valid = false;
            g.bk = 0u;
            return g;
        }
        g.k = __ffs(kr) - 1;
        g.h = 0;
        g.bk = blocks_with(g.k);
        return g;
    };

    // registers of one pipeline stage: this wave's weight fragments of a
    // group and the rows it loads
    struct Stage {
        u32x4 w[C::RW];
        u32x4 r[C::RL];
    };
    // Row load j of a wave covers rows 8 (j % 2) .. +7 of block WB w + j / 2:
    // lane l takes row 8 (j % 2) + l / 8 and stores its 16-byte chunk at
    // position l % 8 of the slab row, which holds data chunk
    // (l % 8) ^ (row % 8) (swizzled so that the fragment reads hit distinct
    // banks).  Weight fragment f = (s, j) is lane (c, q)'s 16 bytes of B_k
    // rows 64 h + 32 s + 8 q .. +7, column w NC + 16 j + c.
    const int lrow = lane >> 3;
    const uint32_t lchunk = 16u * (uint32_t)((lane & 7) ^ (lrow & 7));
    uint32_t woff[C::RW];
#pragma unroll
    for (int f = 0; f < C::RW; ++f)
        woff[f] = (uint32_t)(((col0 + wave * C::NC + 16 * (f % C::NB) + r16) * CA + 32 * (f / C::NB) + 8 * q) * 2);
    // byte offsets of this lane's rows for group g (kBufNone: none)
    auto row_offsets = [&](const BfGroup& g, uint32_t (&off)[C::RL]) {
#pragma unroll
        for (int j = 0; j < C::RL; ++j) {
            const uint32_t m = bmw[j / 2];
            const bool has = g.valid && ((m >> g.k) & 1u);
            const int il = has ? iblw[j / 2] + __popc(m & ((1u << g.k) - 1u)) : 0;
            const int32_t v = idx_s[il * 16 + 8 * (j % 2) + lrow];
            off[j] = has && v >= 0 && v < n_x ? (uint32_t)v * (uint32_t)(CA * 2) + lchunk : kBufNone;
        }
    };
    auto load = [&](const BfGroup& g, int b, const uint32_t (&off)[C::RL], Stage& st) {
        const int h = g.valid ? g.h : 0;
        if (b < C::RL) st.r[b] = __builtin_amdgcn_raw_buffer_load_b128(xr, off[b], h * C::CAH * 2, 0);
        if (b < C::RW) {
            const int wsel = readlane_i32(sel_lane, g.valid ? g.k : 0);
            st.w[b] = __builtin_amdgcn_raw_buffer_load_b128(wr, woff[b], (wsel * cb_full * CA + h * C::CAH) * 2, 0);
        }
        // keep the loads here: their uses sit in conditional blocks two groups
        // on, and sinking them there would undo the pipeline
        asm volatile("" ::: "memory");
    };
    auto store = [&](const Stage& st, int b, int par) {
        if (b < C::RL)
            *reinterpret_cast<u32x4*>(&slab[par][C::WB * wave + b / 2][(b % 2) * 1024 + lane * 16]) = st.r[b];
    };
    // row r16's 16-byte chunks 4 s + q (s < KH) of block b in slab par
    auto read_a = [&](int par, int b, u32x4 (&a)[C::KH]) {
#pragma unroll
        for (int s2 = 0; s2 < C::KH; ++s2) {
            const int c = 4 * s2 + q;
            a[s2] = *reinterpret_cast<const u32x4*>(&slab[par][b][r16 * 128 + ((c ^ (r16 & 7)) * 16)]);
        }
    };

    floatx4 acc[kBfT][C::NB];
#pragma unroll
    for (int b = 0; b < kBfT; ++b)
#pragma unroll
        for (int j = 0; j < C::NB; ++j) acc[b][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    if (U != 0) {
        // The walk starts two empty groups early, so that entering the loop
        // leaves no loads in flight and the loop's own waits hold from its
        // first group on; an empty group loads (and stores) but computes
        // nothing.  left counts the groups until the last one is computed.
        Stage S[3] = {};
        BfGroup g0{0, 0, 0u, false}, g1 = g0, g2{__ffs(U) - 1, 0, 0u, true};
        g2.bk = blocks_with(g2.k);
        int left = __popc(U) * C::H + 2;
        int par = 0;   // slab of the current group
        // one group: load g+2 into stage (p+2)%3, store g+1 (stage (p+1)%3) to
        // the other slab, MFMAs of g (stage p) from this slab
        auto group = [&](auto P) {
            constexpr int p = decltype(P)::value;
            Stage& cur = S[p];
            Stage& nxt = S[(p + 1) % 3];
            Stage& far = S[(p + 2) % 3];
            uint32_t off[C::RL];
            row_offsets(g2, off);
            u32x4 a[2][C::KH];
            read_a(par, 0, a[0]);
#pragma unroll
            for (int b = 0; b < kBfT; ++b) {
                load(g2, b, off, far);
                store(nxt, b, par ^ 1);
                if (b + 1 < kBfT) read_a(par, b + 1, a[(b + 1) & 1]);
                if ((g0.bk >> b) & 1u) {
#pragma unroll
                    for (int s2 = 0; s2 < C::KH; ++s2)
#pragma unroll
                        for (int j = 0; j < C::NB; ++j)
                            acc[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8, a[b & 1][s2]),
                                __builtin_bit_cast(bf16x8, cur.w[s2 * C::NB + j]), acc[b][j], 0, 0, 0);
                }
            }
            __syncthreads();   // slab par ^ 1 written, slab par read by every wave
            par ^= 1;
            g0 = g1;
            g1 = g2;
            g2 = next_of(g2);
            --left;
        };
        // one exit, after whole rounds of three groups (the last round's
        // extra groups are empty): an exit after each group would give the
        // compiler a path around the later groups' loads, and with it
        // waits as if every load were recent
        do {
            group(std::integral_constant<int, 0>{});
            group(std::integral_constant<int, 1>{});
            group(std::integral_constant<int, 2>{});
        } while (left > 0);
    }
    // Write the tile through LDS, 64 positions per pass: the sums become bf16
    // pairs (lane (c, q) holds rows 4q .. 4q+3 of column c; after an
    // exchange with lane c ^ 1 an even lane holds rows 4q, 4q+1 of columns
    // c, c+1 and an odd one rows 4q+2, 4q+3 of columns c-1, c), and whole
    // output rows go out 16 bytes per lane.
    constexpr int LPR = CB / 8;                  // lanes per output row
    constexpr int RPI = kBfThreads / LPR;        // rows per pass of the workgroup
    static_assert(64 * CB * 2 <= (int)sizeof(slab), "a pass of 64 positions fits the slabs");
    uint32_t* out_s = reinterpret_cast<uint32_t*>(&slab[0][0][0]);
    const bool odd = r16 & 1;
    // epilogue coefficients of the lane's output columns (before rounding to bf16)
    float esc[C::NB], esh[C::NB];
#pragma unroll
    for (int j = 0; j < C::NB; ++j) {
        const int col = col0 + wave * C::NC + 16 * j + r16;
        esc[j] = EP && ep.scale ? ep.scale[col] : 1.f;
        esh[j] = EP && ep.shift ? ep.shift[col] : 0.f;
    }
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        if (half) __syncthreads();   // the first pass has been read
#pragma unroll
        for (int b = 4 * half; b < 4 * half + 4; ++b)
#pragma unroll
            for (int j = 0; j < C::NB; ++j) {
                floatx4 v = acc[b][j];
                if constexpr (EP) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = epi_apply(v[i], esc[j], esh[j], ep.relu);
                }
                const float e0 = xor1(odd ? v[0] : v[2]);
                const float e1 = xor1(odd ? v[1] : v[3]);
                const uint32_t p0 = odd ? pack_bf16(e0, v[2]) : pack_bf16(v[0], e0);
                const uint32_t p1 = odd ? pack_bf16(e1, v[3]) : pack_bf16(v[1], e1);
                const int row = 16 * (b - 4 * half) + 4 * q + (odd ? 2 : 0);
                const int cp = (wave * C::NC + 16 * j + (r16 & ~1)) / 2;
                out_s[row * (CB / 2) + cp] = p0;
                out_s[(row + 1) * (CB / 2) + cp] = p1;
            }
        __syncthreads();   // the pass is staged
#pragma unroll
        for (int r0 = 0; r0 < 64; r0 += RPI) {
            const int pos = r0 + tid / LPR;
            const int32_t row = perm_s[64 * half + pos];
            if (row >= 0 && row < n_y) {
                const u32x4 val = *reinterpret_cast<const u32x4*>(&out_s[pos * (CB / 2) + (tid % LPR) * 4]);
                *reinterpret_cast<u32x4*>(Y + (int64_t)row * cb_full + col0 + (tid % LPR) * 8) = val;
            }
        }
    }
}

bool blk_bf16_supported(int ca, int cb, int K) {
    return (ca == 64 || ca == 128 || ca == 256) && (cb == 64 || cb == 128 || cb == 256) && K >= 1 && K <= kPlanMaxK;
}

bool blk_bf16_fits(int64_t n_x, int ca) { return n_x >= 0 && n_x * ca < ((int64_t)1 << 30); }

template <int CA, int CB, typename Sel>
static void launch_blk_bf16(const uint16_t* X, int64_t n_x, const uint16_t* Bt, int K, const Sel& sel,
                            const BlockPlan& p, int64_t nb, int64_t n_y, int cb_full, const Epilogue& ep, uint16_t* Y,
                            hipStream_t s) {
    const int64_t tiles = (nb + kBfT - 1) / kBfT;
    const int64_t grid = 8 * (int64_t)(cb_full / CB) * ((tiles + 7) / 8);
    if constexpr (std::is_same<Sel, WIdentity>::value) {   // the epilogue is a forward-pass option
        if (ep.on()) {
            hipLaunchKernelGGL((k_conv_blk_bf16<CA, CB, Sel, true>), dim3((unsigned)grid), dim3(kBfThreads), 0, s, X,
                               n_x, Bt, K, sel, p.perm, p.bmask, p.ibase, p.items, nb, n_y, cb_full, tiles, ep, Y);
            return;
        }
    }
    hipLaunchKernelGGL((k_conv_blk_bf16<CA, CB, Sel, false>), dim3((unsigned)grid), dim3(kBfThreads), 0, s, X, n_x,
                       Bt, K, sel, p.perm, p.bmask, p.ibase, p.items, nb, n_y, cb_full, tiles, ep, Y);
}

__global__ void k_zero_u16(uint16_t* __restrict__ y, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        y[i] = 0;
}

template <typename Sel>
int conv_blk_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const Sel& sel, int K,
                  const BlockPlan& plan, int64_t n_y, void* Y, hipStream_t s, const Epilogue& ep) {
    if (!blk_bf16_supported(ca, cb, K)) return fail(GSC_EINVAL, "conv: no bf16 block engine for %dx%d, K=%d", ca, cb, K);
    if (ep.on() && !std::is_same<Sel, WIdentity>::value)
        return fail(GSC_EINVAL, "conv: the epilogue applies to the forward pass only");
    if (!blk_bf16_fits(n_x, ca)) return fail(GSC_EINVAL, "conv: bf16 block engine takes at most 2^30 input elements");
    const int64_t nb = (n_y + kPlanBlockRows - 1) / kPlanBlockRows;
    if (nb == 0) return GSC_OK;
    auto Y16 = reinterpret_cast<uint16_t*>(Y);
    if (n_x == 0) {   // no input rows to read (the engine always issues its row loads)
        const int64_t n = n_y * cb;
        hipLaunchKernelGGL(k_zero_u16, dim3((unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096)), dim3(256),
                           0, s, Y16, n);
        GSC_LAUNCH_CHECK();
        return ep.on() ? affine_act(GSC_BF16, Y16, n_y, cb, ep, s) : GSC_OK;
    }
    auto X16 = reinterpret_cast<const uint16_t*>(X);
    auto B16 = reinterpret_cast<const uint16_t*>(Bt);
    // 256 output columns go in two 128-column slices (two workgroups per
    // tile): a slice's sums fit in 167 VGPRs, so two workgroups share a CU
    // (two waves per SIMD), where one 256-column workgroup holds a CU alone
#define GSC_BFB_CASE(A, B, S)                                                         \
    if (ca == A && cb == B) {                                                         \
        launch_blk_bf16<A, S, Sel>(X16, n_x, B16, K, sel, plan, nb, n_y, B, ep, Y16, s); \
        GSC_LAUNCH_CHECK();                                                           \
        return GSC_OK;                                                                \
    }
    GSC_BFB_CASE(64, 64, 64) GSC_BFB_CASE(64, 128, 128) GSC_BFB_CASE(64, 256, 128) GSC_BFB_CASE(128, 64, 64)
    GSC_BFB_CASE(128, 128, 128) GSC_BFB_CASE(128, 256, 128) GSC_BFB_CASE(256, 64, 64) GSC_BFB_CASE(256, 128, 128)
    GSC_BFB_CASE(256, 256, 128)
#undef GSC_BFB_CASE
    return fail(GSC_EINVAL, "conv: no bf16 block engine for %dx%d", ca, cb);
}

template int conv_blk_bf16<WIdentity>(int, int, const void*, int64_t, const void*, const WIdentity&, int,
                                      const BlockPlan&, int64_t, void*, hipStream_t, const Epilogue&);
template int conv_blk_bf16<WSel>(int, int, const void*, int64_t, const void*, const WSel&, int, const BlockPlan&,
                                 int64_t, void*, hipStream_t, const Epilogue&);

bool blk_f32_supported(int ca, int cb, int K) {
    auto ok = [](int c) { return c == 16 || c == 32 || c == 64; };
    return ok(ca) && ok(cb) && K >= 1 && K <= kPlanMaxK && (int64_t)K * ca * cb * 4 <= kBlkLdsBytes;
}

template <int CA, int CB, bool WT, bool EP>
static void launch_blk_f32(const float* X, int64_t n_x, const float* W, const WSel& sel, int K, const BlockPlan& p,
                           int64_t nb, int64_t n_y, const Epilogue& ep, bool accum, float* Y, hipStream_t s) {
    // (accum is a template argument: a run-time test would leave a wait for every load in flight at each store)
    using C = BlkF32<CA, CB>;
    int64_t grid = (nb + C::WAVES - 1) / C::WAVES;
    const int cus = device_cus();
    if (grid > cus) grid = cus;
    if (accum)
        hipLaunchKernelGGL((k_conv_blk_f32<CA, CB, WT, EP, true>), dim3((unsigned)grid), dim3(C::THREADS), 0, s, X,
                           n_x, W, K, sel, p.perm, p.bmask, p.ibase, p.items, nb, n_y, ep, Y);
    else
        hipLaunchKernelGGL((k_conv_blk_f32<CA, CB, WT, EP, false>), dim3((unsigned)grid), dim3(C::THREADS), 0, s, X,
                           n_x, W, K, sel, p.perm, p.bmask, p.ibase, p.items, nb, n_y, ep, Y);
}

int conv_blk_f32(int ca, int cb, const float* X, int64_t n_x, const float* W, bool wt, const WSel& sel, int K,
                 const BlockPlan& plan, int64_t n_y, float* Y, hipStream_t s, const Epilogue& ep, bool accum) {
    if (!blk_f32_supported(ca, cb, K)) return fail(GSC_EINVAL, "conv: no fp32 block engine for %dx%d, K=%d", ca, cb, K);
    if (ep.on() && wt) return fail(GSC_EINVAL, "conv: the epilogue applies to the forward pass only");
    const int64_t nb = (n_y + kPlanBlockRows - 1) / kPlanBlockRows;
    if (nb == 0) return GSC_OK;
    if (n_x == 0) {   // no input rows to read (the engine always issues its row loads)
        const int64_t n = n_y * cb;
        if (!accum) {
            hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096)),
                               dim3(256), 0, s, Y, n);
            GSC_LAUNCH_CHECK();
        }
        return ep.on() ? affine_act(GSC_F32, Y, n_y, cb, ep, s) : GSC_OK;
    }
#define GSC_BLK_CASE(A, B)                                                                         \
    if (ca == A && cb == B) {                                                                      \
        if (wt)                                                                                    \
            launch_blk_f32<A, B, true, false>(X, n_x, W, sel, K, plan, nb, n_y, ep, accum, Y, s);  \
        else if (ep.on())                                                                          \
            launch_blk_f32<A, B, false, true>(X, n_x, W, sel, K, plan, nb, n_y, ep, accum, Y, s);  \
        else                                                                                       \
            launch_blk_f32<A, B, false, false>(X, n_x, W, sel, K, plan, nb, n_y, ep, accum, Y, s); \
        GSC_LAUNCH_CHECK();                                                                        \
        return GSC_OK;                                                                             \
    }
    GSC_BLK_CASE(16, 16) GSC_BLK_CASE(16, 32) GSC_BLK_CASE(16, 64) GSC_BLK_CASE(32, 16) GSC_BLK_CASE(32, 32)
    GSC_BLK_CASE(32, 64) GSC_BLK_CASE(64, 16) GSC_BLK_CASE(64, 32) GSC_BLK_CASE(64, 64)
#undef GSC_BLK_CASE
    return fail(GSC_EINVAL, "conv: no fp32 block engine for %dx%d", ca, cb);
}

}  // namespace gsc
