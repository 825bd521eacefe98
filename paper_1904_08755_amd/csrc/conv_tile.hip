// bf16 tile engine for wide layers: the sum of Eq. 3 over a block plan, a
// tile of 16 blocks (256 output positions) by all output columns per
// workgroup, v_mfma_f32_16x16x32_bf16 with fp32 sums, bf16 output (nearest
// even).
//
// The tile is computed step by step; a step is one offset k of the union of
// the tile's block masks and 32 channels of the reduction.  Per step the
// workgroup copies into LDS, with buffer loads that write LDS directly:
//   - the 16 input rows of every block having k (32 channels of each: one
//     load instruction of 64 lanes x 16 bytes per block; a block without k,
//     or a position without a pair, reads out of range and so gets zeros),
//   - the 32 x C_out slice of the offset's weight matrix.
// Steps go through a ring of four LDS stages.  During step s the copies of
// step s + 4 are issued into the stage step s has just left, the MFMA
// operands of step s + 1 are read from LDS into registers, and the products
// of step s run on the operands read during step s - 1; the step ends once
// the copies of step s + 2 are complete (three steps after they were
// issued).  The steps of an offset are unrolled, and what they need of the
// offset (its blocks, its weight matrix, its input rows) is worked out once
// per offset: the scalar instructions of the bookkeeping share the SIMD's
// issue slots with the MFMAs.  Eight waves (two per SIMD) share the tile: wave (r, c) keeps the
// sums of blocks [16/WR r, 16/WR (r+1)) by 64 output columns c in registers
// and, for each block having k, multiplies the block's 16 x 32 rows by the
// 32 x 64 weights (four MFMAs per block).  Every output row's products are
// added in increasing offset order, so the result does not depend on the
// plan's row order and is bit-reproducible.  The sums are written once, as
// bf16, straight from the registers.
//
// The grid is persistent (one workgroup per CU) and takes tiles from the
// last to the first through a counter in device memory: tiles later in the
// plan hold rows with more neighbours (the plan sorts rows by neighbour
// count, then mask), so the large tiles go out first and the small ones fill
// the gaps.  Without a counter the workgroups take tiles nt-1-g, nt-1-g-G,
// ... .
//
// LDS layout of a stage: block b's rows at b * 1 KiB, row r's 64 bytes at
// r * 64 with 16-byte chunk c at ((c ^ ((r >> 1) & 3)) * 16); output column
// n's 32 weights at n * 64, chunk c at ((c ^ ((n >> 1) & 3)) * 16).  The XOR
// keeps the eight 16-byte reads that the LDS serves together in distinct
// banks.  (A load instruction writes 16 bytes per lane at lane * 16 of its
// destination, so the swizzle is applied to the chunk each lane fetches.)
// The tile's item table (16 row indices per block and offset) sits in
// dynamic LDS, 1 KiB per offset of the region.
#include <type_traits>

#include "conv_blk.h"

namespace gsc {

typedef __bf16 tbf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int tu32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 tbf16x2 __attribute__((ext_vector_type(2)));
typedef float tfloatx2 __attribute__((ext_vector_type(2)));

constexpr int kTileBlocks = 16;                         // blocks (of 16 positions) per tile
constexpr int kTilePos = kTileBlocks * kPlanBlockRows;  // 256 positions
constexpr int kTileThreads = 512;                       // eight waves
constexpr int kTileStageBytes = 16384;                  // rows of a stage; weights of a stage at most as much
constexpr int kTileMaxK = 29;                           // item table in the LDS left by the stages (29 KiB)
constexpr int kTileBufFlags = 0x00020000;               // buffer descriptor word 3: 32-bit data format
constexpr uint32_t kTileNone = 0x80000000u;             // an offset past any buffer the engine reads

// s_waitcnt operand: vmcnt(n) and lgkmcnt(0), expcnt left free (gfx9 encoding)
template <int N>
struct VmLgkmWait {
    static constexpr int value = (N & 15) | ((N >> 4) << 14) | (7 << 4);
};

template <int CA, int CB>
struct TileCfg {
    static constexpr int WC = CB / 64;               // column groups of 64
    static constexpr int WR = 8 / WC;                // position groups
    static constexpr int BPW = kTileBlocks / WR;     // blocks per wave
    static constexpr int NJ = 4;                     // 16-column blocks per wave
    static constexpr int H = CA / 32;                // steps per offset
    static constexpr int BINS = CB / 16;             // weight load instructions per step (1 KiB each)
    static constexpr int BL = BINS >= 8 ? BINS / 8 : 1;   // ... per wave (dummies where BINS < 8)
    static constexpr int LOADS = 2 + BL;             // load instructions per wave and step
    static_assert(CB == 64 || CB == 128 || CB == 256, "output width");
    static_assert(CA == 64 || CA == 128 || CA == 256, "reduction width");
};

__device__ __forceinline__ uint32_t tile_pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(tfloatx2{lo, hi}, tbf16x2));
}
// value of lane l ^ 1 (DPP quad_perm 1, 0, 3, 2)
__device__ __forceinline__ float tile_xor1(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xb1, 0xf, 0xf, false));
}
__device__ __forceinline__ void tile_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// What the steps of one offset need (see the kernel): the offset k (-1:
// none), which of a wave's blocks have it (bk), the byte offset of its
// weight matrix (wb) and the lane's row offsets in the two copied blocks.
struct OffState {
    int k;
    uint32_t bk, wb;
    uint32_t vr[2];
};

template <int CA, int CB, typename Sel, bool EP>
__global__ void __launch_bounds__(kTileThreads, 1)
k_conv_tile_bf16(const uint16_t* __restrict__ X, int64_t n_x, const uint16_t* __restrict__ Bt, int K, Sel sel,
                 const int32_t* __restrict__ perm, const uint32_t* __restrict__ bmask,
                 const int64_t* __restrict__ ibase, const int32_t* __restrict__ items, int64_t nb, int64_t n_y,
                 int64_t ntiles, unsigned* __restrict__ counter, Epilogue ep, uint16_t* __restrict__ Y) {
    using C = TileCfg<CA, CB>;
    // four stages, each array its own object so that the compiler can tell
    // the copies into one stage from the reads of another
    __shared__ __attribute__((aligned(1024))) uint8_t sa0[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sa1[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sa2[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sa3[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sb0[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sb1[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sb2[kTileStageBytes];
    __shared__ __attribute__((aligned(1024))) uint8_t sb3[kTileStageBytes];
    __shared__ int32_t perm_s[kTilePos];
    __shared__ int64_t next_s;                                          // the next tile to take
    __shared__ __attribute__((aligned(1024))) uint8_t sdummy[1024];   // destination of copies that carry nothing
    extern __shared__ __attribute__((aligned(16))) int32_t idx_s[];    // the tile's items: 16 K x 16 ints

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int wr = wave / C::WC, wc = wave % C::WC;
    const int sel_lane = lane < K ? sel(lane) : 0;

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void*)X, (short)0, (int)(n_x * CA * 2), kTileBufFlags);
    const __amdgpu_buffer_rsrc_t wrs =
        __builtin_amdgcn_make_buffer_rsrc((void*)Bt, (short)0, (int)((int64_t)K * CB * CA * 2), kTileBufFlags);

    // load lanes: row (or column) l / 4 of the instruction's 16, data chunk
    // (l % 4) ^ swizzle, stored at l * 16 of the destination
    const int lrow = lane >> 2;
    const uint32_t lchunk = 16u * (uint32_t)((lane & 3) ^ ((lane >> 3) & 3));
    // weight columns this wave copies: instructions wave * BL + i (16 columns each)
    uint32_t bcol[C::BL];
#pragma unroll
    for (int i = 0; i < C::BL; ++i) {
        const int ins = wave * C::BL + i;
        bcol[i] = ins < C::BINS ? (uint32_t)((16 * ins + lrow) * CA * 2) + lchunk : kTileNone;
    }
    // fragment read offsets: lane (r16, q) reads row (or column) r16, chunk q
    const int r16 = lane & 15, q = lane >> 4;
    const int frag = r16 * 64 + ((q ^ ((r16 >> 1) & 3)) * 16);

    auto stage_a = [&](auto P) -> uint8_t* {
        constexpr int p = decltype(P)::value;
        return p == 0 ? sa0 : (p == 1 ? sa1 : (p == 2 ? sa2 : sa3));
    };
    auto stage_b = [&](auto P) -> uint8_t* {
        constexpr int p = decltype(P)::value;
        return p == 0 ? sb0 : (p == 1 ? sb1 : (p == 2 ? sb2 : sb3));
    };

    // tile sequence: from the counter (taken one tile ahead), else static;
    // tile t of the sequence is plan tile ntiles - 1 - t
    auto tile_of = [&](int64_t t) -> int64_t { return t < ntiles ? ntiles - 1 - t : -1; };
    auto uniform = [](int64_t v) {   // a value every lane holds, as a scalar
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
        return (int64_t)(((uint64_t)hi << 32) | lo);
    };
    if (tid == 0) next_s = tile_of(counter ? (int64_t)atomicAdd(counter, 1u) : (int64_t)blockIdx.x);
    __syncthreads();
    int64_t tile = uniform(next_s);
    for (int64_t round = 1; tile >= 0; ++round) {
        const int64_t b0 = tile * kTileBlocks;
        const int nbt = (int)min((int64_t)kTileBlocks, nb - b0);

        // The tile's blocks (wave-uniform): lane b < nbt loads bmask[b0 + b]
        // and lane b <= nbt ibase[b0 + b] (one round trip for all of them),
        // then each value is read out of its lane.
        const uint32_t bm_l = lane < nbt ? bmask[b0 + lane] : 0u;
        const int64_t ib_l = lane <= nbt ? ibase[b0 + lane] : 0;
        const int64_t ib0 = uniform(ib_l);
        const uint32_t ib0_lo = (uint32_t)ib0;
        uint32_t bm[kTileBlocks];
        int32_t ibl[kTileBlocks];
        uint32_t U = 0;
#pragma unroll
        for (int b = 0; b < kTileBlocks; ++b) {
            bm[b] = (uint32_t)__builtin_amdgcn_readlane((int)bm_l, b);   // 0 past the tile's blocks
            ibl[b] = b < nbt ? (int32_t)((uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)ib_l, b) - ib0_lo) : 0;
            U |= bm[b];
        }
        // a tile holds at most 16 K items: the difference fits in 32 bits
        const int n_items = (int)((uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)ib_l, nbt) - ib0_lo);
        // the previous tile's last reads of the LDS (item table, output
        // rows, next tile) are done before they are overwritten
        tile_barrier();
        // The next tile from the counter: the atomic is issued here and its
        // result is first used after the loads below have returned, so the
        // two round trips overlap.  (The address is laundered through an
        // empty asm so that the compiler does not turn the single-lane atomic
        // into a wave reduction that waits for the result on the spot.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Wsometimes-uninitialized"
        unsigned t_raw;   // defined, and used, by thread 0 only (no merge with another value to copy it into)
        if (tid == 0 && counter) {
            __attribute__((address_space(1))) unsigned* c = (__attribute__((address_space(1))) unsigned*)counter;
            asm volatile("" : "+v"(c));
            t_raw = __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        {   // the tile's items (at most 16 K x 16 ints, 16-byte loads) and
            // output rows: all loads in flight before any store
            constexpr int kPer = (kTileBlocks * kTileMaxK * 4 + kTileThreads - 1) / kTileThreads;
            const tu32x4* src = reinterpret_cast<const tu32x4*>(items + ib0 * 16);
            const int last = n_items * 4 - 1;
            const int64_t pos = b0 * kPlanBlockRows + tid;
            int32_t prow = tid < kTilePos && pos < n_y ? perm[pos] : -1;
            tu32x4 v[kPer] = {};
            if (last >= 0) {
#pragma unroll
                for (int u = 0; u < kPer; ++u) v[u] = src[min(tid + u * kTileThreads, last)];
            }
#pragma unroll
            for (int u = 0; u < kPer; ++u) asm volatile("" : "+v"(v[u]));
            asm volatile("" : "+v"(prow));
            if (last >= 0) {
#pragma unroll
                for (int u = 0; u < kPer; ++u)
                    if (tid + u * kTileThreads <= last) reinterpret_cast<tu32x4*>(idx_s)[tid + u * kTileThreads] = v[u];
            }
            if (tid < kTilePos) perm_s[tid] = prow;
        }
        if (tid == 0) next_s = tile_of(counter ? (int64_t)t_raw : blockIdx.x + round * (int64_t)gridDim.x);
#pragma clang diagnostic pop
        __syncthreads();   // items and output rows staged

        // the blocks whose rows this wave copies: wave and wave + 8
        uint32_t bmw[2];
        int32_t iblw[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            bmw[j] = 0u;
            iblw[j] = 0;
#pragma unroll
            for (int b = 0; b < kTileBlocks; ++b)
                if (b == wave + 8 * j) {
                    bmw[j] = bm[b];
                    iblw[j] = ibl[b];
                }
        }
        // the blocks whose sums this wave keeps: BPW wr .. BPW wr + BPW - 1
        uint32_t bmv[C::BPW];
#pragma unroll
        for (int b = 0; b < C::BPW; ++b) {
            bmv[b] = 0u;
#pragma unroll
            for (int r = 0; r < C::WR; ++r)
                if (r == wr) bmv[b] = bm[C::BPW * r + b];
        }

        // Per-offset state (wave-uniform except the row offsets): the
        // offset k (-1: none), which of this wave's blocks have it (bk), the
        // byte offset of its weight matrix (wb) and the two copied blocks'
        // row offsets for this lane (vr, kTileNone where there is no row).
        // The steps of an iteration (L = max(4, H) steps: one offset, or two
        // when an offset takes two steps) use the states of the current
        // iteration, their copies four steps ahead those of the next one;
        // the states of the iteration after that are taken during step 1,
        // where their LDS reads hide behind the products.
        constexpr int H = C::H;
        constexpr int L = H > 4 ? H : 4;    // steps per iteration
        constexpr int NO = L / H;           // offsets per iteration
        uint32_t urem = U;                  // offsets not yet taken
        auto take_offset = [&](OffState& d) {
            d.k = urem ? __ffs(urem) - 1 : -1;
            urem &= urem - 1u;
            const int k = d.k >= 0 ? d.k : 0;
            d.bk = 0u;
#pragma unroll
            for (int b = 0; b < C::BPW; ++b) d.bk |= ((bmv[b] >> k) & 1u) << b;
            d.bk = d.k >= 0 ? d.bk : 0u;
            d.wb = (uint32_t)__builtin_amdgcn_readlane(sel_lane, k) * (uint32_t)(CB * CA * 2);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const uint32_t m = bmw[j];
                const bool has = d.k >= 0 && ((m >> k) & 1u);
                const int il = has ? iblw[j] + __popc(m & ((1u << k) - 1u)) : 0;
                const int32_t r = idx_s[il * 16 + lrow];
                d.vr[j] = has && r >= 0 && r < n_x ? (uint32_t)r * (uint32_t)(CA * 2) + lchunk : kTileNone;
            }
        };
        // copies of part h of offset state d into stage P: C::LOADS
        // instructions per wave, always; copy p < BL is weight instruction p,
        // the others the rows of the two blocks this wave copies
        auto issue_one = [&](const OffState& d, int h, auto P, int p) {
            if (p < C::BL) {
                const int ins = wave * C::BL + p;
                const uint32_t off = d.k >= 0 ? bcol[p] : kTileNone;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    wrs, (__attribute__((address_space(3))) void*)(ins < C::BINS ? stage_b(P) + ins * 1024 : sdummy),
                    16, off, d.wb + (uint32_t)(h * 64), 0, 0);
            } else {
                const int j = p - C::BL;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    xr, (__attribute__((address_space(3))) void*)(stage_a(P) + (wave + 8 * j) * 1024), 16, d.vr[j],
                    h * 64, 0, 0);
            }
        };
        auto issue = [&](const OffState& d, int h, auto P) {
#pragma unroll
            for (int p = 0; p < C::LOADS; ++p) issue_one(d, h, P, p);
        };

        floatx4 acc[C::BPW][C::NJ];
#pragma unroll
        for (int b = 0; b < C::BPW; ++b)
#pragma unroll
            for (int j = 0; j < C::NJ; ++j) acc[b][j] = floatx4{0.f, 0.f, 0.f, 0.f};

        if (U != 0u) {
            OffState dc[NO], dn[NO], dnn[NO];   // offsets of this iteration, the next and the one after
#pragma unroll
            for (int o = 0; o < NO; ++o) take_offset(dc[o]);
#pragma unroll
            for (int o = 0; o < NO; ++o) take_offset(dn[o]);
            // operands in registers: the weights of two steps (this one and
            // the next), the rows of one block at a time (a block's rows of
            // the next step are read once its products of this step are
            // issued)
            tu32x4 bfr[2][C::NJ], afr[C::BPW];
            issue(dc[0], 0, std::integral_constant<int, 0>{});
            issue(dc[1 / H], 1 % H, std::integral_constant<int, 1>{});
            issue(dc[2 / H], 2 % H, std::integral_constant<int, 2>{});
            issue(dc[3 / H], 3 % H, std::integral_constant<int, 3>{});
            __builtin_amdgcn_s_waitcnt(VmLgkmWait<2 * C::LOADS>::value);   // steps 0 and 1 copied
            tile_barrier();
#pragma unroll
            for (int j = 0; j < C::NJ; ++j)
                bfr[0][j] = *reinterpret_cast<const tu32x4*>(sb0 + (64 * wc + 16 * j) * 64 + frag);
#pragma unroll
            for (int b = 0; b < C::BPW; ++b)
                if ((dc[0].bk >> b) & 1u)
                    afr[b] = *reinterpret_cast<const tu32x4*>(sa0 + (C::BPW * wr + b) * 1024 + frag);
            // every wave has read stage 0 before step 0 copies into it
            __builtin_amdgcn_s_waitcnt(VmLgkmWait<2 * C::LOADS>::value);
            tile_barrier();
            // step j of the iteration (static): stage j % 4; the products of
            // step j on the operands read during the step before, and the
            // operands of step j + 1 read from stage (j + 1) % 4; halfway
            // through the products the copies of the step four ahead go into
            // stage j % 4 (whose operands every wave read during the step
            // before), and in step 1 the offsets of the iteration after next
            // are taken; then wait for the copies of step j + 2
            auto step = [&](auto J) {
                constexpr int j = decltype(J)::value;
                constexpr int st = j % 4, stn = (j + 1) % 4;
                constexpr bool ahead_here = j + 4 < L;               // the step four ahead is in this iteration
                constexpr int ja = ahead_here ? j + 4 : j + 4 - L;
                const uint8_t* san = stage_a(std::integral_constant<int, stn>{});
                const uint8_t* sbn = stage_b(std::integral_constant<int, stn>{});
#pragma unroll
                for (int c = 0; c < C::NJ; ++c)
                    bfr[(j + 1) & 1][c] = *reinterpret_cast<const tu32x4*>(sbn + (64 * wc + 16 * c) * 64 + frag);
                // fresh scalar copies: one bit test and branch per block
                uint32_t bk = dc[j / H].bk;
                asm volatile("" : "+s"(bk));
                // the next step has this step's offset: one test per block
                constexpr bool same = j + 1 < L && (j + 1) % H != 0;
                uint32_t bn = j + 1 < L ? dc[((j + 1) % L) / H].bk : dn[0].bk;
                asm volatile("" : "+s"(bn));
#pragma unroll
                for (int b = 0; b < C::BPW; ++b) {
                    // the copies go out spread over the products (copy p
                    // before block p * BPW / LOADS: issued together they
                    // queue at the vector memory unit and hold up every
                    // wave's products at once)
#pragma unroll
                    for (int p = 0; p < C::LOADS; ++p) {
                        if ((p * C::BPW) / C::LOADS == b) {
                            if constexpr (ahead_here)
                                issue_one(dc[ja / H], ja % H, std::integral_constant<int, st>{}, p);
                            else
                                issue_one(dn[ja / H], ja % H, std::integral_constant<int, st>{}, p);
                        }
                    }
                    if constexpr (j == 1) {
                        if (b == C::BPW / 2) {
#pragma unroll
                            for (int o = 0; o < NO; ++o) take_offset(dnn[o]);
                        }
                    }
                    if (same) {
                        if ((bk >> b) & 1u) {
#pragma unroll
                            for (int c = 0; c < C::NJ; ++c)
                                acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    __builtin_bit_cast(tbf16x8, afr[b]), __builtin_bit_cast(tbf16x8, bfr[j & 1][c]),
                                    acc[b][c], 0, 0, 0);
                            afr[b] = *reinterpret_cast<const tu32x4*>(san + (C::BPW * wr + b) * 1024 + frag);
                        }
                    } else {
                        if ((bk >> b) & 1u) {
#pragma unroll
                            for (int c = 0; c < C::NJ; ++c)
                                acc[b][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                    __builtin_bit_cast(tbf16x8, afr[b]), __builtin_bit_cast(tbf16x8, bfr[j & 1][c]),
                                    acc[b][c], 0, 0, 0);
                        }
                        if ((bn >> b) & 1u)
                            afr[b] = *reinterpret_cast<const tu32x4*>(san + (C::BPW * wr + b) * 1024 + frag);
                    }
                }
                // the copies of two steps on are complete, this step's operand reads done
                __builtin_amdgcn_s_waitcnt(VmLgkmWait<2 * C::LOADS>::value);
                tile_barrier();
            };
            static_assert(L % 4 == 0, "iterations of whole stage rounds");
            while (true) {
                step(std::integral_constant<int, 0>{});
                step(std::integral_constant<int, 1>{});
                step(std::integral_constant<int, 2>{});
                step(std::integral_constant<int, 3>{});
                if constexpr (L == 8) {
                    step(std::integral_constant<int, 4>{});
                    step(std::integral_constant<int, 5>{});
                    step(std::integral_constant<int, 6>{});
                    step(std::integral_constant<int, 7>{});
                }
#pragma unroll
                for (int o = 0; o < NO; ++o) {
                    dc[o] = dn[o];
                    dn[o] = dnn[o];
                }
                if (dc[0].k < 0) break;
            }
            __builtin_amdgcn_s_waitcnt(VmLgkmWait<0>::value);   // the trailing (empty) copies
            tile_barrier();
        }

        // Write the tile straight from registers: the sums become bf16 pairs
        // (lane (c, q) holds rows 4q .. 4q+3 of column c; after an exchange
        // with lane c ^ 1 an even lane holds rows 4q, 4q+1 of columns c, c+1
        // and an odd one rows 4q+2, 4q+3 of columns c-1, c), one 4-byte store
        // per lane, row and column block (measured as fast as staging whole
        // rows through LDS, and it needs no barrier).
        const bool odd = r16 & 1;
        float esc[C::NJ], esh[C::NJ];
#pragma unroll
        for (int j = 0; j < C::NJ; ++j) {
            const int col = 64 * wc + 16 * j + r16;
            esc[j] = EP && ep.scale ? ep.scale[col] : 1.f;
            esh[j] = EP && ep.shift ? ep.shift[col] : 0.f;
        }
#pragma unroll
        for (int b = 0; b < C::BPW; ++b) {
            const int blk = C::BPW * wr + b;
            const int pos = 16 * blk + 4 * q + (odd ? 2 : 0);
            const int32_t row0 = perm_s[pos], row1 = perm_s[pos + 1];
#pragma unroll
            for (int j = 0; j < C::NJ; ++j) {
                floatx4 v = acc[b][j];
                if constexpr (EP) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = epi_apply(v[i], esc[j], esh[j], ep.relu);
                }
                const float e0 = tile_xor1(odd ? v[0] : v[2]);
                const float e1 = tile_xor1(odd ? v[1] : v[3]);
                const uint32_t p0 = odd ? tile_pack_bf16(e0, v[2]) : tile_pack_bf16(v[0], e0);
                const uint32_t p1 = odd ? tile_pack_bf16(e1, v[3]) : tile_pack_bf16(v[1], e1);
                const int col = 64 * wc + 16 * j + (r16 & ~1);
                if (row0 >= 0 && row0 < n_y) *reinterpret_cast<uint32_t*>(Y + (int64_t)row0 * CB + col) = p0;
                if (row1 >= 0 && row1 < n_y) *reinterpret_cast<uint32_t*>(Y + (int64_t)row1 * CB + col) = p1;
            }
        }
        tile = uniform(next_s);   // written before the item staging's barrier
    }
}

// The tile counter starts at zero (a kernel, not a memset, so that the call
// can be captured in a graph).
__global__ void k_tile_counter_zero(unsigned* counter) { *counter = 0u; }

// ---------------------------------------------------------------------------
// Weight gradient for wide layers (the chain rule of Eq. 3): dW_k =
// sum over the pairs p of offset k of X[I_p]^T dY[O_p].  A workgroup takes
// one work item (a chunk of the pairs of one offset, see dw_item) and
// computes the whole C_in x C_out product of its pairs, 32 pairs per step;
// its partial sum goes to part[item], and k_dw_reduce adds an offset's
// partials in item order (so dW is deterministic).
//
// The reduction runs over pairs, while an MFMA operand holds eight
// consecutive reduction elements per lane: here eight pairs of one channel.
// The rows are copied into LDS as they are (pair-major, by buffer loads that
// write LDS directly, in a four-stage ring as in the tile engine), and the
// operands are read with the LDS transpose read (ds_read_b64_tr_b16: within
// each 16 lanes, lane i receives element i % 4 of the 8-byte chunks that
// lanes i / 4, i / 4 + 4, i / 4 + 8, i / 4 + 12 address), two per operand.
// A row of C channels is stored with its 32-byte chunks permuted by the
// row's index modulo 4 (chunk c at (c ^ (p % 4)) * 32), so the four rows a
// transpose read touches fall in distinct banks.  Eight waves: wave (r, c)
// keeps rows [128 r, 128 r + 128) of dW by C_out / WC columns in registers.
// ---------------------------------------------------------------------------
typedef short ts16x4 __attribute__((ext_vector_type(4)));

template <int CI, int CO>
struct DwTileCfg {
    static constexpr int WR = CI / 128;                 // dW row groups of 128
    static constexpr int WC = 8 / WR;                   // column groups
    static constexpr int NI = 8;                        // 16-row blocks per wave
    static constexpr int NJ = CO / WC / 16;             // 16-column blocks per wave
    static constexpr int XI = CI / 128;                 // X copy instructions per wave and step (1 KiB each)
    static constexpr int YI = CO / 128;                 // dY copy instructions per wave and step
    static constexpr int LOADS = XI + YI;
    static constexpr int XB = 32 * CI * 2;              // bytes of a step's X rows
    static constexpr int YB = 32 * CO * 2;
    static_assert(CI == 128 || CI == 256, "dW rows");
    static_assert(CO == 128 || CO == 256, "dW columns");
    static_assert(NJ >= 1, "columns per wave");
};

template <int CI, int CO>
__global__ void __launch_bounds__(kTileThreads, 1)
k_dw_tile_bf16(const uint16_t* __restrict__ X, int64_t n_in, const uint16_t* __restrict__ dY, int64_t n_out,
               const int32_t* __restrict__ in_idx, const int32_t* __restrict__ out_idx,
               const int64_t* __restrict__ seg, const int64_t* __restrict__ ibase, const int64_t* __restrict__ chunk,
               int K, float* __restrict__ part) {
    using C = DwTileCfg<CI, CO>;
    __shared__ __attribute__((aligned(1024))) uint8_t sx0[C::XB];
    __shared__ __attribute__((aligned(1024))) uint8_t sx1[C::XB];
    __shared__ __attribute__((aligned(1024))) uint8_t sx2[C::XB];
    __shared__ __attribute__((aligned(1024))) uint8_t sx3[C::XB];
    __shared__ __attribute__((aligned(1024))) uint8_t sy0[C::YB];
    __shared__ __attribute__((aligned(1024))) uint8_t sy1[C::YB];
    __shared__ __attribute__((aligned(1024))) uint8_t sy2[C::YB];
    __shared__ __attribute__((aligned(1024))) uint8_t sy3[C::YB];

    const int64_t item = blockIdx.x;
    int k;
    int64_t p_begin, p_end;
    if (!dw_item(ibase, chunk, seg, K, item, &k, &p_begin, &p_end)) return;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int wr = wave / C::WC, wc = wave % C::WC;

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc((void*)X, (short)0, (int)(n_in * CI * 2), kTileBufFlags);
    const __amdgpu_buffer_rsrc_t yr =
        __builtin_amdgcn_make_buffer_rsrc((void*)dY, (short)0, (int)(n_out * CO * 2), kTileBufFlags);

    // copy lanes: instruction j of this wave covers rows (pairs) of the
    // step; lane l takes 16 bytes of its row, the data chunk that the
    // permutation puts at position l of the instruction's 1 KiB
    constexpr int XL = CI / 8, YL = CO / 8;            // lanes per row
    auto lane_src = [&](int lanes_per_row, int row) -> uint32_t {
        const int u16 = lane % lanes_per_row;          // 16-byte slot in the row
        const int w = (u16 >> 1) ^ (row & 3);           // its 32-byte data chunk
        return (uint32_t)(w * 32 + (u16 & 1) * 16);
    };
    // the step's 4 pairs of this wave: 4 wave .. 4 wave + 3 (X and dY alike)
    auto sx = [&](auto P) -> uint8_t* {
        constexpr int p = decltype(P)::value;
        return p == 0 ? sx0 : (p == 1 ? sx1 : (p == 2 ? sx2 : sx3));
    };
    auto sy = [&](auto P) -> uint8_t* {
        constexpr int p = decltype(P)::value;
        return p == 0 ? sy0 : (p == 1 ? sy1 : (p == 2 ? sy2 : sy3));
    };
    // row indices of this wave's 4 pairs of the step at pair p0 (scalar
    // loads, taken one step before the copies that use them)
    struct PairRows {
        int32_t gi[4], go[4];
        bool ok[4];
    };
    auto load_rows = [&](int64_t p0, PairRows& pr) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t pp = p0 + 4 * wave + r;
            const int64_t pc = pp < p_end ? pp : p_end - 1;
            pr.gi[r] = __builtin_amdgcn_readfirstlane(in_idx[pc]);
            pr.go[r] = __builtin_amdgcn_readfirstlane(out_idx[pc]);
            pr.ok[r] = pp < p_end;
        }
    };
    auto issue = [&](const PairRows& pr, auto P) {
        uint8_t* dx = sx(P);
        uint8_t* dy = sy(P);
        int32_t gi[4], go[4];
        bool ok[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            gi[r] = pr.gi[r];
            go[r] = pr.go[r];
            ok[r] = pr.ok[r] && gi[r] >= 0 && gi[r] < n_in && go[r] >= 0 && go[r] < n_out;
        }
#pragma unroll
        for (int j = 0; j < C::XI; ++j) {
            const int rl = j * (64 / XL) + lane / XL;   // pair of the wave (0..3)
            const int row = 4 * wave + rl;               // row of the stage
            int32_t g = gi[0];
            bool v = ok[0];
#pragma unroll
            for (int r = 1; r < 4; ++r) {
                g = rl == r ? gi[r] : g;
                v = rl == r ? ok[r] : v;
            }
            const uint32_t off = v ? (uint32_t)g * (uint32_t)(CI * 2) + lane_src(XL, row) : kTileNone;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                xr, (__attribute__((address_space(3))) void*)(dx + (wave * C::XI + j) * 1024), 16, off, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < C::YI; ++j) {
            const int rl = j * (64 / YL) + lane / YL;
            const int row = 4 * wave + rl;
            int32_t g = go[0];
            bool v = ok[0];
#pragma unroll
            for (int r = 1; r < 4; ++r) {
                g = rl == r ? go[r] : g;
                v = rl == r ? ok[r] : v;
            }
            const uint32_t off = v ? (uint32_t)g * (uint32_t)(CO * 2) + lane_src(YL, row) : kTileNone;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                yr, (__attribute__((address_space(3))) void*)(dy + (wave * C::YI + j) * 1024), 16, off, 0, 0, 0);
        }
    };

    // transpose reads: lane (i, q) addresses row 8 q + i / 4 (+ 4 for the
    // second read), 8 bytes at channel base + 4 (i % 4)
    const int i16 = lane & 15, q = lane >> 4;
    const int trow = 8 * q + (i16 >> 2);
    auto tr_addr = [&](int row_bytes, int c0) -> int {   // c0: first channel of the 16-channel block
        return trow * row_bytes + (((c0 >> 4) ^ (trow & 3)) * 32) + 8 * (i16 & 3);
    };
    int xa[C::NI], yb[C::NJ];
#pragma unroll
    for (int a = 0; a < C::NI; ++a) xa[a] = tr_addr(CI * 2, 128 * wr + 16 * a);
#pragma unroll
    for (int b = 0; b < C::NJ; ++b) yb[b] = tr_addr(CO * 2, (CO / C::WC) * wc + 16 * b);
    // A step's 24 transpose reads are one block of inline assembly that
    // also waits for them: the builtin's memory operand does not tell the
    // compiler which stage it reads, so it would wait for every copy in
    // flight (into other stages too) before each read; and no instruction
    // may touch a read's registers before the read has completed.  Block a
    // + 4 of X sits 128 bytes after block a (its chunk index differs in bit
    // 2 only, which the row permutation leaves alone); the second read of an
    // operand is four rows (2 KiB) on.
    auto frags = [&](const uint8_t* bx, const uint8_t* by, tbf16x8 (&av)[C::NI], tbf16x8 (&bv)[C::NJ]) {
        static_assert(C::NI == 8 && C::NJ == 4 && CI == 256 && CO == 256, "the read block is written for 256 x 256");
        const uint32_t x0 = (uint32_t)(uintptr_t)(bx + xa[0]), x1 = (uint32_t)(uintptr_t)(bx + xa[1]);
        const uint32_t x2 = (uint32_t)(uintptr_t)(bx + xa[2]), x3 = (uint32_t)(uintptr_t)(bx + xa[3]);
        const uint32_t y0 = (uint32_t)(uintptr_t)(by + yb[0]), y1 = (uint32_t)(uintptr_t)(by + yb[1]);
        const uint32_t y2 = (uint32_t)(uintptr_t)(by + yb[2]), y3 = (uint32_t)(uintptr_t)(by + yb[3]);
        ts16x4 r[24];
        asm volatile(
            "ds_read_b64_tr_b16 %0, %24\n ds_read_b64_tr_b16 %1, %24 offset:2048\n"
            "ds_read_b64_tr_b16 %2, %25\n ds_read_b64_tr_b16 %3, %25 offset:2048\n"
            "ds_read_b64_tr_b16 %4, %26\n ds_read_b64_tr_b16 %5, %26 offset:2048\n"
            "ds_read_b64_tr_b16 %6, %27\n ds_read_b64_tr_b16 %7, %27 offset:2048\n"
            "ds_read_b64_tr_b16 %8, %28\n ds_read_b64_tr_b16 %9, %28 offset:2048\n"
            "ds_read_b64_tr_b16 %10, %29\n ds_read_b64_tr_b16 %11, %29 offset:2048\n"
            "ds_read_b64_tr_b16 %12, %30\n ds_read_b64_tr_b16 %13, %30 offset:2048\n"
            "ds_read_b64_tr_b16 %14, %31\n ds_read_b64_tr_b16 %15, %31 offset:2048\n"
            "ds_read_b64_tr_b16 %16, %28 offset:128\n ds_read_b64_tr_b16 %17, %28 offset:2176\n"
            "ds_read_b64_tr_b16 %18, %29 offset:128\n ds_read_b64_tr_b16 %19, %29 offset:2176\n"
            "ds_read_b64_tr_b16 %20, %30 offset:128\n ds_read_b64_tr_b16 %21, %30 offset:2176\n"
            "ds_read_b64_tr_b16 %22, %31 offset:128\n ds_read_b64_tr_b16 %23, %31 offset:2176\n"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]),
              "=&v"(r[7]), "=&v"(r[8]), "=&v"(r[9]), "=&v"(r[10]), "=&v"(r[11]), "=&v"(r[12]), "=&v"(r[13]),
              "=&v"(r[14]), "=&v"(r[15]), "=&v"(r[16]), "=&v"(r[17]), "=&v"(r[18]), "=&v"(r[19]), "=&v"(r[20]),
              "=&v"(r[21]), "=&v"(r[22]), "=&v"(r[23])
            : "v"(y0), "v"(y1), "v"(y2), "v"(y3), "v"(x0), "v"(x1), "v"(x2), "v"(x3)
            : "memory");
        auto join = [](ts16x4 lo, ts16x4 hi) {
            const ts16x4 v8[2] = {lo, hi};
            return __builtin_bit_cast(tbf16x8, v8);
        };
#pragma unroll
        for (int b = 0; b < 4; ++b) bv[b] = join(r[2 * b], r[2 * b + 1]);
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            av[a] = join(r[8 + 2 * a], r[9 + 2 * a]);
            av[a + 4] = join(r[16 + 2 * a], r[17 + 2 * a]);
        }
    };

    floatx4 acc[C::NI][C::NJ];
#pragma unroll
    for (int a = 0; a < C::NI; ++a)
#pragma unroll
        for (int b = 0; b < C::NJ; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    // step s reads stage s % 4; the copies of step s + 3 go into the stage
    // that step s - 1 has read; a step ends once step s + 1 is copied
    const int64_t steps = (p_end - p_begin + 31) / 32;
    PairRows pr;
    load_rows(p_begin, pr);
    issue(pr, std::integral_constant<int, 0>{});
    load_rows(p_begin + 32, pr);
    issue(pr, std::integral_constant<int, 1>{});
    load_rows(p_begin + 64, pr);
    issue(pr, std::integral_constant<int, 2>{});
    load_rows(p_begin + 96, pr);
    __builtin_amdgcn_s_waitcnt(VmLgkmWait<2 * C::LOADS>::value);   // step 0 copied
    tile_barrier();
    auto step = [&](int64_t s, auto P) {
        constexpr int p = decltype(P)::value;
        issue(pr, std::integral_constant<int, (p + 3) % 4>{});   // the copies of step s + 3
        load_rows(p_begin + 32 * (s + 4), pr);
        const uint8_t* bx = sx(P);
        const uint8_t* by = sy(P);
        tbf16x8 bv[C::NJ], av[C::NI];
        frags(bx, by, av, bv);
        __builtin_amdgcn_s_waitcnt(VmLgkmWait<2 * C::LOADS>::value);   // step s + 1's copies done
#pragma unroll
        for (int a = 0; a < C::NI; ++a)
#pragma unroll
            for (int b = 0; b < C::NJ; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bv[b], acc[a][b], 0, 0, 0);
        tile_barrier();
    };
    for (int64_t s = 0; s < steps; s += 4) {
        step(s, std::integral_constant<int, 0>{});
        if (s + 1 < steps) step(s + 1, std::integral_constant<int, 1>{});
        if (s + 2 < steps) step(s + 2, std::integral_constant<int, 2>{});
        if (s + 3 < steps) step(s + 3, std::integral_constant<int, 3>{});
    }
    __builtin_amdgcn_s_waitcnt(VmLgkmWait<0>::value);   // the trailing (empty) copies

    // the item's partial sums: lane (c, q) holds rows 4q .. 4q+3 of column c
    float* out = part + (item * CI + 128 * wr) * (int64_t)CO + (CO / C::WC) * wc;
#pragma unroll
    for (int a = 0; a < C::NI; ++a)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int b = 0; b < C::NJ; ++b) out[(int64_t)(16 * a + 4 * q + i) * CO + 16 * b + i16] = acc[a][b][i];
}

bool dw_tile_bf16_supported(int ci, int co) { return ci == 256 && co == 256; }

int dw_tile_bf16(int ci, int co, const void* X, int64_t n_in, const void* dY, int64_t n_out, const int32_t* in_idx,
                 const int32_t* out_idx, const int64_t* seg, const int64_t* ibase, const int64_t* chunk, int K,
                 int64_t items, float* part, hipStream_t s) {
    if (items <= 0) return GSC_OK;
#define GSC_DWT_CASE(A, B)                                                                                    \
    if (ci == A && co == B) {                                                                                 \
        hipLaunchKernelGGL((k_dw_tile_bf16<A, B>), dim3((unsigned)items), dim3(kTileThreads), 0, s,            \
                           reinterpret_cast<const uint16_t*>(X), n_in, reinterpret_cast<const uint16_t*>(dY), n_out, \
                           in_idx, out_idx, seg, ibase, chunk, K, part);                                      \
        GSC_LAUNCH_CHECK();                                                                                   \
        return GSC_OK;                                                                                        \
    }
    GSC_DWT_CASE(256, 256)
#undef GSC_DWT_CASE
    return fail(GSC_EINVAL, "dw_tile_bf16: unsupported channels %d x %d", ci, co);
}

bool tile_bf16_supported(int ca, int cb, int K) {
    return (ca == 64 || ca == 128 || ca == 256) && (cb == 64 || cb == 128 || cb == 256) && K >= 1 && K <= kTileMaxK;
}

template <int CA, int CB, typename Sel, bool EP>
static int launch_tile_kernel(const uint16_t* X, int64_t n_x, const uint16_t* Bt, int K, const Sel& sel,
                              const BlockPlan& p, int64_t nb, int64_t n_y, const Epilogue& ep, uint16_t* Y,
                              unsigned* counter, bool counter_ready, hipStream_t s) {
    const int64_t tiles = (nb + kTileBlocks - 1) / kTileBlocks;
    if (tiles == 0) return GSC_OK;
    const int64_t grid = tiles < device_cus() ? tiles : device_cus();
    const size_t dyn = (size_t)kTileBlocks * K * 16 * sizeof(int32_t);
    auto kern = k_conv_tile_bf16<CA, CB, Sel, EP>;
    GSC_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)dyn));
    if (counter && !counter_ready) {
        hipLaunchKernelGGL(k_tile_counter_zero, dim3(1), dim3(1), 0, s, counter);
        GSC_LAUNCH_CHECK();
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kTileThreads), dyn, s, X, n_x, Bt, K, sel, p.perm, p.bmask,
                       p.ibase, p.items, nb, n_y, tiles, counter, ep, Y);
    GSC_LAUNCH_CHECK();
    return GSC_OK;
}

template <typename Sel>
int conv_tile_bf16(int ca, int cb, const void* X, int64_t n_x, const void* Bt, const Sel& sel, int K,
                   const BlockPlan& plan, int64_t nb, int64_t n_y, void* Y, unsigned* counter, hipStream_t s,
                   const Epilogue& ep, bool counter_ready) {
    auto X16 = reinterpret_cast<const uint16_t*>(X);
    auto B16 = reinterpret_cast<const uint16_t*>(Bt);
    auto Y16 = reinterpret_cast<uint16_t*>(Y);
    const bool epi = std::is_same<Sel, WIdentity>::value && ep.on();   // the epilogue is a forward-pass option
#define GSC_TILE_CASE(A, B)                                                                                    \
    if (ca == A && cb == B) {                                                                                  \
        if (epi)                                                                                               \
            return launch_tile_kernel<A, B, Sel, true>(X16, n_x, B16, K, sel, plan, nb, n_y, ep, Y16, counter,      \
                                                       counter_ready, s);                                          \
        return launch_tile_kernel<A, B, Sel, false>(X16, n_x, B16, K, sel, plan, nb, n_y, ep, Y16, counter,         \
                                                    counter_ready, s);                                             \
    }
    GSC_TILE_CASE(64, 64) GSC_TILE_CASE(64, 128) GSC_TILE_CASE(64, 256) GSC_TILE_CASE(128, 64)
    GSC_TILE_CASE(128, 128) GSC_TILE_CASE(128, 256) GSC_TILE_CASE(256, 64) GSC_TILE_CASE(256, 128)
    GSC_TILE_CASE(256, 256)
#undef GSC_TILE_CASE
    return fail(GSC_EINVAL, "conv: no bf16 tile engine for %dx%d", ca, cb);
}

template int conv_tile_bf16<WIdentity>(int, int, const void*, int64_t, const void*, const WIdentity&, int,
                                       const BlockPlan&, int64_t, int64_t, void*, unsigned*, hipStream_t,
                                       const Epilogue&, bool);
template int conv_tile_bf16<WSel>(int, int, const void*, int64_t, const void*, const WSel&, int, const BlockPlan&,
                                  int64_t, int64_t, void*, unsigned*, hipStream_t, const Epilogue&, bool);

}  // namespace gsc
