/*
 * gsc.h -- C ABI of the generalized sparse convolution library (libgsc.so)
 * for AMD Instinct MI355X (gfx950).
 *
 * The library implements the hot path of the generalized sparse convolution
 * of "4D Spatio-Temporal ConvNets: Minkowski Convolutional Neural Networks"
 * (Choy, Gwak, Savarese, CVPR 2019):
 *
 *   gsc_coords_build     hash table over the coordinates of a sparse tensor
 *                        (Sec. 3, Eq. 1; neighbour queries through a hash
 *                        table, Sec. 2 and Sec. 4.1)
 *   gsc_coords_stride    output coordinates of a strided convolution
 *                        (Sec. 4.2, first paragraph)
 *   gsc_kernel_map       kernel map M = {(I_i, O_i)}_i for an arbitrary
 *                        offset set N^D (Sec. 4.2; Eq. 3 of Sec. 3.1)
 *   gsc_conv_plan        the block plan of a kernel map: its output rows
 *                        ordered by neighbour mask, in 16-row blocks
 *   gsc_sparse_conv_fwd  Alg. 2 (and the transposed convolution of Sec. 4.2,
 *                        run on the role-reversed kernel map)
 *   gsc_sparse_conv_fwd_affine  the same with a per-channel affine map and
 *                        ReLU applied to the sums as they are stored (Sec. 4.5)
 *   gsc_sparse_conv_bwd  gradients of Alg. 2 with respect to the input
 *                        features and the weights (chain rule of Eq. 3)
 *   gsc_sparse_pool_*    max / average / sum pooling over a kernel map and
 *   gsc_global_pool_*    global pooling, with their gradients (Sec. 4.3,
 *                        Alg. 3; Sec. 4.4, Alg. 4); on the role-reversed
 *                        map, the transposed pooling (unpooling)
 *
 * Conventions
 *   - A coordinate row is (b, x_1, ..., x_D) of int32, batch index first;
 *     1 <= D <= 7.  Coordinates are row-major n x (1 + D); the row index is
 *     the position in that array.  The batch index is never offset.
 *   - Features are row-major n x C.  Weights are K x C_in x C_out row-major:
 *     W[k] is the C_in x C_out matrix of offset k, the transpose of the
 *     paper's W_i (Sec. 3.1), so a feature row f contributes f * W[k].
 *   - Offsets follow Eq. 3 literally: output u reads input u + ts (.) o_k.
 *   - Every device buffer is allocated and owned by the caller.  The library
 *     never allocates or frees device memory; it exports size queries.
 *     Host arrays (offsets, strides, counts) are read during the call only.
 *   - `stream` is a hipStream_t (NULL = the default stream).  All work is
 *     enqueued on it.
 *   - Every entry point returns GSC_OK (0) or a negative gsc_status.  On error
 *     gsc_last_error() returns a message (thread-local, valid until the next
 *     call on the same thread).  Arguments are validated on the host before
 *     any HIP call; errors found on the device (duplicate coordinate, table
 *     full, key range) are read back at the call's synchronisation point.
 */
#ifndef GSC_H
#define GSC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GSC_OK = 0,
    GSC_EINVAL = -1,  /* invalid argument (null pointer, negative size, bad D, ...) */
    GSC_ESHORT = -2,  /* caller buffer too small; the required size is returned   */
    GSC_ERANGE = -3,  /* coordinates span more than 92 bits of packed key          */
    GSC_EDUP = -4,    /* a coordinate row occurs twice                             */
    GSC_EFULL = -5,   /* hash table has no free slot                               */
    GSC_EHIP = -6,    /* a HIP runtime call failed                                 */
    GSC_ETIMEOUT = -7 /* a bounded device-side wait gave up: the result is invalid */
} gsc_status;

typedef enum { GSC_F32 = 0, GSC_BF16 = 1 } gsc_dtype;

/* Rows of one kernel-map group: the pairs of every offset are indexed in
 * groups of this many consecutive output rows (see gsc_kernel_map, gidx). */
#define GSC_GROUP_ROWS 64

const char* gsc_last_error(void);
int gsc_abi_version(void);

/* ------------------------------------------------------------------------ */
/* a1. Coordinate hash table (Sec. 3; hash-table neighbour search, Sec. 2).  */
/* ------------------------------------------------------------------------ */
/* Bytes of a table for n coordinates: a 256-byte header (key packing,
 * bounding box, status) followed by a power-of-two number (>= 4n, >= 64) of
 * 16-byte slots {uint64 key, int32 row, int32 hi}.  Open addressing with
 * linear probing; the key is the row packed into <= 92 bits relative to the
 * bounding box of the coordinates (batch column most significant): up to 62
 * bits in `key` alone, a wider key with its low 62 bits in `key` and the rest
 * in `hi` (an insert claims a slot by an atomic compare-and-swap on `key`
 * and then writes `hi`; an insert meeting the same low bits waits for that
 * write, boundedly: past the bound the build reports EFULL).  The home
 * slot keeps each 2 x 2 x 2 block of neighbouring coordinates in one 128-byte
 * line of slots, so a neighbourhood query touches few lines. */
size_t gsc_table_bytes(int64_t n);

/* Build the table of `coords` (device, n x (1+D) int32) into `table` (device,
 * table_bytes >= gsc_table_bytes(n)).  The table maps each row's coordinate to
 * its row index.  Synchronises `stream` once to read the device status.
 * Errors: EINVAL, ESHORT (table_bytes too small), ERANGE (bounding box needs
 * more than 92 key bits), EDUP (a repeated row), EFULL (no free slot: not
 * reached at the table's load factor of at most 1/4; the environment variable
 * GSC_TABLE_CAP_LIMIT, a test hook read by gsc_table_bytes and the builds,
 * caps the slot count to force it), EHIP.  n == 0 builds an empty table. */
int gsc_coords_build(const int32_t* coords, int64_t n, int32_t D,
                     void* table, size_t table_bytes, void* stream);

/* gsc_coords_build without the synchronisation: the build is only enqueued
 * and device-detected errors (EDUP, EFULL, ERANGE) are left in the table
 * header, where gsc_table_status reads them.  A kernel map queried from a
 * table whose build failed comes out empty.  Host-side errors (EINVAL,
 * ESHORT) are returned at once. */
int gsc_coords_build_async(const int32_t* coords, int64_t n, int32_t D,
                           void* table, size_t table_bytes, void* stream);

/* Synchronise `stream` and return the status the build left in `table`:
 * GSC_OK, GSC_EDUP, GSC_EFULL or GSC_ERANGE (GSC_EINVAL if `table` was never
 * built). */
int gsc_table_status(const void* table, void* stream);

/* ------------------------------------------------------------------------ */
/* a2. Output coordinates of a strided convolution (Sec. 4.2).              */
/* ------------------------------------------------------------------------ */
/* Workspace bytes for gsc_coords_stride with n_in input rows. */
size_t gsc_stride_ws_bytes(int64_t n_in);

/* For every input row, the output coordinate is (b, floor(x_d / s_d) * s_d)
 * (floor division, so -1 -> -2 for s = 2); repeated results are merged.  The
 * output rows are written to `out_coords` (device, capacity n_in rows) in the
 * order of the first input row that produces each of them, which is
 * deterministic; `*n_out` (host) receives their number.  `out_table` (device,
 * >= gsc_table_bytes(n_in) bytes) receives the hash table of the output
 * coordinates, usable by gsc_kernel_map.  `stride` is a host array of D
 * positive ints.  Synchronises `stream` once.  Errors: EINVAL, ESHORT (out_table
 * or ws too small), ERANGE, EHIP. */
int gsc_coords_stride(const int32_t* in_coords, int64_t n_in, int32_t D, const int32_t* stride,
                      int32_t* out_coords, int64_t* n_out, void* out_table, size_t out_table_bytes,
                      void* ws, size_t ws_bytes, void* stream);

/* gsc_coords_stride without its host round trip (Sec. 4.2, as above): the
 * kernels are enqueued on `stream`, followed by an asynchronous copy of 16
 * bytes into `result` (host, 2 int64; pinned memory keeps the call from
 * blocking, pageable memory makes the copy, and so the call, wait for the
 * stream).  Once the stream has passed that copy (an event recorded after
 * the call, or a synchronisation), gsc_coords_stride_result turns `result`
 * into the output row count and the build's status.  Work that needs only
 * `out_table` (a kernel map onto other coordinates) can be enqueued before
 * that.  Errors (of this call): EINVAL, ESHORT, EHIP. */
int gsc_coords_stride_async(const int32_t* in_coords, int64_t n_in, int32_t D, const int32_t* stride,
                            int32_t* out_coords, int64_t* result, void* out_table, size_t out_table_bytes,
                            void* ws, size_t ws_bytes, void* stream);

/* The outcome of a gsc_coords_stride_async call from its `result` (host):
 * `*n_out` (host) receives the number of output rows.  Errors: EINVAL (null
 * pointer), ERANGE (the strided box needs more key bits than a key holds),
 * EFULL (no free slot). */
int gsc_coords_stride_result(const int64_t* result, int64_t* n_out);

/* ------------------------------------------------------------------------ */
/* Sparse tensor quantization (Sec. 4.1, Alg. 1): the step before a1.       */
/* ------------------------------------------------------------------------ */
/* Workspace bytes for gsc_quantize with n points in D dimensions. */
size_t gsc_quantize_ws_bytes(int64_t n, int32_t D);

/* Points (device, n x D float32) with batch indices (device, n int32, or NULL
 * for batch 0) become voxels: coordinate (b, floor(p_1 / v_1), ...,
 * floor(p_D / v_D)), the floor of the exact quotient of the stored float32
 * values (0.7f / 0.1f is voxel 6, although the quotient rounded to float32 is
 * 7.0); voxel (host, D positive floats, taken as float32).  One output row per distinct
 * coordinate, written to out_coords (device, capacity n rows of 1 + D int32)
 * in the order of each voxel's first point; *n_out (host) receives their
 * number.  rep (device, capacity n int32): the first point of each voxel (the
 * row whose features it takes).  labels (device, n int32, nullable) and
 * out_labels (device, capacity n, nullable): a voxel's label is its points'
 * common label, or ignore_label when they carry more than one.  inverse
 * (device, n int32, nullable): the voxel row of every point.  out_table
 * (>= gsc_table_bytes(n) bytes) receives the hash table of the voxel
 * coordinates, usable by gsc_kernel_map.  Synchronises `stream` once.
 * Errors: EINVAL, ESHORT, ERANGE (a coordinate outside +-2^30, or a box needing
 * more than 92 key bits), EHIP. */
int gsc_quantize(const float* points, const int32_t* batch, int64_t n, int32_t D, const float* voxel,
                 const int32_t* labels, int32_t ignore_label, int32_t* out_coords, int64_t* n_out, int32_t* rep,
                 int32_t* out_labels, int32_t* inverse, void* out_table, size_t out_table_bytes,
                 void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* a3. Kernel map (Sec. 4.2; Eq. 3, Sec. 3.1).                              */
/* ------------------------------------------------------------------------ */
/* Number of 64-row groups of n_out output rows: ceil(n_out / 64). */
int64_t gsc_kmap_groups(int64_t n_out);
/* Workspace bytes for gsc_kernel_map. */
size_t gsc_kmap_ws_bytes(int64_t n_out, int32_t K, int32_t D);

/* For each offset o_k (host array `offsets`, K x D int32, any region: cube,
 * cross, hybrid, dilated, ...) and each output row j with coordinate u, emit
 * the pair (r, j) when u + ts (.) o_k is the coordinate of input row r in
 * `in_table` (built by gsc_coords_build or gsc_coords_stride).  `tensor_stride`
 * is a host array of D positive ints (the input tensor stride), or NULL for 1.
 *
 * Output (device): in_idx[p], out_idx[p] for p < n_pairs, grouped by offset in
 * the order of `offsets` and, within one offset, in increasing output row
 * (so the kernel map is deterministic).  seg[K + 1]: pairs of offset k are
 * [seg[k], seg[k+1]).  gidx[K * G + 1] with G = gsc_kmap_groups(n_out): the
 * pairs of offset k whose output row lies in [64 g, 64 g + 64) are
 * [gidx[k*G + g], gidx[k*G + g + 1]); gidx[K*G] = n_pairs.  gidx is what the
 * convolution kernels use to find the pairs of a tile of output rows.
 *
 * nbr (nullable, device, K * n_out int32): when given, the call also writes
 * the map's dense form, nbr[k * n_out + j] = the input row paired with output
 * row j at offset k, or -1 (the input of gsc_conv_plan).
 *
 * *n_pairs (host) receives the total.  If it exceeds cap_pairs, nothing is
 * written to in_idx/out_idx and ESHORT is returned with *n_pairs set, so the
 * caller can allocate and call again.  Synchronises `stream` once.
 *
 * Asynchronous mode: with n_pairs == NULL the call only enqueues work and
 * never synchronises.  Then cap_pairs must be at least K * n_out (so no map
 * can overflow), K * D must be at most 768, and the total is available on the
 * device only (seg[K] = gidx[K*G]).  The convolution calls need no host pair
 * count (they take an upper bound), so a whole layer can be enqueued without
 * a round trip to the host.
 *
 * The transposed convolution's map (roles of input and output reversed,
 * Sec. 4.2) is this function applied to the table of the original output
 * coordinates, the original input coordinates as `out_coords` and the negated
 * offsets: it lists the same pairs, ordered by the original input row. */
int gsc_kernel_map(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D,
                   const int32_t* offsets, int32_t K, const int32_t* tensor_stride,
                   int32_t* in_idx, int32_t* out_idx, int64_t cap_pairs,
                   int64_t* seg, int64_t* gidx, int32_t* nbr, int64_t* n_pairs,
                   void* ws, size_t ws_bytes, void* stream);

/* Allocation-free kernel map, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): gsc_kernel_map in its asynchronous mode (never synchronises;
 * cap_pairs >= K * n_out, K * D <= 768; the total is left on the device in
 * seg[K] = gidx[K*G]) with the dense form nbr (device, K * n_out int32)
 * required, and no workspace argument: the per-(offset, group) counts, the
 * scan partials and the status words live in a device array that the
 * library holds, gsc_kernel_map_noalloc_bytes(n_out, K) of its 8 MiB (each
 * GPU the library runs on holds its own copy until the process ends).  The
 * call allocates and frees nothing; it needs every count and flag it reads to
 * be written by itself first, so the array's contents from an earlier call do
 * not matter.  All calls on one GPU share that GPU's array: calls that
 * overlap on one GPU (on different streams, or from several threads) race and
 * must be serialised by the caller.  The stream must belong to the current
 * device.  Arguments and results otherwise as gsc_kernel_map.  Errors:
 * EINVAL (as gsc_kernel_map, and a null nbr), ESHORT (cap_pairs below
 * K * n_out), ERANGE (more scratch than the 8 MiB, e.g. n_out above about
 * 4.9 M rows at K = 27: then call gsc_kernel_map with a workspace), EHIP. */
size_t gsc_kernel_map_noalloc_bytes(int64_t n_out, int32_t K);
int gsc_kernel_map_noalloc(const void* in_table, const int32_t* out_coords, int64_t n_out, int32_t D,
                           const int32_t* offsets, int32_t K, const int32_t* tensor_stride,
                           int32_t* in_idx, int32_t* out_idx, int64_t cap_pairs,
                           int64_t* seg, int64_t* gidx, int32_t* nbr, void* stream);

/* The role-reversed map (Sec. 4.2: the transposed convolution's pairs are
 * the forward ones with input and output exchanged) of a map, built from its
 * pairs alone, without a coordinate table.  Input (device): in_idx, out_idx
 * and seg[K + 1] of a map as gsc_kernel_map writes it (any region, stride or
 * output set: an input row occurs at most once per offset), cap_pairs = the
 * length of the pair arrays (>= seg[K]; only seg[K] pairs are read), n_rev =
 * the number of the map's input rows (they become the output rows).  Output
 * (device, caller-allocated): t_in_idx, t_out_idx (cap_pairs each) with
 * t_in_idx = the former output row and t_out_idx = the former input row,
 * grouped by offset in the same order and increasing in t_out_idx within an
 * offset; t_seg[K + 1]; t_gidx[K * G + 1], G = gsc_kmap_groups(n_rev), as
 * gsc_kernel_map's gidx over the n_rev rows; t_nbr[K * n_rev], the dense form
 * (the input of gsc_conv_plan).  ws: gsc_kernel_map_transpose_ws_bytes(n_rev,
 * K).  Segment k of the result holds the pairs of offset k, so a backward
 * call on it takes the identity as t_wsel.  Asynchronous.  A pair whose
 * input row lies outside [0, n_rev) is left out and flagged in ws:
 * gsc_kernel_map_transpose_status(ws, stream) synchronises and returns EINVAL
 * then, else GSC_OK.  Errors: EINVAL, ESHORT (ws), EHIP. */
size_t gsc_kernel_map_transpose_ws_bytes(int64_t n_rev, int32_t K);
int gsc_kernel_map_transpose(const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg, int32_t K,
                             int64_t cap_pairs, int64_t n_rev, int32_t* t_in_idx, int32_t* t_out_idx,
                             int64_t* t_seg, int64_t* t_gidx, int32_t* t_nbr, void* ws, size_t ws_bytes,
                             void* stream);
int gsc_kernel_map_transpose_status(const void* ws, void* stream);

/* ------------------------------------------------------------------------ */
/* Block plan of a kernel map (an ordering of the output rows for a4 - a6). */
/* ------------------------------------------------------------------------ */
/* Eq. 3 sums, for every output row, one product per offset at which the row
 * has a pair.  The block engines of gsc_sparse_conv_fwd/bwd compute 16 output
 * rows together (one MFMA row block): for each offset that any of the 16 rows
 * has they gather the 16 input rows of that offset (zero where a row has no
 * pair) and multiply them by the offset's weight matrix, keeping the block's
 * sums in registers; so a block costs one product per distinct offset of its
 * rows.  The plan orders the output rows by neighbour mask (bit k set when
 * the row has a pair at offset k), so rows with equal masks share blocks;
 * the sort key puts the mask's popcount (capped) above the mask, so rows
 * with fewer neighbours come first and runs of blocks share offsets too.
 *
 * Input: the dense form of a kernel map over n_out output rows with K <= 32
 * offsets, nbr[k * n_out + j] = input row paired with output row j at offset
 * k or -1 (as gsc_kernel_map writes it).  Output (device, caller-allocated),
 * with
 * nb = gsc_plan_blocks(n_out) = ceil(n_out / 16):
 *   perm[n_out]       perm[i] = the output row at position i: a stable sort
 *                     of the rows by key = (min(popcount(mask), cap) << K)
 *                     | mask, cap = 2^p - 1, p = min(10 ceil(K / 10) - K,
 *                     32 - K, 6) (the bits the sort's last 10-bit digit
 *                     leaves free; K = 27: counts capped at 7);
 *   bmask[nb]         bmask[b] = OR of the masks of positions 16b..16b+15;
 *   ibase[nb + 1]     exclusive scan of popcount(bmask); ibase[nb] = items;
 *   items[16 * cap_items]  item t = ibase[b] + j belongs to block b and the
 *                     j-th set bit k of bmask[b] (increasing k); entry
 *                     items[16t + r] is the input row paired at offset k with
 *                     the output row at position 16b + r, or -1 if none.
 * cap_items must be >= K * nb (an upper bound of the item count).
 *
 * A map with 32 < K <= 128 offsets (the 3^4 tesseract's 81, the 5^3 cube's
 * 125) is planned in R = gsc_plan_ranges(K) = ceil(K / 32) ranges of
 * consecutive offsets: range r holds offsets k0 = r*S .. min(K, k0 + S) - 1
 * with S = ceil(K / R), and is the plan above of the map restricted to them
 * (bit k - k0 of a mask for offset k), stored at perm + r*n_out,
 * bmask + r*nb, ibase + r*(nb+1) (item numbers counted from the range's
 * first item) and items + 16*k0*nb.  So perm, bmask and ibase hold R times
 * the sizes above; cap_items is still >= K * nb.  The engines add the ranges'
 * sums in range order.
 *
 * ws: gsc_conv_plan_ws_bytes(n_out, K) bytes.  Asynchronous, deterministic.
 * Errors: EINVAL (K > 128, null pointers), ESHORT (cap_items, ws), EHIP.
 *
 * The sort's passes find each tile's place by looking back at the counts
 * earlier tiles publish, polling an entry not yet published a bounded number
 * of times (far more than a running tile needs).  Should a pass give up, it
 * finishes with a wrong prefix, sets a status word in ws and every later step
 * of the call stays inside its arrays; gsc_conv_plan_status then returns
 * ETIMEOUT, and the plan must be built again before it is used.
 * (The environment variable GSC_PLAN_SPIN_LIMIT overrides the bound for
 * tests; a negative value gives up at once.) */
int32_t gsc_plan_ranges(int32_t K);
int64_t gsc_plan_blocks(int64_t n_out);
size_t gsc_conv_plan_ws_bytes(int64_t n_out, int32_t K);
int gsc_conv_plan(const int32_t* nbr, int64_t n_out, int32_t K,
                  int32_t* perm, uint32_t* bmask, int64_t* ibase, int32_t* items, int64_t cap_items,
                  void* ws, size_t ws_bytes, void* stream);

/* Synchronise `stream` and return the status of the last gsc_conv_plan call
 * that used `ws` (with the same n_out and K): GSC_OK, or GSC_ETIMEOUT if one
 * of its sort passes gave up (EINVAL, ESHORT for bad arguments, EHIP). */
int gsc_conv_plan_status(const void* ws, size_t ws_bytes, int64_t n_out, int32_t K, void* stream);

/* 1 if gsc_sparse_conv_fwd/bwd have a block engine for a convolution whose
 * gathered rows have c_red channels and whose output rows have c_out channels
 * (forward: c_red = c_in; input gradient: c_red = c_out of the layer and the
 * output is c_in wide), else 0; a plan passed for another shape is ignored
 * and the map's row form is used.  Present engines: float32 with c_red, c_out
 * in {16, 32, 64} and S * c_red * c_out * 4 <= 147456, S = the offsets of a
 * plan range (K itself for K <= 32, ceil(K / ceil(K / 32)) for K <= 128: the
 * ranges run one after another, each adding its sums to the output rows);
 * bfloat16 (fp32 sums) with c_red, c_out in {64, 128, 256} and K <= 32. */
int32_t gsc_conv_block_engine(int32_t dtype, int32_t c_red, int32_t c_out, int32_t K);

/* ------------------------------------------------------------------------ */
/* a4 / a5. Convolution forward (Alg. 2), transposed convolution.           */
/* ------------------------------------------------------------------------ */
/* Workspace bytes for gsc_sparse_conv_fwd (0 when none is needed).  The
 * bfloat16 engines for wide layers (c_in in {32, 64, 128, 256}, c_out in {64,
 * 128, 256}, K <= 64) keep a transposed copy of W there (K * c_in * c_out * 2
 * bytes, rounded up to 256) followed by 256 bytes for the counter with which
 * the block engine hands out its tiles. */
size_t gsc_conv_fwd_ws_bytes(int32_t dtype, int32_t c_in, int32_t c_out, int32_t K);

/* Y = 0; for every offset k and pair p of it: Y[out_idx[p]] += X[in_idx[p]] W[k].
 *
 * dtype GSC_F32: X, W, Y float32.  GSC_BF16: X, W bfloat16, accumulation in
 * float32, Y rounded to bfloat16 (nearest even).  X: n_in x c_in, Y: n_out x
 * c_out (overwritten; rows without pairs become 0), W: K x c_in x c_out.
 * The map (in_idx, out_idx, seg, gidx, n_pairs) must be as gsc_kernel_map
 * produces it for n_out output rows: out_idx increasing within each offset
 * and gidx its 64-row group index.  (perm, bmask, ibase, items) is the map's
 * block plan (gsc_conv_plan), or all four NULL; when given and
 * gsc_conv_block_engine(dtype, c_in, c_out, K) is 1 (and X and W are 16-byte
 * aligned) the block engine computes Y from the plan, otherwise the map is
 * used.  Both give Eq. 3.  The block engines and the row form's specialised
 * float32 kernels add each output row's products in increasing offset order
 * (bit-reproducible); the general row-form kernel (other shapes, K > 64)
 * adds them into its LDS tile atomically, in no fixed order, so its last
 * bits can differ between calls.  The transposed convolution is this call on the
 * role-reversed map (see gsc_kernel_map).  ws: gsc_conv_fwd_ws_bytes
 * bytes of device memory (may be NULL when that is 0), contents not kept.
 * Asynchronous.  Errors: EINVAL, ESHORT (ws), EHIP. */
int gsc_sparse_conv_fwd(int32_t dtype, const void* X, int64_t n_in, int32_t c_in,
                        const void* W, int32_t c_out, int32_t K,
                        const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                        const int64_t* gidx, int64_t n_pairs,
                        const int32_t* perm, const uint32_t* bmask, const int64_t* ibase, const int32_t* items,
                        void* Y, int64_t n_out, void* ws, size_t ws_bytes, void* stream);

/* Forward convolution with a per-output-channel affine map and activation
 * fused into the kernel that writes Y (Sec. 4.5: batch normalisation, whose
 * inference form is an affine map per channel, and ReLU act on the feature
 * matrix alone, so they can be applied to each output row as it is produced):
 *   Y[j][c] = act(S[j][c] * scale[c] + shift[c]),
 * S = the sums of gsc_sparse_conv_fwd (same arguments, same meaning).  scale
 * and shift: device float32 arrays of c_out values, each nullable (null scale
 * = 1, null shift = 0); act: GSC_ACT_NONE or GSC_ACT_RELU (max(v, 0); NaN
 * passes through).  The map is applied to the float32 sums before bf16
 * rounding on the block engines; the row form applies it in a second pass
 * over Y (so a bf16 Y is rounded twice there).  A batch-normalised layer in
 * training takes scale = gamma / sqrt(var + eps), shift = beta - mean * scale
 * once its batch statistics are known.  Asynchronous.  Errors: as
 * gsc_sparse_conv_fwd, and EINVAL for an unknown act. */
typedef enum { GSC_ACT_NONE = 0, GSC_ACT_RELU = 1 } gsc_act;
int gsc_sparse_conv_fwd_affine(int32_t dtype, const void* X, int64_t n_in, int32_t c_in,
                               const void* W, int32_t c_out, int32_t K,
                               const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg,
                               const int64_t* gidx, int64_t n_pairs,
                               const int32_t* perm, const uint32_t* bmask, const int64_t* ibase,
                               const int32_t* items, const float* scale, const float* shift, int32_t act,
                               void* Y, int64_t n_out, void* ws, size_t ws_bytes, void* stream);

/* Backward of that epilogue (the chain rule of Y = act(S * scale + shift),
 * per element): with dY the gradient of Y (n x c, the dtype of Y) and G =
 * dY where the ReLU passed (Y > 0) or everywhere without it,
 *   dZ = G * scale            (n x c, Y's dtype: the dY of gsc_sparse_conv_bwd),
 *   dscale[c] = sum over rows of G * S,   dshift[c] = sum over rows of G
 * (float32, each nullable), S recovered from Y as (Y - shift) / scale, so a
 * channel with scale 0 gets a non-finite dscale (and a bf16 Y gives S to bf16
 * precision).  For batch normalisation with its statistics held fixed:
 * dgamma = (dscale - mean * dshift) / sqrt(var + eps), dbeta = dshift.
 * Y, scale, shift, act as passed to gsc_sparse_conv_fwd_affine.  ws:
 * gsc_affine_act_bwd_ws_bytes(n, c) bytes, needed only for the sums.  The
 * sums are added in a fixed order (deterministic).  Asynchronous.  Errors:
 * EINVAL, ESHORT (ws), EHIP. */
size_t gsc_affine_act_bwd_ws_bytes(int64_t n, int32_t c);
int gsc_affine_act_bwd(int32_t dtype, const void* Y, const void* dY, int64_t n, int32_t c, const float* scale,
                       const float* shift, int32_t act, void* dZ, float* dscale, float* dshift, void* ws,
                       size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* a6 / a7. Backward: dX and dW.                                             */
/* ------------------------------------------------------------------------ */
/* Workspace bytes for gsc_sparse_conv_bwd. */
size_t gsc_conv_bwd_ws_bytes(int64_t n_pairs, int32_t c_in, int32_t c_out, int32_t K);

/* Gradients of gsc_sparse_conv_fwd with the forward map (in_idx, out_idx, seg):
 *   dW[k] = sum over pairs p of offset k of X[in_idx[p]]^T dY[out_idx[p]]
 *           (float32, K x c_in x c_out; zero for an offset without pairs),
 *   dX[r] = sum over pairs (r, j) of offset k of dY[j] W[k]^T (n_in x c_in).
 * dX is computed on the dX map (t_in_idx, t_out_idx, t_seg, t_gidx, t_n_pairs):
 * the same pairs with roles reversed (t_in_idx = output rows, t_out_idx = input
 * rows, increasing within each segment, t_gidx its group index over n_in rows),
 * and t_wsel (host, K ints, a permutation of 0..K-1: each segment of the dX
 * map holds the pairs of one forward offset) names the offset whose weight
 * segment s of the dX map uses: dX[t_out_idx[p]] += dY[t_in_idx[p]]
 * W[t_wsel[s]]^T.  For the
 * role-reversed map from gsc_kernel_map t_wsel is the identity; for a stride-1
 * map whose offset set is symmetric the forward map itself serves, with
 * t_wsel[s] = the offset -o_s.  (t_perm, t_bmask, t_ibase, t_items) is the
 * dX map's block plan or all NULL, used as in gsc_sparse_conv_fwd when
 * gsc_conv_block_engine(dtype, c_out, c_in, K) is 1.
 * dX (nullable: skip) has X's dtype; dW (nullable: skip) is float32.  Both are
 * overwritten.  ws: gsc_conv_bwd_ws_bytes(n_pairs, c_in, c_out, K) bytes (only
 * needed when dW is computed; given in full, it also holds the counter with
 * which the bfloat16 block engine of dX hands out its tiles, large ones
 * first: without it dX takes longer).  The dW reduction order is fixed, so dW is
 * deterministic.  Asynchronous.  Errors: EINVAL (also a t_wsel that is not a
 * permutation), ESHORT (ws), EHIP. */
int gsc_sparse_conv_bwd(int32_t dtype, const void* X, const void* W, const void* dY,
                        int64_t n_in, int32_t c_in, int32_t c_out, int32_t K,
                        const int32_t* in_idx, const int32_t* out_idx, const int64_t* seg, int64_t n_pairs,
                        const int32_t* t_in_idx, const int32_t* t_out_idx, const int64_t* t_seg,
                        const int64_t* t_gidx, int64_t t_n_pairs, const int32_t* t_wsel,
                        const int32_t* t_perm, const uint32_t* t_bmask, const int64_t* t_ibase,
                        const int32_t* t_items,
                        void* dX, float* dW, int64_t n_out, void* ws, size_t ws_bytes, void* stream);

/* gsc_sparse_conv_bwd from the forward map alone (the form that needs no
 * caller-built dX map): X (n_in x c_in) and dY (n_out x c_out) are the
 * forward convolution's input and output gradient, W its K x c_in x c_out
 * weights, and (in_idx, out_idx, seg) its map with cap_pairs = the pair
 * arrays' length.  transpose = 0: the forward convolution ran the map as it
 * is (in_idx: rows of X, out_idx: rows of Y); transpose != 0: it was the
 * transposed convolution on that map (Sec. 4.2: out_idx rows of X, in_idx
 * rows of Y).  The call builds the dX map (gsc_kernel_map_transpose) and,
 * when a block engine applies, its plan (gsc_conv_plan) in ws, then computes
 * dX (nullable) and dW (nullable, float32) as gsc_sparse_conv_bwd does.  ws:
 * gsc_conv_bwd_fwdmap_ws_bytes(dtype, n_in, cap_pairs, c_in, c_out, K)
 * bytes.  Asynchronous; slower than gsc_sparse_conv_bwd with a dX map and
 * plan kept from the forward pass, which is what a training loop should use.
 * Errors: EINVAL, ESHORT (ws), EHIP. */
size_t gsc_conv_bwd_fwdmap_ws_bytes(int32_t dtype, int64_t n_in, int64_t cap_pairs, int32_t c_in, int32_t c_out,
                                    int32_t K);
int gsc_sparse_conv_bwd_fwdmap(int32_t dtype, const void* X, const void* W, const void* dY, int64_t n_in,
                               int32_t c_in, int32_t c_out, int32_t K, const int32_t* in_idx, const int32_t* out_idx,
                               const int64_t* seg, int64_t cap_pairs, int32_t transpose, void* dX, float* dW,
                               int64_t n_out, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Pooling over a kernel map (Sec. 4.3 max pooling, Alg. 3; Sec. 4.4         */
/* average and sum pooling, Alg. 4) and global pooling.  float32.            */
/* ------------------------------------------------------------------------ */
typedef enum { GSC_POOL_MAX = 0, GSC_POOL_AVG = 1, GSC_POOL_SUM = 2 } gsc_pool_mode;

/* Y[j] (n_out x C, overwritten) = the channel-wise maximum (MAX), mean (AVG)
 * or sum (SUM) of the input rows X[i] (n_in x C) paired with output row j in
 * the kernel map whose dense form is nbr (K x n_out int32, nbr[k*n_out + j]
 * = input row or -1, as gsc_kernel_map writes it; a pooling layer's map is
 * the kernel map of its window from the input table to its output
 * coordinates, e.g. gsc_coords_stride's).  An output without inputs is 0.
 * arg (n_out x C int32; required for MAX, else nullable): the input row
 * attaining the maximum, the first in offset order on ties (-1: none).  cnt
 * (n_out int32, nullable): the number of inputs of each output (Alg. 4's N).
 * Unpooling (the transposed pooling of Sec. 4.4) is this call in AVG or SUM
 * mode on the role-reversed map (the map gsc_sparse_pool_bwd takes: coarse
 * rows in, fine rows out): each fine row receives the mean or the sum of the
 * coarse rows it is pooled into; its gradient is gsc_sparse_pool_bwd on the
 * pooling's own map.
 * Asynchronous.  Errors: EINVAL, EHIP. */
int gsc_sparse_pool_fwd(int32_t mode, const float* X, int64_t n_in, int32_t C,
                        const int32_t* nbr, int32_t K, int64_t n_out,
                        float* Y, int32_t* arg, int32_t* cnt, void* stream);

/* dX (n_in x C, overwritten) = gradient of gsc_sparse_pool_fwd: each input row
 * i receives, for every output j it is paired with, dY[j] (SUM), dY[j] /
 * cnt[j] (AVG), or dY[j][c] in the channels c where arg[j][c] == i (MAX).
 * nbrT (K x n_in int32) is the dense form of the role-reversed map
 * (gsc_kernel_map on the output table with the input coordinates and the
 * negated offsets): nbrT[k*n_in + i] = the output fed by input i at offset
 * k, or -1.  arg is required for MAX, cnt for AVG.  The sum over outputs
 * runs in offset order (deterministic, no atomics).  Asynchronous.
 * Errors: EINVAL, EHIP. */
int gsc_sparse_pool_bwd(int32_t mode, const float* dY, int64_t n_out, int32_t C,
                        const int32_t* nbrT, int32_t K, int64_t n_in,
                        const int32_t* arg, const int32_t* cnt, float* dX, void* stream);

/* Global pooling (Sec. 4.4): every row of batch index b (column 0 of coords,
 * n x (1+D) int32) maps to output row b < n_batch <= 32; rows with a batch
 * index outside [0, n_batch) are ignored.  Y (n_batch x C), arg (n_batch x
 * C, required for MAX: the first row attaining the maximum) and cnt
 * (n_batch, nullable) as in gsc_sparse_pool_fwd.  ws:
 * gsc_global_pool_ws_bytes(n, C, n_batch) bytes of device memory (partial
 * reductions; contents not kept).  Asynchronous.  Errors: EINVAL, ESHORT, EHIP. */
size_t gsc_global_pool_ws_bytes(int64_t n, int32_t C, int32_t n_batch);
int gsc_global_pool_fwd(int32_t mode, const float* X, int64_t n, int32_t C, const int32_t* coords, int32_t D,
                        int32_t n_batch, float* Y, int32_t* arg, int32_t* cnt, void* ws, size_t ws_bytes,
                        void* stream);
/* dX (n x C, overwritten) = gradient of gsc_global_pool_fwd. */
int gsc_global_pool_bwd(int32_t mode, const float* dY, int32_t n_batch, int32_t C, const int32_t* coords, int32_t D,
                        int64_t n, const int32_t* arg, const int32_t* cnt, float* dX, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* GSC_H */
