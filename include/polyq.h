/*
 * polyq.h -- C ABI of the MI355X (gfx950) mixed-bit linear-layer library.
 *
 * The operation (PolyQ, Sec. 3-4): a linear layer y = x W^T whose input
 * channels each carry a bit-width from {2, 3, 4, 8, 16}.  At compile time the
 * input channels are permuted and clustered into bit-homogeneous blocks in
 * ascending bit order (Sec. 4.1, Eq. 9: O = A W = (A P^T)(P W)); every block of
 * b <= 8 bits is group-quantized (Sec. 3.4) with one fp16 scale s and one fp16
 * zero point z per output row and per group of 128 channels counted from the
 * block start; 16-bit channels are plain fp16 weights (Sec. 3.1: unquantized).
 * One kernel handles all blocks and accumulates them into one output
 * (Sec. 4.2):
 *
 *     y[m][n] = sum over clustered channels k' of  w_hat[n][k'] * x[m][perm[k']]
 *     w_hat[n][k'] = s[n][g] * (q[n][k'] - z[n][g])   (b <= 8)
 *     w_hat[n][k'] = fp16 weight                      (b = 16)
 *
 * Conventions for every call:
 *   - Shapes: W is n x k (out x in); codes, x and y are row-major.
 *   - Ownership: every array argument is caller-owned memory; the library
 *     allocates nothing, frees nothing and keeps no state between calls, so
 *     calls on different streams may run concurrently.  polyq_plan takes and
 *     writes host memory; every other pointer is device memory unless stated.
 *   - Streams: `stream` is a hipStream_t passed as void* (NULL = null stream).
 *     Device calls only enqueue work on it: they never synchronize the host.
 *   - Errors: argument, shape and capacity errors are detected on the host
 *     before any launch and return a non-zero status with no side effects.
 *     A failed launch returns POLYQ_ERR_DEVICE.  Device-side faults cannot be
 *     reported synchronously; indices read from device memory (perm) are
 *     range-checked in the kernels (an out-of-range entry reads as 0).
 *   - Aliasing: outputs must not overlap inputs.
 */
#ifndef POLYQ_H
#define POLYQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define POLYQ_MAX_BLOCKS 5    /* one block per bit-width in {2,3,4,8,16}            */
#define POLYQ_QUANTUM 32      /* every block length is a multiple of this (Sec. 3.3) */
#define POLYQ_GROUP 128       /* quantization group, counted from each block start   */
#define POLYQ_TILE_ROWS 64    /* output rows per packed tile                         */
#define POLYQ_MAX_M_GEMV 16   /* tokens per polyq_gemv call                          */
#define POLYQ_MAX_BATCH 8     /* linears per polyq_gemv_batch call                   */
#define POLYQ_MAX_K (1 << 20) /* input channels                                      */
#define POLYQ_MAX_N (1 << 24) /* output channels                                     */

typedef enum {
  POLYQ_OK = 0,
  POLYQ_ERR_ARG = 1,         /* null pointer, negative or zero size, bad enum value   */
  POLYQ_ERR_BITS = 2,        /* bit-width not in {2,3,4,8,16} or blocks not ascending */
  POLYQ_ERR_QUANTUM = 3,     /* a block length is not a positive multiple of 32      */
  POLYQ_ERR_SHAPE = 4,       /* block lengths do not sum to k, or n/k out of range    */
  POLYQ_ERR_CAPACITY = 5,    /* m too large, or workspace too small                   */
  POLYQ_ERR_UNSUPPORTED = 6, /* valid request this build cannot serve                 */
  POLYQ_ERR_DEVICE = 7       /* a HIP call failed                                     */
} polyq_status;

typedef struct {
  int32_t bits; /* 2, 3, 4, 8 or 16 */
  int32_t len;  /* channels, a positive multiple of POLYQ_QUANTUM */
} polyq_block;

/*
 * Layout of one packed linear (host POD, filled by polyq_plan).
 *
 * Packed buffer (device, 256-byte aligned base): the regions of the blocks in
 * block order, region i at block_offset[i].  A region holds n_tiles tiles of
 * 64 output rows (rows >= n are zero padding), tile t at
 * block_offset[i] + t * tile_bytes[i].  A tile holds the block's groups of 128
 * channels in order (the last one may hold 32, 64 or 96); group j of a tile
 * starts at j * record_bytes[i] and is
 *     [meta: 256 B, only for b <= 8][chunk 0][chunk 1]...  (up to 4 chunks of
 *     32 channels, chunk c at 256 + c * 256 * b for b <= 8, c * 4096 for b = 16).
 * Meta (fp16 bits): z of tile row R at half (R % 16) * 4 + R / 16, and s of row R
 *     at half 64 + ((R % 16) / 4) * 16 + (R / 16) * 4 + R % 4.
 * Chunk (64 rows x 32 channels, 256 * b bytes): 64 lane slices of 4 * b bytes,
 *     slice l at l * 4b.  Slice l holds channels 8 * (l / 16) .. + 7 of the four
 *     rows 16 * r + l % 16, r = 0..3 (the operand fragment a 64-lane 16x16x32
 *     matrix instruction takes per row sub-tile); its code i = 8 * r + t is row
 *     sub-tile r, channel 8 * (l / 16) + t.  Inside the slice's b words
 *     (32-bit, little endian):
 *   b = 2, 4, 8, 16: word d holds codes d*P .. d*P + P - 1, P = 32 / b; the
 *        even codes fill the low half and the odd codes the high half, in order:
 *        code d*P + 2p + h sits at bits [16h + b*p, 16h + b*p + b).
 *   b = 3: word d (d = 0,1,2) holds codes 10d .. 10d+9 as five pairs; pair p
 *        (codes 10d+2p, 10d+2p+1) sits at bits F..F+2 and 16+F..18+F with
 *        F = {0, 3, 6, 10, 13}[p]; codes 30 and 31 keep bit j in bit 9
 *        (code 30) and bit 25 (code 31) of word j.
 *   b = 16: the raw fp16 bits.
 * Every field of a 64-lane load is therefore one contiguous, aligned run of
 * 64 * 4b bytes.
 */
typedef struct {
  int32_t n;        /* output channels (rows)                          */
  int32_t k;        /* input channels                                  */
  int32_t nblocks;  /* 1 .. POLYQ_MAX_BLOCKS                           */
  int32_t n_groups; /* sum over blocks with b <= 8 of ceil(len / 128)  */
  int32_t n_tiles;  /* ceil(n / 64)                                    */
  int32_t n_chunks; /* k / 32                                          */
  polyq_block block[POLYQ_MAX_BLOCKS];
  int32_t k_begin[POLYQ_MAX_BLOCKS];     /* first clustered channel of the block     */
  int32_t group_begin[POLYQ_MAX_BLOCKS]; /* first group index of the block (b <= 8)   */
  int64_t block_offset[POLYQ_MAX_BLOCKS];/* byte offset of the block region           */
  int64_t tile_bytes[POLYQ_MAX_BLOCKS];  /* bytes per 64-row tile in the region       */
  int64_t record_bytes[POLYQ_MAX_BLOCKS];/* bytes of a full (4-chunk) group record    */
  int64_t packed_bytes;                  /* total packed-buffer size                  */
  int64_t code_bits;   /* n * sum_b b * len_b: B_real (Eq. 7) = code_bits / (n k) */
  int64_t weight_bytes;/* algorithmic bytes of one pass: code_bits/8 + n*n_groups*4 */
} polyq_layout;

/*
 * polyq_plan -- validate a block list and compute the packed layout (host only,
 * no HIP call).  blocks: host array of nblocks entries with strictly ascending
 * bits from {2,3,4,8,16} and lengths that are positive multiples of 32 summing
 * to k (the quanta-matched block sizes of Sec. 3.3).  On error *out is left
 * unchanged.
 */
polyq_status polyq_plan(int32_t n, int32_t k, const polyq_block* blocks, int32_t nblocks,
                        polyq_layout* out);

/*
 * polyq_pack -- write the packed buffer of a layer (compile-time step of
 * Sec. 4.1: only the clustered weight P W is materialized).
 *   codes  [n][k] uint16, clustered channel order: the code q for b <= 8
 *          (only the low b bits are stored), the fp16 bit pattern for b = 16.
 *   scales [n][n_groups] fp16 bits, zeros [n][n_groups] fp16 bits
 *          (ignored when n_groups == 0).
 *   packed layout->packed_bytes bytes, 256-byte aligned; fully overwritten.
 */
polyq_status polyq_pack(const polyq_layout* layout, const uint16_t* codes, const uint16_t* scales,
                        const uint16_t* zeros, void* packed, void* stream);

/*
 * polyq_pack_rows -- polyq_pack with the output rows reordered: the producer
 * side of the cross-layer permutation merge (Sec. 4.3, Eq. 10).  A consumer
 * that wants its input in basis P (its own channel permutation) receives it
 * without an activation shuffle when the producer's weight is stored as
 * W P^T, i.e. with its output rows permuted by P at compile time.
 *   row_perm  int32 [n] (device, not NULL): packed row r holds source row
 *             row_perm[r] of codes, scales and zeros, so polyq_gemv /
 *             polyq_gemm on the packed buffer produce y'[i][r] =
 *             y[i][row_perm[r]].  Passing the consumer's perm (consumer k ==
 *             producer n) makes y' the consumer's clustered input (call it
 *             with perm = NULL).  An entry outside [0, n) packs a zero row
 *             (codes, scales and zeros 0): its output is 0.
 *   Other arguments, layout and errors as for polyq_pack (NULL row_perm:
 *   POLYQ_ERR_ARG).  codes, scales, zeros and row_perm are read only.
 */
polyq_status polyq_pack_rows(const polyq_layout* layout, const uint16_t* codes,
                             const uint16_t* scales, const uint16_t* zeros,
                             const int32_t* row_perm, void* packed, void* stream);

/*
 * polyq_unpack -- inverse of polyq_pack: writes codes [n][k], scales and zeros
 * [n][n_groups] (fp16 bits) from a packed buffer.  Any of the three outputs may
 * be NULL to skip it.  Codes of b <= 8 come back masked to b bits.
 */
polyq_status polyq_unpack(const polyq_layout* layout, const void* packed, uint16_t* codes,
                          uint16_t* scales, uint16_t* zeros, void* stream);

/*
 * polyq_permute -- the explicit activation shuffle of Sec. 4.1 / Eq. 9:
 * x_out[i][k'] = x[i][perm[k']] for i < m, k' < k, for any 2-byte element type
 * (fp16 or bf16).  perm: int32 [k] (device).  An entry outside [0, k) yields 0.
 * m * k must not exceed 2^31 - 1 elements (else POLYQ_ERR_CAPACITY, before any
 * launch).
 */
polyq_status polyq_permute(const int32_t* perm, const uint16_t* x, uint16_t* x_out, int32_t m,
                           int32_t k, void* stream);

/*
 * polyq_gemv -- decode / small-batch product, 1 <= m <= 16 tokens: the
 * clustered product of Eq. 9 (x P^T times P W), one kernel over all bit blocks
 * accumulating into one output (Sec. 4.2), dequantized as in Sec. 3.4:
 *   y[i][n] = sum_k' w_hat[n][k'] * x[i][perm[k']]   (fp32 accumulation)
 *   packed  buffer written by polyq_pack for `layout`.
 *   perm    int32 [k] (device, 16-byte aligned), or NULL when x is already in
 *           clustered order.
 *   x       fp16 [m][k] bits (16-byte aligned).   y fp32 [m][n], fully overwritten.
 *   workspace / workspace_bytes: device memory of at least
 *           polyq_gemv_workspace_bytes(layout, m) bytes (enough with or
 *           without a permutation; may be NULL when that is 0), 256-byte
 *           aligned, laid out as for polyq_gemv_batch with one item: its
 *           first polyq_gemv_batch_workspace_zero_bytes bytes (the split-K
 *           state) must be zero on entry and are zero again when the call
 *           completes; the bytes after them are scratch that the call
 *           overwrites (a clustered copy of x for several tokens, or for a row
 *           too long for the kernel's LDS).  Calls that share a workspace must
 *           be ordered (same stream).
 * Precision: for zero points that are integers of magnitude <= 1023 every
 * w_hat * x product is exact in fp32 (q - z is an exact integer, s is applied
 * once per group) and only fp32 accumulation rounds.  Any other z is applied
 * as zi = rint(z) (clamped to [-1023, 1023]) plus the fp32 correction
 * -(z - zi) * sum x' per group.  |y - y_ref| <= 1e-3 * sum |w_hat x|.
 */
size_t polyq_gemv_workspace_bytes(const polyq_layout* layout, int32_t m);
polyq_status polyq_gemv(const polyq_layout* layout, const void* packed, const int32_t* perm,
                        const uint16_t* x, int32_t m, float* y, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Size of the device array behind polyq_gemv_batch_noalloc (per GPU). */
#define POLYQ_NOALLOC_SCRATCH_BYTES (16u << 20)

/*
 * polyq_gemv_batch -- up to POLYQ_MAX_BATCH independent decode products in one
 * launch (e.g. the q/k/v projections, or gate/up, which share x and perm):
 * item i computes exactly what polyq_gemv(items[i].layout, items[i].packed,
 * items[i].perm, items[i].x, m, items[i].y, ...) computes, with the same
 * argument rules per item.  Items may share x and perm; no y may overlap any
 * input or another y.  The work split of every item is sized for the whole
 * launch, so the workspace is queried for the batch:
 *   workspace of at least polyq_gemv_batch_workspace_bytes(items, count, m)
 *   bytes, 256-byte aligned (the queries read the layout, perm and x fields of
 *   each item and return 0 on an invalid request).  It holds two parts:
 *     [0, Z)  Z = polyq_gemv_batch_workspace_zero_bytes(items, count, m): the
 *             split-K counters and partial sums.  Must be zero on entry; every
 *             completed call leaves them zero.
 *     [Z, ..) scratch: one clustered copy x' = x[:, perm] (times xscale)
 *             per distinct (x, perm, xscale) of the items with several tokens
 *             and a permutation or a scale; overwritten by the call (Eq. 9's
 *             explicit shuffle, made once per launch).
 *   A workspace reused for requests of different shapes must therefore be
 *   zeroed again up to the new request's Z wherever an earlier call left
 *   scratch there.
 */
typedef struct {
  const polyq_layout* layout;
  const void* packed;
  const int32_t* perm; /* may be NULL (x already clustered) */
  const uint16_t* x;   /* fp16 [m][k] */
  float* y;            /* fp32 [m][n] */
  /* Bit-specific activation-aware scaling (Sec. 3.4, Eq. 8): fp16 [k] per
   * clustered channel, the factor 1/s_j folded into the activations,
   * x'[m][k'] = x[m][perm[k']] * xscale[k'], for weights packed from
   * Q_b(diag(s) W); NULL (the default of a zero-initialized item) for none.
   * The product is formed in fp32 and rounded to the activation type, so a
   * power of two (what polyq_bit_scaling produces) is applied exactly.  For
   * several tokens, and in the prefill GEMM, the scaled x' is written to the
   * workspace's scratch part first (also without a permutation).  Device
   * memory, 16-byte aligned for polyq_gemv_batch (read as 16-byte vectors;
   * POLYQ_ERR_ARG otherwise), any alignment for polyq_gemm_batch. */
  const uint16_t* xscale;
} polyq_gemv_item;

size_t polyq_gemv_batch_workspace_bytes(const polyq_gemv_item* items, int32_t count, int32_t m);
size_t polyq_gemv_batch_workspace_zero_bytes(const polyq_gemv_item* items, int32_t count, int32_t m);
polyq_status polyq_gemv_batch(const polyq_gemv_item* items, int32_t count, int32_t m,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * polyq_gemv_batch_noalloc -- polyq_gemv_batch without a workspace argument,
 * for callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  The workspace is a
 * fixed array of POLYQ_NOALLOC_SCRATCH_BYTES bytes inside this library, one
 * copy per GPU, held until the process ends; the call allocates and frees
 * nothing.  Arguments and results as for polyq_gemv_batch (same kernels).
 *   - A request whose workspace (polyq_gemv_batch_workspace_bytes) exceeds
 *     POLYQ_NOALLOC_SCRATCH_BYTES returns POLYQ_ERR_CAPACITY before any launch.
 *   - The library keeps, per GPU, how much of the array is known to be zero;
 *     a call whose split-K state reaches past that clears the difference on
 *     `stream` (one kernel) before the product (the first call on a GPU
 *     always does).
 *   - All calls on one GPU share its array: calls that may overlap (e.g. on
 *     different streams without ordering) race and give undefined results.
 */
polyq_status polyq_gemv_batch_noalloc(const polyq_gemv_item* items, int32_t count, int32_t m,
                                      void* stream);

/*
 * polyq_gemm -- prefill product for any m >= 1 (bf16 activations): the same
 * clustered product (Eq. 9; all blocks into one output, Sec. 4.2) as a dense
 * contraction on the matrix cores:
 *   y[i][n] = sum_k' w_hat[n][k'] * x[i][perm[k']]
 *   x bf16 [m][k] bits, original channel order if perm != NULL, else clustered
 *   (then 16-byte aligned); m * k * 2 < 2^31.
 *   y fp32 [m][n], fully overwritten.
 *   workspace: at least polyq_gemm_workspace_bytes(layout, m, perm != NULL)
 *   bytes of device scratch (the permuted activations when perm != NULL, and
 *   per-split partial sums when the launch splits K, which it does when the
 *   output tiles alone would leave most compute units idle); contents on
 *   entry are ignored.  The split sums are added in a fixed order, so results
 *   do not depend on scheduling.
 * Computed with bf16 MFMA and fp32 accumulation: (q - z) enters as one exact
 * bf16 value when z is an integer in [0, 255]; for any other fp16 z, q - z is
 * formed in fp32 from exact operands with one rounding (relative error at most
 * 2^-24) and enters as the bf16 pair hi + lo (together within 2^-16 relative of
 * q - z); the group scale is applied in fp32; a 16-bit channel enters as the
 * exact bf16 pair hi + lo of its fp16 weight.  |y - y_ref| <= 1e-3 *
 * sum |w_hat x| for any fp16 scale and zero point.
 */
size_t polyq_gemm_workspace_bytes(const polyq_layout* layout, int32_t m, int perm_given);
polyq_status polyq_gemm(const polyq_layout* layout, const void* packed, const int32_t* perm,
                        const uint16_t* x, int32_t m, float* y, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * polyq_gemm_batch -- up to POLYQ_MAX_BATCH independent prefill products in
 * one launch (e.g. q/k/v, or gate/up, which share x and perm): item i computes
 * what polyq_gemm(items[i].layout, items[i].packed, items[i].perm, items[i].x,
 * m, items[i].y, ...) computes, with the same argument rules per item (x holds
 * bf16 bits here).  Items with the same x and perm share one permuted copy.
 *   workspace: at least polyq_gemm_batch_workspace_bytes(items, count, m)
 *   bytes of device scratch (the permuted copies, and for count == 1 the
 *   split partial sums as in polyq_gemm); contents on entry are ignored.  The
 *   query reads the layout, x and perm fields; 0 on an invalid request or
 *   when no scratch is needed.
 */
typedef polyq_gemv_item polyq_gemm_item;

size_t polyq_gemm_batch_workspace_bytes(const polyq_gemm_item* items, int32_t count, int32_t m);
polyq_status polyq_gemm_batch(const polyq_gemm_item* items, int32_t count, int32_t m,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * polyq_read_probe -- measurement utility, not part of the linear-layer
 * computation: reads `bytes` bytes of device memory once and discards them
 * (each of at most work_groups work-groups reads one contiguous share).  The
 * time of this launch is the reference read rate of a launch of that size,
 * against which the decode GEMV's weight stream is measured.
 *   buf: device, 16-byte aligned; bytes: a positive multiple of 16.
 *   sink: device array of work_groups uint32, written only when a checksum
 *         takes one particular value (contents afterwards unspecified).
 *   bytes / work_groups must stay below 2^30 (else POLYQ_ERR_CAPACITY).
 */
polyq_status polyq_read_probe(const void* buf, int64_t bytes, int32_t work_groups, uint32_t* sink,
                              void* stream);

/*
 * ---- Compile-time bit allocation (Sec. 3.1-3.3) --------------------------
 * Host functions on host memory: synchronous, no device work, no global
 * state (thread-safe).  Arrays indexed by bit-width use the palette order
 * {2, 3, 4, 8, 16} (index 0 .. 4).  Channels are input channels in their
 * original order.  Every error is detected before any output is written.
 */
#define POLYQ_NUM_BITS 5

/*
 * polyq_channel_error -- the activation-aware error proxy of Eq. 2 for every
 * input channel and bit-width, E_b[j] = ||w~_j - w_j||^2 * E[x_j^2], with the
 * scaled-and-quantized weight of Eq. 1, W~ = diag(s)^-1 Q_b(diag(s) W).
 *   w:     fp32 [n][k] row-major (output rows x input channels);
 *   x2:    fp64 [k], E[x_j^2] (finite, >= 0);
 *   scale: fp32 [k] per-channel scales s_j (finite, > 0), or NULL for all 1;
 *   err:   fp64 [POLYQ_NUM_BITS][k] out.
 * Q_b is this library's asymmetric min-max quantizer applied per output row
 * to groups of 128 consecutive input channels (the last group partial):
 * s16 = fp16_rne((max - min) / (2^b - 1)), z = clamp(rint(-min / s16), 0,
 * 2^b - 1), q = clamp(rint(w / s16) + z, 0, 2^b - 1), value s16 (q - z), all in
 * fp64 with rint rounding half to even; a group whose s16 is 0 quantizes to 0.
 * E_16 = 0 (16-bit channels are unquantized).
 * Errors: POLYQ_ERR_ARG (null pointer, n or k < 1, an x2 or scale value out of
 * range); POLYQ_ERR_SHAPE (n * k above 2^31).
 */
polyq_status polyq_channel_error(const float* w, int32_t n, int32_t k, const double* x2,
                                 const float* scale, double* err);

/*
 * polyq_waterfill -- per-layer greedy waterfilling under the fractional
 * budget B (Sec. 3.2, Eq. 3-5).  Every channel starts at 2 bits; the budget
 * left is round(B k) - 2 k (round half to even; nothing happens when it is
 * <= 0).  Each channel's next upgrade b -> b' (the next palette value) waits
 * in a max-heap keyed by the gain (E_b[j] - E_b'[j]) / (b' - b), ties to the
 * lower channel index; the top upgrade is applied if it fits the budget left
 * (else dropped: the budget only shrinks) and the channel's next upgrade is
 * pushed, until the budget is spent or the heap is empty.
 *   err: fp64 [POLYQ_NUM_BITS][k] (polyq_channel_error's layout); bits: [k] out.
 * Errors: POLYQ_ERR_ARG (null pointer, k < 1, B not finite or above 16).
 */
polyq_status polyq_waterfill(const double* err, int32_t k, double budget, int32_t* bits);

/*
 * polyq_quanta_match -- ISA-aware quanta matching (Sec. 3.3, Eq. 6-7): the
 * per-bit channel counts of `bits` are rounded to multiples of `quantum`
 * (floors in units of the quantum, the units left to the largest remainders,
 * ties to the higher bit-width); whole-quantum moves between neighbouring
 * levels then bring sum_b b c_b closer to round(B k) while one is strictly
 * better (largest improvement first, ties to the lower pair, promotion
 * first); finally single channels move between neighbouring levels until the
 * counts match: across the lowest boundary whose flow is nonzero and whose
 * source level is not empty, the channel with the largest gain is promoted
 * (or the smallest loss demoted), ties to the lower channel index.
 *   bits: [k] in (palette values) and out; counts: [POLYQ_NUM_BITS] out, or
 *   NULL; B_real = sum_b bits b counts[b] / k (Eq. 7).
 * Errors: POLYQ_ERR_ARG (null pointer, k < 1, quantum < 1, B not finite, a
 * bit-width outside the palette); POLYQ_ERR_QUANTUM (k not a multiple of
 * quantum).
 */
polyq_status polyq_quanta_match(const double* err, int32_t k, int32_t quantum, double budget,
                                int32_t* bits, int32_t* counts);

/*
 * polyq_cluster -- channel clustering (Sec. 4.1, Eq. 9): blocks in ascending
 * bit-width, ascending original index inside a block.
 *   bits: [k] palette values; perm: [k] out, perm[k'] = original channel at
 *   clustered position k'; blocks: [POLYQ_MAX_BLOCKS] out (bits, len) and
 *   *nblocks: the number of nonempty blocks.  The block list is what
 *   polyq_plan takes once every length is a multiple of POLYQ_QUANTUM.
 * Errors: POLYQ_ERR_ARG (null pointer, k < 1, a bit-width outside the palette).
 */
polyq_status polyq_cluster(const int32_t* bits, int32_t k, int32_t* perm, polyq_block* blocks,
                           int32_t* nblocks);

/*
 * polyq_bit_scaling -- bit-specific activation-aware scaling (Sec. 3.4,
 * Eq. 8), run after the bit map is fixed: for every bit-width b <= 8 present,
 * one exponent alpha_b from `grid` (values in [0, 1]) for all its channels,
 * s_j = 2^rint(alpha_b log2 m_j) (Eq. 8's power law kept to powers of two,
 * so that the runtime fold of 1/s_j into x' is exact; the exponent is clamped
 * to [-14, 14], so that 1/s_j is a normal fp16 value), chosen to minimize the
 * block's proxy error sum_j E_b[j] (Eq. 2, x2 weights) with W~ =
 * diag(s)^-1 Q_b(diag(s) W) and Q_b applied as deployed: to the block's
 * channels in ascending index order, groups of 128 per row.  Ties keep the
 * earlier grid point; 16-bit channels get s = 1.
 *   w: fp32 [n][k]; x2: fp64 [k] >= 0; saliency: fp64 [k] m_j > 0 (e.g. mean
 *   |x_j| normalized by its mean); bits: [k] palette values; grid: [ngrid];
 *   scale: fp32 [k] out (powers of two); alpha: [POLYQ_NUM_BITS] out or NULL
 *   (0 for absent bit-widths and for 16 bits).
 * The weights to pack are then Q_b(diag(s) W), and the channel factors passed
 * with them (polyq_gemv_item.xscale) are 1/s in clustered order.
 * Errors: POLYQ_ERR_ARG (null pointer, n, k or ngrid < 1, a value out of
 * range); POLYQ_ERR_SHAPE (n * k above 2^31).
 */
polyq_status polyq_bit_scaling(const float* w, int32_t n, int32_t k, const double* x2,
                               const double* saliency, const int32_t* bits, const float* grid,
                               int32_t ngrid, float* scale, float* alpha);

/* Static description of a status code (never NULL). */
const char* polyq_status_str(polyq_status status);

#ifdef __cplusplus
}
#endif

#endif /* POLYQ_H */
