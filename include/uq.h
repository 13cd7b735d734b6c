/*
 * uq.h -- C ABI of libuq, the MI355X (gfx950) implementation of the unbiased
 * single-scale and multi-scale max-norm quantisers of "Unbiased Single-scale
 * and Multi-scale Quantizers for Distributed Optimization" (arXiv 2109.12497).
 *
 * One aggregation step of Algorithm 1 (one scale) or Algorithm 2 (several
 * scales) for M workers' flat fp32 gradients g^m in R^d is the sequence
 *
 *   uq_shared_scale     W = max_m ||g^m||_2 and, for several scales, the
 *                       shared per-coordinate scale index;
 *   uq_quantize_single  or uq_quantize_multi: the integer codes of each worker;
 *   uq_sum_codes        the all-reduce of the codes (an exact integer sum);
 *   uq_dequantize       the averaged gradient reconstructed from the sum
 *                       (uq_sum_dequantize does these two in one pass).
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers, except `scales`, which is a HOST
 *     array of K floats.  The caller owns every buffer; the library never
 *     allocates device memory and keeps no state between calls (the two test
 *     hooks at the end set process-wide options that change how work is
 *     launched or searched, never a result).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *     asynchronously on it; no entry point synchronises.  Argument checks are
 *     done on the host before anything is enqueued; on an error nothing is
 *     enqueued and no output is touched.
 *   - Gradients are row-major [rows][ldg] fp32 with ldg >= d, ldg % 4 == 0;
 *     only the first d entries of a row are read.  Codes are row-major
 *     [rows][ldc] int8 with ldc >= d, ldc % 16 == 0; only the first d bytes
 *     of a row are written.  Every array pointer must be 16-byte aligned
 *     (`w` 4-byte aligned).
 *   - Scale sets: 1 <= K <= 16 strictly increasing integral floats
 *     s_0 < ... < s_{K-1} with 1 <= s_0 <= 127 (|code| <= s_0 fits int8).
 *     The single-scale call takes s in [1, 127] and is the case K = 1.
 *   - Data-dependent conditions are never errors.  A scale W that is not a
 *     positive finite number, or for which s_0 / W overflows, selects the zero
 *     path: every code is 0, every scale index K-1, every output 0.  Zero,
 *     NaN and infinite gradient coordinates get code 0 (and a row holding a
 *     NaN or infinity has a non-finite norm, hence the zero path).
 *   - d == 0 is a valid no-op (uq_shared_scale still writes W = 0).
 *
 * Arithmetic contract (bit-exact, independent of launch geometry)
 *   inv_k = RN32(s_k / W), deq_k = RN32(W / (M * s_k)).
 *   Scale index (Eq. (11), shared by the minimum over workers): for each
 *   worker the largest k with RN32(|g| * inv_k) <= s_0 (none: 0; zero or
 *   non-finite |g|: K-1); the shared index is the minimum over the workers.
 *   Code (Eq. (8) / Eq. (12)): x = min(RN32(|g| * inv_k), s_0), l = floor(x),
 *   t = floor((x - l) * 2^32); code = sign(g) * (l + [r < t]), where the
 *   32-bit uniform word r of worker m at coordinate i has as its high half
 *   the 16-bit half (i mod 8) of Philox4x32-10 block
 *   (key = seed, counter = (i / 8, m, 0)) and as its low half the same half
 *   of block (i / 8, m, 1); half h of a block is bits 16*(h / 4) .. +15 of
 *   word h mod 4.
 *   Reconstruction (Eq. (9) / Eq. (13) with 1/M): out_i = RN32(sum_i * deq_k).
 *   The norm is an fp64 sum of exact fp32 squares in a fixed order that
 *   depends only on d and on the pass that forms it (one scale or more than
 *   16 rows or one row: the norm pass alone; several scales and 2 to 16 rows: the
 *   pass that also takes the rows' maxima), so W is deterministic; it can
 *   differ from a sequential fp64 sum by at most one binary32 ulp.
 */
#ifndef UQ_H
#define UQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum uq_status {
    UQ_OK = 0,
    UQ_EINVAL = -1,     /* null pointer, negative size, rows/M < 1, ld < d, size overflow */
    UQ_ERANGE = -2,     /* scale set, s, K, M * s_k or worker ids out of range        */
    UQ_EALIGN = -3,     /* misaligned pointer or leading dimension                    */
    UQ_EWORKSPACE = -4, /* workspace smaller than uq_workspace_bytes(d, M)            */
    UQ_EHIP = -5        /* the HIP runtime refused a launch (see uq_last_error)       */
};

#define UQ_MAX_SCALES 16

/*
 * Shared scale of Sec. 3.1/3.2: W = max_m ||g^m||_2 (the all-reduce of the
 * norms by maximum in Algorithm 1 and Algorithm 2), and for K > 1 also the shared scale index
 * of Sec. 3.2 (the per-coordinate rule Eq. (11) followed by scale sharing,
 * s*_i = min_m s*^m_i).
 *   g        [M][ldg] fp32, the M workers' gradients (read)
 *   scales   host array of K floats (may be NULL when K == 1)
 *   w        one fp32 (written): W
 *   idx      [d] uint8 (written when K > 1, may be NULL when K == 1): the
 *            shared scale index k*_i in 0..K-1
 *   ws       device workspace of at least uq_workspace_bytes(d, M) bytes,
 *            16-byte aligned; its contents are scratch
 */
int uq_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg,
                    const float* scales, int32_t K, float* w, uint8_t* idx,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * uq_shared_scale with the shared index stored as 4-bit fields: coordinate i's
 * k*_i in the low nibble of idx4[i / 2] for even i and in the high nibble for
 * odd i (the high nibble of the last byte is 0 when d is odd).  Bit for bit
 * the same W and index values as uq_shared_scale (Sec. 3.2, Eq. (11) with
 * scale sharing); the index takes half the bytes, and so does every pass
 * that reads it (uq_quantize_sum_idx4).
 *   idx4   [(d + 1) / 2] uint8 (written), 16-byte aligned
 *   every other argument and check as for uq_shared_scale; K < 2 returns
 *   UQ_EINVAL (one scale has no index)
 */
int uq_shared_scale_idx4(const float* g, int64_t d, int32_t M, int64_t ldg,
                         const float* scales, int32_t K, float* w, uint8_t* idx4,
                         void* ws, size_t ws_bytes, void* stream);

/*
 * uq_shared_scale for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same checks, kernels and results, bit for bit, with the scratch taken
 * from a static device buffer of UQ_NOALLOC_SCRATCH_BYTES bytes that the
 * library holds on each device it runs on until the process ends.  The call
 * itself allocates nothing; its first call on a device looks up that
 * device's buffer (the current device, which the stream must belong to).
 *   Limit: the scratch the kernels need must fit the buffer.  With one
 *   scale, or more than 16 rows, or one row, that is 8 * M * ceil(d / c)
 *   bytes with c >= 8192 chunks of at most 1024 per row: any d for
 *   M <= 8192.  With several scales and 2 to 16 rows the pass keeps a
 *   16-bit key of the row maximum (2 * d bytes) and one fp64 partial per
 *   row and 1024 coordinates (8 * M * d / 1024 bytes): d up to about 33.3
 *   million with 2 rows, 32.5 million with 8 and 31.6 million with 16.  A
 *   call beyond the limit returns UQ_EWORKSPACE and launches nothing.
 *   Every call on one device shares that device's buffer (nothing in it
 *   needs to start at zero): calls that overlap on one device, on different
 *   streams or threads, race and give undefined results.
 * Arguments as for uq_shared_scale, without ws and ws_bytes.
 */
#define UQ_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int uq_shared_scale_noalloc(const float* g, int64_t d, int32_t M, int64_t ldg,
                            const float* scales, int32_t K, float* w, uint8_t* idx,
                            void* stream);

/* Workspace bytes uq_shared_scale needs for (d, M) and any K; 0 never
 * returned.  With 2 <= M <= 16 this includes 2 * d bytes: with several scales
 * the norm pass also keeps a 16-bit key of the largest |g| over the rows
 * (its exponent and top 8 mantissa bits) at every coordinate, so that the index pass need not read the gradients
 * again (except at the rare coordinates whose key equals a scale limit's). */
size_t uq_workspace_bytes(int64_t d, int32_t M);

/*
 * Single-scale quantiser Q_s of Eq. (7)-(8) (Sec. 3.1): the integer codes
 * zeta = sign(g_i) * s * xi_i of `rows` workers.
 *   g        [rows][ldg] fp32 (read); row r is worker worker0 + r
 *   w        device pointer to W (one fp32, read)
 *   s        number of levels, 1..127
 *   seed     Philox key
 *   codes    [rows][ldc] int8 (written)
 * A call with rows = R equals R calls with rows = 1 and consecutive worker0.
 * worker0 >= 0 and worker0 + rows <= 2^31.
 */
int uq_quantize_single(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                       const float* w, int32_t s, uint64_t seed, int8_t* codes, int64_t ldc,
                       void* stream);

/*
 * Multi-scale quantiser Q_S of Eq. (10) and (12) (Sec. 3.2) with the shared
 * scale index from uq_shared_scale: coordinate i of every worker is
 * quantised on the grid of s*_i = scales[idx[i]] levels; |code| <= s_0.
 *   idx      [d] uint8 (read); entries >= K are read as K-1
 * Other arguments as for uq_quantize_single.
 */
int uq_quantize_multi(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                      const float* w, const float* scales, int32_t K, const uint8_t* idx,
                      uint64_t seed, int8_t* codes, int64_t ldc, void* stream);

/*
 * The all-reduce of Algorithm 1/2 (the step the quantisers keep compatible
 * with aggregation, Sec. 3.1): sum_i = sum over the rows of code_{r,i}, exact
 * in int32.
 *   codes       [rows][ldc] int8 (read)
 *   accumulate  0: sum = the rows' total; 1: sum += the rows' total
 *   sum         [d] int32 (written, or read and written)
 * rows <= 2^24 per call; keeping a running sum in range over many
 * accumulating calls is the caller's concern.
 */
int uq_sum_codes(const int8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t accumulate,
                 int32_t* sum, void* stream);

/*
 * Reconstruction R of Eq. (9) (one scale) / Eq. (13) (several scales) applied
 * to the summed codes, with the 1/M of the averaging step of Algorithm 1/2:
 * out_i = W * sum_i / (M * s*_i).
 *   sum      [d] int32 (read)
 *   M        number of workers whose codes were summed
 *   scales   host array of K floats; for one scale K = 1 and scales = {s}
 *   idx      [d] uint8 shared scale index; must be NULL iff K == 1
 *   out      [d] fp32 (written)
 * M * s_k must be exactly representable in fp32 and M * s_0 < 2^31.
 */
int uq_dequantize(const int32_t* sum, int64_t d, int32_t M, const float* w,
                  const float* scales, int32_t K, const uint8_t* idx, float* out, void* stream);

/*
 * uq_sum_codes (bits = 8) or uq_sum_packed (bits = 4 or 2) followed by
 * uq_dequantize on the sums, in one pass: the same sum and out, bit for bit,
 * without reading the sums back.  The reconstruction is applied to the
 * stored sums, so with accumulate = 1 it sees the running total.
 *   codes    [rows][ldc] int8 codes (bits = 8) or packed rows (bits = 4, 2)
 *   sum      [d] int32 (written, or read and written)
 *   M, w, scales, K, idx, out   as for uq_dequantize
 * The checks of both calls apply.
 */
int uq_sum_dequantize(const uint8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t bits,
                      int32_t accumulate, int32_t* sum, int32_t M, const float* w, const float* scales,
                      int32_t K, const uint8_t* idx, float* out, void* stream);

/*
 * Quantise and sum in one pass: the codes of uq_quantize_single (K = 1,
 * scales = {s}) or uq_quantize_multi (K > 1) for `rows` workers, added into
 * the int32 sum without being stored anywhere: Eq. (8) / Eq. (12) and the
 * all-reduce of Algorithm 1/2 fused.  With out != NULL the reconstruction of
 * Eq. (9) / Eq. (13) with the 1/M of the averaging step is applied to the
 * sums as they are stored (the rule of uq_dequantize).  Bit for bit the same
 * sum and out as uq_quantize_* followed by uq_sum_codes (and uq_dequantize);
 * a worker streamed through a resident accumulator is one call with
 * rows = 1, accumulate = 0 for the first worker and 1 after it, and out set
 * on the last.
 *   g, d, rows, ldg, worker0, w, seed   as for uq_quantize_single
 *   scales, K, idx   as for uq_quantize_multi; idx is not read when K == 1
 *   accumulate       0: sum = the rows' total; 1: sum += the rows' total
 *   sum              [d] int32 (written, or read and written)
 *   M, out           NULL: no reconstruction (M is then ignored); else out
 *                    [d] fp32 (written) and M as for uq_dequantize, whose
 *                    checks then apply
 * Keeping a running sum in range over many accumulating calls is the
 * caller's concern.
 */
int uq_quantize_sum(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                    const float* w, const float* scales, int32_t K, const uint8_t* idx,
                    uint64_t seed, int32_t accumulate, int32_t* sum, int32_t M, float* out,
                    void* stream);

/*
 * uq_quantize_sum reading the shared index as 4-bit fields (the layout of
 * uq_shared_scale_idx4): bit for bit the same sum and out as uq_quantize_sum
 * given the same index values (Eq. (12), the all-reduce of Algorithm 2 and
 * Eq. (13)).  A streamed worker then reads half a byte of index per
 * coordinate instead of one.
 *   idx4   [(d + 1) / 2] uint8 (read), 16-byte aligned
 *   every other argument and check as for uq_quantize_sum; K < 2 returns
 *   UQ_EINVAL
 */
int uq_quantize_sum_idx4(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                         const float* w, const float* scales, int32_t K, const uint8_t* idx4,
                         uint64_t seed, int32_t accumulate, int32_t* sum, int32_t M, float* out,
                         void* stream);

/*
 * The shared scale index of Sec. 3.2 (the rule of Eq. (11) with scale
 * sharing) formed inside the quantise-and-sum over all M workers: Eq. (12),
 * the all-reduce of Algorithm 2 and the reconstruction of Eq. (13) with the
 * 1/M of the averaging step, in one pass over the gradients.  Bit for bit the
 * idx of uq_shared_scale followed by uq_quantize_sum over all M rows
 * (worker0 = 0, accumulate = 0, out set), given the same W.  Every row of a
 * tile is held in registers, so each coordinate's index comes from its exact
 * largest usable |g| over the rows; uq_shared_scale then only has to form W,
 * which does not depend on the scales (call it with K = 1 and idx = NULL).
 *   g        [M][ldg] fp32, 1 <= M <= 16; row m is worker m
 *   w        device pointer to W (one fp32, read)
 *   scales   host array of K floats, 1 <= K <= UQ_MAX_SCALES, as for
 *            uq_quantize_multi
 *   idx      [d] uint8 (written): k*_i in 0..K-1
 *   sum      [d] int32 (written): the sum over the M workers' codes
 *   out      [d] fp32 (written): the reconstruction, the rule of uq_dequantize
 * The checks of uq_quantize_multi and uq_dequantize apply; M > 16 returns
 * UQ_ERANGE (use uq_shared_scale and uq_quantize_sum there).
 */
int uq_index_quantize_sum(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                          const float* scales, int32_t K, uint64_t seed, uint8_t* idx,
                          int32_t* sum, float* out, void* stream);

/*
 * The shared scale index of Sec. 3.2 (the rule of Eq. (11) with scale
 * sharing) formed inside the multi-scale quantiser over all M workers, with
 * every worker's codes stored: Eq. (12) and the code of Sec. 3.2, as int8 or
 * as the 4- or 2-bit fields of uq_quantize_packed.  Bit for bit the idx of
 * uq_shared_scale followed by uq_quantize_multi (bits = 8) or
 * uq_quantize_packed (bits = 4, 2) over all M rows with worker0 = 0, given
 * the same W.  As in uq_index_quantize_sum, every row of a tile is held in
 * registers, so each coordinate's index comes from its exact largest usable
 * |g|; uq_shared_scale then only has to form W (call it with K = 1 and
 * idx = NULL).
 *   g        [M][ldg] fp32, 1 <= M <= 16; row m is worker m
 *   w        device pointer to W (one fp32, read)
 *   scales   host array of K floats, 1 <= K <= UQ_MAX_SCALES, as for
 *            uq_quantize_multi; with bits < 8 the smallest must fit the field
 *            (s_0 <= 7 for 4 bits, s_0 <= 1 for 2 bits)
 *   bits     8, 4 or 2
 *   idx      [d] uint8 (written): k*_i in 0..K-1
 *   codes    [M][ldc] bytes (written): int8 codes, or packed fields in the
 *            layout of uq_quantize_packed (ldc >= ceil(d * bits / 8))
 *   ldc      code row stride in bytes, a multiple of 16
 * The checks of uq_quantize_multi / uq_quantize_packed apply; M > 16
 * returns UQ_ERANGE (use uq_shared_scale and the quantiser there).
 */
int uq_index_quantize(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                      const float* scales, int32_t K, uint64_t seed, int32_t bits, uint8_t* idx,
                      void* codes, int64_t ldc, void* stream);

/* ------------------------------------------------------------------------
 * Sub-byte codes.  The paper stores every code in 8 bits because its
 * framework had no narrower type, and found bit-packing too slow (Sec. 5,
 * Appendix A).  Here the quantiser packs while it stores and the sum
 * unpacks while it adds: the codes are the same as those of
 * uq_quantize_single / uq_quantize_multi, held as `bits`-bit two's
 * complement fields, low bits first: the code of coordinate i occupies bits
 * (i % (8/bits)) * bits .. + bits-1 of byte i / (8/bits).
 * ------------------------------------------------------------------------ */

/*
 * Quantise to packed codes.  bits = 4 needs s_0 <= 7, bits = 2 needs s_0 <= 1.
 *   scales, K, idx  as for uq_quantize_multi (K = 1: one scale, idx may be NULL)
 *   packed          [rows][ldp] bytes, ldp >= ceil(d * bits / 8), ldp % 16 == 0
 *                   (written: the bytes of every 8-coordinate group that
 *                   starts below d, ceil(d / 8) * bits bytes per row, which
 *                   ldp always covers; fields past d hold 0)
 * Other arguments as for uq_quantize_single.
 */
int uq_quantize_packed(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                       const float* w, const float* scales, int32_t K, const uint8_t* idx,
                       uint64_t seed, int32_t bits, uint8_t* packed, int64_t ldp, void* stream);

/*
 * uq_sum_codes for packed rows: sum_i (=, or +=) the rows' unpacked codes.
 */
int uq_sum_packed(const uint8_t* packed, int64_t d, int32_t rows, int64_t ldp, int32_t bits,
                  int32_t accumulate, int32_t* sum, void* stream);

/* ------------------------------------------------------------------------
 * GlobalRandK sparsification (Sec. 3.3 GlobalRandKMaxNorm, Sec. 3.4
 * GlobalRandKMaxNormMultiScale): K coordinates chosen uniformly at random,
 * the same for every worker, are quantised as a K-dimensional problem with
 * the calls above and written back into the d-vector (0 elsewhere; there is
 * no d/K rescaling).  A step is: uq_randk_select -> uq_gather ->
 * uq_shared_scale / uq_quantize_* / uq_sum_codes / uq_dequantize on the
 * [M][K] sub-vectors -> uq_scatter.  In these four calls K is the number of
 * sampled coordinates (the paper's K), not a number of scales.
 * ------------------------------------------------------------------------ */

/* Workspace bytes uq_randk_select needs (a fixed size, about 4.4 MiB). */
size_t uq_randk_workspace_bytes(int64_t d, int64_t K);

/*
 * The uniformly random K-subset: coordinate i has the 64-bit key
 * (hi, lo) = (word i%4 of Philox4x32-10 block (i/4, 0, 2),
 *             word i%4 of block (i/4, 0, 3)) under key `seed`, and the K
 * coordinates with the smallest (hi, lo, i) are written to sel[0..K) in
 * increasing order.
 *   d      1 <= d < 2^32
 *   K      1 <= K <= d
 *   sel    [K] uint32 (written), 16-byte aligned
 *   ws     device workspace of uq_randk_workspace_bytes(d, K) bytes
 * The boundary search keeps the keys that share the K-th key's top 20 bits
 * (about d / 2^20 are expected, at most 4096 with a standard deviation of
 * 64); when more arrive than it keeps, the K-th key's whole 32-bit high word
 * is found by one more histogram and only the keys with that high word are
 * ranked, so the result stays exact.  Only if more than 1024 keys share
 * that 32-bit high word (which pseudo-random keys do not produce for any
 * d < 2^32) is the selection abandoned: then every entry of sel is
 * 0xFFFFFFFF, an index >= d that uq_gather reads as 0 and uq_scatter skips.
 */
int uq_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* sel, void* ws, size_t ws_bytes,
                    void* stream);

/*
 * sub[m][j] = g[m][sel[j]] for the M rows and j < K (an index >= d reads as 0).
 *   g      [M][ldg] fp32, ldg >= d      sub   [M][lds] fp32, lds >= K, lds % 4 == 0
 */
int uq_gather(const float* g, int64_t d, int32_t M, int64_t ldg, const uint32_t* sel, int64_t K,
              float* sub, int64_t lds, void* stream);

/*
 * out[0..d) = 0, then out[sel[j]] = vals[j] for j < K (indices >= d skipped).
 */
int uq_scatter(const float* vals, const uint32_t* sel, int64_t K, float* out, int64_t d, void* stream);

/*
 * Test hook, not part of the aggregation step: caps the grids of the
 * streaming passes (norm, index, quantise, sum, reconstruction) at `blocks`
 * blocks, 8 <= blocks <= 2^22; 0 restores the default 2^22 (the dispatch
 * packet counts work-items in 32 bits).  The passes cover whatever their grid
 * does not with grid-stride loops, which the default reaches only past about
 * 2^33 coordinates; a lower cap lets tests run those loops at small sizes.
 * Outputs do not depend on the cap.  Process-wide: set it only while no other
 * thread issues library calls.  UQ_EINVAL for a value out of range.
 */
int uq_set_grid_cap(int64_t blocks);

/*
 * Test hook, not part of the aggregation step: how uq_randk_select finds the
 * K-subset (for K <= 16384; larger K always use the histogram passes).
 *   1  (default) one collection pass over a bracket of the K-th key computed
 *      from d and K, with an exact fallback inside the selection when the
 *      bracket misses (probability below 1e-20)
 *   0  the histogram passes (two histograms, then the collection pass)
 *   2  the bracket made to miss, so that the fallback always runs
 *   3  as 0, keeping no boundary candidates, so that the exact refinement
 *      by the 32-bit high word always runs
 *   4  as 2, the fallback keeping no boundary candidates (the refinement
 *      always runs there)
 * Every mode selects the same coordinates.  Process-wide: set it only while
 * no other thread issues library calls.  UQ_EINVAL for another value.
 */
int uq_set_randk_mode(int32_t mode);

/* Static text for a status code. */
const char* uq_strerror(int status);

/* Detail of the last error reported on the calling thread ("" if none). */
const char* uq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* UQ_H */
