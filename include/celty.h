/*
 * celty.h -- C ABI of libcelty: dual-sparse SpMSpV y = W x on AMD MI355X (gfx950).
 *
 * The operation (Celty, Sections 2.1 and 3.1): W is an unstructured-pruned
 * fp16 weight matrix (M rows = outputs, K columns = inputs) kept in the
 * paper's run-length compressed CSC format (RLC-CSC, Section 3.2); x is an
 * fp16 activation vector made sparse at run time by magnitude thresholding
 * (Sections 1 and 2.1): column k takes part iff |x_k| > tau.  Then
 *
 *     y[r] = sum over active k of W[r,k] * x_k,     r = 0 .. M-1,
 *
 * with every product formed exactly in fp32 (two fp16 factors), the products
 * summed in integer fixed point on grids derived from the magnitudes of the
 * call's own active columns (celty_spmspv states the arithmetic and its error
 * bound), and y rounded to fp16 (round to nearest even).  Inactive columns of
 * W are never read (Section 3.1).
 *
 * General rules
 * -------------
 * - No function allocates or frees caller-visible memory.  Every buffer is
 *   owned by the caller.  The encoder uses small per-thread host scratch.
 * - No C++ exception crosses this interface; every error is a status code.
 * - Host pointers and device pointers are marked at each argument.
 * - Device calls (celty_select, celty_spmspv*) validate every argument on the
 *   host, synchronously, before any launch; they then enqueue work on the
 *   given HIP stream (NULL = the default stream) and return without
 *   synchronising.  They are stateless: calls on different streams may run
 *   concurrently when their output and workspace buffers differ.
 */
#ifndef CELTY_H
#define CELTY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum celty_status {
  CELTY_OK = 0,
  CELTY_EINVAL = 1,     /* bad argument: null pointer, bad size, NaN tau, short buffer, misalignment */
  CELTY_ENOMEM = 2,     /* host scratch or worker threads could not be created */
  CELTY_EOVERFLOW = 3,  /* the encoded group count does not fit in uint32 */
  CELTY_EFORMAT = 4,    /* malformed RLC-CSC stream (decoder only) */
  CELTY_EHIP = 5        /* the HIP runtime reported an error at launch */
} celty_status;

#define CELTY_FORMAT_VERSION 2
#define CELTY_RUN_BITS 4   /* 4-bit run lengths (Section 3.2) */
#define CELTY_GROUP 8      /* entries per aligned group: one 16-byte fp16 vector */

/* Layouts of the per-entry row information (the `layout` field). */
#define CELTY_LAYOUT_RLC 0         /* 4-bit run lengths, Section 3.2 (the format below) */
#define CELTY_LAYOUT_ROWS16 1      /* 16-bit row offsets instead of runs (decode-free) */
#define CELTY_LAYOUT_INTERLEAVED 2 /* the RLC entries in lane-interleaved order, Section 4.2 */

/*
 * Tiled RLC-CSC, format version 2 (Section 3.2 plus the readings below).
 *
 * Rows are cut into T = ceil(M/R) tiles of R rows.  Segment (t, k) holds the
 * stored entries of column k inside tile t; segments are laid out tile-major,
 * s = t*K + k, so the segments one row tile needs are contiguous.
 *  - A weight is stored iff it is kept by the mask and is not +0/-0.
 *  - Each stored value carries a 4-bit run: the count of zeros since the
 *    previous stored entry of the segment, or since the tile's first row.
 *  - A gap g > 15 is bridged greedily: g/16 padding entries (value 0, run 15)
 *    come first, then the value with run g%16 (the worked example of 3.2).
 *    Trailing zeros are not encoded.
 *  - Row of entry i of a segment = t*R + (sum of runs 0..i) + i (Section 3.3).
 *  - Each segment is padded to a multiple of 8 entries with (0, 0) "dead"
 *    entries, so every segment starts on a 16-byte boundary.
 *  - values[8g + j] is the fp16 bit pattern of entry j of group g; runs[g]
 *    holds entry j's run in bits [4j, 4j+4).
 *  - gptr[s] is the first group of segment s; gptr[T*K] = n_groups.
 *  - colmax[k] is the fp16 bit pattern of the largest |stored value| of
 *    column k (+0 when the column stores nothing).  It is not part of the
 *    paper's format: the product derives its fixed-point scales from it.
 * Version 1 was the same format without colmax.  The descriptor is plain
 * data; the arrays are owned by the caller and are host pointers for the
 * encoder/decoder and device pointers for celty_spmspv*.
 *
 * Two other layouts keep gptr, values, colmax and the 8-entry groups:
 *  - CELTY_LAYOUT_ROWS16 (a decode-free form, for measuring what the run
 *    reconstruction of Sections 3.3 and 4.2 costs): each entry carries its
 *    row offset within the tile (0 .. R-1) as uint16; `runs` then points to
 *    4 words per group, the uint16 at index 8g + j (little-endian) being
 *    entry j's offset.  Only stored values are entries (no padding entries,
 *    n_pad = 0); a segment's alignment entries have value 0 and repeat the
 *    row offset of its last stored entry.  Needs R <= 16376 (4 * (R + 7)
 *    fits in 16 bits for the kernel).
 *  - CELTY_LAYOUT_INTERLEAVED (Section 4.2's offline interleave across
 *    lanes): the RLC entries of every segment, cut into chunks of up to 64
 *    groups (64 per chunk, the segment's last chunk holding the rest); within
 *    a chunk of G_c groups, row-order entry e is stored in group e % G_c,
 *    slot e / G_c, with its run (the runs keep their meaning).  Lane l of a
 *    wavefront that loads the chunk's group l holds entries l, l + G_c, ...
 *    Same arrays and sizes as CELTY_LAYOUT_RLC.
 */
typedef struct celty_rlc_csc {
  int32_t version;          /* CELTY_FORMAT_VERSION */
  int32_t M, K, R, T;       /* rows (outputs), columns (inputs), tile rows, ceil(M/R) */
  int32_t run_bits;         /* CELTY_RUN_BITS */
  int64_t n_groups;         /* G: 8-entry groups, alignment included */
  int64_t n_entries;        /* stored values + padding entries (alignment excluded) */
  int64_t n_nnz;            /* stored values */
  int64_t n_pad;            /* padding entries */
  float max_abs;            /* largest |stored value| (0 if none) = the largest colmax; finite */
  int32_t layout;           /* CELTY_LAYOUT_RLC, _ROWS16 or _INTERLEAVED */
  const uint32_t* gptr;     /* [T*K + 1], 4-byte aligned */
  const uint16_t* values;   /* [8*G] fp16 bits, 16-byte aligned */
  const uint32_t* runs;     /* [G] ([4*G] for ROWS16), 4-byte aligned (16 for ROWS16) */
  const uint16_t* colmax;   /* [K] fp16 bits, 4-byte aligned */
} celty_rlc_csc;

/*
 * Size plan of the encoding of a dense fp16 matrix under a keep-mask (Section
 * 3.2, offline packing).
 *   W      host, fp16 bit patterns, row-major M x K with row stride ldw >= K.
 *   mask   host, uint8 row-major with row stride ldm >= K; non-zero = kept.
 *          NULL keeps every entry (then only +-0 weights are dropped).
 *   R      tile height, 1 <= R (<= 16376 for CELTY_LAYOUT_ROWS16); T = ceil(M/R).
 *   layout CELTY_LAYOUT_RLC, CELTY_LAYOUT_ROWS16 or CELTY_LAYOUT_INTERLEAVED.
 * Outputs (host, may not be NULL): n_groups, n_nnz, n_pad (0 for ROWS16).
 * Errors: EINVAL (null W or output pointer, M/K/R < 1, short stride, unknown
 *         layout, R too tall for ROWS16), EOVERFLOW (n_groups > UINT32_MAX),
 *         ENOMEM.
 */
celty_status celty_encode_plan(const uint16_t* W, int64_t ldw, const uint8_t* mask, int64_t ldm,
                               int32_t M, int32_t K, int32_t R, int32_t layout,
                               int64_t* n_groups, int64_t* n_nnz, int64_t* n_pad);

/*
 * Encode into caller buffers (host): gptr [T*K+1], values [8*n_groups]
 * (16-byte aligned), runs [n_groups] ([4*n_groups], 16-byte aligned, for
 * CELTY_LAYOUT_ROWS16), colmax [K] (4-byte aligned).
 * n_groups must equal the plan's value.  On success *out is filled (pointers
 * = the buffers given here, and max_abs = the largest magnitude among the
 * stored values).  n_threads: worker threads, 0 = all hardware threads.  The
 * result does not depend on n_threads.
 * Errors: EINVAL (as for the plan, null buffers, misaligned values or colmax,
 *         n_groups mismatch, n_threads < 0), EOVERFLOW, ENOMEM.
 */
celty_status celty_encode(const uint16_t* W, int64_t ldw, const uint8_t* mask, int64_t ldm,
                          int32_t M, int32_t K, int32_t R, int32_t layout,
                          uint32_t* gptr, uint16_t* values, uint32_t* runs, uint16_t* colmax,
                          int64_t n_groups, celty_rlc_csc* out, int32_t n_threads);

/*
 * Decode a stream held in host memory back to dense form (host).
 *   W_out    host, M x K fp16 bits, row-major, stride K: stored values, +0 elsewhere.
 *   mask_out host, M x K uint8, stride K: 1 where a value is stored (may be NULL).
 * Every layout is accepted; an interleaved stream is first put back in row
 * order.
 * Errors: EINVAL (null pointers, bad header), EFORMAT (gptr not monotone from
 * 0 to n_groups, a stored value beyond its tile, an alignment entry with a
 * non-zero run (RLC) or another row than the last stored one (ROWS16),
 * stored rows out of order (ROWS16), header counts, max_abs or colmax that
 * disagree with the stream), ENOMEM.
 */
celty_status celty_decode(const celty_rlc_csc* enc, uint16_t* W_out, uint8_t* mask_out);

/*
 * Active-column selection (Sections 1, 2.1 and 3.1: magnitude threshold,
 * then stream compaction by wavefront ballot and prefix sums).
 *   x      device, fp16[K], 2-byte aligned (4-byte alignment lets the kernel
 *          read two columns per 32-bit load; the result is the same).
 *   tau    threshold; column k is active iff |x_k| > tau in fp32 (NaN x_k is
 *          never active; tau < 0 makes every non-NaN column active).
 *   idx    device, int32[K]: receives the active indices in ascending order;
 *          entries past |A| are not written.
 *   count  device, int32[1]: receives |A|.
 * One kernel launch of one workgroup.
 * Errors: EINVAL (null pointers, K < 1 or K > (2^31 - 4) / 2, NaN tau,
 * misaligned x/idx/count), EHIP.
 */
celty_status celty_select(const void* x, int32_t K, float tau, int32_t* idx, int32_t* count,
                          void* stream);

/* Launch shape of celty_spmspv_ex.  Zero fields mean "choose automatically":
 * 16 wavefronts per workgroup for R >= 1024, else 8; slices sized for about
 * 4096 / waves_per_block workgroups (16 wavefronts on each of 256 compute
 * units), never more, and widened to fill two 8-wavefront workgroups per
 * unit evenly when the rounded width would load the units unevenly and the
 * slices stay heavy enough; one group per lane.  The K columns are cut into
 * ceil(K / cols_per_block) slices, at most 63 (the merge counts 6-bit
 * arrivals in a 64-bit word).  A workgroup's lanes scan at most 8 columns
 * each: cols_per_block <= 512 * waves_per_block.
 * lds_swizzle = 1 stores the LDS tile's row r at slot r ^ ((r >> 6) & 63)
 * (an XOR swizzle against bank conflicts in the scatter-adds, Section 4.1;
 * the result is the same).  It applies to CELTY_LAYOUT_RLC only.  The
 * swizzle and the two other layouts run with one group per lane and one
 * product per launch. */
typedef struct celty_launch {
  int32_t cols_per_block;   /* columns of x one workgroup scans (1..4096) */
  int32_t waves_per_block;  /* 2, 4, 8 or 16 wavefronts of 64 lanes */
  int32_t groups_per_lane;  /* 1, 2 or 4 eight-entry groups per lane per pass */
  int32_t lds_swizzle;      /* 0 (plain tile) or 1 (XOR-swizzled tile) */
} celty_launch;

/* A tile height R for encoding an M x K matrix for celty_spmspv (host only):
 * the largest power of two at or below M / 8 (M / 4 when K >= 4 M), clamped
 * to [256, 2048], which gives 4 to 16 row tiles for the LLM projection shapes
 * and keeps one tile's accumulator (4 * (R + 136) bytes of LDS) small.
 * 0 when M < 1. */
int32_t celty_default_tile_rows(int32_t M, int32_t K);

/* Bytes of device workspace celty_spmspv needs for this shape: two 64-bit
 * merge words per output row, rounded up to 256 bytes. */
size_t celty_spmspv_workspace_bytes(int32_t M, int32_t K, int32_t R);

/*
 * Zero-fill a workspace (device) on `stream`.  A workspace must be zero-filled
 * once before its first use; every completed celty_spmspv call leaves it
 * zero-filled again.  Any alignment and size; one fill kernel, no memset, so
 * the call may be recorded in a graph.  Errors: EINVAL (null or size 0), EHIP.
 */
celty_status celty_spmspv_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/*
 * The dual-sparse SpMSpV (Sections 3.1-3.3): y = W x_A.
 *   W          descriptor with DEVICE pointers (e.g. the encoder's arrays
 *              copied to the device); must be a valid encoder output.
 *   x          device fp16[K]; must be finite (an infinite x_k is outside the
 *              operation's domain and yields unspecified rows).
 *   tau        threshold, as for celty_select.
 *   y          device fp16[M]; fully overwritten (rows without contribution
 *              become +0); must not alias x or the workspace.
 *   workspace  device buffer of at least celty_spmspv_workspace_bytes(M,K,R)
 *              bytes, zero-filled before first use (celty_spmspv_workspace_init).
 *              Every completed call leaves it zero; a call that did not
 *              complete (the device reported an error after the launch)
 *              may leave merge words behind, so zero-fill it again before
 *              the next call, or the next y is wrong.
 * One kernel launch.  The grid is (row tile t) x (column slice c).  Every
 * workgroup selects the active columns of its slice that store entries in
 * its tile (the n columns of A_ct), walks their compressed segments, forms
 * each product w * x_k exactly in fp32 and adds it into an LDS tile of R
 * int32 rows:
 *
 *   B_ct = n * max over k in A_ct of colmax[k] * |x_k|   (fp32)
 *   s_ct = 30 - e(B_ct), where 2^(e-1) <= B_ct < 2^e     (clamped to [-64, 64])
 *
 * and each product is rounded to the nearest multiple of 2^-s_ct (ties
 * upward) before the integer add, so no partial sum can leave int32.  With
 * one column slice, y[r] = fp16(fp32(tile[r]) * 2^-s_ct).  With several,
 * the slices of a row tile are merged with one returning 64-bit atomic per
 * row and slice: each partial p, clamped to +-4096, is added as a multiple
 * of 2^-33 (ties upward); a clamped slice also adds p minus the clamp, as a
 * multiple of 2^-8, to a second word of the row (an extra atomic, ordered
 * before its ticket by a release fence).  The slice that arrives last
 * writes y[r] = fp16(fp32(fine) * 2^-33 + fp32(excess) * 2^-8) and clears
 * both words.  Error of a row r before those output roundings, for n_rc
 * products of row r in slice c:
 *
 *   |sum - exact| <= sum over slices c of n_rc * B_ct * 2^-30
 *                    + 2^-34 per slice (2^-9 per slice whose partial was clamped)
 *
 * (when s_ct is not clamped; B_ct bounds every row's sum of |products| in
 * slice c).  The 2^-34 term, below half the spacing of fp16 subnormals, is
 * the only one that does not scale with the data.  (An fp32 sum of n terms
 * in any order has the worst case (n - 1) * 2^-24 * sum_k |W[r,k] x_k|.)
 * colmax must bound every |stored value| of its column (the encoder sets it
 * exactly): a smaller value can overflow the int32 tile and give wrong rows,
 * but never an access outside the arrays.
 * Every layout gives the same y.
 * Errors: EINVAL (null or misaligned pointers, inconsistent header, NaN tau,
 *         non-finite or negative max_abs, short workspace, more than 63
 *         column slices, cols_per_block above 512 * waves_per_block,
 *         16 * n_groups >= 2^31, groups_per_lane > 1 with another layout
 *         than RLC or with lds_swizzle, lds_swizzle with another layout),
 *         EHIP.
 */
celty_status celty_spmspv(const celty_rlc_csc* W, const void* x, float tau, void* y,
                          void* workspace, size_t workspace_bytes, void* stream);

/* As celty_spmspv with an explicit launch shape (NULL = automatic). */
celty_status celty_spmspv_ex(const celty_rlc_csc* W, const void* x, float tau, void* y,
                             void* workspace, size_t workspace_bytes,
                             const celty_launch* launch, void* stream);

/*
 * Several independent SpMSpVs in one launch (Section 3.1's product for each;
 * one launch instead of n: projections of a decoder layer that read the same
 * activation, q/k/v or gate/up, pass the same x).
 *   n          1..8 products.
 *   W[i]       descriptor with device pointers, as for celty_spmspv; the
 *              products may have different shapes and tile heights.
 *   x[i], tau[i], y[i]
 *              as for celty_spmspv; x pointers may repeat, a y may not
 *              overlap any x, any other y or the workspace.
 *   workspace  device buffer of at least
 *              celty_spmspv_batch_workspace_bytes(n, W) bytes (product i's
 *              slots follow those of products 0..i-1), zero-filled before
 *              first use and left zero-filled by every completed call.
 *   launch     as for celty_spmspv_ex; cols_per_block applies to every product,
 *              the automatic choice is made per product, with 16 wavefronts
 *              when any product has R >= 1024.
 * Results are those of n separate celty_spmspv_ex calls with the same launch.
 * With n > 1 every product must use CELTY_LAYOUT_RLC without lds_swizzle.
 * Errors: EINVAL (n outside 1..8, null arrays, any product's celty_spmspv
 *         error, overlapping buffers, short workspace, another layout or
 *         lds_swizzle with n > 1), EHIP.
 */
celty_status celty_spmspv_batch(int32_t n, const celty_rlc_csc* const* W, const void* const* x,
                                const float* tau, void* const* y, void* workspace,
                                size_t workspace_bytes, const celty_launch* launch, void* stream);

/*
 * As celty_spmspv_ex, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the merge words live in a static device array of the library
 * (2 MiB on every GPU it runs on, held until the process ends) instead of a
 * caller workspace, so the call takes no workspace and allocates nothing.
 *   W, x, tau, y, launch, stream   as for celty_spmspv_ex.
 * The array holds two 64-bit words per output row: M up to 131072.  Its
 * device address is looked up once per device (hipGetSymbolAddress, with
 * that device current); the first call on a device also zero-fills it with a
 * kernel on `stream`, and every completed call leaves it zero.  Every call on
 * a GPU shares that GPU's array: calls that overlap on one GPU (concurrent
 * streams, or graphs replayed concurrently) race and give wrong rows.
 * Errors: as celty_spmspv_ex, plus EINVAL when M exceeds 131072, EHIP when
 *         the array's address cannot be found.
 */
celty_status celty_spmspv_noalloc(const celty_rlc_csc* W, const void* x, float tau, void* y,
                                  const celty_launch* launch, void* stream);

/* Workspace bytes of celty_spmspv_batch: the sum over the products of
 * celty_spmspv_workspace_bytes (host only; 0 for n outside 1..8 or null). */
size_t celty_spmspv_batch_workspace_bytes(int32_t n, const celty_rlc_csc* const* W);

/* The launch shape celty_spmspv_ex would use for W and `launch` (host only):
 * fills *resolved and, if not NULL, the workgroup count and LDS bytes. */
celty_status celty_spmspv_plan(const celty_rlc_csc* W, const celty_launch* launch,
                               celty_launch* resolved, int64_t* n_blocks, int64_t* lds_bytes);

/* Static text for a status code. */
const char* celty_status_string(celty_status status);

#ifdef __cplusplus
}
#endif

#endif /* CELTY_H */
