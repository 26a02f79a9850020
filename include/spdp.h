/*
 * spdp.h -- C ABI of the MI355X (gfx950) Tiled-CBC spMspV library.
 *
 * The library implements the decode-time hot path of SPDP ("Unified
 * Static-Dynamic Pruning for Efficient LLM Inference"): an fp16 weight matrix
 * that has been statically pruned (unstructured) is stored in the Tiled-CBC
 * format (Sec. 4.1), and each decode call multiplies it by activations whose
 * small-magnitude entries are dropped at run time (dynamic pruning, Sec. 2.2),
 * fetching only the active columns' metadata and values (Sec. 4.2).
 *
 * Conventions for every entry point:
 *   - Matrices are row-major. W is rows x cols = out-features x in-features,
 *     so y = W x with x of length cols.
 *   - fp16 data travels as raw IEEE binary16 bit patterns (uint16_t).
 *   - Every function returns an spdp_status; on error nothing is launched,
 *     output handles are left NULL and spdp_last_error() holds a message for
 *     the calling thread. No C++ exception crosses this ABI.
 *   - Host pointers are read during the call only and never retained.
 */
#ifndef SPDP_H
#define SPDP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum spdp_status {
  SPDP_OK = 0,
  SPDP_ERR_INVALID_ARG = -1, /* a null pointer, a bad size, NaN, ... */
  SPDP_ERR_UNSUPPORTED = -2, /* valid input the library does not handle */
  SPDP_ERR_OOM = -3,         /* host or device allocation failed */
  SPDP_ERR_HIP = -4          /* a HIP runtime call failed (text in spdp_last_error) */
} spdp_status;

/* Opaque handle to one encoded matrix (host arrays + optional device copy). */
typedef struct spdp_matrix* spdp_handle_t;

/*
 * spdp_encode -- Tiled-CBC encode of W (Sec. 4.1) and upload to the current
 * HIP device.
 *
 *   W        host, rows*cols fp16 bit patterns, row-major, already pruned:
 *            the library stores whatever zeros it is given. An element is
 *            treated as zero iff its magnitude bits are zero (-0 is zero).
 *   rows     M >= 1; cols: K >= 1. Ragged sizes are zero-padded to whole
 *            tiles inside the format.
 *   tile_m   rows of a GTile, a multiple of 64 in [64, 256] (the paper uses
 *            256); each column tile carries tile_m/64 uint64 bitmap words.
 *   tile_k   columns of a GTile, a power of two in [1, 256] (the paper uses 16).
 *   out      receives the handle.
 *
 * Layout produced (byte-exact, inspect with spdp_format):
 *   GTile g = r*C + c for row stripe r < R = ceil(M/tile_m) and column block
 *   c < C = ceil(K/tile_k) (row-major GTile order).
 *   tile_offset[g]  uint32, start of GTile g in values (fp16 elements);
 *                   NGT+1 entries, the last one = number of values.
 *   col_info[g*tile_k+j] uint32 = (offset << 16) | nnz: offset in fp16
 *                   elements from tile_offset[g] (includes earlier columns'
 *                   padding), nnz = nonzeros of column j of the GTile.
 *   bitmap[(g*tile_k+j)*(tile_m/64) + w] uint64: bit i <-> row 64w+i of the
 *                   stripe; 1 iff that element is nonzero.
 *   values          nonzeros GTile by GTile, column by column, rows ascending,
 *                   each column padded with +0 to a multiple of 8 elements
 *                   (16 bytes, Sec. 4.2.3).
 *
 * Device memory for the four arrays plus a small split-K workspace is
 * allocated on the current device and owned by the handle. Returns
 * SPDP_ERR_UNSUPPORTED if the padded values would take 4 GiB or more, or if
 * R * C * tile_k (GTile columns, plus one) reaches 2^26.
 */
int spdp_encode(const uint16_t* W, int64_t rows, int64_t cols, int32_t tile_m,
                int32_t tile_k, spdp_handle_t* out);

/*
 * spdp_encode_host -- the same encoding without any device work: the handle
 * holds host arrays only (usable on machines without a GPU, e.g. to inspect
 * the format). spdp_spmspv on such a handle returns SPDP_ERR_INVALID_ARG.
 */
int spdp_encode_host(const uint16_t* W, int64_t rows, int64_t cols,
                     int32_t tile_m, int32_t tile_k, spdp_handle_t* out);

/*
 * spdp_spmspv -- Y = W_sp . mask(X) for a batch of decode tokens (Sec. 4.2).
 *
 *   h          handle from spdp_encode (device copy on the current device).
 *   X          device, batch x cols fp16, row-major, 16-byte aligned.
 *   batch      number of tokens, 1 <= batch <= 32.
 *   threshold  dynamic-pruning threshold (Sec. 5.1 per-layer ECDF quantile):
 *              column k takes part for token b iff |X[b,k]| > threshold
 *              (strict). A negative threshold keeps every column; NaN is
 *              SPDP_ERR_INVALID_ARG. NaN activations are never active.
 *              Columns inactive for every token of the batch are not read.
 *   Y          device, batch x rows fp16, row-major, fully overwritten with
 *              the fp32-accumulated result rounded once to nearest even.
 *              Must not overlap X.
 *   stream     hipStream_t to enqueue on (NULL = the null stream).
 *
 * Asynchronous: the call validates, enqueues one kernel and returns; X and Y
 * must stay valid until the stream passes the work. The handle's workspace
 * is reused by every call, so one handle must not run on two streams at
 * once. The first call with a larger batch than before grows the workspace:
 * a device allocation, cleared on `stream` ahead of the kernel, with no wait
 * for the device (the old workspace is kept until spdp_free, since work in
 * flight or a captured graph may still use it). Growth is refused with
 * SPDP_ERR_INVALID_ARG while `stream` is capturing. spdp_reserve sizes the
 * workspace ahead of time, after which calls allocate nothing and may be
 * captured into a HIP graph (replays are exact: the call keeps no host-side
 * state).
 *
 * Deterministic: the fp32 summation order depends only on the matrix, the
 * batch and which columns are active (and on the tuning variables
 * SPDP_SPLITK, SPDP_PASSES, SPDP_MFMA and SPDP_EARLY_FIRST, when set), so
 * equal inputs give equal bits on every call, and a product gives the same
 * bits alone and inside spdp_spmspv_many.
 */
int spdp_spmspv(spdp_handle_t h, const uint16_t* X, int32_t batch,
                float threshold, uint16_t* Y, void* stream);

/*
 * spdp_spmspv_noalloc -- spdp_spmspv that allocates nothing, for callers that
 * cannot call hipMalloc (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Same arguments, semantics, summation
 * order and bits as spdp_spmspv; the split-K partials live in one static
 * workspace of the library per device (SPDP_NOALLOC_PARTIAL_BYTES bytes,
 * held until the process ends) instead of the handle's own.
 *
 *   A product needing more than SPDP_NOALLOC_PARTIAL_BYTES of partials
 *   (8 bytes x K segments x batch x rows rounded up to tile_m) returns
 *   SPDP_ERR_UNSUPPORTED and launches nothing: a 4096 x 4096 product fits
 *   at every batch up to 32, and so does every Llama-7B, -13B and -70B
 *   projection (the most any needs is 39.9 MiB: 8192 x 8192 at batch
 *   29, two K ranges per workgroup).
 *   The workspace is shared by every call on one GPU and keeps the last
 *   call's contents (tagged with a device-wide call epoch, so a call never
 *   reads another's partials): calls that overlap on one GPU (two streams,
 *   or two host threads) race and must not be issued.
 *   The first call on a device looks up the workspace's address
 *   (hipGetSymbolAddress); no call allocates, frees or waits for the device.
 */
#define SPDP_NOALLOC_PARTIAL_BYTES ((size_t)40 << 20)
int spdp_spmspv_noalloc(spdp_handle_t h, const uint16_t* X, int32_t batch,
                        float threshold, uint16_t* Y, void* stream);

/*
 * spdp_spmspv_many -- several independent products in one launch:
 * Y[i] = W_i . mask(X[i]) with threshold thresholds[i], for i < count. This
 * is how a decoder issues the projections that read the same layer input
 * (q, k and v; gate and up), whose fixed per-launch latency would otherwise
 * be paid once per matrix. Each product follows the rules of spdp_spmspv.
 *
 *   handles     count handles (device copies on the current device), all
 *               with the same tile_m; no handle may appear twice (its
 *               workspace serves one product at a time).
 *   count       1 <= count <= 8.
 *   X, Y        count device pointers each (X[i]: batch x cols_i, Y[i]:
 *               batch x rows_i, 16-byte aligned). An output must not overlap
 *               any input or any other output of the call; inputs may be
 *               shared (q, k and v read one X).
 *   batch       tokens of every product, 1 <= batch <= 32.
 *   thresholds  count thresholds (host array).
 *   stream      hipStream_t to enqueue on.
 *
 * Errors are those of spdp_spmspv plus SPDP_ERR_INVALID_ARG for a bad count,
 * a repeated handle, mixed tile_m or overlapping outputs; on any error
 * nothing is launched. spdp_spmspv(h, ...) is this call with count 1.
 */
int spdp_spmspv_many(const spdp_handle_t* handles, int32_t count,
                     const uint16_t* const* X, int32_t batch,
                     const float* thresholds, uint16_t* const* Y, void* stream);

/*
 * spdp_spmspv_many_mask -- spdp_spmspv_many with a choice of how the batch's
 * activations select columns (batched dynamic pruning, which the paper
 * leaves to future work in Sec. 4.3 and Sec. 7):
 *
 *   SPDP_MASK_TOKEN  per-token masks, the rule of spdp_spmspv: column k takes
 *                    part for token b iff |X[b,k]| > threshold; the columns
 *                    read are the union over the batch, which grows as
 *                    1 - p^batch and reaches every column by batch 4-8.
 *   SPDP_MASK_BATCH  one column set for the whole batch: column k takes part
 *                    for every token iff the fp32 running sum of |X[b,k]|
 *                    over b = 0, 1, ... (each addition rounded to nearest
 *                    even) exceeds fp32(batch * threshold), i.e. the batch's
 *                    mean magnitude exceeds the threshold; in that column
 *                    every token's activation is used as it is. The set keeps
 *                    the per-token rule's size at any batch; at batch 1 the
 *                    two rules are the same.
 *
 * Other arguments, ownership and errors are those of spdp_spmspv_many; a
 * mask other than the two values is SPDP_ERR_INVALID_ARG (nothing is
 * launched).
 */
enum { SPDP_MASK_TOKEN = 0, SPDP_MASK_BATCH = 1 };
int spdp_spmspv_many_mask(const spdp_handle_t* handles, int32_t count,
                          const uint16_t* const* X, int32_t batch,
                          const float* thresholds, int32_t mask,
                          uint16_t* const* Y, void* stream);

/*
 * spdp_spmm -- the prefill product on the same encoded matrix (Sec. 4.3):
 * Y = X W_sp^T for n_tokens tokens, static pruning only (no activation
 * test: every column takes part), on the matrix cores: each 256 x 16 GTile
 * is expanded into a dense tile in LDS and multiplied with fp16 MFMA
 * instructions, fp32 accumulation, one rounding to fp16 (nearest even).
 *
 *   h          handle from spdp_encode with tile_m = 256 and tile_k >= 16
 *              (a power of two); fp16 Values. Other handles:
 *              SPDP_ERR_UNSUPPORTED.
 *   X          device, n_tokens x cols fp16, row-major, 16-byte aligned.
 *   n_tokens   1 <= n_tokens <= 65535 * 128.
 *   Y          device, n_tokens x rows fp16, row-major, 16-byte aligned,
 *              fully overwritten; must not overlap X.
 *   stream     hipStream_t to enqueue on.
 *
 * Asynchronous. When the grid of (256-row stripe, token tile) pairs
 * leaves compute units idle (few tokens), or when a stripe has more than
 * 1799 GTiles, the columns are split into k <= 8 ranges (more for very wide
 * matrices; never more workgroups than the device has compute units): one kernel writes k fp32 partial products into a workspace of
 * the handle (k * n_tokens * rows * 4 bytes) and a second adds them in
 * range order and rounds once to fp16. That workspace grows on the first
 * call that needs more (hipMalloc; the old one is kept until spdp_free,
 * so graphs captured earlier stay valid); growing it while `stream` is
 * being captured is refused with SPDP_ERR_INVALID_ARG (make one call with
 * at least as many tokens before the capture). SPDP_ERR_OOM if it cannot
 * be allocated. Calls on one handle that overlap in time on different
 * streams share the workspace and race. The fp32 summation order is fixed
 * by the matrix, the token count and the device's compute-unit count, so
 * equal inputs give equal bits on one device.
 */
int spdp_spmm(spdp_handle_t h, const uint16_t* X, int64_t n_tokens,
              uint16_t* Y, void* stream);

/* spdp_reserve -- size the handle's workspace for batches up to max_batch. */
int spdp_reserve(spdp_handle_t h, int32_t max_batch);

/*
 * spdp_split_plan -- the split-K plan (Sec. 4.2.3) a call with `batch`
 * tokens uses on this matrix, for inspection and tests: *segments
 * workgroups per stripe of tile_m rows (the K segments), *wave_cols columns per
 * wave and range (four waves per workgroup), and *passes consecutive ranges
 * walked by each workgroup. Segment s covers the columns from
 * s * passes * 4 * wave_cols on, so every column lies in exactly one range
 * (segments * passes * 4 * wave_cols >= cols). A property of the matrix and
 * the batch (and of the tuning variables SPDP_SPLITK and SPDP_PASSES), the
 * same on host-only handles. SPDP_ERR_INVALID_ARG for a NULL handle or
 * output, or batch outside [1, 32]; the outputs are then unchanged.
 */
int spdp_split_plan(spdp_handle_t h, int32_t batch, int32_t* segments,
                    int32_t* wave_cols, int32_t* passes);

/*
 * spdp_free -- release a handle. Waits for the device to finish work that
 * may still use it (a device synchronization, so it must not run while a
 * stream capture is in progress). spdp_free(NULL) does nothing. Using h
 * afterwards is undefined.
 */
void spdp_free(spdp_handle_t h);

/* Read-only view of an encoded matrix. Host arrays are owned by the handle
 * and live until spdp_free; device pointers are NULL for host-only handles. */
typedef struct spdp_format {
  int64_t rows, cols;
  int32_t tile_m, tile_k;
  int64_t n_stripes;   /* R */
  int64_t n_colblocks; /* C */
  int64_t n_gtiles;    /* R*C */
  int64_t n_values;    /* length of values (= tile_offset[n_gtiles]) */
  const uint32_t* tile_offset; /* host, n_gtiles + 1 */
  const uint32_t* col_info;    /* host, n_gtiles * tile_k */
  const uint64_t* bitmap;      /* host, n_gtiles * tile_k * tile_m / 64 */
  const uint16_t* values;      /* host, n_values */
  const void* d_tile_offset;   /* device copies (or NULL) */
  const void* d_col_info;
  const void* d_bitmap;
  const void* d_values;
  int32_t device; /* HIP device ordinal of the copies, -1 if host-only */
  /* 16 for fp16 values; 2..8 for a handle from spdp_encode_rtn, whose
     Values are codes (then `values` is NULL, n_values counts codes, and
     tile_offset and the ColInfo offsets count codes) */
  int32_t value_bits;
  const int8_t* codes;  /* host, n_values, or NULL */
  const float* scales;  /* host, rows, or NULL */
  const void* d_scales; /* device copy (or NULL) */
} spdp_format_t;

int spdp_format(spdp_handle_t h, spdp_format_t* out);

/*
 * spdp_encode_rtn -- low-bit Values (Sec. 5.1's quantization setup: the
 * weights are quantized after pruning, and dynamic pruning runs on top at
 * inference; Sec. 6: Values are stored apart from the sparsity metadata).
 * W (already pruned, as for spdp_encode) is quantized to `bits`-bit
 * round-to-nearest codes, symmetric, one fp32 scale per row:
 *     s[m] = fp32(max over the row's nonzeros of |W[m,k]|) / (2^(bits-1) - 1)
 *     q[m,k] = clamp(rint(fp32(W[m,k]) / s[m]), -(2^(bits-1)-1), 2^(bits-1)-1)
 * (fp32 division, ties to even; a row without nonzeros has s = 0). The
 * Tiled-CBC layout is that of spdp_encode -- the same GTiles, column order,
 * bitmaps and nonzero counts (the pruning's pattern: a nonzero whose code is
 * 0 stays stored) -- with one two's-complement byte per code in Values,
 * each column padded with 0 to a multiple of 16 codes (16 bytes), and
 * tile_offset / ColInfo offsets counted in codes. spdp_spmspv* on such a
 * handle computes y[b,m] = fp16(s[m] * sum_k q[m,k] xm[b,k]) (fp32
 * accumulation, the scale applied once per row, one rounding to fp16).
 *
 *   bits     2..8 (the paper uses 4); otherwise SPDP_ERR_INVALID_ARG.
 *   Non-finite weights: SPDP_ERR_INVALID_ARG. Other arguments, ownership
 *   and errors as spdp_encode. Products of one spdp_spmspv_many call must
 *   all be fp16 or all be codes.
 */
int spdp_encode_rtn(const uint16_t* W, int64_t rows, int64_t cols,
                    int32_t tile_m, int32_t tile_k, int32_t bits,
                    spdp_handle_t* out);
/* spdp_encode_rtn_host -- the same without a device copy (host-only handle,
 * for spdp_format; spdp_spmspv on it is SPDP_ERR_INVALID_ARG). */
int spdp_encode_rtn_host(const uint16_t* W, int64_t rows, int64_t cols,
                         int32_t tile_m, int32_t tile_k, int32_t bits,
                         spdp_handle_t* out);


/*
 * Offline preparation helpers (host only, no device work).
 *
 * spdp_prune_magnitude -- global unstructured magnitude pruning (Sec. 2.2,
 * static pruning by magnitude): out = W with the floor(sparsity*n) entries of
 * smallest |W| set to +0. Ties in magnitude go by index, lowest first. W and
 * out may alias. NaN entries are SPDP_ERR_INVALID_ARG; sparsity in [0, 1].
 */
int spdp_prune_magnitude(const uint16_t* W, int64_t n, double sparsity,
                         uint16_t* out);

/*
 * spdp_calibrate_threshold -- TEAL-style threshold (Sec. 5.1: a quantile of
 * the empirical distribution of |x| over calibration activations): *t is
 * the ceil(p*n)-th smallest |X| over all n entries, so the strict rule
 * |x| > t drops at least that many; p == 0 (or n == 0) gives -1, which keeps
 * everything. NaN entries are SPDP_ERR_INVALID_ARG; p in [0, 1].
 */
int spdp_calibrate_threshold(const uint16_t* X, int64_t n, double p, float* t);

/*
 * spdp_threshold_code -- the integer form of a threshold that the kernels
 * use: for finite-or-infinite, non-NaN fp16 x, |x| > threshold holds iff
 * code < (x & 0x7FFF) <= 0x7C00. code = -1 for a negative threshold, else the
 * bit pattern of the largest fp16 magnitude not above the threshold.
 */
int spdp_threshold_code(float threshold, int32_t* code);

/* Static text for a status code, and the calling thread's last error detail. */
const char* spdp_strerror(int status);
const char* spdp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPDP_H */
