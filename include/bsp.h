/*
 * bsp.h - block-structured pruned conv / FC inference on AMD MI355X (gfx950).
 *
 * The pruning regularity is the paper's block-based scheme (Sec. 4.1.1): the
 * GEMM-form weight matrix of a layer (rows = output filters, columns =
 * Cin*kh*kw with column q = (c*kh + r)*kw + s, Sec. 4.2) is cut into blocks
 * of bh x bw, and inside every block whole columns (BSP_COL) or whole rows
 * (BSP_ROW) are removed.  The group measure is the squared Frobenius norm of
 * a block's column / row (Eqs. 2-3), selected one-shot by magnitude
 * (Sec. 5.1).  A block size of 0 means the whole extent, so a whole-matrix
 * block is structured (filter / channel) pruning (Sec. 4.4).
 *
 * Block-punched pruning (BSP_PUNCHED, Sec. 4.1.2 with the group norm of
 * Eq. 4) is the conv-layer variant: the weight tensor is cut into blocks of
 * bh filters x bw input channels, and a kernel location (r, s) is kept or
 * removed in every kernel of a block at once; its score is the squared norm
 * of the weights at (r, s) over the block's kernels.
 *
 * Conventions for every entry point
 *  - Pointers named w, mask, values, indices, rowptr, dev_tiles, x, y, bias
 *    are DEVICE pointers owned by the caller.  The library keeps no state
 *    between calls and owns no memory after a call returns.
 *  - `stream` is a hipStream_t passed as void* (NULL = legacy default stream).
 *    Calls are asynchronous on it unless stated otherwise.
 *  - Arguments are validated before anything is launched; on an argument
 *    error nothing is written and a negative status is returned.  A launch
 *    failure returns BSP_EDEVICE.  Faults inside kernels surface at the
 *    caller's next synchronisation.
 *  - Kept groups per block = ceil(extent / rate) with an integer rate >= 1;
 *    ties in the score go to the lower index; scores are summed in fp64 in
 *    ascending index order; blocks are anchored at (0, 0) and a ragged last
 *    block keeps ceil(its own extent / rate).
 *  - No exceptions cross this interface.  Calls on different streams may run
 *    concurrently.
 */
#ifndef BSP_H
#define BSP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BSP_OK = 0,
    BSP_EINVAL = -1,        /* bad argument, shape or null pointer            */
    BSP_EUNSUPPORTED = -2,  /* valid request this library does not implement  */
    BSP_EDEVICE = -3,       /* HIP launch / copy / allocation failure          */
    BSP_EMASK = -4,         /* mask given to bsp_pack lacks the block structure */
    BSP_ETOOLARGE = -5      /* input beyond the fixed scratch of bsp_prune_noalloc */
} bsp_status;

typedef enum { BSP_F32 = 0, BSP_BF16 = 1 } bsp_dtype;

typedef enum {
    BSP_ROW = 0,            /* whole rows removed inside each block   (Eq. 2) */
    BSP_COL = 1,            /* whole columns removed inside each block (Eq. 3) */
    BSP_UNSTRUCTURED = 2,   /* magnitude top-k over the whole layer (Sec. 2.1.1) */
    BSP_DENSE = 3,          /* nothing removed                                 */
    BSP_PUNCHED = 4,        /* kernel locations removed per block of filters x
                               input channels (Sec. 4.1.2, Eq. 4)              */
    BSP_ROWCOL = 5,         /* rows and columns removed in the same block
                               (Eqs. 2 and 3 together, Sec. 4.2): a block keeps
                               ceil(bh/rate) rows x ceil(bw/rate) columns;
                               packed like BSP_COL with zeros for its removed
                               rows; no per-block counts                       */
    BSP_PATTERN = 6         /* pattern-based pruning of 3x3 kernels (Sec. 2.1,
                               the comparison point of Sec. 5.2.3): 4 weights
                               per kept kernel in one of a library of bh
                               patterns (0 -> 8; the most frequent top-4 sets),
                               connectivity pruning keeps ceil(kernels*9 /
                               (4*rate)) kernels; khw must be 9; packed and run
                               like BSP_UNSTRUCTURED                           */
} bsp_regularity;

typedef struct {
    int32_t rows, cols;     /* GEMM form: rows = Cout / out_features,
                               cols = Cin*kh*kw / in_features                 */
    int32_t bh, bw;         /* block size; 0 => whole extent.  BSP_PUNCHED:
                               bh filters x bw input channels                  */
    int32_t regularity;     /* bsp_regularity                                  */
    int32_t rate;           /* integer >= 1; kept per block = ceil(extent/rate);
                               UNSTRUCTURED keeps ceil(rows*cols/rate);
                               PUNCHED keeps ceil(khw/rate) locations          */
    int32_t khw;            /* BSP_PUNCHED: kernel locations per input channel
                               (kh*kw; cols = Cin*khw, column = c*khw + r*kw + s);
                               must equal kh*kw of the conv shape.  Ignored by
                               the other regularities (0 reads as 1).          */
    const int32_t *counts;  /* HOST array or NULL.  Kept groups of every block
                               (Sec. 4.1.1: the same or a different number per
                               block), n_block_rows x n_block_cols row-major
                               (PUNCHED: filter blocks x channel blocks), each
                               0 .. the block's group count (columns, rows or
                               kernel locations); replaces ceil(extent/rate)
                               for BSP_ROW, BSP_COL and BSP_PUNCHED.  Read by
                               every call that takes the scheme; tiles packed
                               with other counts are detected like another
                               geometry.  NULL: the uniform rule.             */
} bsp_scheme;

/* Convolution geometry: dilation 1, groups 1, NCHW activations, OIHW weights. */
typedef struct {
    int32_t n, cin, h, w, kh, kw, stride_h, stride_w, pad_h, pad_w;
} bsp_conv_shape;

/* Sizes (in elements, and bytes for dev_tiles) of the buffers bsp_pack fills.
 * Host-only, pure.  conv_or_null selects the conv layout (its n is ignored);
 * NULL means a linear layer.  The canonical arrays are
 *   COL, PUNCHED, ROWCOL: values = rows * kept_per_row, indices = n_block_rows * kept_per_row,
 *        rowptr = n_block_rows + 1 (PUNCHED keeps Cin*ceil(khw/rate) per row)
 *   ROW: values = nnz, indices = kept rows summed over blocks, rowptr = n_blocks + 1
 *   DENSE / UNSTRUCTURED / PATTERN: values = rows * cols, indices = rowptr = 0. */
bsp_status bsp_packed_sizes(const bsp_scheme *scheme, const bsp_conv_shape *conv_or_null,
                            bsp_dtype wdt, int64_t *n_values, int64_t *n_indices,
                            int64_t *n_rowptr, int64_t *dev_tile_bytes);

/* Prune (Sec. 4.1.1 with the group norms of Eqs. 2-3, Sec. 4.1.2 with the
 * norm of Eq. 4, one-shot magnitude selection of Sec. 5.1): w is the GEMM-form
 * weight matrix, row-major rows x cols, of dtype wdt; mask (rows x cols bytes,
 * row-major) receives 1 for kept and 0 for removed weights.  Async.  The
 * whole-layer rankings of BSP_UNSTRUCTURED and BSP_PATTERN allocate a scratch
 * buffer on `stream` (stream-ordered) and free it before returning.  With
 * per-block counts the counts go to such a buffer and the call waits for
 * `stream` before returning. */
bsp_status bsp_prune(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, uint8_t *mask,
                     void *stream);

/* bsp_prune for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same masks, bit for bit, and no allocation of any kind.
 *  - BSP_UNSTRUCTURED ranks the layer in the library's fixed scratch: one
 *    static device array per GPU (about 257 KB, held until the process ends)
 *    that serves rows * cols <= 2^28 weights; larger layers return
 *    BSP_ETOOLARGE before anything is launched.  Every call on a GPU shares
 *    that GPU's array: calls that overlap on one GPU (concurrent streams or
 *    threads) race and must be serialised by the caller.  What the select
 *    reads of the array is first written by the same call.
 *  - The block regularities (ROW, COL, PUNCHED, ROWCOL) and DENSE use no
 *    scratch.
 *  - BSP_PATTERN and per-block counts (which need a buffer sized by the
 *    layer) return BSP_EUNSUPPORTED.
 * Async on `stream`; nothing else changes from bsp_prune. */
bsp_status bsp_prune_noalloc(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, uint8_t *mask,
                             void *stream);

/* Pack the masked weights (the compact storage idea of Sec. 4.3, in this
 * library's own layout).  SYNCHRONOUS: checks on the device that the mask
 * has the block structure of the scheme with exactly ceil(extent/rate) kept
 * groups per block and returns BSP_EMASK otherwise (outputs then unspecified).
 *   values / indices / rowptr: the canonical packing
 *     COL: for block-row i, indices[rowptr[i] .. rowptr[i+1]) are its kept
 *          columns in ascending order; values[rowptr[i]*bh + p*len + t] =
 *          W[i*bh + p][indices[rowptr[i] + t]] (len = rowptr[i+1]-rowptr[i]).
 *     PUNCHED: as COL; block-row i (bh filters) keeps whole GEMM columns, the
 *          kept locations of each input channel.
 *     ROW: for block b = i*n_block_cols + j, indices[rowptr[b] .. rowptr[b+1])
 *          are its kept rows ascending; its values are those rows restricted
 *          to the block's columns, [t][q_local], blocks stored in order b.
 *     DENSE / UNSTRUCTURED / PATTERN: values = W * mask (rows x cols); indices and
 *          rowptr are not written (may be NULL).
 *   dev_tiles: the kernels' private layout (pre-decoded gather offsets for
 *     the given conv geometry, MFMA-ordered weight tiles, channel-chunk
 *     table), dev_tile_bytes from bsp_packed_sizes.  It is only valid for the
 *     same scheme, dtype and geometry (conv_or_null) at bsp_conv2d /
 *     bsp_linear time; a mismatch is detected on the device and the output
 *     is filled with NaN.
 * Returns BSP_EUNSUPPORTED when one 32-wide step of a kept-column list spans
 * more input channels than one LDS stage holds (only possible for very
 * sparse whole-width column blocks of 1x1 convs). */
bsp_status bsp_pack(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, const uint8_t *mask,
                    void *values, int32_t *indices, int32_t *rowptr, void *dev_tiles,
                    const bsp_conv_shape *conv_or_null, void *stream);

/* Inverse of the canonical packing (the compact storage of Sec. 4.3 read
 * back): w_masked_out (rows x cols, dtype) = W * mask, bit-exact.  Async.
 * For tests and checkpoints. */
bsp_status bsp_unpack(const bsp_scheme *scheme, bsp_dtype wdt, const void *values,
                      const int32_t *indices, const int32_t *rowptr, void *w_masked_out,
                      void *stream);

/* Blocked Compressed Storage (BCS, Sec. 4.3) of a BSP_COL or BSP_PUNCHED
 * packing (indices / rowptr from bsp_pack, same scheme): CSR whose column
 * indices are stored once per run of consecutive rows that keep the same
 * columns.  The BCS weights array is the canonical `values` array itself (the
 * kept weights row by row, ascending columns).  Outputs (device, int32):
 *   occurrence   first row of each run, then rows    (up to n_block_rows + 1)
 *   compact_cols each run's kept columns, run by run (up to n_indices)
 *   col_stride   start of each run in compact_cols, then its length
 *                                                     (up to n_block_rows + 1)
 *   row_offset   start of each row in values          (rows + 1)
 *   n_runs       the number of runs (one int32)
 * Runs never split a block-row; neighbouring block-rows with identical lists
 * merge.  Other regularities return BSP_EUNSUPPORTED.  Async. */
bsp_status bsp_to_bcs(const bsp_scheme *scheme, const int32_t *indices, const int32_t *rowptr,
                      int32_t *occurrence, int32_t *compact_cols, int32_t *col_stride, int32_t *row_offset,
                      int32_t *n_runs, void *stream);

/* Forward of a pruned conv layer (the layer of Sec. 4.2 with pruned weights):
 *   y[n,o,oh,ow] = bias[o] + sum_{kept (c,r,s)} W[o,c,r,s] * x[n,c,oh*sh-ph+r,ow*sw-pw+s]
 * then ReLU if relu != 0.  x: NCHW of in_dt (must equal the packed dtype);
 * y: NCHW [n][rows][Ho][Wo] of out_dt (fp32 accumulation, RNE to bf16).
 * Only kept weights are multiplied; inputs must be finite (a removed weight
 * is never multiplied, so Inf/NaN inputs do not propagate through it).
 * bias may be NULL.  Async.
 * Device workspace: some calls use a workspace that the library allocates
 * on the device at the first call that needs it (or a larger one) and keeps
 * until the process ends:
 *  - layers with a kernel larger than 1x1 whose output plane has at most 16
 *    pixels, and bf16 layers with per-block-row lists (COL, PUNCHED, ROWCOL
 *    without counts) whose plane has at most 64 pixels (strided, or whose
 *    expanded input for 64 images stays within 24 MiB), and bf16 1x1
 *    stride-2 layers without padding over one identity list (ROW or DENSE
 *    without counts) whose plane has at most 196 pixels, expand x into it
 *    (n x cin*kh*kw planes of Ho*Wo elements, rounded up to 8 for the bf16
 *    pipelined kernel);
 *  - bf16 layers run by the pipelined pointwise kernel (1x1, linear and the
 *    expanded layers above) whose output splits into at most 128 workgroup
 *    tiles (64 or 128 output pixels x 64 to 256 rows) split their K loop
 *    over workgroups and keep fp32 partial sums there (parts x n x rows x
 *    Ho*Wo floats).
 * Calls that use the workspace must not overlap on one device (other
 * streams, other threads), and the first one cannot be captured into a
 * graph. */
bsp_status bsp_conv2d(const bsp_scheme *scheme, const bsp_conv_shape *shape, bsp_dtype in_dt,
                      bsp_dtype out_dt, const void *x, const void *dev_tiles,
                      const float *bias_or_null, int32_t relu, void *y, void *stream);

/* Forward of a pruned FC layer on feature-major activations (an FC layer's
 * weight matrix is its own GEMM form, pruned in blocks as in Sec. 4.1.1; the
 * layer computation with weights W_i and bias b_i of Sec. 4.2):
 *   y[o][b] = bias[o] + sum_{kept k} W[o][k] * x[k][b], then ReLU if relu.
 * x: [cols][batch], y: [rows][batch].  dev_tiles packed with conv_or_null =
 * NULL.  Async.  bf16 layers with small batches (at most 128 workgroup
 * tiles) split the K loop and use the device workspace described at
 * bsp_conv2d, with the same rules. */
bsp_status bsp_linear(const bsp_scheme *scheme, int32_t batch, bsp_dtype in_dt, bsp_dtype out_dt,
                      const void *x, const void *dev_tiles, const float *bias_or_null,
                      int32_t relu, void *y, void *stream);

/* 2x2 max pooling, stride 2 (floor), NCHW, same dtype in and out: the glue
 * between VGG-16 stages (not part of the pruning method).  y is
 * [n][c][h/2][w/2]; each output is the largest of its four inputs, copied
 * bit-exactly; a NaN in a window makes the output NaN.  Async. */
bsp_status bsp_maxpool2x2(bsp_dtype dt, int32_t n, int32_t c, int32_t h, int32_t w,
                          const void *x, void *y, void *stream);

/* Static string for a status code. */
const char *bsp_status_string(bsp_status status);

/* Library version, e.g. 100 for 0.1.0. */
int32_t bsp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BSP_H */
