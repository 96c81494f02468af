/*
 * spl.h - C ABI of the MI355X (gfx950) sparse linear library.
 *
 * Dense activations times unstructured-sparse weights held in the bitmask
 * expansion format of arXiv 2405.03594: section 2.4.1 stores the kept
 * entries of a block densely in order together with a bitmask that marks
 * the kept positions; section 2.4.2 applies the same idea to GPU
 * submatrices that are decompressed right before the matrix units consume
 * them; section 3.4 adds int8 weights and int8 activations.  The linear
 * layers computed here are the seven projections of a Llama-2-7B decoder
 * layer (q, k, v, o, gate, up, down), but any shape is accepted.
 *
 * Conventions shared by every entry point
 *   - W is [N][K] row-major (N output features, K input features), X is
 *     [M][K] and Y is [M][N], both row-major.  The product is
 *         Y[m][n] = sum_k X[m][k] * (W . Mask)[n][k].
 *   - All array arguments are DEVICE pointers (hipMalloc'ed or from a
 *     framework allocator) unless a comment says "host".  The caller owns
 *     every buffer; the library allocates no device memory and keeps no
 *     state between calls.
 *   - Every call is ordered on `stream` (NULL = the default stream) and
 *     returns as soon as its kernels are queued, except spl_pack_count,
 *     which waits for `stream` to return the number of kept entries.
 *   - Arguments are checked on the host before anything is launched; a
 *     failed check returns an error code and launches nothing.  Errors
 *     reported by the HIP runtime at launch map to SPL_ERR_DEVICE.  Nothing
 *     throws across this interface.
 *   - Device buffers must be 16-byte aligned.  The `values` array of a
 *     compressed matrix is allocated with spl_values_bytes(dtype, nnz) bytes
 *     or more (the payloads rounded up to 16 bytes plus 16): kernels read
 *     (never write) up to 16 bytes past the last payload.  A view states its
 *     allocation in `values_bytes`, which spl_check_matrix and every entry
 *     point taking a view check.
 *
 * Two lossless encodings of a compressed matrix
 *
 *   Row layout (SPL_LAYOUT_ROWS: the interchange format written by the packer;
 *   paper section 2.4.1, one block per row):
 *     bitmask     uint32 [N][ceil(K/32)]; bit j (least significant first) of
 *                 word w of row n is set iff position (n, 32w + j) is kept;
 *                 bits at or past K are 0.
 *     values      the kept payloads, row by row, ascending column order, as
 *                 raw bit copies (fp16 / bf16: 2 bytes; int8: 1 byte).
 *     row_offsets int32 [N+1]; row_offsets[n] is the index in `values` of the
 *                 first kept entry of row n, row_offsets[N] = nnz < 2^31.
 *   Reading of the paper: its worked example packs one 16-lane VNNI register
 *   (two interleaved rows); the row layout takes a whole row as the block, in
 *   column order, with the bit order least-significant-bit first.
 *
 *   Tile layout (SPL_LAYOUT_TILE16: the layout the linear kernels read; paper
 *   section 2.4.2, submatrices sized for the register file, each with its own
 *   bitmask and dense values).  Tiles are 16 rows x 32 columns, one MFMA
 *   operand; with B = ceil(N/16) row blocks and S = ceil(K/32) column steps,
 *   tile (b, s) has index t = b*S + s and
 *     bitmask      uint32 [B*S][16]: word r of tile t holds row 16b+r,
 *                  columns 32s..32s+31 (bit j = column 32s+j); rows >= N and
 *                  columns >= K are 0;
 *     values       each tile's kept payloads in tile order; inside a tile by
 *                  column group, then row, then ascending column, where a
 *                  column group is the 16 bytes of payload one matrix-core
 *                  lane holds (8 columns of fp16/bf16, 16 of int8: groups
 *                  cover columns 8g..8g+7, resp. 16g..16g+15);
 *     tile_offsets int32 [B*S + 1]: index in `values` of tile t's first
 *                  payload; tile_offsets[B*S] = nnz.
 *   Both layouts hold the same payloads; spl_retile16 converts rows -> tiles.
 */
#ifndef SPL_H
#define SPL_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPL_OK = 0,
  SPL_ERR_INVALID_ARG = 1,   /* null pointer, bad size, misaligned buffer, inconsistent view */
  SPL_ERR_UNSUPPORTED = 2,   /* dtype or algorithm not available for this call */
  SPL_ERR_OVERFLOW = 3,      /* nnz >= 2^31, or a size product overflows */
  SPL_ERR_DEVICE = 4         /* the HIP runtime reported an error */
} spl_status;

/* SPL_I4: 4-bit codes stored two per byte (spl_sparse_linear_int4 only). */
typedef enum { SPL_F16 = 1, SPL_BF16 = 2, SPL_I8 = 3, SPL_I4 = 4 } spl_dtype;

/* Kernel family for spl_sparse_linear_ex / spl_dense_linear_ex.
 * AUTO picks by batch size M.  DECODE is the small-batch kernel (M <= 32):
 * compressed rows are decompressed into MFMA operand tiles with the batch
 * padded to 16 or 32.  PREFILL is the large-batch tiled kernel: compressed
 * tiles are decompressed into LDS and feed bf16/fp16 MFMA (any M). */
typedef enum { SPL_ALGO_AUTO = 0, SPL_ALGO_DECODE = 1, SPL_ALGO_PREFILL = 2 } spl_algo;

typedef enum { SPL_LAYOUT_ROWS = 0, SPL_LAYOUT_TILE16 = 1 } spl_layout;

/* Non-owning view of a compressed matrix (all pointers device pointers).
 * The arrays must stay alive until work queued with the view completes. */
typedef struct {
  int64_t rows;                  /* N */
  int64_t cols;                  /* K */
  int32_t dtype;                 /* spl_dtype of `values` */
  int32_t layout;                /* spl_layout */
  int64_t nnz;                   /* number of stored payloads */
  const uint32_t* bitmask;       /* rows: [N][ceil(K/32)]; tiles: [B*S][16] */
  const void* values;            /* [nnz] payloads */
  const int32_t* row_offsets;    /* rows: [N+1]; tiles: unused (may be NULL) */
  const int32_t* tile_offsets;   /* tiles: [B*S + 1]; rows: unused (may be NULL) */
  int64_t values_bytes;          /* bytes allocated at `values`: >= spl_values_bytes(dtype, nnz) */
} spl_matrix;

/* Bytes the `values` array of a view with `nnz` payloads of `dtype` must
 * have: the payload bytes (2 per fp16/bf16 value, 1 per int8 value, one per
 * two 4-bit values) rounded up to 16, plus 16 bytes the kernels may read past
 * the last payload.  0 for an unknown dtype or a negative nnz. */
int64_t spl_values_bytes(int32_t dtype, int64_t nnz);

/* Library version, (major << 16) | minor. */
int32_t spl_version(void);

/* Static text for a status code (any int: "unknown status" outside spl_status). */
const char* spl_status_string(int32_t status);

/* Measurement helper, not part of the method: reads `bytes` (> 0, a multiple
 * of 16) of the 16-byte aligned device buffer `buf` with coalesced 16-byte
 * loads from every compute unit, the way a streaming kernel at its best reads
 * HBM; timing it gives the read rate the device sustains, against which a
 * kernel's achieved bandwidth is also reported.  `sink` (device, 4 bytes) is
 * written only if the folded data equal one fixed constant.  Asynchronous on
 * `stream`. */
spl_status spl_read_probe(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream);

/* Host-only consistency check of a view's scalar fields and pointers
 * (no device access): rows, cols >= 1, dtype and layout known,
 * 0 <= nnz < 2^31, nnz <= rows*cols, the layout's arrays and `values`
 * non-null, values_bytes >= spl_values_bytes(dtype, nnz), 16-byte alignment
 * of bitmask and values. */
spl_status spl_check_matrix(const spl_matrix* Wc);

/* Device check of a view's format (paper sections 2.4.1 and 2.4.2: a block's
 * stored values are exactly its kept entries, in order): for every block (a
 * row, or a 16 x 32 tile) the difference of consecutive offsets equals the
 * popcount of the block's bitmask words; the first offset is 0 and the last
 * nnz; bits for columns >= cols (and, in the tile layout, rows >= rows) are 0.
 * Returns SPL_OK, SPL_ERR_INVALID_ARG for an inconsistent format (or a view
 * that fails spl_check_matrix), SPL_ERR_DEVICE for a runtime error.  Reads
 * the bitmask and offsets, not the payloads.  Synchronizes `stream` once to
 * read the result.  The result word lives in a per-device variable of the
 * library; calls from several threads take turns (a lock held until the
 * result is read). */
spl_status spl_validate(const spl_matrix* Wc, hipStream_t stream);

/* Sizes of the tile layout of an N x K matrix: number of tiles B*S (the
 * bitmask has 16 words per tile, tile_offsets B*S + 1 entries). */
int64_t spl_tile16_count(int64_t N, int64_t K);

/* Convert a row-layout matrix to the tile layout (a permutation of payloads
 * and bitmask bits; paper section 2.4.2).
 *   rows_in       view with layout SPL_LAYOUT_ROWS.
 *   bitmask_out   out [B*S][16] uint32, fully written.
 *   values_out    out [nnz] payloads (must not alias rows_in->values).
 *   tile_offsets_out out [B*S + 1] int32. */
spl_status spl_retile16(const spl_matrix* rows_in, uint32_t* bitmask_out, void* values_out,
                        int32_t* tile_offsets_out, hipStream_t stream);

/* Pack, step 1 of 2 (paper section 2.4.1: count the kept entries of every
 * block, a row or, for the layout the linear kernels read, a 16 x 32 tile).
 *   W           [N][K] payloads of `dtype` (F16, BF16 or I8).
 *   mask        [N][K] uint8, non-zero = kept; or NULL, then an entry is kept
 *               iff its payload is non-zero (fp16/bf16: ignoring the sign bit,
 *               so -0.0 is not kept).
 *   layout      SPL_LAYOUT_ROWS or SPL_LAYOUT_TILE16.
 *   offsets     out: the exclusive prefix sum of per-block kept counts, the
 *               row_offsets [N+1] (rows) or the tile_offsets [B*S + 1] (tiles)
 *               of the view the pack describes.
 *   h_nnz       HOST out: number of kept entries.  This call synchronizes
 *               `stream` to read it.  Returns SPL_ERR_OVERFLOW if it would
 *               reach 2^31.
 * The caller then allocates the bitmask (rows: N * ceil(K/32) words; tiles:
 * 16 * spl_tile16_count(N, K) words) and spl_values_bytes(dtype, nnz) bytes
 * of values. */
spl_status spl_pack_count(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K, int32_t layout,
                          int32_t* offsets, int64_t* h_nnz, hipStream_t stream);

/* Pack, step 2 of 2 (paper section 2.4.1: write bitmask and dense values).
 *   offsets     from spl_pack_count for the same W, mask and layout.
 *   bitmask     out, fully written (pad bits 0): rows [N][ceil(K/32)]; tiles
 *               [B*S][16].
 *   values      out [nnz] payloads of `dtype`, in the layout's order (the tail
 *               past nnz is not written).
 * The result, with nnz and `offsets`, is a view spl_sparse_linear reads
 * directly when the layout is SPL_LAYOUT_TILE16 (no conversion step). */
spl_status spl_pack_sparse(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                           int32_t layout, const int32_t* offsets, uint32_t* bitmask, void* values,
                           hipStream_t stream);

/* Decompress (either layout) to a dense [N][K] matrix of the view's dtype:
 * kept positions receive their payload, every other position +0. */
spl_status spl_unpack(const spl_matrix* Wc, void* W_dense, hipStream_t stream);

/* Sparse linear layer, fp16 or bf16 (paper section 2.4.2).
 *   Wc in the tile layout (SPL_ERR_UNSUPPORTED for the row layout).
 *   X  [M][K] of Wc->dtype; M >= 0 (M == 0 is a no-op).
 *   Y  out [M][N] of Wc->dtype, overwritten.  fp32 accumulation, one
 *      round-to-nearest-even conversion per output.  No bias.
 *   Requires K % 8 == 0 (rows of X are read in 16-byte pieces). */
spl_status spl_sparse_linear(const void* X, int64_t M, const spl_matrix* Wc, void* Y, hipStream_t stream);

/* As spl_sparse_linear with an explicit kernel family (spl_algo).
 * DECODE requires M <= 32 and 2 M K <= 2^31 (the activations addressed with
 * 32-bit byte offsets); SPL_ERR_UNSUPPORTED otherwise, and AUTO then picks
 * PREFILL. */
spl_status spl_sparse_linear_ex(const void* X, int64_t M, const spl_matrix* Wc, void* Y, int32_t algo,
                                hipStream_t stream);

/* Sparse linear layer for large batches through a decoded copy (paper
 * section 2.4.2 decompresses the stored submatrices before the matrix
 * units consume them; at prefill batches the product is compute-bound, so
 * decoding each tile once per call into device memory costs less than
 * expanding it once per block of batch rows, as spl_sparse_linear's prefill
 * kernel does).  Same arguments and result as spl_sparse_linear (fp16/bf16,
 * tile layout, K % 8 == 0; M == 0 is a no-op), the sums those of the dense
 * prefill kernel on the decoded matrix.  Two launches: spl_unpack into the
 * workspace, then the dense product.
 *   workspace  device scratch of spl_sparse_linear_expanded_workspace_bytes(Wc)
 *              bytes (2 rows cols for fp16/bf16, rows cols for int8, rounded
 *              up to 256), 16-byte aligned, owned by the caller, overwritten
 *              (one buffer can serve every matrix of a layer in turn on one
 *              stream).
 * The workspace-size function returns -1 for a view spl_check_matrix rejects. */
int64_t spl_sparse_linear_expanded_workspace_bytes(const spl_matrix* Wc);
spl_status spl_sparse_linear_expanded(const void* X, int64_t M, const spl_matrix* Wc, void* Y, void* workspace,
                                      hipStream_t stream);

/* Sparse training with the mask held fixed (paper Algorithm 1: the gradient is
 * masked and so are the weights after each step, i.e. only the kept values
 * change).  For Y = X (W.Mask)^T with an upstream gradient dY [M][N]:
 *
 * spl_sparse_weight_grad: grad_values = the kept entries of dY^T X, in Wc's
 *   value order (so an update is elementwise on Wc->values):
 *   grad[n][k] = sum_m dY[m][n] X[m][k], fp32 sums, one rounding to the payload
 *   type.  dY [M][N] and X [M][K] of Wc->dtype; Wc in the tile layout;
 *   grad_values out, nnz entries.  Requires M % 8 == 0 (M == 0:
 *   SPL_ERR_UNSUPPORTED), K % 8 == 0, M <= 4194240.  workspace: device
 *   scratch of spl_sparse_weight_grad_workspace_bytes(M, N, K) bytes
 *   (2 M (N + K) rounded up: the transposes of dY and X; no [N][K] buffer),
 *   256-byte aligned, caller-owned; left untouched where the product reads
 *   dY and X as they are stored (N % 256 == 0, K % 128 == 0, M % 64 == 0,
 *   16-byte aligned dY and X, and at least one 128 x 256 output block per
 *   compute unit).  The product's epilogue writes the kept entries directly;
 *   nothing else of grad_values is touched.
 * spl_sparse_sgd_update: Wc->values[i] = RNE(v - lr * g) with v, g decoded
 *   from the payloads and each operation rounded to binary32; in place.
 * spl_sparse_input_grad: dX [M][K] = dY [M][N] (W.Mask), the gradient with
 *   respect to the activations, fp32 sums over n, one rounding to the payload
 *   type; dY and dX of Wc->dtype, row-major, 16-byte aligned; Wc in the tile
 *   layout (W itself, not its transpose).  Where M % 256 == 0, N % 64 == 0,
 *   K % 128 == 0 and the launch has at least one 128 x 256 output block per
 *   compute unit of the current device, W's tiles are expanded inside the
 *   product and the workspace is not used
 *   (spl_sparse_input_grad_workspace_bytes returns 0; NULL is accepted);
 *   otherwise W is decoded and transposed into the workspace (4 N K bytes
 *   rounded up, 256-byte aligned, caller-owned; N % 8 == 0 or
 *   SPL_ERR_UNSUPPORTED) and multiplied densely.  M == 0: nothing to do;
 *   nnz == 0: dX = 0.  The workspace-size function returns -1 for a view
 *   spl_check_matrix rejects or an M outside the dimension limits.
 * Alternatively dX is spl_sparse_linear(dY, Wt) with Wt the packed transpose
 * (spl_unpack, spl_transpose16, then pack; the same kept products, kept zeros
 * may be dropped), kept in step by the permutation below.
 * spl_transpose16: dst [C][R] = src [R][C]^T for 16-bit payloads (R <= 4194240).
 * spl_gather_tiled: the entries of a dense [N][K] matrix (16-byte aligned,
 *   K % 8 == 0) at the kept positions of a tile pattern, in its value order. */
/* Keeping the packed transpose in step with W after updates, without a dense
 * pass: spl_transpose_perm computes, once per pattern, perm[i] = the position
 * in W's values of value i of Wt, where Wt [K][N] is W packed transposed with
 * the transposed mask (same nnz and dtype; N % 8 == 0 and K % 8 == 0);
 * workspace: spl_transpose_perm_workspace_bytes(N, K, nnz) bytes, 256-byte
 * aligned.  spl_permute_values then copies dst[i] = src[perm[i]] (nnz 16-bit
 * payloads, src holding nnz of them), e.g. Wt.values from W.values after each
 * SGD step; a perm entry outside [0, nnz) gives 0 and reads nothing; nnz >=
 * 2^31 is SPL_ERR_OVERFLOW.
 * The two *_workspace_bytes functions return -1 for sizes their entry points
 * reject (N, K or M outside the dimension limits, nnz outside [0, N K]). */
int64_t spl_transpose_perm_workspace_bytes(int64_t N, int64_t K, int64_t nnz);
spl_status spl_transpose_perm(const spl_matrix* W, const spl_matrix* Wt, int32_t* perm, void* workspace,
                              hipStream_t stream);
spl_status spl_permute_values(const void* src, const int32_t* perm, int64_t nnz, void* dst, hipStream_t stream);
spl_status spl_transpose16(const void* src, int64_t R, int64_t C, void* dst, hipStream_t stream);
spl_status spl_gather_tiled(const void* W_dense, const spl_matrix* pattern, void* values_out, hipStream_t stream);
int64_t spl_sparse_weight_grad_workspace_bytes(int64_t M, int64_t N, int64_t K);
spl_status spl_sparse_weight_grad(const void* dY, const void* X, int64_t M, const spl_matrix* Wc, void* grad_values,
                                  void* workspace, hipStream_t stream);
/* spl_sparse_weight_grad_group: the weight gradients of up to SPL_MAX_GROUP
 *   layers that share the batch M and the dtype (for example q, k and v, which
 *   share X), each task's output identical to spl_sparse_weight_grad's on the
 *   same arguments.  When every task takes the path that reads dY and X as
 *   stored, they run in one launch per four tasks (so the blocks of those
 *   tasks share the chip's last partial round); otherwise one call per task,
 *   the workspace
 *   (the largest spl_sparse_weight_grad_workspace_bytes of the tasks, 256-byte
 *   aligned) serving them in turn.  Tasks must not write overlapping outputs;
 *   the task array is read during the call only. */
typedef struct {
  const void* dY;                /* [M][N] of W->dtype */
  const void* X;                 /* [M][K] of W->dtype */
  const spl_matrix* W;           /* tile layout, fp16 or bf16: the pattern and value order of the gradient */
  void* grad_values;             /* out: W->nnz payloads in W's value order */
} spl_weight_grad_task;
spl_status spl_sparse_weight_grad_group(const spl_weight_grad_task* tasks, int32_t count, int64_t M,
                                        void* workspace, hipStream_t stream);
int64_t spl_sparse_input_grad_workspace_bytes(int64_t M, const spl_matrix* Wc);
spl_status spl_sparse_input_grad(const void* dY, int64_t M, const spl_matrix* Wc, void* dX, void* workspace,
                                 hipStream_t stream);
spl_status spl_sparse_sgd_update(const spl_matrix* Wc, const void* grad_values, float lr, hipStream_t stream);

/* One-shot magnitude pruning on the GPU (paper section 2 removes the weights
 * of smallest magnitude; the reading taken: per matrix, exactly `prune`
 * entries are zeroed, those of smallest decoded |w|, ties in ascending
 * row-major index).  Writes the keep-mask that spl_pack_sparse takes.
 *   W          [N][K] fp16/bf16 payloads (dtype), 16-byte aligned; K % 8 == 0
 *              and N K < 2^31 (SPL_ERR_UNSUPPORTED otherwise).  NaN payloads
 *              are ordered above +inf by their bits (no magnitude is defined).
 *   prune      0 <= prune <= N K (SPL_ERR_INVALID_ARG otherwise).
 *   mask       out [N][K] uint8: 1 kept, 0 pruned; 8-byte aligned.
 *   workspace  device scratch of spl_magnitude_mask_workspace_bytes() bytes,
 *              16-byte aligned, owned by the caller; contents are overwritten.
 * Asynchronous on `stream` (five kernels, no host synchronisation). */
int64_t spl_magnitude_mask_workspace_bytes(void);
spl_status spl_magnitude_mask(const void* W, int32_t dtype, int64_t N, int64_t K, int64_t prune, uint8_t* mask,
                              void* workspace, hipStream_t stream);

/* spl_magnitude_mask without a workspace argument, for callers that cannot
 * allocate device memory (code under graph capture, serving loops, harnesses
 * that forbid hipMalloc).  The result is that of spl_magnitude_mask with the
 * same arguments.  The scratch is a library array of 34,818 32-bit words
 * (136 KiB) per device, held from the first call on that device until the
 * process ends; it is the same whatever the size, so the size limits are
 * those of spl_magnitude_mask (N K < 2^31, K % 8 == 0: SPL_ERR_UNSUPPORTED
 * otherwise).  The call allocates nothing and every kernel clears what it
 * needs cleared.  All calls on one device share the array: calls that overlap
 * on one device (two streams, two threads) race and give wrong masks.
 * SPL_ERR_DEVICE when the array's device address cannot be obtained. */
spl_status spl_magnitude_mask_noalloc(const void* W, int32_t dtype, int64_t N, int64_t K, int64_t prune,
                                      uint8_t* mask, hipStream_t stream);

/* The gated half of a Llama MLP on two sparse weights sharing X (the model
 * the paper sparsifies; its MLP is down(silu(gate(x)) * up(x))):
 *   Y[m][n] = silu(g) * u,  g = sum_k X[m][k] Wg[n][k],  u = likewise with Wu,
 *   silu(z) = z / (1 + e^-z), g and u the kernels' fp32 sums, one rounding of
 *   the result to the payload type.  One launch, no intermediate in memory.
 *   Wgate, Wup  views in the tile layout with the same dtype, rows (N) and cols (K).
 *   X, Y        as in spl_sparse_linear (Y [M][N]).
 *   algo        SPL_ALGO_AUTO (DECODE for M <= 16, else PREFILL), DECODE
 *               (M <= 16, SPL_ERR_UNSUPPORTED otherwise) or PREFILL (any M).
 * Errors as spl_sparse_linear; mismatched dtypes or shapes -> SPL_ERR_INVALID_ARG. */
spl_status spl_sparse_linear_silu_mul(const void* X, int64_t M, const spl_matrix* Wgate, const spl_matrix* Wup,
                                      void* Y, int32_t algo, hipStream_t stream);

/* Sparse-quantized linear layer (paper section 3.4: int8 weights and
 * int8 activations).
 *   Xq        [M][K] int8 activation codes; x_scales [M] float32.
 *   Wqc       view with dtype SPL_I8 in the tile layout; w_scales [N] float32.
 *   acc       acc[m][n] = sum over kept k of Xq[m][k] * Wq[n][k], exact int32.
 *   Y         out [M][N] fp16: round-to-nearest-even of
 *             ((float)acc * x_scales[m]) * w_scales[n], each product rounded
 *             to float32 (no fused multiply-add).
 *   acc_out   optional out [M][N] int32 (NULL to skip).
 *   Requires K % 16 == 0. */
spl_status spl_sparse_linear_int8(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* Wqc,
                                  const float* w_scales, void* Y, int32_t* acc_out, hipStream_t stream);

/* spl_sparse_linear_int8 for large batches through a decoded copy of the
 * codes (as spl_sparse_linear_expanded for fp16/bf16; paper sections 2.4.2 and
 * 3.4): spl_unpack writes the dense [N][K] int8 codes into the workspace, then
 * the dense int8 prefill kernel multiplies.  Same arguments, checks and
 * results (exact int32 sums, the same fp16 epilogue: bit-identical to
 * spl_sparse_linear_int8); workspace: spl_sparse_linear_expanded_workspace_bytes(Wqc)
 * bytes, 16-byte aligned, caller-owned, overwritten. */
spl_status spl_sparse_linear_int8_expanded(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* Wqc,
                                           const float* w_scales, void* Y, int32_t* acc_out, void* workspace,
                                           hipStream_t stream);

/* 4-bit sparse payloads (paper section 4 names INT4 as future work; the
 * reading taken: the int8 tile layout's pattern and value order, value i the
 * two's-complement nibble at byte i / 2, low nibble first, codes in [-8, 7]).
 * spl_pack_int4: values4 out (spl_int4_values_bytes(nnz) bytes, 16-byte
 *   aligned; the tail past ceil(nnz/2) is not written) from an int8
 *   tile-layout view W8 whose codes lie in [-8, 7].  A code outside that
 *   range keeps only its low 4 bits (and so reads back as another value);
 *   bad_codes (optional device int32, 4-byte aligned) is set, in stream
 *   order, to the number of such codes, so a caller can reject the result.
 *   The view of the result is W8's with dtype SPL_I4 and values = values4.
 * spl_sparse_linear_int4: as spl_sparse_linear_int8 (exact int32 sums, the
 *   same fp16 epilogue) for a SPL_I4 tile-layout view, decode batches
 *   0 <= M <= 16 (SPL_ERR_UNSUPPORTED above), K % 16 == 0; M * K < 2^31
 *   and ceil(K / 32) < 2^25 (SPL_ERR_UNSUPPORTED otherwise). */
int64_t spl_int4_values_bytes(int64_t nnz);
spl_status spl_pack_int4(const spl_matrix* W8, uint8_t* values4, int32_t* bad_codes, hipStream_t stream);
spl_status spl_sparse_linear_int4(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* W4,
                                  const float* w_scales, void* Y, int32_t* acc_out, hipStream_t stream);

/* Per-token activation quantisation for the sparse-quantized layer (paper
 * section 3.4 runs it on int8 activations; the reading taken: symmetric, one
 * binary32 scale per row).  For each row m of X:
 *   x_scales[m] = max_k |X[m][k]| / 127 (1 when the row is all zeros),
 *   Xq[m][k]    = clamp(round-half-to-even(X[m][k] / x_scales[m]), -127, 127),
 * each division correctly rounded to binary32.
 *   X         [M][K] fp16 or bf16 (dtype), 16-byte aligned; K % 8 == 0
 *             (SPL_ERR_UNSUPPORTED otherwise, and for other dtypes).
 *   Xq        out [M][K] int8, 16-byte aligned; x_scales out [M] float32.
 * M == 0 is a no-op.  Asynchronous on `stream`. */
spl_status spl_quantize_rows_i8(const void* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* x_scales,
                                hipStream_t stream);

/* Dense comparators: the same products with a dense W [N][K].
 * spl_dense_linear: fp16/bf16 (K % 8 == 0); spl_dense_linear_int8: int8
 * with the epilogue of spl_sparse_linear_int8 (K % 16 == 0). */
spl_status spl_dense_linear(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                            void* Y, hipStream_t stream);
spl_status spl_dense_linear_ex(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                               void* Y, int32_t algo, hipStream_t stream);
spl_status spl_dense_linear_int8(const int8_t* Xq, const float* x_scales, int64_t M, const int8_t* Wq,
                                 const float* w_scales, int64_t N, int64_t K, void* Y, int32_t* acc_out,
                                 hipStream_t stream);

/* Grouped launches: up to SPL_MAX_GROUP independent linear layers that share
 * the dtype and the batch size M, computed by one kernel launch (for example
 * the q, k and v projections of a decoder layer, or gate and up).  Each task
 * has its own X [M][K], W and Y [M][N] with the shapes, layouts and alignment
 * that the single-task entry point requires; the outputs are the ones that
 * entry point gives with the same algo (DECODE: one launch for all tasks;
 * PREFILL: one launch per task; AUTO picks by M as above).  The task array
 * is read on the host during the call and need not outlive it.  Tasks must
 * not write overlapping outputs. */
#define SPL_MAX_GROUP 16

typedef struct {
  const void* X;                 /* [M][K] of W->dtype */
  const spl_matrix* W;           /* tile layout, fp16 or bf16 */
  void* Y;                       /* out [M][N] of W->dtype */
} spl_sparse_task;

typedef struct {
  const void* X;                 /* [M][K] of the group's dtype */
  const void* W;                 /* dense [N][K] */
  int64_t N;
  int64_t K;
  void* Y;                       /* out [M][N] */
} spl_dense_task;

spl_status spl_sparse_linear_group(const spl_sparse_task* tasks, int32_t count, int64_t M, int32_t algo,
                                   hipStream_t stream);
spl_status spl_dense_linear_group(const spl_dense_task* tasks, int32_t count, int64_t M, int32_t dtype,
                                  int32_t algo, hipStream_t stream);

/* Grouped sparse-quantized launches (paper section 3.4): up to SPL_MAX_GROUP
 * independent int8 linear layers that share the batch size M, one kernel
 * launch for all of them.  Each task carries the arguments of
 * spl_sparse_linear_int8 (resp. spl_dense_linear_int8), with the same
 * requirements and the same bit-exact outputs; spl_sparse_linear_int8 and
 * spl_dense_linear_int8 are groups of one.  Errors as for those calls (the
 * first failing task's status; nothing is launched then).  The task array is
 * read on the host during the call and need not outlive it.  Tasks must not
 * write overlapping outputs. */
typedef struct {
  const int8_t* Xq;              /* [M][K] activation codes */
  const float* x_scales;         /* [M] */
  const spl_matrix* Wq;          /* tile layout, int8 */
  const float* w_scales;         /* [N] */
  void* Y;                       /* out [M][N] fp16 */
  int32_t* acc_out;              /* optional out [M][N] int32 sums, or NULL */
} spl_int8_task;

typedef struct {
  const int8_t* Xq;              /* [M][K] activation codes */
  const float* x_scales;         /* [M] */
  const int8_t* Wq;              /* dense [N][K] codes */
  const float* w_scales;         /* [N] */
  int64_t N;
  int64_t K;
  void* Y;                       /* out [M][N] fp16 */
  int32_t* acc_out;              /* optional out [M][N] int32 sums, or NULL */
} spl_dense_int8_task;

spl_status spl_sparse_linear_int8_group(const spl_int8_task* tasks, int32_t count, int64_t M, hipStream_t stream);
spl_status spl_dense_linear_int8_group(const spl_dense_int8_task* tasks, int32_t count, int64_t M,
                                       hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPL_H */
