/*
 * convbwd — convolution backward pass with ReLU-derived sparsity on AMD
 * Instinct MI355X (gfx950).
 *
 * The operations are those of "Exploiting Activation based Gradient Output
 * Sparsity to Accelerate Backpropagation in CNNs" (arXiv 2109.07710):
 *
 *   - the data gradient dX = conv_transpose(dY, W), computed only where the
 *     forward ReLU footprint of X is live (output sparsity, Sec. III-B: the
 *     ReLU derivative multiplies the gradient by 1 or 0, so the outputs it
 *     will zero are known from the forward pass) and written as exact +0.0
 *     everywhere else;
 *   - the weight gradient dW = X (star) dY, skipping blocks of dY that are
 *     entirely zero (input sparsity of the incoming gradient, Sec. III-B and
 *     the weight-gradient phase of Sec. IV-B);
 *   - a dense data gradient on the same kernel (the paper's dense-compute
 *     baseline "DC", Sec. VI).
 *
 * Layer notation follows Sec. II-A / Sec. IV-B: an input [C,H,W] is mapped
 * by filters [M,C,R,S] to an output [M,U,V]; here M is K and [U,V] is [P,Q],
 * with P = (H + 2*pad_h - R)/stride_h + 1 (floor), likewise Q.  Convolution is
 * cross-correlation with zero padding:
 *
 *   Y[n,k,p,q]  = sum_{c,r,s} X[n,c,p*sh-ph+r, q*sw-pw+s] W[k,c,r,s]
 *   dX[n,c,h,w] = mask[n,c,h,w] ? sum_{k,r,s : aligned, in range} dY[n,k,p,q] W[k,c,r,s] : +0.0
 *   dW[k,c,r,s] = sum_{n,p,q} dY[n,k,p,q] X[n,c,p*sh-ph+r, q*sw-pw+s]
 *
 * where mask = (X > 0), X being this layer's input, i.e. the output of the
 * preceding ReLU.
 *
 * Conventions for every entry point:
 *   - Tensor, mask and workspace pointers are DEVICE memory owned by the
 *     caller and must stay valid until the work queued on `stream` finishes.
 *     The library never allocates device memory and keeps no per-call state.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All work is queued on it; no entry point synchronizes the device, except
 *     cbw_read_stats, which waits for `stream`.
 *   - Every argument is validated before anything is launched.  On an error
 *     nothing is launched and no output is touched.  No exception or abort
 *     crosses this interface.
 *   - Calls that share a workspace or an output and overlap in time race.
 */
#ifndef CONVBWD_H
#define CONVBWD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CBW_OK = 0,
    CBW_ERR_INVALID_ARG = -1,  /* null pointer, non-positive size, inconsistent P/Q */
    CBW_ERR_UNSUPPORTED = -2,  /* valid but not implemented: layout, channel counts
                                  not a multiple of the 16-byte vector, misaligned
                                  pointer, tensor of 2^31 elements or more */
    CBW_ERR_WORKSPACE = -3,    /* workspace missing or smaller than cbw_workspace_size */
    CBW_ERR_HIP = -4           /* a HIP launch or copy failed (sticky error cleared) */
} cbw_status;

/* Activation layout of X, dX, Y, dY.  Channel-innermost (NHWC) is the native
 * one: the paper stores neurons "channel first" and indexes non-zeros through
 * the channel dimension 32 at a time (Sec. IV-B).  NCHW is accepted by
 * conv_bwd_data, conv_bwd_data_masked, conv_bwd_weight_sparse and
 * conv_bwd_weight_sparse_x: the library transposes the activations (and
 * reorders footprint bits) into NHWC copies in the workspace, runs the NHWC
 * path there and transposes dX back, so an NCHW call adds HBM-bound copies
 * and a larger workspace.  The forward and the per-element data gradient
 * return CBW_ERR_UNSUPPORTED for NCHW.  Footprint bitmaps are always in the
 * caller's layout (bit i = element i of the tensor as the caller stores it). */
typedef enum { CBW_NCHW = 0, CBW_NHWC = 1 } cbw_act_layout;
/* Filter layout of W and dW. */
typedef enum { CBW_KCRS = 0, CBW_KRSC = 1 } cbw_w_layout;
/* Element type of X, W, dY and dX.  dW is always float32. */
typedef enum { CBW_F32 = 0, CBW_BF16 = 1 } cbw_dtype;

typedef struct {
    int32_t N, C, H, W;      /* batch, input channels, input height, width     */
    int32_t K, R, S;         /* output channels (the paper's M), filter size   */
    int32_t P, Q;            /* output height, width; must equal the formula   */
    int32_t stride_h, stride_w, pad_h, pad_w;
    int32_t act_layout;      /* cbw_act_layout; NCHW for the backward calls    */
    int32_t w_layout;        /* cbw_w_layout; both implemented                 */
    int32_t dtype;           /* cbw_dtype                                      */
} cbw_conv_desc;

/* Operation selector for cbw_workspace_size / cbw_read_stats. */
enum { CBW_OP_BWD_DATA = 0, CBW_OP_BWD_DATA_MASKED = 1, CBW_OP_BWD_WEIGHT = 2, CBW_OP_FWD = 3,
       CBW_OP_BWD_DATA_ELEMENTWISE = 4, CBW_OP_BWD_BOTH = 5 };

/* Flags. CBW_FLAG_NO_SKIP runs the same kernels with every skip disabled:
 * the masked data gradient computes all rows and applies the mask in its
 * epilogue; the weight gradient processes every dY block. */
#define CBW_FLAG_NO_SKIP 1u
/* conv_bwd_sparse only: with x_mask given, the weight gradient also skips
 * blocks whose X operand is entirely zero (as conv_bwd_weight_sparse_x). */
#define CBW_FLAG_SKIP_X_BLOCKS 2u

/* Execution statistics written by the kernels into the workspace. */
typedef struct {
    int64_t rows_total;      /* GEMM rows (pixel x channel-group) the dense path would compute */
    int64_t rows_live;       /* rows actually computed                                        */
    int64_t blocks_total;    /* dW GEMM blocks: pixel chunk x k tile x tap group x channel tile */
    int64_t blocks_skipped;  /* dW blocks skipped (dY, or with the _x variant X, all zero)     */
} cbw_stats;

/* Host-only inspection of the data-gradient tiling that conv_bwd_data and
 * the CBW_FLAG_NO_SKIP masked call use for this descriptor (tests and tools):
 * *channels output channels per tile, *capacity pixel rows a tile can hold,
 * and *rows pixel rows each tile covers -- the capacity, or 16 or 32 rows
 * less, whichever lets the busiest CU finish its tiles first given one
 * resident tile per CU (tiles / CUs rounded up, times the rows); the full
 * capacity whenever the tiles are few enough for the reduction to be split.
 * The skipping masked call makes the same choice on the device from the live
 * pixel counts.  Any output pointer may be NULL.  Returns CBW_OK or the
 * descriptor's validation status. */
int cbw_data_tiling(const cbw_conv_desc* desc, int32_t* channels, int32_t* capacity, int32_t* rows);

/* Human-readable name of a cbw_status value (static storage). */
const char* cbw_status_string(int status);

/* Host-only check of a descriptor (no GPU needed).  Returns CBW_OK,
 * CBW_ERR_INVALID_ARG or CBW_ERR_UNSUPPORTED. */
int cbw_validate_desc(const cbw_conv_desc* desc);

/* Number of 32-bit words of the packed X footprint, ceil(N*C*H*W/32), and of
 * a packed dY footprint, ceil(N*K*P*Q/32).  0 for an invalid descriptor. */
size_t cbw_mask_words(const cbw_conv_desc* desc);
size_t cbw_dy_mask_words(const cbw_conv_desc* desc);

/* Workspace bytes needed by `op` for this descriptor (host only; depends on
 * the descriptor alone).  Returns a cbw_status; *bytes is set on success. */
int cbw_workspace_size(const cbw_conv_desc* desc, int op, size_t* bytes);

/* ReLU footprint bitmap of X (Sec. III-B boxed derivative, read as the ReLU
 * output footprint: live iff X > 0; Sec. IV-B: the output bitmap the forward
 * pass leaves in memory for the backward pass).  Bit i of word i/32 (LSB
 * first) is element i of X in X's own linear order; trailing bits of
 * the last word are 0.  x_mask: cbw_mask_words(desc) words. */
int cbw_relu_mask_pack(const cbw_conv_desc* desc, const void* X, uint32_t* x_mask, void* stream);

/* Non-zero bitmap of any tensor of `count` elements of type `dtype` (bit =
 * value != 0; +0.0 and -0.0 are zero), same bit order.  Used for the dY
 * footprint that lets the weight gradient skip all-zero blocks. */
int cbw_nonzero_mask_pack(int32_t dtype, int64_t count, const void* t, uint32_t* bits, void* stream);

/* Dense data gradient (Sec. IV-B, the backward pass as the forward operation
 * with M and C interchanged): dX[N,H,W,C] from dY[N,P,Q,K] and W (KRSC or
 * KCRS); dX[N,C,H,W] from dY[N,K,P,Q] for NCHW.
 * Workspace: cbw_workspace_size(desc, CBW_OP_BWD_DATA). */
int conv_bwd_data(const cbw_conv_desc* desc, const void* dY, const void* W, void* dX,
                  void* workspace, size_t workspace_bytes, void* stream);

/* Masked data gradient (output sparsity, Sec. III-B; output-bitmap-driven
 * address generation, Sec. IV-B): only outputs whose x_mask bit is set are
 * computed; all others are written as +0.0 (bit pattern 0).  x_mask is the
 * packed footprint of X (cbw_relu_mask_pack), 16-byte aligned.  The footprint is compacted per
 * channel group into ascending lists of live pixels and the GEMM runs only
 * over those rows; flags = CBW_FLAG_NO_SKIP computes every row instead.
 * Workspace: cbw_workspace_size(desc, CBW_OP_BWD_DATA_MASKED). */
int conv_bwd_data_masked(const cbw_conv_desc* desc, const void* dY, const void* W,
                         const uint32_t* x_mask, void* dX,
                         void* workspace, size_t workspace_bytes, uint32_t flags, void* stream);

/* conv_bwd_data_masked for callers that cannot allocate device memory (code
 * under stream capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and the same result, with the workspace
 * replaced by a scratch array built into the library (32 MiB, one per GPU,
 * held until the process ends).  Nothing is allocated or freed.  The
 * reduction is never split across workgroups (no partial tiles), so the
 * values equal those of conv_bwd_data_masked whenever that call does not
 * split either (many live tiles), and agree within fp32 summation order
 * otherwise.  Returns CBW_ERR_WORKSPACE when the descriptor needs more
 * scratch than the array holds (roughly: filters K*C*R*S elements plus
 * 4 bytes per pixel and 256-channel group, plus the NCHW copies).  The
 * first call on a device looks up the array's device address.  All calls on
 * one GPU share its array: calls that overlap in time on one GPU (two
 * streams, two threads) race, as two calls sharing a workspace do. */
int conv_bwd_data_masked_noalloc(const cbw_conv_desc* desc, const void* dY, const void* W,
                                 const uint32_t* x_mask, void* dX, uint32_t flags, void* stream);

/* Forward convolution with the ReLU and the footprint of its output fused
 * into one launch (Sec. II-A forward operation; the output bitmap that the
 * backward pass consumes is produced by the forward pass, Sec. IV-B).
 * Y[N,P,Q,K] = relu(conv(X, W)) in desc->dtype: float32 accumulation,
 * round-to-nearest-even to bf16, non-positive (and NaN) sums give +0.0.
 * y_mask (nullable; cbw_dy_mask_words(desc) words, 16-byte aligned) receives
 * the bits (Y > 0) in Y's linear order -- exactly what cbw_relu_mask_pack
 * computes on Y -- which is the next layer's x_mask and, as the ReLU
 * derivative, the footprint of this layer's dY.  X is NHWC, W KRSC or KCRS.
 * Stride 1 only, with pad_h < R and pad_w < S; other shapes return
 * CBW_ERR_UNSUPPORTED.  Y and y_mask are fully overwritten.
 * Workspace: cbw_workspace_size(desc, CBW_OP_FWD). */
int conv_fwd_relu_mask(const cbw_conv_desc* desc, const void* X, const void* W, void* Y, uint32_t* y_mask,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Weight gradient with input sparsity (Sec. III-B; weight-gradient phase of
 * Sec. IV-B): dW (float32, layout desc->w_layout) from X[N,H,W,C] and
 * dY[N,P,Q,K] (NCHW: X[N,C,H,W], dY[N,K,P,Q]).  Blocks of (pixel chunk x output-channel tile) in which dY is
 * entirely zero are skipped; the skipped products are exactly zero.  dy_mask
 * (nullable) is a packed dY footprint (cbw_nonzero_mask_pack or the next
 * layer's ReLU bitmap, any superset of dY's non-zeros; 16-byte aligned);
 * when NULL the occupancy is read from dY itself.  The result is deterministic: partial
 * sums are reduced in a fixed order.  dW is fully overwritten.
 * Workspace: cbw_workspace_size(desc, CBW_OP_BWD_WEIGHT). */
int conv_bwd_weight_sparse(const cbw_conv_desc* desc, const void* X, const void* dY,
                           const uint32_t* dy_mask, float* dW,
                           void* workspace, size_t workspace_bytes, uint32_t flags, void* stream);

/* Weight gradient that also skips blocks whose X operand is entirely zero:
 * activation sparsity used as input sparsity in the weight-gradient phase
 * (Sec. III-A, sources of sparsity; Sec. VI, weight-gradient results).  A
 * (pixel chunk x filter taps x channel tile) block is skipped when dY is zero
 * over the chunk's output channels of the tile (as conv_bwd_weight_sparse
 * does) or when X is zero over the chunk's tap-shifted pixels and the tile's
 * channels; both skips drop only products that are exactly zero (finite
 * inputs).  x_mask (nullable, 16-byte aligned): packed X footprint in X's
 * linear order, cbw_mask_words(desc) words, any superset of X's non-zeros
 * (cbw_nonzero_mask_pack; for a ReLU output X the cbw_relu_mask_pack bitmap);
 * when NULL the X occupancy is read from X itself.  Otherwise as
 * conv_bwd_weight_sparse (same workspace size, deterministic, dW fully
 * overwritten); CBW_FLAG_NO_SKIP disables both skips. */
int conv_bwd_weight_sparse_x(const cbw_conv_desc* desc, const void* X, const void* dY,
                             const uint32_t* x_mask, const uint32_t* dy_mask, float* dW,
                             void* workspace, size_t workspace_bytes, uint32_t flags, void* stream);

/* Both gradients of one layer in one call: the backward-pass phase (data
 * gradient) and the weight-gradient phase of Sec. IV-B, with the results of
 *   - dX: conv_bwd_data_masked(desc, dY, W, x_mask, dX, .., flags & NO_SKIP)
 *     when x_mask is set (output sparsity, Sec. III-B), conv_bwd_data when
 *     x_mask is NULL (dense);
 *   - dW: conv_bwd_weight_sparse(desc, X, dY, dy_mask, dW, .., flags &
 *     NO_SKIP) (input sparsity), or with CBW_FLAG_SKIP_X_BLOCKS and x_mask
 *     set conv_bwd_weight_sparse_x(desc, X, dY, x_mask, dy_mask, ...).
 * Values are those of the separate calls (bitwise, unless a reduction is
 * split differently).  The integer work of both gradients (filter
 * transform, compaction counts, dY block occupancy) shares one launch.
 * With the tiled data gradient the weight GEMM runs next and the data GEMM
 * after it, its tail workgroups summing the weight gradient's split-K
 * partials; a data gradient that may split (the skipping call decides on
 * the device; a dense tiling split by the planner) adds its split
 * reduction: three or four launches.  With the row-window or pointwise data
 * gradient: the data GEMM, the weight GEMM and one reduction launch.
 * NCHW tensors are served by the two separate calls.  Arguments as in the
 * separate calls (X, dY, W, dX, dW and the footprints 16-byte aligned);
 * dX = NULL computes the weight gradient alone (a first layer, whose input
 * needs no gradient; W may then be NULL too); flags: CBW_FLAG_NO_SKIP,
 * CBW_FLAG_SKIP_X_BLOCKS.
 * Workspace: cbw_workspace_size(desc, CBW_OP_BWD_BOTH) bytes; its first
 * cbw_workspace_size(desc, CBW_OP_BWD_DATA_MASKED) bytes are the data
 * gradient's workspace, and the weight gradient's starts at that size
 * rounded up to a multiple of 256 (for cbw_read_live_lists,
 * cbw_read_occupancy and cbw_read_weight_work); cbw_read_stats with
 * CBW_OP_BWD_BOTH reads both. */
int conv_bwd_sparse(const cbw_conv_desc* desc, const void* X, const void* dY, const void* W, const uint32_t* x_mask,
                    const uint32_t* dy_mask, void* dX, float* dW, void* workspace, size_t workspace_bytes,
                    uint32_t flags, void* stream);

/* Data gradient with per-element input and output sparsity on the vector
 * ALUs (Sec. III-B, input and output sparsity; Sec. IV-B, lanes that walk
 * only the non-zero offsets of their gradient column).  Same result as
 * conv_bwd_data_masked up to summation order: dX = x_mask ? sum over the
 * non-zero dY entries only : +0.0.  A pixel whose footprint row is entirely
 * dead costs one zero store; every other pixel sums, per filter tap, only the
 * non-zero entries of its source dY row.  For very sparse inputs, where the
 * matrix-core path cannot skip anything.  Supported: bf16, NHWC, KRSC filters,
 * C in {64, 128, 256, 512}, K < 65536; other descriptors return
 * CBW_ERR_UNSUPPORTED.  Deterministic.  dX is fully overwritten.
 * Workspace: cbw_workspace_size(desc, CBW_OP_BWD_DATA_ELEMENTWISE); after
 * the call it holds, per output pixel, the number of (tap, k) products
 * executed (cbw_read_pixel_counts). */
int conv_bwd_data_elementwise(const cbw_conv_desc* desc, const void* dY, const void* W,
                              const uint32_t* x_mask, void* dX, void* workspace, size_t workspace_bytes,
                              void* stream);

/* After conv_bwd_data_elementwise on `workspace`: copies the per-pixel
 * product counts (N*H*W int32 in pixel order; `counts` may be NULL) and
 * their sum to the host (waits for `stream`). */
int cbw_read_pixel_counts(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes,
                          int32_t* counts, int64_t* total, void* stream);

/* After a weight-gradient call on `workspace` (either entry point): the
 * number of blocks each work item executed, in item order z*ntiles + tile
 * (split z of tile ((tap group * channel tiles + channel tile) * k tiles +
 * k tile)).  With skipping, the live blocks of every tile are shared out in
 * equal ceil(live / nsplit) parts (work redistribution, Sec. IV-F).
 * `work` (nullable) receives nsplit*ntiles int32; waits for `stream`. */
int cbw_read_weight_work(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, int32_t* work,
                         int32_t* nsplit, int32_t* ntiles, void* stream);

/* Copy the statistics of the last `op` call that used `workspace` to the host
 * (waits for `stream`). */
int cbw_read_stats(const cbw_conv_desc* desc, int op, const void* workspace, size_t workspace_bytes,
                   cbw_stats* out, void* stream);

/* Inspection of the integer steps (for tests and tools; waits for `stream`).
 *
 * cbw_read_live_lists: after a conv_bwd_data_masked call without
 * CBW_FLAG_NO_SKIP on `workspace`, copies the compacted footprint of channel
 * group `group` (channels [group*G, min(C, (group+1)*G)), G = the value
 * returned in *group_width) to the host: *count live pixels, in ascending
 * order, into `pixels` (capacity N*H*W entries).  A pixel is listed iff at
 * least one of its channels in the group is live (non-zero indexing of the
 * output bitmap, Sec. IV-B).  `pixels` may be NULL to query count and width.
 *
 * cbw_read_occupancy: after a conv_bwd_weight_sparse call without
 * CBW_FLAG_NO_SKIP, copies the block occupancy map occ[chunk][ktile] (uint8,
 * 1 = dY has a non-zero in that block) to `occ` (capacity *nchunks x
 * *ktiles, both returned; chunk = *chunk_pixels pixels of dY in N,P,Q order,
 * ktile = *ktile_width output channels).  `occ` may be NULL to query sizes. */
int cbw_read_live_lists(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, int group,
                        int32_t* pixels, int32_t* count, int32_t* group_width, void* stream);
int cbw_read_occupancy(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, uint8_t* occ,
                       int32_t* nchunks, int32_t* ktiles, int32_t* chunk_pixels, int32_t* ktile_width,
                       void* stream);

/* Profiling hook (for benchmarks; not needed for computing).  Until changed,
 * every call on this host thread of the given op family records `start`
 * (a hipEvent_t as void*) on the call's stream right before the op's main
 * GEMM kernel is launched and `stop` right after it, so that
 * hipEventElapsedTime(start, stop) is that kernel's duration.  op is
 * CBW_OP_BWD_DATA (covers both data-gradient entry points),
 * CBW_OP_BWD_WEIGHT or CBW_OP_FWD; NULL events switch the hook off. */
int cbw_set_profile_events(int op, void* start, void* stop);

#ifdef __cplusplus
}
#endif
#endif /* CONVBWD_H */
