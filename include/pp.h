/*
 * pp.h -- C ABI of the pattern/connectivity-pruned 3x3 convolution library
 * for AMD Instinct MI355X (gfx950).
 *
 * The method is the one of Niu et al., "Towards Real-Time DNN Inference on
 * Mobile Platforms with Model Pruning and Compiler Optimization":
 *   - pattern pruning keeps a fixed subset of the 9 taps of every 3x3 kernel,
 *     chosen from a small pattern library; connectivity pruning removes whole
 *     (out-channel, in-channel) kernels (Sec. 2, structured pruning);
 *   - the pruned weights are stored in a compact format with no zero weights
 *     and no per-weight indices (Sec. 3, "sparse model storage"), with the
 *     filters reordered so that filters of the same or similar patterns sit
 *     together and the weights compacted along the kernel direction (Sec. 3,
 *     "matrix reorder");
 *   - a convolution is fused with its bias and activation (Sec. 3, "DSL
 *     related optimization": conv + BN + activation fused into one layer).
 *
 * Conventions for every call:
 *   - All calls return pp_status; 0 is success, negative values are errors.
 *     No call aborts, throws or prints.  pp_last_error() gives a detail
 *     string for the calling thread's most recent error.
 *   - The caller owns every buffer.  The library allocates no device memory
 *     and keeps no global state beyond its loaded GPU code.
 *   - Device work is enqueued asynchronously on the caller's HIP stream
 *     (hipStream_t passed as void*, NULL = default stream).  Nothing
 *     synchronises; a device fault surfaces at the caller's next sync.
 *   - Every argument is validated on the host before any device work is
 *     enqueued.  A call that returns an error has enqueued nothing.
 *   - Activations are NCHW, contiguous, fp32 or bf16 (pp_dtype).
 */
#ifndef PP_H_
#define PP_H_

#ifndef __HIPCC_RTC__   /* the run-time compiler provides these itself */
#include <stddef.h>
#include <stdint.h>
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PP_OK = 0,
  PP_EINVAL = -1,        /* bad argument: NULL pointer, out-of-range value     */
  PP_ESIZE = -2,         /* a buffer is smaller than required                  */
  PP_EBLOB = -3,         /* packed blob is malformed or inconsistent           */
  PP_EUNSUPPORTED = -4,  /* valid request the GPU kernels do not implement     */
  PP_EHIP = -5           /* the HIP runtime reported an error at launch        */
} pp_status;

typedef enum { PP_F32 = 0, PP_BF16 = 1 } pp_dtype;

/* flags of pp_conv2d_fwd / pp_net_op.  The others than PP_RELU are for
 * pp_conv2d_fwd only and fuse the op before or after the conv into its
 * loads or its store (graph-level fusion, Sec. 3): PP_UPSAMPLE2 convolves
 * the nearest x2 upsampling of x; PP_MAXPOOL2 stores the 2 x 2, stride 2 max
 * pool of the activated output instead of the output itself; PP_ACCUMULATE
 * adds the activated output to what y holds (a residual connection);
 * PP_PIXSHUF2 stores the activated output through PixelShuffle(2).
 * PP_PREPARED (pp_conv2d_fwd only): the workspace starts with this
 * layer's prepared weights, written by pp_conv2d_prepare, which are read
 * and not rewritten (see there); bytes past them, from the next 256-byte
 * boundary, serve as the workspace a call without the flag would get. */
enum { PP_RELU = 1u, PP_MAXPOOL2 = 2u, PP_ACCUMULATE = 4u, PP_PIXSHUF2 = 8u, PP_UPSAMPLE2 = 16u,
       PP_PREPARED = 32u };

/* Shape and storage of one pruned 3x3 layer. */
typedef struct {
  int32_t c_out;     /* output channels (filters), 1..65535                 */
  int32_t c_in;      /* input channels, 1..65535                            */
  int32_t stride;    /* 1..16 (the GPU kernels run 1 and 2)                 */
  int32_t pad;       /* zero padding on every side, 0..16                   */
  int32_t dilation;  /* 1..16 (the GPU kernels run 1 and 2)                 */
  int32_t wdtype;    /* pp_dtype of the stored weights                      */
} pp_layer_desc;

/*
 * pp_pack -- pattern projection + compact storage + filter reorder (Sec. 2
 * structured pruning; Sec. 3 "sparse model storage" and "matrix reorder").
 * Host-only, pure and deterministic: equal inputs give equal bytes.
 *
 *   d           layer description (c_out, c_in, stride, pad, dilation, wdtype)
 *   w           host fp32 [c_out][c_in][3][3] dense weights.  Taps outside a
 *               kernel's pattern and kernels with conn = 0 are dropped, even
 *               when nonzero; zero weights inside a kept pattern are stored.
 *   bias        host fp32 [c_out], or NULL for zeros
 *   pattern_id  host u8 [c_out][c_in]: index into lib_masks; read only where
 *               conn = 1
 *   conn        host u8 [c_out][c_in]: 1 = kernel kept, 0 = pruned (other
 *               values are an error)
 *   lib_masks   host u16 [n_patterns]: 9-bit tap masks, bit t = tap
 *               (ky, kx) with t = 3*ky + kx; each must be in 1..511
 *   n_patterns  1..255
 *   out         host buffer for the blob, or NULL to query the size
 *   inout_bytes in: capacity of out; out: bytes required / written
 *
 * Errors: PP_EINVAL (NULL pointer other than bias/out, ranges, conn not 0/1,
 * pattern id >= n_patterns where conn = 1, bad mask, more than 2^24 - 1
 * stored weights), PP_ESIZE (capacity too small; *inout_bytes then holds the
 * required size).
 *
 * Blob layout "PPK1" (little-endian, each section 64-byte aligned, padding
 * zero):
 *   header  u32[24]: magic 0x314B5050, version (2) | wdtype<<16, c_out, c_in,
 *           stride, pad, dilation, n_patterns, group (=8), n_groups,
 *           n_kept, n_wt, off_masks, off_perm, off_codes, off_woff, off_w,
 *           off_bias, total_bytes, 0 x 5
 *   masks   u16[n_patterns]
 *   perm    u32[n_groups*8]: packed slot -> original filter, 0xFFFFFFFF for
 *           padding slots; n_groups = ceil(c_out/8)
 *   codes   u8[n_groups][c_in][8]: pattern id of kernel (perm[8g+s], c) or
 *           0xFF when pruned
 *   woff    u32[n_groups*c_in + 1]: entry (g, c) holds in bits 0..23 the
 *           index in w of its first weight and in bits 24..31 the mask of its
 *           kept slots (bit s set = slot s kept); the last entry is n_wt
 *   w       fp32 or bf16 [n_wt]: for g, c, slot ascending, kept kernels only,
 *           the pattern's taps in ascending tap order (bf16: each kernel
 *           padded to an even element count with a zero)
 *   bias    fp32[n_groups*8] in packed slot order
 * Filter order: kept-kernel count descending, then pattern histogram
 * (count of pattern 0, 1, ... each descending), then filter index.
 */
pp_status pp_pack(const pp_layer_desc* d, const float* w, const float* bias,
                  const uint8_t* pattern_id, const uint8_t* conn,
                  const uint16_t* lib_masks, int32_t n_patterns,
                  void* out, size_t* inout_bytes);

/*
 * Pruning-structure helpers (host-only, pure, deterministic).  ADMM-based
 * structured pruning (Sec. 2) alternates training with a Euclidean
 * projection of each layer's weights onto its structure set; these are those
 * projections, for the structures the paper names, plus the conv + batch
 * norm fusion of its graph rewrite (Sec. 3).  Sums of squares are taken in
 * double, in ascending tap (filter) order.  w is fp32 [c_out][c_in][3][3];
 * channel counts 1..65535.  Errors: PP_EINVAL (NULL pointer, sizes, bad mask,
 * n_keep out of range, negative or NaN energy).
 *
 * pp_project_patterns -- pattern pruning: pattern_id[o][c] (u8) = the library
 *   pattern with the largest sum of w[o][c][t]^2 over its taps t (ties: the
 *   lowest index), i.e. the nearest kernel that keeps one pattern's taps;
 *   kept_energy (double [c_out][c_in], may be NULL) receives that sum.
 * pp_project_connectivity -- connectivity pruning: conn[o][c] = 1 for the
 *   n_keep kernels of largest energy[o][c] (e.g. kept_energy above; ties:
 *   the lower o * c_in + c), else 0.
 * pp_project_columns -- column pruning (one (input channel, tap) position of
 *   every filter): keep the n_keep columns with the largest sum over filters
 *   of w^2 (ties: the lower 9 c + t); col_mask[c] (u16) = 9-bit mask of
 *   channel c's kept taps.
 * pp_column_library -- a column-pruned layer in pp_pack's terms: lib_masks
 *   (capacity 255) = the distinct nonzero channel masks ascending, its count
 *   in *n_patterns, pattern_id / conn (u8 [c_out][c_in]) = channel c's mask
 *   and (mask != 0) for every filter.  PP_EUNSUPPORTED: more than 255
 *   distinct masks.
 * pp_fold_bn -- fold an inference-mode batch norm that follows a conv into
 *   it, in place: s = gamma / sqrt(var + eps) per output channel, w[o][*] *=
 *   s, bias[o] = s (bias[o] - mean[o]) + beta (double, one rounding to fp32);
 *   w is [c_out][k_elems], bias [c_out] (zeros for a conv without one).
 *   PP_EINVAL also when var + eps <= 0.
 */
pp_status pp_project_patterns(const float* w, int32_t c_out, int32_t c_in, const uint16_t* lib_masks,
                              int32_t n_patterns, uint8_t* pattern_id, double* kept_energy);
pp_status pp_project_connectivity(const double* energy, int32_t c_out, int32_t c_in, int64_t n_keep,
                                  uint8_t* conn);
pp_status pp_project_columns(const float* w, int32_t c_out, int32_t c_in, int64_t n_keep, uint16_t* col_mask);
pp_status pp_column_library(const uint16_t* col_mask, int32_t c_out, int32_t c_in, uint16_t* lib_masks,
                            int32_t* n_patterns, uint8_t* pattern_id, uint8_t* conn);
pp_status pp_fold_bn(float* w, float* bias, int32_t c_out, int32_t k_elems, const float* gamma,
                     const float* beta, const float* mean, const float* var, float eps);

/*
 * pp_blob_info -- validate a host copy of a blob (the compact stored model
 * of Sec. 3, "Sparse model storage": kept weights only, filters in their
 * reordered sequence of "Matrix reorder", per-kernel pattern codes in place
 * of per-weight indices) and return its description.
 *   h_blob, bytes  host blob as written by pp_pack; read only
 *   d              out: shape and storage of the layer
 *   n_kept         out: kernels kept by connectivity pruning (Sec. 2)
 *   n_wt           out: stored weights (the kept kernels' pattern taps summed)
 * Any output pointer may be NULL.  Errors: PP_EINVAL (blob NULL), PP_EBLOB
 * (bad magic/version, sizes or offsets inconsistent with `bytes`, woff not
 * monotone, a code >= n_patterns, a perm entry out of range).
 */
pp_status pp_blob_info(const void* h_blob, size_t bytes, pp_layer_desc* d,
                       int32_t* n_kept, int64_t* n_wt);

/*
 * pp_conv2d_fwd -- y = act(conv3x3_pruned(x) + bias) for one packed layer:
 * the 3x3 convolution whose kernels keep only the taps of their pattern
 * and whose connectivity-pruned kernels are absent (Sec. 2, "Structured
 * Model Pruning"), run from the compact reordered storage (Sec. 3, "Sparse
 * model storage", "Matrix reorder") with the bias and activation fused
 * into the same launch (Sec. 3, "DSL related optimization").
 *   h_blob, blob_bytes  host copy of the blob (its header is read here, so no
 *                       device-to-host copy is needed)
 *   d_blob              the same bytes in device memory, 256-byte aligned
 *   x                   device [n][c_in][h][w] in act_dtype
 *   y                   device [n][c_out][h_out][w_out] in act_dtype,
 *                       h_out = (h + 2 pad - 2 dilation - 1)/stride + 1;
 *                       with PP_MAXPOOL2 [n][c_out][h_out/2][w_out/2]
 *                       (floor); must not overlap x
 *   flags               PP_RELU, PP_MAXPOOL2 (y = maxpool2x2(act(conv +
 *                       bias)): the max of the same activated values the
 *                       unpooled call would store when both run the same
 *                       tiling (within the fp32 accumulation tolerance
 *                       otherwise); needs h_out, w_out >= 2 and a tiling
 *                       that holds whole 2 x 2 windows per lane: the
 *                       canonical or all-ones library with pad = dilation,
 *                       else PP_EUNSUPPORTED; with a channel split the
 *                       second pass takes the pool),
 *                       PP_ACCUMULATE (y holds a residual r on entry and
 *                       becomes r + act(conv + bias), element by element, the
 *                       activated value rounded to act_dtype before the add:
 *                       bitwise what a separate add of the stored output
 *                       gives; canonical or all-ones library with pad =
 *                       dilation, else PP_EUNSUPPORTED), PP_PIXSHUF2 (y is
 *                       [n][c_out/4][2 h_out][2 w_out], y[c][2i+a][2j+b] =
 *                       act(conv + bias)[4c+2a+b][i][j]; c_out a multiple of
 *                       4, else PP_EINVAL; same libraries as PP_ACCUMULATE);
 *                       at most one of PP_MAXPOOL2, PP_ACCUMULATE and
 *                       PP_PIXSHUF2, else PP_EINVAL; PP_UPSAMPLE2 (the conv
 *                       reads x [n][c_in][h][w] as its nearest x2 upsampling
 *                       [n][c_in][2h][2w]: h_out, w_out are those of a 2h x 2w
 *                       input; same libraries as PP_ACCUMULATE; combines with
 *                       the others)
 *   workspace, ws_bytes optional device scratch (NULL, 0 for none), 256-byte
 *                       aligned.  With pp_conv2d_workspace() bytes the
 *                       kernel may split the input channels over more
 *                       workgroups (grids that underfill the GPU); partial
 *                       sums go there and a second kernel adds them.  A
 *                       bf16 layer may instead run on the matrix cores
 *                       (pp_conv2d_recipe id 64): its weights are expanded
 *                       to a dense matrix there first.  Calls sharing one
 *                       workspace must be ordered (same stream).
 * Output channels are in the original filter order.  Accumulation is fp32
 * in a fixed order, so repeated calls with the same workspace size give
 * bitwise-identical results.
 * Errors: PP_EINVAL, PP_EBLOB, PP_EUNSUPPORTED (stride or dilation outside
 * {1,2}, pad > 2*dilation, weight dtype not the activation dtype, h_out or
 * w_out < 1), PP_EHIP.
 */
pp_status pp_conv2d_fwd(const void* h_blob, size_t blob_bytes, const void* d_blob,
                        const void* x, void* y, int32_t n, int32_t h, int32_t w,
                        int32_t act_dtype, uint32_t flags, void* workspace, size_t ws_bytes,
                        void* hip_stream);

/*
 * pp_conv2d_fwd_noalloc -- pp_conv2d_fwd for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation): the same plan and result as pp_conv2d_fwd with a
 * pp_conv2d_workspace()-sized workspace, the scratch taken from a 16 MiB
 * array in device memory that the library holds on each device it runs on
 * until the process ends.  The call allocates nothing.  Every call on one
 * GPU shares that GPU's array: calls that overlap on one GPU (different
 * streams, host threads) race, so order them on one stream.  Arguments as
 * pp_conv2d_fwd without the workspace.  Errors: as pp_conv2d_fwd, PP_ESIZE
 * (the layer needs more than 16 MiB of scratch), PP_EHIP (the array's device
 * address could not be found).
 */
pp_status pp_conv2d_fwd_noalloc(const void* h_blob, size_t blob_bytes, const void* d_blob,
                                const void* x, void* y, int32_t n, int32_t h, int32_t w,
                                int32_t act_dtype, uint32_t flags, void* hip_stream);

/*
 * pp_conv2d_prepare -- write, once, a layer's weights in the form its
 * kernels read them, which pp_conv2d_fwd otherwise re-derives from the blob
 * on every call, in up to two parts.  The matrix-core part (bf16 layers
 * with c_in a multiple of 32): the layer as the masked dense contraction of
 * Sec. 2's pruning structure, bf16 [c_out][9][c_in] in original filter
 * order, zeros for taps off a kernel's pattern and for pruned kernels, then
 * the fp32 bias.  The lean part (layers of the canonical library with pad =
 * dilation: stride and dilation 1 (fp32 or bf16), or stride 1 and dilation
 * 2, or stride 2 and dilation 1 (fp32)), from the next 256-byte boundary after
 * the matrix-core part (at the start when there is none): each (slot group,
 * input channel)'s 8 slots x 4 taps of the compact storage (Sec. 3)
 * expanded, zeros for pruned slots, fp32 [ceil(c_out/8)][c_in][32] (bf16
 * weights widened, exact), which the lean kernel reads by scalar loads
 * instead of staging them through LDS.  The
 * weights never change, so a caller that keeps the buffer passes it as the
 * workspace of later calls with PP_PREPARED (or as pp_net_op.d_w of the
 * layer in pp_net_fwd), and the per-call expansion is skipped.  A call whose
 * plan does not read them ignores the buffer and runs without a workspace
 * (pp_conv2d_fwd; pp_net_fwd keeps its own scratch for splits).
 *   h_blob, blob_bytes, d_blob  as pp_conv2d_fwd
 *   prepared     device buffer, 256-byte aligned, or NULL to query the size
 *   inout_bytes  in: capacity of prepared; out: bytes required
 *   hip_stream   stream the expansion is enqueued on (NULL: default)
 * Errors: PP_EBLOB, PP_EINVAL (NULL pointers, misaligned buffers),
 * PP_EUNSUPPORTED (a layer with neither part: bf16 with c_in not a multiple
 * of 32 or too large for the matrix-core form and another library, stride,
 * dilation or pad than the lean part's; fp32 with another library, pad not
 * equal to the dilation, or both stride and dilation 2 or either above 2),
 * PP_ESIZE (capacity too small; *inout_bytes then holds
 * the required size), PP_EHIP.
 */
pp_status pp_conv2d_prepare(const void* h_blob, size_t blob_bytes, const void* d_blob, void* prepared,
                            size_t* inout_bytes, void* hip_stream);

/*
 * pp_conv2d_workspace -- device scratch bytes pp_conv2d_fwd can use for this
 * layer and input (0: it would not use any); h, w are the conv's input size
 * (for a PP_UPSAMPLE2 call the upsampled size 2h x 2w; a call with fused
 * flags needs no more than the plain call).  Host-only.  Errors: as
 * pp_conv2d_out_size, PP_EINVAL (bytes NULL, act_dtype), PP_EUNSUPPORTED.
 */
pp_status pp_conv2d_workspace(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h,
                              int32_t w, int32_t act_dtype, size_t* bytes);

/*
 * pp_conv2d_recipe -- the GPU tiling ("recipe" id) and the channel split
 * pp_conv2d_fwd uses for this layer, batch and input size, with
 * (with_workspace != 0) or without a pp_conv2d_workspace()-sized workspace.
 * Informational: lets callers and tests see which compiled kernel runs: ids
 * below 40 are vector-ALU tilings, 64 the bf16 matrix-core form (the layer as
 * a zero-filled dense contraction on the matrix cores; needs the workspace,
 * c_in a multiple of 32 and no fused max pool).  The environment variables
 * PP_RECIPE=<id> and PP_KSPLIT=<k> force a tiling (when it can run the layer)
 * and a split; otherwise the planner's choice is reported.  ksplit may be NULL.  Host-only.  Errors: as pp_conv2d_out_size,
 * PP_EINVAL (recipe NULL, act_dtype), PP_EUNSUPPORTED.
 */
pp_status pp_conv2d_recipe(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h, int32_t w,
                           int32_t act_dtype, int32_t with_workspace, int32_t* recipe,
                           int32_t* ksplit);

/*
 * pp_jit_library -- compile (on the host, with the device compiler at run
 * time: seconds) the wave-pipeline kernels specialised for this layer's own
 * pattern library, for the plans pp_conv2d_fwd makes for this input (n, h,
 * w, act_dtype; with a pp_conv2d_workspace()-sized workspace when
 * with_workspace != 0, and without), and load them on the current device.
 * From then on pp_conv2d_fwd and pp_net_fwd (unfused convs) run such a
 * layer with them, as fast as the canonical library, instead of the generic
 * kernel that tests taps against run-time masks (the per-layer code
 * generation of the paper's compiler, Sec. 3); pp_conv2d_recipe reports
 * their tiling.  For libraries of up to 8 patterns of exactly 4 taps other
 * than the canonical one, with pad = dilation.  Idempotent and thread-safe;
 * the kernels stay loaded until the process ends.  Errors: as
 * pp_conv2d_out_size, PP_EUNSUPPORTED (library or layer not of that form),
 * PP_EHIP (compilation or loading failed; pp_last_error starts the log).
 */
pp_status pp_jit_library(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h, int32_t w,
                         int32_t act_dtype, int32_t with_workspace);

/* pp_conv2d_out_size -- h_out, w_out of a packed layer for an h x w input. */
pp_status pp_conv2d_out_size(const void* h_blob, size_t blob_bytes, int32_t h, int32_t w,
                             int32_t* h_out, int32_t* w_out);

/* ------------------------------------------------------------------------
 * Network execution: an ordered op list over activation slots, the flat
 * layer-wise representation of a model (Sec. 3, "DSL related optimization":
 * each layer one entry, conv fused with its activation).
 * Slot 0 is the network input x, slot 1 the output y, slots 2..15 live in
 * the caller's workspace.
 * ---------------------------------------------------------------------- */
typedef enum {
  PP_OP_CONV_PP = 0,     /* pruned 3x3 conv: h_blob/blob_bytes/d_blob          */
  PP_OP_CONV_DENSE = 1,  /* dense k x k conv, stride 1: k, pad, c_in, c_out,   */
                         /* d_w [c_out][c_in][k][k], d_b fp32 [c_out]          */
  PP_OP_DECONV = 2,      /* transposed conv: k, stride, pad, c_in, c_out,      */
                         /* d_w [c_in][c_out][k][k], d_b fp32 [c_out]          */
  PP_OP_MAXPOOL2 = 3,    /* 2x2 max pool, stride 2 (floor)                     */
  PP_OP_UPSAMPLE2 = 4,   /* nearest-neighbour x2                               */
  PP_OP_PIXSHUF2 = 5,    /* PixelShuffle(2): out[c,2h+i,2w+j] = in[4c+2i+j,h,w] */
  PP_OP_ADD = 6          /* dst = src + src2 (same shape)                      */
} pp_op_kind;

#define PP_MAX_SLOTS 16

typedef struct {
  int32_t kind;              /* pp_op_kind                                      */
  int32_t src, src2, dst;    /* slots; dst must differ from src and src2        */
  uint32_t flags;            /* PP_RELU (conv / deconv ops)                     */
  int32_t k, stride, pad, dilation, c_in, c_out;   /* dense conv / deconv       */
  const void* h_blob;        /* PP_OP_CONV_PP: host blob                        */
  size_t blob_bytes;
  const void* d_blob;        /* PP_OP_CONV_PP: device blob                      */
  const void* d_w;           /* dense ops: device weights in the act dtype;     */
                             /* PP_OP_CONV_PP: NULL, or the layer's prepared    */
                             /* weights (pp_conv2d_prepare), read when the net  */
                             /* runs the layer in the form they are for         */
  const float* d_b;          /* dense ops: device fp32 bias, or NULL            */
} pp_net_op;

/*
 * pp_net_workspace -- bytes of workspace pp_net_fwd needs for this op list
 * and input shape (intermediate activations, plus scratch for the pruned
 * convs' channel splits), and the output shape (any output pointer may be
 * NULL).
 * Errors: PP_EINVAL (bad op, slot or shape chain), PP_EBLOB.
 */
pp_status pp_net_workspace(const pp_net_op* ops, int32_t n_ops, int32_t n, int32_t c,
                           int32_t h, int32_t w, int32_t act_dtype, size_t* bytes,
                           int32_t* out_c, int32_t* out_h, int32_t* out_w);

/*
 * pp_net_fwd -- run the op list on the stream, one launch per op, no host
 * synchronisation.  x is device [n][c][h][w]; y receives slot 1 (shape from
 * pp_net_workspace).  A pruned conv (canonical or all-ones library, pad =
 * dilation) whose output slot only feeds the next op -- a max pool, a pixel
 * shuffle, or an add whose other operand is dead afterwards too -- runs
 * fused with that op in one launch (pp_conv2d_fwd's PP_MAXPOOL2,
 * PP_PIXSHUF2, PP_ACCUMULATE); the result is the same.  The workspace is
 * only valid for the op list and shape it was sized for.  With the
 * environment variable PP_TRACE set (and not "0") when the library first
 * runs a net, each op's (or fused pair's) launches sit in a named roctx
 * range, "pp op <index> <kind>", for rocprofv3 --marker-trace; the roctx
 * library is loaded at run time, and without it there are no ranges.
 * Errors: as pp_net_workspace, PP_ESIZE (ws_bytes too small),
 * PP_EUNSUPPORTED, PP_EHIP.
 */
pp_status pp_net_fwd(const pp_net_op* ops, int32_t n_ops, const void* x, void* y,
                     int32_t n, int32_t c, int32_t h, int32_t w, int32_t act_dtype,
                     void* workspace, size_t ws_bytes, void* hip_stream);

/*
 * pp_net_plan -- how pp_net_fwd runs this op list for this input shape: the
 * graph-level fusion it applies (Sec. 3, "DSL related optimization": a conv
 * and the cheap op next to it become one launch) and the tiling of each
 * pruned conv.  Host-only; reads the host blobs and the op fields, never a
 * device pointer (those may be NULL here).
 *   op_flags  host u32 [n_ops], written: for a pruned conv, the fusion flags
 *             its launch carries (PP_UPSAMPLE2: it takes the upsample before
 *             it; PP_MAXPOOL2, PP_PIXSHUF2 or PP_ACCUMULATE: it takes the
 *             max pool, pixel shuffle or add after it); PP_NET_TAKEN for an
 *             op so taken (it has no launch of its own); 0 otherwise
 *   recipe    host i32 [n_ops], or NULL: the pp_conv2d_recipe id of each
 *             pruned conv's launch (with the workspace pp_net_workspace
 *             sizes), -1 for the other ops
 * Errors: as pp_net_workspace (without the device-pointer checks),
 * PP_EINVAL (op_flags NULL).
 */
#define PP_NET_TAKEN 0x80000000u
pp_status pp_net_plan(const pp_net_op* ops, int32_t n_ops, int32_t n, int32_t c, int32_t h,
                      int32_t w, int32_t act_dtype, uint32_t* op_flags, int32_t* recipe);

/*
 * pp_round_bf16 -- fp32 -> bf16 bit patterns, round to nearest, ties to
 * even (the rounding pp_pack applies to bf16 pruned weights), for the dense
 * layers' weights of a bf16 network (pp_net_op.d_w).  NaN stays NaN.
 * Host-only: src host fp32 [count], dst host u16 [count]; they must not
 * overlap.  Errors: PP_EINVAL (NULL pointer with count > 0).
 */
pp_status pp_round_bf16(const float* src, uint16_t* dst, size_t count);

const char* pp_status_str(pp_status s);
const char* pp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* PP_H_ */
