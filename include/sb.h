/*
 * sb.h -- C ABI of libsb, the MI355X (gfx950) compute library for one
 * SplitBrain worker's share of a training step (arXiv 2112.15317).
 *
 * The paper splits a CNN into two halves (sec. 3.1, Model Parallelism): the
 * convolutional layers, compute-heavy with few parameters, run data-parallel
 * on each worker's local batch; the fully connected layers, which hold most
 * parameters, are split to 1/K of their outputs and run on the batch that
 * the modulo layer gathers from the K workers.  One worker's compute is
 * therefore: 3x3 convolution forward / data gradient / weight gradient, the
 * ReLU and 2x2 max pooling between them (sec. 2.2), and the forward and
 * backward of its FC column shard.  Those are the calls below, together
 * with the data movement of the modulo and shard layers around the FC
 * shards for the case where every worker's buffers sit on one device.
 * Exchanges between devices and model averaging are not part of this
 * library.
 *
 * Conventions for every call
 * --------------------------
 *  * Tensor pointers are DEVICE pointers, owned by the caller, that stay
 *    valid until the enqueued work has finished.  The library never
 *    allocates, frees or synchronises inside these calls; scratch memory is
 *    the caller's workspace (query its size first).
 *  * The workspace holds split-reduction partial sums; its contents need no
 *    initialisation and are dead after the call.  Calls that share one
 *    workspace must not run concurrently (use one workspace per stream).
 *  * `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    All work is enqueued on it, asynchronously.
 *  * Arguments are validated before anything is enqueued; on any error
 *    nothing is launched and the status says why.  A launch failure
 *    returns SB_ERR_HIP.  Faults during execution surface, as in HIP, at
 *    the caller's next synchronisation.
 *  * Outputs must not overlap inputs (checked by address range).
 *  * Layouts: activations NCHW row-major, or channel-blocked NCHW8C
 *    (sb_layout) for the conv and pooling calls; conv weights KCRS
 *    ([out][in][3][3]); FC input X [M][Kin] and shard weights
 *    W_shard [Kin][Ns] row-major.  Element strides are in elements.
 *  * dtype SB_F32: every tensor fp32.  SB_BF16: activations, activation
 *    gradients and conv weights are bfloat16 (round-to-nearest-even on
 *    store); accumulation is fp32; bias, weight gradient and bias gradient
 *    are fp32.
 *  * Calls are thread-safe; the library keeps no state between calls.
 */
#ifndef SB_H
#define SB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SB_OK = 0,
    SB_ERR_INVALID_ARG = 1,   /* null pointer, bad size, overlap, bad flag */
    SB_ERR_UNSUPPORTED = 2,   /* valid request this build does not provide */
    SB_ERR_WORKSPACE = 3,     /* workspace missing or smaller than needed  */
    SB_ERR_HIP = 4            /* a HIP runtime call or launch failed       */
} sb_status;

typedef enum { SB_F32 = 0, SB_BF16 = 1 } sb_dtype;

/* Activation layouts.  SB_NCHW: [n][c][h][w].  SB_NCHW8C (channel-blocked):
 * [n][c/8][h][w][c%8], i.e. element (n, c, h, w) at
 * ((n * C/8 + c/8) * H + h) * W + w) * 8 + c % 8, for channel counts that
 * are multiples of 8; the 8 channels of a pixel are one 16-byte bf16 piece.
 * Filters are KCRS in both. */
typedef enum { SB_NCHW = 0, SB_NCHW8C = 1 } sb_layout;

/* flags */
#define SB_FUSE_RELU 1u       /* apply ReLU to the output (conv fwd, FC fwd) */
#define SB_PACKED_FILTERS 2u  /* conv fwd / data gradient: `w` holds filters
                                 packed by sb_conv3x3_pack_filters */

/* Returns a static string naming the status. */
const char *sb_status_string(sb_status s);

/* Library version as major*10000 + minor*100 + patch. */
int sb_version(void);

/* ------------------------------------------------------------------------
 * 3x3 convolution, stride 1, zero padding 1 (sec. 2.2: each convolutional
 * stage multiplies successive input patches with square filters; the
 * operation is the cross-correlation used by deep-learning frameworks).
 *
 *   x  [n][c][h][w]    input activations (or channel-blocked, see layout)
 *   w  [k][c][3][3]    filters
 *   y  [n][k][h][w]    output (same layout as x)
 * The layout applies to every activation tensor of a call (x, y, dy, dx,
 * the ReLU mask).  SB_NCHW8C is provided for SB_BF16 with c and k multiples
 * of 8 and w >= 8 (the bf16 MFMA kernels); other combinations return
 * SB_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------- */
typedef struct {
    int n, c, h, w;       /* batch, input channels, height, width (all > 0) */
    int k;                /* output channels (> 0)                          */
    int dtype;            /* sb_dtype                                       */
    unsigned flags;       /* SB_FUSE_RELU (forward only), SB_PACKED_FILTERS
                             (forward and data gradient)                    */
    int layout;           /* sb_layout of the activations                   */
} sb_conv3x3_desc;

/* SB_PASS_FWD_POOL: the forward with ReLU + 2x2 max pooling fused
 * (sb_conv3x3_fwd_pool); it takes the forward's workspace and packing. */
enum { SB_PASS_FWD = 0, SB_PASS_BWD_DATA = 1, SB_PASS_BWD_WEIGHT = 2, SB_PASS_FWD_POOL = 3 };

/* Workspace bytes that `pass` needs for `desc` (0 is a valid answer, and a
 * NULL workspace is then accepted).  With SB_PACKED_FILTERS set the answer
 * leaves out the room the call would otherwise use to pack the filters.
 * Returns (size_t)-1 for an invalid or unsupported descriptor. */
size_t sb_conv3x3_workspace_bytes(const sb_conv3x3_desc *desc, int pass);

/* Packed filters.  The forward and data-gradient kernels read the filters
 * rearranged into the order they stage them (slices per output-channel tile
 * and input-channel chunk; for the data gradient the filters transposed and
 * rotated by 180 degrees).  Every such call packs them first, into its
 * workspace.  A caller that runs several calls with the same filters (a
 * training step: forward, then data gradient), or wants the packing off the
 * critical path (on another stream, ahead of the call), packs them once with
 * sb_conv3x3_pack_filters and sets SB_PACKED_FILTERS on the calls, which
 * then take the packed buffer as `w`.
 *
 * sb_conv3x3_packed_bytes: bytes of the packed filters of `pass`
 * (SB_PASS_FWD or SB_PASS_BWD_DATA) for `desc`; 0 for an invalid descriptor
 * or pass.  The flags of desc other than the dtype's are ignored.
 *
 * sb_conv3x3_pack_filters: packs w [k][c][3][3] (desc->dtype, device) into
 * `packed` (device, packed_bytes >= sb_conv3x3_packed_bytes, not
 * overlapping w), on `stream`.  The result serves every call of that pass
 * on a descriptor with the same n, c, h, w, k and dtype, until w changes;
 * the caller orders it before those calls (same stream, or an event).
 * SB_ERR_INVALID_ARG for a bad descriptor, pass, pointer or size. */
size_t sb_conv3x3_packed_bytes(const sb_conv3x3_desc *desc, int pass);
sb_status sb_conv3x3_pack_filters(const sb_conv3x3_desc *desc, int pass,
                                  const void *w, void *packed,
                                  size_t packed_bytes, void *stream);

/* The packing of `count` (1..64) filter tensors in one launch, each as
 * sb_conv3x3_pack_filters(&descs[i], passes[i], w[i], packed[i],
 * packed_bytes[i]) would do it; all descriptors of one dtype, the packed
 * buffers disjoint.  A packing moves little data, so packing every layer of
 * a network this way costs about one launch instead of one per layer and
 * pass.  The host arrays are read before the call returns. */
sb_status sb_conv3x3_pack_filters_many(int count, const sb_conv3x3_desc *descs,
                                       const int *passes, const void *const *w,
                                       void *const *packed,
                                       const size_t *packed_bytes, void *stream);

/* Forward:  y[n,k,h,w] = bias[k] + sum_{c,r,s} x[n,c,h+r-1,w+s-1] * w[k,c,r,s]
 * (x = 0 outside the image), then max(y, 0) when SB_FUSE_RELU is set.
 * bias may be NULL (zero).  With SB_PACKED_FILTERS, w is the forward
 * packing of the filters (sb_conv3x3_pack_filters, SB_PASS_FWD). */
sb_status sb_conv3x3_fwd(const sb_conv3x3_desc *desc, const void *x,
                         const void *w, const float *bias, void *y,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Forward followed by ReLU + 2x2 / stride 2 max pooling in one call
 * (sec. 2.2: a convolution, its ReLU and the pooling layer after it; the
 * pooled layer's pre-activation is read by nothing else in a step, so it is
 * never written): the forward's output z as sb_conv3x3_fwd would store it
 * without SB_FUSE_RELU (bias added, rounded to the storage type), then
 * y and idx exactly as sb_relu_maxpool_fwd computes them from z.  y is
 * [n][k][h/2][w/2] and idx one byte per element of y, both in desc->layout.
 * Supported with even h and w for SB_NCHW8C bf16 when the forward's channel
 * loop is not split, and for SB_NCHW fp32 (an unsplit plan pools in the
 * kernel, a split one in its split reduction; not the few-output-channel
 * kernel): sb_conv3x3_workspace_bytes(desc, SB_PASS_FWD_POOL) is then not
 * (size_t)-1.  SB_ERR_UNSUPPORTED otherwise, SB_ERR_INVALID_ARG
 * for odd h or w, SB_FUSE_RELU, NULL pointers or overlapping outputs.
 * With SB_PACKED_FILTERS, w is the forward packing (SB_PASS_FWD). */
sb_status sb_conv3x3_fwd_pool(const sb_conv3x3_desc *desc, const void *x,
                              const void *w, const float *bias, void *y,
                              uint8_t *idx, void *workspace,
                              size_t workspace_bytes, void *stream);

/* Data gradient (sec. 2.2 backward propagation):
 *   dx[n,c,i,j] = sum_{k,r,s} dy[n,k,i-r+1,j-s+1] * w[k,c,r,s]
 * over in-image output positions.  When relu_mask_src is non-NULL (shape of
 * dx: the activation of the layer below, whose ReLU this gradient crosses),
 * dx is set to 0 wherever relu_mask_src <= 0.  desc->flags must be 0 or
 * SB_PACKED_FILTERS (w then the data-gradient packing, SB_PASS_BWD_DATA). */
sb_status sb_conv3x3_bwd_data(const sb_conv3x3_desc *desc, const void *dy,
                              const void *w, const void *relu_mask_src,
                              void *dx, void *workspace,
                              size_t workspace_bytes, void *stream);

/* Weight gradient (sec. 2.2 backward propagation; sec. 3.1 Modulo Layer:
 * the conv parameters are updated from the gradient of the whole local
 * batch):
 *   dw[k,c,r,s] = sum_{n,h,w} x[n,c,h+r-1,w+s-1] * dy[n,k,h,w]   (fp32)
 *   db[k]       = sum_{n,h,w} dy[n,k,h,w]                        (fp32)
 * dw and db are overwritten; db may be NULL.  The summation order is fixed
 * (no atomics): repeated calls give bit-identical results. */
sb_status sb_conv3x3_bwd_weight(const sb_conv3x3_desc *desc, const void *x,
                                const void *dy, float *dw, float *db,
                                void *workspace, size_t workspace_bytes,
                                void *stream);

/* Weight gradients of `count` layers (1..SB_MANY_MAX) in one call, each as
 * sb_conv3x3_bwd_weight computes it (bit-identical results).  The weight
 * gradient of a step reads nothing a later layer's backward writes, so a
 * caller may defer several layers' weight gradients and issue them
 * together; consecutive layers whose plans run the same kernel then share
 * one launch (one round of blocks ramping up and draining instead of one
 * per layer).
 *  * descs[i], x[i], dy[i], dw[i] as for sb_conv3x3_bwd_weight; db may be
 *    NULL (no bias gradients) or an array whose entries may be NULL.  The
 *    arrays are host memory, read during the call only.
 *  * workspace: sb_conv3x3_bwd_weight_many_workspace_bytes(count, descs)
 *    bytes, layer i's split partials in its own region; needs no
 *    initialisation.
 *  * SB_ERR_INVALID_ARG for a count out of range, null arrays or pointers,
 *    an invalid descriptor, an output overlapping any layer's input or any
 *    other output, or a workspace overlapping any operand;
 *    SB_ERR_WORKSPACE for a short workspace.  Nothing is enqueued then. */
#define SB_MANY_MAX 64
size_t sb_conv3x3_bwd_weight_many_workspace_bytes(int count,
                                                  const sb_conv3x3_desc *descs);
sb_status sb_conv3x3_bwd_weight_many(int count, const sb_conv3x3_desc *descs,
                                     const void *const *x,
                                     const void *const *dy, float *const *dw,
                                     float *const *db, void *workspace,
                                     size_t workspace_bytes, void *stream);

/* Weight gradient for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Computes exactly what sb_conv3x3_bwd_weight computes, with the same kernels
 * and the same summation order (bit-identical results), but takes no
 * workspace: the split partial sums go to a scratch array of
 * SB_NOALLOC_SCRATCH_BYTES that the library keeps in device memory, one per
 * device, reserved when the library's device code is first loaded on that
 * device and held until the process ends.  The call itself allocates and
 * frees nothing.
 *  * The stream must belong to the current device (the scratch array used is
 *    the current device's).
 *  * Every call on a device shares that device's array, and its contents
 *    after a call are dead.  Calls on one device that may overlap in time
 *    (different streams without ordering between them) race on it: the
 *    caller serialises them.
 *  * SB_ERR_WORKSPACE when sb_conv3x3_workspace_bytes(desc,
 *    SB_PASS_BWD_WEIGHT) exceeds SB_NOALLOC_SCRATCH_BYTES (nothing enqueued);
 *    other errors as for sb_conv3x3_bwd_weight. */
#define SB_NOALLOC_SCRATCH_BYTES (40u << 20)
sb_status sb_conv3x3_bwd_weight_noalloc(const sb_conv3x3_desc *desc,
                                        const void *x, const void *dy,
                                        float *dw, float *db, void *stream);

/* Describes the launch plan `pass` would use for `desc`: the name of the
 * main kernel as a profiler reports it, the grid and whether a split
 * reduction follows.  Writes at most `len` bytes (NUL-terminated) into buf
 * and returns the length of the full string plus one; returns 0 for an
 * invalid or unsupported descriptor.  Enqueues nothing. */
size_t sb_conv3x3_plan_string(const sb_conv3x3_desc *desc, int pass, char *buf,
                              size_t len);

/* ------------------------------------------------------------------------
 * Fused ReLU + 2x2 max pooling, stride 2 (sec. 2.2: pooling layers
 * subsample; sec. 3.1 Layer Partitioning: pooling is never partitioned).
 *
 *   x   [n][c][h][w]       h and w even and > 0
 *   y   [n][c][h/2][w/2]   y = max(0, max of the window)
 *   idx [n][c][h/2][w/2]   uint8 code per window: bits 0-1 = row-major
 *                          position of the first maximum (0:(0,0) 1:(0,1)
 *                          2:(1,0) 3:(1,1)); bit 7 set when that maximum
 *                          is <= 0 (the ReLU blocks the gradient); bits
 *                          2-6 zero.
 * Backward: dx (un-pooled shape) is zero except dx[window position] = dy
 * for windows whose bit 7 is clear.  dx is fully overwritten.
 * layout (sb_layout) applies to x, y, dy, dx and idx alike (idx one byte per
 * element of y); SB_NCHW8C needs c a multiple of 8 (SB_ERR_INVALID_ARG
 * otherwise).
 * ---------------------------------------------------------------------- */
sb_status sb_relu_maxpool_fwd(int n, int c, int h, int w, int dtype, int layout,
                              const void *x, void *y, uint8_t *idx,
                              void *stream);
sb_status sb_relu_maxpool_bwd(int n, int c, int h, int w, int dtype, int layout,
                              const void *dy, const uint8_t *idx, void *dx,
                              void *stream);

/* ------------------------------------------------------------------------
 * FC column shard (sec. 3.1 Layer Partitioning: a LINEAR layer is split to
 * 1/K of its outputs; Modulo Layer: it runs on the batch gathered from the
 * K workers; Shard Layer: its backward yields gradients over the full
 * input, which are reduced across workers later).
 *
 *   x        [m][k_in]      gathered activations, row stride ldx
 *   w_shard  [k_in][n_shard] this worker's columns of W, dense
 *   y, dy    [m][n_shard]   row stride ldy
 * ---------------------------------------------------------------------- */
typedef struct {
    int m, k_in, n_shard;  /* gathered rows, input features, shard columns */
    int dtype;             /* sb_dtype: SB_F32, or SB_BF16 (x, w_shard, y,
                              dy, relu_mask_src, dx_partial bfloat16; b_shard,
                              dw_shard, db_shard fp32; products on fp32 MFMA
                              from the exactly widened values, y and
                              dx_partial rounded to nearest-even)          */
    int ldx;               /* row stride of x and dx_partial (>= k_in)     */
    int ldy;               /* row stride of y, dy, relu_mask_src (>= n_shard) */
    unsigned flags;        /* SB_FUSE_RELU (forward only)                  */
} sb_fc_desc;

enum { SB_FC_FWD = 0, SB_FC_BWD = 1 };

/* Workspace bytes for `pass`; (size_t)-1 for an invalid descriptor. */
size_t sb_fc_workspace_bytes(const sb_fc_desc *desc, int pass);

/* y = x * w_shard + b_shard, then max(y, 0) with SB_FUSE_RELU.  b_shard
 * [n_shard] may be NULL. */
sb_status sb_fc_shard_fwd(const sb_fc_desc *desc, const void *x,
                          const void *w_shard, const float *b_shard, void *y,
                          void *workspace, size_t workspace_bytes, void *stream);

/* With g = dy, or g = dy * [relu_mask_src > 0] when relu_mask_src (shape
 * and stride of dy: this shard's ReLU output) is non-NULL:
 *   dx_partial[i,k] = sum_j g[i,j] * w_shard[k,j]   (may be NULL: skipped)
 *   dw_shard[k,j]   = (accumulate ? dw_shard[k,j] : 0) + sum_i x[i,k] g[i,j]
 *   db_shard[j]     = (accumulate ? db_shard[j]   : 0) + sum_i g[i,j]
 * dw_shard and db_shard are fp32; db_shard may be NULL.  accumulate = 1
 * adds the gradient of the K successive modulo iterations in place.  The
 * division by K that the paper applies to FC gradients is the optimiser's
 * and is not done here. */
sb_status sb_fc_shard_bwd(const sb_fc_desc *desc, const void *x,
                          const void *w_shard, const void *dy,
                          const void *relu_mask_src, void *dx_partial,
                          float *dw_shard, float *db_shard, int accumulate,
                          void *workspace, size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Modulo and shard layers on one device (sec. 3.1, Modulo Layer and Shard
 * Layer; sec. 3.2, Group MP Extension).
 *
 * The buffers of `workers` emulated workers sit on this device, worker w's
 * slot at w * stride elements from the base pointer (the layout an
 * exchange between devices would fill, one slot per peer).  Workers form MP
 * groups of `mp` consecutive ids (group of worker i: first id
 * g = (i / mp) * mp); inside a group the paper's K is mp, so mp = 1 is plain
 * data parallelism and mp = workers a single group.  A call serves the
 * group of worker `iproc`: all workers of a group gather the same data, and
 * a backward call writes the results of every worker of the group.  All
 * tensors are fp32, row-major; sums run over the group's workers in
 * increasing id (the result does not depend on the launch).  Strides are
 * in elements and at least one slot's size; input and output slots of the
 * group must not overlap.  Invalid arguments return SB_ERR_INVALID_ARG with
 * nothing enqueued.
 * ---------------------------------------------------------------------- */
typedef struct {
    int workers;   /* N, a multiple of mp                                  */
    int mp;        /* MP group size (the paper's K), >= 1                  */
    int batch;     /* B: examples per local batch, a multiple of mp        */
    int features;  /* F: elements per example                              */
} sb_modulo_desc;

/* Modulo layer forward, iteration k (the counter modulo mp, 0 <= k < mp).
 * Gathered example b comes from worker g + b / s (the paper's b / size
 * within the group, s = B / mp), block k of its local batch:
 *   gathered[b][f] = local[(g + b/s) * local_stride + (k*s + b%s) * F + f]
 * local: `workers` slots of [B][F]; gathered: [B][F]. */
sb_status sb_modulo_fwd(const sb_modulo_desc *desc, int iproc, int k,
                        const float *local, size_t local_stride,
                        float *gathered, void *stream);

/* Modulo layer backward, iteration k.  dgathered: `workers` slots of [B][F],
 * each worker's gradient with respect to its gathered batch (a partial sum:
 * its FC shard covers 1/mp of the layer's outputs).  For each worker g + r
 * of the group, rows k*s .. k*s + s - 1 of its dlocal slot receive the
 * group's sum at the gathered examples it supplied:
 *   dlocal[(g + r) * dl_stride + (k*s + j) * F + f]
 *       = sum_{w = 0 .. mp-1} dgathered[(g + w) * dg_stride + (r*s + j) * F + f]
 * Other rows of dlocal are left as they are (the mp iterations fill them in
 * turn). */
sb_status sb_modulo_bwd(const sb_modulo_desc *desc, int iproc, int k,
                        const float *dgathered, size_t dg_stride,
                        float *dlocal, size_t dl_stride, void *stream);

typedef struct {
    int workers;   /* N, a multiple of mp                                  */
    int mp;        /* MP group size, >= 1                                  */
    int rows;      /* M: rows of the batch                                 */
    int shard;     /* Ns: output columns of one worker's partition         */
} sb_shard_desc;

/* Shard layer forward: the next layer's full input [M][mp*Ns] from the
 * group's partitioned outputs (`workers` slots of [M][Ns]):
 *   full[m][r*Ns + c] = parts[(g + r) * parts_stride + m*Ns + c] */
sb_status sb_shard_fwd(const sb_shard_desc *desc, int iproc,
                       const float *parts, size_t parts_stride, float *full,
                       void *stream);

/* Shard layer backward: dfull holds `workers` slots of [M][mp*Ns], each
 * worker's gradient with respect to the full input (partial sums from its
 * shard of the layer above).  Worker g + r receives its column slice,
 * summed over the group:
 *   dparts[(g + r) * dp_stride + m*Ns + c]
 *       = sum_{w = 0 .. mp-1} dfull[(g + w) * df_stride + m*mp*Ns + r*Ns + c] */
sb_status sb_shard_bwd(const sb_shard_desc *desc, int iproc,
                       const float *dfull, size_t df_stride, float *dparts,
                       size_t dp_stride, void *stream);

/* Model averaging (sec. 2: data-parallel replicas reach a global model by
 * averaging; sec. 4: every worker exchanges its parameters up to the modulo
 * layer every few batches, and the FC model shards are averaged across the
 * MP groups).  params holds `workers` slots of n fp32 elements (worker w at
 * w * stride elements, stride >= n).  Worker g * mp + r holds shard r of
 * group g (sec. 3.2), so each slot is replaced, in place, by the mean over
 * the workers holding the same parameters:
 *   mp = 1: all workers (the conv layers' replicas);
 *   mp > 1: the workers r, mp + r, 2 mp + r, ... (FC shard r across groups).
 * Each mean is the sum in increasing worker id, divided once by the count.
 * workers must be a multiple of mp; slots must not overlap (stride >= n).
 * n = 0 does nothing. */
sb_status sb_model_average(int workers, int mp, size_t n, float *params,
                           size_t stride, void *stream);

/* Model averaging of replicas in separate buffers (the same reduce as
 * sb_model_average, sec. 2 and sec. 4, for replicas that do not share one
 * slotted allocation: one call per parameter tensor, with the tensor of
 * every replica, e.g. a conv layer's filters in every MP group, or FC shard
 * r of every group).  params is a HOST array of `replicas` device pointers,
 * each to n fp32 elements; every one is replaced, in place, by the mean
 * over the replicas (the sum in increasing replica index, divided once by
 * the count).  1 <= replicas <= SB_MAX_REPLICAS; the pointers must be
 * non-NULL and their ranges must not overlap (SB_ERR_INVALID_ARG).  n = 0
 * or a single replica does nothing. */
#define SB_MAX_REPLICAS 64
sb_status sb_model_average_replicas(int replicas, size_t n, float *const *params,
                                    void *stream);

/* ------------------------------------------------------------------------
 * Loss and parameter update (NEXT after the worker's forward and backward).
 *
 * Log-softmax and negative log-likelihood on the complete model output
 * (sec. 3.1 Layer Partitioning: when the last FC layer is partitioned, a
 * shard layer before the LOG_SOFTMAX layer hands every worker the full
 * output, so the output error is evaluated as for a complete local model).
 * Per row i of the logits z [m][classes] (row stride ldz, fp32):
 *   logp[i][c] = z[i][c] - log(sum_j exp(z[i][j]))
 *   loss[i]    = -logp[i][labels[i]]
 *   dz[i][c]   = scale * (exp(logp[i][c]) - [c == labels[i]])
 * i.e. dz is the gradient of scale * sum_i loss[i] (scale = 1/m for the
 * batch mean).  labels [m] are int32 device values; the kernel never
 * indexes memory with them: a label outside [0, classes) gives loss[i] =
 * NaN and a NaN row of dz.  logp, loss and dz may each be NULL (not
 * written); logp and dz use row stride ldz.  Outputs must not overlap z or
 * labels.  Sums run in a fixed order (bitwise reproducible).
 * ---------------------------------------------------------------------- */
sb_status sb_log_softmax_nll(int m, int classes, int ldz, const float *z,
                             const int32_t *labels, float scale, float *logp,
                             float *loss, float *dz, void *stream);

/* Plain SGD step on `count` fp32 tensors (sec. 4: SGD on mini-batches;
 * sec. 3.1 Modulo Layer: the FC layers, updated K times per local batch,
 * divide their gradients by K):
 *   w[t][i] = w[t][i] - (lr * scale[t]) * g[t][i],  i < n[t]
 * with the product lr * scale[t] formed once (fp32) and one fused
 * multiply-add per element.  w, g, n and scale are HOST arrays of `count`
 * entries (1 <= count <= SB_SGD_MAX_TENSORS); w[t] and g[t] are device
 * pointers, n[t] may be 0 (nothing to do; pointers may then be NULL).  A
 * gradient must not overlap any parameter tensor of the call, and the
 * parameter tensors must not overlap each other. */
enum { SB_SGD_MAX_TENSORS = 64 };
sb_status sb_sgd_update(int count, float *const *w, const float *const *g,
                        const size_t *n, const float *scale, float lr,
                        void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SB_H */
