/*
 * reuse_net — frame-to-frame convolutional activation reuse on MI355X (gfx950).
 *
 * The method (Abstract; Sec. 1): keep each conv layer's activations from the
 * previous frame, find which input pixels changed, and recompute only the
 * outputs those changes can reach, reusing the cached activations everywhere
 * else.  A k x k convolution spreads a change by (k-1)/2 pixels on each side
 * per layer (Fig. 1 caption).  Instead of the paper's single rectangle per
 * frame, changes are tracked as small dirty tiles (the local-area variant of
 * Sec. 3), and many independent streams (environments, cameras, occlusion
 * variants) are processed per launch.
 *
 * Network: n_conv conv layers, each followed by bias and ReLU, then a dense
 * layer to n_out logits (Sec. 2: two conv layers and a dense layer).  The
 * dense input is the last conv output flattened in (channel, row, column)
 * order, as torch's NCHW .flatten(1).  A change spreads through a layer by its
 * window (Fig. 1): output pixel (y, x) of a k x k layer with stride s and zero
 * pad p changed iff an input pixel in rows s y - p .. s y - p + k - 1 and the
 * same columns changed.
 *
 * Conventions
 *   - Every function returns an rn_status (0 = RN_OK, negative = error) unless
 *     stated otherwise; on an argument error nothing is changed and
 *     reuse_net_last_error() describes the failure.  No function aborts.
 *   - "dev_" pointers are device memory owned by the caller.  The library
 *     never allocates or frees device memory: all of its device state lives in
 *     the caller's workspace, which must outlive the net.
 *   - hip_stream is a hipStream_t passed as void* (NULL = the null stream).
 *     reuse_net_step and reuse_net_full only enqueue kernels on it and return;
 *     launch failures return RN_EHIP, device faults surface at the caller's
 *     next synchronisation.  No host synchronisation happens inside them.
 *   - Introspection calls (get_*, read_activation) synchronise the stream of
 *     the last step and copy into caller host buffers.
 *   - A net is not thread-safe; calls on one net must not overlap.
 */
#ifndef REUSE_NET_H
#define REUSE_NET_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RN_MAX_CONV 8

typedef enum {
    RN_OK = 0,
    RN_EINVAL = -1,        /* bad argument or null pointer */
    RN_EUNSUPPORTED = -2,  /* valid request the library does not implement */
    RN_ENOSPACE = -3,      /* workspace or caller buffer too small */
    RN_EHIP = -4,          /* a HIP runtime call failed */
    RN_ESTATE = -5         /* call not valid in the net's current state */
} rn_status;

typedef enum { RN_F32 = 0, RN_BF16 = 1, RN_U8 = 2 } rn_dtype;

/* How the dense head is evaluated.  Both give the same logits up to float32
 * rounding order; each is deterministic.
 *   RN_HEAD_TILES: the head is linear, so the logits are a sum over tiles of
 *     each tile's contribution (the reuse idea of Sec. 1 applied to the dense
 *     layer).  The contribution of every tile the last conv layer recomputes
 *     is recomputed with it (in that layer's epilogue, or, for bf16 and for
 *     float32 layers too large to keep their weights in LDS, by a matrix
 *     kernel that takes the recomputed tiles position by position), and the
 *     head adds the cached contributions in a fixed tile order.  Needs
 *     n_conv >= 2.
 *   RN_HEAD_FULL: the head reads the whole last-layer cache of every stream
 *     every step (split-K GEMV over C_L*H_L*W_L). */
typedef enum { RN_HEAD_TILES = 0, RN_HEAD_FULL = 1 } rn_head_mode;

/* One conv layer (OIHW weights), output grid ((H + 2 pad - k) / stride + 1) per
 * side.  Valid: k >= 1, stride >= 1, 0 <= pad <= (k - 1) / 2.  Kernels exist for
 * 3x3 stride 1 pad 1 (float32 and bf16, the channel pairs listed in the design
 * notes), and, float32 only, for k <= 8 with stride 1, 2 or 4 at the
 * (k, stride, cin, cout) shapes of the general-layer kernel; other layers make
 * reuse_net_create return RN_EUNSUPPORTED naming the shape. */
typedef struct {
    int32_t cin, cout, k, stride, pad;
} rn_conv_spec;

typedef struct {
    int32_t in_c, in_h, in_w;     /* channels, rows, columns of one frame */
    int32_t stack;                /* 1, or 4: the last 4 frames are conv1's input channels,
                                     oldest first (Sec. 1 and Sec. 3: multiple input frames);
                                     conv[0].cin must equal in_c * stack */
    int32_t n_conv;               /* 1..RN_MAX_CONV */
    const rn_conv_spec *conv;     /* host array [n_conv], read during create only */
    int32_t n_out;                /* logits per stream, 1..64 */
    int32_t tile_h, tile_w;       /* dirty-tile grid cell on every layer; supported: 4 x 4 */
    int32_t max_streams;          /* cache slots, 1..65535 */
    rn_dtype act_dtype;           /* RN_F32, or RN_BF16 (bf16 weights and activations,
                                     fp32 accumulation, fp32 logits) */
    rn_head_mode head_mode;       /* RN_HEAD_TILES (default, zero) or RN_HEAD_FULL */
    int32_t options;              /* bit set of RN_OPT_*, 0 = defaults */
} rn_config;

/* Options.
 *   RN_OPT_SEPARATE_FIRST: keep layer 1 as its own kernel writing its cache.
 *     By default, when the frame has one channel and layer 2 runs on the
 *     resident-weight MFMA kernel, layer 1 is folded into layer 2: each dirty
 *     layer-2 tile computes the layer-1 activations of its halo from the input
 *     patch around it (the same arithmetic, so the same bits) instead of
 *     reading a layer-1 cache.  Layer-1 masks and work lists are produced
 *     either way; reuse_net_read_activation(layer 1) then computes the layer
 *     on demand. */
#define RN_OPT_SEPARATE_FIRST 1

typedef struct {                  /* HOST pointers, float32, read during create only */
    const float *const *conv_w;   /* [n_conv], each [cout][cin][k][k] (OIHW) */
    const float *const *conv_b;   /* [n_conv], each [cout] */
    const float *dense_w;         /* [n_out][C_L * H * W], (c, y, x) flatten order */
    const float *dense_b;         /* [n_out] */
} rn_weights;

typedef struct reuse_net reuse_net;   /* opaque host object owned by the library */

/* Bytes of device workspace a net with this config needs (0 if the config is
 * invalid or unsupported). */
size_t reuse_net_workspace_bytes(const rn_config *cfg);

/* Validate cfg, lay out the caller's workspace (dev_workspace, >= the size
 * above, 256-byte aligned), pack the weights into the kernels' layouts and
 * upload them on hip_stream, clear every cache and mark every slot unprimed.
 * Synchronises hip_stream before returning.  *out receives the net. */
rn_status reuse_net_create(const rn_config *cfg, const rn_weights *w, void *dev_workspace,
                           size_t workspace_bytes, void *hip_stream, reuse_net **out);

/* One reuse step (Abstract; Sec. 1) for n streams.
 *   dev_stream_ids: [n] distinct cache slots in [0, max_streams), or NULL for 0..n-1.
 *   dev_frames:     [n][in_c][in_h][in_w], RN_F32 values, or RN_U8 levels k read as
 *                   k / 255 (correctly rounded float32).  With stack = 4 this is the
 *                   newest frame only; the library keeps the older three.
 *   dev_boxes, dev_box_off: NULL for change detection by diff.  Otherwise the
 *                   caller states the change (Sec. 1, known-change use such as
 *                   occlusion): boxes [nb][4] int32 (y0, x0, y1, x1), half-open, clipped
 *                   to the frame; stream i owns boxes [box_off[i], box_off[i+1]);
 *                   box_off has n+1 entries and box_off[0] = 0.  On a primed slot only
 *                   pixels inside the boxes are read from dev_frames; a slot that was
 *                   never primed (or was reset) ignores its boxes and reads and caches
 *                   the whole frame, so its frame must be complete.
 *   dev_logits:     [n][n_out] float32 output.
 * Change rule: a pixel changed iff the float32 bits of some channel differ from
 * the cached input (so -0 vs +0 is a change and an identical NaN is not).  A
 * slot that was never primed, or was reset, is treated as all-changed.
 * Enqueues diff (or boxes) -> dilation and tile masks -> work-list compaction ->
 * dirty-tile conv per layer (bias, ReLU and scatter into the caches fused) ->
 * dense head. */
rn_status reuse_net_step(reuse_net *net, int32_t n, const int32_t *dev_stream_ids,
                         const void *dev_frames, rn_dtype frame_dtype,
                         const int32_t *dev_boxes, const int32_t *dev_box_off,
                         float *dev_logits, void *hip_stream);

/* Dense recompute of every layer for n streams (the comparison path): the
 * frames are copied into the input caches and every tile of every layer is
 * recomputed, without work lists.  Gives the same bits as a step on which
 * every pixel changed, and leaves the slots primed.  With stack = 4 the frame
 * enters the slot's frame ring as a step's frame does (a never-primed slot
 * takes it as all four frames), and its change against the previous newest
 * frame is kept for the steps that follow, so a full call in the middle of a
 * stream leaves the same state as a step on the same frame.  The pixel and
 * tile masks of the slots are left as they were; reuse_net_get_worklist
 * reports RN_ESTATE until the next step. */
rn_status reuse_net_full(reuse_net *net, int32_t n, const int32_t *dev_stream_ids,
                         const void *dev_frames, rn_dtype frame_dtype, float *dev_logits,
                         void *hip_stream);

/* Mark one slot (or all, stream_id = -1) unprimed: its next step recomputes
 * everything.  Synchronises the last step's stream. */
rn_status reuse_net_reset(reuse_net *net, int32_t stream_id);

/* Replace the weights (training between rollouts: activations are reused
 * within a rollout whose weights are fixed, Sec. 1 and Sec. 2).  Same layout,
 * packing and host pointers as reuse_net_create.  Waits for the last step's
 * stream, uploads on hip_stream, marks every slot unprimed (the caches hold
 * activations of the old weights, so each slot's next step recomputes
 * everything; with stacked frames the frame ring restarts as at an episode
 * start, the next frame standing for the older ones) and synchronises
 * hip_stream.  On an argument error nothing changes. */
rn_status reuse_net_set_weights(reuse_net *net, const rn_weights *w, void *hip_stream);

/* ---- training (Sec. 2: the policy is trained with REINFORCE) ----
 *
 * Within a rollout the weights are fixed, so every forward step reuses
 * activations as in inference; a step's gradient is taken from the
 * activations the slots' caches hold after it.  A REINFORCE update over an
 * episode replays its frames through reuse steps and, after each, adds that
 * step's gradient (reuse_net_backward with accumulate = 1), then applies one
 * SGD step.  Supported for float32 nets of 3x3 stride-1 pad-1 layers at the
 * channel pairs of the backward kernels (first layer 1 or 4 -> 20, 40, 64 or
 * 80 channels; later layers 40->80, 64->128, 128->128); other nets return
 * RN_EUNSUPPORTED from the calls below.
 *
 * Gradient buffer (float32, device, caller-owned): the weights of rn_weights
 * in that order and layout, conv layer l's OIHW weights [cout][cin][3][3]
 * then its bias [cout] for l = 1..n_conv, then the dense weights
 * [n_out][C_L * H_L * W_L] in (c, y, x) order and the dense bias [n_out];
 * reuse_net_grad_elems floats in all. */

/* Floats of a gradient buffer (0 if the net does not support training). */
size_t reuse_net_grad_elems(const reuse_net *net);

/* Device scratch bytes reuse_net_backward needs for a batch of n streams
 * (0 if n is outside 1..max_streams or the net does not support training). */
size_t reuse_net_backward_scratch_bytes(const reuse_net *net, int32_t n);

/* REINFORCE's logit gradient (Sec. 2): for n streams with logits z [n][n_out],
 * sampled actions a [n] (0..n_out-1) and returns G [n],
 *   dlogits[i][o] = G_i (softmax(z_i)[o] - [o == a_i]),
 * the derivative of -G_i log softmax(z_i)[a_i].  Device pointers, enqueued on
 * hip_stream; RN_EINVAL for NULL pointers or n_out outside 1..64. */
rn_status reuse_net_reinforce_dlogits(int32_t n, int32_t n_out, const float *dev_logits,
                                      const int32_t *dev_actions, const float *dev_returns,
                                      float *dev_dlogits, void *hip_stream);

/* Gradient of J = sum_i sum_o dlogits[i][o] logits[i][o] with respect to
 * every weight and bias, for the n streams dev_stream_ids (NULL: 0..n-1) at the
 * inputs their slots' caches hold (the last step or full call on them; the
 * ReLU derivative is taken as 0 where an activation is 0).
 *   dev_dlogits: [n][n_out] float32.
 *   dev_grads:   reuse_net_grad_elems floats; accumulate = 0 overwrites it,
 *                accumulate != 0 adds this gradient to it.
 *   dev_scratch: caller-owned, 256-byte aligned, at least
 *                reuse_net_backward_scratch_bytes(net, n) bytes.
 * Deterministic (fixed summation order).  Enqueued on hip_stream; with layer
 * 1 folded into layer 2 (the default for one-channel frames) it first
 * recomputes the slots' layer-1 activations into the layer-1 cache. */
rn_status reuse_net_backward(reuse_net *net, int32_t n, const int32_t *dev_stream_ids,
                             const float *dev_dlogits, float *dev_grads, int32_t accumulate,
                             void *dev_scratch, size_t scratch_bytes, void *hip_stream);

/* One SGD step on the device: every weight w becomes fl(w - fl(lr * g)) with g
 * its entry of dev_grads (layout above), in every packed copy the kernels
 * read, so the net computes exactly as one created with the updated weights.
 * Marks every slot unprimed (the caches hold activations of the old weights;
 * the next step of each slot recomputes everything, and with stacked frames
 * the frame ring restarts as at an episode start).  Enqueued on hip_stream,
 * no host synchronisation. */
rn_status reuse_net_sgd_step(reuse_net *net, const float *dev_grads, float lr, void *hip_stream);

/* Replace the weights from device memory (training between rollouts, Sec. 1
 * and Sec. 2, when the new weights are already on the GPU: a learner's
 * parameters, or a copy kept beside the net).  dev_params: float32, device,
 * reuse_net_grad_elems floats in the gradient-buffer layout above (each conv
 * layer's OIHW weights then its bias, then the dense weights in (c, y, x)
 * order and the dense bias); read only, owned by the caller, and not
 * referenced after the call's work on hip_stream has run.  Every packed copy
 * the kernels read is rewritten from it on the device, so the net computes
 * exactly as one created with those weights (the same bits), and every slot
 * is marked unprimed as by reuse_net_set_weights.  Enqueued on hip_stream, no
 * host synchronisation and no host copy of the weights; work on other streams
 * that still reads the old weights must be ordered before it by the caller.
 * RN_EINVAL for a NULL net or dev_params; RN_EUNSUPPORTED (nothing changes)
 * for nets the training calls do not support; RN_EHIP if a launch fails. */
rn_status reuse_net_set_weights_device(reuse_net *net, const float *dev_params, void *hip_stream);

/* ---- variants of one slot: copy-on-write overlays (Sec. 1, known change) ---- */

/* Device scratch bytes reuse_net_variants needs for n variants when no variant
 * has more than max_tiles dirty tiles in any layer 1..n_conv (max_tiles <= 0:
 * no limit, room for every tile).  0 if n is outside 1..65535 or the net
 * cannot run variants (head_mode RN_HEAD_FULL, fewer than 2 layers, stack = 4). */
size_t reuse_net_variant_scratch_bytes(const reuse_net *net, int32_t n, int32_t max_tiles);

/* Evaluate n variants of one primed slot in a single pass, as used for
 * occlusion maps (Sec. 1): variant i is the slot's cached input with the
 * pixels of its boxes [box_off[i], box_off[i+1]) replaced by the same pixels
 * of frame i (frame_count = n) or of frame 0 (frame_count = 1: e.g. one
 * all-zero frame for zero patches).  Boxes are (y0, x0, y1, x1) int32,
 * half-open, clipped; box_off has n+1 entries, box_off[0] = 0.
 * The result is what a step with those boxes would give on a copy of the slot,
 * to float32 rounding (the same tiles are recomputed).  Nothing of the slot
 * changes: each variant recomputes only the tiles its change reaches, writes
 * them to per-layer overlays in dev_scratch (row = position in the layer's
 * work list) and reads every other activation and per-tile head contribution
 * from the base slot.  Logits go to dev_logits [n][n_out].
 *   dev_frames:   [frame_count][in_c][in_h][in_w], RN_F32 or RN_U8 (k / 255);
 *                 only pixels inside the variant's boxes are read.
 *   max_tiles:    per-variant limit that sizes the scratch (see above).  A
 *                 variant over the limit is left out and its logits are NaN;
 *                 all logits are NaN if the base slot was never primed.
 *   dev_scratch:  caller-owned device memory, 256-byte aligned, at least
 *                 reuse_net_variant_scratch_bytes(net, n, max_tiles) bytes.
 * Needs head_mode RN_HEAD_TILES, n_conv >= 2 and stack = 1 (RN_EUNSUPPORTED
 * otherwise).  Enqueues on hip_stream only.  Until the next step, full or
 * variants call, the introspection functions below describe the variants
 * (stream_id = variant index i; work-list entries i << 16 | ty << 8 | tx) and
 * read them from dev_scratch, which must then still hold them. */
rn_status reuse_net_variants(reuse_net *net, int32_t base_stream, int32_t n, const void *dev_frames,
                             rn_dtype frame_dtype, int32_t frame_count, const int32_t *dev_boxes,
                             const int32_t *dev_box_off, int32_t max_tiles, void *dev_scratch,
                             size_t scratch_bytes, float *dev_logits, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * reuse_net_variants with the library's own scratch instead of dev_scratch.
 * That scratch is a static device array of RN_STATIC_SCRATCH_BYTES per GPU
 * (64 MiB; 4096 variants of a 105x80 frame with max_tiles = 16 need about
 * 44 MB), held by each GPU the library runs on until the process ends.  The
 * call allocates nothing; a request whose scratch
 * (reuse_net_variant_scratch_bytes) exceeds the limit returns RN_ENOSPACE and
 * launches nothing.  Every call on one GPU, from any net, shares that GPU's
 * array and leaves its contents there: calls that overlap on one GPU (on
 * different streams or from different threads) race, and the introspection
 * functions describe a static call's variants only until the next one on
 * that GPU.  The net must be used with the device that was current at
 * reuse_net_create.  Arguments and results as reuse_net_variants. */
#define RN_STATIC_SCRATCH_BYTES (64u << 20)
rn_status reuse_net_variants_static(reuse_net *net, int32_t base_stream, int32_t n, const void *dev_frames,
                                    rn_dtype frame_dtype, int32_t frame_count, const int32_t *dev_boxes,
                                    const int32_t *dev_box_off, int32_t max_tiles, float *dev_logits,
                                    void *hip_stream);

/* ---- introspection (synchronous; for parity checks and statistics) ---- */

/* Pixel change mask of a slot after its last step, layer 0 (input) .. n_conv.
 * Row-major bit rows: word (y * words_per_row + x / 64), bit x % 64, with
 * words_per_row = ceil(in_w / 64).  words >= in_h * words_per_row. */
rn_status reuse_net_get_pixel_mask(reuse_net *net, int32_t layer, int32_t stream_id,
                                   uint64_t *out, size_t words);

/* Dirty-tile mask of a slot after its last step: bit t = ty * TW + tx of word
 * t / 64, TW = ceil(in_w / tile_w).  words >= ceil(TH * TW / 64). */
rn_status reuse_net_get_tile_mask(reuse_net *net, int32_t layer, int32_t stream_id,
                                  uint64_t *out, size_t words);

/* Work list of layer 1..n_conv from the last step: the dirty tiles in
 * ascending (ty, tx, batch index i) order, encoded i << 16 | ty << 8 | tx, where
 * i indexes that call's stream batch (RN_ESTATE after a full).  *count receives the length; at most
 * cap entries are copied (RN_ENOSPACE if cap < count, with *count still set). */
rn_status reuse_net_get_worklist(reuse_net *net, int32_t layer, uint32_t *out, size_t cap,
                                 int32_t *count);

/* Cached activations of a slot, layer 0 (the float32 input cache, newest frame
 * for stack = 4) .. n_conv, as float32 [C][H][W] in host memory. */
rn_status reuse_net_read_activation(reuse_net *net, int32_t stream_id, int32_t layer,
                                    float *host_out);

typedef struct {
    int64_t streams;              /* n of the last step */
    int64_t changed_px;           /* changed input pixels, summed over the streams */
    int64_t dirty_tiles[RN_MAX_CONV + 1];   /* per layer 0..n_conv */
    int64_t useful_mac;           /* MACs of in-image pixels of dirty tiles + dense head */
    int64_t issued_mac;           /* MACs the kernels issued (whole tiles) + dense head */
    int64_t dense_mac;            /* MACs of a dense recompute of the same streams */
} rn_stats;

/* Statistics of the last step or full call. */
rn_status reuse_net_get_stats(reuse_net *net, rn_stats *out);

/* ---- kernel timing with HIP events (measurement support) ---- */

#define RN_PHASES 9
typedef enum {
    RN_PHASE_MASKS = 0,   /* diff or boxes, dilation, tile masks */
    RN_PHASE_COMPACT = 1, /* work-list compaction */
    RN_PHASE_CONV1 = 2,   /* first conv layer on dirty tiles */
    RN_PHASE_CONVN = 3,   /* conv layers 2..n_conv on dirty tiles (MFMA) */
    RN_PHASE_HEAD = 4,    /* dense head */
    RN_PHASE_BWD_HEAD = 5,/* backward: dense head and the last layer's gradient (and a layer-1 recompute) */
    RN_PHASE_BWD_DW = 6,  /* backward: weight and bias gradients of the conv layers (MFMA) */
    RN_PHASE_BWD_DX = 7,  /* backward: gradients at the conv layers' inputs (MFMA) */
    RN_PHASE_SGD = 8      /* SGD step on the packed weights */
} rn_phase;

typedef struct {
    double ms[RN_PHASES];         /* summed event time per phase */
    int64_t launches[RN_PHASES];  /* kernel launches per phase */
    double layer_ms[RN_MAX_CONV + 1];          /* conv kernels of layer l = 1..n_conv
                                                  (index 0: every other kernel) */
    int64_t layer_launches[RN_MAX_CONV + 1];
} rn_profile;

/* enable != 0: bracket every later kernel launch with HIP events on the
 * launch stream and accumulate; 0 stops.  Either way the totals restart. */
rn_status reuse_net_set_profiling(reuse_net *net, int32_t enable);

/* Synchronise and return the totals since profiling was enabled. */
rn_status reuse_net_get_profile(reuse_net *net, rn_profile *out);

/* Text of the last error on this net (never NULL; "" if none).  net may be
 * NULL for errors of reuse_net_create. */
const char *reuse_net_last_error(const reuse_net *net);

/* Release the host object.  The caller then owns (and may free) the workspace. */
void reuse_net_destroy(reuse_net *net);

#ifdef __cplusplus
}
#endif
#endif
