/*
 * CPU oracle for frame-to-frame convolutional activation reuse.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path includes, links or
 * calls this code: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load it.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * What it computes is the plain definition, not the reuse method: the reuse
 * method (Abstract; Sec. 1) recomputes only what changed and must reach
 * exactly what a full recompute of the current frame gives, so the full
 * recompute is the expected result.  Change sets, their per-layer growth
 * (Fig. 1 caption: a k x k convolution spreads a change by (k-1)/2 pixels on
 * each side), dirty-tile masks and the work list depend only on the change
 * set and are written out from their definitions.
 *
 * Conventions (readings where the paper is silent):
 *   - tensors are C-contiguous float32, channel-major [C][H][W];
 *   - convolution is cross-correlation with OIHW weights, zero padding,
 *     output size floor((n + 2p - k) / s) + 1, then bias, then ReLU;
 *   - sums accumulate in double and round once to float32;
 *   - masks are one byte per pixel / per tile, 1 = dirty;
 *   - a tile grid of tile_h x tile_w cells is anchored at (0, 0) on every
 *     layer's output grid; edge tiles may be partial.
 */
#ifndef REUSE_ORACLE_H
#define REUSE_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_MAX_LAYERS 8

typedef struct {
    int in_c, h, w;                    /* input frame (channels, rows, cols) */
    int n_conv;                        /* conv layers, 1..ORC_MAX_LAYERS */
    int cin[ORC_MAX_LAYERS], cout[ORC_MAX_LAYERS];
    int k[ORC_MAX_LAYERS], s[ORC_MAX_LAYERS], p[ORC_MAX_LAYERS];
    int n_out;                         /* logits */
    int tile_h, tile_w;                /* dirty-tile grid cell */
    int bf16;                          /* 1: bf16 weights/activations, see orc_forward */
} orc_net;

/* Input levels (Sec. 2: grayscale frames): uint8 level k -> fl32(k / 255). */
float orc_level_to_f32(uint8_t k);
void orc_levels_to_f32(const uint8_t *k, size_t n, float *out);

/* Round-to-nearest-even to bfloat16, returned as the float it represents. */
float orc_bf16_rne(float x);
void orc_bf16_rne_array(const float *x, size_t n, float *out);

/* floor((n + 2p - k) / s) + 1 */
int orc_out_size(int n, int k, int s, int p);

/* Shape of layer l (0 = input) of a net. */
void orc_layer_shape(const orc_net *net, int l, int *c, int *h, int *w);

/* Change detection (Abstract; Sec. 1): d0[y][x] = 1 iff some channel's
 * float32 bit pattern differs between prev and cur. */
void orc_diff(int c, int h, int w, const float *prev, const float *cur, uint8_t *d0);

/* Known-change mode (Sec. 1, occlusion): d0 = union of the boxes, each
 * (y0, x0, y1, x1) half-open, clipped to the frame. */
void orc_box_mask(int h, int w, int nb, const int32_t *boxes, uint8_t *d0);

/* Change growth through one conv layer (Fig. 1 caption): output pixel
 * (y', x') is dirty iff its k x k input window at (s*y'-p, s*x'-p) holds a
 * dirty input pixel.  Output grid size from orc_out_size. */
void orc_dilate(int h, int w, const uint8_t *din, int k, int s, int p, uint8_t *dout);

/* Dirty-tile mask: m[ty][tx] = 1 iff the tile holds a dirty pixel
 * (local-area recompute, Sec. 3). */
void orc_tile_mask(int h, int w, const uint8_t *d, int tile_h, int tile_w, uint8_t *m);

/* Work list of one layer: every (stream, ty, tx) with m = 1, ordered by
 * (ty, tx, stream) ascending, encoded stream << 16 | ty << 8 | tx.
 * masks: [n][th][tw].  Returns the count. */
int orc_worklist(int n, int th, int tw, const uint8_t *masks, uint32_t *out);

/* One conv layer, full recompute: y = ReLU(fl32(b + sum w * x)).  bf16 != 0
 * additionally rounds each output to bfloat16 (inputs and weights are taken
 * as given). */
void orc_conv2d_relu(int cin, int h, int w, const float *x, int cout, int k, int s, int p,
                     const float *wt, const float *b, int bf16, float *y);

/* The same layer, recomputed only at the pixels of tiles with tmask = 1; every
 * other output keeps the value already in y (plain reuse, Sec. 1). */
void orc_conv2d_relu_tiles(int cin, int h, int w, const float *x, int cout, int k, int s, int p,
                           const float *wt, const float *b, int bf16,
                           const uint8_t *tmask, int tile_h, int tile_w, float *y);

/* Dense head: logits[n] = fl32(bd[n] + sum_j wd[n][j] * a[j]). */
void orc_dense(int kdim, const float *a, int n, const float *wd, const float *bd, float *logits);

/* Full recompute of n independent inputs x [n][in_c][h][w] (OpenMP over the
 * inputs).  acts: NULL, or n_conv pointers (each may be NULL) receiving layer
 * outputs [n][C_l][H_l][W_l].  logits [n][n_out].
 * bf16 mode: weights (conv and dense) and the input are rounded to bfloat16
 * once, every conv output is rounded to bfloat16, logits stay float32;
 * biases stay float32.  Returns 0, or -1 on a bad net description. */
int orc_forward(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                const float *dense_w, const float *dense_b, int n, const float *x,
                float *const *acts, float *logits);

/* Masks of one step for n streams (OpenMP over streams).  d0: [n][h][w].
 * d: NULL or n_conv + 1 pointers, d[l] = [n][H_l][W_l] (d[0] gets a copy of d0).
 * m: n_conv + 1 pointers, m[l] = [n][TH_l][TW_l].  Returns 0 or -1. */
int orc_masks(const orc_net *net, int n, const uint8_t *d0, uint8_t *const *d, uint8_t *const *m);

/* Plain reuse step of one stream (Sec. 1): diff x against cache[0] (or take
 * d0_given if non-NULL; all dirty if primed == 0), copy x into cache[0] where
 * changed, grow the change set layer by layer, recompute each layer only on
 * its dirty tiles (cache[l] updated in place) and run the dense head.
 * cache[l] holds layer l's activations [C_l][H_l][W_l], l = 0..n_conv.
 * Weights must already be in the precision the mode uses (bf16 mode: rounded
 * to bfloat16; the cached input stays float32 and is rounded as layer 1 reads
 * it).  Returns 0 or -1. */
int orc_reuse_step(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                   const float *dense_w, const float *dense_b, const float *x,
                   const uint8_t *d0_given, int primed, float *const *cache, float *logits);

/* ---- training (Sec. 2: the policy is trained with REINFORCE) ---- */

/* dJ/dlogits of the REINFORCE loss J = sum_i -returns[i] log softmax(logits_i)[actions[i]]:
 * g[i][o] = returns[i] (softmax(logits_i)[o] - [o == actions[i]]).  Double inside. */
void orc_reinforce_dlogits(int n, int n_out, const float *logits, const int32_t *actions,
                           const float *returns, float *g);

/* Pre-activations of one input: z[l] = fl32(b + sum w a_{l-1}) of layer l + 1,
 * [C][H][W], before the ReLU (a = the float32 activations of orc_forward).
 * Float32 nets only.  Returns 0 or -1. */
int orc_forward_preact(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                       const float *x, float *const *z);

/* Gradients of J = sum_i sum_o g[i][o] logits[i][o] with respect to every
 * weight and bias, summed over the n inputs x [n][in_c][h][w] (backpropagation
 * through orc_forward, double accumulation, ReLU derivative 0 at the kink).
 * Outputs in the layouts of the weights: dconv_w[l] OIHW, dconv_b[l] [cout],
 * ddense_w [n_out][C_L H_L W_L] in (c, y, x) order, ddense_b [n_out].
 * Float32 nets only.  Returns 0 or -1. */
int orc_backward(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                 const float *dense_w, const float *dense_b, int n, const float *x, const float *g,
                 float *const *dconv_w, float *const *dconv_b, float *ddense_w, float *ddense_b);

#ifdef __cplusplus
}
#endif
#endif
