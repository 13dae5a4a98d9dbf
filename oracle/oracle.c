/*
 * CPU oracle for frame-to-frame convolutional activation reuse — test
 * infrastructure only (see oracle.h).  Plain loops, double accumulation,
 * no blocking or fusion, so that each function can be checked against its
 * definition by eye.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- scalars */

float orc_level_to_f32(uint8_t k) {
    /* Sec. 2: grayscale frames; a level k maps to k / 255.  The division is
     * done in double and rounded once to float: k / 255 is never within half a
     * double ulp of a float rounding midpoint, so this is the correctly
     * rounded float quotient. */
    return (float)((double)k / 255.0);
}

void orc_levels_to_f32(const uint8_t *k, size_t n, float *out) {
    for (size_t i = 0; i < n; ++i) out[i] = orc_level_to_f32(k[i]);
}

static uint32_t f32_bits(float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    return u;
}

static float bits_f32(uint32_t u) {
    float x;
    memcpy(&x, &u, sizeof x);
    return x;
}

float orc_bf16_rne(float x) {
    /* bfloat16 keeps the top 16 bits of a float.  Round to nearest, ties to
     * even: look at the 16 dropped bits; above half rounds up, below half
     * rounds down, exactly half rounds to the even kept value. */
    uint32_t u = f32_bits(x);
    if (isnan(x)) return bits_f32((u | 0x00400000u) & 0xFFFF0000u);
    uint32_t kept = u & 0xFFFF0000u;
    uint32_t dropped = u & 0x0000FFFFu;
    uint32_t lsb = (u >> 16) & 1u;
    if (dropped > 0x8000u || (dropped == 0x8000u && lsb)) kept += 0x00010000u;
    return bits_f32(kept);
}

void orc_bf16_rne_array(const float *x, size_t n, float *out) {
    for (size_t i = 0; i < n; ++i) out[i] = orc_bf16_rne(x[i]);
}

int orc_out_size(int n, int k, int s, int p) {
    /* Convolution output length for input n, kernel k, stride s, padding p. */
    int num = n + 2 * p - k;
    if (num < 0) return 0;
    return num / s + 1;
}

void orc_layer_shape(const orc_net *net, int l, int *c, int *h, int *w) {
    int cc = net->in_c, hh = net->h, ww = net->w;
    for (int i = 0; i < l; ++i) {
        hh = orc_out_size(hh, net->k[i], net->s[i], net->p[i]);
        ww = orc_out_size(ww, net->k[i], net->s[i], net->p[i]);
        cc = net->cout[i];
    }
    *c = cc;
    *h = hh;
    *w = ww;
}

static int ceil_div(int a, int b) { return (a + b - 1) / b; }

static int net_ok(const orc_net *net) {
    if (net->n_conv < 1 || net->n_conv > ORC_MAX_LAYERS) return 0;
    if (net->in_c < 1 || net->h < 1 || net->w < 1 || net->n_out < 1) return 0;
    if (net->tile_h < 1 || net->tile_w < 1) return 0;
    int c = net->in_c;
    for (int i = 0; i < net->n_conv; ++i) {
        if (net->cin[i] != c || net->cout[i] < 1 || net->k[i] < 1 || net->s[i] < 1 ||
            net->p[i] < 0)
            return 0;
        c = net->cout[i];
    }
    int lc, lh, lw;
    orc_layer_shape(net, net->n_conv, &lc, &lh, &lw);
    return lh > 0 && lw > 0;
}

/* ---------------------------------------------------------- change sets */

void orc_diff(int c, int h, int w, const float *prev, const float *cur, uint8_t *d0) {
    /* A pixel changed iff any of its channels changed; "changed" is an exact
     * test on the stored float32 bits (Sec. 1: reuse where the input pixels
     * have not changed). */
    for (int y = 0; y < h; ++y)
        for (int x = 0; x < w; ++x) {
            int changed = 0;
            for (int ch = 0; ch < c; ++ch) {
                size_t i = ((size_t)ch * h + y) * w + x;
                if (f32_bits(prev[i]) != f32_bits(cur[i])) changed = 1;
            }
            d0[(size_t)y * w + x] = (uint8_t)changed;
        }
}

void orc_box_mask(int h, int w, int nb, const int32_t *boxes, uint8_t *d0) {
    /* Sec. 1: when the caller defines the change itself (occlusion), the
     * change set is known; it is the union of the given rectangles. */
    memset(d0, 0, (size_t)h * w);
    for (int b = 0; b < nb; ++b) {
        int y0 = boxes[4 * b + 0], x0 = boxes[4 * b + 1];
        int y1 = boxes[4 * b + 2], x1 = boxes[4 * b + 3];
        for (int y = 0; y < h; ++y)
            for (int x = 0; x < w; ++x)
                if (y >= y0 && y < y1 && x >= x0 && x < x1) d0[(size_t)y * w + x] = 1;
    }
}

void orc_dilate(int h, int w, const uint8_t *din, int k, int s, int p, uint8_t *dout) {
    /* Fig. 1 caption: an output pixel depends on the k x k input window that
     * starts at (s*y' - p, s*x' - p); it must be recomputed iff that window
     * holds a changed pixel.  Window cells outside the input are padding and
     * never change. */
    int ho = orc_out_size(h, k, s, p), wo = orc_out_size(w, k, s, p);
    for (int yo = 0; yo < ho; ++yo)
        for (int xo = 0; xo < wo; ++xo) {
            int dirty = 0;
            for (int ky = 0; ky < k; ++ky)
                for (int kx = 0; kx < k; ++kx) {
                    int y = s * yo - p + ky, x = s * xo - p + kx;
                    if (y >= 0 && y < h && x >= 0 && x < w && din[(size_t)y * w + x]) dirty = 1;
                }
            dout[(size_t)yo * wo + xo] = (uint8_t)dirty;
        }
}

void orc_tile_mask(int h, int w, const uint8_t *d, int tile_h, int tile_w, uint8_t *m) {
    /* Sec. 3: recompute small local areas.  Tile (ty, tx) covers rows
     * [ty*tile_h, (ty+1)*tile_h) and columns [tx*tile_w, (tx+1)*tile_w),
     * clipped to the grid; it is dirty iff one of its pixels is. */
    int th = ceil_div(h, tile_h), tw = ceil_div(w, tile_w);
    for (int ty = 0; ty < th; ++ty)
        for (int tx = 0; tx < tw; ++tx) {
            int dirty = 0;
            for (int y = ty * tile_h; y < (ty + 1) * tile_h && y < h; ++y)
                for (int x = tx * tile_w; x < (tx + 1) * tile_w && x < w; ++x)
                    if (d[(size_t)y * w + x]) dirty = 1;
            m[(size_t)ty * tw + tx] = (uint8_t)dirty;
        }
}

int orc_worklist(int n, int th, int tw, const uint8_t *masks, uint32_t *out) {
    /* Every dirty tile of one layer, ordered by tile row, then tile column,
     * then stream: tiles at the same position are adjacent. */
    int cnt = 0;
    for (int ty = 0; ty < th; ++ty)
        for (int tx = 0; tx < tw; ++tx)
            for (int s = 0; s < n; ++s)
                if (masks[((size_t)s * th + ty) * tw + tx])
                    out[cnt++] = ((uint32_t)s << 16) | ((uint32_t)ty << 8) | (uint32_t)tx;
    return cnt;
}

/* --------------------------------------------------------- convolution */

static float conv_pixel(int cin, int h, int w, const float *x, int k, int s, int p,
                        const float *wt, const float *b, int bf16, int co, int yo, int xo) {
    /* out[co][yo][xo] = ReLU(fl32(b[co] + sum_{ci,ky,kx} w[co][ci][ky][kx] *
     * x[ci][s*yo-p+ky][s*xo-p+kx])), zero outside the input. */
    double acc = (double)b[co];
    for (int ci = 0; ci < cin; ++ci)
        for (int ky = 0; ky < k; ++ky)
            for (int kx = 0; kx < k; ++kx) {
                int y = s * yo - p + ky, xx = s * xo - p + kx;
                if (y < 0 || y >= h || xx < 0 || xx >= w) continue;
                double wv = (double)wt[(((size_t)co * cin + ci) * k + ky) * k + kx];
                double xv = (double)x[((size_t)ci * h + y) * w + xx];
                acc += wv * xv;
            }
    float v = (float)acc;
    v = v > 0.0f ? v : 0.0f;
    if (bf16) v = orc_bf16_rne(v);
    return v;
}

void orc_conv2d_relu(int cin, int h, int w, const float *x, int cout, int k, int s, int p,
                     const float *wt, const float *b, int bf16, float *y) {
    int ho = orc_out_size(h, k, s, p), wo = orc_out_size(w, k, s, p);
    for (int co = 0; co < cout; ++co)
        for (int yo = 0; yo < ho; ++yo)
            for (int xo = 0; xo < wo; ++xo)
                y[((size_t)co * ho + yo) * wo + xo] =
                    conv_pixel(cin, h, w, x, k, s, p, wt, b, bf16, co, yo, xo);
}

void orc_conv2d_relu_tiles(int cin, int h, int w, const float *x, int cout, int k, int s, int p,
                           const float *wt, const float *b, int bf16,
                           const uint8_t *tmask, int tile_h, int tile_w, float *y) {
    int ho = orc_out_size(h, k, s, p), wo = orc_out_size(w, k, s, p);
    int tw = ceil_div(wo, tile_w);
    for (int yo = 0; yo < ho; ++yo)
        for (int xo = 0; xo < wo; ++xo) {
            if (!tmask[(size_t)(yo / tile_h) * tw + xo / tile_w]) continue;
            for (int co = 0; co < cout; ++co)
                y[((size_t)co * ho + yo) * wo + xo] =
                    conv_pixel(cin, h, w, x, k, s, p, wt, b, bf16, co, yo, xo);
        }
}

void orc_dense(int kdim, const float *a, int n, const float *wd, const float *bd, float *logits) {
    /* Sec. 2: the dense layer after the convolutions.  Input flattened in
     * (c, y, x) order. */
    for (int o = 0; o < n; ++o) {
        double acc = (double)bd[o];
        for (int j = 0; j < kdim; ++j) acc += (double)wd[(size_t)o * kdim + j] * (double)a[j];
        logits[o] = (float)acc;
    }
}

/* ------------------------------------------------------------ networks */

static float *rounded_copy(const float *src, size_t n) {
    float *dst = (float *)malloc(n * sizeof(float));
    if (!dst) return NULL;
    for (size_t i = 0; i < n; ++i) dst[i] = orc_bf16_rne(src[i]);
    return dst;
}

static size_t layer_elems(const orc_net *net, int l) {
    int c, h, w;
    orc_layer_shape(net, l, &c, &h, &w);
    return (size_t)c * h * w;
}

int orc_forward(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                const float *dense_w, const float *dense_b, int n, const float *x,
                float *const *acts, float *logits) {
    if (!net_ok(net)) return -1;
    int L = net->n_conv;
    const float *wl[ORC_MAX_LAYERS];
    float *owned[ORC_MAX_LAYERS + 1] = {0};
    const float *wd = dense_w;
    size_t kdim = layer_elems(net, L);
    for (int l = 0; l < L; ++l) {
        wl[l] = conv_w[l];
        if (net->bf16) {
            size_t cnt = (size_t)net->cout[l] * net->cin[l] * net->k[l] * net->k[l];
            owned[l] = rounded_copy(conv_w[l], cnt);
            wl[l] = owned[l];
        }
    }
    if (net->bf16) {
        owned[L] = rounded_copy(dense_w, (size_t)net->n_out * kdim);
        wd = owned[L];
    }
    size_t in_elems = layer_elems(net, 0);
    int status = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < n; ++i) {
        float *buf[ORC_MAX_LAYERS + 1];
        buf[0] = (float *)malloc(in_elems * sizeof(float));
        for (size_t e = 0; e < in_elems; ++e) {
            float v = x[(size_t)i * in_elems + e];
            buf[0][e] = net->bf16 ? orc_bf16_rne(v) : v;
        }
        for (int l = 0; l < L; ++l) {
            int c, h, w;
            orc_layer_shape(net, l, &c, &h, &w);
            buf[l + 1] = (float *)malloc(layer_elems(net, l + 1) * sizeof(float));
            orc_conv2d_relu(c, h, w, buf[l], net->cout[l], net->k[l], net->s[l], net->p[l],
                            wl[l], conv_b[l], net->bf16, buf[l + 1]);
            if (acts && acts[l]) {
                size_t e = layer_elems(net, l + 1);
                memcpy(acts[l] + (size_t)i * e, buf[l + 1], e * sizeof(float));
            }
        }
        orc_dense((int)kdim, buf[L], net->n_out, wd, dense_b, logits + (size_t)i * net->n_out);
        for (int l = 0; l <= L; ++l) free(buf[l]);
    }
    for (int l = 0; l <= L; ++l) free(owned[l]);
    return status;
}

int orc_masks(const orc_net *net, int n, const uint8_t *d0, uint8_t *const *d, uint8_t *const *m) {
    if (!net_ok(net)) return -1;
    int L = net->n_conv;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < n; ++i) {
        uint8_t *cur = NULL;
        int c, h, w;
        orc_layer_shape(net, 0, &c, &h, &w);
        cur = (uint8_t *)malloc((size_t)h * w);
        memcpy(cur, d0 + (size_t)i * h * w, (size_t)h * w);
        for (int l = 0; l <= L; ++l) {
            orc_layer_shape(net, l, &c, &h, &w);
            if (l > 0) {
                int ph, pw, pc;
                orc_layer_shape(net, l - 1, &pc, &ph, &pw);
                uint8_t *nxt = (uint8_t *)malloc((size_t)h * w);
                orc_dilate(ph, pw, cur, net->k[l - 1], net->s[l - 1], net->p[l - 1], nxt);
                free(cur);
                cur = nxt;
            }
            if (d && d[l]) memcpy(d[l] + (size_t)i * h * w, cur, (size_t)h * w);
            int th = ceil_div(h, net->tile_h), tw = ceil_div(w, net->tile_w);
            orc_tile_mask(h, w, cur, net->tile_h, net->tile_w, m[l] + (size_t)i * th * tw);
        }
        free(cur);
    }
    return 0;
}

int orc_reuse_step(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                   const float *dense_w, const float *dense_b, const float *x,
                   const uint8_t *d0_given, int primed, float *const *cache, float *logits) {
    if (!net_ok(net)) return -1;
    int L = net->n_conv;
    int c0, h0, w0;
    orc_layer_shape(net, 0, &c0, &h0, &w0);
    size_t px = (size_t)h0 * w0;
    uint8_t *d = (uint8_t *)malloc(px);
    if (!primed) memset(d, 1, px);
    else if (d0_given) memcpy(d, d0_given, px);
    else orc_diff(c0, h0, w0, cache[0], x, d);
    /* The cached input takes the new values at the changed pixels. */
    for (int ch = 0; ch < c0; ++ch)
        for (size_t q = 0; q < px; ++q)
            if (d[q]) cache[0][(size_t)ch * px + q] = x[(size_t)ch * px + q];
    for (int l = 1; l <= L; ++l) {
        int pc, ph, pw, c, h, w;
        orc_layer_shape(net, l - 1, &pc, &ph, &pw);
        orc_layer_shape(net, l, &c, &h, &w);
        uint8_t *dn = (uint8_t *)malloc((size_t)h * w);
        orc_dilate(ph, pw, d, net->k[l - 1], net->s[l - 1], net->p[l - 1], dn);
        free(d);
        d = dn;
        int th = ceil_div(h, net->tile_h), tw = ceil_div(w, net->tile_w);
        uint8_t *tm = (uint8_t *)malloc((size_t)th * tw);
        orc_tile_mask(h, w, d, net->tile_h, net->tile_w, tm);
        const float *in = cache[l - 1];
        float *rounded_in = NULL;
        if (l == 1 && net->bf16) {
            rounded_in = rounded_copy(cache[0], (size_t)pc * ph * pw);
            in = rounded_in;
        }
        orc_conv2d_relu_tiles(pc, ph, pw, in, c, net->k[l - 1], net->s[l - 1], net->p[l - 1],
                              conv_w[l - 1], conv_b[l - 1], net->bf16, tm, net->tile_h,
                              net->tile_w, cache[l]);
        free(rounded_in);
        free(tm);
    }
    free(d);
    orc_dense((int)layer_elems(net, L), cache[L], net->n_out, dense_w, dense_b, logits);
    return 0;
}

/* ------------------------------------------------------------- training */

/* Sec. 2: the policy is trained with REINFORCE.  For input i with logits z,
 * sampled action a and return G, the loss is -G log softmax(z)[a]; its
 * derivative with respect to z[o] is G (softmax(z)[o] - [o == a]). */
void orc_reinforce_dlogits(int n, int n_out, const float *logits, const int32_t *actions,
                           const float *returns, float *g) {
    for (int i = 0; i < n; ++i) {
        const float *z = logits + (size_t)i * n_out;
        double zmax = z[0];
        for (int o = 1; o < n_out; ++o)
            if (z[o] > zmax) zmax = z[o];
        double den = 0.0;
        for (int o = 0; o < n_out; ++o) den += exp((double)z[o] - zmax);
        for (int o = 0; o < n_out; ++o) {
            double p = exp((double)z[o] - zmax) / den;
            double onehot = (o == actions[i]) ? 1.0 : 0.0;
            g[(size_t)i * n_out + o] = (float)((double)returns[i] * (p - onehot));
        }
    }
}

static double conv_sum(int cin, int h, int w, const float *x, int k, int s, int p,
                       const float *wt, const float *b, int co, int yo, int xo) {
    /* b[co] + sum_{ci,ky,kx} w[co][ci][ky][kx] * x[ci][s*yo-p+ky][s*xo-p+kx] */
    double acc = (double)b[co];
    for (int ci = 0; ci < cin; ++ci)
        for (int ky = 0; ky < k; ++ky)
            for (int kx = 0; kx < k; ++kx) {
                int y = s * yo - p + ky, xx = s * xo - p + kx;
                if (y < 0 || y >= h || xx < 0 || xx >= w) continue;
                acc += (double)wt[(((size_t)co * cin + ci) * k + ky) * k + kx] *
                       (double)x[((size_t)ci * h + y) * w + xx];
            }
    return acc;
}

int orc_forward_preact(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                       const float *x, float *const *z) {
    /* One input: each layer's pre-activation fl32(b + sum w a) (before the
     * ReLU), with the layer inputs a the float32 activations of orc_forward. */
    if (!net_ok(net) || net->bf16) return -1;
    int L = net->n_conv;
    float *a = (float *)malloc(layer_elems(net, 0) * sizeof(float));
    memcpy(a, x, layer_elems(net, 0) * sizeof(float));
    for (int l = 0; l < L; ++l) {
        int c, h, w, co, ho, wo;
        orc_layer_shape(net, l, &c, &h, &w);
        orc_layer_shape(net, l + 1, &co, &ho, &wo);
        float *an = (float *)malloc((size_t)co * ho * wo * sizeof(float));
#pragma omp parallel for schedule(dynamic, 1)
        for (int o = 0; o < co; ++o)
            for (int yo = 0; yo < ho; ++yo)
                for (int xo = 0; xo < wo; ++xo) {
                    float v = (float)conv_sum(c, h, w, a, net->k[l], net->s[l], net->p[l], conv_w[l],
                                              conv_b[l], o, yo, xo);
                    z[l][((size_t)o * ho + yo) * wo + xo] = v;
                    an[((size_t)o * ho + yo) * wo + xo] = v > 0.0f ? v : 0.0f;
                }
        free(a);
        a = an;
    }
    free(a);
    return 0;
}

int orc_backward(const orc_net *net, const float *const *conv_w, const float *const *conv_b,
                 const float *dense_w, const float *dense_b, int n, const float *x, const float *g,
                 float *const *dconv_w, float *const *dconv_b, float *ddense_w, float *ddense_b) {
    /* Backpropagation of J = sum_i sum_o g[i][o] logits[i][o] through the
     * network of orc_forward (float32 activations a_l = ReLU(fl32(z_l))),
     * summed over the n inputs x [n][in_c][h][w].  Chain rule, all in double:
     *   dbd[o]      = sum_i g[i][o]
     *   dWd[o][j]   = sum_i g[i][o] a_L[i][j]
     *   da_L[i][j]  = sum_o Wd[o][j] g[i][o]
     *   dz_l        = da_l where a_l > 0, else 0   (ReLU derivative, 0 at the kink)
     *   dW_l[co][ci][ky][kx] = sum_i sum_{yo,xo} dz_l[co][yo][xo] a_{l-1}[ci][s yo-p+ky][s xo-p+kx]
     *   db_l[co]    = sum_i sum_{yo,xo} dz_l[co][yo][xo]
     *   da_{l-1}[ci][y][x] = sum over (co, ky, kx, yo, xo) with s yo-p+ky = y and
     *                        s xo-p+kx = x of W_l[co][ci][ky][kx] dz_l[co][yo][xo]
     * Each gradient is rounded once to float32.  Float32 weights only. */
    if (!net_ok(net) || net->bf16) return -1;
    int L = net->n_conv;
    size_t kdim = layer_elems(net, L);
    size_t nw[ORC_MAX_LAYERS];
    double *gw[ORC_MAX_LAYERS], *gb[ORC_MAX_LAYERS];
    for (int l = 0; l < L; ++l) {
        nw[l] = (size_t)net->cout[l] * net->cin[l] * net->k[l] * net->k[l];
        gw[l] = (double *)calloc(nw[l], sizeof(double));
        gb[l] = (double *)calloc((size_t)net->cout[l], sizeof(double));
    }
    double *gwd = (double *)calloc((size_t)net->n_out * kdim, sizeof(double));
    double *gbd = (double *)calloc((size_t)net->n_out, sizeof(double));
    float *act[ORC_MAX_LAYERS + 1];
    for (int l = 0; l <= L; ++l) act[l] = (float *)malloc(layer_elems(net, l) * sizeof(float));
    double *da = (double *)malloc(kdim * sizeof(double));
    for (int i = 0; i < n; ++i) {
        const float *gi = g + (size_t)i * net->n_out;
        /* forward: the float32 activations of every layer */
        memcpy(act[0], x + (size_t)i * layer_elems(net, 0), layer_elems(net, 0) * sizeof(float));
        for (int l = 0; l < L; ++l) {
            int c, h, w, co, ho, wo;
            orc_layer_shape(net, l, &c, &h, &w);
            orc_layer_shape(net, l + 1, &co, &ho, &wo);
#pragma omp parallel for schedule(dynamic, 1)
            for (int o = 0; o < co; ++o)
                for (int yo = 0; yo < ho; ++yo)
                    for (int xo = 0; xo < wo; ++xo)
                        act[l + 1][((size_t)o * ho + yo) * wo + xo] =
                            conv_pixel(c, h, w, act[l], net->k[l], net->s[l], net->p[l], conv_w[l],
                                       conv_b[l], 0, o, yo, xo);
        }
        /* dense layer */
        for (int o = 0; o < net->n_out; ++o) gbd[o] += (double)gi[o];
#pragma omp parallel for schedule(static)
        for (size_t j = 0; j < kdim; ++j) {
            double s = 0.0;
            for (int o = 0; o < net->n_out; ++o) {
                gwd[(size_t)o * kdim + j] += (double)gi[o] * (double)act[L][j];
                s += (double)dense_w[(size_t)o * kdim + j] * (double)gi[o];
            }
            da[j] = s;
        }
        /* conv layers, last to first; da holds dJ/da_l on entry */
        double *da_cur = da;
        for (int l = L - 1; l >= 0; --l) {
            int c, h, w, co, ho, wo;
            orc_layer_shape(net, l, &c, &h, &w);
            orc_layer_shape(net, l + 1, &co, &ho, &wo);
            int k = net->k[l], s = net->s[l], p = net->p[l];
            size_t nout = (size_t)co * ho * wo;
            double *dz = (double *)malloc(nout * sizeof(double));
            for (size_t e = 0; e < nout; ++e) dz[e] = act[l + 1][e] > 0.0f ? da_cur[e] : 0.0;
#pragma omp parallel for schedule(dynamic, 1)
            for (int o = 0; o < co; ++o)
                for (int yo = 0; yo < ho; ++yo)
                    for (int xo = 0; xo < wo; ++xo) {
                        double d = dz[((size_t)o * ho + yo) * wo + xo];
                        gb[l][o] += d;
                        for (int ci = 0; ci < c; ++ci)
                            for (int ky = 0; ky < k; ++ky)
                                for (int kx = 0; kx < k; ++kx) {
                                    int y = s * yo - p + ky, xx = s * xo - p + kx;
                                    if (y < 0 || y >= h || xx < 0 || xx >= w) continue;
                                    gw[l][(((size_t)o * c + ci) * k + ky) * k + kx] +=
                                        d * (double)act[l][((size_t)ci * h + y) * w + xx];
                                }
                    }
            double *da_prev = NULL;
            if (l > 0) {
                da_prev = (double *)malloc((size_t)c * h * w * sizeof(double));
#pragma omp parallel for schedule(dynamic, 1)
                for (int ci = 0; ci < c; ++ci)
                    for (int y = 0; y < h; ++y)
                        for (int xx = 0; xx < w; ++xx) {
                            double acc = 0.0;
                            for (int o = 0; o < co; ++o)
                                for (int ky = 0; ky < k; ++ky)
                                    for (int kx = 0; kx < k; ++kx) {
                                        int ny = y + p - ky, nx = xx + p - kx;
                                        if (ny < 0 || nx < 0 || ny % s || nx % s) continue;
                                        int yo = ny / s, xo = nx / s;
                                        if (yo >= ho || xo >= wo) continue;
                                        acc += (double)conv_w[l][(((size_t)o * c + ci) * k + ky) * k + kx] *
                                               dz[((size_t)o * ho + yo) * wo + xo];
                                    }
                            da_prev[((size_t)ci * h + y) * w + xx] = acc;
                        }
            }
            free(dz);
            if (da_cur != da) free(da_cur);
            da_cur = da_prev;
        }
    }
    for (int l = 0; l < L; ++l) {
        for (size_t e = 0; e < nw[l]; ++e) dconv_w[l][e] = (float)gw[l][e];
        for (int o = 0; o < net->cout[l]; ++o) dconv_b[l][o] = (float)gb[l][o];
        free(gw[l]);
        free(gb[l]);
    }
    for (size_t e = 0; e < (size_t)net->n_out * kdim; ++e) ddense_w[e] = (float)gwd[e];
    for (int o = 0; o < net->n_out; ++o) ddense_b[o] = (float)gbd[o];
    free(gwd);
    free(gbd);
    free(da);
    for (int l = 0; l <= L; ++l) free(act[l]);
    return 0;
}
