// Training support (Sec. 2: the policy is trained with REINFORCE): argument
// blocks and launchers of the backward and update kernels (rn_train.hip).
// Float32 nets of 3x3 stride-1 pad-1 layers.  Not part of the public ABI.
#pragma once

#include "rn_internal.hpp"

namespace rn {

// Dense-head backward for a batch of n streams (one block per tile position
// of the last layer): gwd/gbd (+)= the head's weight and bias gradients and
// dz = the gradient at the last layer's pre-activations (ReLU derivative
// applied), [n][ntiles][16][C] by batch index.
struct HeadBwdArgs {
    int n, n_out, C, ntiles, TW, H, W;
    size_t K;                     // head inputs per stream (ntiles * 16 * C)
    const int32_t *ids;           // [n] slots
    const float *act;             // last-layer cache [S][ntiles][16][C]
    size_t act_stride;
    const float *wd;              // dense weights in the cache order [n_out][K], 0 at padded pixels
    const float *g;               // [n][n_out] dJ/dlogits
    float *dz;                    // [n][ntiles][16][C]
    float *gwd;                   // [n_out][C][H][W]
    float *gbd;                   // [n_out]
    int accumulate;
};

// One conv layer l's backward: dz_in = dJ/dz_l [n][ntiles][16][cz]; act_prev
// the layer-(l-1) activations (a tiled cache, or the float32 input planes for
// layer 1); dW (split over teams of blocks into part, then reduced) and, for
// l >= 2, dz_out = dJ/dz_{l-1} = (W_l^T * dz_l) where a_{l-1} > 0.
struct BwdArgs {
    int n, H, W, TH, TW, ntiles;
    int ca, cz;                   // channels of a_{l-1} and of layer l
    const int32_t *ids;           // [n] slots
    const float *dz_in;
    const float *act_prev;
    size_t prev_stride;           // elements per slot of act_prev
    int first;                    // act_prev is the input cache (planar; a ring of 4 frames when stacking)
    int stack, cin0;              // layer 1: frames stacked, channels per frame
    const int32_t *ring_head;
    float *dz_out;                // l >= 2
    const float *wt;              // dx weights (pack_dx_weights)
    float *part;                  // [cz][9 ca + 1][teams]
    int teams;
    float *gw, *gb;               // OIHW [cz][ca][3][3], [cz]
    int accumulate;
};

// Plain SGD step applied in place to one packed weight buffer: every element
// that holds weight v of the natural layout becomes fl(v - fl(lr * g)), with g
// the gradient of that weight, so each packed copy stays the packing of the
// updated weights.  With assign set, the element becomes g itself (and a
// padding element 0): the packing of the weights g, written on the device.
// kind: what layout dst has.
enum SgdKind { SGD_PLAIN = 0, SGD_FIRST = 1, SGD_MFMA = 2, SGD_DENSE = 3, SGD_TILE_HEAD = 4, SGD_DX = 5, SGD_TILE_PART = 6 };
struct SgdArgs {
    float *dst;
    size_t count;                 // elements of dst
    int kind;
    const float *g;               // gradient (or, with assign, the weights) in the natural layout (OIHW, or [n_out][C][H][W])
    float lr;
    int assign;
    int cin, cout;                // conv layers
    int C, H, W, TW, ntiles, n_out;   // dense / tile head / tile partials: last layer
    size_t K;
};

bool train_shapes_supported(int ca, int cz, bool first);
bool train_dx_supported(int cz, int ca);
size_t dx_weights_elems(int cz, int ca);
// W_l (OIHW, cz outputs, ca inputs) -> the B operand of the dx product.
void pack_dx_weights(const float *oihw, int ca, int cz, float *dst);
// Teams of the split-K dW product for n streams of ntiles tiles, and the
// partial-sum elements they need.
int bwd_dw_teams(int ca, int cz, bool first, int n, int ntiles, int cus);
size_t bwd_dw_part_elems(int ca, int cz, int teams);

hipError_t launch_reinforce(int n, int n_out, const float *logits, const int32_t *actions, const float *returns,
                            float *g, hipStream_t s);
hipError_t launch_bwd_head(const HeadBwdArgs &a, hipStream_t s);
hipError_t launch_bwd_dw(const BwdArgs &a, int cus, hipStream_t s);   // partials, then the reduction
hipError_t launch_bwd_dx(const BwdArgs &a, int cus, hipStream_t s);
hipError_t launch_sgd(const SgdArgs &a, hipStream_t s);
hipError_t launch_unprime(int32_t *primed, int S, hipStream_t s);

}  // namespace rn
