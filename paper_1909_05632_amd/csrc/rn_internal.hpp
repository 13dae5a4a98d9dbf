// Internal declarations shared by the reuse_net host planner and its kernels.
// Not part of the public ABI (that is include/reuse_net.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include <string>
#include <vector>

#include "reuse_net.h"

namespace rn {

constexpr int kTile = 4;          // dirty-tile edge on every layer
constexpr int kTilePx = kTile * kTile;
constexpr int kHeadMaxOut = 64;

// Geometry shared by the mask kernels.  Layer l's grid is Hl[l] x Wl[l]
// (layer 0: the input); a 3x3 stride-1 pad-1 layer keeps its input grid, other
// layers shrink it (pad <= (k - 1) / 2).
struct MaskGeom {
    int L;                        // conv layers
    int H, W, WW;                 // input rows, columns, 64-bit words per mask row
    int TH, TW, TMW;              // input tile rows, tile columns, 64-bit words per tile mask
    int cin;                      // channels per frame
    int stack;                    // 1, or 4 (ring of the last 4 frames)
    int dil;                      // every layer 3x3/1/1: layer l's mask is the change set dilated by l (set by the launcher)
    int Hl[RN_MAX_CONV + 1], Wl[RN_MAX_CONV + 1], WWl[RN_MAX_CONV + 1];
    int THl[RN_MAX_CONV + 1], TWl[RN_MAX_CONV + 1], TMWl[RN_MAX_CONV + 1];
    int ks[RN_MAX_CONV], st[RN_MAX_CONV], pd[RN_MAX_CONV];   // kernel, stride, pad of layer l + 1
    uint64_t *pmask[RN_MAX_CONV + 1];   // [S][Hl][WWl] per layer
    uint64_t *tmask[RN_MAX_CONV + 1];   // [S][TMWl] per layer
    int32_t *tpfx[RN_MAX_CONV + 1];     // [S][TMWl] per layer 1..L: dirty tiles in the slot's earlier tile words (NULL: not kept)
};

// Per-step inputs of the mask kernel.
struct MaskArgs {
    int n;
    const int32_t *ids;           // [n] slots, or NULL: slot i for batch index i
    const void *frames;           // [n][cin][H][W]
    int frame_u8;                 // 1: uint8 levels, 0: float32
    const int32_t *boxes;         // NULL: diff
    const int32_t *box_off;       // [n+1]
    int force_all;                // 1: every pixel changed (dense path)
    const float *lut;             // [256] level -> float32
    float *xin;                   // [S][stack][cin][H][W] input cache (ring for stack=4)
    int32_t *ring_head;           // [S] newest ring position (stack=4)
    uint64_t *dring;              // [S][stack][H][WW] last single-frame change masks (stack=4)
    int32_t *primed;              // [S]
    int32_t *nchg;                // [n] changed pixels
    int32_t *ntile;               // [n][L+1] dirty tiles per layer
    // Work lists of layers 1..L (as CompactArgs); with one stream the mask
    // kernel writes them itself (fuse_lists, set by launch_masks) and no
    // compaction launch follows.
    uint32_t *wl[RN_MAX_CONV + 1];
    uint32_t *wls[RN_MAX_CONV + 1];
    int32_t *cnt;
    int fuse_lists;
};

struct CompactArgs {
    int n, L;
    int TWl[RN_MAX_CONV + 1], TMWl[RN_MAX_CONV + 1], ntl[RN_MAX_CONV + 1];   // per layer
    const int32_t *ids;           // [n] slots, or NULL: slot i for batch index i
    const int32_t *ntile;         // [n][L+1]
    uint64_t *tmask[RN_MAX_CONV + 1];
    const int32_t *tpfx[RN_MAX_CONV + 1];   // per-slot word prefixes written by k_masks
    uint32_t *wl[RN_MAX_CONV + 1];  // entries i << 16 | ty << 8 | tx (batch index i)
    uint32_t *wls[RN_MAX_CONV + 1]; // the same list as slot << 16 | ty << 8 | tx, for the kernels
    int32_t *cnt;                 // [L+1]
    size_t cap[RN_MAX_CONV + 1];  // entries each layer's list can hold
};

// Masks and work lists of n variants straight from their boxes (variant i's
// change set is the union of boxes [box_off[i], box_off[i+1])).  Masks are
// indexed by variant.  A variant with more than vmax (> 0) dirty tiles in a
// layer 1..L is left out of every list; vmap[l][i][t] receives the list index
// of tile t of variant i (written for listed tiles only).
struct VarMaskArgs {
    int n, L, H, W, WW, TH, TW, TMW, ntiles, nch, vmax;
    int R[RN_MAX_CONV + 1];       // growth radius of layer l's change set (R[0] = 0)
    const int32_t *boxes, *box_off;
    uint64_t *pmask[RN_MAX_CONV + 1];   // [n][H][WW]
    uint64_t *tmask[RN_MAX_CONV + 1];   // [n][TMW]
    int32_t *nchg;                // [n]
    int32_t *ntile;               // [n][L+1]
    uint64_t *bits[RN_MAX_CONV + 1];    // layers 1..L: [ntiles][nch] listed variants per position
    int32_t *pos_cnt;             // [L][ntiles] listed entries per position
    uint32_t *wl[RN_MAX_CONV + 1];
    int32_t *vmap[RN_MAX_CONV + 1];     // [n][ntiles]
    int32_t *cnt;
    size_t cap;
};

struct ConvArgs {
    const uint32_t *wl;           // work list of this layer, slot-encoded (NULL: dense mode)
    const int32_t *cnt;           // device count of this layer
    const int32_t *ids;
    const void *in;               // previous layer cache (layer 1: float32 input ring)
    void *out;                    // this layer's cache [S][TH][TW][16][cout]
    const void *w;                // packed weights
    const float *bias;            // [cout]
    const int32_t *ring_head;     // stack=4 only
    int H, W, TH, TW;             // this layer's output grid and its tile grid
    int cin, cout;
    int stack;
    int Hin, Win, TWin;           // input grid (layers other than 3x3 stride 1 pad 1)
    int pad;
    size_t in_stride, out_stride; // elements per slot
    int dense_n;                  // dense mode (wl == NULL): every tile of streams 0..dense_n-1
    int max_tiles;                // host bound on the tiles of this launch (sizes the grid)
    // Tile-partial dense head fused into the last layer's epilogue (n_out > 0):
    // hpart[slot][tile][o] = sum over the tile's outputs of hw * activation.
    int n_out;
    const float *hw;              // [n_out][TH*TW][16*cout] in the epilogue's fragment order
    float *hpart;                 // [S][TH*TW][n_out]
    // Layer 1 folded into this layer's halo staging (this is layer 2 and the
    // input has one channel): `in` is the float32 input cache and the halo's
    // layer-1 activations are computed from the input patch with w1/b1.
    int fuse_first;
    const float *w1;              // layer-1 weights, [k][c1] (first-layer packing, one input channel)
    const float *b1;              // [c1]
    // Variant mode (kernels instantiated with VAR): the work items are
    // i << 16 | ty << 8 | tx for variant i of base slot vbase, and item t of
    // the list writes its outputs to row t of this layer's overlay instead of
    // a cache.  A variant's layer-(l-1) tile is its own overlay row where its
    // tile mask has the tile, else the base slot's cached tile.
    int vbase;
    int vcin;                     // input channels of the frames (layer-1 reads)
    int WW;                       // 64-bit words per pixel-mask row
    const uint64_t *vtm_in;       // layer l-1 tile masks [n][TMW]
    const int32_t *vmap_in;       // layer l-1 list index of (variant, tile) [n][TH*TW]
    const void *vov_in;           // layer l-1 overlay [list index][16][cin]
    void *vov_out;                // this layer's overlay [list index][16][cout] (NULL: not stored)
    float *vhpart;                // head partials [list index][n_out]
    const uint64_t *vpm0;         // layer-0 change masks [n][H][WW]: input pixels taken from the frame
    const void *vframes;          // [1 or n][vcin][H][W]
    int vframe_u8;
    int vframe_shared;            // 1: every variant reads frame 0
    const float *lut;             // [256] level -> float32
};

// Dense path: copy the frames into the input cache and mark the slots primed.
struct PrimeArgs {
    int n, L, cin, stack, H, W, WW;
    int ntl[RN_MAX_CONV + 1];     // tiles per layer
    const int32_t *ids;
    const void *frames;
    int frame_u8;
    const float *lut;
    float *xin;
    int32_t *ring_head;
    uint64_t *dring;
    int32_t *primed;
    int32_t *nchg;
    int32_t *ntile;
    size_t dring_words;           // per slot (stack = 4)
};

// Sum of the per-tile head partials: logits[i][o] = bd[o] + sum_t hpart[ids[i]][t][o].
struct TileHeadArgs {
    int n, n_out, ntiles;
    const int32_t *ids;           // [n] slots, or NULL: slot i for batch index i
    const float *hpart;
    const float *bias;
    float *logits;
    // Variant mode (var = 1): tile t of variant i takes its partials from
    // vhpart[vmap[i][t]] where the variant recomputed it (vtm), else from the
    // base slot; variants left out of the lists (more than vmax dirty tiles in
    // a layer) and variants of an unprimed base get NaN logits.
    int var, vbase, L, TMW, vmax;
    const uint64_t *vtm;          // [n][TMW] last layer
    const int32_t *vmap;          // [n][ntiles] last layer
    const float *vhpart;          // [list index][n_out]
    const int32_t *ntile;         // [n][L+1]
    const int32_t *primed;        // [S]
};

struct HeadArgs {
    int n, n_out;
    const int32_t *ids;
    const void *act;              // last cache [S][K]
    const void *w;                // [n_out][K] tiled order, zero at padded pixels
    const float *bias;            // [n_out]
    float *part;                  // [nsplit][n][n_out]
    float *logits;                // [n][n_out]
    size_t K;                     // elements per slot
    int nsplit;
    size_t chunk;                 // elements per split (multiple of 4)
};

// Launchers (each returns the hipGetLastError of its launch).
// Sets *fused when the kernel also wrote the work lists (one stream, lists
// given in a.wl / a.wls / a.cnt): the caller then skips launch_compact.
hipError_t launch_masks(const MaskGeom &g, const MaskArgs &a, int cus, hipStream_t s, bool *fused);
size_t masks_lds_bytes(int H, int WW, int L, int TMW);   // dynamic LDS of the layer-by-layer mask kernel
constexpr size_t kMasksLdsMax = 160 * 1024 - 1024;       // per block, less the static arrays
hipError_t launch_prime(const PrimeArgs &a, hipStream_t s);
hipError_t launch_tile_head(const TileHeadArgs &a, hipStream_t s);
size_t tile_head_w_elems(int ntiles, int cout, int n_out);
void pack_tile_head(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, float *dst);
hipError_t launch_compact(const CompactArgs &a, hipStream_t s);
hipError_t launch_var_masks(const VarMaskArgs &a, hipStream_t s);
hipError_t launch_var_lists(const VarMaskArgs &a, hipStream_t s);
// Conv launchers: list mode (a.wl set), dense mode (a.wl NULL), or variant
// mode (var = true, a.wl set).
hipError_t launch_conv_first(const ConvArgs &a, rn_dtype dt, int grid, hipStream_t s, bool var = false);
hipError_t launch_conv_mfma(const ConvArgs &a, rn_dtype dt, int grid, hipStream_t s, bool var = false);
bool conv_mfma_supported(int cin, int cout, rn_dtype dt);
bool conv_first_supported(int cin, int cout, rn_dtype dt);
// General layers (any k <= 8, stride 1, 2 or 4, pad <= (k - 1) / 2; float32):
// first = the layer reads the input frames.
bool conv_gen_supported(int k, int s, int cin, int cout, bool first);
size_t conv_gen_packed_elems(int k, int cin, int cout);
void pack_conv_gen(const float *oihw, int k, int cin, int cout, float *dst);
hipError_t launch_conv_gen(const ConvArgs &a, int k, int s, bool first, int cus, hipStream_t st);
bool conv_fused_first_supported(int c1, int c2, rn_dtype dt);
bool conv_mfma_bf16_supported(int cin, int cout);
bool conv_first_bf16_supported(int cin, int cout);
hipError_t launch_conv_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var = false);
hipError_t launch_conv_first_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var = false);
void pack_conv_mfma_bf16(const float *oihw, int cin, int cout, void *dst);
float round_bf16_host(float v);
uint16_t bf16_bits_host(float v);
// bf16 tile head partials (last layer bf16, tile head): hw is the packed bf16
// weights of pack_tile_part_bf16, `in` the last cache, cout its channels.
bool tile_part_bf16_supported(int C);
size_t tile_part_bf16_elems(int ntiles, int C, int n_out);
void pack_tile_part_bf16(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, uint16_t *dst);
hipError_t launch_tile_part_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var = false);
// float32 tile partials by position for a last layer on the staged conv
// kernel (its epilogue then computes none): hw the packed weights of
// pack_tile_part_f32, `in` the last cache, cout its channels.
bool conv_mfma_is_staged(int cin, int cout);
bool tile_part_f32_supported(int C);
size_t tile_part_f32_elems(int ntiles, int C, int n_out);
void pack_tile_part_f32(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, float *dst);
hipError_t launch_tile_part_f32(const ConvArgs &a, int cus, hipStream_t s, bool var = false);
hipError_t launch_head(const HeadArgs &a, rn_dtype dt, hipStream_t s);
int head_streams_per_block(int n_out);

// Packed weight sizes (elements of the act dtype) for the kernels' layouts.
size_t conv_first_packed_elems(int cin, int cout);
size_t conv_mfma_packed_elems(int cin, int cout, rn_dtype dt);
void pack_conv_first(const float *oihw, int cin, int cout, rn_dtype dt, void *dst);
void pack_conv_mfma(const float *oihw, int cin, int cout, rn_dtype dt, void *dst);

}  // namespace rn
