// Dense head (Sec. 2: the dense layer after the two conv layers):
//   logits[i][o] = bd[o] + sum_j Wd[o][j] * a_L[i][j].
// The weights were permuted at create into the cache's tiled order, with zeros
// at the padded pixels of ragged edge tiles, so the head streams each stream's
// whole cache contiguously.  It reads all of a_L every step: the kernel is
// HBM-bound.
//
// Split-K: block (split, stream group) reduces one K-chunk for SG streams,
// keeping the chunk's weights in registers across the streams of the group.
// Partials go to [split][stream][o]; a second kernel adds them in split order.
// Both orders are fixed, so the result is deterministic and a step on an
// unchanged cache reproduces the previous logits bit for bit.
#include "rn_device.hpp"

namespace rn {
namespace {

constexpr int kThreads = 256;

using dev::floatx4;
using dev::XcdRange;
using dev::TileRef;
using dev::xcd_range;
using dev::item_ref;
using dev::item_word;
using dev::work_count;
using dev::lds_barrier;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Four consecutive activations as float32 (float32 or bf16 caches).
template <typename AT>
__device__ inline float4 load_act4(const AT *p);
template <>
__device__ inline float4 load_act4<float>(const float *p) { return *reinterpret_cast<const float4 *>(p); }
template <>
__device__ inline float4 load_act4<uint16_t>(const uint16_t *p) {
    const uint2 q = *reinterpret_cast<const uint2 *>(p);
    return make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xFFFF0000u),
                       __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xFFFF0000u));
}

template <int NO, int SG, typename AT>
__global__ __launch_bounds__(kThreads) void k_head_partial_f32(HeadArgs a) {
    __shared__ float red[kThreads / 64][SG * NO];
    const int split = blockIdx.x, g = blockIdx.y;
    const size_t k0 = (size_t)split * a.chunk;
    const size_t k1 = min(k0 + a.chunk, a.K);
    const float *W = static_cast<const float *>(a.w);
    const AT *act = static_cast<const AT *>(a.act);
    const AT *rows[SG];
    int ns = 0;
#pragma unroll
    for (int s = 0; s < SG; ++s) {
        const int i = g * SG + s;
        rows[s] = nullptr;
        if (i < a.n) {
            rows[s] = act + (size_t)a.ids[i] * a.K;
            ns = s + 1;
        }
    }
    float acc[SG][NO];
#pragma unroll
    for (int s = 0; s < SG; ++s)
#pragma unroll
        for (int o = 0; o < NO; ++o) acc[s][o] = 0.f;

    for (size_t k = k0 + 4 * (size_t)threadIdx.x; k < k1; k += 4 * kThreads) {
        float4 wv[NO];
#pragma unroll
        for (int o = 0; o < NO; ++o) wv[o] = *reinterpret_cast<const float4 *>(W + (size_t)o * a.K + k);
#pragma unroll
        for (int s = 0; s < SG; ++s) {
            if (s < ns) {
                const float4 av = load_act4<AT>(rows[s] + k);
#pragma unroll
                for (int o = 0; o < NO; ++o) {
                    float t = acc[s][o];
                    t = fmaf(av.x, wv[o].x, t);
                    t = fmaf(av.y, wv[o].y, t);
                    t = fmaf(av.z, wv[o].z, t);
                    t = fmaf(av.w, wv[o].w, t);
                    acc[s][o] = t;
                }
            }
        }
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int s = 0; s < SG; ++s)
#pragma unroll
        for (int o = 0; o < NO; ++o) {
            float v = acc[s][o];
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[wave][s * NO + o] = v;
        }
    __syncthreads();
    for (int j = threadIdx.x; j < SG * NO; j += kThreads) {
        const int s = j / NO, o = j - s * NO;
        const int i = g * SG + s;
        if (i < a.n) {
            float v = red[0][j];
            for (int w = 1; w < kThreads / 64; ++w) v += red[w][j];
            a.part[((size_t)split * a.n + i) * a.n_out + o] = v;
        }
    }
}

// One wave per (stream, logit): lanes add the split partials, then a fixed
// butterfly adds the lanes.
__global__ __launch_bounds__(kThreads) void k_head_reduce(HeadArgs a) {
    const int lane = threadIdx.x & 63;
    const int j = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (j >= a.n * a.n_out) return;
    const int o = j % a.n_out;
    float v = 0.f;
    for (int s = lane; s < a.nsplit; s += 64) v += a.part[(size_t)s * a.n * a.n_out + j];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if (lane == 0) a.logits[j] = v + a.bias[o];
}

// Tile-partial head: logits[i][o] = bd[o] + sum over tiles of the cached
// per-tile partials of stream i, added in a fixed order: thread j adds tiles
// j, j + 256, ... (each tile's NO partials are one contiguous read), then a
// fixed butterfly per wave and the 4 waves in order.
template <int NO>
__global__ __launch_bounds__(kThreads) void k_tile_head(TileHeadArgs a) {
    __shared__ float red[kThreads / 64][NO];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = blockIdx.x;
    const float *P = a.hpart + (size_t)(a.ids ? a.ids[i] : i) * a.ntiles * NO;
    float acc[NO];
#pragma unroll
    for (int o = 0; o < NO; ++o) acc[o] = 0.f;
    for (int t = threadIdx.x; t < a.ntiles; t += kThreads) {
#pragma unroll
        for (int o = 0; o < NO; ++o) acc[o] += P[(size_t)t * NO + o];
    }
#pragma unroll
    for (int o = 0; o < NO; ++o) {
        float v = acc[o];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0) red[wave][o] = v;
    }
    __syncthreads();
    if (threadIdx.x < NO) {
        float v = red[0][threadIdx.x];
        for (int w = 1; w < kThreads / 64; ++w) v += red[w][threadIdx.x];
        a.logits[(size_t)i * NO + threadIdx.x] = v + a.bias[threadIdx.x];
    }
}

// Variant mode: a variant that was left out of the work lists (more than vmax
// dirty tiles in some layer), or whose base slot holds no state yet, gets NaN.
__device__ inline bool var_bad(const TileHeadArgs &a, int i) {
    if (!a.primed[a.vbase]) return true;
    if (a.vmax <= 0) return false;
    for (int l = 1; l <= a.L; ++l)
        if (a.ntile[(size_t)i * (a.L + 1) + l] > a.vmax) return true;
    return false;
}

// Partials of tile t as variant i sees them: its own row where it recomputed
// the tile, else the base slot's.  Only for variants that passed var_bad: a
// variant left out of the lists has tile-mask bits but no list rows.
__device__ inline const float *var_part(const TileHeadArgs &a, int i, int t, int no) {
    const uint64_t w = a.vtm[(size_t)i * a.TMW + (t >> 6)];
    if ((w >> (t & 63)) & 1ull) return a.vhpart + (size_t)a.vmap[(size_t)i * a.ntiles + t] * no;
    return a.hpart + ((size_t)a.vbase * a.ntiles + t) * no;
}

// k_tile_head for variants: the same fixed order of tiles and of the sums, so
// a variant whose boxes are empty gets the base slot's logits bit for bit.
template <int NO>
__global__ __launch_bounds__(kThreads) void k_tile_head_var(TileHeadArgs a) {
    __shared__ float red[kThreads / 64][NO];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = blockIdx.x;
    if (var_bad(a, i)) {                                   // uniform per block
        if (threadIdx.x < NO) a.logits[(size_t)i * NO + threadIdx.x] = __builtin_nanf("");
        return;
    }
    float acc[NO];
#pragma unroll
    for (int o = 0; o < NO; ++o) acc[o] = 0.f;
    for (int t = threadIdx.x; t < a.ntiles; t += kThreads) {
        const float *P = var_part(a, i, t, NO);
#pragma unroll
        for (int o = 0; o < NO; ++o) acc[o] += P[o];
    }
#pragma unroll
    for (int o = 0; o < NO; ++o) {
        float v = acc[o];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0) red[wave][o] = v;
    }
    __syncthreads();
    if (threadIdx.x < NO) {
        float v = red[0][threadIdx.x];
        for (int w = 1; w < kThreads / 64; ++w) v += red[w][threadIdx.x];
        a.logits[(size_t)i * NO + threadIdx.x] = v + a.bias[threadIdx.x];
    }
}

__global__ __launch_bounds__(kThreads) void k_tile_head_var_generic(TileHeadArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = blockIdx.x;
    if (var_bad(a, i)) {                                   // uniform per block
        for (int o = threadIdx.x; o < a.n_out; o += kThreads) a.logits[(size_t)i * a.n_out + o] = __builtin_nanf("");
        return;
    }
    for (int o = wave; o < a.n_out; o += kThreads / 64) {
        float v = 0.f;
        for (int t = lane; t < a.ntiles; t += 64) v += var_part(a, i, t, a.n_out)[o];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0) a.logits[(size_t)i * a.n_out + o] = v + a.bias[o];
    }
}

// Any n_out: wave w of the block handles logits o = w, w + 4, ...
__global__ __launch_bounds__(kThreads) void k_tile_head_generic(TileHeadArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = blockIdx.x;
    const float *P = a.hpart + (size_t)(a.ids ? a.ids[i] : i) * a.ntiles * a.n_out;
    for (int o = wave; o < a.n_out; o += kThreads / 64) {
        float v = 0.f;
        for (int t = lane; t < a.ntiles; t += 64) v += P[(size_t)t * a.n_out + o];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0) a.logits[(size_t)i * a.n_out + o] = v + a.bias[o];
    }
}

// Generic head for any n_out (<= kHeadMaxOut): 8 outputs per pass over a_L.
template <int SG, typename AT>
__global__ __launch_bounds__(kThreads) void k_head_partial_generic(HeadArgs a, int o0) {
    constexpr int NO = 8;
    __shared__ float red[kThreads / 64][SG * NO];
    const int split = blockIdx.x, g = blockIdx.y;
    const size_t k0 = (size_t)split * a.chunk;
    const size_t k1 = min(k0 + a.chunk, a.K);
    const float *W = static_cast<const float *>(a.w);
    const AT *act = static_cast<const AT *>(a.act);
    float acc[SG][NO];
    for (int s = 0; s < SG; ++s)
        for (int o = 0; o < NO; ++o) acc[s][o] = 0.f;
    const int no = min(NO, a.n_out - o0);
    for (size_t k = k0 + 4 * (size_t)threadIdx.x; k < k1; k += 4 * kThreads) {
        for (int s = 0; s < SG; ++s) {
            const int i = g * SG + s;
            if (i >= a.n) break;
            const float4 av = load_act4<AT>(act + (size_t)a.ids[i] * a.K + k);
            for (int o = 0; o < no; ++o) {
                const float4 wv = *reinterpret_cast<const float4 *>(W + (size_t)(o0 + o) * a.K + k);
                float t = acc[s][o];
                t = fmaf(av.x, wv.x, t);
                t = fmaf(av.y, wv.y, t);
                t = fmaf(av.z, wv.z, t);
                t = fmaf(av.w, wv.w, t);
                acc[s][o] = t;
            }
        }
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int s = 0; s < SG; ++s)
        for (int o = 0; o < NO; ++o) {
            float v = acc[s][o];
            for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
            if (lane == 0) red[wave][s * NO + o] = v;
        }
    __syncthreads();
    for (int j = threadIdx.x; j < SG * NO; j += kThreads) {
        const int s = j / NO, o = j - s * NO;
        const int i = g * SG + s;
        if (i < a.n && o < no) {
            float v = red[0][j];
            for (int w = 1; w < kThreads / 64; ++w) v += red[w][j];
            a.part[((size_t)split * a.n + i) * a.n_out + o0 + o] = v;
        }
    }
}

// ------------------------------------------------------------------ bf16 tile partials

// Tile contributions to the logits for a bf16 last layer, as a matrix product
// per tile position: for the tiles of one position P (rows), with the head
// weights of P (bf16, packed [P][k-step][n-block][k-quarter][column][8] with
// only the n_out real columns stored: a last n-block of w < 16 logits holds w
// columns and its other lanes take zeros without a load),
//   hpart[tile][o] = sum_k act_tile[k] * hw[P][k][o],  k = pixel * C + channel,
// on v_mfma_f32_16x16x32_bf16 (A: the tile's cache slice read straight from
// memory, 16 bytes per lane per k-step; products of two bf16 values are exact
// in float32).  A block takes 64 consecutive work items (four 16-row groups);
// the work list is position-major, so the 64 items mostly share one or two
// positions, and the block makes one pass per distinct position.  In a pass
// the four waves split K: wave w runs k-steps [w KS/4, (w + 1) KS/4) for all
// four row groups, so each weight fragment of P is read once per block (the
// weights of the positions in flight do not fit in L2; reading them once per
// wave cost more than the activations), rows not at P contributing zeros.
// The four K-quarter partials go through LDS and wave g adds those of row
// group g in wave order.  A row's sum therefore has a fixed order that does
// not depend on which rows share the block: list and dense passes agree bit
// for bit.  VAR: variant work items; the tile's activations are its overlay
// row (the item's list index) and its partials go to the same row of the
// variant partials.
template <int C, int NBO, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_tile_part_bf16(ConvArgs a) {
    constexpr int KS = 16 * C / 32;           // k-steps
    constexpr int KW = KS / 4;                // k-steps per wave
    constexpr int KB = 4;                     // k-steps per batch of loads
    static_assert(KW % KB == 0, "whole batches");
    __shared__ int s_pos[64];
    __shared__ floatx4 s_acc[4][4][NBO][64];  // [wave][row group][n-block][lane]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, 64);
    const uint16_t *act = static_cast<const uint16_t *>(a.in);
    const uint16_t *hw = reinterpret_cast<const uint16_t *>(a.hw);
    const int ntiles = a.TH * a.TW;
    const int row = lane & 15, kq = lane >> 4;
    // This lane's B fragment of n-block nb within a k-step's n_out x 32 weights
    // (column `row`, k-quarter kq), or none past the last real column.
    const int kstep_elems = a.n_out * 32;
    int boff[NBO];
    bool bval[NBO];
#pragma unroll
    for (int nb = 0; nb < NBO; ++nb) {
        const int wb = min(16, a.n_out - 16 * nb);
        bval[nb] = row < wb;
        boff[nb] = nb * 16 * 32 + (kq * wb + row) * 8;
    }
    for (int g = xr.first; g < xr.end; g += xr.stride) {   // uniform per block
        // This lane's A rows: row `row` of each group (items g + 16 rg + row).
        uint32_t e[4];
        int pos[4];
        const uint16_t *arow[4];
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int it = g + 16 * rg + row;
            const bool valid = it < xr.end;
            e[rg] = valid ? item_word<DENSE>(a, it) : 0u;
            const TileRef r = item_ref(a, e[rg]);
            pos[rg] = valid ? r.tile : -1;
            arow[rg] = (VAR ? static_cast<const uint16_t *>(a.vov_in) + (size_t)it * kTilePx * C
                            : act + (size_t)r.slot * a.in_stride + (size_t)r.tile * kTilePx * C) +
                       8 * kq + 32 * KW * wave;
        }
        if (tid < 64) {
            const int t2 = g + tid;
            s_pos[tid] = t2 < xr.end ? item_ref(a, item_word<DENSE>(a, t2)).tile : -1;
        }
        lds_barrier();
        // Lane q of every wave holds row q's position; the passes take the
        // positions in order of first appearance, found by ballots.
        const int my_sp = s_pos[lane];
        uint64_t left = __ballot(my_sp >= 0);                // rows of the block not yet handled
        while (left) {                                       // uniform per block
            const int P = __builtin_amdgcn_readlane(my_sp, __ffsll((long long)left) - 1);
            const uint64_t pmask = __ballot(my_sp == P);
            left &= ~pmask;
            const uint16_t *wp = hw + ((size_t)P * KS + KW * wave) * kstep_elems;
            if constexpr (KW * NBO <= 32) {
                // The wave's whole K quarter of P's weights is loaded at once,
                // then per row group holding rows at P its activations: one
                // memory round trip for the weights and one per such group.
                // Products in k-step order, as in the batched loop below.
                u32x4 bq[KW][NBO];
#pragma unroll
                for (int s = 0; s < KW; ++s)
#pragma unroll
                    for (int nb = 0; nb < NBO; ++nb)
                        bq[s][nb] = bval[nb] ? *reinterpret_cast<const u32x4 *>(wp + (size_t)s * kstep_elems + boff[nb])
                                             : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                for (int rg = 0; rg < 4; ++rg) {
                    if (((pmask >> (16 * rg)) & 0xFFFFu) == 0) continue;   // uniform: no row of this group at P
                    u32x4 aq[KW];
                    const bool mine = pos[rg] == P;
#pragma unroll
                    for (int s = 0; s < KW; ++s)
                        aq[s] = mine ? *reinterpret_cast<const u32x4 *>(arow[rg] + 32 * s) : u32x4{0u, 0u, 0u, 0u};
                    floatx4 acc[NBO];
#pragma unroll
                    for (int nb = 0; nb < NBO; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < KW; ++s)
#pragma unroll
                        for (int nb = 0; nb < NBO; ++nb)
                            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8, aq[s]), __builtin_bit_cast(bf16x8, bq[s][nb]), acc[nb], 0, 0, 0);
#pragma unroll
                    for (int nb = 0; nb < NBO; ++nb) s_acc[wave][rg][nb][lane] = acc[nb];
                }
            } else {
            floatx4 acc[4][NBO];
#pragma unroll
            for (int rg = 0; rg < 4; ++rg)
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) acc[rg][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
            for (int s0 = 0; s0 < KW; s0 += KB) {
                u32x4 av[KB][4], bv[KB][NBO];
#pragma unroll
                for (int s = 0; s < KB; ++s) {
#pragma unroll
                    for (int nb = 0; nb < NBO; ++nb)
                        bv[s][nb] = bval[nb] ? *reinterpret_cast<const u32x4 *>(wp + (size_t)(s0 + s) * kstep_elems + boff[nb])
                                             : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg)
                        av[s][rg] = pos[rg] == P ? *reinterpret_cast<const u32x4 *>(arow[rg] + 32 * (s0 + s))
                                                 : u32x4{0u, 0u, 0u, 0u};
                }
#pragma unroll
                for (int s = 0; s < KB; ++s)
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg)
#pragma unroll
                        for (int nb = 0; nb < NBO; ++nb)
                            acc[rg][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8, av[s][rg]), __builtin_bit_cast(bf16x8, bv[s][nb]), acc[rg][nb],
                                0, 0, 0);
            }
#pragma unroll
            for (int rg = 0; rg < 4; ++rg)
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) s_acc[wave][rg][nb][lane] = acc[rg][nb];
            }
            lds_barrier();
            // Wave `wave` finishes row group `wave`: the K quarters in wave order.
            const uint64_t gmask = (pmask >> (16 * wave)) & 0xFFFFu;
            if (gmask) {                                     // uniform per wave
                const uint32_t ew = wave == 0 ? e[0] : wave == 1 ? e[1] : wave == 2 ? e[2] : e[3];
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) {
                    const floatx4 v = s_acc[0][wave][nb][lane] + s_acc[1][wave][nb][lane] +
                                      s_acc[2][wave][nb][lane] + s_acc[3][wave][nb][lane];
                    // D: rows 4 kq + i of the group, column lane % 16 = logit nb * 16 + row.
                    const int o = nb * 16 + row;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int q = 4 * kq + i;
                        const uint32_t eq = __shfl(ew, q, 64);   // lane q holds row q's item
                        if (o < a.n_out && ((gmask >> q) & 1)) {
                            const TileRef rq = item_ref(a, eq);
                            float *hp = VAR ? a.vhpart + (size_t)(g + 16 * wave + q) * a.n_out
                                            : a.hpart + ((size_t)rq.slot * ntiles + rq.tile) * a.n_out;
                            hp[o] = v[i];
                        }
                    }
                }
            }
            lds_barrier();                                   // s_acc is rewritten by the next pass
        }
    }
}


// ------------------------------------------------------------------ float32 tile partials

// The same product for a float32 last layer on the staged conv kernel, whose
// epilogue would otherwise read the tile's whole n_out x 16 C slice of head
// weights from L2 for every tile:
//   hpart[tile][o] = sum_k act_tile[k] * hw[P][k][o],  k = pixel * C + channel,
// on v_mfma_f32_16x16x4_f32 with K walked in 16-deep blocks: in block b lane
// group kq takes k = 16 b + 4 kq + j, j = 0..3 (one 16-byte load of the
// tile's cache slice per lane), the weights packed [P][b][kq][o][4] with only
// the n_out real logits (lanes of padding columns take zeros without a load).
// Rows, one pass per distinct position, K quarters per wave and their sum in
// wave order as in k_tile_part_bf16, so list and dense passes agree bit for
// bit.  VAR: variant work items, as in k_tile_part_bf16 (activations from the
// item's overlay row, partials to the same row of the variant partials).
template <int C, int NBO, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_tile_part_f32(ConvArgs a) {
    constexpr int KBL = C;                    // 16-deep K blocks per tile (16 C / 16)
    constexpr int KW = KBL / 4;               // blocks per wave
    constexpr int KB = 4;                     // blocks per batch of loads
    static_assert(KW % KB == 0, "whole batches");
    __shared__ int s_pos[64];
    __shared__ floatx4 s_acc[4][4][NBO][64];  // [wave][row group][n-block][lane]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, 64);
    const float *act = static_cast<const float *>(a.in);
    const int ntiles = a.TH * a.TW;
    const int row = lane & 15, kq = lane >> 4;
    const int blk_elems = a.n_out * 16;       // weights of one K block
    int boff[NBO];
    bool bval[NBO];
#pragma unroll
    for (int nb = 0; nb < NBO; ++nb) {
        const int o = nb * 16 + row;
        bval[nb] = o < a.n_out;
        boff[nb] = (kq * a.n_out + o) * 4;
    }
    for (int g = xr.first; g < xr.end; g += xr.stride) {   // uniform per block
        uint32_t e[4];
        int pos[4];
        const float *arow[4];
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int it = g + 16 * rg + row;
            const bool valid = it < xr.end;
            e[rg] = valid ? item_word<DENSE>(a, it) : 0u;
            const TileRef r = item_ref(a, e[rg]);
            pos[rg] = valid ? r.tile : -1;
            arow[rg] = (VAR ? static_cast<const float *>(a.vov_in) + (size_t)it * kTilePx * C
                            : act + (size_t)r.slot * a.in_stride + (size_t)r.tile * kTilePx * C) +
                       4 * kq + 16 * KW * wave;
        }
        if (tid < 64) {
            const int t2 = g + tid;
            s_pos[tid] = t2 < xr.end ? item_ref(a, item_word<DENSE>(a, t2)).tile : -1;
        }
        lds_barrier();
        const int my_sp = s_pos[lane];
        uint64_t left = __ballot(my_sp >= 0);                // rows of the block not yet handled
        while (left) {                                       // uniform per block
            const int P = __builtin_amdgcn_readlane(my_sp, __ffsll((long long)left) - 1);
            const uint64_t pmask = __ballot(my_sp == P);
            left &= ~pmask;
            const float *wp = a.hw + ((size_t)P * KBL + KW * wave) * blk_elems;
            floatx4 acc[4][NBO];
#pragma unroll
            for (int rg = 0; rg < 4; ++rg)
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) acc[rg][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
            // Row groups with no row at P skip their loads and matrix ops
            // (the flags are uniform: whole groups, from the ballot).
            bool gact[4];
#pragma unroll
            for (int rg = 0; rg < 4; ++rg) gact[rg] = ((pmask >> (16 * rg)) & 0xFFFFu) != 0;
            for (int s0 = 0; s0 < KW; s0 += KB) {
                floatx4 av[KB][4], bv[KB][NBO];
#pragma unroll
                for (int s = 0; s < KB; ++s) {
#pragma unroll
                    for (int nb = 0; nb < NBO; ++nb)
                        bv[s][nb] = bval[nb] ? *reinterpret_cast<const floatx4 *>(wp + (size_t)(s0 + s) * blk_elems + boff[nb])
                                             : floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int rg = 0; rg < 4; ++rg)
                        av[s][rg] = gact[rg] && pos[rg] == P ? *reinterpret_cast<const floatx4 *>(arow[rg] + 16 * (s0 + s))
                                                             : floatx4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int rg = 0; rg < 4; ++rg) {
                    if (!gact[rg]) continue;
#pragma unroll
                    for (int s = 0; s < KB; ++s)
#pragma unroll
                        for (int j = 0; j < 4; ++j)
#pragma unroll
                            for (int nb = 0; nb < NBO; ++nb)
                                acc[rg][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s][rg][j], bv[s][nb][j],
                                                                                   acc[rg][nb], 0, 0, 0);
                }
            }
#pragma unroll
            for (int rg = 0; rg < 4; ++rg)
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) s_acc[wave][rg][nb][lane] = acc[rg][nb];
            lds_barrier();
            // Wave `wave` finishes row group `wave`: the K quarters in wave order.
            const uint64_t gmask = (pmask >> (16 * wave)) & 0xFFFFu;
            if (gmask) {                                     // uniform per wave
                const uint32_t ew = wave == 0 ? e[0] : wave == 1 ? e[1] : wave == 2 ? e[2] : e[3];
#pragma unroll
                for (int nb = 0; nb < NBO; ++nb) {
                    const floatx4 v = s_acc[0][wave][nb][lane] + s_acc[1][wave][nb][lane] +
                                      s_acc[2][wave][nb][lane] + s_acc[3][wave][nb][lane];
                    const int o = nb * 16 + row;             // D: rows 4 kq + i of the group, column `row`
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int q = 4 * kq + i;
                        const uint32_t eq = __shfl(ew, q, 64);   // lane q holds row q's item
                        if (o < a.n_out && ((gmask >> q) & 1)) {
                            const TileRef rq = item_ref(a, eq);
                            float *hp = VAR ? a.vhpart + (size_t)(g + 16 * wave + q) * a.n_out
                                            : a.hpart + ((size_t)rq.slot * ntiles + rq.tile) * a.n_out;
                            hp[o] = v[i];
                        }
                    }
                }
            }
            lds_barrier();                                   // s_acc is rewritten by the next pass
        }
    }
}

}  // namespace

int head_streams_per_block(int n_out) { return n_out == 18 ? 4 : 8; }

template <typename AT>
void launch_head_partials(const HeadArgs &a, hipStream_t s) {
    const int sg = head_streams_per_block(a.n_out);
    dim3 grid(a.nsplit, (a.n + sg - 1) / sg);
    if (a.n_out == 6)
        hipLaunchKernelGGL((k_head_partial_f32<6, 8, AT>), grid, dim3(kThreads), 0, s, a);
    else if (a.n_out == 18)
        hipLaunchKernelGGL((k_head_partial_f32<18, 4, AT>), grid, dim3(kThreads), 0, s, a);
    else
        for (int o0 = 0; o0 < a.n_out; o0 += 8)
            hipLaunchKernelGGL((k_head_partial_generic<8, AT>), grid, dim3(kThreads), 0, s, a, o0);
}

hipError_t launch_head(const HeadArgs &a, rn_dtype dt, hipStream_t s) {
    if (dt == RN_BF16) launch_head_partials<uint16_t>(a, s);
    else launch_head_partials<float>(a, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int tot = a.n * a.n_out;
    hipLaunchKernelGGL(k_head_reduce, dim3((tot + 3) / 4), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

size_t tile_part_bf16_elems(int ntiles, int C, int n_out) {
    return (size_t)ntiles * kTilePx * C * n_out;
}

void pack_tile_part_bf16(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, uint16_t *dst) {
    // [tile][k-step][n-block][kq][column][j] with the n-block of width
    // wb = min(16, n_out - 16 n-block): k = 32 step + 8 kq + j is pixel k / C
    // (row-major in the tile) and channel k % C; logit o = 16 n-block + column.
    // Zero outside the image.
    const int nbo = (n_out + 15) / 16;
    const int ntiles = TH * TW, KS = kTilePx * C / 32;
    size_t d = 0;
    for (int t = 0; t < ntiles; ++t) {
        const int ty = t / TW, tx = t % TW;
        for (int s = 0; s < KS; ++s)
            for (int nb = 0; nb < nbo; ++nb) {
                const int wb = std::min(16, n_out - 16 * nb);
                for (int kq = 0; kq < 4; ++kq)
                    for (int col = 0; col < wb; ++col)
                        for (int j = 0; j < 8; ++j) {
                            const int k = 32 * s + 8 * kq + j, m = k / C, c = k % C;
                            const int o = nb * 16 + col, y = ty * kTile + (m >> 2), x = tx * kTile + (m & 3);
                            const float v = (y < H && x < W)
                                                ? dense_w[(size_t)o * C * H * W + ((size_t)c * H + y) * W + x]
                                                : 0.f;
                            dst[d++] = bf16_bits_host(v);
                        }
            }
    }
}

template <int C, bool DENSE, bool VAR>
hipError_t run_tile_part_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    // Two blocks per CU are resident (registers), so a larger grid would only
    // run in a second generation.
    const int grid = dev::persistent_grid(cus * (a.n_out <= 32 ? 2 : 1), (a.max_tiles + 63) / 64);
    if (a.n_out <= 16) hipLaunchKernelGGL((k_tile_part_bf16<C, 1, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    else if (a.n_out <= 32) hipLaunchKernelGGL((k_tile_part_bf16<C, 2, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_tile_part_bf16<C, 4, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

bool tile_part_bf16_supported(int C) { return C == 64 || C == 128; }

hipError_t launch_tile_part_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var) {
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
    if (a.cout == 64)
        return var ? run_tile_part_bf16<64, false, true>(a, cus, s)
                   : dense ? run_tile_part_bf16<64, true, false>(a, cus, s) : run_tile_part_bf16<64, false, false>(a, cus, s);
    if (a.cout == 128)
        return var ? run_tile_part_bf16<128, false, true>(a, cus, s)
                   : dense ? run_tile_part_bf16<128, true, false>(a, cus, s)
                           : run_tile_part_bf16<128, false, false>(a, cus, s);
    return hipErrorInvalidValue;
}

template <int C, bool DENSE, bool VAR>
hipError_t run_tile_part_f32(const ConvArgs &a, int cus, hipStream_t s) {
    const int grid = dev::persistent_grid(cus * 2, (a.max_tiles + 63) / 64);
    if (a.n_out <= 16) hipLaunchKernelGGL((k_tile_part_f32<C, 1, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    else if (a.n_out <= 32) hipLaunchKernelGGL((k_tile_part_f32<C, 2, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_tile_part_f32<C, 4, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

bool tile_part_f32_supported(int C) { return C == 128; }

hipError_t launch_tile_part_f32(const ConvArgs &a, int cus, hipStream_t s, bool var) {
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
    if (a.cout == 128)
        return var ? run_tile_part_f32<128, false, true>(a, cus, s)
                   : dense ? run_tile_part_f32<128, true, false>(a, cus, s) : run_tile_part_f32<128, false, false>(a, cus, s);
    return hipErrorInvalidValue;
}

size_t tile_part_f32_elems(int ntiles, int C, int n_out) { return (size_t)ntiles * kTilePx * C * n_out; }

void pack_tile_part_f32(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, float *dst) {
    // [tile][b][kq][o][j]: k = 16 b + 4 kq + j is pixel k / C (row-major in the
    // tile) and channel k % C; zero outside the image.
    const int ntiles = TH * TW;
    size_t d = 0;
    for (int t = 0; t < ntiles; ++t) {
        const int ty = t / TW, tx = t % TW;
        for (int b = 0; b < C; ++b)
            for (int kq = 0; kq < 4; ++kq)
                for (int o = 0; o < n_out; ++o)
                    for (int j = 0; j < 4; ++j) {
                        const int k = 16 * b + 4 * kq + j, m = k / C, c = k % C;
                        const int y = ty * kTile + (m >> 2), x = tx * kTile + (m & 3);
                        dst[d++] = (y < H && x < W) ? dense_w[(size_t)o * C * H * W + ((size_t)c * H + y) * W + x] : 0.f;
                    }
    }
}

hipError_t launch_tile_head(const TileHeadArgs &a, hipStream_t s) {
    if (a.var) {
        if (a.n_out == 6)
            hipLaunchKernelGGL(k_tile_head_var<6>, dim3(a.n), dim3(kThreads), 0, s, a);
        else if (a.n_out == 18)
            hipLaunchKernelGGL(k_tile_head_var<18>, dim3(a.n), dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL(k_tile_head_var_generic, dim3(a.n), dim3(kThreads), 0, s, a);
        return hipGetLastError();
    }
    if (a.n_out == 6)
        hipLaunchKernelGGL(k_tile_head<6>, dim3(a.n), dim3(kThreads), 0, s, a);
    else if (a.n_out == 18)
        hipLaunchKernelGGL(k_tile_head<18>, dim3(a.n), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(k_tile_head_generic, dim3(a.n), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace rn
