// bf16 variants of the dirty-tile conv kernels: bf16 weights and activations
// (caches hold bf16), float32 accumulation, every output rounded to bf16
// (round to nearest even).  Same tiles, work lists, layouts and epilogue
// duties as the float32 kernels in rn_conv.hip (bias, ReLU, zero outside the
// image, scatter into the tiled cache, tile head partials).
#include <cstring>
#include <utility>

#include "rn_device.hpp"

namespace rn {
namespace {

using namespace dev;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// float -> bf16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ inline uint16_t f2bf(float v) {
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ inline float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// ------------------------------------------------------------------ first layer

// Direct conv for a few input channels; the input is rounded to bf16 as it is
// staged, the weights arrive rounded, the output is rounded and stored as bf16.
// Lane l owns output channels l, l + 64 (weights in registers); the halo is
// read once from LDS into every lane's registers (the layout of the float32
// first-layer kernel).  VAR: variant tiles (input from the base slot and the
// variant's frame, output to the work item's overlay row).
template <int CIN, int COUT, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_conv_first_bf16(ConvArgs a) {
    constexpr int CPL = (COUT + 63) / 64;
    constexpr int HN = 36 * CIN;
    __shared__ float s_halo[4][HN];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float *wg = static_cast<const float *>(a.w);
    float wr[CPL][CIN * 9], br[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        const int co = min(lane + 64 * j, COUT - 1);
#pragma unroll
        for (int k = 0; k < CIN * 9; ++k) wr[j][k] = wg[k * COUT + co];
        br[j] = a.bias[co];
    }

    const int cnt = work_count<DENSE>(a);
    const size_t HW = (size_t)a.H * a.W;
    const int cin1 = CIN / a.stack;
    float *halo = s_halo[wave];
    const float *xin = static_cast<const float *>(a.in);
    uint16_t *outp = static_cast<uint16_t *>(a.out);

    // The halo values of the next tile (past the end: the last tile again,
    // never used) are loaded into registers, HPL per lane, before this tile's
    // FMAs, so their latency overlaps the arithmetic.
    constexpr int HPL = (HN + 63) / 64;
    const XcdRange xr = xcd_range(cnt, 4);
    auto load_tile = [&](int t, float *pv) __attribute__((always_inline)) {
        const TileRef r = decode<DENSE>(a, t);
        int head = 0;
        if (!VAR && a.stack != 1) head = a.ring_head[r.slot];
#pragma unroll
        for (int k = 0; k < HPL; ++k) {
            const int h = lane + 64 * k;
            const int c = h / 36, pos = h - c * 36;
            const int hy = pos / 6, hx = pos - hy * 6;
            const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
            float v = 0.0f;
            if (h < HN && y >= 0 && y < a.H && x >= 0 && x < a.W) {
                if constexpr (VAR) {
                    v = bf2f(f2bf(var_input(a, r.slot, c, y, x)));
                } else {
                    const float *plane;
                    if (a.stack == 1) {
                        plane = xin + ((size_t)r.slot * CIN + c) * HW;
                    } else {
                        // Channel c = frame j (oldest first) of the ring, channel c1 of it.
                        const int j = c / cin1, c1 = c - j * cin1;
                        const int rp = (head - (a.stack - 1) + j + 4 * a.stack) & 3;
                        plane = xin + (((size_t)r.slot * 4 + rp) * cin1 + c1) * HW;
                    }
                    v = bf2f(f2bf(plane[(size_t)y * a.W + x]));
                }
            }
            pv[k] = v;
        }
    };
    int t = xr.first + wave;
    if (t >= xr.end) return;
    float pv[HPL];
    load_tile(t, pv);
    for (; t < xr.end; t += xr.stride) {
        const TileRef r = decode<DENSE>(a, t);
#pragma unroll
        for (int k = 0; k < HPL; ++k) {
            const int h = lane + 64 * k;
            if (h < HN) {
                const int c = h / 36, pos = h - c * 36;
                halo[pos * CIN + c] = pv[k];
            }
        }
        wave_sync();
        // One output row at a time: its three halo rows (18 pixels x CIN,
        // contiguous in LDS) go to registers by broadcast reads.
        float hr[18 * CIN];
        load_tile(min(t + xr.stride, xr.end - 1), pv);
        uint16_t *dst = VAR ? static_cast<uint16_t *>(a.vov_out) + (size_t)t * kTilePx * COUT
                            : outp + (size_t)r.slot * a.out_stride + (size_t)r.tile * kTilePx * COUT;
#pragma unroll
        for (int py = 0; py < kTile; ++py) {
            if constexpr (CIN % 4 == 0) {
#pragma unroll
                for (int q = 0; q < 18 * CIN / 4; ++q) {
                    const float4 v4 = reinterpret_cast<const float4 *>(halo + py * 6 * CIN)[q];
                    hr[4 * q] = v4.x;
                    hr[4 * q + 1] = v4.y;
                    hr[4 * q + 2] = v4.z;
                    hr[4 * q + 3] = v4.w;
                }
            } else {
#pragma unroll
                for (int q = 0; q < 18 * CIN; ++q) hr[q] = halo[py * 6 * CIN + q];
            }
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const int co = lane + 64 * j;
                if (co >= COUT) continue;
#pragma unroll
                for (int px = 0; px < kTile; ++px) {
                    const int m = py * kTile + px;
                    float acc = 0.0f;
#pragma unroll
                    for (int c = 0; c < CIN; ++c)
#pragma unroll
                        for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                            for (int kx = 0; kx < 3; ++kx)
                                acc = fmaf(wr[j][c * 9 + ky * 3 + kx], hr[(ky * 6 + px + kx) * CIN + c], acc);
                    float v = acc + br[j];
                    v = v > 0.0f ? v : 0.0f;
                    if (r.ty * kTile + py >= a.H || r.tx * kTile + px >= a.W) v = 0.0f;
                    dst[m * COUT + co] = f2bf(v);
                }
            }
        }
        wave_sync();                                   // halo reads done before the next tile's writes
    }
}

// ------------------------------------------------------------------ MFMA layers

// Implicit GEMM over a group of T = 16 tiles: M = 256 pixels, N = COUT,
// K = 9 CIN, on v_mfma_f32_32x32x16_bf16 (one wave per SIMD issues this
// instruction at close to the full matrix rate; the 16x16x32 one needs two).
// Operand layout (lane l, h = l / 32):
//   A: row l % 32, k = 8 h + j (j = 0..7);  B: k = 8 h + j, column l % 32;
//   D: element i of lane l is row 8 (i / 4) + 4 h + i % 4, column l % 32.
// The product is formed transposed, D = W^T X: A holds 32 output channels,
// B the 32 pixels of a pair of tiles (column c = tile 2 p + c / 16, pixel c %
// 16 in column-major order: pixel (c % 4, (c % 16) / 4)).  Lane l of D then
// holds, for each g = 0..3, the four neighbouring channels 8 g + 4 h .. + 3 of
// one pixel, which the epilogue rounds and stores as one 8-byte word.  K is
// walked in steps of 16 channels of one kernel position; lane half h reads
// channels 8 h .. + 7 of the step, one 16-byte LDS read per operand.  The
// weights are packed [kpos][step][n-block][lane][8] (lane l: output 32 n-block
// + l % 32).
//
// Register blocking: four waves (one per SIMD) form a 2 x 2 grid; a wave owns
// 8 tiles (256 rows of the transposed product... 4 tile pairs) x COUT / 2
// outputs, so every weight fragment it reads feeds four matrix ops and every
// halo fragment COUT / 64.  At the matrix rate this keeps the LDS traffic near
// 100 of its 256 bytes per clock.
//
// Loop nest per group: for each chunk of HC = min(CIN, 64) input channels (a
// "pass"), the chunk's halos of the 16 tiles sit in LDS and the nine kernel
// positions stream their weights for that chunk through LDS, one position per
// stage, in three buffers.  Each weight byte brought to the CU serves 16 tiles
// and each halo byte is brought once.  The weights of a stage are fetched into
// registers four stages ahead and written to the free buffer two stages ahead
// (two stages of registers, so a weight load, and the group's output stores
// that precede it in the memory counter, have two stages to complete before a
// wait counts them); the next pass's halo chunk (the next
// group's first chunk after the last pass) is fetched in two halves, after the
// matrix ops of stages 1 and 3, and written to LDS once the pass is done.  The
// nine stages are unrolled and every load is issued on every path (a halo
// chunk outside the image reads a fixed valid address and is dropped when
// stored), so each wait names exactly the loads it needs, all issued at least
// a stage earlier.  Each stage ends with one block barrier.
//
// Halo layout in LDS: chunk c of halo pixel (hy, hx) at 16-byte chunk
// hy RS + hx CS + c, padded strides with CS = 9, RS = 60 for 8 chunks per
// pixel (CS = 4, RS = 25 for 4).  The LDS serves 16 lanes of a 16-byte read
// per clock (256 bytes, 16 bank groups); the 16 pixels such a group reads (one
// tile, one chunk: rows a = 0..3, columns b = 0..3 shifted by the kernel
// position) sit at a RS + b CS + const, and a RS + b CS mod 16 takes all 16
// values, so every read is conflict-free.  Unlike an XOR swizzle, the layout
// makes every read of a stage a per-lane base plus a constant, which the
// instruction's offset field holds (no per-position address registers).
// Within a stage the fragments of the next k-step are read before the matrix
// ops of the current one.
template <int CIN, int COUT>
struct GrpBf {
    static constexpr int THREADS = 512;              // eight waves, 4 (M) x 2 (N)
    static constexpr int WM = 4;
    static constexpr int MP = 2;                     // tile pairs per wave
    static constexpr int T = WM * 2 * MP;            // tiles per group
    static constexpr int NB = COUT / 32;             // 32-output blocks
    static constexpr int NBW = NB / 2;               // per wave
    static constexpr int HC = CIN < 64 ? CIN : 64;   // channels per pass
    static constexpr int NPASS = CIN / HC;
    static constexpr int C8 = HC / 8;                // 16-byte chunks per pixel and pass
    // Halo pixel (hy, hx) of a pass at chunk hy RS + hx CS (16-byte chunks):
    // a padded layout whose every read offset is a lane base plus a constant.
    static constexpr int CS = C8 == 8 ? 9 : 4;
    static constexpr int RS = C8 == 8 ? 60 : 25;
    static constexpr int HALO = (5 * RS + 6 * CS) * 8;   // bf16 elements per tile halo chunk
    static constexpr int KS = HC / 16;               // k-steps per stage
    static constexpr int WST = HC * COUT;            // bf16 elements per weight stage
    static constexpr int WPT = (WST / 8 + THREADS - 1) / THREADS;   // 16-byte weight loads per thread and stage
    static constexpr int PSTEP = THREADS / T / C8;   // pixel step of a thread's halo chunks
    static constexpr int HPT = (36 + PSTEP - 1) / PSTEP;            // halo chunks per thread and pass
    static constexpr size_t lds_bytes = (size_t)(T * HALO + 3 * WST) * 2;
    static_assert(CIN % HC == 0 && HC % 32 == 0 && COUT % 64 == 0, "bf16 MFMA tiling");
    static_assert(C8 == 4 || C8 == 8, "halo swizzle is defined for 32- and 64-channel chunks");
    static_assert(THREADS % (T * C8) == 0, "whole halo pixels per thread group");
};

// Element offset (bf16) of chunk c of halo pixel (hy, hx).
template <int CIN, int COUT>
__device__ inline int halo_chunk(int hy, int hx, int c) {
    using G = GrpBf<CIN, COUT>;
    return (hy * G::RS + hx * G::CS + c) * 8;
}

// Halo chunk j of pass `pass` of a group: the THREADS / T threads tid / (THREADS
// / T) = t serve tile t; thread tid takes chunk c = tid % C8 of pixel p0 +
// PSTEP j, p0 = (tid % (THREADS / T)) / C8.  The load is always issued (from
// the cache's first element when the pixel is outside the image, past 36 or
// of an absent tile) and bit j of `ok` says whether it counts.
template <int CIN, int COUT, bool VAR, int J>
__device__ inline void fetch_halo_chunk(const ConvArgs &a, const uint32_t *items, int nvalid, int pass, u32x4 *regs,
                                        uint32_t &ok, int tid) {
    using G = GrpBf<CIN, COUT>;
    constexpr int TPT = G::THREADS / G::T;           // threads per tile
    const uint16_t *inp = static_cast<const uint16_t *>(a.in);
    const int t = tid / TPT, c = tid % G::C8, p0 = (tid % TPT) / G::C8;
    const TileRef r = item_ref(a, items[t]);
    const int pos = p0 + G::PSTEP * J;
    const int hy = pos / 6, hx = pos - hy * 6;
    const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
    const bool in = t < nvalid && pos < 36 && y >= 0 && y < a.H && x >= 0 && x < a.W;
    const uint16_t *src;
    if constexpr (VAR) {
        src = in ? var_src<uint16_t>(a, r.slot, y, x, CIN) + pass * G::HC + c * 8 : inp;
    } else {
        src = inp + (in ? (size_t)r.slot * a.in_stride + pass * G::HC + c * 8 +
                              ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN
                        : 0);
    }
    regs[J] = *reinterpret_cast<const u32x4 *>(src);
    ok = in ? ok | (1u << J) : ok & ~(1u << J);
}

template <int CIN, int COUT, bool VAR, int J0, int J1>
__device__ inline void fetch_halos(const ConvArgs &a, const uint32_t *items, int nvalid, int pass, u32x4 *regs,
                                   uint32_t &ok, int tid) {
    [&]<int... J>(std::integer_sequence<int, J...>) {
        (fetch_halo_chunk<CIN, COUT, VAR, J0 + J>(a, items, nvalid, pass, regs, ok, tid), ...);
    }(std::make_integer_sequence<int, J1 - J0>{});
}

template <int CIN, int COUT>
__device__ inline void store_halos(uint16_t *halos, const u32x4 *regs, uint32_t ok, int tid) {
    using G = GrpBf<CIN, COUT>;
    constexpr int TPT = G::THREADS / G::T;
    const int t = tid / TPT, c = tid % G::C8, p0 = (tid % TPT) / G::C8;
#pragma unroll
    for (int j = 0; j < G::HPT; ++j) {
        const int pos = p0 + G::PSTEP * j;
        if (36 % G::PSTEP != 0 && pos >= 36) break;
        const int hy = pos / 6, hx = pos - hy * 6;
        const u32x4 z = {0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4 *>(halos + t * G::HALO + halo_chunk<CIN, COUT>(hy, hx, c)) =
            (ok >> j) & 1 ? regs[j] : z;
    }
}

// Weight stage q = pass * 9 + kpos: kernel position kpos, channels of the pass.
template <int CIN, int COUT>
__device__ inline void fetch_stage(const uint16_t *wg, int q, u32x4 *regs, int tid) {
    using G = GrpBf<CIN, COUT>;
    const int pass = q / 9, kpos = q - pass * 9;
    const u32x4 *src = reinterpret_cast<const u32x4 *>(wg + (size_t)kpos * CIN * COUT + (size_t)pass * G::WST);
#pragma unroll
    for (int j = 0; j < G::WPT; ++j) {
        const int e = tid + G::THREADS * j;
        if ((G::WST / 8) % G::THREADS == 0 || e < G::WST / 8) regs[j] = src[e];
    }
}

template <int CIN, int COUT>
__device__ inline void store_stage(uint16_t *dst, const u32x4 *regs, int tid) {
    using G = GrpBf<CIN, COUT>;
#pragma unroll
    for (int j = 0; j < G::WPT; ++j) {
        const int e = tid + G::THREADS * j;
        if ((G::WST / 8) % G::THREADS == 0 || e < G::WST / 8) reinterpret_cast<u32x4 *>(dst)[e] = regs[j];
    }
}

// Fragments of one 16-channel k-step: the halo columns of the wave's MP tile
// pairs and the weight rows of its NBW 32-output blocks.
template <int MP, int NBW>
struct FragsBf {
    bf16x8 xb[MP];
    bf16x8 wa[NBW];
};

// Lane bases of the k-step reads: this lane's halo chunk (tile pair 0 of the
// wave, pixel m of column l % 32, chunk half h) and its weight fragment in
// stage buffer 0.  Every read of a stage is then base + a constant.
template <int CIN, int COUT>
__device__ inline const uint16_t *halo_lane(const uint16_t *halos, int wm, int lane) {
    using G = GrpBf<CIN, COUT>;
    const int col = lane & 31, h = lane >> 5, m = col & 15;
    return halos + (wm * 2 * G::MP + (col >> 4)) * G::HALO + halo_chunk<CIN, COUT>(m & 3, m >> 2, h);
}

template <int CIN, int COUT>
__device__ inline const uint16_t *weight_lane(const uint16_t *wbuf, int half, int lane) {
    using G = GrpBf<CIN, COUT>;
    return wbuf + ((size_t)half * G::NBW * 64 + lane) * 8;
}

// Fragments of k-step S of kernel position KPOS (weights in stage buffer
// KPOS % 3).
template <int CIN, int COUT, int KPOS, int S>
__device__ inline void load_kstep(FragsBf<GrpBf<CIN, COUT>::MP, GrpBf<CIN, COUT>::NBW> &f, const uint16_t *hl,
                                  const uint16_t *wl) {
    using G = GrpBf<CIN, COUT>;
    constexpr int ky = KPOS / 3, kx = KPOS % 3;
    constexpr int hoff = (ky * G::RS + kx * G::CS + 2 * S) * 8;
    constexpr int woff = (KPOS % 3) * G::WST + S * G::NB * 512;
#pragma unroll
    for (int p = 0; p < G::MP; ++p)
        f.xb[p] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(hl + hoff + 2 * p * G::HALO));
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb)
        f.wa[nb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(wl + woff + nb * 512));
}

// The matrix work of one stage (kernel position KPOS) on the wave's MP tile
// pairs x NBW 32-output blocks, from k-step S on.  The fragments of k-step S
// arrive in f; those of the next k-step (past the stage's last: the first of
// stage KPOS + 1, whose weight buffer the previous barrier published) are
// read before the matrix ops of this one, so each read has a k-step of matrix
// work to arrive.  On return f holds the next stage's first k-step.
template <int CIN, int COUT, int KPOS, int S, int MP, int NBW, typename Mid>
__device__ inline void stage_mma(floatx16 (&acc)[MP][NBW], FragsBf<MP, NBW> &f, const uint16_t *hl, const uint16_t *wl,
                                 Mid &&mid) {
    using G = GrpBf<CIN, COUT>;
    static_assert(MP == G::MP && NBW == G::NBW, "accumulator shape");
    FragsBf<MP, NBW> nxt;
    if constexpr (S + 1 < G::KS) load_kstep<CIN, COUT, KPOS, S + 1>(nxt, hl, wl);
    else if constexpr (KPOS < 8) load_kstep<CIN, COUT, KPOS + 1, 0>(nxt, hl, wl);
#pragma unroll
    for (int p = 0; p < G::MP; ++p)
#pragma unroll
        for (int nb = 0; nb < G::NBW; ++nb)
            acc[p][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.wa[nb], f.xb[p], acc[p][nb], 0, 0, 0);
    if constexpr (S + 1 < G::KS || KPOS < 8) {
        __builtin_amdgcn_sched_group_barrier(0x100, MP + NBW, 0);   // the next reads first,
        __builtin_amdgcn_sched_group_barrier(0x008, MP * NBW, 0);   // then the matrix ops
    }
    // The stage's memory work goes out while the first k-step's matrix ops
    // run (pinned there: the scheduler would sink the loads to the end of the
    // stage, leaving them a barrier's distance to arrive).
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (S == 0) {
        mid();
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (S + 1 < G::KS || KPOS < 8) f = nxt;
    if constexpr (S + 1 < G::KS) stage_mma<CIN, COUT, KPOS, S + 1, MP, NBW>(acc, f, hl, wl, mid);
}

template <int CIN, int COUT, bool DENSE, bool VAR>
__global__ __launch_bounds__(512) void k_conv_bf16_grp(ConvArgs a) {
    using G = GrpBf<CIN, COUT>;
    constexpr int NQ = 9 * G::NPASS;                      // stages per group
    extern __shared__ uint16_t smem16[];
    __shared__ __align__(16) float s_bias[COUT];
    __shared__ uint32_t s_items[3][G::T];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % G::WM, half = wave / G::WM;
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, G::T);
    if (xr.first >= xr.end) return;                       // uniform per block
    uint16_t *halos = smem16;
    uint16_t *wbuf = smem16 + G::T * G::HALO;             // three stages; stage q of a group in q % 3
    const uint16_t *hl = halo_lane<CIN, COUT>(halos, wm, lane);
    const uint16_t *wl = weight_lane<CIN, COUT>(wbuf, half, lane);
    const uint16_t *wg = static_cast<const uint16_t *>(a.w);
    uint16_t *outp = static_cast<uint16_t *>(a.out);
    for (int j = tid; j < COUT; j += G::THREADS) s_bias[j] = a.bias[j];
    // Work items of group k (k strides after the first), 0 past the end.
    auto items_of = [&](int k) -> uint32_t {
        const int t = xr.first + k * xr.stride + tid;
        return t < xr.end && tid < G::T ? item_word<DENSE>(a, t) : 0u;
    };
    auto nvalid_of = [&](int k) { return max(0, min(G::T, xr.end - (xr.first + k * xr.stride))); };

    // Prologue: items of groups 0 and 1 in LDS, of group 2 in flight (items are
    // written to LDS a group before the halo fetch that reads them and loaded
    // a group before that); pass 0 halos and weight stages 0 and 1 in LDS,
    // stages 2 and 3 in flight to registers.
    if (tid < G::T) {
        s_items[0][tid] = items_of(0);
        s_items[1][tid] = items_of(1);
    }
    uint32_t ireg = items_of(2);
    u32x4 wreg[G::WPT], wnext[G::WPT];
    fetch_stage<CIN, COUT>(wg, 0, wreg, tid);
    lds_barrier();
    u32x4 hreg[G::HPT];
    uint32_t hok = 0;
    fetch_halos<CIN, COUT, VAR, 0, G::HPT>(a, s_items[0], nvalid_of(0), 0, hreg, hok, tid);
    store_halos<CIN, COUT>(halos, hreg, hok, tid);
    store_stage<CIN, COUT>(wbuf, wreg, tid);
    fetch_stage<CIN, COUT>(wg, 1, wreg, tid);
    store_stage<CIN, COUT>(wbuf + G::WST, wreg, tid);
    fetch_stage<CIN, COUT>(wg, 2, wreg, tid);
    fetch_stage<CIN, COUT>(wg, 3 % NQ, wnext, tid);
    lds_barrier();
    FragsBf<G::MP, G::NBW> f0;                            // first k-step of the next stage
    load_kstep<CIN, COUT, 0, 0>(f0, hl, wl);
    for (int it = 0;; ++it) {                             // groups, uniform per block
        const int g = xr.first + it * xr.stride;
        if (g >= xr.end) break;
        const int cur = it % 3;
        const int nvalid = nvalid_of(it);
        __builtin_amdgcn_sched_barrier(0);
        floatx16 acc[G::MP][G::NBW];
#pragma unroll
        for (int p = 0; p < G::MP; ++p)
#pragma unroll
            for (int nb = 0; nb < G::NBW; ++nb)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[p][nb][e] = 0.f;

#pragma unroll 1
        for (int pass = 0; pass < G::NPASS; ++pass) {
            // What the halo prefetch of this pass loads: the group's next
            // chunk, or the next group's first chunk.
            const bool last_pass = pass + 1 == G::NPASS;
            const uint32_t *hitems = last_pass ? s_items[(it + 1) % 3] : s_items[cur];
            const int hvalid = last_pass ? nvalid_of(it + 1) : nvalid;
            const int hpass = last_pass ? 0 : pass + 1;
            auto stage = [&](auto kc) __attribute__((always_inline)) {
                constexpr int kpos = decltype(kc)::value;
                const int q = pass * 9 + kpos;
                __builtin_amdgcn_sched_barrier(0);            // keep each stage's work in its stage
                // The matrix work on stage q (buffer q % 3 = kpos % 3, as 9
                // divides the stages of a group), which also reads the first
                // k-step of stage q + 1 unless the pass ends here; during it,
                // stage q + 2 (in registers since stage q - 2) goes to buffer
                // (q + 2) % 3, last read in stage q - 1, and stage q + 4
                // (wrapping into the next group) is fetched to registers;
                // halo loads after the matrix ops of stages 1 and 3.  The
                // barrier publishes stage q + 2 and frees stage q's buffer.
                stage_mma<CIN, COUT, kpos, 0, G::MP, G::NBW>(acc, f0, hl, wl, [&] {
                    store_stage<CIN, COUT>(wbuf + ((kpos + 2) % 3) * G::WST, wreg, tid);
                    fetch_stage<CIN, COUT>(wg, (q + 4) % NQ, wreg, tid);
#pragma unroll
                    for (int j = 0; j < G::WPT; ++j) {                // wreg: stage q + 3, wnext: q + 4
                        const u32x4 t = wreg[j];
                        wreg[j] = wnext[j];
                        wnext[j] = t;
                    }
                });
                if constexpr (kpos == 1)
                    fetch_halos<CIN, COUT, VAR, 0, G::HPT / 2>(a, hitems, hvalid, hpass, hreg, hok, tid);
                if constexpr (kpos == 3)
                    fetch_halos<CIN, COUT, VAR, G::HPT / 2, G::HPT>(a, hitems, hvalid, hpass, hreg, hok, tid);
                lds_barrier();
            };
            [&]<int... K>(std::integer_sequence<int, K...>) {
                (stage(std::integral_constant<int, K>{}), ...);
            }(std::make_integer_sequence<int, 9>{});
            if (!last_pass) {
                store_halos<CIN, COUT>(halos, hreg, hok, tid);    // every wave is past the pass's last read
                lds_barrier();
                load_kstep<CIN, COUT, 0, 0>(f0, hl, wl);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        // Items of group it + 2 to LDS (its slot last served group it - 1),
        // then the load of group it + 3's items.
        if (tid < G::T) s_items[(it + 2) % 3][tid] = ireg;
        ireg = items_of(it + 3);

        // The next group's first halo chunk goes to LDS now (every wave is
        // past the last read of this group's halos), then the epilogue: bias,
        // ReLU, zero outside the image, round to bf16 and store straight to
        // the cache.  Lanes l and l + 32 hold the two halves of each 8-channel
        // group of a pixel; one v_permlane32_swap per word gives the lower
        // lane the whole of groups 0 and 2 and the upper lane groups 1 and 3,
        // so every lane stores 16 contiguous bytes.
        if (nvalid_of(it + 1) > 0) store_halos<CIN, COUT>(halos, hreg, hok, tid);
        const int col = lane & 31, h = lane >> 5, m = col & 15;
        const int py = m & 3, px = m >> 2;
#pragma unroll
        for (int p = 0; p < G::MP; ++p) {
            const int t = wm * 2 * G::MP + 2 * p + (col >> 4);
            const TileRef r = item_ref(a, s_items[cur][t]);
            const bool inside = (r.ty * kTile + py < a.H) & (r.tx * kTile + px < a.W);
            // VAR: the work item's index is g + t, its overlay row.
            uint16_t *dst = VAR ? static_cast<uint16_t *>(a.vov_out) + ((size_t)(g + t) * kTilePx + py * 4 + px) * COUT
                                : outp + (size_t)r.slot * a.out_stride + ((size_t)r.tile * kTilePx + py * 4 + px) * COUT;
#pragma unroll
            for (int nb = 0; nb < G::NBW; ++nb) {
                const int nbase = (half * G::NBW + nb) * 32;
                uint32_t wd[4][2];                         // [channel group][word]
#pragma unroll
                for (int gq = 0; gq < 4; ++gq) {
                    const int n0 = nbase + 8 * gq + 4 * h;
                    const float4 b = *reinterpret_cast<const float4 *>(s_bias + n0);
                    float x[4] = {acc[p][nb][4 * gq] + b.x, acc[p][nb][4 * gq + 1] + b.y,
                                  acc[p][nb][4 * gq + 2] + b.z, acc[p][nb][4 * gq + 3] + b.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i) x[i] = inside && x[i] > 0.0f ? x[i] : 0.0f;
                    const bf16x2 lo = {(__bf16)x[0], (__bf16)x[1]}, hi = {(__bf16)x[2], (__bf16)x[3]};
                    wd[gq][0] = __builtin_bit_cast(uint32_t, lo);
                    wd[gq][1] = __builtin_bit_cast(uint32_t, hi);
                }
#pragma unroll
                for (int g0 = 0; g0 < 4; g0 += 2) {
                    const auto s0 = __builtin_amdgcn_permlane32_swap(wd[g0][0], wd[g0 + 1][0], false, false);
                    const auto s1 = __builtin_amdgcn_permlane32_swap(wd[g0][1], wd[g0 + 1][1], false, false);
                    const u32x4 v = {s0[0], s1[0], s0[1], s1[1]};
                    if (t < nvalid) *reinterpret_cast<u32x4 *>(dst + nbase + 8 * (g0 + h)) = v;
                }
            }
        }
        lds_barrier();
        load_kstep<CIN, COUT, 0, 0>(f0, hl, wl);
    }
}

template <int CIN, int COUT, bool DENSE, bool VAR>
hipError_t run_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    using G = GrpBf<CIN, COUT>;
    if (a.n_out > 0) return hipErrorInvalidValue;          // head partials come from their own kernel
    constexpr size_t lds = G::lds_bytes;
    auto kern = k_conv_bf16_grp<CIN, COUT, DENSE, VAR>;
    static hipError_t attr = set_lds(kern, lds);
    if (attr != hipSuccess) return attr;
    const int grid = persistent_grid(cus, (a.max_tiles + G::T - 1) / G::T);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(G::THREADS), lds, s, a);
    return hipGetLastError();
}

template <int CIN, int COUT, bool DENSE, bool VAR>
hipError_t run_first_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    const int grid = persistent_grid(cus * 8, (a.max_tiles + 3) / 4);
    hipLaunchKernelGGL((k_conv_first_bf16<CIN, COUT, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

#define RN_BF16_MFMA_SHAPES(X) X(64, 128) X(128, 128) X(32, 64) X(64, 64)
#define RN_BF16_FIRST_SHAPES(X) X(1, 32) X(1, 64) X(4, 32) X(4, 64)

uint16_t host_bf16(float v) {
    uint32_t u;
    memcpy(&u, &v, 4);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

}  // namespace

bool conv_mfma_bf16_supported(int cin, int cout) {
#define X(ci, co) if (cin == ci && cout == co) return true;
    RN_BF16_MFMA_SHAPES(X)
#undef X
    return false;
}

bool conv_first_bf16_supported(int cin, int cout) {
#define X(ci, co) if (cin == ci && cout == co) return true;
    RN_BF16_FIRST_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_conv_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var) {
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
#define X(ci, co)                                                                                \
    if (a.cin == ci && a.cout == co)                                                             \
        return var ? run_mfma_bf16<ci, co, false, true>(a, cus, s)                               \
                   : dense ? run_mfma_bf16<ci, co, true, false>(a, cus, s) : run_mfma_bf16<ci, co, false, false>(a, cus, s);
    RN_BF16_MFMA_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_conv_first_bf16(const ConvArgs &a, int cus, hipStream_t s, bool var) {
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
#define X(ci, co)                                                                                \
    if (a.cin == ci && a.cout == co)                                                             \
        return var ? run_first_bf16<ci, co, false, true>(a, cus, s)                              \
                   : dense ? run_first_bf16<ci, co, true, false>(a, cus, s) : run_first_bf16<ci, co, false, false>(a, cus, s);
    RN_BF16_FIRST_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

uint16_t bf16_bits_host(float v) { return host_bf16(v); }

float round_bf16_host(float v) {
    const uint32_t u = (uint32_t)host_bf16(v) << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

void pack_conv_mfma_bf16(const float *oihw, int cin, int cout, void *dst) {
    // [kpos][step][n-block][lane][j]: step s covers channels [16 s, 16 s + 16);
    // element j of lane l is W[n][c] with n = 32 n-block + l % 32 and
    // c = 16 s + 8 (l / 32) + j.
    uint16_t *d = static_cast<uint16_t *>(dst);
    const int nbn = cout / 32, ns = cin / 16;
    size_t o = 0;
    for (int kpos = 0; kpos < 9; ++kpos)
        for (int st = 0; st < ns; ++st)
            for (int nb = 0; nb < nbn; ++nb)
                for (int l = 0; l < 64; ++l)
                    for (int j = 0; j < 8; ++j) {
                        const int ci = 16 * st + 8 * (l / 32) + j, n = nb * 32 + l % 32;
                        d[o++] = host_bf16(oihw[((size_t)n * cin + ci) * 9 + kpos]);
                    }
}

}  // namespace rn
