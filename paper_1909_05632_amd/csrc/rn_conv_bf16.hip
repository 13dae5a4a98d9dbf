// bf16 variants of the dirty-tile conv kernels: bf16 weights and activations
// (caches hold bf16), float32 accumulation, every output rounded to bf16
// (round to nearest even).  Same tiles, work lists, layouts and epilogue
// duties as the float32 kernels in rn_conv.hip (bias, ReLU, zero outside the
// image, scatter into the tiled cache, tile head partials).
#include <cstring>

#include "rn_device.hpp"

namespace rn {
namespace {

using namespace dev;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
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
template <int CIN, int COUT, bool DENSE>
__global__ __launch_bounds__(256) void k_conv_first_bf16(ConvArgs a) {
    __shared__ float s_w[CIN * 9 * COUT];
    __shared__ float s_b[COUT];
    __shared__ float s_halo[4][CIN * 36];
    const float *wg = static_cast<const float *>(a.w);
    for (int j = threadIdx.x; j < CIN * 9 * COUT; j += blockDim.x) s_w[j] = wg[j];
    for (int j = threadIdx.x; j < COUT; j += blockDim.x) s_b[j] = a.bias[j];
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int cnt = work_count<DENSE>(a);
    const size_t HW = (size_t)a.H * a.W;
    const int cin1 = CIN / a.stack;
    float *halo = s_halo[wave];
    const float *xin = static_cast<const float *>(a.in);
    uint16_t *outp = static_cast<uint16_t *>(a.out);

    const XcdRange xr = xcd_range(cnt, 4);
    for (int t = xr.first + wave; t < xr.end; t += xr.stride) {
        const TileRef r = decode<DENSE>(a, t);
        int head = 0;
        if (a.stack != 1) head = a.ring_head[r.slot];
        for (int h = lane; h < CIN * 36; h += 64) {
            const int c = h / 36, pos = h - c * 36;
            const int hy = pos / 6, hx = pos - hy * 6;
            const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
            float v = 0.0f;
            if (y >= 0 && y < a.H && x >= 0 && x < a.W) {
                const float *plane;
                if (a.stack == 1) {
                    plane = xin + ((size_t)r.slot * CIN + c) * HW;
                } else {
                    const int j = c / cin1, c1 = c - j * cin1;
                    const int rp = (head - (a.stack - 1) + j + 4 * a.stack) & 3;
                    plane = xin + (((size_t)r.slot * 4 + rp) * cin1 + c1) * HW;
                }
                v = bf2f(f2bf(plane[(size_t)y * a.W + x]));
            }
            halo[h] = v;
        }
        wave_sync();
        uint16_t *dst = outp + (size_t)r.slot * a.out_stride + (size_t)r.tile * kTilePx * COUT;
        for (int o = lane; o < kTilePx * COUT; o += 64) {
            const int m = o / COUT, co = o - m * COUT;
            const int py = m >> 2, px = m & 3;
            float acc = 0.0f;
#pragma unroll
            for (int c = 0; c < CIN; ++c)
#pragma unroll
                for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                    for (int kx = 0; kx < 3; ++kx)
                        acc = fmaf(s_w[(c * 9 + ky * 3 + kx) * COUT + co],
                                   halo[c * 36 + (py + ky) * 6 + px + kx], acc);
            float v = acc + s_b[co];
            v = v > 0.0f ? v : 0.0f;
            if (r.ty * kTile + py >= a.H || r.tx * kTile + px >= a.W) v = 0.0f;
            dst[o] = f2bf(v);
        }
        wave_sync();
    }
}

// ------------------------------------------------------------------ MFMA layers

// Implicit GEMM over a group of T tiles: M = 16 T pixels, N = COUT, K = 9 CIN.
// v_mfma_f32_16x16x32_bf16 operand layout (lane l, kq = l / 16):
//   A: row l % 16, k = 8 kq + j (j = 0..7);  B: k = 8 kq + j, column l % 16;
//   D: rows 4 kq + i, column l % 16.
// Rows are tile pixels in column-major order (row m = pixel (m % 4, m / 4)), so
// lane l of D holds pixels (i, kq), i = 0..3.  K is walked per kernel position
// in steps of 32 channels; lane group kq of step b takes channels 32 b + 8 kq
// .. + 7, one 16-byte LDS read for A.  The weights are packed
// [kpos][step][nb][lane][8] so that B is one 16-byte read per 16 outputs.
//
// Register blocking: four waves (one per SIMD) form a 2 x 2 grid; a wave owns
// MT tiles (16 MT rows) x COUT / 2 outputs, so every A fragment it reads feeds
// COUT / 32 matrix ops and every B fragment MT.  At the bf16 matrix rate this
// keeps the LDS traffic at or below half of its 256 bytes per clock.
//
// Weights stream through LDS one kernel position per stage, double-buffered:
// the next stage is fetched into registers while the matrix cores work on the
// current one, then written to the other buffer, one block barrier per stage.
// Every group walks the nine positions in the same order, so the stage after
// position 8 is the next group's position 0 and the pipeline never drains.
// The halos of the next group are fetched into registers during the second
// half of the current group.
//
// Halo layout in LDS: pixel p = 6 hy + hx at p * PS 16-byte chunks, chunk c of
// the pixel stored at slot c ^ g(hy, hx) with g taking hy % 4 (and hx % 4 for
// 16 chunks per pixel).  For every kernel position the 16 rows of a read then
// fall in 16 distinct bank groups, and so do the 8 rows of each half (checked
// exhaustively on the host for 32, 64 and 128 channels; 64 channels need the
// 12-chunk pixel stride).
template <int CIN, int COUT>
struct GrpBf {
    static constexpr int WM = 2;                     // waves along M
    static constexpr int WAVES = 2 * WM;
    static constexpr int THREADS = 64 * WAVES;
    static constexpr int MT = CIN >= 128 ? 4 : 8;    // tiles per wave
    static constexpr int T = WM * MT;                // tiles per group
    static constexpr int NB = COUT / 16;
    static constexpr int NBW = NB / 2;               // 16-output blocks per wave
    static constexpr int C8 = CIN / 8;               // 16-byte chunks per pixel
    static constexpr int PS = C8 == 8 ? 12 : C8;     // pixel stride in chunks
    static constexpr int HALO = 36 * PS * 8;         // bf16 elements per tile halo
    static constexpr int KB = CIN / 32;              // k-steps per kernel position
    static constexpr int WST = CIN * COUT;           // bf16 elements per weight stage
    static constexpr int WPT = (WST / 8 + THREADS - 1) / THREADS;      // 16-byte weight loads per thread
    static constexpr int HCH = T * 36 * C8;                            // 16-byte halo chunks per group
    static constexpr int HPT = (HCH + THREADS - 1) / THREADS;          // per thread
    static constexpr int SR = COUT + 8;              // output staging row stride (bf16)
    static constexpr size_t lds_bytes = (size_t)(T * HALO + 2 * WST) * 2;
    static_assert(CIN % 32 == 0 && COUT % 32 == 0, "bf16 MFMA tiling");
    static_assert(C8 == 4 || C8 == 8 || C8 == 16, "halo swizzle is defined for 32, 64, 128 channels");
    static_assert(16 * SR <= HALO, "output staging must fit in the halo area");
};

template <int C8>
__device__ inline int halo_swz(int hy, int hx) {
    return C8 == 16 ? (hy & 3) | ((hx & 3) << 2) : (hy & 3);
}

// Element offset (bf16) of chunk c of halo pixel (hy, hx).
template <int CIN, int COUT>
__device__ inline int halo_chunk(int hy, int hx, int c) {
    using G = GrpBf<CIN, COUT>;
    return ((hy * 6 + hx) * G::PS + (c ^ halo_swz<G::C8>(hy, hx))) * 8;
}

// Fetch this thread's share of a group's halos: chunk h = tid + THREADS j of
// T x 36 pixels x C8 chunks; zero outside the image and for absent tiles.
template <int CIN, int COUT>
__device__ inline void fetch_group_halos(const ConvArgs &a, const uint32_t *items, int nvalid, u32x4 *regs,
                                         int tid) {
    using G = GrpBf<CIN, COUT>;
    const uint16_t *inp = static_cast<const uint16_t *>(a.in);
#pragma unroll
    for (int j = 0; j < G::HPT; ++j) {
        const int h = tid + G::THREADS * j;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (h < G::HCH) {
            const int t = h / (36 * G::C8), rem = h - t * (36 * G::C8);
            const int pos = rem / G::C8, c = rem - pos * G::C8;
            if (t < nvalid) {
                const TileRef r = item_ref(a, items[t]);
                const int hy = pos / 6, hx = pos - hy * 6;
                const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
                if (y >= 0 && y < a.H && x >= 0 && x < a.W)
                    v = *reinterpret_cast<const u32x4 *>(
                        inp + (size_t)r.slot * a.in_stride +
                        ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN + c * 8);
            }
        }
        regs[j] = v;
    }
}

template <int CIN, int COUT>
__device__ inline void store_group_halos(uint16_t *halos, const u32x4 *regs, int tid) {
    using G = GrpBf<CIN, COUT>;
#pragma unroll
    for (int j = 0; j < G::HPT; ++j) {
        const int h = tid + G::THREADS * j;
        if (h < G::HCH) {
            const int t = h / (36 * G::C8), rem = h - t * (36 * G::C8);
            const int pos = rem / G::C8, c = rem - pos * G::C8;
            const int hy = pos / 6, hx = pos - hy * 6;
            *reinterpret_cast<u32x4 *>(halos + t * G::HALO + halo_chunk<CIN, COUT>(hy, hx, c)) = regs[j];
        }
    }
}

template <int CIN, int COUT>
__device__ inline void fetch_stage(const uint16_t *wg, int kpos, u32x4 *regs, int tid) {
    using G = GrpBf<CIN, COUT>;
    const u32x4 *src = reinterpret_cast<const u32x4 *>(wg + (size_t)kpos * G::WST);
#pragma unroll
    for (int j = 0; j < G::WPT; ++j) {
        const int e = tid + G::THREADS * j;
        if (e < G::WST / 8) regs[j] = src[e];
    }
}

template <int CIN, int COUT>
__device__ inline void store_stage(uint16_t *dst, const u32x4 *regs, int tid) {
    using G = GrpBf<CIN, COUT>;
#pragma unroll
    for (int j = 0; j < G::WPT; ++j) {
        const int e = tid + G::THREADS * j;
        if (e < G::WST / 8) reinterpret_cast<u32x4 *>(dst)[e] = regs[j];
    }
}

template <int MT, int NBW>
struct FragsBf {
    bf16x8 a[MT];
    bf16x8 b[NBW];
};

// A and B fragments of k-step kb at kernel position (ky, kx).
template <int CIN, int COUT>
__device__ inline void load_frags(FragsBf<GrpBf<CIN, COUT>::MT, GrpBf<CIN, COUT>::NBW> &f, const uint16_t *halos, const uint16_t *wst,
                                  int ky, int kx, int kb, int wm, int half, int lane) {
    using G = GrpBf<CIN, COUT>;
    const int m = lane & 15, kq = lane >> 4;
    const int hy = (m & 3) + ky, hx = (m >> 2) + kx;
    const int off = halo_chunk<CIN, COUT>(hy, hx, 4 * kb + kq);
#pragma unroll
    for (int mt = 0; mt < G::MT; ++mt)
        f.a[mt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(
                                                 halos + (wm * G::MT + mt) * G::HALO + off));
    const uint16_t *wb = wst + ((size_t)(kb * G::NB + half * G::NBW) * 64 + lane) * 8;
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb)
        f.b[nb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(wb + nb * 64 * 8));
}

template <int MT, int NBW>
__device__ inline void mma_frags(floatx4 (&acc)[MT][NBW], const FragsBf<MT, NBW> &f) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
            acc[mt][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[mt], f.b[nb], acc[mt][nb], 0, 0, 0);
}

template <int CIN, int COUT, bool DENSE>
__global__ __launch_bounds__((GrpBf<CIN, COUT>::THREADS)) void k_conv_bf16_grp(ConvArgs a) {
    using G = GrpBf<CIN, COUT>;
    extern __shared__ uint16_t smem16[];
    __shared__ float s_bias[COUT];
    __shared__ uint32_t s_items[2][G::T];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % G::WM, half = wave / G::WM;
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, G::T);
    if (xr.first >= xr.end) return;                       // uniform per block
    uint16_t *halos = smem16;
    uint16_t *wbuf = smem16 + G::T * G::HALO;             // two stages
    const uint16_t *wg = static_cast<const uint16_t *>(a.w);
    uint16_t *outp = static_cast<uint16_t *>(a.out);
    for (int j = tid; j < COUT; j += G::THREADS) s_bias[j] = a.bias[j];

    // Prologue: items, halos and weight stage 0 of the first group.
    int g = xr.first;
    if (tid < G::T) s_items[0][tid] = g + tid < xr.end ? item_word<DENSE>(a, g + tid) : 0u;
    u32x4 wreg[G::WPT];
    fetch_stage<CIN, COUT>(wg, 0, wreg, tid);
    __syncthreads();
    {
        u32x4 hreg[G::HPT];
        fetch_group_halos<CIN, COUT>(a, s_items[0], min(G::T, xr.end - g), hreg, tid);
        store_group_halos<CIN, COUT>(halos, hreg, tid);
    }
    store_stage<CIN, COUT>(wbuf, wreg, tid);
    __syncthreads();

    int buf = 0;                                          // weight buffer of the current stage
    for (int it = 0; g < xr.end; g += xr.stride, ++it) {  // uniform per block
        const int cur = it & 1;
        const int nvalid = min(G::T, xr.end - g);
        const int gn = g + xr.stride;
        const bool has_next = gn < xr.end;
        if (tid < G::T) s_items[cur ^ 1][tid] = has_next && gn + tid < xr.end ? item_word<DENSE>(a, gn + tid) : 0u;
        u32x4 hreg[G::HPT];
        floatx4 acc[G::MT][G::NBW];
#pragma unroll
        for (int mt = 0; mt < G::MT; ++mt)
#pragma unroll
            for (int nb = 0; nb < G::NBW; ++nb) acc[mt][nb] = floatx4{0.f, 0.f, 0.f, 0.f};

        for (int kpos = 0; kpos < 9; ++kpos) {
            // Weights of the next stage (next group's position 0 after position 8).
            fetch_stage<CIN, COUT>(wg, kpos == 8 ? 0 : kpos + 1, wreg, tid);
            // Next group's halos: its items were published by the barrier of stage 0.
            if (kpos == 4 && has_next)
                fetch_group_halos<CIN, COUT>(a, s_items[cur ^ 1], min(G::T, xr.end - gn), hreg, tid);
            const uint16_t *wst = wbuf + buf * G::WST;
            const int ky = kpos / 3, kx = kpos - ky * 3;
            FragsBf<G::MT, G::NBW> f0, f1;
            load_frags<CIN, COUT>(f0, halos, wst, ky, kx, 0, wm, half, lane);
#pragma unroll
            for (int kb = 0; kb < G::KB; ++kb) {
                if (kb + 1 < G::KB) {
                    if (kb & 1) load_frags<CIN, COUT>(f0, halos, wst, ky, kx, kb + 1, wm, half, lane);
                    else load_frags<CIN, COUT>(f1, halos, wst, ky, kx, kb + 1, wm, half, lane);
                }
                __builtin_amdgcn_sched_barrier(0);
                if (kb & 1) mma_frags<G::MT, G::NBW>(acc, f1);
                else mma_frags<G::MT, G::NBW>(acc, f0);
                __builtin_amdgcn_sched_barrier(0);
            }
            store_stage<CIN, COUT>(wbuf + (buf ^ 1) * G::WST, wreg, tid);
            buf ^= 1;
            __syncthreads();
        }

        // Epilogue: bias, ReLU, zero outside the image, round to bf16, stage the
        // group's outputs in the (now free) halo area, then coalesced stores.
        uint16_t *stage = halos;
        const int m = lane & 15, kq = lane >> 4;
#pragma unroll
        for (int mt = 0; mt < G::MT; ++mt) {
            const int t = wm * G::MT + mt;
            const TileRef r = item_ref(a, s_items[cur][t]);
            const bool col_in = r.tx * kTile + kq < a.W;
#pragma unroll
            for (int nb = 0; nb < G::NBW; ++nb) {
                const int n = (half * G::NBW + nb) * 16 + m;
                const float b = s_bias[n];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float v = acc[mt][nb][i] + b;
                    v = v > 0.0f ? v : 0.0f;
                    const bool inside = col_in & (r.ty * kTile + i < a.H);
                    v = inside ? v : 0.0f;
                    stage[(t * 16 + i * 4 + kq) * G::SR + n] = f2bf(v);
                }
            }
        }
        __syncthreads();
        constexpr int V8 = 16 * COUT / 8;                  // 16-byte vectors per tile
        for (int e = tid; e < G::T * V8; e += G::THREADS) {
            const int t = e / V8, o8 = e - t * V8;
            if (t < nvalid) {
                const TileRef r = item_ref(a, s_items[cur][t]);
                const int px = (8 * o8) / COUT, n = 8 * o8 - px * COUT;
                reinterpret_cast<u32x4 *>(outp + (size_t)r.slot * a.out_stride +
                                          (size_t)r.tile * kTilePx * COUT)[o8] =
                    *reinterpret_cast<const u32x4 *>(stage + (t * 16 + px) * G::SR + n);
            }
        }
        __syncthreads();
        if (has_next) store_group_halos<CIN, COUT>(halos, hreg, tid);
        __syncthreads();
    }
}

template <int CIN, int COUT, bool DENSE>
hipError_t run_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    using G = GrpBf<CIN, COUT>;
    if (a.n_out > 0) return hipErrorInvalidValue;          // head partials come from their own kernel
    constexpr size_t lds = G::lds_bytes;
    auto kern = k_conv_bf16_grp<CIN, COUT, DENSE>;
    static hipError_t attr = set_lds(kern, lds);
    if (attr != hipSuccess) return attr;
    const int grid = persistent_grid(cus, (a.max_tiles + G::T - 1) / G::T);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(G::THREADS), lds, s, a);
    return hipGetLastError();
}

template <int CIN, int COUT, bool DENSE>
hipError_t run_first_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    const int grid = persistent_grid(cus * 8, (a.max_tiles + 3) / 4);
    hipLaunchKernelGGL((k_conv_first_bf16<CIN, COUT, DENSE>), dim3(grid), dim3(256), 0, s, a);
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

hipError_t launch_conv_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    const bool dense = a.wl == nullptr;
#define X(ci, co)                                                                                \
    if (a.cin == ci && a.cout == co)                                                             \
        return dense ? run_mfma_bf16<ci, co, true>(a, cus, s) : run_mfma_bf16<ci, co, false>(a, cus, s);
    RN_BF16_MFMA_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_conv_first_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    const bool dense = a.wl == nullptr;
#define X(ci, co)                                                                                \
    if (a.cin == ci && a.cout == co)                                                             \
        return dense ? run_first_bf16<ci, co, true>(a, cus, s) : run_first_bf16<ci, co, false>(a, cus, s);
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
    // [kpos][block][nb][lane][j]: block b covers channels [32 b, 32 b + 32);
    // element j of lane l is B[channel][n], n = nb * 16 + l % 16,
    // channel = 32 b + 8 (l / 16) + j.
    uint16_t *d = static_cast<uint16_t *>(dst);
    const int nb_n = cout / 16, nblk = cin / 32;
    size_t o = 0;
    for (int kpos = 0; kpos < 9; ++kpos)
        for (int b = 0; b < nblk; ++b)
            for (int nb = 0; nb < nb_n; ++nb)
                for (int l = 0; l < 64; ++l)
                    for (int j = 0; j < 8; ++j) {
                        const int ci = 32 * b + 8 * (l / 16) + j, n = nb * 16 + l % 16;
                        d[o++] = host_bf16(oihw[((size_t)n * cin + ci) * 9 + kpos]);
                    }
}

}  // namespace rn
