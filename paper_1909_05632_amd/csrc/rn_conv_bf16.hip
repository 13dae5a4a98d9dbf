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

// v_mfma_f32_16x16x32_bf16 operand layout (lane l, kq = l / 16):
//   A: row l % 16, k = 8 kq + j (j = 0..7);  B: k = 8 kq + j, column l % 16;
//   D: rows 4 kq + i, column l % 16 (as the float32 16x16x4 instruction).
// Rows are tile pixels in column-major order (row m = pixel (m % 4, m / 4)).
// K per kernel position is walked in blocks of 32 channels; lane group kq of
// block b takes channels 32 b + 8 kq .. + 7, one 16-byte LDS read for A; the
// weights are packed [kpos][block][nb][lane][8] so B is one 16-byte read per
// nb.  Halo pixel stride CIN + 8 bf16 (a 16-byte pad) puts the 16-byte A reads
// of each 8-lane phase in distinct banks.  Weights are streamed through LDS
// in stages of KPS kernel positions for a group of 4 tiles (one per wave).
template <int CIN, int COUT>
struct MfmaBf {
    static constexpr int NB = COUT / 16;
    static constexpr int CS = CIN + 8;          // halo pixel stride (bf16 elements)
    static constexpr int NBLK = CIN / 32;       // k-steps per kernel position
    static constexpr int C8 = CIN / 8;          // 16-byte chunks per pixel
    static constexpr int HALO = 36 * CS;        // bf16 elements of one halo in LDS
    static constexpr int SR = COUT + 8;         // output staging row stride (bf16)
    static constexpr int HV = (36 * C8 + 63) / 64;
    static constexpr int WTOT = 9 * CIN * COUT; // bf16 elements
    static_assert(CIN % 32 == 0 && COUT % 16 == 0, "bf16 MFMA tiling");
    static_assert(16 * SR <= HALO, "output staging must fit in the halo area");
};

template <int CIN, int COUT, int KPS>
struct StagedBf {
    static constexpr int NST = (9 + KPS - 1) / KPS;
    static constexpr int WST = KPS * CIN * COUT;                       // bf16 elements per stage
    static constexpr size_t lds_bytes = (size_t)(WST + 4 * MfmaBf<CIN, COUT>::HALO) * 2;
};

template <int CIN, int COUT, int KPS, bool DENSE>
__global__ __launch_bounds__(256) void k_conv_mfma_bf16(ConvArgs a) {
    using M = MfmaBf<CIN, COUT>;
    using S = StagedBf<CIN, COUT, KPS>;
    extern __shared__ uint16_t smem16[];
    __shared__ float s_bias[COUT];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, 4);
    if (xr.first >= xr.end) return;                       // uniform per block
    uint16_t *s_w = smem16;
    uint16_t *halo = smem16 + S::WST + wave * M::HALO;
    const uint16_t *wg = static_cast<const uint16_t *>(a.w);
    const uint16_t *inp = static_cast<const uint16_t *>(a.in);
    uint16_t *outp = static_cast<uint16_t *>(a.out);
    for (int j = tid; j < COUT; j += blockDim.x) s_bias[j] = a.bias[j];
    const int mrow = lane & 15, kq = lane >> 4;
    const int pix = (mrow & 3) * 6 + (mrow >> 2);

    for (int g = xr.first; g < xr.end; g += xr.stride) {   // uniform per block
        const int t = g + wave;
        const bool valid = t < xr.end;
        TileRef r{0, 0, 0, 0};
        if (valid) {
            r = decode<DENSE>(a, t);
            const uint16_t *src = inp + (size_t)r.slot * a.in_stride;
#pragma unroll
            for (int j = 0; j < M::HV; ++j) {
                const int h = lane + 64 * j;
                if (h < 36 * M::C8) {
                    const int pos = h / M::C8, c8 = h - pos * M::C8;
                    const int hy = pos / 6, hx = pos - hy * 6;
                    const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
                    u32x4 v = {0u, 0u, 0u, 0u};
                    if (y >= 0 && y < a.H && x >= 0 && x < a.W)
                        v = *reinterpret_cast<const u32x4 *>(
                            src + ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN +
                            c8 * 8);
                    *reinterpret_cast<u32x4 *>(halo + pos * M::CS + c8 * 8) = v;
                }
            }
        }
        floatx4 acc[M::NB];
#pragma unroll
        for (int nb = 0; nb < M::NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        for (int st = 0; st < S::NST; ++st) {
            __syncthreads();                               // previous stage fully consumed
            const int n0 = st * S::WST;
            const int nf = min(S::WST, M::WTOT - n0);
            for (int j = tid; j < nf / 8; j += blockDim.x)
                reinterpret_cast<u32x4 *>(s_w)[j] = reinterpret_cast<const u32x4 *>(wg + n0)[j];
            __syncthreads();
            if (valid) {
#pragma unroll
                for (int kp = 0; kp < KPS; ++kp) {
                    const int kpos = st * KPS + kp;
                    if (kpos >= 9) break;
                    const int ky = kpos / 3, kx = kpos - ky * 3;
                    const uint16_t *ap = halo + (pix + ky * 6 + kx) * M::CS + 8 * kq;
#pragma unroll
                    for (int blk = 0; blk < M::NBLK; ++blk) {
                        const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(ap + 32 * blk));
                        const uint16_t *wb = s_w + (size_t)((kp * M::NBLK + blk) * M::NB) * 64 * 8 + lane * 8;
#pragma unroll
                        for (int nb = 0; nb < M::NB; ++nb) {
                            const bf16x8 bv = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(wb + nb * 64 * 8));
                            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[nb], 0, 0, 0);
                        }
                    }
                }
            }
        }
        if (valid) {
            wave_sync();
            // Epilogue: bias, ReLU, zero outside the image, round to bf16.
            uint16_t *stage = halo;
            const bool col_in = r.tx * kTile + kq < a.W;
#pragma unroll
            for (int nb = 0; nb < M::NB; ++nb) {
                const float b = s_bias[nb * 16 + mrow];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float v = acc[nb][i] + b;
                    v = v > 0.0f ? v : 0.0f;
                    if (!col_in || r.ty * kTile + i >= a.H) v = 0.0f;
                    const uint16_t h = f2bf(v);
                    acc[nb][i] = bf2f(h);                  // the stored value feeds the head
                    stage[(i * 4 + kq) * M::SR + nb * 16 + mrow] = h;
                }
            }
            wave_sync();
            u32x4 *d = reinterpret_cast<u32x4 *>(outp + (size_t)r.slot * a.out_stride +
                                                 (size_t)r.tile * kTilePx * COUT);
#pragma unroll
            for (int j = 0; j < (16 * COUT / 8 + 63) / 64; ++j) {
                const int o8 = lane + 64 * j;
                if (o8 < 16 * COUT / 8) {
                    const int e = 8 * o8, m = e / COUT, n = e - m * COUT;
                    d[o8] = *reinterpret_cast<const u32x4 *>(stage + m * M::SR + n);
                }
            }
            if (a.n_out > 0) {
                const int ntiles = a.TH * a.TW;
                for (int o = 0; o < a.n_out; ++o) {
                    const float4 *w4 = reinterpret_cast<const float4 *>(
                                           a.hw + ((size_t)o * ntiles + r.tile) * kTilePx * COUT) + lane;
                    float p = 0.f;
#pragma unroll
                    for (int nb = 0; nb < M::NB; ++nb) {
                        const float4 w = w4[nb * 64];
                        p = fmaf(acc[nb][0], w.x, p);
                        p = fmaf(acc[nb][1], w.y, p);
                        p = fmaf(acc[nb][2], w.z, p);
                        p = fmaf(acc[nb][3], w.w, p);
                    }
                    for (int off = 32; off > 0; off >>= 1) p += __shfl_xor(p, off, 64);
                    if (lane == 0) a.hpart[((size_t)r.slot * ntiles + r.tile) * a.n_out + o] = p;
                }
            }
            wave_sync();
        }
    }
}

constexpr size_t kLdsBudgetBf = 160 * 1024 - 1024;

template <int CIN, int COUT>
constexpr int pick_kps_bf() {
    return StagedBf<CIN, COUT, 9>::lds_bytes <= kLdsBudgetBf   ? 9
           : StagedBf<CIN, COUT, 3>::lds_bytes <= kLdsBudgetBf ? 3
                                                               : 1;
}

template <int CIN, int COUT, bool DENSE>
hipError_t run_mfma_bf16(const ConvArgs &a, int cus, hipStream_t s) {
    constexpr int KPS = pick_kps_bf<CIN, COUT>();
    constexpr size_t lds = StagedBf<CIN, COUT, KPS>::lds_bytes;
    auto kern = k_conv_mfma_bf16<CIN, COUT, KPS, DENSE>;
    static hipError_t attr = set_lds(kern, lds);
    if (attr != hipSuccess) return attr;
    const int grid = persistent_grid(cus, (a.max_tiles + 3) / 4);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, s, a);
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
