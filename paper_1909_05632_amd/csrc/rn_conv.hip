// Dirty-tile convolution kernels (Sec. 1: recompute only where the change can
// reach and reuse the cached activations elsewhere).
//
// Every conv layer is 3x3, stride 1, zero pad 1, then bias and ReLU:
//   out[y][x][co] = ReLU(b[co] + sum_{ky,kx,ci} w[co][ci][ky][kx] * in[y-1+ky][x-1+kx][ci]).
// Each work-list entry names one 4x4 output tile of one stream; the kernels
// compute its 16 pixels x cout outputs from the 6x6 input halo and write them
// in place into the stream's cache (scatter fused with bias and ReLU).
// Pixels of a ragged edge tile that fall outside the image are written as 0:
// they are the next layer's zero padding and carry zero dense weights.
//
// Cache layout ("tiled NHWC"): per slot [TH][TW][16][C], a tile's 16 pixels in
// row-major order, channels innermost; one tile is 16 * C contiguous elements.
//
// Both kernels are persistent: the grid is sized to the chip and each block
// walks the device-side work list until the device-side count is exhausted,
// so no host synchronisation is needed to size a launch.
#include "rn_internal.hpp"

namespace rn {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

[[maybe_unused]] __device__ inline float bf16_round(float v) {
    // Round to nearest even on the upper 16 bits (finite values; NaN kept NaN).
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7F800000u) == 0x7F800000u) return __uint_as_float((u | ((u & 0xFFFF) ? 0x00400000u : 0u)) & 0xFFFF0000u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return __uint_as_float(u & 0xFFFF0000u);
}

// ------------------------------------------------------------------ first layer

// Direct conv for a few input channels (1, or 4 stacked frames): 9 * CIN FMAs
// per output, too few for a matrix core to pay off; the layer is HBM-bound on
// its output writes.  One wave per tile; weights and bias in LDS.
template <int CIN, int COUT>
__global__ __launch_bounds__(256) void k_conv_first_f32(ConvArgs a) {
    __shared__ float s_w[CIN * 9 * COUT];
    __shared__ float s_b[COUT];
    __shared__ float s_halo[4][CIN * 36];
    const float *wg = static_cast<const float *>(a.w);
    for (int j = threadIdx.x; j < CIN * 9 * COUT; j += blockDim.x) s_w[j] = wg[j];
    for (int j = threadIdx.x; j < COUT; j += blockDim.x) s_b[j] = a.bias[j];
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int cnt = *a.cnt;
    const size_t HW = (size_t)a.H * a.W;
    const int cin1 = CIN / a.stack;               // channels per frame
    float *halo = s_halo[wave];
    const float *xin = static_cast<const float *>(a.in);
    float *outp = static_cast<float *>(a.out);

    for (int base = blockIdx.x * 4; base < cnt; base += gridDim.x * 4) {
        const int t = base + wave;
        const bool valid = t < cnt;
        int slot = 0, ty = 0, tx = 0;
        if (valid) {
            const uint32_t e = a.wl[t];
            slot = a.ids[e >> 16];
            ty = (e >> 8) & 255;
            tx = e & 255;
            int head = 0;
            if (a.stack != 1) head = a.ring_head[slot];
            for (int h = lane; h < CIN * 36; h += 64) {
                const int c = h / 36, pos = h - c * 36;
                const int hy = pos / 6, hx = pos - hy * 6;
                const int y = ty * kTile - 1 + hy, x = tx * kTile - 1 + hx;
                float v = 0.0f;
                if (y >= 0 && y < a.H && x >= 0 && x < a.W) {
                    const float *plane;
                    if (a.stack == 1) {
                        plane = xin + ((size_t)slot * CIN + c) * HW;
                    } else {
                        // Channel c = frame j (oldest first) of the ring, channel c1 of it.
                        const int j = c / cin1, c1 = c - j * cin1;
                        const int rp = (head - (a.stack - 1) + j + 4 * a.stack) & 3;
                        plane = xin + (((size_t)slot * 4 + rp) * cin1 + c1) * HW;
                    }
                    v = plane[(size_t)y * a.W + x];
                }
                halo[h] = v;
            }
        }
        __syncthreads();
        if (valid) {
            float *dst = outp + (size_t)slot * a.out_stride + (size_t)(ty * a.TW + tx) * kTilePx * COUT;
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
                if (ty * kTile + py >= a.H || tx * kTile + px >= a.W) v = 0.0f;
                dst[o] = v;
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ MFMA layers

// Implicit GEMM per tile: M = 16 pixels, N = COUT, K = 9 * CIN ordered
// (ky, kx, ci).  v_mfma_f32_16x16x4_f32 operand layout (lane l):
//   A: row l % 16, k l / 16;  B: k l / 16, column l % 16;
//   D: rows 4 (l / 16) + i, column l % 16, i = 0..3.
// So row m = pixel (m / 4, m % 4) of the tile; the A operand is read straight
// from the 6x6 x CIN halo in LDS (im2col is an address computation), and lane l
// ends up holding tile row l / 16, columns i = 0..3, of channel l % 16 + 16 nb.
// The weights are pre-packed in fragment order [kstep][nb][lane] so each B
// read is one conflict-free 256-byte LDS row.  When all of them fit in LDS
// (KPS = 9) they are loaded once per persistent block; otherwise they are
// streamed in stages of KPS kernel positions per tile group.
template <int CIN, int COUT, int KPS, int WAVES>
struct MfmaCfg {
    static constexpr int NB = COUT / 16;
    static constexpr int CS = CIN + 1;       // halo channel stride in LDS (odd: spreads banks)
    static constexpr int KSP = CIN / 4;      // k-steps per kernel position
    static constexpr int NST = (9 + KPS - 1) / KPS;
    static constexpr int WST = KPS * CIN * COUT;
    static constexpr size_t lds_bytes = (size_t)(WST + WAVES * 36 * CS) * sizeof(float);
};

template <int CIN, int COUT, int KPS, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void k_conv_mfma_f32(ConvArgs a) {
    using C = MfmaCfg<CIN, COUT, KPS, WAVES>;
    constexpr int NB = C::NB, CS = C::CS, KSP = C::KSP, NST = C::NST, WST = C::WST;
    constexpr int WTOT = 9 * CIN * COUT;
    extern __shared__ float smem[];
    __shared__ float s_bias[COUT];
    float *s_w = smem;
    float *s_halo = smem + WST;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int cnt = *a.cnt;
    const int ngroups = (cnt + WAVES - 1) / WAVES;
    if ((int)blockIdx.x >= ngroups) return;       // uniform per block
    const float *wg = static_cast<const float *>(a.w);
    for (int j = tid; j < COUT; j += blockDim.x) s_bias[j] = a.bias[j];
    if constexpr (NST == 1) {
        for (int j = tid; j < WTOT / 4; j += blockDim.x)
            reinterpret_cast<float4 *>(s_w)[j] = reinterpret_cast<const float4 *>(wg)[j];
    }
    const int mrow = lane & 15, kq = lane >> 4;
    const int py = mrow >> 2, px = mrow & 3;
    float *my_halo = s_halo + wave * 36 * CS;
    const float *inp = static_cast<const float *>(a.in);
    float *outp = static_cast<float *>(a.out);

    for (int grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
        const int t = grp * WAVES + wave;
        const bool valid = t < cnt;
        int slot = 0, ty = 0, tx = 0;
        if (valid) {
            const uint32_t e = a.wl[t];
            slot = a.ids[e >> 16];
            ty = (e >> 8) & 255;
            tx = e & 255;
            const float *src = inp + (size_t)slot * a.in_stride;
            for (int h = lane; h < 36 * KSP; h += 64) {
                const int pos = h / KSP, c4 = h - pos * KSP;
                const int hy = pos / 6, hx = pos - hy * 6;
                const int y = ty * kTile - 1 + hy, x = tx * kTile - 1 + hx;
                float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                if (y >= 0 && y < a.H && x >= 0 && x < a.W)
                    v = *reinterpret_cast<const float4 *>(
                        src + ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN +
                        c4 * 4);
                float *d = my_halo + pos * CS + c4 * 4;
                d[0] = v.x;
                d[1] = v.y;
                d[2] = v.z;
                d[3] = v.w;
            }
        }
        floatx4 acc[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};

        for (int st = 0; st < NST; ++st) {
            if constexpr (NST > 1) {
                __syncthreads();
                const int n0 = st * WST;
                const int nf = min(WST, WTOT - n0);
                for (int j = tid; j < nf / 4; j += blockDim.x)
                    reinterpret_cast<float4 *>(s_w)[j] = reinterpret_cast<const float4 *>(wg + n0)[j];
            }
            __syncthreads();
            if (valid) {
#pragma unroll
                for (int kp = 0; kp < KPS; ++kp) {
                    const int kpos = st * KPS + kp;
                    if (NST > 1 && kpos >= 9) break;
                    const int ky = kpos / 3, kx = kpos - ky * 3;
                    const float *arow = my_halo + ((py + ky) * 6 + px + kx) * CS + kq;
                    const float *brow = s_w + kp * KSP * NB * 64 + lane;
#pragma unroll
                    for (int cs = 0; cs < KSP; ++cs) {
                        const float av = arow[cs * 4];
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
                            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, brow[(cs * NB + nb) * 64],
                                                                           acc[nb], 0, 0, 0);
                    }
                }
            }
        }
        if (valid) {
            float *dst = outp + (size_t)slot * a.out_stride + (size_t)(ty * a.TW + tx) * kTilePx * COUT;
            const bool row_in = ty * kTile + kq < a.H;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int n = nb * 16 + mrow;
                const float b = s_bias[n];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float v = acc[nb][i] + b;
                    v = v > 0.0f ? v : 0.0f;
                    if (!row_in || tx * kTile + i >= a.W) v = 0.0f;
                    dst[(kq * 4 + i) * COUT + n] = v;
                }
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ dispatch

template <int CIN, int COUT>
constexpr int pick_kps() {
    // Largest stage (9, 3 or 1 kernel positions) that fits 160 KiB of LDS
    // next to the halos of 4 waves.
    return MfmaCfg<CIN, COUT, 9, 4>::lds_bytes <= 160 * 1024 - 2048   ? 9
           : MfmaCfg<CIN, COUT, 3, 4>::lds_bytes <= 160 * 1024 - 2048 ? 3
                                                                      : 1;
}

template <int CIN, int COUT>
hipError_t run_mfma(const ConvArgs &a, int grid, hipStream_t s) {
    constexpr int KPS = pick_kps<CIN, COUT>();
    constexpr size_t lds = MfmaCfg<CIN, COUT, KPS, 4>::lds_bytes;
    auto kern = k_conv_mfma_f32<CIN, COUT, KPS, 4>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, s, a);
    return hipGetLastError();
}

template <int CIN, int COUT>
hipError_t run_first(const ConvArgs &a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((k_conv_first_f32<CIN, COUT>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

#define RN_MFMA_SHAPES(X) X(20, 40) X(40, 80) X(80, 160) X(64, 128) X(128, 128)
#define RN_FIRST_SHAPES(X) X(1, 20) X(1, 40) X(1, 64) X(1, 80) X(4, 20) X(4, 40) X(4, 64) X(4, 80)

}  // namespace

bool conv_mfma_supported(int cin, int cout, rn_dtype dt) {
    if (dt != RN_F32) return false;
#define X(ci, co) if (cin == ci && cout == co) return true;
    RN_MFMA_SHAPES(X)
#undef X
    return false;
}

bool conv_first_supported(int cin, int cout, rn_dtype dt) {
    if (dt != RN_F32) return false;
#define X(ci, co) if (cin == ci && cout == co) return true;
    RN_FIRST_SHAPES(X)
#undef X
    return false;
}

hipError_t launch_conv_mfma(const ConvArgs &a, rn_dtype dt, int grid, hipStream_t s) {
    (void)dt;
#define X(ci, co) if (a.cin == ci && a.cout == co) return run_mfma<ci, co>(a, grid, s);
    RN_MFMA_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_conv_first(const ConvArgs &a, rn_dtype dt, int grid, hipStream_t s) {
    (void)dt;
#define X(ci, co) if (a.cin == ci && a.cout == co) return run_first<ci, co>(a, grid, s);
    RN_FIRST_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

size_t conv_first_packed_elems(int cin, int cout) { return (size_t)cin * 9 * cout; }

size_t conv_mfma_packed_elems(int cin, int cout, rn_dtype dt) {
    (void)dt;
    return (size_t)9 * cin * cout;
}

void pack_conv_first(const float *oihw, int cin, int cout, rn_dtype dt, void *dst) {
    // [ci * 9 + ky * 3 + kx][co]
    (void)dt;
    float *d = static_cast<float *>(dst);
    for (int co = 0; co < cout; ++co)
        for (int ci = 0; ci < cin; ++ci)
            for (int k = 0; k < 9; ++k) d[(ci * 9 + k) * cout + co] = oihw[((size_t)co * cin + ci) * 9 + k];
}

void pack_conv_mfma(const float *oihw, int cin, int cout, rn_dtype dt, void *dst) {
    // Fragment order [kstep][nb][lane]: element B[k][n] with
    // k = kstep * 4 + lane / 16 = (ky * 3 + kx) * cin + ci, n = nb * 16 + lane % 16.
    (void)dt;
    float *d = static_cast<float *>(dst);
    const int nb_n = cout / 16, ksteps = 9 * cin / 4;
    for (int ks = 0; ks < ksteps; ++ks)
        for (int nb = 0; nb < nb_n; ++nb)
            for (int l = 0; l < 64; ++l) {
                const int k = ks * 4 + l / 16, n = nb * 16 + l % 16;
                const int kpos = k / cin, ci = k - kpos * cin;
                d[((size_t)ks * nb_n + nb) * 64 + l] = oihw[((size_t)n * cin + ci) * 9 + kpos];
            }
}

}  // namespace rn
