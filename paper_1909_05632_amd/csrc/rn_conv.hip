// Dirty-tile convolution kernels (Sec. 1: recompute only where the change can
// reach and reuse the cached activations elsewhere).
//
// A conv layer is bias and ReLU after a k x k cross-correlation with stride s
// and zero padding p:
//   out[y][x][co] = ReLU(b[co] + sum_{ky,kx,ci} w[co][ci][ky][kx] * in[s y-p+ky][s x-p+kx][ci]).
// Most kernels here are for 3x3, stride 1, pad 1 (6x6 input halo per tile); the
// general-layer kernel k_conv_gen takes other k and s.  Each work-list entry
// names one 4x4 output tile of one stream; the kernels compute its 16 pixels x
// cout outputs and write them in place into the stream's cache (scatter fused
// with bias and ReLU).
// Pixels of a ragged edge tile that fall outside the image are written as 0:
// they are the next layer's zero padding and carry zero dense weights.
//
// Cache layout ("tiled NHWC"): per slot [TH][TW][16][C], a tile's 16 pixels in
// row-major order, channels innermost; one tile is 16 * C contiguous elements.
//
// The kernels are persistent: the grid is sized to the chip and the blocks walk
// the device-side work list until the device-side count is exhausted, so no
// host synchronisation is needed to size a launch.  In dense mode (the
// comparison path) they walk every tile of every stream instead of a list;
// the arithmetic per tile is the same code, so a dense pass and a reuse pass
// give the same bits.
//
// Tile-partial head (last layer only): the dense head is linear, so the logits
// are a sum over tiles of each tile's own contribution.  The epilogue computes
// that contribution for the tiles it recomputes and stores it per (stream,
// tile); clean tiles keep theirs.  The head then only adds partials.
#include "rn_device.hpp"

namespace rn {
namespace {

using namespace dev;

// ------------------------------------------------------------------ first layer

// Direct conv for a few input channels (1, or 4 stacked frames): 9 * CIN FMAs
// per output, too few for a matrix core to pay off; the layer is HBM-bound on
// its output writes.  One wave per tile: lane l owns output channels l, l + 64
// (its 9 CIN weights in registers for the kernel's life); the 6x6 x CIN halo
// goes to LDS channel-innermost and from there, by broadcast reads, into every
// lane's registers, so the 16 x 9 CIN FMAs of a lane touch registers only.
// Each output is accumulated with fmaf over (c, ky, kx) in that order, then the
// bias is added (the order the folded layer-1 staging of the layer-2 kernel
// uses, so both give the same bits).  Stores: the lanes of one pixel write
// consecutive channels.  VAR: the tiles of variants (input from the base slot
// and the variant's frame, output to the overlay row of the work item).
template <int CIN, int COUT, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_conv_first_f32(ConvArgs a) {
    constexpr int CPL = (COUT + 63) / 64;         // channels per lane
    constexpr int HN = 36 * CIN;                  // halo values
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
    const int cin1 = CIN / a.stack;               // channels per frame
    float *halo = s_halo[wave];
    const float *xin = static_cast<const float *>(a.in);
    float *outp = static_cast<float *>(a.out);

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
                    v = var_input(a, r.slot, c, y, x);
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
                    v = plane[(size_t)y * a.W + x];
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
        float *dst = VAR ? static_cast<float *>(a.vov_out) + (size_t)t * kTilePx * COUT
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
                    dst[m * COUT + co] = v;
                }
            }
        }
        wave_sync();                                   // halo reads done before the next tile's writes
    }
}

// Layer 1 with four input channels (stacked frames, or a 4-channel input) on
// the matrix cores: for every output channel count a lane-per-channel kernel
// leaves lanes idle (40 channels use 40 of 64 lanes) and runs its FMAs at the
// VALU rate.  Per tile an implicit GEMM on v_mfma_f32_16x16x4_f32: M = 16
// pixels (row m = pixel (m / 4, m % 4)), N = COUT in blocks of 16 (padded with
// zero weights), K = 36 in (c, ky, kx) order, nine k-steps; step s gives lane
// group kq the K index 4 s + kq, a halo value gathered from LDS (offsets fixed
// per lane), and the B fragments stay in registers for the kernel's life.
// D: lane (n, kq) holds pixels 4 kq + i (row kq, column i) of channel
// 16 nb + n.  The halo prefetch and the VAR handling are those of
// k_conv_first_f32.
template <int COUT, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_conv_first4_mfma(ConvArgs a) {
    constexpr int CIN = 4, KS = 9, NB = (COUT + 15) / 16;
    constexpr int HN = 36 * CIN;                  // halo values
    constexpr int HPL = (HN + 63) / 64;
    __shared__ float s_halo[4][HN];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int mrow = lane & 15, kq = lane >> 4;
    const float *wg = static_cast<const float *>(a.w);
    float bw[KS][NB], bias[NB];
    int aoff[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int k = 4 * s + kq, c = k / 9, r = k - 9 * c, ky = r / 3, kx = r - 3 * ky;
        aoff[s] = (((mrow >> 2) + ky) * 6 + (mrow & 3) + kx) * CIN + c;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int n = 16 * nb + mrow;
            bw[s][nb] = n < COUT ? wg[k * COUT + n] : 0.f;
        }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bias[nb] = 16 * nb + mrow < COUT ? a.bias[16 * nb + mrow] : 0.f;

    const int cnt = work_count<DENSE>(a);
    const size_t HW = (size_t)a.H * a.W;
    const int cin1 = CIN / a.stack;               // channels per frame
    float *halo = s_halo[wave];
    const float *xin = static_cast<const float *>(a.in);
    float *outp = static_cast<float *>(a.out);
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
                    v = var_input(a, r.slot, c, y, x);
                } else {
                    const float *plane;
                    if (a.stack == 1) {
                        plane = xin + ((size_t)r.slot * CIN + c) * HW;
                    } else {
                        const int j = c / cin1, c1 = c - j * cin1;
                        const int rp = (head - (a.stack - 1) + j + 4 * a.stack) & 3;
                        plane = xin + (((size_t)r.slot * 4 + rp) * cin1 + c1) * HW;
                    }
                    v = plane[(size_t)y * a.W + x];
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
        float av[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) av[s] = halo[aoff[s]];
        load_tile(min(t + xr.stride, xr.end - 1), pv);
        floatx4 acc[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s], bw[s][nb], acc[nb], 0, 0, 0);
        float *dst = VAR ? static_cast<float *>(a.vov_out) + (size_t)t * kTilePx * COUT
                         : outp + (size_t)r.slot * a.out_stride + (size_t)r.tile * kTilePx * COUT;
        const bool row_in = r.ty * kTile + kq < a.H;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int n = 16 * nb + mrow;
            if (n >= COUT) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float v = acc[nb][i] + bias[nb];
                v = v > 0.0f ? v : 0.0f;
                if (!row_in || r.tx * kTile + i >= a.W) v = 0.0f;
                dst[(4 * kq + i) * COUT + n] = v;
            }
        }
        wave_sync();                                   // halo reads done before the next tile's writes
    }
}

// ------------------------------------------------------------------ MFMA layers

// Implicit GEMM per tile: M = 16 pixels, N = COUT, K = 9 * CIN.
// v_mfma_f32_16x16x4_f32 operand layout (lane l, kq = l / 16):
//   A: row l % 16, k-row kq;  B: k-row kq, column l % 16;
//   D: rows 4 kq + i, column l % 16, i = 0..3.
// Rows are tile pixels in column-major order, row m = pixel (m % 4, m / 4), so
// lane l of D holds pixels (i, kq), i = 0..3, of channel l % 16 + 16 nb.
// K is walked per kernel position in channel blocks of 16 (plus one block of
// 8 when CIN % 16 = 8).  Inside a block, k-step j gives lane group kq the
// channel c0 + 4 kq + j (c0 + 2 kq + j in a block of 8), so each lane's A
// values for the block's 4 (2) k-steps are contiguous channels of one halo
// pixel: one 16-byte (8-byte) LDS read.  The weights are packed to match,
// [kpos][block][nb][lane][j], so the B values are one 16-byte read per nb.
// Bank layout of the halo: the LDS serves 16 lanes of a 16-byte read per
// clock (64 banks), and the A reads of such a group touch 16 pixels of the
// 6x6 halo, one chunk each.  The halo is stored unpadded (pixel stride CIN,
// which lets 8 waves' halos fit in LDS next to the 40->80 weights) with the
// 16-byte chunk index of halo pixel (hy, hx) XOR-ed with g(hy, hx): hy % 2
// for 10 chunks per pixel, hy % 4 for 20, (hy % 4) + 4 (hx % 4) for 16 or
// 32; every group then falls in 16 distinct bank groups for all 9 kernel
// positions, and the 8-byte reads of the 8-channel tail block in distinct
// banks too (checked exhaustively on the host).  Blocks are double-buffered:
// the operands of the next block are read while the matrix cores work on the
// current one.
template <int CIN, int COUT>
struct Mfma {
    static constexpr int NB = COUT / 16;
    static constexpr int CS = CIN;            // halo pixel stride in LDS (floats)
    static constexpr int NF = CIN / 16;       // full channel blocks per kernel position
    static constexpr int TAIL = (CIN % 16) ? 1 : 0;
    static constexpr int NBLK = NF + TAIL;
    static constexpr int C4 = CIN / 4;        // float4 per halo pixel
    static constexpr int HALO = 36 * CS;      // floats of one halo in LDS
    static constexpr int SR = COUT + 4;       // row stride of the output staging area
    static constexpr int HV = (36 * C4 + 63) / 64;   // 16-byte halo loads per lane
    static constexpr int WTOT = 9 * CIN * COUT;
    static_assert(16 * SR <= HALO, "output staging must fit in the halo area");
    static_assert(COUT % 16 == 0 && CIN % 8 == 0, "MFMA tiling");
    static_assert(C4 == 10 || C4 == 20 || C4 == 16 || C4 == 32, "halo swizzle defined for 40, 64, 80, 128 channels");
};

// Global -> registers: the halo of one tile, 16 bytes per lane per load.
template <int CIN, int COUT, bool VAR>
__device__ inline void fetch_halo(const ConvArgs &a, const TileRef &r, float4 *regs, int lane) {
    using M = Mfma<CIN, COUT>;
    const float *src = static_cast<const float *>(a.in) + (VAR ? 0 : (size_t)r.slot * a.in_stride);
#pragma unroll
    for (int j = 0; j < M::HV; ++j) {
        const int h = lane + 64 * j;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (h < 36 * M::C4) {
            const int pos = h / M::C4, c4 = h - pos * M::C4;
            const int hy = pos / 6, hx = pos - hy * 6;
            const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
            if (y >= 0 && y < a.H && x >= 0 && x < a.W)
                v = *reinterpret_cast<const float4 *>(
                    (VAR ? var_src<float>(a, r.slot, y, x, CIN)
                         : src + ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN) +
                    c4 * 4);
        }
        regs[j] = v;
    }
}

// Offset (floats) of 16-byte channel chunk c of halo pixel p.
template <int CIN, int COUT>
__device__ inline int chunk_off(int p, int c) {
    using M = Mfma<CIN, COUT>;
    const int hy = p / 6, hx = p - 6 * hy;
    const int g = M::C4 == 10 ? (hy & 1) : M::C4 == 20 ? (hy & 3) : (hy & 3) | ((hx & 3) << 2);
    return p * M::CS + 4 * (c ^ g);
}

template <int CIN, int COUT>
__device__ inline void store_halo(float *halo, const float4 *regs, int lane) {
    using M = Mfma<CIN, COUT>;
#pragma unroll
    for (int j = 0; j < M::HV; ++j) {
        const int h = lane + 64 * j;
        if (h < 36 * M::C4) {
            const int pos = h / M::C4, c4 = h - pos * M::C4;
            *reinterpret_cast<float4 *>(halo + chunk_off<CIN, COUT>(pos, c4)) = regs[j];
        }
    }
}

// Layer 1 folded into the halo staging (one input channel): the 6x6 x CIN
// layer-1 activations around the tile are computed from the 8x8 input patch
// around it, in the same FMA order as k_conv_first_f32 (so the values are the
// bits that kernel would have cached).  Halo pixels outside the image are the
// layer-2 zero padding.
template <bool VAR>
__device__ inline float fetch_patch(const ConvArgs &a, const TileRef &r, int lane) {
    const int y = r.ty * kTile - 2 + (lane >> 3), x = r.tx * kTile - 2 + (lane & 7);
    const bool in = y >= 0 && y < a.H && x >= 0 && x < a.W;
    if constexpr (VAR) return in ? var_input(a, r.slot, 0, y, x) : 0.f;
    const float *plane = static_cast<const float *>(a.in) + (size_t)r.slot * a.in_stride;
    return in ? plane[(size_t)y * a.W + x] : 0.f;
}

// The 8x8 input patch sits in the last 64 floats of the wave's halo area
// (written there by the caller before the previous tile's epilogue, whose
// output staging ends below it).
template <int CIN, int COUT>
__device__ inline float *patch_area(float *halo) {
    return halo + Mfma<CIN, COUT>::HALO - 64;
}

template <int CIN, int COUT>
__device__ inline void build_halo_fused(float *halo, const ConvArgs &a, const TileRef &r, const float *s_w1,
                                        const float *s_b1, int lane) {
    using M = Mfma<CIN, COUT>;
    constexpr int NU = 36 * M::C4;            // 4-channel units of the halo
    constexpr int UV = (NU + 63) / 64;
    static_assert(16 * M::SR <= M::HALO - 64, "output staging must end below the patch");
    const float *patch = patch_area<CIN, COUT>(halo);
    wave_sync();
    float4 v[UV];
#pragma unroll
    for (int k = 0; k < UV; ++k) {
        const int u = lane + 64 * k;
        v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (u < NU) {
            const int pos = u / M::C4, c4 = u - pos * M::C4;
            const int hy = pos / 6, hx = pos - hy * 6;
            const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
            if (y >= 0 && y < a.H && x >= 0 && x < a.W) {
                float o[4];
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
                    const int c = 4 * c4 + cc;
                    float acc = 0.0f;
#pragma unroll
                    for (int ky = 0; ky < 3; ++ky)
#pragma unroll
                        for (int kx = 0; kx < 3; ++kx)
                            acc = fmaf(s_w1[(ky * 3 + kx) * CIN + c], patch[(hy + ky) * 8 + hx + kx], acc);
                    const float t = acc + s_b1[c];
                    o[cc] = t > 0.0f ? t : 0.0f;
                }
                v[k] = make_float4(o[0], o[1], o[2], o[3]);
            }
        }
    }
    wave_sync();                              // patch reads done before the halo overwrites it
#pragma unroll
    for (int k = 0; k < UV; ++k) {
        const int u = lane + 64 * k;
        if (u < NU) {
            const int pos = u / M::C4, c4 = u - pos * M::C4;
            *reinterpret_cast<float4 *>(halo + chunk_off<CIN, COUT>(pos, c4)) = v[k];
        }
    }
}

template <int NB>
struct BlockOps {
    float4 a;
    float4 b[NB];
};

// Operands of channel block `blk` at kernel position `kpos` (s_w holds the
// weights from kernel position k0 on).
template <int CIN, int COUT>
__device__ inline void load_block(BlockOps<Mfma<CIN, COUT>::NB> &o, const float *halo, int pix, const float *s_w,
                                  int kpos, int k0, int blk, int lane) {
    using M = Mfma<CIN, COUT>;
    const int kq = lane >> 4;
    const int ky = kpos / 3, kx = kpos - ky * 3;
    const int p = pix + ky * 6 + kx;
    const float *wb = s_w + (size_t)(kpos - k0) * CIN * COUT + blk * 16 * COUT;
    if (blk < M::NF) {
        o.a = *reinterpret_cast<const float4 *>(halo + chunk_off<CIN, COUT>(p, 4 * blk + kq));
#pragma unroll
        for (int nb = 0; nb < M::NB; ++nb)
            o.b[nb] = *reinterpret_cast<const float4 *>(wb + (nb * 64 + lane) * 4);
    } else {
        const float2 a2 = *reinterpret_cast<const float2 *>(
            halo + chunk_off<CIN, COUT>(p, 4 * blk + (kq >> 1)) + 2 * (kq & 1));
        o.a = make_float4(a2.x, a2.y, 0.f, 0.f);
#pragma unroll
        for (int nb = 0; nb < M::NB; ++nb) {
            const float2 b2 = *reinterpret_cast<const float2 *>(wb + (nb * 64 + lane) * 2);
            o.b[nb] = make_float4(b2.x, b2.y, 0.f, 0.f);
        }
    }
}

template <int CIN, int COUT>
__device__ inline void mma_block(floatx4 *acc, const BlockOps<Mfma<CIN, COUT>::NB> &o, int blk) {
    using M = Mfma<CIN, COUT>;
    const int steps = blk < M::NF ? 4 : 2;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (j >= steps) break;
        const float av = j == 0 ? o.a.x : j == 1 ? o.a.y : j == 2 ? o.a.z : o.a.w;
#pragma unroll
        for (int nb = 0; nb < M::NB; ++nb) {
            const float bv = j == 0 ? o.b[nb].x : j == 1 ? o.b[nb].y : j == 2 ? o.b[nb].z : o.b[nb].w;
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[nb], 0, 0, 0);
        }
    }
}

// acc += A(halo, kernel positions [k0, k0 + NK)) x B(weights in LDS from kernel position k0).
template <int CIN, int COUT, int NK>
__device__ inline void mfma_positions(floatx4 *acc, const float *halo, const float *s_w, int k0, int lane) {
    using M = Mfma<CIN, COUT>;
    const int mrow = lane & 15;
    const int pix = (mrow & 3) * 6 + (mrow >> 2);   // column-major pixel rows
    BlockOps<M::NB> cur, nxt;
    load_block<CIN, COUT>(cur, halo, pix, s_w, k0, k0, 0, lane);
    for (int kp = 0; kp < NK; ++kp) {
        const int kpos = k0 + kp;
#pragma unroll
        for (int blk = 0; blk < M::NBLK; ++blk) {
            if (blk + 1 < M::NBLK) load_block<CIN, COUT>(nxt, halo, pix, s_w, kpos, k0, blk + 1, lane);
            else if (kp + 1 < NK) load_block<CIN, COUT>(nxt, halo, pix, s_w, kpos + 1, k0, 0, lane);
            // Keep the next block's LDS reads ahead of this block's matrix ops
            // (the scheduler would otherwise sink them to their first use).
            __builtin_amdgcn_sched_barrier(0);
            mma_block<CIN, COUT>(acc, cur, blk);
            __builtin_amdgcn_sched_barrier(0);
            cur = nxt;
        }
    }
}

// Bias, ReLU, zero outside the image, coalesced store of the 16 x COUT tile
// through LDS (the halo area is free by now), and the tile's head partials.
// NO is the number of logits when known at compile time (0: this layer feeds
// no head partials), else -1 (a.n_out at run time).  A fixed count keeps the
// number of memory operations per tile fixed, so the next tile's waits can
// name exactly the loads they need instead of draining this tile's stores.
// VAR: work item widx of a variant list; the outputs go to overlay row widx
// (none for a last layer, which only feeds the head), the partials to row
// widx of the variant partials.
template <int COUT>
struct Epi {
    static constexpr int NB = COUT / 16;      // 16-column blocks of the 16x16x4 product
    static constexpr int SR = COUT + 4;       // row stride of the output staging area
};

template <int COUT, int NO, bool VAR>
__device__ inline void epilogue(const ConvArgs &a, const TileRef &r, floatx4 *acc, const float *s_bias,
                                float *stage, int lane, int widx) {
    using M = Epi<COUT>;
    const int mrow = lane & 15, kq = lane >> 4;       // D holds pixels (py = i, px = kq)
    // Bias, then ReLU and the zero outside the image on the bit patterns, with
    // no per-value compare into a lane mask: a float above zero has a positive
    // int pattern (zeros, negatives go to +0 under the int max), and pixels
    // outside the image are masked to +0 (all-ones / all-zero row masks; the
    // row bound is the same for the whole wave).
    const int col_keep = ~((a.W - 1 - (r.tx * kTile + kq)) >> 31);
    int keep[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) keep[i] = col_keep & ~((a.H - 1 - (r.ty * kTile + i)) >> 31);
#pragma unroll
    for (int nb = 0; nb < M::NB; ++nb) {
        const float b = s_bias[nb * 16 + mrow];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[nb][i] = __int_as_float(max(__float_as_int(acc[nb][i] + b), 0) & keep[i]);
            stage[(i * 4 + kq) * M::SR + nb * 16 + mrow] = acc[nb][i];
        }
    }
    wave_sync();
    const int n_out = NO >= 0 ? NO : a.n_out;
    if (NO != 0 && n_out > 0) {
        // Tile contribution to each logit: per-lane partial dot products, then
        // the lane sums, 8 logits at a time (lane_sums8).
        const int ntiles = a.TH * a.TW;
        for (int o0 = 0; o0 < n_out; o0 += 8) {
            float p[8];
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                // Two logits per batch: their 2 x NB weight loads are issued
                // together (indices clamped, results of absent logits dropped).
                const int oa = min(o0 + q, n_out - 1), ob = min(o0 + q + 1, n_out - 1);
                const float4 *wa = reinterpret_cast<const float4 *>(
                                       a.hw + ((size_t)oa * ntiles + r.tile) * kTilePx * COUT) + lane;
                const float4 *wb = reinterpret_cast<const float4 *>(
                                       a.hw + ((size_t)ob * ntiles + r.tile) * kTilePx * COUT) + lane;
                float4 va[M::NB], vb[M::NB];
#pragma unroll
                for (int nb = 0; nb < M::NB; ++nb) {
                    va[nb] = wa[nb * 64];
                    vb[nb] = wb[nb * 64];
                }
                float pa = 0.f, pb = 0.f;
#pragma unroll
                for (int nb = 0; nb < M::NB; ++nb) {
                    pa = fmaf(acc[nb][0], va[nb].x, pa);
                    pa = fmaf(acc[nb][1], va[nb].y, pa);
                    pa = fmaf(acc[nb][2], va[nb].z, pa);
                    pa = fmaf(acc[nb][3], va[nb].w, pa);
                    pb = fmaf(acc[nb][0], vb[nb].x, pb);
                    pb = fmaf(acc[nb][1], vb[nb].y, pb);
                    pb = fmaf(acc[nb][2], vb[nb].z, pb);
                    pb = fmaf(acc[nb][3], vb[nb].w, pb);
                }
                p[q] = pa;
                p[q + 1] = pb;
                if (o0 + q + 2 >= n_out) {
                    for (int z = q + 2; z < 8; ++z) p[z] = 0.f;
                    break;
                }
            }
            const float v = lane_sums8(p, lane);
            const int q = (lane >> 5) * 4 + ((lane >> 4) & 1) * 2 + ((lane >> 3) & 1);
            if ((lane & 7) == 0 && o0 + q < n_out) {
                float *hp = VAR ? a.vhpart + (size_t)widx * n_out
                                : a.hpart + ((size_t)r.slot * ntiles + r.tile) * n_out;
                hp[o0 + q] = v;
            }
        }
    }
    // The tile's stores go last: the next tile's waits on its own loads then
    // never have to drain them.
    if (!VAR || n_out == 0) {
        float4 *d4 = reinterpret_cast<float4 *>(
            VAR ? static_cast<float *>(a.vov_out) + (size_t)widx * kTilePx * COUT
                : static_cast<float *>(a.out) + (size_t)r.slot * a.out_stride + (size_t)r.tile * kTilePx * COUT);
#pragma unroll
        for (int j = 0; j < M::NB; ++j) {              // 16 * COUT / 4 float4 = 64 * NB
            const int o4 = lane + 64 * j;
            const int e = 4 * o4, m = e / COUT, n = e - m * COUT;
            d4[o4] = *reinterpret_cast<const float4 *>(stage + m * M::SR + n);
        }
    }
    wave_sync();
}

// Weights resident in LDS for the whole persistent kernel, 8 waves per block
// (two per SIMD: waves w and w + 4 share one); every wave walks its own tiles
// independently.  A tile's input (the next halo, or fused, the next 8x8 input
// patch) is fetched into registers a whole tile ahead.  Measured on gfx950: a
// wave's VALU work makes no progress while the other wave of its SIMD issues
// float32 matrix ops, so the two add up and the per-tile VALU work is what
// this kernel keeps small (item words 64 at a time, one per lane, read with
// readlane; the epilogue masks on bit patterns).
template <int CIN, int COUT, int WAVES>
struct Resident {
    static constexpr size_t lds_bytes =
        (size_t)(Mfma<CIN, COUT>::WTOT + WAVES * Mfma<CIN, COUT>::HALO) * sizeof(float);
};

// Item words of a wave's items, 64 at a time: lane j of chunk c holds the
// word of the wave's item 64 c + j (items past the last repeat the range's
// last word, so every load reads a valid entry).  The words of a whole chunk
// arrive in one load, long before they are read with readlane, so no per-tile
// word load is waited for.
template <bool DENSE>
__device__ inline uint32_t word_chunk(const ConvArgs &a, int first, int stride, int end, int c, int lane) {
    return item_word<DENSE>(a, (int)min((long long)first + (long long)(64 * c + lane) * stride, (long long)end - 1));
}

// Word of item j, held in chunk c0 (w0) or c0 + 1 (w1); j is wave-uniform.
__device__ inline TileRef item_of(const ConvArgs &a, uint32_t w0, uint32_t w1, int c0, int j) {
    const uint32_t src = (j >> 6) == c0 ? w0 : w1;
    return item_ref(a, (uint32_t)__builtin_amdgcn_readlane((int)src, j & 63));
}

// Halo of tile r into LDS, then the input loads of tile rn (when there is
// one) into the registers just freed (fused: the patch was written to its
// area, above the output staging, before the previous tile's epilogue).
template <int CIN, int COUT, bool FUSE, bool VAR>
__device__ inline void res_build(const ConvArgs &a, float *halo, const float *s_w1, const float *s_b1, float4 *pre,
                                 float &pin, const TileRef &r, const TileRef &rn, bool next, int lane) {
    if constexpr (FUSE) {
        if (next) pin = fetch_patch<VAR>(a, rn, lane);
        build_halo_fused<CIN, COUT>(halo, a, r, s_w1, s_b1, lane);
    } else {
        store_halo<CIN, COUT>(halo, pre, lane);
        if (next) fetch_halo<CIN, COUT, VAR>(a, rn, pre, lane);
    }
}

template <int CIN, int COUT, int WAVES, bool DENSE, bool FUSE, int NO, bool VAR>
__global__ __launch_bounds__(WAVES * 64) void k_conv_mfma_res(ConvArgs a) {
    using M = Mfma<CIN, COUT>;
    static_assert(WAVES == 8, "item mapping for two waves per SIMD");
    extern __shared__ float smem[];
    __shared__ float s_bias[COUT];
    __shared__ float s_w1[FUSE ? 9 * CIN : 1];
    __shared__ float s_b1[FUSE ? CIN : 1];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cnt = work_count<DENSE>(a);
    const XcdRangeW xr = xcd_range_simd2(cnt, wave);
    if (xr.block_first >= xr.end) return;                 // uniform per block
    const int stride = xr.stride;
    const int n_me = xr.first < xr.end ? (xr.end - xr.first + stride - 1) / stride : 0;
    float *s_w = smem;
    float *halo = smem + M::WTOT + wave * M::HALO;

    // Item words in two chunks of 64 (w0: chunk c0, w1: chunk c0 + 1); the
    // first tile's input is fetched before the weights are staged.
    int c0 = 0;
    uint32_t w0 = word_chunk<DENSE>(a, xr.first, stride, xr.end, 0, lane);
    uint32_t w1 = word_chunk<DENSE>(a, xr.first, stride, xr.end, 1, lane);
    constexpr int HVR = FUSE ? 1 : M::HV;
    float4 pre[HVR];
    float pin = 0.f;
    if (n_me > 0) {
        if constexpr (FUSE) pin = fetch_patch<VAR>(a, item_of(a, w0, w1, c0, 0), lane);
        else fetch_halo<CIN, COUT, VAR>(a, item_of(a, w0, w1, c0, 0), pre, lane);
    }
    // Weights into LDS in batches of 8 loads per thread, each batch issued
    // before any of it is written (indices past the end read the last
    // element and are not stored): a few memory round trips, not one per
    // 16 bytes.
    // The biases and the folded layer's weights (at most one value of each
    // per thread) are loaded up front, in flight with the weights below.
    static_assert(COUT <= WAVES * 64 && 9 * CIN <= WAVES * 64, "one small value per thread");
    const float bias_v = tid < COUT ? a.bias[tid] : 0.f;
    float w1_v = 0.f, b1_v = 0.f;
    if constexpr (FUSE) {
        if (tid < 9 * CIN) w1_v = a.w1[tid];
        if (tid < CIN) b1_v = a.b1[tid];
    }
    const float4 *wg = static_cast<const float4 *>(a.w);
    constexpr int NW4 = M::WTOT / 4, WPER = (NW4 + WAVES * 64 - 1) / (WAVES * 64), WB = 8;
#pragma unroll
    for (int k0 = 0; k0 < WPER; k0 += WB) {
        float4 wv[WB];
#pragma unroll
        for (int k = 0; k < WB; ++k)
            if (k0 + k < WPER) wv[k] = wg[min(tid + (k0 + k) * WAVES * 64, NW4 - 1)];
#pragma unroll
        for (int k = 0; k < WB; ++k) {
            const int j = tid + (k0 + k) * WAVES * 64;
            if (k0 + k < WPER && j < NW4) reinterpret_cast<float4 *>(s_w)[j] = wv[k];
        }
    }
    if (tid < COUT) s_bias[tid] = bias_v;
    if constexpr (FUSE) {
        if (tid < 9 * CIN) s_w1[tid] = w1_v;
        if (tid < CIN) s_b1[tid] = b1_v;
    }
    lds_barrier();                                        // the first input loads stay in flight

    if (n_me == 0) return;                                // no block barrier after this point

    // Per tile: halo (issuing the next tile's input loads first), matrix
    // work, epilogue; fused, the next patch goes to its area after the
    // epilogue, its load having had the whole tile to arrive.
    if constexpr (FUSE) patch_area<CIN, COUT>(halo)[lane] = pin;
    for (int k = 0; k < n_me; ++k) {
        if (k >= 64 * (c0 + 1)) {                         // tile k starts the next chunk of words
            w0 = w1;
            ++c0;
            w1 = word_chunk<DENSE>(a, xr.first, stride, xr.end, c0 + 1, lane);
        }
        res_build<CIN, COUT, FUSE, VAR>(a, halo, s_w1, s_b1, pre, pin, item_of(a, w0, w1, c0, k),
                                        item_of(a, w0, w1, c0, k + 1), k + 1 < n_me, lane);
        wave_sync();
        floatx4 acc[M::NB];
#pragma unroll
        for (int nb = 0; nb < M::NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // A wave in its matrix phase issues ahead of the other wave of its SIMD.
        __builtin_amdgcn_s_setprio(2);
        mfma_positions<CIN, COUT, 9>(acc, halo, s_w, 0, lane);
        __builtin_amdgcn_s_setprio(0);
        wave_sync();
        epilogue<COUT, NO, VAR>(a, item_of(a, w0, w1, c0, k), acc, s_bias, halo, lane, xr.first + k * stride);
        if constexpr (FUSE) {
            if (k + 1 < n_me) patch_area<CIN, COUT>(halo)[lane] = pin;
        }
    }
}

// Weights too large for LDS: a block works on a group of T tiles (8 for 64
// input channels, 4 for 128: the halos that fit next to the weights) and
// splits the outputs, not the tiles, across its waves (one per SIMD: the
// float32 matrix op issues at full rate from a single wave): wave w computes
// output channels [w COUT / 4, (w + 1) COUT / 4) of all T tiles.  The halos of
// the T tiles sit in LDS for the whole group (wave w fetches and stores those
// of tiles w, w + 4, ...);
// each wave streams only its quarter of the weights through its own pair of
// LDS buffers, in stages of one kernel position x SC input channels: stage
// q + 1 goes straight from global memory into the free buffer at the start of
// stage q (global_load_lds_dwordx4: no registers, no LDS store instructions)
// and the wave waits for its own loads at the end of the stage.  No wave reads
// another's weights, so the stages need no block barrier: two per group remain
// (halos read by all waves before the epilogue reuses the LDS, halos of the
// next group stored before its first stage).  Per 16-channel block a wave
// reads T halo fragments and COUT / 64 weight fragments for T x COUT / 64 x 4
// matrix ops.  Each wave fetches its halos of the next group into registers
// in the group's last stage (every load issued, out-of-image and absent ones
// from a fixed valid address and dropped when stored).
template <int CIN, int COUT>
struct Staged {
    static constexpr int SC = (CIN > 64 && CIN % 64 == 0) ? 64 : CIN;   // channels per stage
    static constexpr int NCH = CIN / SC;             // stages per kernel position
    static constexpr int NQ = 9 * NCH;               // stages per group
    static constexpr int SB = SC / 16;               // 16-channel blocks per stage
    static constexpr int NBW = COUT / 64;            // 16-output blocks per wave
    static constexpr int CW = 16 * NBW;              // output channels per wave
    static constexpr int WSW = SC * CW;              // floats per stage and wave
    static constexpr int WPW = WSW / 256;            // 1 KB wave loads per stage (16 bytes a lane)
    static constexpr int SR = CW + 4;                // row stride of a tile's output staging (floats)
    static constexpr int T = CIN <= 64 ? 8 : 4;      // tiles per group
    static constexpr int TW = T / 4;                 // halos fetched per wave
    static constexpr size_t lds_bytes = (size_t)(4 * 2 * WSW + T * Mfma<CIN, COUT>::HALO) * sizeof(float);
    static_assert(COUT % 64 == 0 && SC % 16 == 0 && WSW % 256 == 0, "whole 16-output blocks and 1 KB loads per wave");
    static_assert(4 * 16 * SR <= Mfma<CIN, COUT>::HALO, "four tiles' output staging fit one halo area");
};

// Stage q's weights for wave w (its CW output channels) straight from global
// memory into the wave's LDS buffer dst, [block][n-block][lane][4]
// (global_load_lds_dwordx4: lane i writes the 16 bytes at the wave-uniform
// base + 16 i); the WPW loads are in flight on return.
template <int CIN, int COUT>
__device__ inline void dma_wstage(const float *wg, int q, float *dst, int w, int lane) {
    using M = Mfma<CIN, COUT>;
    using S = Staged<CIN, COUT>;
    const int kpos = q / S::NCH, ch = q - kpos * S::NCH;
    const uint32_t l0 = lds_addr(dst);
#pragma unroll
    for (int j = 0; j < S::WPW; ++j) {
        const int b = j / S::NBW, nbw = j - b * S::NBW;
        lds_dma16(wg + ((size_t)(kpos * M::NBLK + ch * S::SB + b) * M::NB + w * S::NBW + nbw) * 256 + 4 * lane,
                  l0 + 1024u * j);
    }
}

// Halo of tile r into registers with every load issued; bit j of `ok` says
// whether element j counts (inside the image and `valid`).
template <int CIN, int COUT, bool VAR>
__device__ inline void fetch_halo_all(const ConvArgs &a, const TileRef &r, bool valid, floatx4 *regs, uint32_t &ok,
                                      int lane) {
    using M = Mfma<CIN, COUT>;
    static_assert(M::HV <= 32, "halo mask width");
    const float *base = static_cast<const float *>(a.in);
    ok = 0;
#pragma unroll
    for (int j = 0; j < M::HV; ++j) {
        const int h = lane + 64 * j;
        const int pos = h / M::C4, c4 = h - pos * M::C4;
        const int hy = pos / 6, hx = pos - hy * 6;
        const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
        const bool in = valid && h < 36 * M::C4 && y >= 0 && y < a.H && x >= 0 && x < a.W;
        const float *src;
        if constexpr (VAR) {
            src = in ? var_src<float>(a, r.slot, y, x, CIN) + c4 * 4 : base;
        } else {
            src = base + (in ? (size_t)r.slot * a.in_stride +
                                   ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN +
                                   c4 * 4
                             : 0);
        }
        regs[j] = *reinterpret_cast<const floatx4 *>(src);
        ok |= (uint32_t)in << j;
    }
}

template <int CIN, int COUT>
__device__ inline void store_halo_masked(float *halo, const floatx4 *regs, uint32_t ok, int lane) {
    using M = Mfma<CIN, COUT>;
#pragma unroll
    for (int j = 0; j < M::HV; ++j) {
        const int h = lane + 64 * j;
        if (h < 36 * M::C4) {
            const int pos = h / M::C4, c4 = h - pos * M::C4;
            *reinterpret_cast<floatx4 *>(halo + chunk_off<CIN, COUT>(pos, c4)) =
                (ok >> j) & 1 ? regs[j] : floatx4{0.f, 0.f, 0.f, 0.f};
        }
    }
}

// Operands of one 16-channel block: the A fragments of the T tiles and the B
// fragments of the wave's NBW output blocks.
template <int T, int NBW>
struct SplitOps {
    float4 a[T];
    float4 b[NBW];
};

// Block b of stage (kpos, ch): A from the T halos (channels of block
// ch * SB + b at kernel position kpos), B from the wave's stage buffer.
template <int CIN, int COUT, int T, int NBW>
__device__ inline void split_block(SplitOps<T, NBW> &o, const float *halos, const float *wst, int kpos, int ch, int b,
                                   int lane) {
    using M = Mfma<CIN, COUT>;
    using S = Staged<CIN, COUT>;
    static_assert(T == S::T && NBW == S::NBW, "operand shape");
    const int mrow = lane & 15, kq = lane >> 4;
    const int pix = (mrow & 3) * 6 + (mrow >> 2);   // column-major pixel rows
    const int ky = kpos / 3, kx = kpos - ky * 3;
    const int off = chunk_off<CIN, COUT>(pix + ky * 6 + kx, 4 * (ch * S::SB + b) + kq);
#pragma unroll
    for (int t = 0; t < T; ++t) o.a[t] = *reinterpret_cast<const float4 *>(halos + t * M::HALO + off);
#pragma unroll
    for (int nb = 0; nb < S::NBW; ++nb)
        o.b[nb] = *reinterpret_cast<const float4 *>(wst + ((b * S::NBW + nb) * 64 + lane) * 4);
}

template <int T, int NBW>
__device__ inline void split_mma(floatx4 (&acc)[T][NBW], const SplitOps<T, NBW> &o) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const float av = j == 0 ? o.a[t].x : j == 1 ? o.a[t].y : j == 2 ? o.a[t].z : o.a[t].w;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const float bv = j == 0 ? o.b[nb].x : j == 1 ? o.b[nb].y : j == 2 ? o.b[nb].z : o.b[nb].w;
                acc[t][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[t][nb], 0, 0, 0);
            }
        }
    }
}

// acc += the stage's channels (blocks ch * SB .. + SB) at kernel position
// kpos; `cur` holds block 0's operands on entry, each later block's are read
// during the previous block's matrix ops.
template <int CIN, int COUT, int T, int NBW>
__device__ inline void split_stage(floatx4 (&acc)[T][NBW], const float *halos, const float *wst, int kpos, int ch,
                                   int lane, SplitOps<T, NBW> &cur) {
    using S = Staged<CIN, COUT>;
    static_assert(T == S::T && NBW == S::NBW, "accumulator shape");
    SplitOps<T, NBW> nxt;
#pragma unroll
    for (int b = 0; b < S::SB; ++b) {
        if (b + 1 < S::SB) split_block<CIN, COUT, T, NBW>(nxt, halos, wst, kpos, ch, b + 1, lane);
        __builtin_amdgcn_sched_barrier(0);
        split_mma<T, NBW>(acc, cur);
        __builtin_amdgcn_sched_barrier(0);
        cur = nxt;
    }
}

// ---- staged layers, chunk-streamed form (launches without variant overlays)
//
// A block of four waves computes a group of T tiles, each wave COUT / 4 output
// channels of all of them, walking K one 16-channel chunk at a time and, within
// a chunk, the nine kernel positions (a stage = one position of one chunk:
// 4 k-steps x T x COUT / 64 matrix ops per wave).  Only three chunks of the
// group's halos are in LDS at once: chunk K is read, K + 1 is ready, K + 2 is
// in flight, each loaded straight from global memory into LDS with
// global_load_lds_dwordx4 (lane i writes 16 bytes at base + 16 i, so the
// lanes' source addresses lay out the buffer: tile t's 6 x 6 pixels x 4
// channel quads at 16-byte slot 144 t + 24 hy + 4 hx + quad; pixels outside
// the image and tiles past the end load from a zero page).  Rows padded to
// 25 or 27 slots, which put the 16 pixels of a 16-lane read in 16 distinct
// bank groups, measured no faster and with the same bank-conflict count.
// The stage sequence runs on across groups: when a chunk's last stage starts,
// the waves have read all of it, so after one block barrier it is refilled
// with the chunk three ahead (the next group's when the group runs out), 18
// stages before it is read.  Weights stream per stage through a ring of five
// LDS slots per wave (stage q + 4 loaded at the start of stage q) and each
// stage's operands are read during the previous stage's matrix ops.  The
// memory counter the waits use retires loads and stores in issue order, so
// every wait names how many later operations it may leave in flight; the work
// items are loaded into LDS the same way, and the only loads the compiler
// issues (the bias) are waited for before the first ring load.  The epilogue
// applies bias, ReLU and the zero outside the image, transposes each lane
// quad's 4 x 4 values with DPP moves so a lane holds four channels of one
// pixel, and stores 16 bytes a lane straight to the cache.  The order of the
// sums over K (chunk, then position, then channel) is the same for every T,
// so a tile's outputs do not depend on the group size a launch picks.
template <int CIN, int COUT, int T>
struct Chunked {
    static constexpr int NCH = CIN / 16;             // 16-channel chunks
    static constexpr int NQ = 9 * NCH;               // stages per group
    static constexpr int NB = COUT / 16;             // 16-output blocks
    static constexpr int NBW = COUT / 64;            // 16-output blocks per wave
    static constexpr int CW = 16 * NBW;              // output channels per wave
    static constexpr int WSW = 16 * CW;              // weight floats per stage and wave
    static constexpr int NWB = 5;                    // weight ring slots per wave
    static constexpr int WL = NWB - 2;               // stages between a weight load and its wait
    static constexpr int RS = 24;                    // 16-byte slots per halo row
    static constexpr int HT = 6 * RS;                // slots per tile of a chunk buffer
    static constexpr int HD = (T * HT * 16 + 1023) / 1024;   // 1 KB loads per chunk buffer
    static constexpr int HB = HD * 1024;             // bytes per chunk buffer
    static constexpr int HDW = (HD + 3) / 4;         // most loads of one wave per chunk
    static constexpr int HDMIN = HD / 4;             // fewest
    static constexpr int NS = T * NBW;               // 16-byte-a-lane stores per group and wave
    static constexpr size_t lds_bytes = 3 * (size_t)HB + (size_t)4 * NWB * WSW * sizeof(float) + 4 * 256;
    static_assert(CIN % 16 == 0 && COUT % 64 == 0 && NCH >= 4, "whole chunks, at least four per group");
    static_assert(WSW == 256 * NBW, "one 1 KB load per output block and stage");
    static_assert(T <= 16 && T % 4 == 0, "group size");
    static_assert(WL >= 2 && WL <= 8 && WL * NBW + HDMIN + NS <= 63, "the stage waits below assume these");
};

// Zero page (512 bytes): the source of every halo slot that holds no input
// value (chunk c reads 16 c floats further on).
__device__ __align__(16) float g_zero_page[128];

// Work items of a group, staged per wave in LDS: lane u loads the word of
// tile g + u (clamped to the last item) straight into the wave's item slot
// (global_load_lds_dword), so no register is written behind the compiler's
// back and the load is counted with the ring loads; in dense mode the words
// loaded are the stream ids and the positions are computed on reading.
template <bool DENSE>
__device__ inline const uint32_t *item_src(const ConvArgs &a, int t) {
    if constexpr (DENSE) {
        constexpr int CH = 32;                            // as item_word<true>
        const int per_chunk = CH * a.TH * a.TW;
        const int c = t / per_chunk, rr = t - c * per_chunk;
        const int nc = min(CH, a.dense_n - c * CH);
        const int tile = rr / nc;
        return reinterpret_cast<const uint32_t *>(a.ids) + c * CH + (rr - tile * nc);
    } else {
        return a.wl + t;
    }
}

template <bool DENSE>
__device__ inline uint32_t item_from(const ConvArgs &a, int t, uint32_t raw) {
    if constexpr (DENSE) {
        constexpr int CH = 32;
        const int per_chunk = CH * a.TH * a.TW;
        const int c = t / per_chunk, rr = t - c * per_chunk;
        const int nc = min(CH, a.dense_n - c * CH);
        const int tile = rr / nc;
        const int ty = tile / a.TW;
        return (raw << 16) | ((uint32_t)ty << 8) | (uint32_t)(tile - ty * a.TW);
    } else {
        return raw;
    }
}

template <bool DENSE, int T>
__device__ inline void dma_items(const ConvArgs &a, int g, int end, uint32_t dst, int lane) {
    lds_dma4(item_src<DENSE>(a, min(g + min(lane, T - 1), end - 1)), dst);
}

// Source of each of this wave's halo loads for chunk 0 of the group at g.
template <int CIN, int COUT, int T, bool DENSE>
__device__ inline void chunk_sources(const ConvArgs &a, int g, int end, const uint32_t *items,
                                     const float *(&src)[Chunked<CIN, COUT, T>::HDW], int wave, int lane) {
    using C = Chunked<CIN, COUT, T>;
    const float *in = static_cast<const float *>(a.in);
#pragma unroll
    for (int k = 0; k < C::HDW; ++k) {
        const int s = 64 * (wave + 4 * k) + lane;
        const int t = s / C::HT, rem = s - t * C::HT;
        const int hy = rem / C::RS, r2 = rem - hy * C::RS;
        const int hx = r2 >> 2, kq = r2 & 3;
        const int tc = min(t, T - 1);
        const TileRef r = item_ref(a, item_from<DENSE>(a, min(g + tc, end - 1), items[tc]));
        const int y = r.ty * kTile - 1 + hy, x = r.tx * kTile - 1 + hx;
        const bool ok = t < T && g + t < end && r2 < 24 && y >= 0 && y < a.H && x >= 0 && x < a.W;
        src[k] = ok ? in + (size_t)r.slot * a.in_stride +
                          ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN + 4 * kq
                    : g_zero_page + 4 * kq;
    }
}

// Chunk c of the halos into the chunk buffer at LDS byte address dst.
template <int CIN, int COUT, int T>
__device__ inline void dma_chunk(const float *const (&src)[Chunked<CIN, COUT, T>::HDW], int c, uint32_t dst,
                                 int wave) {
    using C = Chunked<CIN, COUT, T>;
#pragma unroll
    for (int k = 0; k < C::HDW; ++k) {
        const int j = wave + 4 * k;
        if (k + 1 < C::HDW || j < C::HD) lds_dma16(src[k] + 16 * c, dst + 1024u * j);
    }
}

// Stage s (chunk s / 9, position s % 9) of this wave's weights into the ring
// slot at LDS byte address dst, [output block][lane][4].
template <int CIN, int COUT, int T>
__device__ inline void dma_wchunk(const float *wg, int s, uint32_t dst, int wave, int lane) {
    using C = Chunked<CIN, COUT, T>;
    const int c = s / 9, kpos = s - 9 * c;
#pragma unroll
    for (int nb = 0; nb < C::NBW; ++nb)
        lds_dma16(wg + ((size_t)(kpos * C::NCH + c) * C::NB + wave * C::NBW + nb) * 256 + 4 * lane,
                  dst + 1024u * nb);
}

// A fragments of the T tiles at kernel position kpos from the chunk buffer
// (hb: this lane's slot of tile 0, position 0) and the B fragments of the
// stage's ring slot (wb: this lane's 16 bytes of output block 0).
template <int CIN, int COUT, int T>
__device__ inline void chunk_ops(SplitOps<T, Chunked<CIN, COUT, T>::NBW> &o, const float *hb, const float *wb,
                                 int kpos) {
    using C = Chunked<CIN, COUT, T>;
    const int ky = kpos / 3, kx = kpos - 3 * ky;
#pragma unroll
    for (int t = 0; t < T; ++t)
        o.a[t] = *reinterpret_cast<const float4 *>(hb + 4 * (t * C::HT + ky * C::RS + kx * 4));
#pragma unroll
    for (int nb = 0; nb < C::NBW; ++nb) o.b[nb] = *reinterpret_cast<const float4 *>(wb + 256 * nb);
}

// Parts of a stage, issued interleaved: A fragments of tiles [t0, t1), the
// B fragments, and the matrix ops of one k-step (the order of the matrix ops
// over a stage is that of split_mma).
template <int CIN, int COUT, int T, int T0, int T1>
__device__ inline void chunk_ops_a(SplitOps<T, Chunked<CIN, COUT, T>::NBW> &o, const float *hb, int kpos) {
    using C = Chunked<CIN, COUT, T>;
    const int ky = kpos / 3, kx = kpos - 3 * ky;
#pragma unroll
    for (int t = T0; t < T1; ++t)
        o.a[t] = *reinterpret_cast<const float4 *>(hb + 4 * (t * C::HT + ky * C::RS + kx * 4));
}

template <int CIN, int COUT, int T>
__device__ inline void chunk_ops_b(SplitOps<T, Chunked<CIN, COUT, T>::NBW> &o, const float *wb) {
#pragma unroll
    for (int nb = 0; nb < Chunked<CIN, COUT, T>::NBW; ++nb) o.b[nb] = *reinterpret_cast<const float4 *>(wb + 256 * nb);
}

template <int T, int NBW, int J>
__device__ inline void mma_kstep(floatx4 (&acc)[T][NBW], const SplitOps<T, NBW> &o) {
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const float av = J == 0 ? o.a[t].x : J == 1 ? o.a[t].y : J == 2 ? o.a[t].z : o.a[t].w;
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            const float bv = J == 0 ? o.b[nb].x : J == 1 ? o.b[nb].y : J == 2 ? o.b[nb].z : o.b[nb].w;
            acc[t][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[t][nb], 0, 0, 0);
        }
    }
}

// 4 x 4 transpose inside each lane quad: lane 4 m + b holds v[i] = X[i][b] on
// entry and X[b][i] on return (two exchanges, over lane bit 0 with element
// bit 0, then over lane bit 1 with element bit 1).
__device__ inline void quad_transpose(float (&v)[4], int b) {
    {
        const bool hi = b & 1;
        const float s0 = hi ? v[0] : v[1], s1 = hi ? v[2] : v[3];
        const float r0 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s0), 0xb1, 0xf, 0xf, false));
        const float r1 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s1), 0xb1, 0xf, 0xf, false));
        if (hi) {
            v[0] = r0;
            v[2] = r1;
        } else {
            v[1] = r0;
            v[3] = r1;
        }
    }
    {
        const bool hi = b & 2;
        const float s0 = hi ? v[0] : v[2], s1 = hi ? v[1] : v[3];
        const float r0 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s0), 0x4e, 0xf, 0xf, false));
        const float r1 = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(s1), 0x4e, 0xf, 0xf, false));
        if (hi) {
            v[0] = r0;
            v[1] = r1;
        } else {
            v[2] = r0;
            v[3] = r1;
        }
    }
}

template <int CIN, int COUT, bool DENSE, int T>
__device__ void chunk_path(const ConvArgs &a, int cnt, float *smem) {
    using C = Chunked<CIN, COUT, T>;
    constexpr int NBW = C::NBW;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const XcdRange xr = xcd_range(cnt, T);
    if (xr.first >= xr.end) return;                       // uniform per block
    const int mrow = lane & 15, kq = lane >> 4;
    unsigned char *lds = reinterpret_cast<unsigned char *>(smem);
    float *wring = reinterpret_cast<float *>(lds + 3 * C::HB) + wave * C::NWB * C::WSW;
    const uint32_t *items = reinterpret_cast<const uint32_t *>(lds + 3 * C::HB + 4 * C::NWB * C::WSW * 4) + 64 * wave;
    const uint32_t hlds = lds_addr(lds), wlds = lds_addr(wring), ilds = lds_addr(items);
    const float *wg = static_cast<const float *>(a.w);
    // this lane's A slot (halo pixel (mrow & 3, mrow >> 2), channel quad kq) and B slot
    const float *ha = reinterpret_cast<const float *>(lds) + 4 * ((mrow & 3) * C::RS + (mrow >> 2) * 4 + kq);
    const float *wa = wring + 4 * lane;

    // Bias of the lane's output channels, waited for before any ring load.
    float bias[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) bias[nb] = a.bias[wave * C::CW + nb * 16 + mrow];
    asm volatile("" ::"v"(bias[0]), "v"(bias[NBW - 1]));

    // Prologue: halo chunks 0-2 and weight stages 0 .. NWB - 2 of the first group.
    const float *src[C::HDW];
    dma_items<DENSE, T>(a, xr.first, xr.end, ilds, lane);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    chunk_sources<CIN, COUT, T, DENSE>(a, xr.first, xr.end, items, src, wave, lane);
#pragma unroll
    for (int k = 0; k < 3; ++k) dma_chunk<CIN, COUT, T>(src, k, hlds + k * C::HB, wave);
#pragma unroll
    for (int q = 0; q < C::NWB - 1; ++q) dma_wchunk<CIN, COUT, T>(wg, q, wlds + q * C::WSW * 4, wave, lane);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();

    int hk = 0;                                           // chunk buffer of the current chunk
    int qs = 0;                                           // ring slot of the current stage
    int dc = 3;                                           // next chunk to load (of the group at g, or, once
                                                          // past NCH, of the next group)
    SplitOps<T, NBW> cur;
    chunk_ops<CIN, COUT, T>(cur, ha, wa, 0);
    for (int g = xr.first; g < xr.end; g += xr.stride) {   // uniform per block
        const bool stores_before = g != xr.first;         // the previous group's stores are in flight
        floatx4 acc[T][NBW];
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) acc[t][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        for (int c = 0; c < C::NCH; ++c) {
#pragma unroll
            for (int kp = 0; kp < 9; ++kp) {
                if (kp == 8) {
                    // This chunk's reads are done in every wave, chunk + 1 is
                    // in LDS: its loads (issued two chunks ago) are followed
                    // by 17 stages' weight loads and one chunk's halo loads.
                    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(17 * NBW + C::HDMIN) : "memory");
                    lds_barrier();
                }
                // Matrix ops of this stage, one k-step at a time, with the
                // rest of the stage's work in between so the matrix pipe is
                // never left waiting on a burst of other instructions: stage
                // q + NWB - 1's weights into the slot stage q - 1 used (its
                // reads fed matrix ops that have issued), at a chunk boundary
                // the item and halo loads, and the next stage's operands,
                // its weights once they are in: they were loaded WL stages
                // ago and are followed by WL stages' weight loads, plus a
                // chunk's halo loads when a chunk boundary is that close,
                // plus the previous group's stores at a group's start.
                SplitOps<T, NBW> nxt;
                const int qn = qs + 1 == C::NWB ? 0 : qs + 1;
                const int hn = kp == 8 ? (hk + 1 == 3 ? 0 : hk + 1) : hk;
                const int kn = kp == 8 ? 0 : kp + 1;
                mma_kstep<T, NBW, 0>(acc, cur);
                __builtin_amdgcn_sched_barrier(0);
                const int s4 = c * 9 + kp + C::NWB - 1;
                dma_wchunk<CIN, COUT, T>(wg, s4 >= C::NQ ? s4 - C::NQ : s4,
                                         wlds + ((qs + C::NWB - 1) % C::NWB) * C::WSW * 4, wave, lane);
                if (kp == 8) {
                    // The wave's item slot: the next group's items a chunk
                    // before its halo sources are needed, then this group's
                    // for the epilogue (each followed by this boundary's halo
                    // loads and the next nine stages' weight loads).
                    const int gn = min(g + xr.stride, xr.end - 1);
                    if (c == C::NCH - 4) dma_items<DENSE, T>(a, gn, xr.end, ilds, lane);
                    if (c == C::NCH - 2) dma_items<DENSE, T>(a, g, xr.end, ilds, lane);
                    // Refill this chunk's buffer with the chunk three ahead.
                    if (dc == C::NCH) {                       // on to the next group
                        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(9 * NBW + C::HDMIN) : "memory");
                        chunk_sources<CIN, COUT, T, DENSE>(a, g + xr.stride, xr.end, items, src, wave, lane);
                        dc = 0;
                    }
                    dma_chunk<CIN, COUT, T>(src, dc, hlds + hk * C::HB, wave);
                    ++dc;
                }
                chunk_ops_a<CIN, COUT, T, 0, T / 2>(nxt, ha + hn * (C::HB / 4), kn);
                __builtin_amdgcn_sched_barrier(0);
                mma_kstep<T, NBW, 1>(acc, cur);
                __builtin_amdgcn_sched_barrier(0);
                chunk_ops_a<CIN, COUT, T, T / 2, T>(nxt, ha + hn * (C::HB / 4), kn);
                __builtin_amdgcn_sched_barrier(0);
                mma_kstep<T, NBW, 2>(acc, cur);
                __builtin_amdgcn_sched_barrier(0);
                if (kp >= C::WL && kp <= 7) {
                    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(C::WL * NBW) : "memory");
                } else if (c == 0 && kp <= C::WL - 1 && stores_before) {
                    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(C::WL * NBW + C::HDMIN + C::NS) : "memory");
                } else {
                    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(C::WL * NBW + C::HDMIN) : "memory");
                }
                chunk_ops_b<CIN, COUT, T>(nxt, wa + qn * C::WSW);
                __builtin_amdgcn_sched_barrier(0);
                mma_kstep<T, NBW, 3>(acc, cur);
                __builtin_amdgcn_sched_barrier(0);
                cur = nxt;
                qs = qn;
                hk = hn;
            }
        }
        // Epilogue: bias, ReLU and the zero outside the image on the bit
        // patterns (a float above zero has a positive int pattern), the quad
        // transpose, 16 bytes a lane: pixel (b, kq) of the tile, channels
        // 16 nb + 4 m .. + 3 of the wave's, for lane 16 kq + 4 m + b.
        const int qb = lane & 3, qm = (lane >> 2) & 3;
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(9 * NBW + 2 * C::HDMIN) : "memory");
#pragma unroll
        for (int t = 0; t < T; ++t) {
            if (g + t >= xr.end) break;                   // uniform
            const TileRef r = item_ref(a, item_from<DENSE>(a, g + t, items[t]));
            const int col_keep = ~((a.W - 1 - (r.tx * kTile + kq)) >> 31);
            float *dst = static_cast<float *>(a.out) + (size_t)r.slot * a.out_stride +
                         (size_t)r.tile * kTilePx * COUT + (qb * 4 + kq) * COUT + wave * C::CW + 4 * qm;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int keep = col_keep & ~((a.H - 1 - (r.ty * kTile + i)) >> 31);
                    v[i] = __int_as_float(max(__float_as_int(acc[t][nb][i] + bias[nb]), 0) & keep);
                }
                quad_transpose(v, qb);
                *reinterpret_cast<float4 *>(dst + 16 * nb) = make_float4(v[0], v[1], v[2], v[3]);
            }
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");      // loads issued for a group that does not come
}

template <int CIN, int COUT, bool DENSE, bool VAR>
__global__ __launch_bounds__(256) void k_conv_mfma_staged(ConvArgs a) {
    using M = Mfma<CIN, COUT>;
    using S = Staged<CIN, COUT>;
    static_assert(M::TAIL == 0, "staged layers take whole 16-channel blocks");
    extern __shared__ float smem[];
    if constexpr (!VAR) {
        // Launches without overlays stream the halos by chunk: groups of 8
        // tiles when every block has at least 16 of them to do, else of 4.
        const int cnt = work_count<DENSE>(a);
        if (cnt >= 16 * 8 * (int)gridDim.x) chunk_path<CIN, COUT, DENSE, 8>(a, cnt, smem);
        else chunk_path<CIN, COUT, DENSE, 4>(a, cnt, smem);
    } else {
    __shared__ float s_bias[COUT];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cnt = work_count<DENSE>(a);
    constexpr int T = S::T;
    const XcdRange xr = xcd_range(cnt, T);
    if (xr.first >= xr.end) return;                       // uniform per block
    float *halos = smem;                                  // tile t's halo at t * HALO
    float *wbuf = smem + T * M::HALO + wave * 2 * S::WSW; // this wave's two stage buffers
    const float *wg = static_cast<const float *>(a.w);
    for (int j = tid; j < COUT; j += blockDim.x) s_bias[j] = a.bias[j];
    const int mrow = lane & 15, kq = lane >> 4;

    // Prologue: the wave's halos (tiles wave + 4 h) of group 0; its stage 0 in LDS.
    dma_wstage<CIN, COUT>(wg, 0, wbuf, wave, lane);
    floatx4 hreg[S::TW][M::HV];
    uint32_t hok[S::TW];
#pragma unroll
    for (int h = 0; h < S::TW; ++h) {
        const int t = xr.first + wave + 4 * h;
        const uint32_t e = t < xr.end ? item_word<DENSE>(a, t) : 0u;
        fetch_halo_all<CIN, COUT, VAR>(a, item_ref(a, e), t < xr.end, hreg[h], hok[h], lane);
    }
#pragma unroll
    for (int h = 0; h < S::TW; ++h) store_halo_masked<CIN, COUT>(halos + (wave + 4 * h) * M::HALO, hreg[h], hok[h], lane);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();

    int buf = 0;
    for (int g = xr.first; g < xr.end; g += xr.stride) {   // uniform per block
        uint32_t e_nxt[S::TW];                            // the wave's items of the next group
#pragma unroll
        for (int h = 0; h < S::TW; ++h) {
            const int tn = g + xr.stride + wave + 4 * h;
            e_nxt[h] = tn < xr.end ? item_word<DENSE>(a, tn) : 0u;
        }
        uint32_t e_grp[T];                                // the group's items, for the epilogue
#pragma unroll
        for (int tt = 0; tt < T; ++tt) e_grp[tt] = g + tt < xr.end ? item_word<DENSE>(a, g + tt) : 0u;
        floatx4 acc[T][S::NBW];
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
#pragma unroll
            for (int nb = 0; nb < S::NBW; ++nb) acc[tt][nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // Three stages per loop iteration where the group has 18: rolled one
        // stage at a time the compiler permutes the accumulator registers
        // within an iteration and moves them back at its end.
        constexpr int QU = S::NQ == 18 ? 3 : 1;
#pragma unroll QU
        for (int q = 0; q < S::NQ; ++q) {
            // The stage's first operands, then stage q + 1 (wrapping into the
            // next group) straight into the wave's other buffer (its last
            // reads, of stage q - 1, fed matrix ops that have issued) and,
            // in the last stage, the wave's halos of the next group into
            // registers; then the matrix work and the wait for the weight
            // loads (the halo loads, issued after them, stay in flight: the
            // waits count in issue order).
            const int kpos = q / S::NCH, ch = q - kpos * S::NCH;
            const float *wst = wbuf + buf * S::WSW;
            SplitOps<T, S::NBW> first;
            split_block<CIN, COUT, T, S::NBW>(first, halos, wst, kpos, ch, 0, lane);
            dma_wstage<CIN, COUT>(wg, (q + 1) % S::NQ, wbuf + (buf ^ 1) * S::WSW, wave, lane);
            const bool last = q == S::NQ - 1;
            if (last) {
#pragma unroll
                for (int h = 0; h < S::TW; ++h) {
                    const int tn = g + xr.stride + wave + 4 * h;
                    fetch_halo_all<CIN, COUT, VAR>(a, item_ref(a, e_nxt[h]), tn < xr.end, hreg[h], hok[h], lane);
                }
            }
            split_stage<CIN, COUT, T, S::NBW>(acc, halos, wst, kpos, ch, lane, first);
            buf ^= 1;
            if (last) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(S::TW * M::HV) : "memory");
            else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        lds_barrier();                                    // every wave is past its last halo read
        // Epilogue, tile by tile: bias, ReLU and the zero outside the image on
        // the bit patterns (a float above zero has a positive int pattern),
        // staged through LDS rows of the wave's CW channels, then stored 16
        // bytes a lane.
#pragma unroll
        for (int tt = 0; tt < T; ++tt) {
            const int it = g + tt;
            if (it >= xr.end) break;                      // uniform
            const TileRef r = item_ref(a, e_grp[tt]);
            const int col_keep = ~((a.W - 1 - (r.tx * kTile + kq)) >> 31);
            // staging: the wave's own halo areas (tiles wave + 4 h), four tiles each
            float *stg = halos + (wave + 4 * (tt / 4)) * M::HALO + (tt % 4) * 16 * S::SR;
#pragma unroll
            for (int nb = 0; nb < S::NBW; ++nb) {
                const float bb = s_bias[(wave * S::NBW + nb) * 16 + mrow];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int keep = col_keep & ~((a.H - 1 - (r.ty * kTile + i)) >> 31);
                    stg[(i * 4 + kq) * S::SR + nb * 16 + mrow] =
                        __int_as_float(max(__float_as_int(acc[tt][nb][i] + bb), 0) & keep);
                }
            }
            wave_sync();
            float *dst = VAR ? static_cast<float *>(a.vov_out) + (size_t)it * kTilePx * COUT
                             : static_cast<float *>(a.out) + (size_t)r.slot * a.out_stride + (size_t)r.tile * kTilePx * COUT;
            if (!VAR || a.vov_out != nullptr) {
#pragma unroll
                for (int j = 0; j < S::CW / 16; ++j) {    // 16 x CW / 4 float4 = 64 x CW / 16
                    const int o4 = lane + 64 * j;
                    const int m = (4 * o4) / S::CW, n = 4 * o4 - m * S::CW;
                    *reinterpret_cast<float4 *>(dst + m * COUT + wave * S::CW + n) =
                        *reinterpret_cast<const float4 *>(stg + m * S::SR + n);
                }
            }
        }
        wave_sync();                                      // staging reads done before the halo store
#pragma unroll
        for (int h = 0; h < S::TW; ++h) store_halo_masked<CIN, COUT>(halos + (wave + 4 * h) * M::HALO, hreg[h], hok[h], lane);
        lds_barrier();                                    // the next group's halos visible to every wave
    }
    }
}

// ------------------------------------------------------------------ general layers

// Any k x k kernel with stride s and zero padding p <= (k - 1) / 2 (the growth
// rule of Fig. 1 for general k and s; DQN-style trunks: 8x8/4, 4x4/2, 3x3/1
// without padding).  A 4x4 output tile reads an E x E input patch, E = 3 s + k,
// whose corner is input pixel (4 s ty - p, 4 s tx - p); out-of-grid pixels are
// zero.  Implicit GEMM on v_mfma_f32_16x16x4_f32 (operand layout as in Mfma):
// M = 16 tile pixels (column-major rows), N = COUT, K = k k CIN in (ky, kx, c)
// order, walked in blocks of 16 K values: in block b, k-step j gives lane group
// kq the K index 16 b + 4 kq + j, so a lane's four k-steps are consecutive K
// values (four consecutive channels of one input pixel when CIN % 4 = 0: one
// 16-byte LDS read).  K is padded to a multiple of 16 with zero weights and
// zero A values.  The patch sits in LDS channel-innermost; the weights,
// packed [block][n-block][lane][j], stream from global memory (the same few
// hundred KB for every wave, served by L1/L2), one 16-byte load per lane and
// n-block, three blocks ahead of their use (a ring of three register sets
// with fixed roles, the loop unrolled by three).  A block of four waves works
// on one tile at a time and splits its K blocks four ways (these layers have
// few tiles on their small grids, so a launch lasts about one tile's latency);
// the four partial products are added in LDS in wave order and wave 0 runs
// the epilogue; the next tile's patch is fetched into registers during this
// tile's matrix work;
// the epilogue is the one of the 3x3 kernels (bias, ReLU, zero outside the
// output grid, tile head partials on the last layer, cache store).
// FIRST: the input is the float32 input cache (planar, a ring of 4 frames when
// stacking) instead of a tiled layer cache.
template <int KS, int ST, int CIN, int COUT>
struct Gen {
    static constexpr int E = 3 * ST + KS;
    static constexpr int KT = KS * KS * CIN;
    static constexpr int KSPLIT = 4;                             // waves per tile, each a quarter of K
    static constexpr int NBLK = ((KT + 15) / 16 + 11) / 12 * 12;  // 16-K blocks, padded to 4 x whole triples
    static constexpr int NBW = NBLK / KSPLIT;                    // blocks per wave
    static constexpr int NB = COUT / 16;
    static constexpr int HALO = E * E * CIN;
    static constexpr int STAGE = 16 * Epi<COUT>::SR;
    static constexpr int AREA = HALO > STAGE ? HALO : STAGE;   // floats per wave
    static constexpr int PART = (KSPLIT - 1) * NB * 64 * 4;     // partial products of waves 1..3
    static constexpr size_t lds_bytes = (size_t)(AREA + PART) * sizeof(float);
    static_assert(COUT % 16 == 0, "16-column blocks");
};

// The patch of tile r, thread idx's share (elements idx, idx + 256, ...), in
// registers: PF values per thread (scalars from the input frames, FIRST), or
// PF 16-byte channel groups (cache layers).  Every load is issued before any
// is used; out-of-image elements are zero.
template <int KS, int ST, int CIN, int COUT, bool FIRST>
struct GenPatch {
    using G = Gen<KS, ST, CIN, COUT>;
    static constexpr int N = FIRST ? G::HALO : G::E * G::E * (CIN / 4);   // elements
    static constexpr int PF = (N + 255) / 256;                            // per thread
    using T = typename std::conditional<FIRST, float, float4>::type;
};

template <int KS, int ST, int CIN, int COUT, bool FIRST>
__device__ inline void gen_fetch_patch(const ConvArgs &a, const TileRef &r,
                                       typename GenPatch<KS, ST, CIN, COUT, FIRST>::T *v, int idx) {
    using G = Gen<KS, ST, CIN, COUT>;
    using P = GenPatch<KS, ST, CIN, COUT, FIRST>;
    const int y0 = 4 * ST * r.ty - a.pad, x0 = 4 * ST * r.tx - a.pad;
    if constexpr (FIRST) {
        const float *xin = static_cast<const float *>(a.in);
        const size_t HW = (size_t)a.Hin * a.Win;
        const int cin1 = CIN / a.stack;
        const int head = a.stack != 1 ? a.ring_head[r.slot] : 0;
#pragma unroll
        for (int k = 0; k < P::PF; ++k) {
            const int h = idx + 256 * k;
            const int c = h / (G::E * G::E), pos = h - c * (G::E * G::E);
            const int hy = pos / G::E, hx = pos - hy * G::E;
            const int y = y0 + hy, x = x0 + hx;
            float val = 0.0f;
            if (h < P::N && y >= 0 && y < a.Hin && x >= 0 && x < a.Win) {
                const float *plane;
                if (a.stack == 1) {
                    plane = xin + ((size_t)r.slot * CIN + c) * HW;
                } else {
                    const int j = c / cin1, c1 = c - j * cin1;
                    const int rp = (head - (a.stack - 1) + j + 4 * a.stack) & 3;
                    plane = xin + (((size_t)r.slot * 4 + rp) * cin1 + c1) * HW;
                }
                val = plane[(size_t)y * a.Win + x];
            }
            v[k] = val;
        }
    } else {
        static_assert(CIN % 4 == 0, "cache layers carry whole 16-byte channel groups");
        constexpr int C4 = CIN / 4;
        const float *src = static_cast<const float *>(a.in) + (size_t)r.slot * a.in_stride;
#pragma unroll
        for (int k = 0; k < P::PF; ++k) {
            const int h = idx + 256 * k;
            const int pos = h / C4, c4 = h - pos * C4;
            const int hy = pos / G::E, hx = pos - hy * G::E;
            const int y = y0 + hy, x = x0 + hx;
            float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
            if (h < P::N && y >= 0 && y < a.Hin && x >= 0 && x < a.Win)
                val = *reinterpret_cast<const float4 *>(
                    src + ((size_t)((y >> 2) * a.TWin + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CIN + 4 * c4);
            v[k] = val;
        }
    }
}

// The fetched patch into LDS, channel-innermost.
template <int KS, int ST, int CIN, int COUT, bool FIRST>
__device__ inline void gen_store_patch(float *halo, const typename GenPatch<KS, ST, CIN, COUT, FIRST>::T *v, int idx) {
    using G = Gen<KS, ST, CIN, COUT>;
    using P = GenPatch<KS, ST, CIN, COUT, FIRST>;
#pragma unroll
    for (int k = 0; k < P::PF; ++k) {
        const int h = idx + 256 * k;
        if (h >= P::N) break;
        if constexpr (FIRST) {
            const int c = h / (G::E * G::E), pos = h - c * (G::E * G::E);
            halo[pos * CIN + c] = v[k];
        } else {
            constexpr int C4 = CIN / 4;
            const int pos = h / C4, c4 = h - pos * C4;
            *reinterpret_cast<float4 *>(halo + pos * CIN + 4 * c4) = v[k];
        }
    }
}


// A values of block b for this lane: K = 16 b + 4 kq + j, j = 0..3, of tile
// pixel (py, px).
template <int KS, int ST, int CIN, int COUT>
__device__ inline float4 gen_a(const float *halo, int b, int kq, int py, int px) {
    using G = Gen<KS, ST, CIN, COUT>;
    const int K0 = 16 * b + 4 * kq;
    if constexpr (CIN % 4 == 0) {
        if (K0 >= G::KT) return make_float4(0.f, 0.f, 0.f, 0.f);
        const int kpos = K0 / CIN, c = K0 - kpos * CIN;
        const int ky = kpos / KS, kx = kpos - ky * KS;
        return *reinterpret_cast<const float4 *>(halo + ((py * ST + ky) * G::E + px * ST + kx) * CIN + c);
    } else {
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int K = K0 + j < G::KT ? K0 + j : G::KT - 1;   // padded K: an in-patch address, value 0
            const int kpos = K / CIN, c = K - kpos * CIN;
            const int ky = kpos / KS, kx = kpos - ky * KS;
            const float hv = halo[((py * ST + ky) * G::E + px * ST + kx) * CIN + c];
            v[j] = K0 + j < G::KT ? hv : 0.f;
        }
        return make_float4(v[0], v[1], v[2], v[3]);
    }
}

template <int KS, int ST, int CIN, int COUT, bool DENSE, bool FIRST>
__global__ __launch_bounds__(256) void k_conv_gen(ConvArgs a) {
    using G = Gen<KS, ST, CIN, COUT>;
    extern __shared__ float smem[];
    __shared__ float s_bias[COUT];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int j = tid; j < COUT; j += blockDim.x) s_bias[j] = a.bias[j];
    float *halo = smem;                                   // patch, then the epilogue's staging
    floatx4 *part = reinterpret_cast<floatx4 *>(smem + G::AREA);
    const floatx4 *wg = static_cast<const floatx4 *>(a.w);
    const int cnt = work_count<DENSE>(a);
    const XcdRange xr = xcd_range(cnt, 1);
    const int m = lane & 15, kq = lane >> 4;
    const int py = m & 3, px = m >> 2;
    const int b0 = wave * G::NBW;                         // this wave's K blocks [b0, b0 + NBW)
    // The next tile's patch is fetched into registers while this tile's
    // matrix work runs (past the end: the last tile again, never used).
    using P = GenPatch<KS, ST, CIN, COUT, FIRST>;
    typename P::T pv[P::PF];
    if (xr.first < xr.end) gen_fetch_patch<KS, ST, CIN, COUT, FIRST>(a, decode<DENSE>(a, xr.first), pv, tid);
    for (int t = xr.first; t < xr.end; t += xr.stride) {  // uniform per block
        const TileRef r = decode<DENSE>(a, t);
        lds_barrier();                                    // the previous tile's epilogue is done with the area
        gen_store_patch<KS, ST, CIN, COUT, FIRST>(halo, pv, tid);
        gen_fetch_patch<KS, ST, CIN, COUT, FIRST>(a, decode<DENSE>(a, min(t + xr.stride, xr.end - 1)), pv, tid);
        lds_barrier();
        floatx4 acc[G::NB];
#pragma unroll
        for (int nb = 0; nb < G::NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // Weight ring: block b's fragments live in set (b - b0) % 3 (ext-vector arrays stay in registers).
        floatx4 w0[G::NB], w1[G::NB], w2[G::NB];
        auto fetch = [&](floatx4 *dst, int b) __attribute__((always_inline)) {
            const int bb = b < b0 + G::NBW ? b : b0 + G::NBW - 1;   // past this wave's range: unused
#pragma unroll
            for (int nb = 0; nb < G::NB; ++nb) dst[nb] = wg[(bb * G::NB + nb) * 64 + lane];
        };
        auto block = [&](floatx4 *w, int b) __attribute__((always_inline)) {
            const float4 av = gen_a<KS, ST, CIN, COUT>(halo, b, kq, py, px);
            const float al[4] = {av.x, av.y, av.z, av.w};
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int nb = 0; nb < G::NB; ++nb)
                    acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(al[j], w[nb][j], acc[nb], 0, 0, 0);
        };
        fetch(w0, b0);
        fetch(w1, b0 + 1);
        fetch(w2, b0 + 2);
#pragma unroll 1
        for (int b = b0; b < b0 + G::NBW; b += 3) {
            block(w0, b);
            fetch(w0, b + 3);
            block(w1, b + 1);
            fetch(w1, b + 4);
            block(w2, b + 2);
            fetch(w2, b + 5);
        }
        if (wave > 0) {
#pragma unroll
            for (int nb = 0; nb < G::NB; ++nb) part[((wave - 1) * G::NB + nb) * 64 + lane] = acc[nb];
        }
        lds_barrier();
        if (wave == 0) {
#pragma unroll
            for (int w = 0; w < G::KSPLIT - 1; ++w)
#pragma unroll
                for (int nb = 0; nb < G::NB; ++nb) acc[nb] += part[(w * G::NB + nb) * 64 + lane];
            epilogue<COUT, -1, false>(a, r, acc, s_bias, halo, lane, t);
        }
    }
}

// ------------------------------------------------------------------ dispatch

constexpr size_t kLdsBudget = 160 * 1024 - 1024;   // 160 KiB per CU, less the static arrays

template <int CIN, int COUT>
constexpr bool use_resident() { return Resident<CIN, COUT, 8>::lds_bytes <= kLdsBudget; }

// Static LDS of the fused variant: bias, layer-1 weights and bias.
template <int CIN, int COUT>
constexpr bool fused_fits() {
    return Resident<CIN, COUT, 8>::lds_bytes + (COUT + 10 * CIN) * sizeof(float) <= 160 * 1024;
}

template <int CIN, int COUT, bool DENSE, bool FUSE, int NO, bool VAR>
hipError_t run_resident_no(const ConvArgs &a, int cus, hipStream_t s) {
    constexpr size_t lds = Resident<CIN, COUT, 8>::lds_bytes;
    auto kern = k_conv_mfma_res<CIN, COUT, 8, DENSE, FUSE, NO, VAR>;
    static hipError_t attr = set_lds(kern, lds);
    if (attr != hipSuccess) return attr;
    const int grid = persistent_grid(cus, (a.max_tiles + 7) / 8);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(512), lds, s, a);
    return hipGetLastError();
}

// Logit count as a template argument where it is a common one.
template <int CIN, int COUT, bool DENSE, bool FUSE, bool VAR>
hipError_t run_resident(const ConvArgs &a, int cus, hipStream_t s) {
    if (a.n_out == 0) return run_resident_no<CIN, COUT, DENSE, FUSE, 0, VAR>(a, cus, s);
    if (a.n_out == 6) return run_resident_no<CIN, COUT, DENSE, FUSE, 6, VAR>(a, cus, s);
    return run_resident_no<CIN, COUT, DENSE, FUSE, -1, VAR>(a, cus, s);
}

template <int CIN, int COUT, bool DENSE, bool VAR>
hipError_t run_mfma(const ConvArgs &a, int cus, hipStream_t s) {
    if constexpr (use_resident<CIN, COUT>()) {
        if (a.fuse_first) return run_resident<CIN, COUT, DENSE, true, VAR>(a, cus, s);
        return run_resident<CIN, COUT, DENSE, false, VAR>(a, cus, s);
    } else {
        if (a.fuse_first || a.n_out > 0) return hipErrorInvalidValue;   // head partials come from their own kernel
        constexpr size_t lds = VAR ? Staged<CIN, COUT>::lds_bytes : Chunked<CIN, COUT, 8>::lds_bytes;
        static_assert(lds <= kLdsBudget && Chunked<CIN, COUT, 4>::lds_bytes <= lds, "staged layer exceeds LDS");
        auto kern = k_conv_mfma_staged<CIN, COUT, DENSE, VAR>;
        static hipError_t attr = set_lds(kern, lds);
        if (attr != hipSuccess) return attr;
        const int grid = persistent_grid(cus, (a.max_tiles + Staged<CIN, COUT>::T - 1) / Staged<CIN, COUT>::T);
        hipLaunchKernelGGL(kern, dim3(grid), dim3(256), lds, s, a);
    }
    return hipGetLastError();
}

template <int CIN, int COUT, bool DENSE, bool VAR>
hipError_t run_first(const ConvArgs &a, int cus, hipStream_t s) {
    const int total_max = a.max_tiles;
    if constexpr (CIN == 4) {
        // about 100-150 registers: four blocks of four waves are resident per CU
        const int grid = persistent_grid(cus * 4, (total_max + 3) / 4);
        hipLaunchKernelGGL((k_conv_first4_mfma<COUT, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    } else {
        const int grid = persistent_grid(cus * 8, (total_max + 3) / 4);
        hipLaunchKernelGGL((k_conv_first_f32<CIN, COUT, DENSE, VAR>), dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

#define RN_MFMA_SHAPES(X) X(40, 80) X(64, 128) X(128, 128)
// General layers: (k, stride, cin, cout); first layers read the input frames.
#define RN_GEN_FIRST_SHAPES(X) X(8, 4, 4, 32) X(8, 4, 1, 32) X(5, 1, 1, 32) X(7, 2, 1, 32) X(5, 2, 4, 32)
#define RN_GEN_SHAPES(X) X(4, 2, 32, 64) X(3, 1, 64, 64) X(3, 1, 32, 64) X(3, 2, 32, 64) X(5, 2, 32, 64) X(5, 1, 32, 32)

template <int KS, int ST, int CIN, int COUT, bool FIRST>
hipError_t run_gen(const ConvArgs &a, int cus, hipStream_t s) {
    using G = Gen<KS, ST, CIN, COUT>;
    const bool dense = a.wl == nullptr;
    auto kern = dense ? k_conv_gen<KS, ST, CIN, COUT, true, FIRST> : k_conv_gen<KS, ST, CIN, COUT, false, FIRST>;
    static hipError_t attr = set_lds(k_conv_gen<KS, ST, CIN, COUT, true, FIRST>, G::lds_bytes);
    static hipError_t attr2 = set_lds(k_conv_gen<KS, ST, CIN, COUT, false, FIRST>, G::lds_bytes);
    if (attr != hipSuccess) return attr;
    if (attr2 != hipSuccess) return attr2;
    // As many blocks as the CUs hold at once (registers and LDS decide), so
    // every block starts in the first generation and walks several tiles.
    static int occ = [] {
        int b = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, k_conv_gen<KS, ST, CIN, COUT, false, FIRST>,
                                                         64 * G::KSPLIT, G::lds_bytes) != hipSuccess || b < 1)
            b = 2;
        return b;
    }();
    const int grid = persistent_grid(cus * occ, a.max_tiles);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * G::KSPLIT), G::lds_bytes, s, a);
    return hipGetLastError();
}
#define RN_FIRST_SHAPES(X) X(1, 20) X(1, 40) X(1, 64) X(1, 80) X(4, 20) X(4, 40) X(4, 64) X(4, 80)

}  // namespace

bool conv_gen_supported(int k, int s, int cin, int cout, bool first) {
#define X(kk, ss, ci, co) if (k == kk && s == ss && cin == ci && cout == co) return true;
    if (first) {
        RN_GEN_FIRST_SHAPES(X)
    } else {
        RN_GEN_SHAPES(X)
    }
#undef X
    return false;
}

hipError_t launch_conv_gen(const ConvArgs &a, int k, int s, bool first, int cus, hipStream_t st) {
#define X(kk, ss, ci, co) \
    if (k == kk && s == ss && a.cin == ci && a.cout == co) return run_gen<kk, ss, ci, co, FIRSTV>(a, cus, st);
    if (first) {
#define FIRSTV true
        RN_GEN_FIRST_SHAPES(X)
#undef FIRSTV
    } else {
#define FIRSTV false
        RN_GEN_SHAPES(X)
#undef FIRSTV
    }
#undef X
    return hipErrorInvalidValue;
}

// 16-K blocks of a general layer, padded like Gen::NBLK (four waves x whole
// triples of the kernel's weight ring).
static int gen_blocks(int k, int cin) { return ((k * k * cin + 15) / 16 + 11) / 12 * 12; }

size_t conv_gen_packed_elems(int k, int cin, int cout) { return (size_t)gen_blocks(k, cin) * 16 * cout; }
#define X(kk, ss, ci, co) static_assert(Gen<kk, ss, ci, co>::NBLK == ((kk * kk * ci + 15) / 16 + 11) / 12 * 12, "padding");
RN_GEN_FIRST_SHAPES(X)
RN_GEN_SHAPES(X)
#undef X

void pack_conv_gen(const float *oihw, int k, int cin, int cout, float *dst) {
    // [block][n-block][lane][j]: K = 16 block + 4 (lane / 16) + j in (ky, kx, c)
    // order, n = 16 n-block + lane % 16; zero past K = k k cin.
    const int kt = k * k * cin, nblk = gen_blocks(k, cin), nbn = cout / 16;
    size_t o = 0;
    for (int b = 0; b < nblk; ++b)
        for (int nb = 0; nb < nbn; ++nb)
            for (int l = 0; l < 64; ++l)
                for (int j = 0; j < 4; ++j) {
                    const int K = 16 * b + 4 * (l / 16) + j, n = nb * 16 + l % 16;
                    float v = 0.f;
                    if (K < kt) {
                        const int kpos = K / cin, c = K % cin, ky = kpos / k, kx = kpos % k;
                        v = oihw[(((size_t)n * cin + c) * k + ky) * k + kx];
                    }
                    dst[o++] = v;
                }
}

bool conv_mfma_supported(int cin, int cout, rn_dtype dt) {
    if (dt != RN_F32) return false;
#define X(ci, co) if (cin == ci && cout == co) return true;
    RN_MFMA_SHAPES(X)
#undef X
    return false;
}

bool conv_fused_first_supported(int c1, int c2, rn_dtype dt) {
    if (dt != RN_F32) return false;
#define X(ci, co) if (c1 == ci && c2 == co) return use_resident<ci, co>() && fused_fits<ci, co>();
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

// cus: compute units of the device; the persistent grid is at most one block
// (resident or staged MFMA kernel) or eight blocks (first layer) per CU.
hipError_t launch_conv_mfma(const ConvArgs &a, rn_dtype dt, int cus, hipStream_t s, bool var) {
    (void)dt;
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
#define X(ci, co)                                                                          \
    if (a.cin == ci && a.cout == co)                                                       \
        return var ? run_mfma<ci, co, false, true>(a, cus, s)                              \
                   : dense ? run_mfma<ci, co, true, false>(a, cus, s) : run_mfma<ci, co, false, false>(a, cus, s);
    RN_MFMA_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_conv_first(const ConvArgs &a, rn_dtype dt, int cus, hipStream_t s, bool var) {
    (void)dt;
    const bool dense = a.wl == nullptr;
    if (var && dense) return hipErrorInvalidValue;
#define X(ci, co)                                                                          \
    if (a.cin == ci && a.cout == co)                                                       \
        return var ? run_first<ci, co, false, true>(a, cus, s)                             \
                   : dense ? run_first<ci, co, true, false>(a, cus, s) : run_first<ci, co, false, false>(a, cus, s);
    RN_FIRST_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

bool conv_mfma_is_staged(int cin, int cout) {
#define X(ci, co) \
    if (cin == ci && cout == co) return !use_resident<ci, co>();
    RN_MFMA_SHAPES(X)
#undef X
    return false;
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
    // [kpos][block][nb][lane][j]: block b of a kernel position covers channels
    // [16 b, 16 b + 16) (the last block [16 nf, 16 nf + 8) when cin % 16 = 8);
    // element j of lane l is B[channel][n] with n = nb * 16 + l % 16 and
    // channel = 16 b + 4 (l / 16) + j (block of 8: 16 nf + 2 (l / 16) + j).
    (void)dt;
    float *d = static_cast<float *>(dst);
    const int nb_n = cout / 16, nf = cin / 16;
    size_t o = 0;
    for (int kpos = 0; kpos < 9; ++kpos) {
        for (int b = 0; b < nf + (cin % 16 ? 1 : 0); ++b) {
            const bool full = b < nf;
            const int steps = full ? 4 : 2;
            for (int nb = 0; nb < nb_n; ++nb)
                for (int l = 0; l < 64; ++l)
                    for (int j = 0; j < steps; ++j) {
                        const int ci = 16 * b + (full ? 4 : 2) * (l / 16) + j;
                        const int n = nb * 16 + l % 16;
                        d[o++] = oihw[((size_t)n * cin + ci) * 9 + kpos];
                    }
        }
    }
}

size_t tile_head_w_elems(int ntiles, int cout, int n_out) { return (size_t)n_out * ntiles * kTilePx * cout; }

void pack_tile_head(const float *dense_w, int n_out, int C, int H, int W, int TH, int TW, float *dst) {
    // [o][tile][nb][lane][i]: the weight of the output the MFMA epilogue holds
    // in lane `lane`, register i of block nb: channel nb * 16 + lane % 16,
    // tile pixel (row i, column lane / 16).  Zero outside the image.
    const int NB = C / 16, ntiles = TH * TW;
    for (int o = 0; o < n_out; ++o)
        for (int t = 0; t < ntiles; ++t) {
            const int ty = t / TW, tx = t % TW;
            for (int nb = 0; nb < NB; ++nb)
                for (int l = 0; l < 64; ++l)
                    for (int i = 0; i < 4; ++i) {
                        const int c = nb * 16 + l % 16, y = ty * kTile + i, x = tx * kTile + l / 16;
                        const size_t di = ((((size_t)o * ntiles + t) * NB + nb) * 64 + l) * 4 + i;
                        dst[di] = (y < H && x < W) ? dense_w[(size_t)o * C * H * W + ((size_t)c * H + y) * W + x]
                                                   : 0.f;
                    }
        }
}

}  // namespace rn
