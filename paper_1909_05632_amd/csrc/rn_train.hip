// Training kernels (Sec. 2: the policy is trained with REINFORCE; within a
// rollout the weights are fixed, so the forward steps reuse activations as in
// inference, and the gradient of a step is taken from the activations the
// caches then hold).
//
// For a batch of streams and given dJ/dlogits g, backpropagation through
// logits = Wd a_L + bd and a_l = ReLU(conv(a_{l-1}, W_l) + b_l):
//   head:   dWd (+)= sum_i g_i a_L,i^T,  dbd (+)= sum_i g_i,
//           dz_L = (Wd^T g_i) where a_L > 0 (the ReLU derivative, 0 at the kink);
//   layer l: dW_l (+)= sum over pixels of dz_l x im2col(a_{l-1}), db_l (+)= sum dz_l,
//           dz_{l-1} = (transposed conv of dz_l with W_l) where a_{l-1} > 0.
// Both conv products run on the float32 matrix cores (v_mfma_f32_16x16x4_f32):
//   dx: per 4x4 tile of layer l-1 an implicit GEMM, M = 16 pixels, N = C_{l-1},
//       K = 9 C_l, i.e. a forward 3x3 conv of dz_l with the weights transposed
//       (input <-> output channels) and flipped (kernel position 8 - k);
//   dW: M = C_l, N = 9 C_{l-1} + 1 (the last column, all ones, gives the bias
//       gradient), K = every pixel of every stream, split over teams of blocks
//       whose partial sums are added in team order (no atomics, so the result
//       is deterministic).
// The SGD step updates every packed copy of a weight in place.
#include <type_traits>

#include "rn_device.hpp"
#include "rn_train.hpp"

namespace rn {
namespace {

using dev::floatx4;

// ------------------------------------------------------------------ REINFORCE

// g[i][o] = G_i (softmax(z_i)[o] - [o == a_i]): the derivative of
// -G_i log softmax(z_i)[a_i] with respect to z_i (one thread per stream).
__global__ __launch_bounds__(256) void k_reinforce(int n, int n_out, const float *z, const int32_t *act,
                                                   const float *ret, float *g) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float *zi = z + (size_t)i * n_out;
    float m = zi[0];
    for (int o = 1; o < n_out; ++o) m = fmaxf(m, zi[o]);
    float den = 0.f;
    for (int o = 0; o < n_out; ++o) den += expf(zi[o] - m);
    const float G = ret[i];
    const int a = act[i];
    for (int o = 0; o < n_out; ++o) {
        const float p = expf(zi[o] - m) / den;
        g[(size_t)i * n_out + o] = G * (p - (o == a ? 1.f : 0.f));
    }
}

// ------------------------------------------------------------------ dense head

// Block (t, c) takes blockDim.x V of the 16 C head inputs of tile position t
// of the last layer (chunk c); a thread owns V consecutive inputs j (one
// 16-byte access per stream for V = 4), keeps their NO weights and NO
// gradient sums in registers and walks the streams (their g rows staged in
// LDS).  Each input's sums run over o and over the streams in order, whatever
// V is.
template <int NO, int V>
__global__ __launch_bounds__(512) void k_bwd_head(HeadBwdArgs a) {
    static_assert(V == 1 || V == 4, "one float or one float4 per thread");
    using VT = typename std::conditional<V == 4, float4, float>::type;
    constexpr int kHeadStreams = NO <= 32 ? 256 : 128;    // streams per LDS stage of g (32 KB at most)
    __shared__ float s_g[kHeadStreams * NO];
    __shared__ int32_t s_slot[kHeadStreams];
    const int t = blockIdx.x;
    const int E = kTilePx * a.C;                          // a multiple of V
    const int ty = t / a.TW, tx = t - ty * a.TW;
    {
        const int j0 = (blockIdx.y * blockDim.x + threadIdx.x) * V;
        const bool ok = j0 < E;
        float w[V][NO], acc[V][NO];
#pragma unroll
        for (int v = 0; v < V; ++v)
#pragma unroll
            for (int o = 0; o < NO; ++o) {
                w[v][o] = ok && o < a.n_out ? a.wd[(size_t)o * a.K + (size_t)t * E + j0 + v] : 0.f;
                acc[v][o] = 0.f;
            }
        for (int i0 = 0; i0 < a.n; i0 += kHeadStreams) {
            const int nc = min(kHeadStreams, a.n - i0);
            __syncthreads();                      // the previous stage's readers are done
            for (int k = threadIdx.x; k < nc * NO; k += blockDim.x) {
                const int ii = k / NO, o = k - ii * NO;
                s_g[k] = o < a.n_out ? a.g[(size_t)(i0 + ii) * a.n_out + o] : 0.f;
            }
            for (int k = threadIdx.x; k < nc; k += blockDim.x) s_slot[k] = a.ids[i0 + k];
            __syncthreads();
            if (ok) {
#pragma unroll 4
                for (int ii = 0; ii < nc; ++ii) {
                    const VT in = *reinterpret_cast<const VT *>(a.act + (size_t)s_slot[ii] * a.act_stride + (size_t)t * E + j0);
                    const float *vin = reinterpret_cast<const float *>(&in);
                    VT out;
                    float *vout = reinterpret_cast<float *>(&out);
#pragma unroll
                    for (int v = 0; v < V; ++v) {
                        float da = 0.f;
#pragma unroll
                        for (int o = 0; o < NO; ++o) {
                            const float gv = s_g[ii * NO + o];
                            da = fmaf(w[v][o], gv, da);
                            acc[v][o] = fmaf(gv, vin[v], acc[v][o]);
                        }
                        vout[v] = vin[v] > 0.f ? da : 0.f;
                    }
                    *reinterpret_cast<VT *>(a.dz + ((size_t)(i0 + ii) * a.ntiles + t) * E + j0) = out;
                }
            }
        }
        if (ok) {
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int j = j0 + v, m = j / a.C, c = j - m * a.C;
                const int y = ty * kTile + (m >> 2), x = tx * kTile + (m & 3);
                if (y < a.H && x < a.W) {
#pragma unroll
                    for (int o = 0; o < NO; ++o) {
                        if (o >= a.n_out) break;
                        float *d = a.gwd + (size_t)o * a.C * a.H * a.W + ((size_t)c * a.H + y) * a.W + x;
                        *d = a.accumulate ? *d + acc[v][o] : acc[v][o];
                    }
                }
            }
        }
    }
    if (t == 0 && blockIdx.y == 0 && (int)threadIdx.x < a.n_out) {
        float s = 0.f;
        for (int i = 0; i < a.n; ++i) s += a.g[(size_t)i * a.n_out + threadIdx.x];
        a.gbd[threadIdx.x] = a.accumulate ? a.gbd[threadIdx.x] + s : s;
    }
}

// ------------------------------------------------------------------ dx

// Offset (floats) of 16-byte channel chunk c4 of halo pixel p (6x6 halo,
// pixel stride CZ): the chunk index XOR-ed with a function of the pixel, so
// the 16 pixels one 16-lane group reads at a kernel position fall in distinct
// bank groups (the scheme of the forward MFMA kernels).
template <int CZ>
__device__ inline int hoff(int p, int c4) {
    constexpr int C4 = CZ / 4;
    static_assert(C4 == 10 || C4 == 20 || C4 == 16 || C4 == 32, "halo swizzle defined for 40, 64, 80, 128 channels");
    const int hy = p / 6, hx = p - 6 * hy;
    const int g = C4 == 10 ? (hy & 1) : C4 == 20 ? (hy & 3) : (hy & 3) | ((hx & 3) << 2);
    return p * CZ + 4 * (c4 ^ g);
}

// Input gradients dz_{l-1} = (W_l^T * dz_l) where a_{l-1} > 0, as a forward
// convolution of dz_l (CZ channels) with the transposed, flipped weights
// (pack_dx_weights) into CA channels.  A block works on a group of WV tiles
// of layer l-1 (one per wave: 8 where two weight stages and eight halos fit
// one CU's LDS, so two waves per SIMD, else 4) and streams the weights
// through LDS in stages of one kernel position x SC channels of dz_l, two
// buffers: stage q + 1 goes straight from global memory into the free buffer
// at the start of stage q (lds_dma16, the block's loads split over its
// waves), each wave waits for its own loads and a block barrier ends the
// stage.  So each weight byte brought from L2 serves WV tiles.  Each wave
// keeps its tile's 6x6 x CZ halo of dz_l in its own LDS area (the next
// group's fetched into registers three stages before the group ends, stored
// after the epilogue: fetched in the last stage it arrived late, 14% of the
// time).  Operand layout of v_mfma_f32_16x16x4_f32 as in the forward
// kernels: A row m = tile pixel (m % 4, m / 4), lane group kq takes
// K = 16 b + 4 kq + j; D lane (n, kq) holds pixels (i, kq), i = 0..3, of
// output channel 16 nb + n.
template <int CZ, int CA>
struct Dx {
    static constexpr int NB = (CA + 15) / 16;   // 16-column output blocks (CA padded with zero weights)
    static constexpr int SC = (CZ > 64 && CZ % 64 == 0) ? 64 : CZ;   // channels of dz_l per stage
    static constexpr int NCH = CZ / SC;         // stages per kernel position
    static constexpr int NQ = 9 * NCH;          // stages per group
    static constexpr int SB = SC / 16;          // 16-deep K blocks per stage
    static constexpr int KBP = CZ / 16;         // K blocks per kernel position
    static constexpr int WL = SB * NB;          // 1 KB wave loads per stage
    static constexpr int WST = WL * 256;        // floats per stage
    static constexpr int HALO = 36 * CZ;        // floats of one tile's halo
    static constexpr int HV = (9 * CZ + 63) / 64;   // 16-byte halo loads per lane
    // waves (tiles of a group) per block: 8 where two weight stages and 8 halos fit one CU
    static constexpr int WV = (2 * WST + 8 * HALO) * 4 <= 160 * 1024 ? 8 : 4;
    static constexpr size_t lds_bytes = (size_t)(2 * WST + WV * HALO) * sizeof(float);
    static_assert(CZ % 16 == 0 && SC % 16 == 0, "whole 16-channel K blocks per stage");
    static_assert(CA % 4 == 0, "whole 16-byte channel groups in the epilogue");
    static_assert(HV <= 32, "halo mask width");
};

template <int CZ, int CA>
__device__ inline void dx_fetch_halo(const BwdArgs &a, int tid, bool valid, float4 *regs, uint32_t &ok, int lane) {
    using D = Dx<CZ, CA>;
    constexpr int C4 = CZ / 4;
    const int i = valid ? tid / a.ntiles : 0, t = valid ? tid - i * a.ntiles : 0;
    const int ty = t / a.TW, tx = t - ty * a.TW;
    const float *src = a.dz_in + (size_t)i * a.ntiles * kTilePx * CZ;
    ok = 0;
#pragma unroll
    for (int k = 0; k < D::HV; ++k) {
        const int e = lane + 64 * k;
        const int pos = e / C4, c4 = e - pos * C4;
        const int y = ty * kTile - 1 + pos / 6, x = tx * kTile - 1 + pos % 6;
        const bool in = valid && e < 36 * C4 && y >= 0 && y < a.H && x >= 0 && x < a.W;
        // every load issued (an absent one reads the tile's first chunk)
        regs[k] = *reinterpret_cast<const float4 *>(
            src + (in ? ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CZ + 4 * c4 : 0));
        ok |= (uint32_t)in << k;
    }
}

template <int CZ, int CA>
__device__ inline void dx_store_halo(float *halo, const float4 *regs, uint32_t ok, int lane) {
    using D = Dx<CZ, CA>;
    constexpr int C4 = CZ / 4;
#pragma unroll
    for (int k = 0; k < D::HV; ++k) {
        const int e = lane + 64 * k;
        if (e < 36 * C4) {
            const int pos = e / C4, c4 = e - pos * C4;
            *reinterpret_cast<float4 *>(halo + hoff<CZ>(pos, c4)) = (ok >> k) & 1 ? regs[k] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
}

// The block's share of stage q's weights straight into LDS: wave w issues
// the stage's wave loads w, w + 4, ...
template <int CZ, int CA>
__device__ inline void dx_dma_stage(const float *wt, int q, float *dst, int wave, int lane) {
    using D = Dx<CZ, CA>;
    const int kpos = q / D::NCH, ch = q - kpos * D::NCH;
    const float *src = wt + (size_t)(kpos * D::KBP + ch * D::SB) * D::NB * 256;
    const uint32_t l0 = dev::lds_addr(dst);
#pragma unroll
    for (int j = 0; j < (D::WL + D::WV - 1) / D::WV; ++j) {
        const int wl = wave + D::WV * j;
        if (wl < D::WL) dev::lds_dma16(src + wl * 256 + 4 * lane, l0 + 1024u * wl);   // uniform per wave
    }
}

// One exchange of a quad transpose: lanes that differ in lane bit BIT swap
// the elements that differ in element bit BIT (DPP quad permutation [1,0,3,2]
// for bit 0, [2,3,0,1] for bit 1).
template <int BIT>
__device__ inline void dx_quad_xchg(float (&v)[4], int b) {
    constexpr int step = 1 << BIT, ctrl = BIT == 0 ? 0xb1 : 0x4e;
    const bool hi = b & step;
    float r[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int lo = BIT == 0 ? 2 * k : k;              // the pair (lo, lo + step)
        r[k] = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(hi ? v[lo] : v[lo + step]), ctrl, 0xf, 0xf, false));
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {                         // selects on values: constant indices only
        const int lo = BIT == 0 ? 2 * k : k;
        v[lo] = hi ? r[k] : v[lo];
        v[lo + step] = hi ? v[lo + step] : r[k];
    }
}

// 4 x 4 transpose inside each lane quad: lane 4 m + b holds v[i] = X[i][b]
// on entry and X[b][i] on return.
__device__ inline void dx_quad_transpose(float (&v)[4], int b) {
    dx_quad_xchg<0>(v, b);
    dx_quad_xchg<1>(v, b);
}

template <int CZ, int CA>
__global__ __launch_bounds__((64 * Dx<CZ, CA>::WV)) void k_bwd_dx(BwdArgs a) {
    using D = Dx<CZ, CA>;
    extern __shared__ float smem[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int NT = a.n * a.ntiles, NG = (NT + D::WV - 1) / D::WV;
    if ((int)blockIdx.x >= NG) return;                             // uniform per block
    float *wbuf = smem;                                            // two stages
    float *halo = smem + 2 * D::WST + wave * D::HALO;              // this wave's tile
    const int mrow = lane & 15, kq = lane >> 4;
    const int pix = (mrow & 3) * 6 + (mrow >> 2);

    int g = blockIdx.x;
    dx_dma_stage<CZ, CA>(a.wt, 0, wbuf, wave, lane);
    float4 hreg[D::HV];
    uint32_t hok;
    dx_fetch_halo<CZ, CA>(a, D::WV * g + wave, D::WV * g + wave < NT, hreg, hok, lane);
    dx_store_halo<CZ, CA>(halo, hreg, hok, lane);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    dev::lds_barrier();
    int buf = 0;
    for (; g < NG; g += gridDim.x) {                               // uniform per block
        const int tid = D::WV * g + wave, tidn = D::WV * (g + (int)gridDim.x) + wave;
        floatx4 acc[D::NB];
#pragma unroll
        for (int nb = 0; nb < D::NB; ++nb) acc[nb] = floatx4{0.f, 0.f, 0.f, 0.f};
        // The epilogue's view, after a quad transpose of the accumulators:
        // lane (qb, qm, kq) holds pixel qb * 4 + kq of the tile, channels
        // c0(nb) = 16 nb + 4 qm .. + 3.  Its ReLU mask (a_{l-1} at those
        // places, 16 bytes per block) is loaded now, waited for by the end of
        // this stage, so the epilogue waits for no load.
        const int qb = lane & 3, qm = (lane >> 2) & 3, em = qb * 4 + kq;
        float4 msk[D::NB];
        {
            const bool tv = tid < NT;
            const int i = tv ? tid / a.ntiles : 0, t = tv ? tid - i * a.ntiles : 0;
            const float *ap = a.act_prev + (size_t)a.ids[i] * a.prev_stride + ((size_t)t * kTilePx + em) * CA;
#pragma unroll
            for (int nb = 0; nb < D::NB; ++nb) {
                const int c0 = nb * 16 + 4 * qm;
                msk[nb] = *reinterpret_cast<const float4 *>(ap + (c0 < CA ? c0 : 0));
            }
        }
        for (int q = 0; q < D::NQ; ++q) {
            const int kpos = q / D::NCH, ch = q - kpos * D::NCH;
            const int ky = kpos / 3, kx = kpos - ky * 3;
            const float *wst = wbuf + buf * D::WST;
            float4 av = *reinterpret_cast<const float4 *>(halo + hoff<CZ>(pix + ky * 6 + kx, 4 * ch * D::SB + kq));
            float4 bv[D::NB];
#pragma unroll
            for (int nb = 0; nb < D::NB; ++nb) bv[nb] = *reinterpret_cast<const float4 *>(wst + (nb * 64 + lane) * 4);
            dx_dma_stage<CZ, CA>(a.wt, q + 1 < D::NQ ? q + 1 : 0, wbuf + (buf ^ 1) * D::WST, wave, lane);
            // The next group's halo is fetched three stages before the end
            // (issued after this stage's weight loads: the wait below leaves
            // it in flight, the next stages' waits find it arrived).
            const bool hstage = q == (D::NQ >= 3 ? D::NQ - 3 : 0);
            if (hstage) dx_fetch_halo<CZ, CA>(a, tidn, tidn < NT, hreg, hok, lane);
#pragma unroll
            for (int b = 0; b < D::SB; ++b) {
                float4 an = av, bn[D::NB];
#pragma unroll
                for (int nb = 0; nb < D::NB; ++nb) bn[nb] = bv[nb];
                if (b + 1 < D::SB) {                               // the next block's operands during this one's ops
                    an = *reinterpret_cast<const float4 *>(halo + hoff<CZ>(pix + ky * 6 + kx, 4 * (ch * D::SB + b + 1) + kq));
#pragma unroll
                    for (int nb = 0; nb < D::NB; ++nb)
                        bn[nb] = *reinterpret_cast<const float4 *>(wst + (((b + 1) * D::NB + nb) * 64 + lane) * 4);
                }
                __builtin_amdgcn_sched_barrier(0);
                const float al[4] = {av.x, av.y, av.z, av.w};
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int nb = 0; nb < D::NB; ++nb) {
                        const float bj = j == 0 ? bv[nb].x : j == 1 ? bv[nb].y : j == 2 ? bv[nb].z : bv[nb].w;
                        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(al[j], bj, acc[nb], 0, 0, 0);
                    }
                __builtin_amdgcn_sched_barrier(0);
                av = an;
#pragma unroll
                for (int nb = 0; nb < D::NB; ++nb) bv[nb] = bn[nb];
            }
            buf ^= 1;
            if (hstage) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(D::HV) : "memory");
            else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            dev::lds_barrier();
        }
        if (tid < NT) {                                            // uniform per wave
            const int i = tid / a.ntiles, t = tid - i * a.ntiles;
            float *dst = a.dz_out + (((size_t)i * a.ntiles + t) * kTilePx + em) * CA;
#pragma unroll
            for (int nb = 0; nb < D::NB; ++nb) {
                float v[4] = {acc[nb][0], acc[nb][1], acc[nb][2], acc[nb][3]};   // pixels r * 4 + kq, channel 16 nb + 4 qm + qb
                dx_quad_transpose(v, qb);
                const int c0 = nb * 16 + 4 * qm;
                if (c0 < CA)                                       // CA % 4 == 0: whole float4s
                    *reinterpret_cast<float4 *>(dst + c0) =
                        make_float4(msk[nb].x > 0.f ? v[0] : 0.f, msk[nb].y > 0.f ? v[1] : 0.f,
                                    msk[nb].z > 0.f ? v[2] : 0.f, msk[nb].w > 0.f ? v[3] : 0.f);
            }
        }
        dev::wave_sync();                                          // this wave's halo reads are done
        dx_store_halo<CZ, CA>(halo, hreg, hok, lane);
        dev::wave_sync();
    }
}

// ------------------------------------------------------------------ dW

// dW for layers 2..L (a_{l-1} a tiled cache), operands read 16 bytes at a
// time.  The K index of the product is the tile's pixel: in 4 consecutive
// k-steps lane group kq takes k = 4 kq + j, j = 0..3, pixel (row kq, column j),
// so a lane's A values (dz at those pixels, output channel 16 mb + n) are
// one 16-byte read of a transposed dz tile [channel][pixel], and its B values
// (a_{l-1} at those pixels shifted by the column's kernel position (ky, kx),
// channel ci) one 16-byte read of the halo copy for kx, [ci][halo row][4]
// (halo columns kx .. kx + 3 of each row).  Wave u of a team owns all MBU
// row blocks and QW column blocks (MBU x QW x 4 accumulators), so one staged
// tile feeds MBU x QW x 4 matrix ops from MBU + QW reads.  Two staging
// buffers of P tiles each alternate: the matrix ops read one while the next P
// tiles are written to the other between their k-steps, one barrier per pass
// (P = 2 where both buffers fit one CU's LDS, else 1).  Row strides (20
// and 28 floats) put the 16 lanes of a read group in distinct bank groups.
template <int CA, int CZ>
struct Dw2 {
    static constexpr int NQ = 9 * CA + 1;                 // columns: (kernel position, input channel), bias
    static constexpr int NBQ = (NQ + 15) / 16;            // 16-column blocks
    static constexpr int MB = CZ / 16;                    // 16-row blocks (output channels)
    static constexpr int MBU = MB;                        // row blocks per wave
    static constexpr int QW0 = 32 / MBU;                  // column blocks per wave, at most 32 blocks of accumulators
    static constexpr int NCH = (NBQ + QW0 - 1) / QW0;     // column chunks (waves per team)
    static constexpr int QW = (NBQ + NCH - 1) / NCH;
    static constexpr int BPT = (NCH + 3) / 4;             // blocks per team
    static constexpr int SZ = 20;                         // dz row stride (16 pixels + pad)
    static constexpr int HS = 28;                         // halo copy channel stride (6 rows x 4 + pad)
    static constexpr int DZT = CZ * SZ;                   // floats of one staged dz tile
    static constexpr int HT = 3 * CA * HS;                // floats of one staged halo (three copies)
    static constexpr int P = 16 * (DZT + HT) <= 160 * 1024 ? 2 : 1;  // tiles per buffer
    static constexpr int DZV = (4 * CZ + 255) / 256;      // 16-byte dz chunks per thread and tile
    static constexpr int HV = (9 * CA + 255) / 256;       // 16-byte halo chunks per thread and tile
    static constexpr int BUF = P * (DZT + HT);            // floats of one staging buffer
    static constexpr size_t lds_bytes = (size_t)2 * BUF * sizeof(float);   // two buffers
    static_assert(lds_bytes <= 160 * 1024, "two buffers fit one CU");
    static_assert(CZ % 16 == 0 && CA % 4 == 0, "whole row blocks and 16-byte channel chunks");
};

// Staging of one fetched tile into an LDS buffer by 256 threads (tix the
// thread's index among them): dz transposed to [channel][pixel] (PART 0), the
// halo as three column-shifted copies [kx][channel][row-major 6 x 4 window]
// (PART 1).
template <int CA, int CZ, int PART>
__device__ inline void dw2_stage(float *dz, float *h, const float4 *rdz, const float4 *rh, int tix) {
    using D = Dw2<CA, CZ>;
    if constexpr (PART == 0) {
#pragma unroll
        for (int k = 0; k < D::DZV; ++k) {
            const int e = tix + 256 * k;
            if (e < 4 * CZ) {
                const int m = e / (CZ / 4), c4 = e - m * (CZ / 4);   // pixel m, channels 4 c4 ..
                const float4 v = rdz[k];
                dz[(4 * c4 + 0) * D::SZ + m] = v.x;
                dz[(4 * c4 + 1) * D::SZ + m] = v.y;
                dz[(4 * c4 + 2) * D::SZ + m] = v.z;
                dz[(4 * c4 + 3) * D::SZ + m] = v.w;
            }
        }
    } else {
#pragma unroll
        for (int k = 0; k < D::HV; ++k) {
            const int e = tix + 256 * k;
            if (e < 9 * CA) {
                const int pos = e / (CA / 4), c4 = e - pos * (CA / 4);
                const int hy = pos / 6, hx = pos - 6 * hy;
                const float4 v = rh[k];
#pragma unroll
                for (int kx = 0; kx < 3; ++kx) {
                    const int j = hx - kx;
                    if (j < 0 || j > 3) continue;
                    float *d = h + (kx * CA + 4 * c4) * D::HS + hy * 4 + j;
                    d[0] = v.x;
                    d[D::HS] = v.y;
                    d[2 * D::HS] = v.z;
                    d[3 * D::HS] = v.w;
                }
            }
        }
    }
}

// One tile's A (dz rows) and B (halo columns) fragments from a staged buffer.
template <int MBU, int QW>
struct Dw2Ops {
    float4 av[MBU], bv[QW];
};

template <int CA, int CZ, int QW = Dw2<CA, CZ>::QW>
__device__ inline void dw2_ops(Dw2Ops<Dw2<CA, CZ>::MBU, QW> &o, const float *dz, const float *h, const int *boff,
                               int col, int kq) {
    using D = Dw2<CA, CZ>;
#pragma unroll
    for (int m = 0; m < D::MBU; ++m) o.av[m] = *reinterpret_cast<const float4 *>(dz + (16 * m + col) * D::SZ + 4 * kq);
#pragma unroll
    for (int k = 0; k < QW; ++k)
        o.bv[k] = boff[k] >= 0 ? *reinterpret_cast<const float4 *>(h + boff[k])
                               : (boff[k] == -1 ? make_float4(1.f, 1.f, 1.f, 1.f) : make_float4(0.f, 0.f, 0.f, 0.f));
}

// Matrix ops of k-steps J0 .. J1 - 1 of one tile.
template <int MBU, int QW, int J0, int J1>
__device__ inline void dw2_mma(floatx4 (&acc)[MBU][QW], const Dw2Ops<MBU, QW> &o) {
#pragma unroll
    for (int j = J0; j < J1; ++j)
#pragma unroll
        for (int m = 0; m < MBU; ++m)
#pragma unroll
            for (int k = 0; k < QW; ++k) {
                const float x = j == 0 ? o.av[m].x : j == 1 ? o.av[m].y : j == 2 ? o.av[m].z : o.av[m].w;
                const float y = j == 0 ? o.bv[k].x : j == 1 ? o.bv[k].y : j == 2 ? o.bv[k].z : o.bv[k].w;
                acc[m][k] = __builtin_amdgcn_mfma_f32_16x16x4f32(x, y, acc[m][k], 0, 0, 0);
            }
}

template <int CA, int CZ>
__global__ __launch_bounds__(256) void k_bwd_dw2(BwdArgs a) {
    using D = Dw2<CA, CZ>;
    extern __shared__ float smem[];                       // two buffers of [P][CZ][SZ] dz, [P][3][CA][HS] halo
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int team = blockIdx.x / D::BPT, u = (blockIdx.x - team * D::BPT) * 4 + wave;
    const bool active = u < D::NCH;
    const int qb0 = active ? u * D::QW : 0;
    const int kq = lane >> 4, col = lane & 15;
    // This lane's B offset per column block within a staged halo, or -1 for
    // the bias column (all ones), -2 for a padding column (zeros).
    int boff[D::QW];
#pragma unroll
    for (int k = 0; k < D::QW; ++k) {
        const int q = (qb0 + k) * 16 + col;
        if (q < 9 * CA) {
            const int kpos = q / CA, ci = q - kpos * CA, ky = kpos / 3, kx = kpos - 3 * ky;
            boff[k] = (kx * CA + ci) * D::HS + (kq + ky) * 4;
        } else {
            boff[k] = q == 9 * CA ? -1 : -2;
        }
    }
    floatx4 acc[D::MBU][D::QW];
#pragma unroll
    for (int m = 0; m < D::MBU; ++m)
#pragma unroll
        for (int k = 0; k < D::QW; ++k) acc[m][k] = floatx4{0.f, 0.f, 0.f, 0.f};
    // The team's tiles [t0, t1) of the batch (batch index i, tile t), walked
    // in order: (fi, ft) is the next tile to fetch.
    const long long NT = (long long)a.n * a.ntiles;
    const int t0 = (int)(NT * team / a.teams), t1 = (int)(NT * (team + 1) / a.teams);
    int fi = t0 / a.ntiles, ft = t0 - fi * a.ntiles;
    // Operands of tiles c .. c + P - 1 (this thread's share) into registers,
    // every load issued; tiles past t1, out-of-image halo pixels: zero.  The
    // slot of each tile's stream is read first, as a scalar load of a
    // wave-uniform index, so that only the halo addresses wait for it (a
    // vector load there would make the wait drain the dz loads as well).
    float4 rdz[D::P][D::DZV], rh[D::P][D::HV];
    const __attribute__((address_space(4))) int32_t *ids =
        (const __attribute__((address_space(4))) int32_t *)a.ids;
    auto fetch = [&](int c) __attribute__((always_inline)) {
        bool ok[D::P];
        int tl[D::P], slot[D::P];
#pragma unroll
        for (int pp = 0; pp < D::P; ++pp) {
            ok[pp] = c + pp < t1;
            const int i = __builtin_amdgcn_readfirstlane(ok[pp] ? fi : 0);
            tl[pp] = ok[pp] ? ft : 0;
            if (++ft == a.ntiles) {
                ft = 0;
                ++fi;
            }
            slot[pp] = ids[i];
            const float4 *dzp = reinterpret_cast<const float4 *>(a.dz_in + ((size_t)i * a.ntiles + tl[pp]) * kTilePx * CZ);
#pragma unroll
            for (int k = 0; k < D::DZV; ++k) {
                const int e = threadIdx.x + 256 * k;
                rdz[pp][k] = ok[pp] && e < 4 * CZ ? dzp[e] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
#pragma unroll
        for (int pp = 0; pp < D::P; ++pp) {
            const int t = tl[pp], ty = t / a.TW, tx = t - ty * a.TW;
            const float *ap = a.act_prev + (size_t)slot[pp] * a.prev_stride;
#pragma unroll
            for (int k = 0; k < D::HV; ++k) {
                const int e = threadIdx.x + 256 * k;
                const int pos = e / (CA / 4), c4 = e - pos * (CA / 4);
                const int y = ty * kTile - 1 + pos / 6, x = tx * kTile - 1 + pos % 6;
                float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
                if (ok[pp] && e < 9 * CA && y >= 0 && y < a.H && x >= 0 && x < a.W)
                    v = *reinterpret_cast<const float4 *>(
                        ap + ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CA + 4 * c4);
                rh[pp][k] = v;
            }
        }
    };
    // Two staging buffers: while the matrix ops read the P tiles of one, the
    // next P tiles (fetched into registers during the previous pass) are
    // written to the other between k-steps, and the tiles after those are
    // fetched; one block barrier per pass.  Fetching and staging run
    // unconditionally (tiles past t1 load zeros from valid addresses): a
    // guarded pass would make the compiler copy the accumulators between
    // register files.
    fetch(t0);
#pragma unroll
    for (int pp = 0; pp < D::P; ++pp) {
        dw2_stage<CA, CZ, 0>(smem + pp * D::DZT, smem + D::P * D::DZT + pp * D::HT, rdz[pp], rh[pp], threadIdx.x);
        dw2_stage<CA, CZ, 1>(smem + pp * D::DZT, smem + D::P * D::DZT + pp * D::HT, rdz[pp], rh[pp], threadIdx.x);
    }
    fetch(t0 + D::P);
    dev::lds_barrier();
    int b = 0;
    for (int c = t0; c < t1; c += D::P) {
        float *cb = smem + b * D::BUF, *nb = smem + (b ^ 1) * D::BUF;
        Dw2Ops<D::MBU, D::QW> cur;
        dw2_ops<CA, CZ>(cur, cb, cb + D::P * D::DZT, boff, col, kq);
#pragma unroll
        for (int pp = 0; pp < D::P; ++pp) {
            Dw2Ops<D::MBU, D::QW> nxt;
            if (pp + 1 < D::P) dw2_ops<CA, CZ>(nxt, cb + (pp + 1) * D::DZT, cb + D::P * D::DZT + (pp + 1) * D::HT, boff, col, kq);
            __builtin_amdgcn_sched_barrier(0);
            dw2_mma<D::MBU, D::QW, 0, 2>(acc, cur);
            __builtin_amdgcn_sched_barrier(0);
            dw2_stage<CA, CZ, 0>(nb + pp * D::DZT, nb + D::P * D::DZT + pp * D::HT, rdz[pp], rh[pp], threadIdx.x);
            __builtin_amdgcn_sched_barrier(0);
            dw2_mma<D::MBU, D::QW, 2, 4>(acc, cur);
            __builtin_amdgcn_sched_barrier(0);
            dw2_stage<CA, CZ, 1>(nb + pp * D::DZT, nb + D::P * D::DZT + pp * D::HT, rdz[pp], rh[pp], threadIdx.x);
            __builtin_amdgcn_sched_barrier(0);
            if (pp + 1 < D::P) cur = nxt;
        }
        fetch(c + 2 * D::P);                               // in flight during the next pass
        dev::lds_barrier();                                // the other buffer staged, this one read
        b ^= 1;
    }
    if (!active) return;
#pragma unroll
    for (int m = 0; m < D::MBU; ++m)
#pragma unroll
        for (int k = 0; k < D::QW; ++k) {
            const int q = (qb0 + k) * 16 + col;
            if (q >= D::NQ) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = m * 16 + 4 * kq + r;
                a.part[((size_t)co * D::NQ + q) * a.teams + team] = acc[m][k][r];
            }
        }
}

// The same weight gradients with a block of 8 waves per team, for layers
// whose row blocks and a third as many column blocks as above fit 64
// accumulators (40 -> 80: 5 x 3 blocks): two waves per SIMD.  A pass takes
// four tiles (two buffers of four fit one CU's LDS: one barrier per four
// tiles); waves 0-3 stage and fetch tiles 0 and 2 of each pass, waves 4-7
// tiles 1 and 3, each half between the k-steps of its own tiles, so that
// while one wave of a SIMD runs its staging the other issues matrix ops.
// Teams, tile ranges and the k-step order of every column block are those of
// the 4-wave kernel: the same partial sums bit for bit.
template <int CA, int CZ>
struct Dw8 {
    using D = Dw2<CA, CZ>;
    static constexpr int QW = (D::NBQ + 7) / 8;           // column blocks per wave
    static constexpr int P = 4;                            // tiles per pass: 0 and 2 of half 0, 1 and 3 of half 1
    static constexpr int BUF = P * (D::DZT + D::HT);
    static constexpr size_t lds_bytes = (size_t)2 * BUF * sizeof(float);
    static constexpr bool FITS = D::MBU * QW * 4 <= 64 && lds_bytes <= 160 * 1024;
};

template <int CA, int CZ>
__global__ __launch_bounds__(512) void k_bwd_dw8(BwdArgs a) {
    using D = Dw2<CA, CZ>;
    constexpr int QW = Dw8<CA, CZ>::QW;
    static_assert(Dw8<CA, CZ>::FITS, "8-wave layout");
    extern __shared__ float smem[];                       // two buffers of [P][CZ][SZ] dz, [P][3][CA][HS] halo
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int half = wave >> 2, hix = threadIdx.x & 255;  // tiles half, half + 2 of a pass are this half's to stage
    const int team = blockIdx.x;
    const int qb0 = wave * QW;
    const int kq = lane >> 4, col = lane & 15;
    int boff[QW];
#pragma unroll
    for (int k = 0; k < QW; ++k) {
        const int q = (qb0 + k) * 16 + col;
        if (q < 9 * CA) {
            const int kpos = q / CA, ci = q - kpos * CA, ky = kpos / 3, kx = kpos - 3 * ky;
            boff[k] = (kx * CA + ci) * D::HS + (kq + ky) * 4;
        } else {
            boff[k] = q == 9 * CA ? -1 : -2;
        }
    }
    floatx4 acc[D::MBU][QW];
#pragma unroll
    for (int m = 0; m < D::MBU; ++m)
#pragma unroll
        for (int k = 0; k < QW; ++k) acc[m][k] = floatx4{0.f, 0.f, 0.f, 0.f};
    const long long NT = (long long)a.n * a.ntiles;
    const int t0 = (int)(NT * team / a.teams), t1 = (int)(NT * (team + 1) / a.teams);
    // This half's tiles t0 + half, t0 + half + 2, ...: (fi, ft) the next one.
    int fi = (t0 + half) / a.ntiles, ft = (t0 + half) - fi * a.ntiles;
    float4 rdz[2][D::DZV], rh[2][D::HV];
    const __attribute__((address_space(4))) int32_t *ids =
        (const __attribute__((address_space(4))) int32_t *)a.ids;
    auto fetch = [&](int c, int s) __attribute__((always_inline)) {   // tile c into register set s
        const bool ok = c < t1;
        const int i = __builtin_amdgcn_readfirstlane(ok ? fi : 0), tl = ok ? ft : 0;
        ft += 2;
        while (ft >= a.ntiles) {
            ft -= a.ntiles;
            ++fi;
        }
        const int slot = ids[i];
        const float4 *dzp = reinterpret_cast<const float4 *>(a.dz_in + ((size_t)i * a.ntiles + tl) * kTilePx * CZ);
#pragma unroll
        for (int k = 0; k < D::DZV; ++k) {
            const int e = hix + 256 * k;
            rdz[s][k] = ok && e < 4 * CZ ? dzp[e] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        const int ty = tl / a.TW, tx = tl - ty * a.TW;
        const float *ap = a.act_prev + (size_t)slot * a.prev_stride;
#pragma unroll
        for (int k = 0; k < D::HV; ++k) {
            const int e = hix + 256 * k;
            const int pos = e / (CA / 4), c4 = e - pos * (CA / 4);
            const int y = ty * kTile - 1 + pos / 6, x = tx * kTile - 1 + pos % 6;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (ok && e < 9 * CA && y >= 0 && y < a.H && x >= 0 && x < a.W)
                v = *reinterpret_cast<const float4 *>(
                    ap + ((size_t)((y >> 2) * a.TW + (x >> 2)) * kTilePx + (y & 3) * 4 + (x & 3)) * CA + 4 * c4);
            rh[s][k] = v;
        }
    };
    constexpr int P = Dw8<CA, CZ>::P, BUF = Dw8<CA, CZ>::BUF;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        fetch(t0 + half + 2 * s, s);
        dw2_stage<CA, CZ, 0>(smem + (half + 2 * s) * D::DZT, smem + P * D::DZT + (half + 2 * s) * D::HT, rdz[s], rh[s], hix);
        dw2_stage<CA, CZ, 1>(smem + (half + 2 * s) * D::DZT, smem + P * D::DZT + (half + 2 * s) * D::HT, rdz[s], rh[s], hix);
    }
    fetch(t0 + P + half, 0);
    fetch(t0 + P + half + 2, 1);
    dev::lds_barrier();
    int b = 0;
    for (int c = t0; c < t1; c += P) {
        float *cb = smem + b * BUF, *nb = smem + (b ^ 1) * BUF;
        Dw2Ops<D::MBU, QW> cur;
        dw2_ops<CA, CZ, QW>(cur, cb, cb + P * D::DZT, boff, col, kq);
#pragma unroll
        for (int pp = 0; pp < P; ++pp) {
            Dw2Ops<D::MBU, QW> nxt;
            if (pp + 1 < P) dw2_ops<CA, CZ, QW>(nxt, cb + (pp + 1) * D::DZT, cb + P * D::DZT + (pp + 1) * D::HT, boff, col, kq);
            __builtin_amdgcn_sched_barrier(0);
            dw2_mma<D::MBU, QW, 0, 2>(acc, cur);
            __builtin_amdgcn_sched_barrier(0);
            if (half == (pp & 1)) dw2_stage<CA, CZ, 0>(nb + pp * D::DZT, nb + P * D::DZT + pp * D::HT, rdz[pp >> 1], rh[pp >> 1], hix);
            __builtin_amdgcn_sched_barrier(0);
            dw2_mma<D::MBU, QW, 2, 4>(acc, cur);
            __builtin_amdgcn_sched_barrier(0);
            if (half == (pp & 1)) {
                dw2_stage<CA, CZ, 1>(nb + pp * D::DZT, nb + P * D::DZT + pp * D::HT, rdz[pp >> 1], rh[pp >> 1], hix);
                fetch(c + 2 * P + pp, pp >> 1);                // in flight during the next pass
            }
            __builtin_amdgcn_sched_barrier(0);
            if (pp + 1 < P) cur = nxt;
        }
        dev::lds_barrier();                                // the other buffer staged, this one read
        b ^= 1;
    }
#pragma unroll
    for (int m = 0; m < D::MBU; ++m)
#pragma unroll
        for (int k = 0; k < QW; ++k) {
            const int q = (qb0 + k) * 16 + col;
            if (q >= D::NQ) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = m * 16 + 4 * kq + r;
                a.part[((size_t)co * D::NQ + q) * a.teams + team] = acc[m][k][r];
            }
        }
}

// dW for layer 1 (a_0 the float32 input planes, 1 or 4 channels): so few
// columns (9 cin + 1) that staging a tile through LDS for a handful of matrix
// ops costs more than the ops.  Each wave is a team of its own and walks its
// tiles with the operands loaded straight into the matrix layout (lane
// (m, kq), k-step j: A = dz at pixel (row kq, column j), channel 16 mb + m;
// B = the input at that pixel shifted by the column's kernel position, or 1
// for the bias column), the next tile's loads issued before this tile's
// matrix ops.  Memory-bound: each tile's dz (16 x CZ floats) is read once.
template <int CA, int CZ>
struct DwFirst {
    static constexpr int NQ = 9 * CA + 1;
    static constexpr int NBQ = (NQ + 15) / 16;            // 16-column blocks
    static constexpr int MB = (CZ + 15) / 16;             // 16-row blocks
};

template <int CA, int CZ>
__global__ __launch_bounds__(256) void k_bwd_dw_first(BwdArgs a) {
    using D = DwFirst<CA, CZ>;
    const int lane = threadIdx.x & 63;
    const int team = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int kq = lane >> 4, col = lane & 15;
    const long long NT = (long long)a.n * a.ntiles;
    const int t0 = (int)(NT * team / a.teams), t1 = (int)(NT * (team + 1) / a.teams);
    if (team >= a.teams) return;                           // uniform per wave
    // This lane's column per block: kernel position offset (ky, kx) and input
    // channel, or the bias / padding column.
    int qky[D::NBQ], qkx[D::NBQ], qci[D::NBQ], qkind[D::NBQ];   // kind 0: input, 1: bias, 2: zero
#pragma unroll
    for (int k = 0; k < D::NBQ; ++k) {
        const int q = 16 * k + col;
        const int kpos = q / CA;
        qci[k] = q - kpos * CA;
        qky[k] = kpos / 3;
        qkx[k] = kpos - 3 * (kpos / 3);
        qkind[k] = q < 9 * CA ? 0 : q == 9 * CA ? 1 : 2;
    }
    floatx4 acc[D::MB][D::NBQ];
#pragma unroll
    for (int m = 0; m < D::MB; ++m)
#pragma unroll
        for (int k = 0; k < D::NBQ; ++k) acc[m][k] = floatx4{0.f, 0.f, 0.f, 0.f};
    const size_t HW = (size_t)a.H * a.W;
    float av[2][D::MB][4], bv[2][D::NBQ][4];
    int fi = t0 / a.ntiles, ft = t0 - fi * a.ntiles;
    auto fetch = [&](int slot_buf) __attribute__((always_inline)) {
        const int i = fi, t = ft;
        if (++ft == a.ntiles) {
            ft = 0;
            ++fi;
        }
        const int ty = t / a.TW, tx = t - ty * a.TW;
        const int slot = a.ids[i];
        const float *dz = a.dz_in + ((size_t)i * a.ntiles + t) * kTilePx * CZ;
#pragma unroll
        for (int m = 0; m < D::MB; ++m) {
            const int co = 16 * m + col;
#pragma unroll
            for (int j = 0; j < 4; ++j) av[slot_buf][m][j] = co < CZ ? dz[(4 * kq + j) * CZ + co] : 0.f;
        }
        const int head = a.stack != 1 ? a.ring_head[slot] : 0;
#pragma unroll
        for (int k = 0; k < D::NBQ; ++k) {
            const float *plane;
            if (a.stack == 1) {
                plane = a.act_prev + ((size_t)slot * CA + qci[k]) * HW;
            } else {
                const int jj = qci[k] / a.cin0, c1 = qci[k] - jj * a.cin0;
                const int rp = (head - (a.stack - 1) + jj + 4 * a.stack) & 3;
                plane = a.act_prev + (((size_t)slot * 4 + rp) * a.cin0 + c1) * HW;
            }
            const int y = ty * kTile - 1 + kq + qky[k];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int x = tx * kTile - 1 + j + qkx[k];
                const bool in = qkind[k] == 0 && y >= 0 && y < a.H && x >= 0 && x < a.W;
                bv[slot_buf][k][j] = in ? plane[(size_t)y * a.W + x] : (qkind[k] == 1 ? 1.f : 0.f);
            }
        }
    };
    if (t0 < t1) fetch(0);
    for (int tt = t0; tt < t1; tt += 2) {
        if (tt + 1 < t1) fetch(1);                         // in flight during tile tt's matrix ops
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int m = 0; m < D::MB; ++m)
#pragma unroll
                for (int k = 0; k < D::NBQ; ++k)
                    acc[m][k] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[0][m][j], bv[0][k][j], acc[m][k], 0, 0, 0);
        if (tt + 1 >= t1) break;
        if (tt + 2 < t1) fetch(0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int m = 0; m < D::MB; ++m)
#pragma unroll
                for (int k = 0; k < D::NBQ; ++k)
                    acc[m][k] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[1][m][j], bv[1][k][j], acc[m][k], 0, 0, 0);
    }
#pragma unroll
    for (int m = 0; m < D::MB; ++m)
#pragma unroll
        for (int k = 0; k < D::NBQ; ++k) {
            const int q = 16 * k + col;
            if (q >= D::NQ) continue;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = 16 * m + 4 * kq + r;
                if (co < CZ) a.part[((size_t)co * D::NQ + q) * a.teams + team] = acc[m][k][r];
            }
        }
}

// dW_l and db_l from the teams' partial sums ([co][column][team]): one wave
// per weight, lane j adding teams j, j + 64, ... in order, then the lanes'
// sums by a fixed butterfly, so the order never changes.
__global__ __launch_bounds__(256) void k_bwd_reduce(BwdArgs a) {
    const int NQ = 9 * a.ca + 1;
    const int e = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (e >= a.cz * NQ) return;                            // uniform per wave
    const int co = e / NQ, q = e - co * NQ;
    const float *p = a.part + (size_t)e * a.teams;
    float s = 0.f;
    for (int team = lane; team < a.teams; team += 64) s += p[team];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane != 0) return;
    float *d;
    if (q < 9 * a.ca) {
        const int kpos = q / a.ca, ci = q - kpos * a.ca;
        d = a.gw + ((size_t)co * a.ca + ci) * 9 + kpos;
    } else {
        d = a.gb + co;
    }
    *d = a.accumulate ? *d + s : s;
}

// ------------------------------------------------------------------ SGD

// Natural-layout index of packed element d (or -1 for a padding zero).
__device__ inline long long sgd_src(const SgdArgs &a, size_t d) {
    switch (a.kind) {
    case SGD_FIRST: {                                         // [ci * 9 + k][co]
        const int co = (int)(d % a.cout);
        const size_t r = d / a.cout;
        const int ci = (int)(r / 9), k = (int)(r % 9);
        return ((long long)co * a.cin + ci) * 9 + k;
    }
    case SGD_MFMA: {                                          // [kpos][block][nb][lane][j]
        const size_t per = (size_t)a.cin * a.cout;
        const int kpos = (int)(d / per);
        size_t r = d - (size_t)kpos * per;
        const int nf = a.cin / 16;
        const size_t full = (size_t)nf * 16 * a.cout;
        int ci, n;
        if (r < full) {
            const int b = (int)(r / (16 * a.cout));
            const int rb = (int)(r - (size_t)b * 16 * a.cout);
            const int nb = rb / 256, l = (rb / 4) % 64, j = rb % 4;
            ci = 16 * b + 4 * (l / 16) + j;
            n = nb * 16 + l % 16;
        } else {
            const int rt = (int)(r - full);
            const int nb = rt / 128, l = (rt / 2) % 64, j = rt % 2;
            ci = 16 * nf + 2 * (l / 16) + j;
            n = nb * 16 + l % 16;
        }
        return ((long long)n * a.cin + ci) * 9 + kpos;
    }
    case SGD_DENSE: {                                         // [o][tile][16][C], 0 outside the image
        const int o = (int)(d / a.K);
        const size_t e = d - (size_t)o * a.K;
        const int c = (int)(e % a.C), m = (int)((e / a.C) % kTilePx), tile = (int)(e / ((size_t)kTilePx * a.C));
        const int ty = tile / a.TW, tx = tile - ty * a.TW;
        const int y = ty * kTile + m / 4, x = tx * kTile + m % 4;
        if (y >= a.H || x >= a.W) return -1;
        return (long long)o * a.C * a.H * a.W + ((long long)c * a.H + y) * a.W + x;
    }
    case SGD_TILE_HEAD: {                                     // [o][tile][nb][lane][i]
        const int NB = a.C / 16;
        const int i = (int)(d % 4), l = (int)((d / 4) % 64), nb = (int)((d / 256) % NB);
        const size_t r = d / (256 * (size_t)NB);
        const int tile = (int)(r % a.ntiles), o = (int)(r / a.ntiles);
        const int ty = tile / a.TW, tx = tile - ty * a.TW;
        const int c = nb * 16 + l % 16, y = ty * kTile + i, x = tx * kTile + l / 16;
        if (y >= a.H || x >= a.W) return -1;
        return (long long)o * a.C * a.H * a.W + ((long long)c * a.H + y) * a.W + x;
    }
    case SGD_TILE_PART: {                                     // [tile][b][kq][o][j], b < C
        const int j = (int)(d % 4);
        size_t r = d / 4;
        const int o = (int)(r % a.n_out);
        r /= a.n_out;
        const int kq = (int)(r % 4);
        r /= 4;
        const int b = (int)(r % a.C), tile = (int)(r / a.C);
        const int k = 16 * b + 4 * kq + j, m = k / a.C, c = k - m * a.C;
        const int ty = tile / a.TW, tx = tile - ty * a.TW;
        const int y = ty * kTile + m / 4, x = tx * kTile + m % 4;
        if (y >= a.H || x >= a.W) return -1;
        return (long long)o * a.C * a.H * a.W + ((long long)c * a.H + y) * a.W + x;
    }
    case SGD_DX: {                                            // [b][nb][lane][j], cin = ca, cout = cz
        const int NB = (a.cin + 15) / 16;
        const int j = (int)(d % 4), l = (int)((d / 4) % 64), nb = (int)((d / 256) % NB);
        const int b = (int)(d / (256 * (size_t)NB));
        const int K = 16 * b + 4 * (l / 16) + j, n = nb * 16 + l % 16;
        if (n >= a.cin) return -1;
        const int kpos = K / a.cout, co = K - kpos * a.cout;
        return ((long long)co * a.cin + n) * 9 + (8 - kpos);
    }
    default:
        return (long long)d;
    }
}

// Two roundings, fl(w - fl(lr g)), as a host computing the same update in
// float32 does: contraction into one fused multiply-add is switched off.
// assign: a plain gather into the packed layout (padding elements 0).
__global__ __launch_bounds__(256) void k_sgd(SgdArgs a) {
#pragma clang fp contract(off)
    for (size_t d = (size_t)blockIdx.x * blockDim.x + threadIdx.x; d < a.count; d += (size_t)gridDim.x * blockDim.x) {
        const long long s = sgd_src(a, d);
        if (a.assign) {
            a.dst[d] = s >= 0 ? a.g[s] : 0.f;
        } else if (s >= 0) {
            const float step = a.lr * a.g[s];
            a.dst[d] = a.dst[d] - step;
        }
    }
}

__global__ __launch_bounds__(256) void k_unprime(int32_t *primed, int S) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < S) primed[i] = 0;
}

// ------------------------------------------------------------------ launchers

#define RN_DW_FIRST_SHAPES(X) X(1, 20) X(1, 40) X(1, 64) X(1, 80) X(4, 20) X(4, 40) X(4, 64) X(4, 80)
#define RN_DW_SHAPES(X) X(40, 80) X(64, 128) X(128, 128)
#define RN_DX_SHAPES(X) X(80, 40) X(128, 64) X(128, 128)

int dw_blocks_per_team(int ca, int cz, bool first) {
#define X(a_, z_) \
    if (first && ca == a_ && cz == z_) return 1;
    RN_DW_FIRST_SHAPES(X)
#undef X
#define X(a_, z_) \
    if (!first && ca == a_ && cz == z_) return Dw8<a_, z_>::FITS ? 1 : Dw2<a_, z_>::BPT;
    RN_DW_SHAPES(X)
#undef X
    return 0;
}

template <int CA, int CZ>
hipError_t run_dw_first(const BwdArgs &a, hipStream_t s) {
    hipLaunchKernelGGL((k_bwd_dw_first<CA, CZ>), dim3((a.teams + 3) / 4), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int total = CZ * DwFirst<CA, CZ>::NQ;
    hipLaunchKernelGGL(k_bwd_reduce, dim3((total + 3) / 4), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int CA, int CZ>
hipError_t run_dw2(const BwdArgs &a, hipStream_t s) {
    using D = Dw2<CA, CZ>;
    if constexpr (Dw8<CA, CZ>::FITS) {
        auto kern = k_bwd_dw8<CA, CZ>;
        constexpr size_t lds8 = Dw8<CA, CZ>::lds_bytes;
        static hipError_t attr = dev::set_lds(kern, lds8);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL(kern, dim3(a.teams), dim3(512), lds8, s, a);
    } else {
        auto kern = k_bwd_dw2<CA, CZ>;
        static hipError_t attr = dev::set_lds(kern, D::lds_bytes);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL(kern, dim3(D::BPT * a.teams), dim3(256), D::lds_bytes, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int total = CZ * D::NQ;
    hipLaunchKernelGGL(k_bwd_reduce, dim3((total + 3) / 4), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int CZ, int CA>
hipError_t run_dx(const BwdArgs &a, int cus, hipStream_t s) {
    using D = Dx<CZ, CA>;
    auto kern = k_bwd_dx<CZ, CA>;
    static hipError_t attr = dev::set_lds(kern, D::lds_bytes);
    if (attr != hipSuccess) return attr;
    const long long groups = ((long long)a.n * a.ntiles + D::WV - 1) / D::WV;
    const int per_cu = D::lds_bytes <= 78 * 1024 ? 2 : 1;       // blocks that fit one CU's LDS
    const int grid = (int)std::min<long long>(groups, (long long)per_cu * cus);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * D::WV), D::lds_bytes, s, a);
    return hipGetLastError();
}

}  // namespace

bool train_shapes_supported(int ca, int cz, bool first) { return dw_blocks_per_team(ca, cz, first) > 0; }

bool train_dx_supported(int cz, int ca) {
#define X(z_, a_) \
    if (cz == z_ && ca == a_) return true;
    RN_DX_SHAPES(X)
#undef X
    return false;
}

size_t dx_weights_elems(int cz, int ca) { return (size_t)9 * cz * ((ca + 15) / 16) * 16; }

void pack_dx_weights(const float *oihw, int ca, int cz, float *dst) {
    // [b][nb][lane][j]: K = 16 b + 4 (lane / 16) + j is (kernel position
    // K / cz, channel K % cz of layer l), column n = 16 nb + lane % 16 is
    // channel n of layer l-1; the value is W_l[K % cz][n] at the flipped
    // position 8 - K / cz, 0 for padding columns.
    const int NB = (ca + 15) / 16, KB = 9 * cz / 16;
    size_t d = 0;
    for (int b = 0; b < KB; ++b)
        for (int nb = 0; nb < NB; ++nb)
            for (int l = 0; l < 64; ++l)
                for (int j = 0; j < 4; ++j) {
                    const int K = 16 * b + 4 * (l / 16) + j, n = nb * 16 + l % 16;
                    const int kpos = K / cz, co = K % cz;
                    dst[d++] = n < ca ? oihw[((size_t)co * ca + n) * 9 + (8 - kpos)] : 0.f;
                }
}

int bwd_dw_teams(int ca, int cz, bool first, int n, int ntiles, int cus) {
    if (first) {
        // a team per wave, 16 waves per CU, at least 8 tiles each
        const long long tiles = (long long)n * ntiles;
        return (int)std::max(1LL, std::min(16LL * cus, (tiles + 7) / 8));
    }
    const int bpt = std::max(1, dw_blocks_per_team(ca, cz, first));
    const long long tiles = (long long)n * ntiles;
    // One block per CU, one round: the accumulators and operands take more
    // than half the register file, so one wave per SIMD is resident anyway,
    // and equal tile ranges finish together (more, shorter teams measured
    // slower, and each adds a partial to reduce).
    const long long want = std::max(1, cus / bpt);
    return (int)std::max(1LL, std::min(want, (tiles + 7) / 8));
}

size_t bwd_dw_part_elems(int ca, int cz, int teams) { return (size_t)teams * cz * (9 * ca + 1); }

hipError_t launch_reinforce(int n, int n_out, const float *logits, const int32_t *actions, const float *returns,
                            float *g, hipStream_t s) {
    hipLaunchKernelGGL(k_reinforce, dim3((n + 255) / 256), dim3(256), 0, s, n, n_out, logits, actions, returns, g);
    return hipGetLastError();
}

hipError_t launch_bwd_head(const HeadBwdArgs &a, hipStream_t s) {
    const int E = kTilePx * a.C;
    if (a.n_out <= 8) {
        // a float4 of inputs per thread, one block per tile up to 512 threads
        const int q = E / 4, th = std::min(512, (q + 63) / 64 * 64);
        hipLaunchKernelGGL((k_bwd_head<8, 4>), dim3(a.ntiles, (q + th - 1) / th), dim3(th), 0, s, a);
    } else {
        // 32 or 64 weights and sums per input: one input per thread
        const dim3 grid(a.ntiles, (E + 255) / 256), block(256);
        if (a.n_out <= 32) hipLaunchKernelGGL((k_bwd_head<32, 1>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((k_bwd_head<64, 1>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dw(const BwdArgs &a, int cus, hipStream_t s) {
    (void)cus;
    const bool first = a.first != 0;
#define X(a_, z_) \
    if (first && a.ca == a_ && a.cz == z_) return run_dw_first<a_, z_>(a, s);
    RN_DW_FIRST_SHAPES(X)
#undef X
#define X(a_, z_) \
    if (!first && a.ca == a_ && a.cz == z_) return run_dw2<a_, z_>(a, s);
    RN_DW_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_bwd_dx(const BwdArgs &a, int cus, hipStream_t s) {
#define X(z_, a_) \
    if (a.cz == z_ && a.ca == a_) return run_dx<z_, a_>(a, cus, s);
    RN_DX_SHAPES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_sgd(const SgdArgs &a, hipStream_t s) {
    if (a.count == 0) return hipSuccess;
    const size_t blocks = std::min<size_t>((a.count + 255) / 256, 65536);
    hipLaunchKernelGGL(k_sgd, dim3((unsigned)blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_unprime(int32_t *primed, int S, hipStream_t s) {
    hipLaunchKernelGGL(k_unprime, dim3((S + 255) / 256), dim3(256), 0, s, primed, S);
    return hipGetLastError();
}

}  // namespace rn
