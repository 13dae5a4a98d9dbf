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
#include "rn_internal.hpp"

namespace rn {
namespace {

constexpr int kThreads = 256;

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
    const float *P = a.hpart + (size_t)a.ids[i] * a.ntiles * NO;
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

// Any n_out: wave w of the block handles logits o = w, w + 4, ...
__global__ __launch_bounds__(kThreads) void k_tile_head_generic(TileHeadArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int i = blockIdx.x;
    const float *P = a.hpart + (size_t)a.ids[i] * a.ntiles * a.n_out;
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

hipError_t launch_tile_head(const TileHeadArgs &a, hipStream_t s) {
    if (a.n_out == 6)
        hipLaunchKernelGGL(k_tile_head<6>, dim3(a.n), dim3(kThreads), 0, s, a);
    else if (a.n_out == 18)
        hipLaunchKernelGGL(k_tile_head<18>, dim3(a.n), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(k_tile_head_generic, dim3(a.n), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace rn
