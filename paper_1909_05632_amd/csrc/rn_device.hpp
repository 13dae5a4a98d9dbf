// Device helpers shared by the conv kernels: work-item decoding, the XCD
// split of a work list, wave-level LDS ordering, persistent grid sizing.
#pragma once

#include "rn_internal.hpp"

namespace rn {
namespace dev {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Order this wave's LDS writes before its later LDS reads (and keep the
// compiler from moving memory operations across).
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Block barrier for data exchanged through LDS only: waits for this wave's
// LDS (and scalar) operations, then s_barrier.  Unlike __syncthreads it does
// not wait for the wave's outstanding global loads and stores, so prefetches
// stay in flight across it.  Use only where no global-memory data passes
// between the waves of the block.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// 16 bytes per lane from global memory straight into LDS
// (global_load_lds_dwordx4: lane i writes the 16 bytes at the wave-uniform LDS
// byte address lds + 16 i).  Issued in assembly so the compiler does not make
// every later LDS read wait for it; the caller waits (s_waitcnt vmcnt) before
// the data is read.  M0, the instruction's LDS base, is restored afterwards.
__device__ inline void lds_dma16(const void *src, uint32_t lds) {
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds)
                 : "memory");
}

// 4 bytes per lane (global_load_lds_dword: lane i writes the 4 bytes at lds
// + 4 i); as lds_dma16 otherwise.
__device__ inline void lds_dma4(const void *src, uint32_t lds) {
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dword %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(lds)
                 : "memory");
}

// LDS byte address of a pointer into LDS (the low half of a generic pointer to
// LDS is its LDS offset), made wave-uniform.
__device__ inline uint32_t lds_addr(const void *p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}

// Sums over the 64 lanes of a wave of eight per-lane values p[0..7], by
// halving: at each step (partner lane l ^ 32, 16, 8, 4, 2, 1) a lane keeps
// half of the values it still holds and adds the partner's copy of them, so
// 8 + 4 + ... values cross lanes in 10 moves instead of 48.  Each sum is
// formed by the same pairings as the full xor butterfly (p += its value at
// lane l ^ off, off = 32 .. 1), so the results are the butterfly's bits.  The
// moves are the gfx950 permlane swaps for 32 and 16 (rows of 16 lanes) and
// DPP row moves for the rest.  Lane l returns the sum of p[4 b5 + 2 b4 + b3]
// (b_i: bit i of l).
__device__ inline float lane_sums8(const float *p, int lane) {
    float h[4], g[2];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        // Lanes 0-31 keep p[k], lanes 32-63 p[4 + k]; each half receives the
        // other half's copy of the value it keeps.
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(p[k]), __float_as_uint(p[4 + k]), false,
                                                        false);
        h[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        // Even rows keep h[k], odd rows h[2 + k].
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(h[k]), __float_as_uint(h[2 + k]), false,
                                                        false);
        g[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    const bool b3 = (lane >> 3) & 1;
    const float keep = b3 ? g[1] : g[0], send = b3 ? g[0] : g[1];
    // row_ror:8 reads lane l ^ 8 within a row.
    float v = keep + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(send), 0x128, 0xf, 0xf, false));
    // Lane l ^ 4: row_shl:4 into lanes 0-3 and 8-11 of each row (banks 0, 2),
    // row_shr:4 into lanes 4-7 and 12-15 (banks 1, 3).
    int x = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x104, 0xf, 0x5, false);
    x = __builtin_amdgcn_update_dpp(x, __float_as_int(v), 0x114, 0xf, 0xa, false);
    v += __int_as_float(x);
    // Lane l ^ 2 and l ^ 1: quad permutations [2, 3, 0, 1] and [1, 0, 3, 2].
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4e, 0xf, 0xf, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false));
    return v;
}

struct TileRef {
    int slot, tile, ty, tx;
};

// A work item is named by one 32-bit word: list mode, the slot-encoded entry
// slot << 16 | ty << 8 | tx (one load); dense mode, the same word built from
// the stream id (one load) and the position.  item_word issues the load;
// item_ref only decodes, so the load can be issued iterations ahead.
template <bool DENSE>
__device__ inline uint32_t item_word(const ConvArgs &a, int t) {
    if constexpr (DENSE) {
        // Every tile of every stream, in chunks of 32 streams, position-major
        // within a chunk: 32 consecutive tiles share a head-weight slice, and
        // a chunk's neighbouring halos are still in L2 when they are reused.
        constexpr int CH = 32;
        const int per_chunk = CH * a.TH * a.TW;
        const int c = t / per_chunk;
        const int rr = t - c * per_chunk;
        const int nc = min(CH, a.dense_n - c * CH);
        const int tile = rr / nc;
        const int i = c * CH + (rr - tile * nc);
        const int ty = tile / a.TW;
        return ((uint32_t)a.ids[i] << 16) | ((uint32_t)ty << 8) | (uint32_t)(tile - ty * a.TW);
    } else {
        return a.wl[t];
    }
}

__device__ inline TileRef item_ref(const ConvArgs &a, uint32_t e) {
    TileRef r;
    r.slot = (int)(e >> 16);
    r.ty = (e >> 8) & 255;
    r.tx = e & 255;
    r.tile = r.ty * a.TW + r.tx;
    return r;
}

template <bool DENSE>
__device__ inline TileRef decode(const ConvArgs &a, int t) {
    return item_ref(a, item_word<DENSE>(a, t));
}

template <bool DENSE>
__device__ inline int work_count(const ConvArgs &a) {
    if constexpr (DENSE) return a.dense_n * a.TH * a.TW;
    else return *a.cnt;
}

// ---- variant mode: copy-on-write overlays of one base slot
//
// A variant is the base slot's input with the pixels of its change boxes
// taken from its own frame.  It owns no caches: the tiles it recomputes in a
// layer go to that layer's overlay, row = their index in the layer's work
// list, and everything else is read from the base slot.

// Input value (float32, channel c, pixel (y, x) inside the image) of variant i.
__device__ inline float var_input(const ConvArgs &a, int i, int c, int y, int x) {
    const size_t HW = (size_t)a.H * a.W, px = (size_t)y * a.W + x;
    const uint64_t w = a.vpm0[((size_t)i * a.H + y) * a.WW + (x >> 6)];
    if ((w >> (x & 63)) & 1ull) {
        const size_t f = (a.vframe_shared ? 0 : (size_t)i * a.vcin) * HW + (size_t)c * HW + px;
        return a.vframe_u8 ? a.lut[static_cast<const uint8_t *>(a.vframes)[f]]
                           : static_cast<const float *>(a.vframes)[f];
    }
    return static_cast<const float *>(a.in)[(size_t)a.vbase * a.in_stride + (size_t)c * HW + px];
}

// Address of channel 0 of pixel (y, x) (inside the image) of layer l-1 as
// variant i sees it: its overlay row where it recomputed the tile, else the
// base slot's cache.
template <typename T>
__device__ inline const T *var_src(const ConvArgs &a, int i, int y, int x, int cin) {
    const int ntiles = a.TH * a.TW, TMW = (ntiles + 63) >> 6;
    const int t = (y >> 2) * a.TW + (x >> 2);
    const int m = ((y & 3) * 4 + (x & 3)) * cin;
    const uint64_t w = a.vtm_in[(size_t)i * TMW + (t >> 6)];
    if ((w >> (t & 63)) & 1ull)
        return static_cast<const T *>(a.vov_in) + (size_t)a.vmap_in[(size_t)i * ntiles + t] * kTilePx * cin + m;
    return static_cast<const T *>(a.in) + (size_t)a.vbase * a.in_stride + (size_t)t * kTilePx * cin + m;
}

// XCD-aware split of the work items [0, cnt): workgroups are dispatched round
// robin over the chip's 8 XCDs (block b runs on XCD b % 8), each with its own
// L2.  Item range [cnt x / 8, cnt (x + 1) / 8) goes to the blocks of XCD x, so
// the tiles of neighbouring positions (same head weights, overlapping halos)
// are served from one L2.  `units` work items per block per round.
struct XcdRange {
    int first, end, stride;
};

__device__ inline XcdRange xcd_range(int cnt, int units) {
    constexpr int kXcd = 8;
    const int x = blockIdx.x % kXcd, k = blockIdx.x / kXcd;
    const int blocks_x = ((int)gridDim.x - x + kXcd - 1) / kXcd;
    XcdRange r;
    r.first = (int)((long long)cnt * x / kXcd) + k * units;
    r.end = (int)((long long)cnt * (x + 1) / kXcd);
    r.stride = blocks_x * units;
    return r;
}

// The same segments for blocks of 8 waves, two per SIMD (waves w and w + 4 of
// a block share one), returning wave `wave`'s own first item.  A round of the
// segment holds 8 B items (B blocks on the XCD): its first 4 B go to waves 0-3,
// four consecutive items per block (neighbouring tiles stay on one CU), the
// next 4 B to waves 4-7.  The partial last round then gives every SIMD of the
// XCD one extra item before any SIMD gets a second, where a block-major split
// would give both waves of a SIMD one.  `block_first` is the block's smallest
// item (wave 0's), for a block-uniform early exit.
struct XcdRangeW {
    int first, block_first, end, stride;
};

__device__ inline XcdRangeW xcd_range_simd2(int cnt, int wave) {
    constexpr int kXcd = 8;
    const int x = blockIdx.x % kXcd, k = blockIdx.x / kXcd;
    const int blocks_x = ((int)gridDim.x - x + kXcd - 1) / kXcd;
    const int seg = (int)((long long)cnt * x / kXcd);
    XcdRangeW r;
    r.block_first = seg + 4 * k;
    r.first = r.block_first + (wave & 3) + (wave >> 2) * 4 * blocks_x;
    r.end = (int)((long long)cnt * (x + 1) / kXcd);
    r.stride = blocks_x * 8;
    return r;
}

// Persistent grid: at most `cap` blocks, no more than the work needs, and a
// multiple of 8 so that every XCD segment of xcd_range has blocks.
inline int persistent_grid(int cap, int need) {
    int g = std::max(1, std::min(cap, need));
    return (g + 7) / 8 * 8;
}

template <typename K>
hipError_t set_lds(K kern, size_t lds) {
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)lds);
}

}  // namespace dev
}  // namespace rn
