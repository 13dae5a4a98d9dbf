// Change detection, change growth, dirty-tile masks and work-list compaction.
//
// Change detection (Abstract; Sec. 1): a pixel changed iff the float32 bits of
// one of its channels differ from the cached input.  Growth (Fig. 1 caption):
// a 3x3 stride-1 layer spreads a change by one pixel on each side; in general
// an output pixel of a k x k layer with stride s and pad p changed iff its
// window (rows s y - p .. s y - p + k - 1, the same for columns) holds a
// changed input pixel.  Dirty
// tiles (Sec. 3, local areas instead of one rectangle): a 4x4 cell of a
// layer's grid is dirty iff it holds a dirty pixel.  The work list of a layer
// is its dirty tiles in (tile row, tile column, batch index) order.
//
// The work list of a layer is ordered by tile position first (see k_poswrite).
//
// Masks are bit rows: word (y * WW + x / 64), bit x % 64.  One workgroup owns
// one stream: it diffs the frame against the cache with 16-byte loads, ORs the
// change bits into a mask held in LDS, grows it layer by layer in LDS with
// shifts and ORs, and reduces 4x4 cells to tile bits with one ballot per 64
// tiles.  No global atomics; every output word has exactly one writer.
// The lists are then built position-major from the tile masks.
#include "rn_internal.hpp"

namespace rn {
namespace {

constexpr int kThreads = 256;
// k_masks: one block per stream, of 1024 threads when the streams fit one
// block per CU, else smaller blocks so that several streams share a CU and
// their serial phases overlap: 512 threads up to four streams per CU (1024
// full-resolution streams: 82 -> 77 us against 256 threads), 256 beyond.

__device__ inline uint32_t f32_bits(float v) { return __float_as_uint(v); }

// Block barrier for data exchanged through LDS only (waits for this wave's LDS
// operations, then s_barrier).  __syncthreads would also drain every global
// store in flight (its release fence), a full memory round trip per barrier;
// no kernel here reads global data that another wave of its block wrote.
__device__ inline void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline uint64_t row_valid_bits(int W, int wx) {
    int nb = W - 64 * wx;
    return nb >= 64 ? ~0ull : ((1ull << nb) - 1ull);
}

__device__ inline int block_sum(int v, int *red) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    lds_sync();
    if (lane == 0) red[wave] = v;
    lds_sync();
    int s = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) s += red[w];
    return s;
}

// Load 4 consecutive pixels of one channel plane as float32.
template <bool U8>
__device__ inline float4 load4(const void *frames, size_t off, const float *lut) {
    if constexpr (U8) {
        uint32_t q = *reinterpret_cast<const uint32_t *>(static_cast<const uint8_t *>(frames) + off);
        return make_float4(lut[q & 255u], lut[(q >> 8) & 255u], lut[(q >> 16) & 255u], lut[q >> 24]);
    } else {
        return *reinterpret_cast<const float4 *>(static_cast<const float *>(frames) + off);
    }
}

template <bool U8>
__device__ inline float load1(const void *frames, size_t off, const float *lut) {
    if constexpr (U8) return lut[static_cast<const uint8_t *>(frames)[off]];
    else return static_cast<const float *>(frames)[off];
}

// OR of mask word wx of the tile rows y0 .. y0 + 3 that lie inside the H rows
// (the four LDS reads issued together, not one round trip per row).
__device__ inline uint64_t tile_rows(const uint64_t *M, int y0, int H, int WW, int wx) {
    static_assert(kTile == 4, "four rows per tile");
    uint64_t r[kTile];
#pragma unroll
    for (int k = 0; k < kTile; ++k) r[k] = y0 + k < H ? M[(y0 + k) * WW + wx] : 0ull;
    return (r[0] | r[1]) | (r[2] | r[3]);
}

// Write layer l's pixel mask and tile mask of one slot; returns the dirty tiles.
__device__ int emit_layer(const MaskGeom &g, const uint64_t *A, int l, int slot, int *red, int *s_wc,
                          uint64_t *s_tw) {
    const int H = g.Hl[l], WW = g.WWl[l], TW = g.TWl[l];
    const int HWW = H * WW;
    uint64_t *pm = g.pmask[l] + (size_t)slot * HWW;
    for (int w = threadIdx.x; w < HWW; w += blockDim.x) pm[w] = A[w];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ntiles = g.THl[l] * TW;
    uint64_t *tm = g.tmask[l] + (size_t)slot * g.TMWl[l];
    int cnt = 0;
    for (int base = wave * 64; base < ntiles; base += (int)blockDim.x) {
        const int t = base + lane;
        bool dirty = false;
        if (t < ntiles) {
            const int ty = t / TW, tx = t - ty * TW;
            const int x0 = tx * kTile, wx = x0 >> 6, sh = x0 & 63;
            const uint64_t bits = tile_rows(A, ty * kTile, H, WW, wx) >> sh;
            dirty = (bits & ((1ull << kTile) - 1ull)) != 0;
        }
        const uint64_t m = __ballot(dirty);
        if (lane == 0) {
            tm[base >> 6] = m;
            if (l) s_wc[(l - 1) * g.TMW + (base >> 6)] = __popcll(m);
            if (l && s_tw) s_tw[(l - 1) * g.TMW + (base >> 6)] = m;
            cnt += __popcll(m);
        }
    }
    return block_sum(lane == 0 ? cnt : 0, red);
}

// tpfx[l][slot][w] = dirty tiles in tile words 0 .. w - 1 of layer l (1..L),
// from the per-word counts in s_wc ([l - 1][w], row stride TMW); one wave per
// layer, a wave scan per 64 words.
__device__ void write_tpfx(const MaskGeom &g, const int *s_wc, int slot) {
    if (g.tpfx[1] == nullptr) return;            // few words per layer: the list build sums them itself
    const int lane = threadIdx.x & 63, nw = (int)(blockDim.x >> 6);
    for (int l = 1 + (int)(threadIdx.x >> 6); l <= g.L; l += nw) {
        const int TMWl = g.TMWl[l];
        int run = 0;
        for (int b = 0; b < TMWl; b += 64) {
            const int w = b + lane;
            const int c = w < TMWl ? s_wc[(l - 1) * g.TMW + w] : 0;
            int x = c;
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(x, o, 64);
                if (lane >= o) x += y;
            }
            if (w < TMWl) g.tpfx[l][(size_t)slot * TMWl + w] = run + x - c;
            run += __shfl(x, 63, 64);
        }
    }
}

// Work lists of a batch of one stream (batch index 0), from the tile words
// and per-word counts in LDS: layer l's entries are its dirty tiles in
// position order, as the compaction kernel writes them.  One wave per layer:
// a wave scan of the word counts gives each word's offset, then a lane per
// tile bit writes the entry at offset + the set bits below it (mbcnt).
__device__ void write_lists(const MaskGeom &g, const MaskArgs &a, const int *s_wc, const uint64_t *s_tw, int slot) {
    const int lane = threadIdx.x & 63, nw = (int)(blockDim.x >> 6);
    for (int l = 1 + (int)(threadIdx.x >> 6); l <= g.L; l += nw) {
        const int TMWl = g.TMWl[l], TWl = g.TWl[l];
        int run = 0;
        for (int b = 0; b < TMWl; b += 64) {
            const int w = b + lane;
            const int c = w < TMWl ? s_wc[(l - 1) * g.TMW + w] : 0;
            int x = c;
            for (int o = 1; o < 64; o <<= 1) {
                const int y = __shfl_up(x, o, 64);
                if (lane >= o) x += y;
            }
            const int pre = run + x - c;
            const int nwc = min(64, TMWl - b);
            for (int j = 0; j < nwc; ++j) {
                const uint64_t m = s_tw[(l - 1) * g.TMW + b + j];
                const int base = __shfl(pre, j, 64);
                if ((m >> lane) & 1ull) {
                    const int t = 64 * (b + j) + lane;
                    const uint32_t pos = ((uint32_t)(t / TWl) << 8) | (uint32_t)(t % TWl);
                    const int idx = base + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                                           __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                    a.wl[l][idx] = pos;                           // batch index 0
                    a.wls[l][idx] = ((uint32_t)slot << 16) | pos;
                }
            }
            run += __shfl(x, 63, 64);
        }
        if (lane == 0) a.cnt[l] = run;                            // at most the layer's tiles: the list's capacity
    }
}

// Grow a change set by one pixel on every side (3x3 window), clipped to the
// H x W grid (3x3 stride-1 pad-1 layer: the output grid is the input grid).
__device__ void grow1(int H, int W, int WW, const uint64_t *src, uint64_t *dst) {
    const int HWW = H * WW;
    for (int w = threadIdx.x; w < HWW; w += blockDim.x) {
        const int y = w / WW, wx = w - y * WW;
        uint64_t acc = 0;
        for (int dy = -1; dy <= 1; ++dy) {
            const int yy = y + dy;
            if (yy < 0 || yy >= H) continue;
            const uint64_t *row = src + yy * WW;
            const uint64_t c = row[wx];
            const uint64_t lft = wx > 0 ? row[wx - 1] : 0ull;
            const uint64_t rgt = wx + 1 < WW ? row[wx + 1] : 0ull;
            acc |= c | (c << 1) | (lft >> 63) | (c >> 1) | (rgt << 63);
        }
        dst[w] = acc & row_valid_bits(W, wx);
    }
}

// Dilation of a change set by R pixels (every pixel within Chebyshev
// distance R of a changed one), clipped to the H x W grid, in two separable
// passes: the OR of rows y - R .. y + R (k_masks), then the OR of bits
// x - R .. x + R of that row (hdilate_word, word wx).
// Growing by one pixel per 3x3 stride-1 layer, clipped each time, gives the
// same set after R layers: inside a rectangle, a point within distance R of a
// changed pixel is reached by R one-pixel steps that stay in the rectangle.
__device__ inline uint64_t hdilate_word(const uint64_t *row, int W, int WW, int wx, int R) {
    const uint64_t mid = row[wx], lft = wx > 0 ? row[wx - 1] : 0ull, rgt = wx + 1 < WW ? row[wx + 1] : 0ull;
    uint64_t out = mid;
    for (int d = 1; d <= R; ++d) out |= (mid << d) | (lft >> (64 - d)) | (mid >> d) | (rgt << (64 - d));
    return out & row_valid_bits(W, wx);
}

// Bits of the index range [x0, x1) that fall in 64-bit word wx.
__device__ inline uint64_t range_bits(int x0, int x1, int wx) {
    const int lo = max(x0 - 64 * wx, 0), hi = min(x1 - 64 * wx, 64);
    if (hi <= lo) return 0ull;
    const uint64_t upto = hi == 64 ? ~0ull : ((1ull << hi) - 1ull);
    return upto & ~((1ull << lo) - 1ull);
}

// Growth through a general layer l (k x k, stride s, pad p), separably: rows
// first (V row y = OR of the input rows s y - p .. s y - p + k - 1 inside the
// grid, on the input columns), then columns (output bit x = any bit of V row y
// in s x - p .. s x - p + k - 1).  src: layer l - 1's rows; mid: scratch of
// Hl[l] x WWl[l - 1] words; the result goes back to src.
__device__ void grow_general(const MaskGeom &g, int l, uint64_t *src, uint64_t *mid) {
    const int Hi = g.Hl[l - 1], Wi = g.Wl[l - 1], WWi = g.WWl[l - 1];
    const int Ho = g.Hl[l], Wo = g.Wl[l], WWo = g.WWl[l];
    const int k = g.ks[l - 1], s = g.st[l - 1], p = g.pd[l - 1];
    for (int w = threadIdx.x; w < Ho * WWi; w += blockDim.x) {
        const int y = w / WWi, wx = w - y * WWi;
        const int r0 = max(s * y - p, 0), r1 = min(s * y - p + k, Hi);
        uint64_t acc = 0;
        for (int r = r0; r < r1; ++r) acc |= src[r * WWi + wx];
        mid[w] = acc;
    }
    lds_sync();
    // One wave per output word, one lane per output bit (the window spans at
    // most two input words: k <= 8), the word by ballot.
    const int lane = threadIdx.x & 63;
    for (int w = (int)(threadIdx.x >> 6); w < Ho * WWo; w += (int)(blockDim.x >> 6)) {
        const int y = w / WWo, wx = w - y * WWo;
        const uint64_t *row = mid + y * WWi;
        const int x = 64 * wx + lane;
        const int c0 = max(s * x - p, 0), c1 = min(s * x - p + k, Wi);
        bool any = false;
        if (x < Wo && c0 < c1) {
            const int w0 = c0 >> 6, w1 = (c1 - 1) >> 6, sh = c0 & 63;
            uint64_t bits = row[w0] >> sh;
            if (w1 != w0) bits |= row[w1] << (64 - sh);     // sh > 0 here: the window crosses a word edge
            any = (bits & ((1ull << (c1 - c0)) - 1ull)) != 0;
        }
        const uint64_t word = __ballot(any);
        if (lane == 0) src[w] = word;
    }
}

__device__ inline bool standard_layer(const MaskGeom &g, int l) {
    return g.ks[l - 1] == 3 && g.st[l - 1] == 1 && g.pd[l - 1] == 1;
}

template <bool U8, int NT>
__global__ __launch_bounds__(NT) void k_masks(MaskGeom g, MaskArgs a) {
    extern __shared__ uint64_t smem[];
    __shared__ int red[NT / 64];
    __shared__ int s_tiles[RN_MAX_CONV + 1];
    const int HWW = g.H * g.WW;
    uint64_t *A = smem;
    uint64_t *B = smem + HWW;
    // After the bit planes: the tile words of layers 1..L when this kernel
    // writes the lists ([L][TMW]), the level LUT, the per-word tile counts.
    uint64_t *s_tw = a.fuse_lists ? smem + (g.dil ? 2 * g.L + 1 : 2) * HWW : nullptr;
    float *lut = reinterpret_cast<float *>(smem + (g.dil ? 2 * g.L + 1 : 2) * HWW +
                                           (a.fuse_lists ? g.L * g.TMW : 0));
    int *s_wc = reinterpret_cast<int *>(lut + 256);            // [L][TMW] dirty tiles per tile word

    const int i = blockIdx.x;
    const int slot = a.ids ? a.ids[i] : i;
    const int primed = a.force_all ? 0 : a.primed[slot];
    const size_t HW = (size_t)g.H * g.W;
    const int C = g.cin;

    for (int w = threadIdx.x; w < HWW; w += blockDim.x) A[w] = 0ull;
    if (U8)
        for (int j = threadIdx.x; j < 256; j += blockDim.x) lut[j] = a.lut[j];
    lds_sync();

    // Cache planes: the previous newest frame, and where the new frame goes.
    float *prev, *next;
    int head = 0, nhead = 0;
    if (g.stack == 1) {
        prev = next = a.xin + (size_t)slot * C * HW;
    } else {
        head = a.ring_head[slot];
        nhead = (head + 1) & 3;
        prev = a.xin + ((size_t)slot * 4 + head) * C * HW;
        next = a.xin + ((size_t)slot * 4 + nhead) * C * HW;
    }
    const size_t fbase = (size_t)i * C * HW;

    if (a.boxes != nullptr && primed) {
        // Known change (Sec. 1): the boxes are the change set; only box pixels
        // are read from the frame and copied into the cache.
        const int b0 = a.box_off[i], b1 = a.box_off[i + 1];
        for (int b = b0; b < b1; ++b) {
            const int y0 = max(a.boxes[4 * b + 0], 0), x0 = max(a.boxes[4 * b + 1], 0);
            const int y1 = min(a.boxes[4 * b + 2], g.H), x1 = min(a.boxes[4 * b + 3], g.W);
            const int bh = y1 - y0, bw = x1 - x0;
            if (bh <= 0 || bw <= 0) continue;
            for (int e = threadIdx.x; e < bh * bw; e += blockDim.x) {
                const int y = y0 + e / bw, x = x0 + e % bw;
                const size_t px = (size_t)y * g.W + x;
                for (int c = 0; c < C; ++c)
                    next[c * HW + px] = load1<U8>(a.frames, fbase + c * HW + px, lut);
                atomicOr(reinterpret_cast<unsigned long long *>(&A[y * g.WW + (x >> 6)]),
                         1ull << (x & 63));
            }
        }
    } else {
        // Diff, 4 pixels (one 16-byte load per plane) per thread per item; the
        // loads of U items are issued before any compare so that many are in
        // flight per thread.
        constexpr int U = 4;
        const int n4 = (int)(HW / 4);
        for (int q0 = threadIdx.x; q0 < n4; q0 += U * (int)blockDim.x) {
            uint32_t ch[U];
#pragma unroll
            for (int u = 0; u < U; ++u) ch[u] = primed ? 0u : 0xFu;
            for (int c = 0; c < C; ++c) {
                float4 nv[U], ov[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int q = q0 + u * (int)blockDim.x;
                    if (q < n4) {
                        nv[u] = load4<U8>(a.frames, fbase + c * HW + 4 * (size_t)q, lut);
                        ov[u] = *reinterpret_cast<const float4 *>(prev + c * HW + 4 * (size_t)q);
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int q = q0 + u * (int)blockDim.x;
                    if (q >= n4) continue;
                    const uint32_t d = (f32_bits(nv[u].x) != f32_bits(ov[u].x) ? 1u : 0u) |
                                       (f32_bits(nv[u].y) != f32_bits(ov[u].y) ? 2u : 0u) |
                                       (f32_bits(nv[u].z) != f32_bits(ov[u].z) ? 4u : 0u) |
                                       (f32_bits(nv[u].w) != f32_bits(ov[u].w) ? 8u : 0u);
                    ch[u] |= d;
                    if (g.stack != 1 || d != 0u || !primed)
                        *reinterpret_cast<float4 *>(next + c * HW + 4 * (size_t)q) = nv[u];
                    if (g.stack != 1 && !primed) {
                        // Priming a stacked input: every older frame is this frame.
                        for (int r = 0; r < 4; ++r)
                            *reinterpret_cast<float4 *>(a.xin + ((size_t)slot * 4 + r) * C * HW + c * HW +
                                                        4 * (size_t)q) = nv[u];
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = q0 + u * (int)blockDim.x;
                if (q < n4 && ch[u]) {
                    const int p = 4 * q, y = p / g.W, x = p - y * g.W;
                    atomicOr(reinterpret_cast<unsigned long long *>(&A[y * g.WW + (x >> 6)]),
                             (unsigned long long)ch[u] << (x & 63));
                }
            }
        }
    }
    lds_sync();

    if (g.stack != 1) {
        // Stacked input: channel j of step t is frame t-3+j, so the stack
        // changed where any of the last 4 single-frame diffs did.  Keep this
        // step's single-frame diff in the ring and OR the ring together.
        uint64_t *ring = a.dring + (size_t)slot * 4 * HWW;
        for (int w = threadIdx.x; w < HWW; w += blockDim.x) {
            const uint64_t d = A[w];
            if (!primed) {
                for (int r = 0; r < 4; ++r) ring[r * HWW + w] = 0ull;
            } else {
                ring[nhead * HWW + w] = d;
                A[w] = d | ring[((nhead + 1) & 3) * HWW + w] | ring[((nhead + 2) & 3) * HWW + w] |
                       ring[((nhead + 3) & 3) * HWW + w];
            }
        }
        lds_sync();
    }

    if (g.dil) {
        // Every layer 3x3 stride 1 pad 1 (one grid): all layers' masks at once
        // (layer l: the change set dilated by l, rows then columns), then all
        // layers' tile words; three barriers instead of four per layer.
        // LDS: the change set, then the vertical ORs V_l (l = 1..L), then the
        // masks M_l.  Each thread keeps its words' coordinates for all layers
        // (V_l = V_{l-1} | the rows y - l and y + l; M_l from V_l's row).
        __shared__ int s_cnt[RN_MAX_CONV + 2];
        if (threadIdx.x < RN_MAX_CONV + 2) s_cnt[threadIdx.x] = 0;
        int nc = 0;
        for (int w = threadIdx.x; w < HWW; w += blockDim.x) {
            const int y = w / g.WW;
            uint64_t v = A[w];
            nc += __popcll(v);
            g.pmask[0][(size_t)slot * HWW + w] = v;
            for (int l = 1; l <= g.L; ++l) {
                if (y - l >= 0) v |= A[w - l * g.WW];
                if (y + l < g.H) v |= A[w + l * g.WW];
                smem[(size_t)l * HWW + w] = v;
            }
        }
        lds_sync();
        for (int w = threadIdx.x; w < HWW; w += blockDim.x) {
            const int y = w / g.WW, wx = w - y * g.WW;
            for (int l = 1; l <= g.L; ++l) {
                const uint64_t v = hdilate_word(smem + (size_t)l * HWW + y * g.WW, g.W, g.WW, wx, l);
                smem[(size_t)(g.L + l) * HWW + w] = v;
                g.pmask[l][(size_t)slot * HWW + w] = v;
            }
        }
        lds_sync();
        if (nc) atomicAdd(&s_cnt[RN_MAX_CONV + 1], nc);
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int TMW = g.TMW, ntiles = g.TH * g.TW;
        for (int wd = wave; wd < TMW; wd += (int)(blockDim.x >> 6)) {
            const int t = 64 * wd + lane;
            const bool in = t < ntiles;
            const int ty = in ? t / g.TW : 0, tx = in ? t - ty * g.TW : 0;
            const int x0 = tx * kTile, wx = x0 >> 6, sh = x0 & 63;
            const int y0 = ty * kTile;
            for (int l = 0; l <= g.L; ++l) {
                const uint64_t *M = smem + (size_t)(l == 0 ? 0 : g.L + l) * HWW;
                const uint64_t bits = in ? tile_rows(M, y0, g.H, g.WW, wx) >> sh : 0ull;
                const uint64_t m = __ballot((bits & ((1ull << kTile) - 1ull)) != 0);
                if (lane == 0) {
                    g.tmask[l][(size_t)slot * TMW + wd] = m;
                    if (l) s_wc[(l - 1) * TMW + wd] = __popcll(m);
                    if (l && s_tw) s_tw[(l - 1) * TMW + wd] = m;
                    if (m) atomicAdd(&s_cnt[l], __popcll(m));
                }
            }
        }
        lds_sync();
        write_tpfx(g, s_wc, slot);
        if (a.fuse_lists) write_lists(g, a, s_wc, s_tw, slot);
        if (threadIdx.x == 0) {
            a.nchg[i] = s_cnt[RN_MAX_CONV + 1];
            for (int l = 0; l <= g.L; ++l) a.ntile[(size_t)i * (g.L + 1) + l] = s_cnt[l];
            a.primed[slot] = 1;
            if (g.stack != 1) a.ring_head[slot] = nhead;
        }
        return;
    }

    int nchg = 0;
    for (int w = threadIdx.x; w < HWW; w += blockDim.x) nchg += __popcll(A[w]);
    nchg = block_sum(nchg, red);

    int t0 = emit_layer(g, A, 0, slot, red, s_wc, s_tw);
    if (threadIdx.x == 0) s_tiles[0] = t0;
    for (int l = 1; l <= g.L; ++l) {
        lds_sync();
        if (standard_layer(g, l)) {
            grow1(g.Hl[l], g.Wl[l], g.WWl[l], A, B);
            lds_sync();
            uint64_t *t = A;
            A = B;
            B = t;
        } else {
            grow_general(g, l, A, B);
            lds_sync();
        }
        const int tl = emit_layer(g, A, l, slot, red, s_wc, s_tw);
        if (threadIdx.x == 0) s_tiles[l] = tl;
    }
    write_tpfx(g, s_wc, slot);                   // the last block_sum published every count
    if (a.fuse_lists) write_lists(g, a, s_wc, s_tw, slot);
    if (threadIdx.x == 0) {
        a.nchg[i] = nchg;
        for (int l = 0; l <= g.L; ++l) a.ntile[(size_t)i * (g.L + 1) + l] = s_tiles[l];
        a.primed[slot] = 1;
        if (g.stack != 1) a.ring_head[slot] = nhead;
    }
}

// Dense path: copy every pixel of the frames into the input cache, mark the
// slots primed and report every pixel and tile as recomputed.
// Stacked input (one block per slot: the block reads the slot's primed flag
// and ring head before its thread 0 updates them): an unprimed slot takes the
// frame at all four ring positions (before 4 frames exist, frame 0 repeats)
// and an empty change ring, as a first step does; a primed slot pushes the
// frame into its ring as a step does, with the frame's own change against
// the newest cached frame in the change ring, so the steps that follow see
// the stack's change exactly as after a step on this frame.
template <bool U8>
__global__ __launch_bounds__(kThreads) void k_prime(PrimeArgs a) {
    const int i = blockIdx.x;
    const int slot = a.ids[i];
    const size_t HW = (size_t)a.H * a.W;
    const int C = a.cin;
    const size_t fbase = (size_t)i * C * HW;
    if (a.stack == 1) {
        const int n4 = (int)(HW / 4);
        for (int q = blockIdx.y * blockDim.x + threadIdx.x; q < n4; q += gridDim.y * blockDim.x)
            for (int c = 0; c < C; ++c) {
                const float4 v = load4<U8>(a.frames, fbase + c * HW + 4 * (size_t)q, a.lut);
                *reinterpret_cast<float4 *>(a.xin + (size_t)slot * C * HW + c * HW + 4 * (size_t)q) = v;
            }
    } else {
        const int primed = a.primed[slot];
        const int head = a.ring_head[slot];
        const int nhead = primed ? (head + 1) & 3 : 0;
        float *planes = a.xin + (size_t)slot * 4 * C * HW;        // ring position r: planes + r C HW
        const float *prev = planes + (size_t)head * C * HW;
        uint64_t *ring = a.dring + (size_t)slot * a.dring_words;  // [4][H][WW]
        const size_t HWW = (size_t)a.H * a.WW;
        for (size_t w = threadIdx.x; w < HWW; w += blockDim.x) {
            const int y = (int)(w / a.WW), x0 = (int)(w - (size_t)y * a.WW) * 64;
            const int x1 = min(x0 + 64, a.W);
            uint64_t bits = 0ull;
            for (int c = 0; c < C; ++c)
                for (int x = x0; x < x1; x += 4) {
                    const size_t px = c * HW + (size_t)y * a.W + x;
                    const float4 v = load4<U8>(a.frames, fbase + px, a.lut);
                    if (primed) {
                        const float4 o = *reinterpret_cast<const float4 *>(prev + px);
                        const uint64_t d = (f32_bits(v.x) != f32_bits(o.x) ? 1u : 0u) |
                                           (f32_bits(v.y) != f32_bits(o.y) ? 2u : 0u) |
                                           (f32_bits(v.z) != f32_bits(o.z) ? 4u : 0u) |
                                           (f32_bits(v.w) != f32_bits(o.w) ? 8u : 0u);
                        bits |= d << (x - x0);
                        *reinterpret_cast<float4 *>(planes + (size_t)nhead * C * HW + px) = v;
                    } else {
                        for (int r = 0; r < 4; ++r)
                            *reinterpret_cast<float4 *>(planes + (size_t)r * C * HW + px) = v;
                    }
                }
            if (primed) {
                ring[(size_t)nhead * HWW + w] = bits;
            } else {
                for (int r = 0; r < 4; ++r) ring[(size_t)r * HWW + w] = 0ull;
            }
        }
        __syncthreads();                      // every thread has read the flags
        if (threadIdx.x == 0) a.ring_head[slot] = nhead;
    }
    if (blockIdx.y == 0 && threadIdx.x == 0) {
        a.primed[slot] = 1;
        a.nchg[i] = (int)HW;
        for (int l = 0; l <= a.L; ++l) a.ntile[(size_t)i * (a.L + 1) + l] = a.ntl[l];
    }
}

// Work lists, position-major: the entries of layer l are its dirty tiles in
// (ty, tx, batch index) order.  One block per (64-position word wd, layer):
//   - its offset is the number of dirty tiles at earlier positions: over
//     the streams, the popcount of tile-mask words 0..wd-1 (for grids of
//     more than 16 words, the per-slot word prefix that k_masks wrote);
//   - a 64 x 64 bit transpose per chunk of 64 streams (lane r holds stream
//     r's word; six exchange stages leave lane j with position j's stream
//     bitmap) gives per-position counts and the streams of each position.
// Every entry has exactly one writer; no global atomics.
constexpr int kChunksPerPass = 16;          // 1024 streams per pass

// 64 x 64 bit-matrix transpose across a wave: on entry lane r holds row r
// (bit c = element (r, c)); on return lane c holds column c (bit r = element
// (r, c)).  Stage s (32, 16, .., 1) swaps the off-diagonal s x s blocks of
// every 2s x 2s block between lanes r and r ^ s.
__device__ inline uint64_t transpose64(uint64_t x, int lane) {
    const uint64_t masks[6] = {0x00000000FFFFFFFFull, 0x0000FFFF0000FFFFull, 0x00FF00FF00FF00FFull,
                               0x0F0F0F0F0F0F0F0Full, 0x3333333333333333ull, 0x5555555555555555ull};
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        const int sh = 32 >> k;
        const uint64_t m = masks[k];
        const uint32_t lo = __shfl_xor((uint32_t)x, sh, 64), hi = __shfl_xor((uint32_t)(x >> 32), sh, 64);
        const uint64_t y = ((uint64_t)hi << 32) | lo;
        x = (lane & sh) ? (x & ~m) | ((y & ~m) >> sh) : (x & m) | ((y & m) << sh);
    }
    return x;
}

// Stage the slots and this word's tile bits of streams [64 c0, 64 (c0 + nc)) in LDS.
__device__ inline void stage_pass(const CompactArgs &a, int l, int wd, int c0, int nc, int32_t *s_slot,
                                  uint64_t *s_word) {
    for (int j = threadIdx.x; j < nc * 64; j += blockDim.x) {
        const int i = 64 * c0 + j;
        const int slot = i >= a.n ? -1 : a.ids ? a.ids[i] : i;
        s_slot[j] = slot;
        s_word[j] = slot >= 0 ? a.tmask[l][(size_t)slot * a.TMWl[l] + wd] : 0ull;
    }
}

__global__ __launch_bounds__(kThreads) void k_compact_pos(CompactArgs a) {
    __shared__ int red[kThreads / 64];
    __shared__ int s_cnt[64];
    __shared__ int s_run[64];
    __shared__ int s_most;
    __shared__ int s_base[kChunksPerPass][64];
    __shared__ uint64_t s_bal[kChunksPerPass][64];
    __shared__ int32_t s_slot[kChunksPerPass * 64];
    __shared__ uint64_t s_word[kChunksPerPass * 64];
    const int wd = blockIdx.x, l = blockIdx.y + 1;
    const int TMW = a.TMWl[l], TW = a.TWl[l], ntiles = a.ntl[l];
    if (wd >= TMW) return;                       // the grid covers the widest layer; uniform per block
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nwaves = (int)(blockDim.x >> 6);
    const int nch = (a.n + 63) / 64;
    const int nc0 = min(kChunksPerPass, nch);

    // One pass over the streams (thread per stream): dirty tiles at positions
    // before this word (the per-slot word prefix k_masks wrote), and the first
    // pass's slots and words of this word staged in LDS.
    // Four streams per thread at a time, their loads issued together.
    constexpr int UB = 4;
    int pre = 0;
    for (int i0 = threadIdx.x; i0 < 64 * nc0 || i0 < a.n; i0 += UB * (int)blockDim.x) {
        int slot[UB];
#pragma unroll
        for (int u = 0; u < UB; ++u) {
            const int i = i0 + u * (int)blockDim.x;
            slot[u] = i >= a.n ? -1 : a.ids ? a.ids[i] : i;
        }
        int pf[UB];
        uint64_t word[UB];
#pragma unroll
        for (int u = 0; u < UB; ++u) {
            const int i = i0 + u * (int)blockDim.x;
            pf[u] = slot[u] >= 0 && wd > 0 && a.tpfx[l] != nullptr ? a.tpfx[l][(size_t)slot[u] * TMW + wd] : 0;
            word[u] = i < 64 * nc0 && slot[u] >= 0 ? a.tmask[l][(size_t)slot[u] * TMW + wd] : 0ull;
        }
#pragma unroll
        for (int u = 0; u < UB; ++u) {
            const int i = i0 + u * (int)blockDim.x;
            pre += pf[u];
            if (slot[u] >= 0 && wd > 0 && a.tpfx[l] == nullptr) {
                const uint64_t *tm = a.tmask[l] + (size_t)slot[u] * TMW;
                for (int w = 0; w < wd; ++w) pre += __popcll(tm[w]);
            }
            if (i < 64 * nc0) {
                s_slot[i] = slot[u];
                s_word[i] = word[u];
            }
        }
    }
    pre = block_sum(pre, red);                   // its barriers also publish the staging
    if (threadIdx.x < 64) s_cnt[threadIdx.x] = 0;

    // Per-position counts of this word over all streams.
    for (int c0 = 0; c0 < nch; c0 += kChunksPerPass) {
        const int nc = min(kChunksPerPass, nch - c0);
        if (c0 > 0) {
            lds_sync();
            stage_pass(a, l, wd, c0, nc, s_slot, s_word);
        }
        lds_sync();
        for (int cc = wave; cc < nc; cc += nwaves) {
            const uint64_t b = transpose64(s_word[cc * 64 + lane], lane);
            s_bal[cc][lane] = b;
            atomicAdd(&s_cnt[lane], __popcll(b));   // LDS
        }
    }
    lds_sync();
    if (threadIdx.x < 64) {
        // Exclusive scan of the position counts, after the earlier words' total.
        const int c = s_cnt[lane];
        int x = c;
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(x, o, 64);
            if (lane >= o) x += y;
        }
        s_run[lane] = pre + x - c;
        if (lane == 63 && wd == TMW - 1) a.cnt[l] = (int)min((size_t)(pre + x), a.cap[l]);   // the last word closes the list
    }
    lds_sync();

    const size_t cap = a.cap[l];
    for (int c0 = 0; c0 < nch; c0 += kChunksPerPass) {
        const int nc = min(kChunksPerPass, nch - c0);
        if (nch > kChunksPerPass) {
            // More than one pass: stage and transpose this pass again (with a
            // single pass, LDS still holds it from the counting loop).
            lds_sync();
            stage_pass(a, l, wd, c0, nc, s_slot, s_word);
            lds_sync();
            for (int cc = wave; cc < nc; cc += nwaves) s_bal[cc][lane] = transpose64(s_word[cc * 64 + lane], lane);
            lds_sync();
        }
        const int npos = min(64, ntiles - 64 * wd);       // positions of this word inside the grid
        if (threadIdx.x < 64) {
            int r = s_run[threadIdx.x], most = 0;
            for (int cc = 0; cc < nc; ++cc) {
                s_base[cc][threadIdx.x] = r;
                const int c = __popcll(s_bal[cc][threadIdx.x]);
                r += c;
                most = max(most, c);
            }
            s_run[threadIdx.x] = r;
            for (int o = 32; o > 0; o >>= 1) most = max(most, __shfl_xor(most, o, 64));
            if (threadIdx.x == 0) s_most = most;
        }
        lds_sync();
        // Entries of (chunk cc, position j) are [base, base + popcount) in
        // stream order.  Either one thread per (chunk, position) walks the set
        // bits of its stream bitmap, or, when the busiest bitmap has more bits
        // than a wave has bitmaps to visit (few positions, dense bitmaps: small
        // grids of strided layers), one wave per bitmap with a lane per stream
        // (rank among the set bits by mbcnt).  Both write the same entries.
        if (s_most > (nc * npos + nwaves - 1) / nwaves) {
            for (int q = wave; q < nc * npos; q += nwaves) {
                const int cc = q / npos, j = q - cc * npos;
                const uint64_t b = s_bal[cc][j];
                if ((b >> lane) & 1ull) {
                    const int t = 64 * wd + j;
                    const uint32_t pos = ((uint32_t)(t / TW) << 8) | (uint32_t)(t % TW);
                    const int idx = s_base[cc][j] + (int)__builtin_amdgcn_mbcnt_hi(
                                        (uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
                    if ((size_t)idx < cap) {
                        a.wl[l][idx] = ((uint32_t)(64 * (c0 + cc) + lane) << 16) | pos;
                        a.wls[l][idx] = ((uint32_t)s_slot[cc * 64 + lane] << 16) | pos;
                    }
                }
            }
        } else {
            for (int pi = threadIdx.x; pi < nc * 64; pi += blockDim.x) {
                const int cc = pi >> 6, j = pi & 63;
                const int t = 64 * wd + j;
                uint64_t b = s_bal[cc][j];
                if (j >= npos) continue;
                const uint32_t pos = ((uint32_t)(t / TW) << 8) | (uint32_t)(t % TW);
                int idx = s_base[cc][j];
                while (b) {
                    const int k = __ffsll((long long)b) - 1;  // next stream of this position
                    b &= b - 1;
                    const int i = 64 * (c0 + cc) + k;
                    if ((size_t)idx < cap) {
                        a.wl[l][idx] = ((uint32_t)i << 16) | pos;
                        a.wls[l][idx] = ((uint32_t)s_slot[cc * 64 + k] << 16) | pos;
                    }
                    ++idx;
                }
            }
        }
    }
}

// ------------------------------------------------------------------ variants
//
// The change set of a variant is a union of boxes, and growing a union grows
// each member: the layer-l set is every box clipped to the frame, widened by
// R_l (the summed growth radii of layers 1..l) on each side and clipped again
// (Fig. 1's one-pixel growth per 3x3 layer, composed; exact for rectangles).
// Every mask word is therefore a direct test against the boxes, with no
// layer-to-layer dependence, and the tiles a box touches form a rectangle of
// the tile grid.
//
// k_var_pix: one wave per (variant, layer); lanes own pixel rows and 64-tile
// words; per-variant counts by wave reduction.
// k_var_bits: one wave per (64-variant chunk, layer 1..L, tile word): the
// chunk's words transposed across the lanes (transpose64) into one
// 64-variant bitmap per tile position, bits[l][t][chunk], with variants over the per-variant limit
// cleared, and each position's entry count summed (integer atomics: the sum
// does not depend on their order).
// k_var_lists: block (b, l) owns positions [b P, b P + P); its entries start
// after those of every earlier position, and a block scan over its
// (position, chunk) bitmaps places each entry: position-major, variants
// ascending within a position, as for streams.

constexpr int kVarThreads = 1024;

__device__ inline int wave_sum(int v) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Box k grown by R and clipped, (y0, x0, y1, x1); empty (y1 <= y0 or x1 <= x0)
// when the box is empty after clipping to the frame.
__device__ inline int4 grown_box(const VarMaskArgs &a, int k, int R) {
    const int32_t *b = a.boxes + 4 * (size_t)k;
    const int y0 = max(b[0], 0), x0 = max(b[1], 0), y1 = min(b[2], a.H), x1 = min(b[3], a.W);
    if (y1 <= y0 || x1 <= x0) return make_int4(0, 0, 0, 0);
    return make_int4(max(y0 - R, 0), max(x0 - R, 0), min(y1 + R, a.H), min(x1 + R, a.W));
}

__global__ __launch_bounds__(256) void k_var_pix(VarMaskArgs a) {
    const int lane = threadIdx.x & 63;
    const int task = blockIdx.x * 4 + (threadIdx.x >> 6);
    // Block 0 also clears the per-position entry counts that k_var_bits adds to.
    if (blockIdx.x == 0)
        for (int j = threadIdx.x; j < a.L * a.ntiles; j += blockDim.x) a.pos_cnt[j] = 0;
    if (task >= a.n * (a.L + 1)) return;
    const int i = task / (a.L + 1), l = task - i * (a.L + 1);
    const int R = a.R[l];
    const int k0 = a.box_off[i], k1 = a.box_off[i + 1];
    int px = 0, tl = 0;
    for (int y = lane; y < a.H; y += 64) {
        uint64_t *dst = a.pmask[l] + ((size_t)i * a.H + y) * a.WW;
        for (int wx = 0; wx < a.WW; ++wx) {
            uint64_t word = 0;
            for (int k = k0; k < k1; ++k) {
                const int4 g = grown_box(a, k, R);
                if (y >= g.x && y < g.z) word |= range_bits(g.y, g.w, wx);
            }
            dst[wx] = word;
            px += __popcll(word);
        }
    }
    for (int wd = lane; wd < a.TMW; wd += 64) {
        uint64_t word = 0;
        const int t0 = 64 * wd, t1 = t0 + 64;
        for (int k = k0; k < k1; ++k) {
            const int4 g = grown_box(a, k, R);
            if (g.z <= g.x) continue;
            const int ty0 = g.x / kTile, ty1 = (g.z + kTile - 1) / kTile;
            const int tx0 = g.y / kTile, tx1 = (g.w + kTile - 1) / kTile;
            // tile rows whose index range [ty TW + tx0, ty TW + tx1) can meet [t0, t1)
            const int r0 = max(ty0, (t0 - tx1) / a.TW), r1 = min(ty1, t1 / a.TW + 1);
            for (int ty = r0; ty < r1; ++ty) word |= range_bits(ty * a.TW + tx0, ty * a.TW + tx1, wd);
        }
        a.tmask[l][(size_t)i * a.TMW + wd] = word;
        tl += __popcll(word);
    }
    px = wave_sum(px);
    tl = wave_sum(tl);
    if (lane == 0) {
        a.ntile[(size_t)i * (a.L + 1) + l] = tl;
        if (l == 0) a.nchg[i] = px;
    }
}

__global__ __launch_bounds__(256) void k_var_bits(VarMaskArgs a) {
    const int lane = threadIdx.x & 63;
    const int task = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (task >= a.nch * a.L * a.TMW) return;
    const int wd = task % a.TMW, r = task / a.TMW;
    const int l = 1 + r % a.L, c = r / a.L;
    const int i = 64 * c + lane;
    bool ok = i < a.n;
    if (ok && a.vmax > 0)
        for (int q = 1; q <= a.L; ++q) ok = ok && a.ntile[(size_t)i * (a.L + 1) + q] <= a.vmax;
    const uint64_t w = ok ? a.tmask[l][(size_t)i * a.TMW + wd] : 0ull;
    const uint64_t mine = transpose64(w, lane);         // position 64 wd + lane's variant bitmap
    const int t = 64 * wd + lane;
    if (t < a.ntiles) {
        a.bits[l][(size_t)t * a.nch + c] = mine;
        if (mine) atomicAdd(&a.pos_cnt[(size_t)(l - 1) * a.ntiles + t], __popcll(mine));
    }
}

// Exclusive block-wide prefix sum of v; *total receives the block's sum.
__device__ inline int block_excl_scan(int v, int *s_w, int *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = (int)(blockDim.x >> 6);
    int x = v;
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    lds_sync();                      // s_w of the previous call has been read
    if (lane == 63) s_w[wave] = x;
    lds_sync();
    int off = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
        const int s = s_w[w];
        off += w < wave ? s : 0;
        tot += s;
    }
    *total = tot;
    return off + x - v;
}

__global__ __launch_bounds__(kVarThreads) void k_var_lists(VarMaskArgs a) {
    __shared__ int red[kVarThreads / 64];
    __shared__ int s_w[kVarThreads / 64];
    const int l = blockIdx.y + 1;
    const int P = max(1, (int)blockDim.x / a.nch);
    const int t0 = blockIdx.x * P, t1 = min(t0 + P, a.ntiles);
    const uint64_t *B = a.bits[l];
    int pre = 0;
    for (int t = threadIdx.x; t < t0; t += blockDim.x) pre += a.pos_cnt[(size_t)(l - 1) * a.ntiles + t];
    int run = block_sum(pre, red);
    const size_t k0 = (size_t)t0 * a.nch, k1 = (size_t)t1 * a.nch;
    for (size_t base = k0; base < k1; base += blockDim.x) {
        const size_t k = base + threadIdx.x;
        const uint64_t w = k < k1 ? B[k] : 0ull;
        int total;
        int idx = run + block_excl_scan(__popcll(w), s_w, &total);
        if (w) {
            const int t = (int)(k / a.nch), cc = (int)(k - (size_t)t * a.nch);
            const uint32_t pos = ((uint32_t)(t / a.TW) << 8) | (uint32_t)(t % a.TW);
            uint64_t b = w;
            while (b) {
                const int j = __ffsll((long long)b) - 1;
                b &= b - 1;
                const int i = 64 * cc + j;
                if ((size_t)idx < a.cap) {
                    a.wl[l][idx] = ((uint32_t)i << 16) | pos;
                    a.vmap[l][(size_t)i * a.ntiles + t] = idx;
                }
                ++idx;
            }
        }
        run += total;
    }
    if (t1 == a.ntiles && threadIdx.x == 0) a.cnt[l] = (int)min((size_t)run, a.cap);
}

}  // namespace

hipError_t launch_var_masks(const VarMaskArgs &a, hipStream_t s) {
    const int waves = a.n * (a.L + 1);
    hipLaunchKernelGGL(k_var_pix, dim3((waves + 3) / 4), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int tw = a.nch * a.L * a.TMW;
    hipLaunchKernelGGL(k_var_bits, dim3((tw + 3) / 4), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_var_lists(const VarMaskArgs &a, hipStream_t s) {
    const int P = std::max(1, kVarThreads / a.nch);
    hipLaunchKernelGGL(k_var_lists, dim3((a.ntiles + P - 1) / P, a.L), dim3(kVarThreads), 0, s, a);
    return hipGetLastError();
}

// Dynamic LDS of k_masks growing layer by layer: two bit planes of the input
// grid, the LUT and the per-word tile counts.
size_t masks_lds_bytes(int H, int WW, int L, int TMW) {
    return (size_t)2 * H * WW * sizeof(uint64_t) + 256 * sizeof(float) + (size_t)L * TMW * sizeof(int);
}

hipError_t launch_masks(const MaskGeom &geom, const MaskArgs &args, int cus, hipStream_t s, bool *fused) {
    MaskGeom g = geom;
    MaskArgs a = args;
    const size_t hww = (size_t)g.H * g.WW;
    bool all_std = true;
    for (int l = 0; l < g.L; ++l) all_std = all_std && g.ks[l] == 3 && g.st[l] == 1 && g.pd[l] == 1;
    const size_t tail = 256 * sizeof(float) + (size_t)g.L * g.TMW * sizeof(int);   // LUT, per-word tile counts
    const size_t dil_bytes = (size_t)(2 * g.L + 1) * hww * sizeof(uint64_t) + tail;
    g.dil = all_std && dil_bytes <= 48 * 1024 ? 1 : 0;
    size_t shm = g.dil ? dil_bytes : masks_lds_bytes(g.H, g.WW, g.L, g.TMW);
    // One stream: the block that has its tile words also writes the lists
    // (saving the compaction launch), when their words fit the default LDS.
    const size_t tw_bytes = (size_t)g.L * g.TMW * sizeof(uint64_t);
    a.fuse_lists = a.n == 1 && a.wl[1] != nullptr && shm + tw_bytes <= 64 * 1024 ? 1 : 0;
    if (a.fuse_lists) shm += tw_bytes;
    *fused = a.fuse_lists != 0;
    const int nt = a.n <= cus ? 1024 : a.n <= 4 * cus ? 512 : 256;
    hipError_t attr = hipSuccess;
    auto go = [&](auto kern) {
        // Above the default 64 KiB of dynamic LDS (frames of more than ~4 K
        // mask words) the kernel has to be allowed more; create checks the limit.
        if (shm > 64 * 1024)
            attr = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)shm);
        if (attr == hipSuccess) hipLaunchKernelGGL(kern, dim3(a.n), dim3(nt), shm, s, g, a);
    };
    if (a.frame_u8) {
        if (nt == 1024) go(k_masks<true, 1024>);
        else if (nt == 512) go(k_masks<true, 512>);
        else go(k_masks<true, 256>);
    } else {
        if (nt == 1024) go(k_masks<false, 1024>);
        else if (nt == 512) go(k_masks<false, 512>);
        else go(k_masks<false, 256>);
    }
    return attr != hipSuccess ? attr : hipGetLastError();
}

hipError_t launch_prime(const PrimeArgs &a, hipStream_t s) {
    dim3 grid(a.n, a.stack == 1 ? 4 : 1);     // stacked: one block per slot (see k_prime)
    if (a.frame_u8)
        hipLaunchKernelGGL(k_prime<true>, grid, dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(k_prime<false>, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_compact(const CompactArgs &a, hipStream_t s) {
    int tmw = 1;
    for (int l = 1; l <= a.L; ++l) tmw = std::max(tmw, a.TMWl[l]);
    dim3 grid(tmw, a.L);
    hipLaunchKernelGGL(k_compact_pos, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace rn
