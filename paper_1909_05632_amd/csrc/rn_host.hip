// Host side of reuse_net: config validation, workspace layout, weight packing,
// and the per-step launch sequence
//   masks (diff or boxes, growth, tile masks) -> work lists -> conv layer 1 ->
//   conv layers 2..L -> dense head,
// all enqueued on the caller's stream with no host synchronisation.
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "rn_internal.hpp"
#include "rn_train.hpp"

using namespace rn;

namespace {

thread_local std::string g_create_error;

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

struct Plan {
    int L = 0, H = 0, W = 0, WW = 0, TH = 0, TW = 0, TMW = 0, ntiles = 0;   // input grid
    // Layer l's output grid (l = 0: the input) and its tiles.
    int Hl[RN_MAX_CONV + 1] = {0}, Wl[RN_MAX_CONV + 1] = {0}, WWl[RN_MAX_CONV + 1] = {0};
    int THl[RN_MAX_CONV + 1] = {0}, TWl[RN_MAX_CONV + 1] = {0}, TMWl[RN_MAX_CONV + 1] = {0};
    int ntl[RN_MAX_CONV + 1] = {0};
    int ks[RN_MAX_CONV] = {0}, st[RN_MAX_CONV] = {0}, pd[RN_MAX_CONV] = {0};   // of layer l + 1
    bool gen[RN_MAX_CONV] = {false};       // layer l + 1 is not 3x3 stride 1 pad 1 (general kernel)
    bool any_gen = false;
    int in_c = 0, stack = 1, S = 0, N = 0;
    rn_dtype dt = RN_F32;
    size_t esz = 4;
    int C[RN_MAX_CONV + 1] = {0};          // channels per layer (0 = conv1 input)
    int radius[RN_MAX_CONV] = {0};         // change growth per layer, (k - 1) / 2
    size_t K = 0;                          // head input elements per slot (tiled)
    int head_mode = RN_HEAD_TILES;
    bool part_f32 = false;                 // float32 tile partials by position (own kernel) instead of in the epilogue
    bool fuse_first = false;               // layer 1 folded into layer 2's halo staging
    int head_sg = 8;
    size_t part_elems = 0;
    // byte offsets into the workspace
    size_t o_lut, o_xin, o_ring, o_dring, o_primed, o_ids, o_act[RN_MAX_CONV + 1], o_w[RN_MAX_CONV],
        o_b[RN_MAX_CONV], o_wd, o_bd, o_pm[RN_MAX_CONV + 1], o_tm[RN_MAX_CONV + 1], o_tpfx[RN_MAX_CONV + 1], o_nchg, o_ntile,
        o_wl[RN_MAX_CONV + 1], o_wls[RN_MAX_CONV + 1], o_cnt, o_part, o_hw, o_hw2, o_hp;
    size_t w_elems[RN_MAX_CONV] = {0};
    size_t w_bytes[RN_MAX_CONV] = {0};
    // Training (backward and SGD step): float32 nets of 3x3 stride-1 pad-1
    // layers at the kernels' shapes; o_wt[l] holds layer l's weights
    // transposed and flipped for the input-gradient product (l >= 1, i.e.
    // conv layers 2..L).
    const char *train_why = nullptr;        // NULL: training supported
    size_t o_wt[RN_MAX_CONV] = {0};
    size_t wt_elems[RN_MAX_CONV] = {0};
    size_t act_stride[RN_MAX_CONV + 1] = {0};   // elements per slot
    size_t total = 0;
};

void head_split(const Plan &p, int n, int *nsplit, size_t *chunk) {
    const int groups = ceil_div(n, p.head_sg);
    const size_t max_split = std::max<size_t>(1, (p.K + 1023) / 1024);
    size_t ns = std::min<size_t>(max_split, std::max<size_t>(1, (size_t)ceil_div(2048, groups)));
    size_t ch = (p.K + ns - 1) / ns;
    ch = (ch + 1023) / 1024 * 1024;
    *chunk = ch;
    *nsplit = (int)((p.K + ch - 1) / ch);
}

rn_status plan_config(const rn_config *cfg, Plan *p, std::string *err) {
    auto fail = [&](rn_status st, const std::string &m) {
        *err = m;
        return st;
    };
    if (!cfg) return fail(RN_EINVAL, "config is NULL");
    if (cfg->n_conv < 1 || cfg->n_conv > RN_MAX_CONV) return fail(RN_EINVAL, "n_conv must be 1..8");
    if (!cfg->conv) return fail(RN_EINVAL, "conv specs are NULL");
    if (cfg->in_c < 1 || cfg->in_h < 1 || cfg->in_w < 1) return fail(RN_EINVAL, "bad frame shape");
    if (cfg->stack != 1 && cfg->stack != 4) return fail(RN_EINVAL, "stack must be 1 or 4");
    if (cfg->n_out < 1 || cfg->n_out > kHeadMaxOut) return fail(RN_EINVAL, "n_out must be 1..64");
    if (cfg->max_streams < 1 || cfg->max_streams > 65535) return fail(RN_EINVAL, "max_streams must be 1..65535");
    if (cfg->act_dtype != RN_F32 && cfg->act_dtype != RN_BF16) return fail(RN_EINVAL, "act_dtype must be F32 or BF16");
    if (cfg->tile_h < 1 || cfg->tile_w < 1) return fail(RN_EINVAL, "bad tile");
    int c = cfg->in_c * cfg->stack;
    for (int l = 0; l < cfg->n_conv; ++l) {
        const rn_conv_spec &s = cfg->conv[l];
        if (s.cin != c) return fail(RN_EINVAL, "conv channel chain is inconsistent at layer " + std::to_string(l + 1));
        if (s.cout < 1 || s.k < 1 || s.stride < 1 || s.pad < 0) return fail(RN_EINVAL, "bad conv spec");
        if (s.pad > (s.k - 1) / 2) return fail(RN_EINVAL, "conv pad must be at most (k-1)/2");
        if (s.k > 8 || (s.stride != 1 && s.stride != 2 && s.stride != 4))
            return fail(RN_EUNSUPPORTED, "conv layers need k <= 8 and stride 1, 2 or 4");
        c = s.cout;
    }
    if (cfg->tile_h != kTile || cfg->tile_w != kTile) return fail(RN_EUNSUPPORTED, "only 4x4 tiles are implemented");
    if (cfg->in_w % 4 != 0) return fail(RN_EUNSUPPORTED, "in_w must be a multiple of 4");
    if (cfg->stack == 4 && cfg->in_c != 1) return fail(RN_EUNSUPPORTED, "stack = 4 needs in_c = 1");
    if (cfg->head_mode != RN_HEAD_TILES && cfg->head_mode != RN_HEAD_FULL) return fail(RN_EINVAL, "bad head_mode");
    if (cfg->options & ~RN_OPT_SEPARATE_FIRST) return fail(RN_EINVAL, "unknown option bits");
    p->L = cfg->n_conv;
    p->H = cfg->in_h;
    p->W = cfg->in_w;
    p->WW = ceil_div(p->W, 64);
    p->TH = ceil_div(p->H, kTile);
    p->TW = ceil_div(p->W, kTile);
    if (p->TH > 256 || p->TW > 256) return fail(RN_EUNSUPPORTED, "frames above 1024 x 1024 are not implemented");
    p->ntiles = p->TH * p->TW;
    p->TMW = ceil_div(p->ntiles, 64);
    if (masks_lds_bytes(p->H, p->WW, cfg->n_conv, p->TMW) > kMasksLdsMax)
        return fail(RN_EUNSUPPORTED, "frame too large: the mask kernel keeps two bit planes of it in LDS "
                                     "(in_h x ceil(in_w / 64) must stay under about 10000 words)");
    p->Hl[0] = p->H;
    p->Wl[0] = p->W;
    for (int l = 0; l < cfg->n_conv; ++l) {
        const rn_conv_spec &cs = cfg->conv[l];
        p->ks[l] = cs.k;
        p->st[l] = cs.stride;
        p->pd[l] = cs.pad;
        p->gen[l] = !(cs.k == 3 && cs.stride == 1 && cs.pad == 1);
        p->any_gen = p->any_gen || p->gen[l];
        const int nh = p->Hl[l] + 2 * cs.pad - cs.k, nw = p->Wl[l] + 2 * cs.pad - cs.k;
        if (nh < 0 || nw < 0) return fail(RN_EINVAL, "layer " + std::to_string(l + 1) + " leaves no output pixels");
        p->Hl[l + 1] = nh / cs.stride + 1;
        p->Wl[l + 1] = nw / cs.stride + 1;
    }
    for (int l = 0; l <= cfg->n_conv; ++l) {
        p->WWl[l] = ceil_div(p->Wl[l], 64);
        p->THl[l] = ceil_div(p->Hl[l], kTile);
        p->TWl[l] = ceil_div(p->Wl[l], kTile);
        p->ntl[l] = p->THl[l] * p->TWl[l];
        p->TMWl[l] = ceil_div(p->ntl[l], 64);
    }
    p->in_c = cfg->in_c;
    p->stack = cfg->stack;
    p->S = cfg->max_streams;
    p->N = cfg->n_out;
    p->dt = cfg->act_dtype;
    p->esz = p->dt == RN_F32 ? 4 : 2;
    p->C[0] = cfg->in_c * cfg->stack;
    for (int l = 0; l < p->L; ++l) {
        p->C[l + 1] = cfg->conv[l].cout;
        p->radius[l] = (cfg->conv[l].k - 1) / 2;
    }
    const bool bf = p->dt == RN_BF16;
    const char *dts = bf ? " (bf16)" : " (float32)";
    if (bf && p->any_gen) return fail(RN_EUNSUPPORTED, "bf16 needs 3x3 stride-1 pad-1 layers");
    auto shape = [&](int l) {
        return std::to_string(p->C[l - 1]) + "->" + std::to_string(p->C[l]) +
               (p->gen[l - 1] ? " (" + std::to_string(p->ks[l - 1]) + "x" + std::to_string(p->ks[l - 1]) + " stride " +
                                    std::to_string(p->st[l - 1]) + ")"
                              : "") +
               dts;
    };
    if (p->gen[0] ? !conv_gen_supported(p->ks[0], p->st[0], p->C[0], p->C[1], true)
                  : !(bf ? conv_first_bf16_supported(p->C[0], p->C[1]) : conv_first_supported(p->C[0], p->C[1], p->dt)))
        return fail(RN_EUNSUPPORTED, "no first-layer kernel for " + shape(1));
    for (int l = 2; l <= p->L; ++l)
        if (p->gen[l - 1] ? !conv_gen_supported(p->ks[l - 1], p->st[l - 1], p->C[l - 1], p->C[l], false)
                          : !(bf ? conv_mfma_bf16_supported(p->C[l - 1], p->C[l])
                                 : conv_mfma_supported(p->C[l - 1], p->C[l], p->dt)))
            return fail(RN_EUNSUPPORTED, "no MFMA conv kernel for " + shape(l));
    p->K = (size_t)p->ntl[p->L] * kTilePx * p->C[p->L];
    p->fuse_first = !(cfg->options & RN_OPT_SEPARATE_FIRST) && p->L >= 2 && p->C[0] == 1 && p->stack == 1 &&
                    !p->gen[0] && !p->gen[1] && conv_fused_first_supported(p->C[1], p->C[2], p->dt);
    // The tile-partial head lives in the epilogue of an MFMA layer (float32) or
    // in its own matrix kernel after the last layer (bf16).
    p->head_mode = (cfg->head_mode == RN_HEAD_TILES && (p->L >= 2 || p->gen[p->L - 1]) &&
                    (!bf || tile_part_bf16_supported(p->C[p->L])))
                       ? RN_HEAD_TILES
                       : RN_HEAD_FULL;
    p->part_f32 = p->head_mode == RN_HEAD_TILES && !bf && p->L >= 2 && !p->gen[p->L - 1] &&
                  conv_mfma_is_staged(p->C[p->L - 1], p->C[p->L]) && tile_part_f32_supported(p->C[p->L]);
    p->head_sg = head_streams_per_block(p->N);
    size_t part = 0;
    for (int n = 1; n <= p->S; ++n) {
        int ns;
        size_t ch;
        head_split(*p, n, &ns, &ch);
        part = std::max(part, (size_t)ns * n);
    }
    p->part_elems = part * p->N;

    const size_t S = p->S, HW = (size_t)p->H * p->W, HWW = (size_t)p->H * p->WW;   // input grid
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + std::max<size_t>(bytes, 1));
        return o;
    };
    p->o_lut = take(256 * 4);
    p->o_xin = take(S * p->stack * p->in_c * HW * 4);
    p->o_ring = take(S * 4);
    p->o_dring = take(p->stack == 4 ? S * 4 * HWW * 8 : 0);
    p->o_primed = take(S * 4);
    p->o_ids = take(S * 4);
    p->act_stride[0] = (size_t)p->stack * p->in_c * HW;
    for (int l = 1; l <= p->L; ++l) {
        p->act_stride[l] = (size_t)p->ntl[l] * kTilePx * p->C[l];
        p->o_act[l] = take(S * p->act_stride[l] * p->esz);
    }
    for (int l = 0; l < p->L; ++l) {
        p->w_elems[l] = p->gen[l] ? conv_gen_packed_elems(p->ks[l], p->C[l], p->C[l + 1])
                        : l == 0  ? conv_first_packed_elems(p->C[0], p->C[1])
                                  : conv_mfma_packed_elems(p->C[l], p->C[l + 1], p->dt);
        // layer 1 keeps float32 weights (bf16-rounded values in bf16 mode); MFMA layers store bf16.
        p->w_bytes[l] = p->w_elems[l] * ((l > 0 && p->dt == RN_BF16) ? 2 : 4);
        p->o_w[l] = take(p->w_bytes[l]);
        p->o_b[l] = take((size_t)p->C[l + 1] * 4);
    }
    if (p->dt != RN_F32) p->train_why = "training needs a float32 net";
    else if (p->any_gen) p->train_why = "training needs 3x3 stride-1 pad-1 layers";
    else if (!train_shapes_supported(p->C[0], p->C[1], true)) p->train_why = "no backward kernel for the first layer's channels";
    for (int l = 1; l < p->L && !p->train_why; ++l)
        if (!train_shapes_supported(p->C[l], p->C[l + 1], false) || !train_dx_supported(p->C[l + 1], p->C[l]))
            p->train_why = "no backward kernels for a layer's channel pair";
    for (int l = 1; l < p->L; ++l) {
        p->wt_elems[l] = p->train_why ? 0 : dx_weights_elems(p->C[l + 1], p->C[l]);
        p->o_wt[l] = take(p->wt_elems[l] * 4);
    }
    p->o_wd = take((size_t)p->N * p->K * 4);
    p->o_bd = take((size_t)p->N * 4);
    for (int l = 0; l <= p->L; ++l) {
        p->o_pm[l] = take(S * p->Hl[l] * p->WWl[l] * 8);
        p->o_tm[l] = take(S * p->TMWl[l] * 8);
        p->o_tpfx[l] = take(l ? S * p->TMWl[l] * 4 : 0);
    }
    p->o_nchg = take(S * 4);
    p->o_ntile = take(S * (p->L + 1) * 4);
    for (int l = 1; l <= p->L; ++l) {
        p->o_wl[l] = take(S * p->ntl[l] * 4);
        p->o_wls[l] = take(S * p->ntl[l] * 4);
    }
    p->o_cnt = take((RN_MAX_CONV + 1) * 4);
    const bool tiles_head = p->head_mode == RN_HEAD_TILES;
    p->o_part = take(tiles_head ? 0 : p->part_elems * 4);
    // Epilogue head weights: float32 last layers whose conv kernel forms the
    // tile partials (a staged last layer leaves them to k_tile_part_f32, o_hw2).
    p->o_hw = take(!tiles_head || p->part_f32 ? 0
                   : p->dt == RN_BF16 ? tile_part_bf16_elems(p->ntl[p->L], p->C[p->L], p->N) * 2
                                      : tile_head_w_elems(p->ntl[p->L], p->C[p->L], p->N) * 4);
    p->o_hw2 = take(p->part_f32 ? tile_part_f32_elems(p->ntl[p->L], p->C[p->L], p->N) * 4 : 0);
    p->o_hp = take(tiles_head ? S * p->ntl[p->L] * p->N * 4 : 0);
    p->total = off;
    return RN_OK;
}

// Scratch layout of a reuse_net_variants call: per-variant masks, the work
// lists, (variant, tile) -> list index maps, the overlays of recomputed tiles
// (row = list index) and the recomputed tiles' head partials.
struct VarPlan {
    int n = 0, vmax = 0;                   // vmax 0: no per-variant limit
    size_t cap = 0;                        // list capacity per layer
    size_t o_pm[RN_MAX_CONV + 1], o_tm[RN_MAX_CONV + 1], o_nchg, o_ntile, o_wl[RN_MAX_CONV + 1],
        o_map[RN_MAX_CONV + 1], o_ov[RN_MAX_CONV + 1], o_bits[RN_MAX_CONV + 1], o_pcnt, o_hp, o_cnt;
    bool has_ov[RN_MAX_CONV + 1] = {false};
    size_t total = 0;
};

// Layer l's recomputed tiles are read back by layer l + 1 (unless layer 1 is
// folded into layer 2) or, bf16 or staged float32 last layer, by the
// head-partial kernel; another float32 last layer feeds the head from its
// epilogue and stores nothing.
VarPlan plan_variants(const Plan &p, int n, int max_tiles) {
    VarPlan v;
    v.n = n;
    v.vmax = (max_tiles <= 0 || max_tiles >= p.ntiles) ? 0 : max_tiles;
    v.cap = (size_t)n * (v.vmax ? v.vmax : p.ntiles);
    const size_t HWW = (size_t)p.H * p.WW;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + std::max<size_t>(bytes, 1));
        return o;
    };
    for (int l = 0; l <= p.L; ++l) {
        v.o_pm[l] = take((size_t)n * HWW * 8);
        v.o_tm[l] = take((size_t)n * p.TMW * 8);
    }
    v.o_nchg = take((size_t)n * 4);
    v.o_ntile = take((size_t)n * (p.L + 1) * 4);
    const size_t nch = ((size_t)n + 63) / 64;
    for (int l = 1; l <= p.L; ++l) {
        v.o_wl[l] = take(v.cap * 4);
        v.o_map[l] = take((size_t)n * p.ntiles * 4);
        v.o_bits[l] = take((size_t)p.ntiles * nch * 8);
        v.has_ov[l] = l < p.L ? !(l == 1 && p.fuse_first) : p.dt == RN_BF16 || p.part_f32;
        v.o_ov[l] = take(v.has_ov[l] ? v.cap * kTilePx * p.C[l] * p.esz : 0);
    }
    v.o_pcnt = take((size_t)p.L * p.ntiles * 4);
    v.o_hp = take(v.cap * p.N * 4);
    v.o_cnt = take((RN_MAX_CONV + 1) * 4);
    v.total = off;
    return v;
}

struct ProfRec {
    int phase;
    int layer;                            // conv layer 1..L of the launch, 0 for other kernels
    hipEvent_t e0, e1;
};

// Scratch of reuse_net_variants_static: a file-scope device array, so the
// call needs no allocation.  Each GPU the library runs on holds its own copy
// until the process ends; host code must use the per-device address from
// hipGetSymbolAddress, never the array's name (a host-side stand-in).
static __device__ __align__(256) unsigned char scratch[RN_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {nullptr};

// Device address of `scratch` on device dev (looked up once per device, with
// dev current).  NULL and a message in *err on failure.
void *static_scratch(int dev, std::string *err) {
    if (dev < 0 || dev >= kMaxDevices) {
        *err = "device index beyond the static scratch table";
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
        void *p = nullptr;
        if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
        if (e != hipSuccess || !p) {
            *err = std::string("static scratch address: ") + hipGetErrorString(e);
            return nullptr;
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

struct reuse_net {
    Plan p;
    rn_config cfg;
    char *ws = nullptr;
    int dev = 0;                         // the device current at create
    int cus = 256;
    hipStream_t last_stream = nullptr;
    int last_n = 0;
    bool has_step = false;
    bool last_was_full = false;
    bool last_was_var = false;           // the last call was reuse_net_variants
    char *var_scratch = nullptr;         // ... with this scratch and layout
    VarPlan var_plan;
    bool prof = false;
    std::vector<hipEvent_t> pool;
    size_t pool_used = 0;
    std::vector<ProfRec> recs;
    std::string err;

    template <typename T>
    T *at(size_t off) const { return reinterpret_cast<T *>(ws + off); }

    rn_status fail(rn_status st, const std::string &m) {
        err = m;
        return st;
    }
    hipEvent_t next_event() {
        if (pool_used == pool.size()) {
            hipEvent_t e;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            pool.push_back(e);
        }
        return pool[pool_used++];
    }
};

namespace {

template <typename F>
hipError_t timed(reuse_net *net, int phase, hipStream_t s, F &&fn, int layer = 0) {
    if (!net->prof) return fn();
    hipEvent_t e0 = net->next_event(), e1 = net->next_event();
    if (!e0 || !e1) return hipErrorOutOfMemory;
    (void)hipEventRecord(e0, s);
    hipError_t e = fn();
    (void)hipEventRecord(e1, s);
    net->recs.push_back({phase, layer, e0, e1});
    return e;
}

rn_status sync_last(reuse_net *net) {
    if (!net->has_step) return RN_OK;
    hipError_t e = hipStreamSynchronize(net->last_stream);
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("stream sync: ") + hipGetErrorString(e));
    return RN_OK;
}

MaskGeom make_geom(reuse_net *net) {
    const Plan &p = net->p;
    MaskGeom g{};
    g.L = p.L;
    g.H = p.H;
    g.W = p.W;
    g.WW = p.WW;
    g.TH = p.TH;
    g.TW = p.TW;
    g.TMW = p.TMW;
    g.cin = p.in_c;
    g.stack = p.stack;
    for (int l = 0; l <= p.L; ++l) {
        g.Hl[l] = p.Hl[l];
        g.Wl[l] = p.Wl[l];
        g.WWl[l] = p.WWl[l];
        g.THl[l] = p.THl[l];
        g.TWl[l] = p.TWl[l];
        g.TMWl[l] = p.TMWl[l];
    }
    for (int l = 0; l < p.L; ++l) {
        g.ks[l] = p.ks[l];
        g.st[l] = p.st[l];
        g.pd[l] = p.pd[l];
    }
    for (int l = 0; l <= p.L; ++l) {
        g.pmask[l] = net->at<uint64_t>(p.o_pm[l]);
        g.tmask[l] = net->at<uint64_t>(p.o_tm[l]);
        // Per-slot word prefixes only pay for grids of many tile words.
        g.tpfx[l] = l && p.TMW > 16 ? net->at<int32_t>(p.o_tpfx[l]) : nullptr;
    }
    return g;
}

// Conv layers 1..L (list mode: the work lists; dense mode: every tile), then the head.
// identity: the batch is slots 0..n-1 in order (ids is then the identity table;
// kernels that only need a stream's slot skip loading it).
hipError_t run_layers(reuse_net *net, int n, const int32_t *ids, bool identity, uint32_t *const *wl,
                      const int32_t *cnt, float *logits, hipStream_t s, bool dense) {
    const Plan &p = net->p;
    const bool tiles_head = p.head_mode == RN_HEAD_TILES;
    hipError_t e = hipSuccess;
    ConvArgs last{};
    for (int l = 1; l <= p.L; ++l) {
        if (l == 1 && p.fuse_first) continue;            // computed inside layer 2
        ConvArgs cv{};
        cv.wl = dense ? nullptr : wl[l];
        cv.cnt = dense ? nullptr : cnt + l;
        cv.ids = ids;
        cv.in = l == 1 ? static_cast<const void *>(net->at<float>(p.o_xin)) : net->at<void>(p.o_act[l - 1]);
        cv.out = net->at<void>(p.o_act[l]);
        cv.w = net->at<void>(p.o_w[l - 1]);
        cv.bias = net->at<float>(p.o_b[l - 1]);
        cv.ring_head = net->at<int32_t>(p.o_ring);
        cv.H = p.Hl[l];
        cv.W = p.Wl[l];
        cv.TH = p.THl[l];
        cv.TW = p.TWl[l];
        cv.Hin = p.Hl[l - 1];
        cv.Win = p.Wl[l - 1];
        cv.TWin = p.TWl[l - 1];
        cv.pad = p.pd[l - 1];
        cv.cin = p.C[l - 1];
        cv.cout = p.C[l];
        cv.stack = p.stack;
        cv.in_stride = p.act_stride[l - 1];
        cv.out_stride = p.act_stride[l];
        cv.dense_n = dense ? n : 0;
        cv.max_tiles = n * p.ntl[l];
        if (l == 2 && p.fuse_first) {
            cv.fuse_first = 1;
            cv.in = net->at<float>(p.o_xin);
            cv.in_stride = p.act_stride[0];
            cv.w1 = net->at<float>(p.o_w[0]);
            cv.b1 = net->at<float>(p.o_b[0]);
        }
        const bool bf = p.dt == RN_BF16;
        if (l == p.L && tiles_head) {
            cv.n_out = p.N;
            cv.hw = net->at<float>(p.o_hw);
            cv.hpart = net->at<float>(p.o_hp);
            last = cv;
            if (bf || p.part_f32) cv.n_out = 0;           // partials from their own kernel below
        }
        if (p.gen[l - 1])
            e = timed(net, l == 1 ? RN_PHASE_CONV1 : RN_PHASE_CONVN, s, [&] {
                return launch_conv_gen(cv, p.ks[l - 1], p.st[l - 1], l == 1, net->cus, s);
            }, l);
        else if (l == 1)
            e = timed(net, RN_PHASE_CONV1, s, [&] {
                return bf ? launch_conv_first_bf16(cv, net->cus, s) : launch_conv_first(cv, p.dt, net->cus, s);
            }, l);
        else
            e = timed(net, RN_PHASE_CONVN, s, [&] {
                return bf ? launch_conv_mfma_bf16(cv, net->cus, s) : launch_conv_mfma(cv, p.dt, net->cus, s);
            }, l);
        if (e != hipSuccess) return e;
    }
    if (tiles_head && (p.dt == RN_BF16 || p.part_f32)) {
        // bf16, or a float32 last layer on the staged kernel: the tiles of the
        // last work list (every tile in dense mode) get their partials from a
        // matrix kernel by position, reading the updated cache.
        last.in = net->at<void>(p.o_act[p.L]);
        last.in_stride = p.act_stride[p.L];
        if (p.part_f32) last.hw = net->at<float>(p.o_hw2);
        e = timed(net, RN_PHASE_HEAD, s, [&] {
            return p.part_f32 ? launch_tile_part_f32(last, net->cus, s) : launch_tile_part_bf16(last, net->cus, s);
        });
        if (e != hipSuccess) return e;
    }
    if (tiles_head) {
        TileHeadArgs ta{};
        ta.n = n;
        ta.n_out = p.N;
        ta.ntiles = p.ntl[p.L];
        ta.ids = identity ? nullptr : ids;
        ta.hpart = net->at<float>(p.o_hp);
        ta.bias = net->at<float>(p.o_bd);
        ta.logits = logits;
        return timed(net, RN_PHASE_HEAD, s, [&] { return launch_tile_head(ta, s); });
    }
    HeadArgs ha{};
    ha.n = n;
    ha.n_out = p.N;
    ha.ids = ids;
    ha.act = net->at<void>(p.o_act[p.L]);
    ha.w = net->at<void>(p.o_wd);
    ha.bias = net->at<float>(p.o_bd);
    ha.part = net->at<float>(p.o_part);
    ha.logits = logits;
    ha.K = p.K;
    head_split(p, n, &ha.nsplit, &ha.chunk);
    return timed(net, RN_PHASE_HEAD, s, [&] { return launch_head(ha, p.dt, s); });
}

rn_status run_step(reuse_net *net, int32_t n, const int32_t *ids_in, const void *frames, rn_dtype fdt,
                   const int32_t *boxes, const int32_t *box_off, float *logits, void *stream) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (n < 1 || n > p.S) return net->fail(RN_EINVAL, "n must be 1..max_streams");
    if (!frames) return net->fail(RN_EINVAL, "frames are NULL");
    if (!logits) return net->fail(RN_EINVAL, "logits are NULL");
    if (fdt != RN_F32 && fdt != RN_U8) return net->fail(RN_EINVAL, "frame dtype must be F32 or U8");
    if (boxes && !box_off) return net->fail(RN_EINVAL, "boxes given without box offsets");
    if (boxes && p.stack != 1) return net->fail(RN_EUNSUPPORTED, "change boxes with stacked frames are not implemented");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int32_t *ids = ids_in ? ids_in : net->at<int32_t>(p.o_ids);

    MaskGeom g = make_geom(net);
    MaskArgs ma{};
    ma.n = n;
    ma.ids = ids_in;                          // NULL: the identity batch, no table load
    ma.frames = frames;
    ma.frame_u8 = fdt == RN_U8;
    ma.boxes = boxes;
    ma.box_off = box_off;
    ma.force_all = 0;
    ma.lut = net->at<float>(p.o_lut);
    ma.xin = net->at<float>(p.o_xin);
    ma.ring_head = net->at<int32_t>(p.o_ring);
    ma.dring = net->at<uint64_t>(p.o_dring);
    ma.primed = net->at<int32_t>(p.o_primed);
    ma.nchg = net->at<int32_t>(p.o_nchg);
    ma.ntile = net->at<int32_t>(p.o_ntile);
    for (int l = 1; l <= p.L; ++l) {
        ma.wl[l] = net->at<uint32_t>(p.o_wl[l]);
        ma.wls[l] = net->at<uint32_t>(p.o_wls[l]);
    }
    ma.cnt = net->at<int32_t>(p.o_cnt);
    bool fused = false;
    hipError_t e = timed(net, RN_PHASE_MASKS, s, [&] { return launch_masks(g, ma, net->cus, s, &fused); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("mask kernel: ") + hipGetErrorString(e));

    CompactArgs ca{};
    ca.n = n;
    ca.L = p.L;
    for (int l = 0; l <= p.L; ++l) {
        ca.TWl[l] = p.TWl[l];
        ca.TMWl[l] = p.TMWl[l];
        ca.ntl[l] = p.ntl[l];
        ca.cap[l] = (size_t)n * p.ntl[l];
    }
    ca.ids = ids_in;
    ca.ntile = ma.ntile;
    for (int l = 0; l <= p.L; ++l) {
        ca.tmask[l] = g.tmask[l];
        ca.tpfx[l] = g.tpfx[l];
        ca.wl[l] = l ? net->at<uint32_t>(p.o_wl[l]) : nullptr;
        ca.wls[l] = l ? net->at<uint32_t>(p.o_wls[l]) : nullptr;
    }
    ca.cnt = net->at<int32_t>(p.o_cnt);
    if (!fused) {
        e = timed(net, RN_PHASE_COMPACT, s, [&] { return launch_compact(ca, s); });
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("compaction kernel: ") + hipGetErrorString(e));
    }

    e = run_layers(net, n, ids, ids_in == nullptr, ca.wls, ca.cnt, logits, s, false);
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("conv/head kernels: ") + hipGetErrorString(e));
    net->last_stream = s;
    net->last_n = n;
    net->has_step = true;
    net->last_was_full = false;
    net->last_was_var = false;
    net->err.clear();
    return RN_OK;
}

const char *variants_unsupported(const Plan &p) {
    if (p.any_gen) return "variants need 3x3 stride-1 pad-1 layers";
    if (p.head_mode != RN_HEAD_TILES) return "variants need the tile-partial head (head_mode RN_HEAD_TILES, >= 2 layers)";
    if (p.stack != 1) return "variants with stacked frames are not implemented";
    return nullptr;
}

// n variants of slot `base` in one pass: masks from the boxes, lists and maps,
// each layer's recomputed tiles into its overlay, the head from base and
// variant partials.
rn_status run_variants(reuse_net *net, int32_t base, int32_t n, const void *frames, rn_dtype fdt,
                       int32_t frame_count, const int32_t *boxes, const int32_t *box_off, int32_t max_tiles,
                       void *scratch, size_t scratch_bytes, float *logits, void *stream) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (const char *why = variants_unsupported(p)) return net->fail(RN_EUNSUPPORTED, why);
    if (base < 0 || base >= p.S) return net->fail(RN_EINVAL, "base_stream out of range");
    if (n < 1 || n > 65535) return net->fail(RN_EINVAL, "n must be 1..65535");
    if (!frames) return net->fail(RN_EINVAL, "frames are NULL");
    if (frame_count != 1 && frame_count != n) return net->fail(RN_EINVAL, "frame_count must be 1 or n");
    if (fdt != RN_F32 && fdt != RN_U8) return net->fail(RN_EINVAL, "frame dtype must be F32 or U8");
    if (!boxes || !box_off) return net->fail(RN_EINVAL, "variants need boxes and box offsets");
    if (!logits) return net->fail(RN_EINVAL, "logits are NULL");
    if (!scratch) return net->fail(RN_EINVAL, "scratch is NULL");
    if (reinterpret_cast<uintptr_t>(scratch) % kAlign) return net->fail(RN_EINVAL, "scratch must be 256-byte aligned");
    const VarPlan vp = plan_variants(p, n, max_tiles);
    if (vp.cap > (size_t)INT32_MAX) return net->fail(RN_EINVAL, "n x max_tiles exceeds 2^31 work-list entries");
    if (scratch_bytes < vp.total)
        return net->fail(RN_ENOSPACE, "scratch too small: need " + std::to_string(vp.total) + " bytes");
    hipStream_t s = static_cast<hipStream_t>(stream);
    char *sc = static_cast<char *>(scratch);
    auto at = [&](size_t off) { return static_cast<void *>(sc + off); };

    VarMaskArgs va{};
    va.n = n;
    va.L = p.L;
    va.H = p.H;
    va.W = p.W;
    va.WW = p.WW;
    va.TH = p.TH;
    va.TW = p.TW;
    va.TMW = p.TMW;
    va.ntiles = p.ntiles;
    va.nch = (n + 63) / 64;
    va.vmax = vp.vmax;
    for (int l = 1; l <= p.L; ++l) va.R[l] = va.R[l - 1] + p.radius[l - 1];
    va.boxes = boxes;
    va.box_off = box_off;
    for (int l = 0; l <= p.L; ++l) {
        va.pmask[l] = static_cast<uint64_t *>(at(vp.o_pm[l]));
        va.tmask[l] = static_cast<uint64_t *>(at(vp.o_tm[l]));
        if (l) {
            va.bits[l] = static_cast<uint64_t *>(at(vp.o_bits[l]));
            va.wl[l] = static_cast<uint32_t *>(at(vp.o_wl[l]));
            va.vmap[l] = static_cast<int32_t *>(at(vp.o_map[l]));
        }
    }
    va.nchg = static_cast<int32_t *>(at(vp.o_nchg));
    va.ntile = static_cast<int32_t *>(at(vp.o_ntile));
    va.cnt = static_cast<int32_t *>(at(vp.o_cnt));
    va.pos_cnt = static_cast<int32_t *>(at(vp.o_pcnt));
    va.cap = vp.cap;
    hipError_t e = timed(net, RN_PHASE_MASKS, s, [&] { return launch_var_masks(va, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("mask kernel: ") + hipGetErrorString(e));
    e = timed(net, RN_PHASE_COMPACT, s, [&] { return launch_var_lists(va, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("work-list kernel: ") + hipGetErrorString(e));

    const bool bf = p.dt == RN_BF16;
    ConvArgs last{};
    for (int l = 1; l <= p.L; ++l) {
        if (l == 1 && p.fuse_first) continue;
        ConvArgs cv{};
        cv.wl = va.wl[l];
        cv.cnt = va.cnt + l;
        cv.in = l == 1 ? static_cast<const void *>(net->at<float>(p.o_xin)) : net->at<void>(p.o_act[l - 1]);
        cv.w = net->at<void>(p.o_w[l - 1]);
        cv.bias = net->at<float>(p.o_b[l - 1]);
        cv.H = p.H;
        cv.W = p.W;
        cv.TH = p.TH;
        cv.TW = p.TW;
        cv.cin = p.C[l - 1];
        cv.cout = p.C[l];
        cv.stack = p.stack;
        cv.in_stride = p.act_stride[l - 1];
        cv.out_stride = p.act_stride[l];
        cv.max_tiles = (int)std::min<size_t>(vp.cap, (size_t)INT32_MAX);
        cv.Hin = p.H;
        cv.Win = p.W;
        cv.TWin = p.TW;
        cv.pad = 1;
        cv.vbase = base;
        cv.vcin = p.in_c;
        cv.WW = p.WW;
        if (l >= 2) {
            cv.vtm_in = va.tmask[l - 1];
            cv.vmap_in = va.vmap[l - 1];
            cv.vov_in = at(vp.o_ov[l - 1]);
        }
        cv.vov_out = vp.has_ov[l] ? at(vp.o_ov[l]) : nullptr;
        cv.vpm0 = va.pmask[0];
        cv.vframes = frames;
        cv.vframe_u8 = fdt == RN_U8;
        cv.vframe_shared = frame_count == 1 ? 1 : 0;
        cv.lut = net->at<float>(p.o_lut);
        if (l == 2 && p.fuse_first) {
            cv.fuse_first = 1;
            cv.in = net->at<float>(p.o_xin);
            cv.in_stride = p.act_stride[0];
            cv.w1 = net->at<float>(p.o_w[0]);
            cv.b1 = net->at<float>(p.o_b[0]);
        }
        if (l == p.L) {
            cv.n_out = p.N;
            cv.hw = net->at<float>(p.o_hw);
            cv.vhpart = static_cast<float *>(at(vp.o_hp));
            last = cv;
            if (bf || p.part_f32) cv.n_out = 0;
        }
        if (l == 1)
            e = timed(net, RN_PHASE_CONV1, s, [&] {
                return bf ? launch_conv_first_bf16(cv, net->cus, s, true) : launch_conv_first(cv, p.dt, net->cus, s, true);
            }, l);
        else
            e = timed(net, RN_PHASE_CONVN, s, [&] {
                return bf ? launch_conv_mfma_bf16(cv, net->cus, s, true) : launch_conv_mfma(cv, p.dt, net->cus, s, true);
            }, l);
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("conv kernels: ") + hipGetErrorString(e));
    }
    if (bf || p.part_f32) {
        last.vov_in = at(vp.o_ov[p.L]);
        if (p.part_f32) last.hw = net->at<float>(p.o_hw2);
        e = timed(net, RN_PHASE_HEAD, s, [&] {
            return p.part_f32 ? launch_tile_part_f32(last, net->cus, s, true) : launch_tile_part_bf16(last, net->cus, s, true);
        });
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("head partials: ") + hipGetErrorString(e));
    }
    TileHeadArgs ta{};
    ta.n = n;
    ta.n_out = p.N;
    ta.ntiles = p.ntiles;
    ta.hpart = net->at<float>(p.o_hp);
    ta.bias = net->at<float>(p.o_bd);
    ta.logits = logits;
    ta.var = 1;
    ta.vbase = base;
    ta.L = p.L;
    ta.TMW = p.TMW;
    ta.vmax = vp.vmax;
    ta.vtm = va.tmask[p.L];
    ta.vmap = va.vmap[p.L];
    ta.vhpart = static_cast<float *>(at(vp.o_hp));
    ta.ntile = va.ntile;
    ta.primed = net->at<int32_t>(p.o_primed);
    e = timed(net, RN_PHASE_HEAD, s, [&] { return launch_tile_head(ta, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("head: ") + hipGetErrorString(e));
    net->last_stream = s;
    net->last_n = n;
    net->has_step = true;
    net->last_was_full = false;
    net->last_was_var = true;
    net->var_scratch = sc;
    net->var_plan = vp;
    net->err.clear();
    return RN_OK;
}

rn_status run_full(reuse_net *net, int32_t n, const int32_t *ids_in, const void *frames, rn_dtype fdt,
                   float *logits, void *stream) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (n < 1 || n > p.S) return net->fail(RN_EINVAL, "n must be 1..max_streams");
    if (!frames) return net->fail(RN_EINVAL, "frames are NULL");
    if (!logits) return net->fail(RN_EINVAL, "logits are NULL");
    if (fdt != RN_F32 && fdt != RN_U8) return net->fail(RN_EINVAL, "frame dtype must be F32 or U8");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int32_t *ids = ids_in ? ids_in : net->at<int32_t>(p.o_ids);
    PrimeArgs pa{};
    pa.n = n;
    pa.L = p.L;
    pa.cin = p.in_c;
    pa.stack = p.stack;
    pa.H = p.H;
    pa.W = p.W;
    pa.WW = p.WW;
    for (int l = 0; l <= p.L; ++l) pa.ntl[l] = p.ntl[l];
    pa.ids = ids;
    pa.frames = frames;
    pa.frame_u8 = fdt == RN_U8;
    pa.lut = net->at<float>(p.o_lut);
    pa.xin = net->at<float>(p.o_xin);
    pa.ring_head = net->at<int32_t>(p.o_ring);
    pa.dring = net->at<uint64_t>(p.o_dring);
    pa.primed = net->at<int32_t>(p.o_primed);
    pa.nchg = net->at<int32_t>(p.o_nchg);
    pa.ntile = net->at<int32_t>(p.o_ntile);
    pa.dring_words = p.stack == 4 ? (size_t)4 * p.H * p.WW : 0;
    hipError_t e = timed(net, RN_PHASE_MASKS, s, [&] { return launch_prime(pa, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("prime kernel: ") + hipGetErrorString(e));
    e = run_layers(net, n, ids, ids_in == nullptr, nullptr, nullptr, logits, s, true);
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("conv/head kernels: ") + hipGetErrorString(e));
    net->last_stream = s;
    net->last_n = n;
    net->has_step = true;
    net->last_was_full = true;
    net->last_was_var = false;
    net->err.clear();
    return RN_OK;
}

// Pack the weights into the kernels' layouts on the host and enqueue their
// upload on s (weights, biases, dense weights, tile-head weights).
hipError_t upload_weights(reuse_net *net, const rn_weights *w, hipStream_t s) {
    const Plan &p = net->p;
    const bool bf = p.dt == RN_BF16;
    auto rnd = [&](float v) { return bf ? round_bf16_host(v) : v; };
    std::vector<std::vector<unsigned char>> wpack(p.L);
    for (int l = 0; l < p.L; ++l) {
        wpack[l].assign(p.w_bytes[l], 0);
        if (p.gen[l]) {
            pack_conv_gen(w->conv_w[l], p.ks[l], p.C[l], p.C[l + 1], reinterpret_cast<float *>(wpack[l].data()));
        } else if (l == 0) {
            float *d = reinterpret_cast<float *>(wpack[l].data());
            pack_conv_first(w->conv_w[0], p.C[0], p.C[1], p.dt, d);
            for (size_t j = 0; j < p.w_elems[0]; ++j) d[j] = rnd(d[j]);
        } else if (bf) {
            pack_conv_mfma_bf16(w->conv_w[l], p.C[l], p.C[l + 1], wpack[l].data());
        } else {
            pack_conv_mfma(w->conv_w[l], p.C[l], p.C[l + 1], p.dt, wpack[l].data());
        }
    }
    std::vector<std::vector<float>> wtpack(p.L);
    for (int l = 1; l < p.L; ++l)
        if (p.wt_elems[l]) {
            wtpack[l].assign(p.wt_elems[l], 0.f);
            pack_dx_weights(w->conv_w[l], p.C[l], p.C[l + 1], wtpack[l].data());
        }
    // Dense weights from (c, y, x) order to the tiled cache order, 0 at padded pixels.
    const int CL = p.C[p.L], HL = p.Hl[p.L], WL = p.Wl[p.L], THL = p.THl[p.L], TWL = p.TWl[p.L];
    std::vector<float> wd((size_t)p.N * p.K, 0.f);
    for (int o = 0; o < p.N; ++o)
        for (int ty = 0; ty < THL; ++ty)
            for (int tx = 0; tx < TWL; ++tx)
                for (int m = 0; m < kTilePx; ++m) {
                    const int y = ty * kTile + m / kTile, x = tx * kTile + m % kTile;
                    if (y >= HL || x >= WL) continue;
                    const size_t dst = (size_t)o * p.K + ((size_t)(ty * TWL + tx) * kTilePx + m) * CL;
                    for (int c = 0; c < CL; ++c)
                        wd[dst + c] = rnd(w->dense_w[(size_t)o * CL * HL * WL + ((size_t)c * HL + y) * WL + x]);
                }
    hipError_t e = hipSuccess;
    auto up = [&](size_t off, const void *src, size_t n) {
        if (e == hipSuccess) e = hipMemcpyAsync(net->ws + off, src, n, hipMemcpyHostToDevice, s);
    };
    for (int l = 0; l < p.L; ++l) {
        up(p.o_w[l], wpack[l].data(), p.w_bytes[l]);
        up(p.o_b[l], w->conv_b[l], (size_t)p.C[l + 1] * 4);
        if (p.wt_elems[l]) up(p.o_wt[l], wtpack[l].data(), p.wt_elems[l] * 4);
    }
    up(p.o_wd, wd.data(), wd.size() * 4);
    std::vector<float> hw;
    std::vector<uint16_t> hwb;
    if (p.head_mode == RN_HEAD_TILES && bf) {
        hwb.assign(tile_part_bf16_elems(p.ntl[p.L], CL, p.N), 0);
        pack_tile_part_bf16(w->dense_w, p.N, CL, HL, WL, THL, TWL, hwb.data());
        up(p.o_hw, hwb.data(), hwb.size() * 2);
    } else if (p.head_mode == RN_HEAD_TILES && !p.part_f32) {
        hw.assign(tile_head_w_elems(p.ntl[p.L], CL, p.N), 0.f);
        pack_tile_head(w->dense_w, p.N, CL, HL, WL, THL, TWL, hw.data());
        for (float &v : hw) v = rnd(v);
        up(p.o_hw, hw.data(), hw.size() * 4);
    }
    std::vector<float> hw2;
    if (p.part_f32) {
        hw2.assign(tile_part_f32_elems(p.ntl[p.L], CL, p.N), 0.f);
        pack_tile_part_f32(w->dense_w, p.N, CL, HL, WL, THL, TWL, hw2.data());
        up(p.o_hw2, hw2.data(), hw2.size() * 4);
    }
    up(p.o_bd, w->dense_b, (size_t)p.N * 4);
    // pageable host buffers: the copies are done with the vectors before they go
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    return e;
}

// NULL checks of a weight set (message in *err).
rn_status check_weights(const Plan &p, const rn_weights *w, std::string *err) {
    if (!w || !w->conv_w || !w->conv_b || !w->dense_w || !w->dense_b) {
        *err = "weights are NULL";
        return RN_EINVAL;
    }
    for (int l = 0; l < p.L; ++l)
        if (!w->conv_w[l] || !w->conv_b[l]) {
            *err = "conv weights of layer " + std::to_string(l + 1) + " are NULL";
            return RN_EINVAL;
        }
    return RN_OK;
}


// Offsets (floats) of each weight's gradient in a gradient buffer: the
// rn_weights order, conv layer l's OIHW weights then its bias, then the
// dense weights [n_out][C_L][H_L][W_L] and the dense bias.
struct GradLayout {
    size_t w[RN_MAX_CONV], b[RN_MAX_CONV], dw, db, total;
};

GradLayout grad_layout(const Plan &p) {
    GradLayout g{};
    size_t off = 0;
    for (int l = 0; l < p.L; ++l) {
        g.w[l] = off;
        off += (size_t)p.C[l + 1] * p.C[l] * 9;
        g.b[l] = off;
        off += (size_t)p.C[l + 1];
    }
    g.dw = off;
    off += (size_t)p.N * p.C[p.L] * p.Hl[p.L] * p.Wl[p.L];
    g.db = off;
    off += (size_t)p.N;
    g.total = off;
    return g;
}

// Scratch of a backward call for n streams: two gradient buffers of the
// largest layer (dJ/dz of layer l and of layer l - 1) and the dW partial sums
// of the largest layer.
struct BwdPlan {
    size_t o_dz0, o_dz1, o_part, total;
    int teams[RN_MAX_CONV];
};

BwdPlan plan_backward(const Plan &p, int n, int cus) {
    BwdPlan b{};
    size_t dzmax = 0, pmax = 0;
    for (int l = 0; l < p.L; ++l) {
        dzmax = std::max(dzmax, (size_t)n * p.act_stride[l + 1]);
        b.teams[l] = bwd_dw_teams(p.C[l], p.C[l + 1], l == 0, n, p.ntl[l + 1], cus);
        pmax = std::max(pmax, bwd_dw_part_elems(p.C[l], p.C[l + 1], b.teams[l]));
    }
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + std::max<size_t>(bytes, 1));
        return o;
    };
    b.o_dz0 = take(dzmax * 4);
    b.o_dz1 = take(dzmax * 4);
    b.o_part = take(pmax * 4);
    b.total = off;
    return b;
}

// Every packed weight copy the kernels read, rewritten from a buffer in the
// gradient layout: assign = false applies fl(w - fl(lr g)) (an SGD step),
// assign = true stores the values themselves (new weights).  Then every slot
// is marked unprimed: the caches hold activations of the old weights.
rn_status write_packed(reuse_net *net, const float *src, float lr, bool assign, hipStream_t s, const char *what) {
    const Plan &p = net->p;
    const GradLayout gl = grad_layout(p);
    hipError_t e = hipSuccess;
    auto upd = [&](size_t off, size_t count, int kind, const float *g, int cin, int cout) {
        if (e != hipSuccess || count == 0) return;
        SgdArgs a{};
        a.dst = net->at<float>(off);
        a.count = count;
        a.kind = kind;
        a.g = g;
        a.lr = lr;
        a.assign = assign ? 1 : 0;
        a.cin = cin;
        a.cout = cout;
        a.C = p.C[p.L];
        a.H = p.Hl[p.L];
        a.W = p.Wl[p.L];
        a.TW = p.TWl[p.L];
        a.ntiles = p.ntl[p.L];
        a.n_out = p.N;
        a.K = p.K;
        e = timed(net, RN_PHASE_SGD, s, [&] { return launch_sgd(a, s); });
    };
    for (int l = 0; l < p.L; ++l) {
        upd(p.o_w[l], p.w_elems[l], l == 0 ? SGD_FIRST : SGD_MFMA, src + gl.w[l], p.C[l], p.C[l + 1]);
        upd(p.o_b[l], p.C[l + 1], SGD_PLAIN, src + gl.b[l], 0, 0);
        if (l > 0) upd(p.o_wt[l], p.wt_elems[l], SGD_DX, src + gl.w[l], p.C[l], p.C[l + 1]);
    }
    upd(p.o_wd, (size_t)p.N * p.K, SGD_DENSE, src + gl.dw, 0, 0);
    if (p.head_mode == RN_HEAD_TILES && !p.part_f32)
        upd(p.o_hw, tile_head_w_elems(p.ntl[p.L], p.C[p.L], p.N), SGD_TILE_HEAD, src + gl.dw, 0, 0);
    if (p.part_f32) upd(p.o_hw2, tile_part_f32_elems(p.ntl[p.L], p.C[p.L], p.N), SGD_TILE_PART, src + gl.dw, 0, 0);
    upd(p.o_bd, p.N, SGD_PLAIN, src + gl.db, 0, 0);
    if (e == hipSuccess) e = timed(net, RN_PHASE_SGD, s, [&] { return launch_unprime(net->at<int32_t>(p.o_primed), p.S, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string(what) + ": " + hipGetErrorString(e));
    net->last_stream = s;
    net->has_step = true;
    net->err.clear();
    return RN_OK;
}

}  // namespace

extern "C" {

size_t reuse_net_workspace_bytes(const rn_config *cfg) {
    Plan p;
    std::string err;
    if (plan_config(cfg, &p, &err) != RN_OK) return 0;
    return p.total;
}

rn_status reuse_net_create(const rn_config *cfg, const rn_weights *w, void *dev_workspace, size_t bytes,
                           void *hip_stream, reuse_net **out) {
    g_create_error.clear();
    if (!out) {
        g_create_error = "out is NULL";
        return RN_EINVAL;
    }
    *out = nullptr;
    Plan p;
    rn_status st = plan_config(cfg, &p, &g_create_error);
    if (st != RN_OK) return st;
    st = check_weights(p, w, &g_create_error);
    if (st != RN_OK) return st;
    if (!dev_workspace) {
        g_create_error = "workspace is NULL";
        return RN_EINVAL;
    }
    if (reinterpret_cast<uintptr_t>(dev_workspace) % kAlign) {
        g_create_error = "workspace must be 256-byte aligned";
        return RN_EINVAL;
    }
    if (bytes < p.total) {
        g_create_error = "workspace too small: need " + std::to_string(p.total) + " bytes";
        return RN_ENOSPACE;
    }
    reuse_net *net = new reuse_net();
    net->p = p;
    net->cfg = *cfg;
    net->cfg.conv = nullptr;
    net->ws = static_cast<char *>(dev_workspace);
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
        net->cus = std::max(1, prop.multiProcessorCount);
    net->dev = dev;
    {
        // Set-up of the static scratch on this device (reuse_net_variants_static);
        // a failure here is reported by that call, which looks it up again.
        std::string ignored;
        (void)static_scratch(dev, &ignored);
    }
    hipStream_t s = static_cast<hipStream_t>(hip_stream);

    // Host-side images of the constant parts.
    std::vector<float> lut(256);
    for (int k = 0; k < 256; ++k) lut[k] = (float)k / 255.0f;   // IEEE division: correctly rounded
    std::vector<int32_t> ids(p.S);
    for (int i = 0; i < p.S; ++i) ids[i] = i;
    hipError_t e = hipMemsetAsync(dev_workspace, 0, p.total, s);
    if (e == hipSuccess) e = hipMemcpyAsync(net->ws + p.o_lut, lut.data(), 256 * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(net->ws + p.o_ids, ids.data(), (size_t)p.S * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = upload_weights(net, w, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        g_create_error = std::string("upload: ") + hipGetErrorString(e);
        delete net;
        return RN_EHIP;
    }
    *out = net;
    return RN_OK;
}

rn_status reuse_net_step(reuse_net *net, int32_t n, const int32_t *ids, const void *frames, rn_dtype fdt,
                         const int32_t *boxes, const int32_t *box_off, float *logits, void *stream) {
    return run_step(net, n, ids, frames, fdt, boxes, box_off, logits, stream);
}

rn_status reuse_net_full(reuse_net *net, int32_t n, const int32_t *ids, const void *frames, rn_dtype fdt,
                         float *logits, void *stream) {
    return run_full(net, n, ids, frames, fdt, logits, stream);
}

size_t reuse_net_variant_scratch_bytes(const reuse_net *net, int32_t n, int32_t max_tiles) {
    if (!net || n < 1 || n > 65535 || variants_unsupported(net->p)) return 0;
    const VarPlan vp = plan_variants(net->p, n, max_tiles);
    return vp.cap > (size_t)INT32_MAX ? 0 : vp.total;
}

rn_status reuse_net_variants(reuse_net *net, int32_t base_stream, int32_t n, const void *frames, rn_dtype fdt,
                             int32_t frame_count, const int32_t *boxes, const int32_t *box_off, int32_t max_tiles,
                             void *scratch, size_t scratch_bytes, float *logits, void *stream) {
    return run_variants(net, base_stream, n, frames, fdt, frame_count, boxes, box_off, max_tiles, scratch,
                        scratch_bytes, logits, stream);
}

rn_status reuse_net_variants_static(reuse_net *net, int32_t base_stream, int32_t n, const void *frames,
                                    rn_dtype fdt, int32_t frame_count, const int32_t *boxes, const int32_t *box_off,
                                    int32_t max_tiles, float *logits, void *stream) {
    if (!net) return RN_EINVAL;
    if (const char *why = variants_unsupported(net->p)) return net->fail(RN_EUNSUPPORTED, why);
    if (n < 1 || n > 65535) return net->fail(RN_EINVAL, "n must be 1..65535");
    const VarPlan vp = plan_variants(net->p, n, max_tiles);
    if (vp.total > (size_t)RN_STATIC_SCRATCH_BYTES)
        return net->fail(RN_ENOSPACE, "variants need " + std::to_string(vp.total) + " bytes of scratch, above the " +
                                          std::to_string((size_t)RN_STATIC_SCRATCH_BYTES) +
                                          "-byte static scratch: use fewer variants or a smaller max_tiles");
    std::string err;
    void *sc = static_scratch(net->dev, &err);
    if (!sc) return net->fail(RN_EHIP, err);
    return run_variants(net, base_stream, n, frames, fdt, frame_count, boxes, box_off, max_tiles, sc,
                        (size_t)RN_STATIC_SCRATCH_BYTES, logits, stream);
}

rn_status reuse_net_set_weights(reuse_net *net, const rn_weights *w, void *hip_stream) {
    if (!net) return RN_EINVAL;
    rn_status st = check_weights(net->p, w, &net->err);
    if (st != RN_OK) return st;
    st = sync_last(net);                     // no step may still read the old weights
    if (st != RN_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    hipError_t e = upload_weights(net, w, s);
    // Every cache now holds activations of the old weights: all slots unprimed.
    if (e == hipSuccess) e = hipMemsetAsync(net->at<int32_t>(net->p.o_primed), 0, (size_t)net->p.S * 4, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("weight upload: ") + hipGetErrorString(e));
    net->err.clear();
    return RN_OK;
}

/* ---- training ---- */

size_t reuse_net_grad_elems(const reuse_net *net) {
    if (!net || net->p.train_why) return 0;
    return grad_layout(net->p).total;
}

size_t reuse_net_backward_scratch_bytes(const reuse_net *net, int32_t n) {
    if (!net || net->p.train_why || n < 1 || n > net->p.S) return 0;
    return plan_backward(net->p, n, net->cus).total;
}

rn_status reuse_net_reinforce_dlogits(int32_t n, int32_t n_out, const float *logits, const int32_t *actions,
                                      const float *returns, float *dlogits, void *stream) {
    if (n < 1 || n_out < 1 || n_out > kHeadMaxOut || !logits || !actions || !returns || !dlogits) return RN_EINVAL;
    return launch_reinforce(n, n_out, logits, actions, returns, dlogits, static_cast<hipStream_t>(stream)) ==
                   hipSuccess
               ? RN_OK
               : RN_EHIP;
}

rn_status reuse_net_backward(reuse_net *net, int32_t n, const int32_t *ids_in, const float *dlogits, float *grads,
                             int32_t accumulate, void *scratch, size_t scratch_bytes, void *stream) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (p.train_why) return net->fail(RN_EUNSUPPORTED, p.train_why);
    if (n < 1 || n > p.S) return net->fail(RN_EINVAL, "n must be 1..max_streams");
    if (!dlogits || !grads) return net->fail(RN_EINVAL, "dlogits and grads must not be NULL");
    if (!scratch) return net->fail(RN_EINVAL, "scratch is NULL");
    if (reinterpret_cast<uintptr_t>(scratch) % kAlign) return net->fail(RN_EINVAL, "scratch must be 256-byte aligned");
    const BwdPlan bp = plan_backward(p, n, net->cus);
    if (scratch_bytes < bp.total)
        return net->fail(RN_ENOSPACE, "scratch too small: need " + std::to_string(bp.total) + " bytes");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int32_t *ids = ids_in ? ids_in : net->at<int32_t>(p.o_ids);
    char *sc = static_cast<char *>(scratch);
    float *dz[2] = {reinterpret_cast<float *>(sc + bp.o_dz0), reinterpret_cast<float *>(sc + bp.o_dz1)};
    const GradLayout gl = grad_layout(p);
    hipError_t e = hipSuccess;
    if (p.fuse_first) {
        // Layer 1 is computed inside layer 2's kernel and has no cache of its
        // own: recompute it for these slots (same arithmetic, same bits).
        ConvArgs cv{};
        cv.ids = ids;
        cv.in = net->at<float>(p.o_xin);
        cv.out = net->at<void>(p.o_act[1]);
        cv.w = net->at<void>(p.o_w[0]);
        cv.bias = net->at<float>(p.o_b[0]);
        cv.ring_head = net->at<int32_t>(p.o_ring);
        cv.H = cv.Hin = p.H;
        cv.W = cv.Win = p.W;
        cv.TH = p.TH;
        cv.TW = cv.TWin = p.TW;
        cv.pad = 1;
        cv.cin = p.C[0];
        cv.cout = p.C[1];
        cv.stack = p.stack;
        cv.in_stride = p.act_stride[0];
        cv.out_stride = p.act_stride[1];
        cv.dense_n = n;
        cv.max_tiles = n * p.ntiles;
        e = timed(net, RN_PHASE_BWD_HEAD, s, [&] { return launch_conv_first(cv, p.dt, net->cus, s); });
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("layer-1 recompute: ") + hipGetErrorString(e));
    }
    const int L = p.L;
    HeadBwdArgs ha{};
    ha.n = n;
    ha.n_out = p.N;
    ha.C = p.C[L];
    ha.ntiles = p.ntl[L];
    ha.TW = p.TWl[L];
    ha.H = p.Hl[L];
    ha.W = p.Wl[L];
    ha.K = p.K;
    ha.ids = ids;
    ha.act = net->at<float>(p.o_act[L]);
    ha.act_stride = p.act_stride[L];
    ha.wd = net->at<float>(p.o_wd);
    ha.g = dlogits;
    ha.dz = dz[0];
    ha.gwd = grads + gl.dw;
    ha.gbd = grads + gl.db;
    ha.accumulate = accumulate != 0;
    e = timed(net, RN_PHASE_BWD_HEAD, s, [&] { return launch_bwd_head(ha, s); });
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("head backward: ") + hipGetErrorString(e));
    int cur = 0;
    for (int l = L - 1; l >= 0; --l) {                  // conv layer l + 1
        BwdArgs ba{};
        ba.n = n;
        ba.H = p.Hl[l + 1];
        ba.W = p.Wl[l + 1];
        ba.TH = p.THl[l + 1];
        ba.TW = p.TWl[l + 1];
        ba.ntiles = p.ntl[l + 1];
        ba.ca = p.C[l];
        ba.cz = p.C[l + 1];
        ba.ids = ids;
        ba.dz_in = dz[cur];
        ba.first = l == 0;
        ba.act_prev = l == 0 ? net->at<float>(p.o_xin) : net->at<float>(p.o_act[l]);
        ba.prev_stride = p.act_stride[l];
        ba.stack = p.stack;
        ba.cin0 = p.in_c;
        ba.ring_head = net->at<int32_t>(p.o_ring);
        ba.dz_out = dz[cur ^ 1];
        ba.wt = l > 0 ? net->at<float>(p.o_wt[l]) : nullptr;
        ba.part = reinterpret_cast<float *>(sc + bp.o_part);
        ba.teams = bp.teams[l];
        ba.gw = grads + gl.w[l];
        ba.gb = grads + gl.b[l];
        ba.accumulate = accumulate != 0;
        e = timed(net, RN_PHASE_BWD_DW, s, [&] { return launch_bwd_dw(ba, net->cus, s); });
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("weight gradient: ") + hipGetErrorString(e));
        if (l > 0) {
            e = timed(net, RN_PHASE_BWD_DX, s, [&] { return launch_bwd_dx(ba, net->cus, s); });
            if (e != hipSuccess) return net->fail(RN_EHIP, std::string("input gradient: ") + hipGetErrorString(e));
            cur ^= 1;
        }
    }
    net->last_stream = s;
    net->has_step = true;
    net->err.clear();
    return RN_OK;
}

rn_status reuse_net_sgd_step(reuse_net *net, const float *grads, float lr, void *stream) {
    if (!net) return RN_EINVAL;
    if (net->p.train_why) return net->fail(RN_EUNSUPPORTED, net->p.train_why);
    if (!grads) return net->fail(RN_EINVAL, "grads are NULL");
    return write_packed(net, grads, lr, false, static_cast<hipStream_t>(stream), "sgd step");
}

rn_status reuse_net_set_weights_device(reuse_net *net, const float *params, void *stream) {
    if (!net) return RN_EINVAL;
    if (net->p.train_why) return net->fail(RN_EUNSUPPORTED, net->p.train_why);
    if (!params) return net->fail(RN_EINVAL, "params are NULL");
    return write_packed(net, params, 0.f, true, static_cast<hipStream_t>(stream), "device weight update");
}

rn_status reuse_net_reset(reuse_net *net, int32_t sid) {
    if (!net) return RN_EINVAL;
    if (sid < -1 || sid >= net->p.S) return net->fail(RN_EINVAL, "stream_id out of range");
    rn_status st = sync_last(net);
    if (st != RN_OK) return st;
    int32_t *pr = net->at<int32_t>(net->p.o_primed);
    hipError_t e = sid < 0 ? hipMemset(pr, 0, (size_t)net->p.S * 4) : hipMemset(pr + sid, 0, 4);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("reset: ") + hipGetErrorString(e));
    return RN_OK;
}

static rn_status copy_out(reuse_net *net, void *dst, const void *src, size_t bytes) {
    rn_status st = sync_last(net);
    if (st != RN_OK) return st;
    hipError_t e = hipMemcpy(dst, src, bytes, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return net->fail(RN_EHIP, std::string("copy: ") + hipGetErrorString(e));
    return RN_OK;
}

// Where the masks, counts and lists of the last call live: the net's own
// buffers (index = slot), or the scratch of the last variants call (index =
// variant).
struct MaskView {
    const uint64_t *pm[RN_MAX_CONV + 1], *tm[RN_MAX_CONV + 1];
    const int32_t *nchg, *ntile, *cnt;
    const uint32_t *wl[RN_MAX_CONV + 1];
    int limit;                    // valid stream / variant indices
};

static MaskView mask_view(reuse_net *net) {
    const Plan &p = net->p;
    MaskView v{};
    if (net->last_was_var) {
        const VarPlan &vp = net->var_plan;
        char *sc = net->var_scratch;
        for (int l = 0; l <= p.L; ++l) {
            v.pm[l] = reinterpret_cast<const uint64_t *>(sc + vp.o_pm[l]);
            v.tm[l] = reinterpret_cast<const uint64_t *>(sc + vp.o_tm[l]);
            v.wl[l] = l ? reinterpret_cast<const uint32_t *>(sc + vp.o_wl[l]) : nullptr;
        }
        v.nchg = reinterpret_cast<const int32_t *>(sc + vp.o_nchg);
        v.ntile = reinterpret_cast<const int32_t *>(sc + vp.o_ntile);
        v.cnt = reinterpret_cast<const int32_t *>(sc + vp.o_cnt);
        v.limit = vp.n;
        return v;
    }
    for (int l = 0; l <= p.L; ++l) {
        v.pm[l] = net->at<uint64_t>(p.o_pm[l]);
        v.tm[l] = net->at<uint64_t>(p.o_tm[l]);
        v.wl[l] = l ? net->at<uint32_t>(p.o_wl[l]) : nullptr;
    }
    v.nchg = net->at<int32_t>(p.o_nchg);
    v.ntile = net->at<int32_t>(p.o_ntile);
    v.cnt = net->at<int32_t>(p.o_cnt);
    v.limit = p.S;
    return v;
}

rn_status reuse_net_get_pixel_mask(reuse_net *net, int32_t layer, int32_t sid, uint64_t *out, size_t words) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    const MaskView v = mask_view(net);
    if (layer < 0 || layer > p.L || sid < 0 || sid >= v.limit || !out)
        return net->fail(RN_EINVAL, "bad layer, stream or buffer");
    const size_t need = (size_t)p.Hl[layer] * p.WWl[layer];
    if (words < need) return net->fail(RN_ENOSPACE, "buffer needs " + std::to_string(need) + " words");
    return copy_out(net, out, v.pm[layer] + (size_t)sid * need, need * 8);
}

rn_status reuse_net_get_tile_mask(reuse_net *net, int32_t layer, int32_t sid, uint64_t *out, size_t words) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    const MaskView v = mask_view(net);
    if (layer < 0 || layer > p.L || sid < 0 || sid >= v.limit || !out)
        return net->fail(RN_EINVAL, "bad layer, stream or buffer");
    const int tmw = p.TMWl[layer];
    if (words < (size_t)tmw) return net->fail(RN_ENOSPACE, "buffer needs " + std::to_string(tmw) + " words");
    return copy_out(net, out, v.tm[layer] + (size_t)sid * tmw, (size_t)tmw * 8);
}

rn_status reuse_net_get_worklist(reuse_net *net, int32_t layer, uint32_t *out, size_t cap, int32_t *count) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (layer < 1 || layer > p.L || !count) return net->fail(RN_EINVAL, "bad layer or count pointer");
    if (net->last_was_full) return net->fail(RN_ESTATE, "the last call was reuse_net_full: no work list");
    const MaskView v = mask_view(net);
    int32_t c = 0;
    rn_status st = copy_out(net, &c, v.cnt + layer, 4);
    if (st != RN_OK) return st;
    *count = c;
    if ((size_t)c > cap) return net->fail(RN_ENOSPACE, "work list has " + std::to_string(c) + " entries");
    if (c == 0) return RN_OK;
    if (!out) return net->fail(RN_EINVAL, "out is NULL");
    return copy_out(net, out, v.wl[layer], (size_t)c * 4);
}

rn_status reuse_net_read_activation(reuse_net *net, int32_t sid, int32_t layer, float *host_out) {
    if (!net) return RN_EINVAL;
    const Plan &p = net->p;
    if (layer < 0 || layer > p.L || sid < 0 || sid >= p.S || !host_out) return net->fail(RN_EINVAL, "bad layer, stream or buffer");
    const size_t HW = (size_t)p.H * p.W;
    if (layer == 0) {
        int head = 0;
        if (p.stack != 1) {
            rn_status st = copy_out(net, &head, net->at<int32_t>(p.o_ring) + sid, 4);
            if (st != RN_OK) return st;
        }
        const float *src = net->at<float>(p.o_xin) + ((size_t)sid * p.stack + head) * p.in_c * HW;
        return copy_out(net, host_out, src, (size_t)p.in_c * HW * 4);
    }
    if (layer == 1 && p.fuse_first) {
        // Layer 1 has no cache of its own in this mode: recompute it for this
        // slot from the input cache with the first-layer kernel.
        rn_status st = sync_last(net);
        if (st != RN_OK) return st;
        ConvArgs cv{};
        cv.ids = net->at<int32_t>(p.o_ids) + sid;   // identity table: points at the value sid
        cv.in = net->at<float>(p.o_xin);
        cv.out = net->at<void>(p.o_act[1]);
        cv.w = net->at<void>(p.o_w[0]);
        cv.bias = net->at<float>(p.o_b[0]);
        cv.ring_head = net->at<int32_t>(p.o_ring);
        cv.H = cv.Hin = p.H;
        cv.W = cv.Win = p.W;
        cv.TH = p.TH;
        cv.TW = cv.TWin = p.TW;
        cv.pad = 1;
        cv.cin = p.C[0];
        cv.cout = p.C[1];
        cv.stack = p.stack;
        cv.in_stride = p.act_stride[0];
        cv.out_stride = p.act_stride[1];
        cv.dense_n = 1;
        cv.max_tiles = p.ntiles;
        hipError_t e = launch_conv_first(cv, p.dt, net->cus, net->last_stream);
        if (e == hipSuccess) e = hipStreamSynchronize(net->last_stream);
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("layer-1 recompute: ") + hipGetErrorString(e));
    }
    const int C = p.C[layer];
    std::vector<float> buf(p.act_stride[layer]);
    rn_status st;
    if (p.dt == RN_BF16) {
        std::vector<uint16_t> hb(p.act_stride[layer]);
        st = copy_out(net, hb.data(), net->at<uint16_t>(p.o_act[layer]) + (size_t)sid * p.act_stride[layer],
                      p.act_stride[layer] * 2);
        for (size_t j = 0; j < hb.size(); ++j) {
            const uint32_t u = (uint32_t)hb[j] << 16;
            memcpy(&buf[j], &u, 4);
        }
    } else {
        st = copy_out(net, buf.data(), net->at<float>(p.o_act[layer]) + (size_t)sid * p.act_stride[layer],
                      p.act_stride[layer] * 4);
    }
    if (st != RN_OK) return st;
    const int Hl = p.Hl[layer], Wl = p.Wl[layer], TWl = p.TWl[layer];
    const size_t HWl = (size_t)Hl * Wl;
    for (int y = 0; y < Hl; ++y)
        for (int x = 0; x < Wl; ++x) {
            const size_t src = ((size_t)((y / kTile) * TWl + x / kTile) * kTilePx + (y % kTile) * kTile + x % kTile) * C;
            for (int c = 0; c < C; ++c) host_out[(size_t)c * HWl + (size_t)y * Wl + x] = buf[src + c];
        }
    return RN_OK;
}

rn_status reuse_net_get_stats(reuse_net *net, rn_stats *out) {
    if (!net) return RN_EINVAL;
    if (!out) return net->fail(RN_EINVAL, "out is NULL");
    memset(out, 0, sizeof *out);
    if (!net->has_step) return RN_OK;
    const Plan &p = net->p;
    const int n = net->last_n;
    const MaskView v = mask_view(net);
    std::vector<int32_t> nchg(n), ntile((size_t)n * (p.L + 1));
    rn_status st = copy_out(net, nchg.data(), v.nchg, (size_t)n * 4);
    if (st == RN_OK) st = copy_out(net, ntile.data(), v.ntile, ntile.size() * 4);
    if (st != RN_OK) return st;
    out->streams = n;
    for (int i = 0; i < n; ++i) {
        out->changed_px += nchg[i];
        for (int l = 0; l <= p.L; ++l) out->dirty_tiles[l] += ntile[(size_t)i * (p.L + 1) + l];
    }
    const int64_t head_mac = (int64_t)n * p.N * p.C[p.L] * p.Hl[p.L] * p.Wl[p.L];
    int64_t useful = head_mac, issued = (int64_t)n * p.N * (int64_t)p.K, dense = head_mac;
    for (int l = 1; l <= p.L; ++l) {
        const int64_t per_px = (int64_t)p.ks[l - 1] * p.ks[l - 1] * p.C[l - 1] * p.C[l];
        const int Hl = p.Hl[l], Wl = p.Wl[l];
        dense += (int64_t)n * Hl * Wl * per_px;
        issued += out->dirty_tiles[l] * kTilePx * per_px;
        if (net->last_was_full) {
            useful += (int64_t)n * Hl * Wl * per_px;
            continue;
        }
        int32_t c = 0;
        std::vector<uint32_t> wl((size_t)n * p.ntl[l]);
        st = reuse_net_get_worklist(net, l, wl.data(), wl.size(), &c);
        if (st != RN_OK) return st;
        for (int j = 0; j < c; ++j) {
            const int ty = (wl[j] >> 8) & 255, tx = wl[j] & 255;
            const int hy = std::min(kTile, Hl - ty * kTile), wx = std::min(kTile, Wl - tx * kTile);
            useful += (int64_t)hy * wx * per_px;
        }
    }
    out->useful_mac = useful;
    out->issued_mac = issued;
    out->dense_mac = dense;
    return RN_OK;
}

rn_status reuse_net_set_profiling(reuse_net *net, int32_t enable) {
    if (!net) return RN_EINVAL;
    rn_status st = sync_last(net);
    if (st != RN_OK) return st;
    net->recs.clear();
    net->pool_used = 0;
    net->prof = enable != 0;
    return RN_OK;
}

rn_status reuse_net_get_profile(reuse_net *net, rn_profile *out) {
    if (!net) return RN_EINVAL;
    if (!out) return net->fail(RN_EINVAL, "out is NULL");
    memset(out, 0, sizeof *out);
    rn_status st = sync_last(net);
    if (st != RN_OK) return st;
    for (const ProfRec &r : net->recs) {
        float ms = 0.f;
        hipError_t e = hipEventElapsedTime(&ms, r.e0, r.e1);
        if (e != hipSuccess) return net->fail(RN_EHIP, std::string("event time: ") + hipGetErrorString(e));
        out->ms[r.phase] += ms;
        out->launches[r.phase] += 1;
        out->layer_ms[r.layer] += ms;
        out->layer_launches[r.layer] += 1;
    }
    return RN_OK;
}

const char *reuse_net_last_error(const reuse_net *net) {
    return net ? net->err.c_str() : g_create_error.c_str();
}

void reuse_net_destroy(reuse_net *net) {
    if (!net) return;
    for (hipEvent_t e : net->pool) (void)hipEventDestroy(e);
    delete net;
}

}  // extern "C"
