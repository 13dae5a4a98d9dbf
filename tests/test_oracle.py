"""Pins of the CPU oracle against things other than itself.

Each group ties one oracle function to a library routine, a brute force, a
closed form or an invariant, chosen so that a plausible slip (a dropped bias,
a flipped kernel, an off-by-one window, a wrong tile edge, a wrong list order)
fails at least one test.
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from synth import frames as synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ inputs

def test_level_to_f32_is_correctly_rounded(orc):
    # IEEE single division is correctly rounded: numpy's float32 k / 255 is the
    # reference for all 256 levels.
    k = np.arange(256, dtype=np.uint8)
    ref = k.astype(np.float32) / np.float32(255)
    got = orc.level_to_f32(k)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    assert got[0] == 0.0 and got[255] == 1.0


def test_bf16_rne_matches_torch(orc):
    rng = np.random.default_rng(5)
    x = np.concatenate([
        rng.normal(0, 1, 5000).astype(np.float32),
        rng.normal(0, 1e-30, 500).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.0e38], np.float32),
        # exact ties: low 16 bits 0x8000, with kept lsb 0 and 1
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x3F80FFFF, 0x3F807FFF],
                 np.uint32).view(np.float32),
    ])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = orc.bf16_rne(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    assert np.isnan(orc.bf16_rne(np.array([np.nan], np.float32))[0])


def test_out_size_closed_form(orc):
    for n in range(1, 30):
        for k in (1, 3, 5, 7):
            for s in (1, 2, 3, 4):
                for p in (0, (k - 1) // 2, k):
                    ref = (n + 2 * p - k) // s + 1 if n + 2 * p >= k else 0
                    assert orc.out_size(n, k, s, p) == ref
    assert orc.out_size(105, 3, 1, 1) == 105
    assert orc.out_size(84, 8, 4, 0) == 20


# ------------------------------------------------------------------ diff

def _diff_brute(prev, cur):
    c, h, w = prev.shape
    out = np.zeros((h, w), np.uint8)
    pb, cb = prev.view(np.uint32), cur.view(np.uint32)
    for y in range(h):
        for x in range(w):
            for ch in range(c):
                if pb[ch, y, x] != cb[ch, y, x]:
                    out[y, x] = 1
    return out


def test_diff_brute_force(orc):
    rng = np.random.default_rng(1)
    for c in (1, 2, 4):
        prev = rng.random((c, 7, 9), dtype=np.float32)
        cur = prev.copy()
        m = rng.random((c, 7, 9)) < 0.2
        cur[m] = rng.random(m.sum(), dtype=np.float32)
        assert np.array_equal(orc.diff(prev, cur), _diff_brute(prev, cur))


def test_diff_special_cases(orc):
    u8 = np.random.default_rng(2).integers(0, 256, (1, 6, 5), dtype=np.uint8)
    a = synth.to_f32(u8)
    assert orc.diff(a, a.copy()).sum() == 0                      # unchanged frame
    b = synth.to_f32(((u8.astype(np.int32) + 1) % 256).astype(np.uint8))
    assert orc.diff(a, b).sum() == 30                            # +1 mod 256 everywhere
    z = np.zeros((1, 2, 2), np.float32)
    nz = z.copy()
    nz[0, 0, 1] = -0.0                                           # -0 vs +0 differ in bits
    nan = np.full((1, 2, 2), np.nan, np.float32)
    assert orc.diff(z, nz).tolist() == [[0, 1], [0, 0]]
    assert orc.diff(nan, nan.copy()).sum() == 0                  # same NaN bits: unchanged


def test_box_mask_union_and_clip(orc):
    boxes = [(1, 1, 3, 4), (2, 3, 5, 5), (-2, -2, 1, 1), (6, 6, 9, 9), (4, 4, 4, 6)]
    got = orc.box_mask(6, 7, boxes)
    ref = np.zeros((6, 7), np.uint8)
    for y0, x0, y1, x1 in boxes:
        ref[max(y0, 0):max(y1, 0), max(x0, 0):max(x1, 0)] = 1
    assert np.array_equal(got, ref)
    assert orc.box_mask(5, 5, np.zeros((0, 4), np.int32)).sum() == 0


# ------------------------------------------------------------------ growth

def _rf_brute(d0, layers, l):
    """Layer-l dirty mask from the composed receptive field of each output pixel.

    Independent of the layer-by-layer dilation: the input interval feeding a
    layer-l pixel is built by composing each layer's window, then tested for any
    changed input pixel."""
    h, w = d0.shape
    hs, ws = [h], [w]
    for (k, s, p) in layers:
        hs.append((hs[-1] + 2 * p - k) // s + 1)
        ws.append((ws[-1] + 2 * p - k) // s + 1)
    out = np.zeros((hs[l], ws[l]), np.uint8)
    for yo in range(hs[l]):
        for xo in range(ws[l]):
            y0 = y1 = yo
            x0 = x1 = xo
            for (k, s, p) in reversed(layers[:l]):
                y0, y1 = s * y0 - p, s * y1 - p + k - 1
                x0, x1 = s * x0 - p, s * x1 - p + k - 1
            y0, x0 = max(y0, 0), max(x0, 0)
            y1, x1 = min(y1, h - 1), min(x1, w - 1)
            if y0 <= y1 and x0 <= x1 and d0[y0:y1 + 1, x0:x1 + 1].any():
                out[yo, xo] = 1
    return out


@pytest.mark.parametrize("layers", [
    [(3, 1, 1), (3, 1, 1), (3, 1, 1)],
    [(5, 1, 2), (3, 1, 1)],
    [(3, 2, 1), (3, 1, 1)],
    [(5, 2, 2), (3, 2, 1)],
    [(1, 1, 0), (3, 1, 0)],
    [(8, 4, 0), (4, 2, 0)],
])
def test_dilation_matches_receptive_field_brute_force(orc, layers):
    rng = np.random.default_rng(len(layers) * 7 + layers[0][0])
    lo = 6 if layers[0][0] < 8 else 20
    for trial in range(6):
        h, w = rng.integers(lo, lo + 7, size=2)
        d0 = (rng.random((h, w)) < (0.02 + 0.05 * trial)).astype(np.uint8)
        cur = d0
        for l, (k, s, p) in enumerate(layers, start=1):
            cur = orc.dilate(cur, k, s, p)
            assert np.array_equal(cur, _rf_brute(d0, layers, l)), (layers, l, trial)


def test_dilation_closed_forms(orc):
    # Fig. 1 caption: k = 3 grows a change by one pixel per side per layer.
    for (y, x) in [(5, 6), (0, 0), (10, 0), (10, 11)]:
        d = np.zeros((11, 12), np.uint8)
        d[y, x] = 1
        for l in range(1, 4):
            d = orc.dilate(d, 3, 1, 1)
            ref = np.zeros_like(d)
            ref[max(0, y - l):y + l + 1, max(0, x - l):x + l + 1] = 1
            assert np.array_equal(d, ref)
    # Monotone in the change set.
    rng = np.random.default_rng(3)
    a = (rng.random((9, 9)) < 0.1).astype(np.uint8)
    b = a | (rng.random((9, 9)) < 0.1).astype(np.uint8)
    assert np.all(orc.dilate(a, 3, 1, 1) <= orc.dilate(b, 3, 1, 1))
    assert orc.dilate(np.zeros((5, 5), np.uint8), 3, 1, 1).sum() == 0


def test_golden_fig1_growth(orc):
    path = os.path.join(GOLDEN, "fig1_growth.txt")
    rows = [l for l in open(path) if l.strip() and not l.startswith("#")]
    assert rows
    for row in rows:
        dims, boxes, l1, l2 = [part.split() for part in row.split("|")]
        h, w = map(int, dims)
        d = orc.box_mask(h, w, np.array(list(map(int, boxes)), np.int32).reshape(-1, 4))
        for want in (l1, l2):
            d = orc.dilate(d, 3, 1, 1)
            ref = orc.box_mask(h, w, np.array(list(map(int, want)), np.int32).reshape(-1, 4))
            assert np.array_equal(d, ref), row


# ------------------------------------------------------------------ tiles

def _tiles_numpy(d, th, tw):
    h, w = d.shape
    H, W = -(-h // th) * th, -(-w // tw) * tw
    pad = np.zeros((H, W), np.uint8)
    pad[:h, :w] = d
    return pad.reshape(H // th, th, W // tw, tw).max(axis=(1, 3))


def test_tile_mask_matches_block_reduction(orc):
    rng = np.random.default_rng(4)
    for (h, w) in [(105, 80), (53, 40), (9, 7), (1, 1), (4, 4), (5, 9)]:
        for (th, tw) in [(4, 4), (8, 8), (1, 1), (3, 5), (16, 16)]:
            d = (rng.random((h, w)) < 0.03).astype(np.uint8)
            assert np.array_equal(orc.tile_mask(d, th, tw), _tiles_numpy(d, th, tw))
    d = np.zeros((105, 80), np.uint8)
    d[104, 79] = 1                                   # last pixel -> ragged last tile
    m = orc.tile_mask(d, 4, 4)
    assert m.shape == (27, 20) and m.sum() == 1 and m[26, 19] == 1


def test_worklist_order_and_encoding(orc):
    rng = np.random.default_rng(6)
    masks = (rng.random((5, 27, 20)) < 0.1).astype(np.uint8)
    wl = orc.worklist(masks)
    # Position-major: argwhere over the [ty][tx][s] transpose lists (ty, tx, s) ascending.
    ref = [(s << 16) | (ty << 8) | tx for (ty, tx, s) in np.argwhere(masks.transpose(1, 2, 0))]
    assert wl.tolist() == ref
    assert sorted(wl.tolist(), key=lambda e: ((e >> 8) & 255, e & 255, e >> 16)) == wl.tolist()
    assert orc.worklist(np.zeros((3, 4, 4), np.uint8)).size == 0
    full = orc.worklist(np.ones((2, 3, 2), np.uint8))
    assert full.tolist() == [(s << 16) | (y << 8) | x for y in range(3) for x in range(2)
                             for s in range(2)]


# ------------------------------------------------------------------ conv / dense

def _torch_conv(x, w, b, s, p):
    y = F.conv2d(torch.from_numpy(x[None].astype(np.float64)), torch.from_numpy(w.astype(np.float64)),
                 torch.from_numpy(b.astype(np.float64)), stride=s, padding=p)
    return torch.relu(y)[0].numpy()


@pytest.mark.parametrize("shape", [
    (1, 5, 7, 4, 3, 1, 1), (3, 6, 6, 5, 3, 1, 1), (4, 9, 8, 7, 5, 1, 2),
    (2, 10, 9, 3, 3, 2, 1), (2, 12, 12, 4, 8, 4, 0), (5, 4, 4, 2, 1, 1, 0),
])
def test_conv_matches_torch_float64(orc, shape):
    cin, h, w, cout, k, s, p = shape
    rng = np.random.default_rng(sum(shape))
    x = rng.random((cin, h, w), dtype=np.float32)
    wt = rng.normal(0, 0.5, (cout, cin, k, k)).astype(np.float32)   # not symmetric: catches flips
    b = rng.normal(0, 0.5, cout).astype(np.float32)                 # non-zero: catches a dropped bias
    got = orc.conv2d_relu(x, wt, b, stride=s, pad=p)
    ref = _torch_conv(x, wt, b, s, p).astype(np.float32)            # fp64 sum, one rounding
    assert got.shape == ref.shape
    np.testing.assert_allclose(got, ref, rtol=2e-7, atol=1e-12)
    assert (got >= 0).all() and not np.signbit(got).any()            # ReLU gives +0, never -0


def test_conv_closed_forms(orc):
    # Delta kernel: output = ReLU(input + b).
    x = np.random.default_rng(8).normal(0, 1, (1, 6, 5)).astype(np.float32)
    wt = np.zeros((1, 1, 3, 3), np.float32)
    wt[0, 0, 1, 1] = 1
    y = orc.conv2d_relu(x, wt, np.zeros(1, np.float32))
    assert np.array_equal(y, np.maximum(x, 0))
    # Off-centre delta at (0, 2): out[y, x] = in[y-1, x+1] (cross-correlation).
    wt[:] = 0
    wt[0, 0, 0, 2] = 1
    y = orc.conv2d_relu(np.abs(x), wt, np.zeros(1, np.float32))
    ref = np.zeros_like(x)
    ref[0, 1:, :-1] = np.abs(x)[0, :-1, 1:]
    assert np.array_equal(y, ref)
    # All-ones kernel on a constant c: interior 9c + b, edges 6c + b, corners 4c + b.
    y = orc.conv2d_relu(np.full((1, 4, 5), 0.5, np.float32), np.ones((1, 1, 3, 3), np.float32),
                        np.array([0.25], np.float32))
    assert y[0, 1, 1] == 4.75 and y[0, 0, 2] == 3.25 and y[0, 0, 0] == 2.25


def test_dense_matches_numpy_float64(orc):
    rng = np.random.default_rng(9)
    a = rng.random(3000, dtype=np.float32)
    wd = rng.normal(0, 0.05, (6, 3000)).astype(np.float32)
    bd = rng.normal(0, 1, 6).astype(np.float32)
    ref = (wd.astype(np.float64) @ a.astype(np.float64) + bd).astype(np.float32)
    np.testing.assert_allclose(orc.dense(a, wd, bd), ref, rtol=1e-7, atol=1e-9)


def _small_net(orc, in_c=1, h=13, w=11, convs=(5, 6), n_out=3, tile=4, bf16=False):
    specs = []
    c = in_c
    for co in convs:
        specs.append((c, co, 3, 1, 1))
        c = co
    return orc.Net(in_c, h, w, specs, n_out, tile, tile, bf16)


def _rand_weights(net, seed, bias=0.3):
    rng = np.random.default_rng(seed)
    cw = [rng.normal(0, 0.3, (co, ci, k, k)).astype(np.float32) for (ci, co, k, s, p) in net.convs]
    cb = [rng.normal(0, bias, co).astype(np.float32) for (ci, co, k, s, p) in net.convs]
    c, h, w = net.layer_shape(len(net.convs))
    dw = rng.normal(0, 0.1, (net.n_out, c * h * w)).astype(np.float32)
    db = rng.normal(0, bias, net.n_out).astype(np.float32)
    return cw, cb, dw, db


def test_forward_matches_torch_model(orc):
    net = _small_net(orc, in_c=2, h=10, w=9, convs=(4, 5, 3), n_out=4)
    cw, cb, dw, db = _rand_weights(net, 11)
    x = np.random.default_rng(12).random((3, 2, 10, 9), dtype=np.float32)
    logits, acts = orc.forward(net, cw, cb, dw, db, x, want_acts=True)
    for i in range(3):
        a = x[i]
        for l, (ci, co, k, s, p) in enumerate(net.convs):
            a = _torch_conv(a, cw[l], cb[l], s, p).astype(np.float32)
            np.testing.assert_allclose(acts[l][i], a, rtol=3e-7, atol=1e-12)
        ref = dw.astype(np.float64) @ a.reshape(-1).astype(np.float64) + db
        np.testing.assert_allclose(logits[i], ref.astype(np.float32), rtol=1e-6, atol=1e-7)


def test_forward_bf16_matches_torch_emulation(orc):
    net = _small_net(orc, bf16=True)
    cw, cb, dw, db = _rand_weights(net, 13)
    x = np.random.default_rng(14).random((2, 1, 13, 11), dtype=np.float32)
    logits, acts = orc.forward(net, cw, cb, dw, db, x, want_acts=True)
    bf = lambda t: torch.from_numpy(np.ascontiguousarray(t)).to(torch.bfloat16).to(torch.float32).numpy()
    for i in range(2):
        a = bf(x[i])
        for l, (ci, co, k, s, p) in enumerate(net.convs):
            a = bf(_torch_conv(a, bf(cw[l]), cb[l], s, p).astype(np.float32))
            assert np.abs(acts[l][i] - a).max() <= 1e-2 * np.abs(a).max()
            # Every stored activation is a bf16 value.
            assert np.array_equal(acts[l][i].view(np.uint32) & 0xFFFF, np.zeros(a.shape, np.uint32))
        ref = bf(dw).astype(np.float64) @ a.reshape(-1).astype(np.float64) + db
        np.testing.assert_allclose(logits[i], ref, rtol=1e-2, atol=1e-3)


# ------------------------------------------------------------------ masks of a step

def test_masks_compose_dilate_and_tiles(orc):
    net = _small_net(orc, h=21, w=18, convs=(3, 4, 2))
    rng = np.random.default_rng(15)
    d0 = (rng.random((4, 21, 18)) < 0.02).astype(np.uint8)
    d, m = orc.masks(net, d0)
    for i in range(4):
        for l in range(len(net.convs) + 1):
            assert np.array_equal(d[l][i], _rf_brute(d0[i], [(3, 1, 1)] * 3, l))
            assert np.array_equal(m[l][i], _tiles_numpy(d[l][i], 4, 4))


# ------------------------------------------------------------------ invariants

def _sprite_inputs(orc, wl, frames, stream=0):
    u8 = synth.sprite_sequence(wl.cid, stream, frames, wl.h, wl.w, wl.n_sprites, wl.smin,
                               wl.smax, wl.vmin, wl.vmax)
    return synth.to_f32(u8)


@pytest.mark.parametrize("bf16", [False, True])
def test_invariant_reuse_equals_full_bitwise(orc, bf16):
    # (i) Reuse on dirty tiles only gives the full recompute's bits, frame after frame.
    net = _small_net(orc, h=23, w=19, convs=(4, 6), n_out=3, bf16=bf16)
    cw, cb, dw, db = _rand_weights(net, 16)
    wl = synth.Workload(cid=99, streams=1, frames=10, h=23, w=19, convs=(4, 6), n_out=3,
                        n_sprites=2, smin=2, smax=4, vmin=1, vmax=2)
    xs = _sprite_inputs(orc, wl, 10)
    rs = orc.ReuseStream(net, cw, cb, dw, db)
    for t in range(10):
        got = rs.step(xs[t][None])
        ref_logits, acts = orc.forward(net, cw, cb, dw, db, xs[t][None, None], want_acts=True)
        for l in range(len(net.convs)):
            assert np.array_equal(rs.cache[l + 1].view(np.uint32), acts[l][0].view(np.uint32)), (t, l)
        assert np.array_equal(got.view(np.uint32), ref_logits[0].view(np.uint32)), t


def test_invariant_reuse_detects_too_small_growth(orc):
    # A recompute on the undilated change set alone must NOT match: this checks
    # that invariant (i) has teeth against a dilation that is too small.
    net = _small_net(orc, h=16, w=16, convs=(3, 3), n_out=2, tile=1)
    cw, cb, dw, db = _rand_weights(net, 17)
    a = np.random.default_rng(18).random((1, 16, 16), dtype=np.float32)
    b = a.copy()
    b[0, 8, 8] += 0.5
    acts_a = orc.forward(net, cw, cb, dw, db, a[None], want_acts=True)[1]
    acts_b = orc.forward(net, cw, cb, dw, db, b[None], want_acts=True)[1]
    stale = acts_a[0][0].copy()
    d0 = orc.diff(a, b)
    orc.conv2d_relu_tiles(b, cw[0], cb[0], d0, 1, 1, stale)   # undilated: misses neighbours
    assert not np.array_equal(stale, acts_b[0][0])
    good = acts_a[0][0].copy()
    orc.conv2d_relu_tiles(b, cw[0], cb[0], orc.dilate(d0, 3, 1, 1), 1, 1, good)
    assert np.array_equal(good, acts_b[0][0])


def test_invariant_unchanged_frame(orc):
    # (ii) An unchanged frame gives zero dirty tiles and the same logits.
    net = _small_net(orc)
    cw, cb, dw, db = _rand_weights(net, 19)
    x = np.random.default_rng(20).random((1, 13, 11), dtype=np.float32)
    rs = orc.ReuseStream(net, cw, cb, dw, db)
    l0 = rs.step(x)
    l1 = rs.step(x.copy())
    assert np.array_equal(l0.view(np.uint32), l1.view(np.uint32))
    d, m = orc.masks(net, orc.diff(x, x)[None])
    assert all(mm.sum() == 0 for mm in m)
    assert all(orc.worklist(mm).size == 0 for mm in m[1:])


def test_invariant_all_changed_frame(orc):
    # (iii) An all-changed frame marks every tile and equals the dense path.
    net = _small_net(orc, h=14, w=10)
    cw, cb, dw, db = _rand_weights(net, 21)
    u8 = np.random.default_rng(22).integers(0, 256, (1, 14, 10), dtype=np.uint8)
    a = synth.to_f32(u8)
    b = synth.to_f32(((u8.astype(np.int32) + 7) % 256).astype(np.uint8))
    d0 = orc.diff(a, b)
    assert d0.all()
    _, m = orc.masks(net, d0[None])
    for l in range(len(net.convs) + 1):
        assert m[l].all()
        if l:
            th, tw = net.tile_grid(l)
            assert orc.worklist(m[l]).size == th * tw
    rs = orc.ReuseStream(net, cw, cb, dw, db)
    rs.step(a)
    got = rs.step(b)
    ref = orc.forward(net, cw, cb, dw, db, b[None])[0][0]
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_boxes_step_equals_full_on_edited_input(orc):
    # Known-change mode: with boxes, the effective input is the previous input
    # with the box pixels taken from the new frame.
    net = _small_net(orc, h=16, w=12)
    cw, cb, dw, db = _rand_weights(net, 23)
    base = np.random.default_rng(24).random((1, 16, 12), dtype=np.float32)
    rs = orc.ReuseStream(net, cw, cb, dw, db)
    rs.step(base)
    for (y, x) in [(0, 0), (3, 5), (10, 8)]:
        frame = base.copy()
        frame[0, y:y + 4, x:x + 4] = 0
        boxes = [(y, x, y + 4, x + 4)]
        got = rs.step(frame, d0=orc.box_mask(16, 12, boxes))
        ref = orc.forward(net, cw, cb, dw, db, frame[None])[0][0]
        np.testing.assert_array_equal(got, ref)
        rs.step(base, d0=orc.box_mask(16, 12, boxes))    # restore


def test_reset_makes_next_step_all_dirty(orc):
    net = _small_net(orc)
    cw, cb, dw, db = _rand_weights(net, 25)
    x = np.random.default_rng(26).random((1, 13, 11), dtype=np.float32)
    rs = orc.ReuseStream(net, cw, cb, dw, db)
    rs.step(x)
    rs.cache[1][:] = 123.0                                # corrupt a cache
    rs.reset()
    got = rs.step(x)                                      # unchanged input, but reset
    ref = orc.forward(net, cw, cb, dw, db, x[None])[0][0]
    assert np.array_equal(got, ref)


def test_variant_input_pins(orc):
    # Closed forms: no boxes -> the base; a box over the whole frame (or past
    # it, clipped) -> the frame; and brute force over every pixel with the
    # half-open box rule written out, for overlapping, clipped and empty boxes.
    rng = np.random.default_rng(31)
    base = rng.random((2, 7, 9), dtype=np.float32)
    frame = -rng.random((2, 7, 9), dtype=np.float32)
    assert np.array_equal(orc.variant_input(base, frame, np.zeros((0, 4), np.int32)), base)
    assert np.array_equal(orc.variant_input(base, frame, [(-3, -1, 20, 30)]), frame)
    boxes = [(1, 2, 4, 5), (3, 4, 6, 9), (-2, 7, 2, 12), (5, 5, 5, 8), (6, 0, 9, 1)]
    got = orc.variant_input(base, frame, boxes)
    for y in range(7):
        for x in range(9):
            inside = any(y0 <= y < y1 and x0 <= x < x1 for (y0, x0, y1, x1) in boxes)
            want = frame[:, y, x] if inside else base[:, y, x]
            assert np.array_equal(got[:, y, x], want), (y, x)


def test_variant_equals_reuse_step_from_base(orc):
    # A variant is what one known-change step from the base state computes:
    # reuse on the boxes' dirty tiles from the base caches gives the full
    # recompute of the variant input bit for bit, and the base is untouched
    # when each variant starts from a fresh copy of the base state.
    net = _small_net(orc, h=15, w=13)
    cw, cb, dw, db = _rand_weights(net, 32)
    rng = np.random.default_rng(33)
    base = rng.random((1, 15, 13), dtype=np.float32)
    for boxes in ([(2, 3, 6, 9)], [(0, 0, 1, 1), (10, 9, 20, 20)], [(4, 4, 4, 9)]):
        frame = np.zeros_like(base)
        x = orc.variant_input(base, frame, boxes)
        rs = orc.ReuseStream(net, cw, cb, dw, db)
        rs.step(base)
        got = rs.step(x, d0=orc.box_mask(15, 13, boxes))
        ref = orc.forward(net, cw, cb, dw, db, x[None])[0][0]
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), boxes


# ------------------------------------------------------------------ training (Sec. 2: REINFORCE)

def _torch_grads(net, cw, cb, dw, db, x, g):
    """Gradients of sum(g * logits) by torch float64 autograd through the same
    function the oracle evaluates: float32 activations (the rounding passes
    the gradient through unchanged), double arithmetic otherwise."""
    T = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
    tw, tb, tdw, tdb = [T(w) for w in cw], [T(b) for b in cb], T(dw), T(db)
    a = torch.tensor(x, dtype=torch.float64)
    for (ci, co, k, s, p), w_, b_ in zip(net.convs, tw, tb):
        a = torch.relu(F.conv2d(a, w_, b_, stride=s, padding=p)).float().double()
    logits = a.flatten(1) @ tdw.T + tdb
    (logits * torch.tensor(g, dtype=torch.float64)).sum().backward()
    return [w.grad.numpy() for w in tw], [b.grad.numpy() for b in tb], tdw.grad.numpy(), tdb.grad.numpy()


def _rand_net(orc, rng, convs, h, w, n_out, in_c=1):
    net = orc.Net(in_c, h, w, convs, n_out)
    cw = [rng.normal(0, 0.3, (co, ci, k, k)).astype(np.float32) for (ci, co, k, s, p) in convs]
    cb = [rng.normal(0, 0.1, co).astype(np.float32) for (ci, co, k, s, p) in convs]
    c, hl, wl = net.layer_shape(len(convs))
    dw = rng.normal(0, 0.1, (n_out, c * hl * wl)).astype(np.float32)
    db = rng.normal(0, 0.1, n_out).astype(np.float32)
    return net, cw, cb, dw, db


@pytest.mark.parametrize("convs,h,w,in_c", [
    ([(1, 5, 3, 1, 1), (5, 7, 3, 1, 1)], 12, 16, 1),                      # the paper's 2 conv + dense
    ([(4, 6, 3, 1, 1), (6, 8, 3, 1, 1), (8, 8, 3, 1, 1)], 9, 13, 4),     # ragged, stacked input
    ([(1, 4, 5, 2, 2), (4, 6, 3, 1, 0)], 17, 15, 1),                      # strided, unpadded
])
def test_backward_matches_torch_autograd(orc, convs, h, w, in_c):
    rng = np.random.default_rng(len(convs) * 100 + h)
    net, cw, cb, dw, db = _rand_net(orc, rng, convs, h, w, 5, in_c)
    x = rng.random((3, in_c, h, w)).astype(np.float32)
    g = rng.normal(0, 1, (3, 5)).astype(np.float32)
    got = orc.backward(net, cw, cb, dw, db, x, g)
    want = _torch_grads(net, cw, cb, dw, db, x, g)
    for gs, ws in zip(got, want):
        for a, b in zip(gs if isinstance(gs, list) else [gs], ws if isinstance(ws, list) else [ws]):
            assert a.shape == b.shape
            assert np.abs(a - b).max() <= 1e-6 * max(1.0, np.abs(b).max())


def test_backward_dense_closed_form_and_linearity(orc):
    # The dense layer's gradients are the outer products g^T a_L and g summed
    # over the batch; every gradient is linear in g and additive over inputs.
    rng = np.random.default_rng(5)
    net, cw, cb, dw, db = _rand_net(orc, rng, [(1, 4, 3, 1, 1), (4, 6, 3, 1, 1)], 10, 12, 3)
    x = rng.random((4, 1, 10, 12)).astype(np.float32)
    g = rng.normal(0, 1, (4, 3)).astype(np.float32)
    _, acts = orc.forward(net, cw, cb, dw, db, x, want_acts=True)
    gw, gb, gdw, gdb = orc.backward(net, cw, cb, dw, db, x, g)
    aL = acts[-1].reshape(4, -1).astype(np.float64)
    assert np.allclose(gdw, g.astype(np.float64).T @ aL, rtol=0, atol=1e-6)
    assert np.allclose(gdb, g.sum(0), rtol=0, atol=1e-6)
    g2 = orc.backward(net, cw, cb, dw, db, x, 2 * g)
    for a, b in zip(gw + gb + [gdw, gdb], g2[0] + g2[1] + [g2[2], g2[3]]):
        assert np.array_equal(2 * a, b)                # scaling by 2 is exact
    parts = [orc.backward(net, cw, cb, dw, db, x[i:i + 1], g[i:i + 1]) for i in range(4)]
    for k, tot in enumerate(gw):
        assert np.allclose(sum(p[0][k] for p in parts), tot, rtol=0, atol=1e-5)
    # an input whose activations are all zero passes no gradient to the conv weights
    z = orc.backward(net, cw, [np.full_like(b, -50.0) for b in cb], dw, db, x[:1], g[:1])
    assert all(np.count_nonzero(a) == 0 for a in z[0] + z[1])


def test_reinforce_dlogits(orc):
    # g = G (softmax(z) - onehot(a)): rows sum to 0, G = 0 gives 0, and it is
    # torch's float64 gradient of -G log_softmax(z)[a].
    rng = np.random.default_rng(9)
    z = rng.normal(0, 3, (7, 6)).astype(np.float32)
    a = rng.integers(0, 6, 7).astype(np.int32)
    G = rng.normal(0, 2, 7).astype(np.float32)
    G[3] = 0.0
    g = orc.reinforce_dlogits(z, a, G)
    assert np.abs(g.sum(1)).max() <= 1e-6
    assert np.count_nonzero(g[3]) == 0
    tz = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    loss = -(torch.tensor(G, dtype=torch.float64) *
             torch.log_softmax(tz, 1)[torch.arange(7), torch.tensor(a, dtype=torch.long)]).sum()
    loss.backward()
    assert np.abs(g - tz.grad.numpy()).max() <= 1e-6
    # large logits do not overflow (the maximum is taken out before exp)
    big = orc.reinforce_dlogits(np.array([[1000.0, 0.0]], np.float32), np.array([0], np.int32),
                                np.array([1.0], np.float32))
    assert np.all(np.isfinite(big)) and abs(big[0, 0]) < 1e-6


def test_forward_preact_relu_gives_forward(orc):
    rng = np.random.default_rng(11)
    net, cw, cb, dw, db = _rand_net(orc, rng, [(1, 4, 3, 1, 1), (4, 6, 3, 1, 1)], 10, 12, 3)
    x = rng.random((1, 1, 10, 12)).astype(np.float32)
    z = orc.forward_preact(net, cw, cb, x[0])
    _, acts = orc.forward(net, cw, cb, dw, db, x, want_acts=True)
    for zl, al in zip(z, acts):
        assert np.array_equal(np.where(zl > 0, zl, np.float32(0)), al[0])
