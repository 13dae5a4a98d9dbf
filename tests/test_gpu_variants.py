"""GPU parity of reuse_net_variants (copy-on-write variants of one primed slot)
against the CPU oracle.

A variant is the base slot's input with the pixels of its boxes taken from its
frame; the expected logits are the oracle's full recompute of that input, the
expected masks and work lists the oracle's change growth of the box mask (one
entry per variant, in (ty, tx, variant) order).  Masks and lists bit-exact;
logits max abs 1e-4 (float32) or 1e-2 of the largest logit (bf16)."""
import numpy as np
import pytest

import oracle
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import ATOL_F32, check_masks, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

BF16_REL = 1e-2


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _net(wl, weights, act_dtype="f32", fuse_first=True, streams=2):
    from paper_1909_05632_amd import ReuseNet
    return ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, streams, weights, act_dtype=act_dtype,
                    fuse_first=fuse_first)


def _random_boxes(rng, n, h, w):
    """Per variant 0..3 boxes: inside, clipped at every edge, empty, and one
    variant whose box covers the whole frame."""
    boxes, off = [], [0]
    for i in range(n):
        k = int(rng.integers(0, 4)) if i else 1
        for _ in range(k):
            if i == 0:
                b = (-2, -3, h + 5, w + 1)                        # whole frame, clipped
            else:
                y0 = int(rng.integers(-4, h))
                x0 = int(rng.integers(-4, w))
                b = (y0, x0, y0 + int(rng.integers(0, 11)), x0 + int(rng.integers(0, 11)))
            boxes.append(b)
        off.append(len(boxes))
    return np.asarray(boxes, np.int32).reshape(-1, 4), np.asarray(off, np.int32)


def _base_frame(wl, seed=0):
    u8 = synth.sprite_batch(wl, streams=[seed], frames=1)
    return synth.to_f32(u8)[0]                                    # [1][H][W]


def _run_variants(torch, wl, weights, n, seed, act_dtype="f32", fuse_first=True, shared=False,
                  u8=False, max_tiles=0, base_slot=1, sample=None, label=""):
    rng = np.random.default_rng(seed)
    base = _base_frame(wl, seed)
    net = _net(wl, weights, act_dtype, fuse_first)
    ids = torch.tensor([base_slot], dtype=torch.int32).cuda()
    net.full(torch.from_numpy(base[None]).cuda(), stream_ids=ids)
    boxes, off = _random_boxes(rng, n, wl.h, wl.w)
    nf = 1 if shared else n
    fu8 = rng.integers(0, 256, (nf, 1, wl.h, wl.w), dtype=np.uint8)
    fx = synth.to_f32(fu8)
    dev_frames = torch.from_numpy(fu8 if u8 else fx).cuda()
    logits = net.variants(base_slot, torch.from_numpy(boxes).cuda(), torch.from_numpy(off).cuda(),
                          dev_frames, max_tiles=max_tiles).cpu().numpy()
    bf = act_dtype == "bf16"
    onet = oracle_net(wl, bf16=bf)
    vb = [boxes[off[i]:off[i + 1]] for i in range(n)]
    d0 = np.stack([oracle.box_mask(wl.h, wl.w, b) for b in vb])
    check_masks(net, onet, d0, np.arange(n), label=label)
    sample = list(range(n)) if sample is None else sample
    xs = np.stack([oracle.variant_input(base, fx[0 if shared else i], vb[i]) for i in sample])
    ref, _ = oracle.forward(onet, *weights, xs)
    got = logits[sample]
    tol = BF16_REL * np.abs(ref).max() if bf else ATOL_F32
    err = np.abs(got - ref).max()
    assert err <= tol, f"{label} logits max abs err {err} > {tol}"
    return net, logits, base, boxes, off


def test_variants_folded_first_layer_105x80(torch):
    # The occlusion workload's net (1->40->80, 6 logits; layer 1 folded into
    # layer 2), per-variant float32 frames and one shared uint8 frame.
    wl = synth.WORKLOADS["occlusion-105x80-4096"]
    weights = synth.net_weights(wl, bias_std=0.05)
    net, *_ = _run_variants(torch, wl, weights, 40, 1, label="folded f32 frames")
    net.close()
    net, *_ = _run_variants(torch, wl, weights, 33, 2, shared=True, u8=True, label="folded shared u8")
    net.close()


def test_variants_separate_first_layer_ragged(torch):
    # Layer 1 as its own kernel: its recomputed tiles go to the layer-1
    # overlay and layer 2's halos read overlay or base tile by tile.
    for (h, w) in [(30, 28), (17, 68)]:
        wl = synth.Workload(cid=90 + h, streams=2, frames=1, h=h, w=w, convs=(40, 80), n_out=6,
                            n_sprites=2, smin=2, smax=5, vmin=1, vmax=3)
        weights = synth.net_weights(wl, bias_std=0.1)
        net, *_ = _run_variants(torch, wl, weights, 25, 3 + h, fuse_first=False, label=f"sep {h}x{w}")
        net.close()


def test_variants_three_layers_staged(torch):
    # 1->64->128->128, 18 logits: first-layer kernel, weight-staged matrix
    # kernels for an intermediate layer (overlay out) and the last layer
    # (head partials only).
    wl = synth.Workload(cid=95, streams=2, frames=1, h=42, w=32, convs=(64, 128, 128), n_out=18,
                        n_sprites=3, smin=3, smax=6, vmin=1, vmax=3)
    weights = synth.net_weights(wl, bias_std=0.05)
    net, *_ = _run_variants(torch, wl, weights, 30, 4, label="3-layer f32")
    net.close()


def test_variants_bf16(torch):
    for convs, n_out, cid in (((64, 128, 128), 18, 96), ((32, 64, 64), 6, 97)):
        wl = synth.Workload(cid=cid, streams=2, frames=1, h=42, w=32, convs=convs, n_out=n_out,
                            n_sprites=3, smin=3, smax=6, vmin=1, vmax=3)
        weights = synth.net_weights(wl, bias_std=0.05)
        net, *_ = _run_variants(torch, wl, weights, 30, cid, act_dtype="bf16", label=f"bf16 {convs}")
        net.close()


def test_variant_edge_cases(torch):
    # Empty boxes -> the base slot's logits bit for bit; the base slot is left
    # as it was (a step on its unchanged frame finds no work and repeats its
    # logits); a variant over the tile limit gets NaN while the others stay
    # exact; an unprimed base gives NaN everywhere.
    wl = synth.WORKLOADS["occlusion-105x80-4096"]
    weights = synth.net_weights(wl, bias_std=0.05)
    base = _base_frame(wl, 5)
    net = _net(wl, weights)
    ids = torch.tensor([1], dtype=torch.int32).cuda()
    dev_base = torch.from_numpy(base[None]).cuda()
    base_logits = net.full(dev_base, stream_ids=ids).cpu().numpy()[0]
    boxes = np.asarray([(10, 10, 14, 14), (0, 0, 105, 80), (50, 30, 58, 38)], np.int32)
    off = np.asarray([0, 0, 1, 2, 3, 3], np.int32)                 # variants 0 and 4: no boxes
    zero = torch.zeros((1, 1, wl.h, wl.w), dtype=torch.float32).cuda()
    tb, to = torch.from_numpy(boxes).cuda(), torch.from_numpy(off).cuda()
    out = net.variants(1, tb, to, zero, max_tiles=40).cpu().numpy()
    assert np.array_equal(out[0].view(np.uint32), base_logits.view(np.uint32))
    assert np.array_equal(out[4].view(np.uint32), base_logits.view(np.uint32))
    assert np.isnan(out[2]).all()                                  # whole frame: over the limit
    assert not np.isnan(out[[0, 1, 3, 4]]).any()
    onet = oracle_net(wl)
    for i in (1, 3):
        x = oracle.variant_input(base, np.zeros_like(base), boxes[off[i]:off[i + 1]])
        ref, _ = oracle.forward(onet, *weights, x[None])
        assert np.abs(out[i] - ref[0]).max() <= ATOL_F32, i
    again = net.step(dev_base, stream_ids=ids).cpu().numpy()[0]
    assert np.array_equal(again.view(np.uint32), base_logits.view(np.uint32))
    assert net.worklist(2).size == 0
    fresh = _net(wl, weights)
    nan = fresh.variants(0, tb, to, zero).cpu().numpy()
    assert np.isnan(nan).all()
    fresh.close()
    net.close()


def test_occlusion_4096_variants_full_size(torch):
    # The occlusion workload at full size: 4096 variants of one 105x80 base,
    # an 8x8 zero patch at every top-left corner of the 64x64 grid, one shared
    # zero frame, at most 16 dirty tiles per variant and layer (as timed).
    # Masks and work lists of every variant bit-exact; logits of a sample.
    wl = synth.WORKLOADS["occlusion-105x80-4096"]
    weights = synth.net_weights(wl)
    P, G = wl.extra["patch"], wl.extra["grid"]
    base = synth.to_f32(synth.occlusion_base(wl))                 # [H][W]
    net = _net(wl, weights)
    net.full(torch.from_numpy(base[None, None]).cuda())
    boxes = np.asarray([(y, x, y + P, x + P) for y in range(G) for x in range(G)], np.int32)
    off = np.arange(G * G + 1, dtype=np.int32)
    zero = torch.zeros((1, 1, wl.h, wl.w), dtype=torch.float32).cuda()
    logits = net.variants(0, torch.from_numpy(boxes).cuda(), torch.from_numpy(off).cuda(), zero,
                          max_tiles=16).cpu().numpy()
    assert not np.isnan(logits).any()
    onet = oracle_net(wl)
    d0 = np.stack([oracle.box_mask(wl.h, wl.w, boxes[i:i + 1]) for i in range(G * G)])
    check_masks(net, onet, d0, np.arange(G * G), label="4096 variants")
    sample = [0, 1, 63, 64, 2047, 2048, 4031, 4095] + list(np.random.default_rng(9).integers(0, 4096, 8))
    xs = np.stack([synth.occlusion_variant_frame(base, i // G, i % G, P)[None] for i in sample])
    ref, _ = oracle.forward(onet, *weights, xs)
    assert np.abs(logits[sample] - ref).max() <= ATOL_F32
    net.close()
