"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
and compare it with the CPU oracle on the same seeded inputs."""
from __future__ import annotations

import numpy as np

import oracle
from synth import frames as synth

ATOL_F32 = 1e-4          # max abs error on activations and logits, float32 path


def oracle_net(wl, bf16=False):
    return oracle.Net(wl.in_c, wl.h, wl.w, wl.conv_specs(), wl.n_out, 4, 4, bf16)


def make_net(wl, streams, weights, act_dtype="f32", head="tiles"):
    from paper_1909_05632_amd import ReuseNet
    return ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, streams, weights, act_dtype=act_dtype,
                    stack=wl.stack, head=head)


def oracle_d0(prev_x, cur_x, primed):
    """Change masks [n][H][W] of one step from float32 inputs [n][C][H][W]."""
    n = cur_x.shape[0]
    if not primed:
        return np.ones((n,) + cur_x.shape[2:], np.uint8)
    return np.stack([oracle.diff(prev_x[i], cur_x[i]) for i in range(n)])


def check_masks(net, onet, d0, slots, label=""):
    """Pixel masks, tile masks and work lists of every layer, bit-exact."""
    d, m = oracle.masks(onet, d0)
    L = len(onet.convs)
    for l in range(L + 1):
        for i, slot in enumerate(slots):
            got = net.pixel_mask_u8(l, int(slot))
            assert np.array_equal(got, d[l][i]), f"{label} pixel mask layer {l} stream {i}"
            got = net.tile_mask_u8(l, int(slot))
            assert np.array_equal(got, m[l][i]), f"{label} tile mask layer {l} stream {i}"
    for l in range(1, L + 1):
        got = net.worklist(l)
        want = oracle.worklist(m[l])
        assert np.array_equal(got, want), f"{label} work list layer {l}: {len(got)} vs {len(want)}"
    return d, m


def check_values(net, onet, weights, x, slots, sample, logits, atol=ATOL_F32, label="",
                 acts=True, rel=None):
    """Logits of every stream and activations of the sampled streams vs the full recompute."""
    ref_logits, ref_acts = oracle.forward(onet, *weights, x, want_acts=acts)
    err = np.abs(logits - ref_logits).max()
    tol = atol if rel is None else rel * max(np.abs(ref_logits).max(), 1e-30)
    assert err <= tol, f"{label} logits max abs err {err} > {tol}"
    if acts:
        for i in sample:
            for l in range(1, len(onet.convs) + 1):
                got = net.activation(int(slots[i]), l)
                want = ref_acts[l - 1][i]
                e = np.abs(got - want).max()
                tol = atol if rel is None else rel * max(np.abs(want).max(), 1e-30)
                assert e <= tol, f"{label} layer {l} stream {i} act max abs err {e} > {tol}"
    return ref_logits


def sprite_inputs(wl, streams, frames, **override):
    u8 = synth.sprite_batch(wl, streams=streams, frames=frames, **override)
    return u8, synth.to_f32(u8)
