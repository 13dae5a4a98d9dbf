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


def condition_biases(onet, weights, xs, rel=2.0 ** -17, tries=400):
    """Seeded test weights whose ReLU decisions are well separated from the kink.

    Backward parity compares gradients whose ReLU derivative (0 or 1) is
    decided by each activation's sign; where a pre-activation lies within the
    float32 evaluation error of 0, both derivatives are correct and two
    implementations may legitimately differ.  The error of a float32 sum of
    terms t_k scales with S = sum |t_k| (about sqrt(K) ulps of S for K terms,
    far below 2^-17 S here), so this shifts each conv channel's bias, layer by
    layer, by the smallest of a fixed sequence of steps that leaves every
    pre-activation of the inputs xs [n][C][H][W] at |z| >= 2 delta_l, delta_l
    = rel * max S_l (S_l from the oracle: the layer with |W|, |b| on the
    non-negative activations; nothing comes from the HIP path).  Returns the
    new weight tuple and the deltas."""
    conv_w, conv_b, dense_w, dense_b = weights
    conv_b = [np.array(b, np.float32, copy=True) for b in conv_b]
    deltas = []
    for l, (ci, co, k, s, p) in enumerate(onet.convs):
        _, acts = oracle.forward(onet, conv_w, conv_b, dense_w, dense_b, xs, want_acts=True)
        prev = xs if l == 0 else acts[l - 1]
        S = max(oracle.conv2d_relu(a, np.abs(conv_w[l]), np.abs(conv_b[l]), s, p).max() for a in prev)
        delta = rel * float(S)
        deltas.append(delta)
        z = np.stack([oracle.forward_preact(onet, conv_w, conv_b, x)[l] for x in xs])   # [n][co][H][W]
        steps = [0.0] + [sgn * 3.0 * delta * j for j in range(1, tries) for sgn in (1.0, -1.0)]
        for c in range(co):
            v = z[:, c].astype(np.float64).ravel()
            for eps in steps:
                if np.abs(v + eps).min() >= 2 * delta:
                    conv_b[l][c] = np.float32(conv_b[l][c] + eps)
                    break
            else:
                raise AssertionError(f"no bias shift separates layer {l + 1} channel {c} from the kink")
    for l in range(len(onet.convs)):
        zmin = min(np.abs(oracle.forward_preact(onet, conv_w, conv_b, x)[l]).min() for x in xs)
        assert zmin >= deltas[l], (l, zmin, deltas[l])
    return (conv_w, conv_b, dense_w, dense_b), deltas
