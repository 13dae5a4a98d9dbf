"""GPU parity of general conv layers (k x k kernels with stride 1, 2 or 4 and
pad <= (k - 1) / 2; the change growth of Fig. 1 for general k and s) against
the CPU oracle.

Masks (every layer's own grid) and work lists bit-exact; activations and logits
max abs 1e-4 against the oracle's full recompute."""
import numpy as np
import pytest

import oracle
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import ATOL_F32, check_masks, check_values, make_net, oracle_d0, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _inputs(wl, n, F, **override):
    """Per-step frames for the library (newest frame) and the oracle (stacked input)."""
    x = synth.to_f32(synth.sprite_batch(wl, streams=range(n), frames=F, **override))   # [F][n][H][W]
    if wl.stack > 1:
        xs = np.stack([np.stack([synth.stacked_view(x[:, i], t) for i in range(n)]) for t in range(F)])
    else:
        xs = x[:, :, None]
    return x, xs


def _run(torch, wl, n, F, weights, head="tiles", sample=None, label=""):
    x, xs = _inputs(wl, n, F)
    net = make_net(wl, n, weights, head=head)
    onet = oracle_net(wl)
    dev = torch.from_numpy(x).cuda()
    sample = list(range(n)) if sample is None else sample
    for t in range(F):
        logits = net.step(dev[t][:, None].contiguous()).cpu().numpy()
        d0 = oracle_d0(xs[t - 1] if t else None, xs[t], primed=t > 0)
        check_masks(net, onet, d0, np.arange(n), label=f"{label} t={t}")
        check_values(net, onet, weights, xs[t], np.arange(n), sample, logits, label=f"{label} t={t}")
    return net


def test_dqn_trunk_84x84_stacked(torch):
    # 4 stacked 84x84 frames, 8x8/4 -> 20x20x32, 4x4/2 -> 9x9x64, 3x3/1 -> 7x7x64
    # (no padding), dense -> 6; both head modes.
    wl = synth.WORKLOADS["dqn-84x84-256x64"]
    weights = synth.net_weights(wl, bias_std=0.05)
    for head in ("tiles", "full"):
        _run(torch, wl, 6, 8, weights, head=head, sample=[0, 5], label=f"dqn head={head}").close()


def test_dqn_trunk_one_stream(torch):
    # A batch of one stream (the mask kernel writes the work lists itself) on
    # the stacked DQN-style trunk: growth layer by layer through strided
    # layers, the single-frame change ring, every step checked.
    wl = synth.WORKLOADS["dqn-84x84-256x64"]
    weights = synth.net_weights(wl, bias_std=0.05)
    _run(torch, wl, 1, 7, weights, label="dqn one stream").close()


def test_general_layers_single_channel_same_and_strided(torch):
    # One input channel: 5x5/1 pad 2 (same grid), 5x5/1 pad 2, 3x3/2 pad 1 on a
    # ragged 44x36 frame, and 7x7/2 pad 3 first.
    cases = [
        ((44, 36), ((32, 5, 1, 2), (32, 5, 1, 2), (64, 3, 2, 1)), 6),
        ((42, 40), ((32, 7, 2, 3), (64, 5, 2, 2)), 18),
    ]
    for cid, ((h, w), convs, n_out) in enumerate(cases):
        wl = synth.Workload(cid=110 + cid, streams=4, frames=6, h=h, w=w, convs=convs, n_out=n_out,
                            n_sprites=3, smin=3, smax=6, vmin=1, vmax=3)
        weights = synth.net_weights(wl, bias_std=0.1)
        _run(torch, wl, 4, 6, weights, label=f"{convs}").close()


def test_general_layers_wide_grid(torch):
    # A 160x168 frame: 1680 tiles (27 tile words) on the 5x5/1 layer's grid, so
    # the list build takes its per-word offsets from the mask kernel's per-slot
    # prefixes; then 3x3/2 pad 1 to 80x84.
    wl = synth.Workload(cid=115, streams=3, frames=4, h=160, w=168, convs=((32, 5, 1, 2), (64, 3, 2, 1)), n_out=6,
                        n_sprites=5, smin=3, smax=8, vmin=1, vmax=3)
    weights = synth.net_weights(wl, bias_std=0.1)
    _run(torch, wl, 3, 4, weights, sample=[0, 2], label="wide general").close()


def test_standard_layers_around_a_general_one(torch):
    # 3x3/1 pad 1 (standard first-layer kernel) -> 3x3/1 pad 0 (general: the grid
    # shrinks by 2) -> 3x3/1 pad 1 64->128 (standard staged MFMA kernel on the
    # smaller grid); and a stacked 5x5/2 first layer.
    for cid, (convs, stack) in enumerate([((64, (64, 3, 1, 0), 128), 1),
                                          (((32, 5, 2, 2), (64, 5, 2, 2)), 4)]):
        wl = synth.Workload(cid=120 + cid, streams=4, frames=6, h=30, w=28, convs=convs, n_out=6,
                            n_sprites=3, smin=3, smax=6, vmin=1, vmax=3, stack=stack)
        weights = synth.net_weights(wl, bias_std=0.1)
        _run(torch, wl, 4, 6, weights, label=f"{convs} stack={stack}").close()


def test_general_all_changed_step_equals_full_bitwise(torch):
    # A step on which every pixel changed (list mode, every tile listed) and the
    # dense path give the same bits through general layers.
    wl = synth.Workload(cid=130, streams=3, frames=2, h=42, w=40, convs=((32, 7, 2, 3), (64, 5, 2, 2)),
                        n_out=6)
    weights = synth.net_weights(wl, bias_std=0.05)
    x, xs = _inputs(wl, 3, 2, full_change=True)
    dev = torch.from_numpy(x).cuda()
    a, b = make_net(wl, 3, weights), make_net(wl, 3, weights)
    a.step(dev[0][:, None].contiguous())
    la = a.step(dev[1][:, None].contiguous()).cpu().numpy()
    lb = b.full(dev[1][:, None].contiguous()).cpu().numpy()
    assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))
    for l in (1, 2):
        th, tw = a.layer_tiles[l]
        assert a.worklist(l).size == 3 * th * tw
        assert np.array_equal(a.activation(2, l).view(np.uint32), b.activation(2, l).view(np.uint32))
    ref, _ = oracle.forward(oracle_net(wl), *weights, xs[1])
    assert np.abs(la - ref).max() <= ATOL_F32
    a.close()
    b.close()
