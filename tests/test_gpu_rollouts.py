"""Reuse inside fixed-weight rollouts with weight updates between them (the
training use of Sec. 1 and Sec. 2): reuse_net_set_weights replaces the weights
and every slot recomputes everything on its next step.

Against the CPU oracle: masks and work lists bit-exact (the first step after
an update is all-changed), logits max abs 1e-4 with the weights in force; and
bitwise against a net created with the new weights."""
import numpy as np
import pytest

import oracle
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import check_masks, check_values, make_net, oracle_d0, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _rollouts(torch, wl, n, episodes, length, label):
    """Episodes of `length` frames; weights k for episode k; stacked views restart per episode."""
    F = episodes * length
    x = synth.to_f32(synth.sprite_batch(wl, streams=range(n), frames=F))           # [F][n][H][W]
    weights = [synth.net_weights(wl, bias_std=0.05, seed_extra=k) for k in range(episodes)]
    onet = oracle_net(wl)
    net = make_net(wl, n, weights[0])
    dev = torch.from_numpy(x).cuda()
    fresh_logits = []
    for ep in range(episodes):
        if ep:
            net.set_weights(weights[ep])
        fresh = make_net(wl, n, weights[ep])
        for j in range(length):
            t = ep * length + j
            seq = x[ep * length:t + 1]                                              # this episode's frames
            if wl.stack > 1:
                cur = np.stack([synth.stacked_view(seq[:, i], j) for i in range(n)])
                prev = (np.stack([synth.stacked_view(seq[:, i], j - 1) for i in range(n)]) if j else None)
            else:
                cur, prev = seq[j][:, None], (seq[j - 1][:, None] if j else None)
            frame = dev[t][:, None].contiguous()
            logits = net.step(frame).cpu().numpy()
            lf = fresh.step(frame).cpu().numpy()
            assert np.array_equal(logits.view(np.uint32), lf.view(np.uint32)), f"{label} ep={ep} t={j}"
            d0 = oracle_d0(prev, cur, primed=j > 0)
            check_masks(net, onet, d0, np.arange(n), label=f"{label} ep={ep} t={j}")
            check_values(net, onet, weights[ep], cur, np.arange(n), [0], logits, label=f"{label} ep={ep} t={j}")
            if j == 0:
                for l in range(len(wl.convs) + 1):
                    assert net.tile_mask_u8(l, 0).all()                            # stale caches never used
        fresh.close()
    net.close()


def test_rollouts_with_weight_updates_105x80(torch):
    wl = synth.WORKLOADS["atari-ds2-256x64"]
    _rollouts(torch, wl, 6, 3, 4, "105x80")


def test_rollouts_with_weight_updates_dqn_stacked(torch):
    wl = synth.WORKLOADS["dqn-84x84-256x64"]
    _rollouts(torch, wl, 4, 2, 5, "dqn")
