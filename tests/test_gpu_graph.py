"""A reuse step captured in a HIP graph (torch.cuda.CUDAGraph over the C ABI).

A step only enqueues kernels on the caller's stream: no memset or copy nodes,
no host synchronisation, per-layer work counts kept on the device.  So a step
captured once replays correctly as long as its buffers stay in place: the frame
(and stream-id) buffers are refilled between replays, with eager work and
synchronisations in between, and every replay's logits, masks and work lists
must equal those of eager steps on a second net, bit for bit."""
import numpy as np
import pytest

from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import make_net, sprite_inputs

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _same_state(a, b, slots, L, label):
    for l in range(L + 1):
        for s in slots:
            assert np.array_equal(a.pixel_mask_u8(l, s), b.pixel_mask_u8(l, s)), f"{label} pixel mask {l} slot {s}"
            assert np.array_equal(a.tile_mask_u8(l, s), b.tile_mask_u8(l, s)), f"{label} tile mask {l} slot {s}"
    for l in range(1, L + 1):
        assert np.array_equal(a.worklist(l), b.worklist(l)), f"{label} work list {l}"


@pytest.mark.parametrize("batch", ["all", "one"])
def test_step_replayed_from_a_graph_equals_eager_steps(torch, batch):
    # 6 slots of 44x48 frames, 3x3 layers 1 -> 40 -> 80, 6 logits.  "all": the
    # whole batch each step (compaction kernel); "one": slot 2 alone (the mask
    # kernel writes the lists).
    n, F = 6, 7
    wl = synth.Workload(cid=150, streams=n, frames=F, h=44, w=48, convs=(40, 80), n_out=6,
                        n_sprites=3, smin=2, smax=6, vmin=1, vmax=3)
    weights = synth.net_weights(wl, bias_std=0.1)
    _, x = sprite_inputs(wl, range(n), F)                       # [F][n][H][W]
    dev = torch.from_numpy(x).cuda()
    slots = list(range(n)) if batch == "all" else [2]
    ids = torch.tensor(slots, dtype=torch.int32, device="cuda")
    sel = ids.long()
    eager, graphed = make_net(wl, n, weights), make_net(wl, n, weights)
    frames = torch.empty((len(slots), 1, wl.h, wl.w), dtype=torch.float32, device="cuda")
    logits = torch.empty((len(slots), wl.n_out), dtype=torch.float32, device="cuda")

    # Frame 0 primes both nets eagerly (and makes every one-time set-up happen
    # outside the capture).
    f0 = dev[0][sel][:, None].contiguous()
    eager.step(f0, stream_ids=ids)
    graphed.step(f0, stream_ids=ids)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    frames.copy_(dev[1][sel][:, None])
    with torch.cuda.graph(g):
        graphed.step(frames, stream_ids=ids, out=logits)
    torch.cuda.synchronize()

    for t in range(1, F):
        frames.copy_(dev[t][sel][:, None])
        g.replay()
        want = eager.step(dev[t][sel][:, None].contiguous(), stream_ids=ids)
        torch.cuda.synchronize()
        got = logits.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.cpu().numpy().view(np.uint32)), f"replay {t} logits"
        _same_state(graphed, eager, slots, 2, label=f"{batch} replay {t}")
        for s in slots[:2]:
            for l in (1, 2):
                assert np.array_equal(graphed.activation(s, l), eager.activation(s, l)), f"replay {t} act {l} slot {s}"
    eager.close()
    graphed.close()
