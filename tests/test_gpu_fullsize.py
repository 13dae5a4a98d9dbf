"""GPU parity at the benchmark workloads' full stream counts and frame sizes
(the launch configuration bench.py times): masks and work lists of every
stream bit-exact on every step, logits and activations of sampled streams
against the oracle's full recompute (float32 max abs 1e-4; bf16 1e-2 of each
tensor's largest magnitude)."""
import numpy as np
import pytest

import oracle
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import ATOL_F32, check_masks, make_net, oracle_d0, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

BF16_REL = 1e-2


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _check_sample(net, onet, weights, cur, sample, logits, rel, label):
    ref_logits, ref_acts = oracle.forward(onet, *weights, cur[sample], want_acts=True)
    tol = ATOL_F32 if rel is None else rel * max(np.abs(ref_logits).max(), 1e-30)
    err = np.abs(logits[sample] - ref_logits).max()
    assert err <= tol, f"{label} logits err {err} > {tol}"
    for j, i in enumerate(sample):
        for l in range(1, len(onet.convs) + 1):
            want = ref_acts[l - 1][j]
            got = net.activation(int(i), l)
            tol = ATOL_F32 if rel is None else rel * max(np.abs(want).max(), 1e-30)
            e = np.abs(got - want).max()
            assert e <= tol, f"{label} stream {i} layer {l} err {e} > {tol}"


def _run(torch, wl, n, F, sample, value_every, act_dtype="f32", preset=None, label="", u8_frames=True):
    weights = synth.net_weights(wl)
    u8 = synth.sprite_batch(wl, streams=range(n), frames=F, **(preset or {}))
    x = synth.to_f32(u8)                                            # [F][n][H][W]
    net = make_net(wl, n, weights, act_dtype=act_dtype)
    onet = oracle_net(wl, bf16=act_dtype == "bf16")
    # uint8 levels (k/255 in the library) or the float32 frames the benchmark feeds
    dev = torch.from_numpy(u8 if u8_frames else x).cuda()
    rel = BF16_REL if act_dtype == "bf16" else None
    prev = None
    for t in range(F):
        logits = net.step(dev[t][:, None].contiguous()).cpu().numpy()
        if wl.stack > 1:
            cur = np.stack([synth.stacked_view(x[:, i], t) for i in range(n)])
        else:
            cur = x[t][:, None]
        d0 = oracle_d0(prev, cur, primed=t > 0)
        check_masks(net, onet, d0, np.arange(n), label=f"{label} t={t}")
        if t % value_every == 0 or t == F - 1:
            _check_sample(net, onet, weights, cur, sample, logits, rel, f"{label} t={t}")
        prev = cur
    net.close()


def test_stack4_512x64_full_size(torch):
    wl = synth.WORKLOADS["stack4-512x64"]
    _run(torch, wl, 512, 64, [0, 1, 256, 511], 16, label="stack4 512x64")


@pytest.mark.parametrize("act_dtype,frac", [("f32", 0.01), ("f32", 0.05), ("bf16", 0.01), ("bf16", 0.05)])
def test_fullres_1024_streams(torch, act_dtype, frac):
    # 1024 streams of 210x160 at the 1% and 5% change presets (the operating
    # points of the benchmark's metric), 8 frames; float32 frames for the
    # float32 net (as the benchmark feeds them), uint8 levels for bf16.
    wl = synth.WORKLOADS["fullres-1024x32"]
    _run(torch, wl, 1024, 8, [0, 511, 1023], 4, act_dtype=act_dtype,
         preset=dict(synth.FRACTION_PRESETS[frac]), label=f"fullres 1024 {act_dtype} {frac}",
         u8_frames=act_dtype != "f32")


def test_dqn_trunk_256_streams_full_size(torch):
    # The DQN-style trunk (4 stacked 84x84 frames; 8x8/4, 4x4/2, 3x3/1 layers)
    # at the 256 streams the benchmark times, 10 frames.
    wl = synth.WORKLOADS["dqn-84x84-256x64"]
    _run(torch, wl, 256, 10, [0, 1, 128, 255], 3, label="dqn 256")
