"""GPU parity of the change rule's edge cases and of paths the workload tests
do not reach, against the CPU oracle.

- Change rule (Sec. 1: activations are reused where the input pixels have
  not changed; reading: a pixel changed iff the float32 bits of some channel
  differ): -0.0 against +0.0 is a change, a bit-identical NaN is not, NaNs
  with different payloads are.  Masks and work lists bit-exact on every
  stream; values within 1e-4 on the streams whose input holds no NaN (NaN
  activations are left unspecified).
- The same levels sent as uint8 (k / 255 in the library) and as float32 give
  the same bits.
- Work-list compaction over more than 1024 streams per step (several passes
  of the compaction kernel), identity and permuted batches.
- A dense call (reuse_net_full) in the middle of a stacked-frame stream
  leaves the same state as a step on the same frame.
"""
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


# float32 bit patterns of the planted pixels (written through a uint32 view so
# that no float conversion can touch a NaN payload)
POS_ZERO, NEG_ZERO = 0x00000000, 0x80000000
NAN_A, NAN_B = 0x7FC00001, 0x7FC00002


def _edge_frames(wl, F):
    """float32 [F][6][H][W]: sprite frames with edge-case pixels planted.

    stream 0: a 5x5 block alternating +0 / -0 every frame (changes every step)
    stream 1: a 3x3 block of the same NaN in every frame (changes only when primed)
    stream 2: one pixel alternating between two NaN payloads (changes every step)
    stream 3: a 4x4 block of -0 in every frame (never changes)
    stream 4: plain sprites
    stream 5: a 2x2 block of -0, turned to +0 from frame 2 on (one change)"""
    x = synth.to_f32(synth.sprite_batch(wl, streams=range(6), frames=F))
    u = x.view(np.uint32)
    for t in range(F):
        u[t, 0, 10:15, 20:25] = POS_ZERO if t % 2 == 0 else NEG_ZERO
        u[t, 1, 40:43, 30:33] = NAN_A
        u[t, 2, 60, 50] = NAN_A if t % 2 == 0 else NAN_B
        u[t, 3, 70:74, 8:12] = NEG_ZERO
        u[t, 5, 90:92, 60:62] = NEG_ZERO if t < 2 else POS_ZERO
    return x


def test_change_rule_signed_zero_and_nan(torch):
    wl = synth.WORKLOADS["atari-ds2-256x64"]
    weights = synth.net_weights(wl, bias_std=0.05)
    F = 6
    x = _edge_frames(wl, F)
    net = make_net(wl, 6, weights)
    onet = oracle_net(wl)
    dev = torch.from_numpy(x).cuda()
    finite = [0, 3, 4, 5]
    for t in range(F):
        logits = net.step(dev[t][:, None].contiguous()).cpu().numpy()
        cur = x[t][:, None]
        d0 = oracle_d0(x[t - 1][:, None] if t else None, cur, primed=t > 0)
        if t:
            # The rule itself, independent of the library: stream 0's block and
            # stream 2's pixel changed, stream 1's NaNs and stream 3's -0 did not.
            assert d0[0, 10:15, 20:25].all() and d0[2, 60, 50] == 1
            assert d0[1, 40:43, 30:33].sum() == 0 and d0[3, 70:74, 8:12].sum() == 0
            assert d0[5, 90:92, 60:62].all() == (t == 2)
        check_masks(net, onet, d0, np.arange(6), label=f"edge t={t}")
        ref, _ = oracle.forward(onet, *weights, cur[finite])
        err = np.abs(logits[finite] - ref).max()
        assert err <= ATOL_F32, f"t={t}: logits err {err}"
        for i in finite:
            for l in (1, 2):
                _, acts = oracle.forward(onet, *weights, cur[i:i + 1], want_acts=True)
                e = np.abs(net.activation(i, l) - acts[l - 1][0]).max()
                assert e <= ATOL_F32, f"t={t} stream {i} layer {l} err {e}"
    net.close()


def test_uint8_and_float32_levels_give_the_same_bits(torch):
    wl = synth.WORKLOADS["atari-ds2-256x64"]
    weights = synth.net_weights(wl, bias_std=0.05)
    n, F = 8, 6
    u8 = synth.sprite_batch(wl, streams=range(n), frames=F)
    x = synth.to_f32(u8)
    a = make_net(wl, n, weights)
    b = make_net(wl, n, weights)
    du, df = torch.from_numpy(u8).cuda(), torch.from_numpy(x).cuda()
    for t in range(F):
        la = a.step(du[t][:, None].contiguous()).cpu().numpy()
        lb = b.step(df[t][:, None].contiguous()).cpu().numpy()
        assert np.array_equal(la.view(np.uint32), lb.view(np.uint32)), f"t={t}"
        for l in range(3):
            wa, wb = a.worklist(l) if l else None, b.worklist(l) if l else None
            if l:
                assert np.array_equal(wa, wb), f"t={t} layer {l}"
            for i in (0, n - 1):
                assert np.array_equal(a.pixel_mask(l, i), b.pixel_mask(l, i))
        for l in (0, 2):
            assert np.array_equal(a.activation(3, l).view(np.uint32), b.activation(3, l).view(np.uint32))
    a.close()
    b.close()


@pytest.mark.parametrize("h,w,n,sprites", [(16, 16, 1100, dict(n_sprites=2, smin=3, smax=4)),
                                           (64, 48, 2100, dict(n_sprites=1, smin=2, smax=3))])
def test_compaction_over_1024_streams(torch, h, w, n, sprites):
    # More than 1024 streams per step: the compaction kernel stages and
    # transposes the streams in passes of 1024 (16 x 64).  The 16x16 grid has
    # dense position bitmaps (a wave per bitmap on the last, short pass); the
    # 64x48 grid sparse ones (a thread per bitmap) over four tile words.
    wl = synth.Workload(cid=120 + n, streams=n, frames=3, h=h, w=w, convs=(40, 80), n_out=6,
                        vmin=1, vmax=2, **sprites)
    weights = synth.net_weights(wl, bias_std=0.05)
    u8 = synth.sprite_batch(wl, frames=3)
    x = synth.to_f32(u8)
    net = make_net(wl, n, weights)
    onet = oracle_net(wl)
    dev = torch.from_numpy(u8).cuda()
    sample = np.array([0, 1023, 1024, n - 1])
    for t in range(3):
        logits = net.step(dev[t][:, None].contiguous()).cpu().numpy()
        d0 = oracle_d0(x[t - 1][:, None] if t else None, x[t][:, None], primed=t > 0)
        check_masks(net, onet, d0, np.arange(n), label=f"{n} streams t={t}")
        _check_sampled(net, onet, weights, x[t][:, None], sample, sample, logits, f"{n} streams t={t}")
    # A permuted batch over most of the slots (ids through the table, several passes).
    rng = np.random.default_rng(7)
    slots = rng.permutation(n)[: n - 40].astype(np.int32)
    ids = torch.from_numpy(slots).cuda()
    u8b = synth.sprite_batch(wl, frames=4)[3]                      # one more frame per stream
    xb = synth.to_f32(u8b)[slots][:, None]
    logits = net.step(torch.from_numpy(u8b[slots][:, None].copy()).cuda(), stream_ids=ids).cpu().numpy()
    d0 = oracle_d0(x[2][slots][:, None], xb, primed=True)
    check_masks(net, onet, d0, slots, label=f"{n} streams permuted")
    pick = np.array([0, len(slots) - 1])
    _check_sampled(net, onet, weights, xb, pick, slots[pick], logits, f"{n} streams permuted")
    net.close()


def _check_sampled(net, onet, weights, x, pick, slots, logits, label):
    """Logits of batch entries `pick` and their slots' activations vs the full recompute."""
    ref, acts = oracle.forward(onet, *weights, x[pick], want_acts=True)
    err = np.abs(logits[pick] - ref).max()
    assert err <= ATOL_F32, f"{label} logits err {err}"
    for j, slot in enumerate(slots):
        for l in range(1, len(onet.convs) + 1):
            e = np.abs(net.activation(int(slot), l) - acts[l - 1][j]).max()
            assert e <= ATOL_F32, f"{label} slot {slot} layer {l} err {e}"


def test_stacked_full_mid_stream_equals_step(torch):
    # Two nets over the same stacked stream: `a` only steps, `b` takes a dense
    # call on frames 3 and 6.  With every pixel changing each frame both
    # recompute everything, so every step's logits are the same bits; with
    # sprite frames the steps after b's dense call see the stack's change
    # exactly (masks bit-exact against the oracle's diff of the stacked
    # inputs) and match the oracle's values.
    wl = synth.WORKLOADS["stack4-512x64"]
    weights = synth.net_weights(wl, bias_std=0.05)
    n, F = 4, 9
    onet = oracle_net(wl)
    for full_change in (True, False):
        u8 = synth.sprite_batch(wl, streams=range(n), frames=F, full_change=full_change)
        x = synth.to_f32(u8)
        xs = np.stack([np.stack([synth.stacked_view(x[:, i], t) for i in range(n)]) for t in range(F)])
        a = make_net(wl, n, weights)
        b = make_net(wl, n, weights)
        dev = torch.from_numpy(u8).cuda()
        for t in range(F):
            f = dev[t][:, None].contiguous()
            la = a.step(f).cpu().numpy()
            lb = (b.full(f) if t in (3, 6) else b.step(f)).cpu().numpy()
            label = f"full_change={full_change} t={t}"
            if full_change:
                assert np.array_equal(la.view(np.uint32), lb.view(np.uint32)), label
            d0 = oracle_d0(xs[t - 1] if t else None, xs[t], primed=t > 0)
            check_masks(a, onet, d0, np.arange(n), label=label + " (steps)")
            if t not in (3, 6):
                check_masks(b, onet, d0, np.arange(n), label=label + " (after full)")
            for net, lg in ((a, la), (b, lb)):
                check_values(net, onet, weights, xs[t], np.arange(n), [0, n - 1], lg, label=label)
            assert np.array_equal(b.activation(1, 0), x[t][1][None])   # newest frame of the ring
        a.close()
        b.close()
