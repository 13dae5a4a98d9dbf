"""GPU parity of the training path (Sec. 2: the policy is trained with
REINFORCE) against the oracle, through the C ABI.

- reuse_net_reinforce_dlogits against the oracle's REINFORCE logit gradient.
- reuse_net_backward after reuse steps (the caches then hold the activations
  of the current frames) against the oracle's backpropagation of the full
  recompute, every weight and bias gradient element by element: max abs error
  <= 1e-4 * max(1, max |oracle|) per tensor.  The test weights have their
  conv biases shifted (tests.gpu_util.condition_biases, oracle only) so that
  no pre-activation lies within the float32 evaluation error of the ReLU kink,
  where either derivative would be correct.
- accumulate adds exactly (2 g), and the result is deterministic.
- reuse_net_sgd_step equals a net created with the updated weights
  fl(w - fl(lr g)): the same logits, masks and next gradients, bit for bit.
"""
import numpy as np
import pytest

import oracle
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import condition_biases, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]

REL = 1e-4


@pytest.fixture(scope="module")
def torch():
    import torch
    return torch


def _wl(base, h, w, n):
    b = synth.WORKLOADS[base]
    return synth.Workload(cid=b.cid + 40, streams=n, frames=4, h=h, w=w, convs=b.convs, n_out=b.n_out,
                          n_sprites=3, smin=3, smax=6, vmin=1, vmax=2, stack=b.stack)


def _inputs(wl, n, F):
    u8 = synth.sprite_batch(wl, streams=range(n), frames=F)
    x = synth.to_f32(u8)
    if wl.stack > 1:
        xs = np.stack([np.stack([synth.stacked_view(x[:, i], t) for i in range(n)]) for t in range(F)])
    else:
        xs = x[:, :, None]
    return u8, xs                                              # xs [F][n][C][H][W]


def _net(wl, slots_n, weights, head, fuse_first=True):
    from paper_1909_05632_amd import ReuseNet
    return ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, slots_n, weights, stack=wl.stack, head=head,
                    fuse_first=fuse_first)


def _grads_np(net, grads):
    cw, cb, dw, db = net.split_grads(grads)
    return [t.cpu().numpy() for t in cw] + [t.cpu().numpy() for t in cb] + [dw.cpu().numpy(), db.cpu().numpy()]


def _oracle_np(onet, weights, x, g):
    gw, gb, gdw, gdb = oracle.backward(onet, *weights, x, g)
    return gw + gb + [gdw, gdb]


def _compare(got, want, label):
    for k, (a, b) in enumerate(zip(got, want)):
        assert a.shape == b.shape, (label, k, a.shape, b.shape)
        tol = REL * max(1.0, float(np.abs(b).max()))
        err = float(np.abs(a.astype(np.float64) - b).max())
        assert err <= tol, f"{label}: gradient tensor {k} err {err} > {tol}"


CASES = [
    # (workload shape source, h, w, streams, slots, head, fuse_first)
    ("atari-ds2-256x64", 40, 32, 3, [4, 0, 2], "tiles", True),       # 1->40->80, layer 1 folded
    ("atari-ds2-256x64", 40, 32, 3, None, "full", False),            # separate layer 1, full-read head
    ("stack4-512x64", 40, 32, 2, [1, 0], "full", True),              # 4 stacked frames -> 40 -> 80
    ("fullres-1024x32", 42, 32, 2, None, "tiles", True),             # 1->64->128->128, 18 logits
    # 99 tiles a stream, 297 in all: weight-gradient teams of 8 and 9 tiles,
    # passes that end past a team's last tile, tile walks across streams
    ("atari-ds2-256x64", 44, 36, 3, [2, 0, 1], "tiles", True),
]


@pytest.mark.parametrize("base,h,w,n,slots,head,fuse", CASES)
def test_backward_matches_oracle(torch, base, h, w, n, slots, head, fuse):
    wl = _wl(base, h, w, n)
    F = 4
    u8, xs = _inputs(wl, n, F)
    onet = oracle_net(wl)
    weights, deltas = condition_biases(onet, synth.net_weights(wl, bias_std=0.05), xs[F - 1])
    S = (max(slots) + 1) if slots else n
    net = _net(wl, S, weights, head, fuse)
    ids = torch.tensor(slots, dtype=torch.int32).cuda() if slots else None
    dev = torch.from_numpy(u8).cuda()
    for t in range(F):                                         # reuse steps; the caches end at frame F-1
        net.step(dev[t][:, None].contiguous(), stream_ids=ids)
    rng = np.random.default_rng(h * 7 + n)
    g = rng.normal(0, 1, (n, wl.n_out)).astype(np.float32)
    gd = torch.from_numpy(g).cuda()
    grads = net.new_grads()
    net.backward(gd, grads, stream_ids=ids)
    got = _grads_np(net, grads)
    _compare(got, _oracle_np(onet, weights, xs[F - 1], g), f"{base} {h}x{w} head={head}")
    # accumulate adds the same gradient again (x2 is exact); a second buffer
    # from scratch has the same bits (fixed summation order)
    net.backward(gd, grads, stream_ids=ids, accumulate=True)
    again = _grads_np(net, grads)
    for a, b in zip(got, again):
        assert np.array_equal((2 * a).view(np.uint32), b.view(np.uint32))
    fresh = net.new_grads()
    net.backward(gd, fresh, stream_ids=ids)
    for a, b in zip(got, _grads_np(net, fresh)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    net.close()


def test_reinforce_dlogits_matches_oracle(torch):
    from paper_1909_05632_amd import ReuseNet  # noqa: F401  (loads the library)
    from paper_1909_05632_amd import binding as B
    rng = np.random.default_rng(4)
    for n, n_out in ((1, 6), (300, 18), (37, 64)):
        z = rng.normal(0, 3, (n, n_out)).astype(np.float32)
        a = rng.integers(0, n_out, n).astype(np.int32)
        G = rng.normal(0, 2, n).astype(np.float32)
        zd, ad, Gd = (torch.from_numpy(v).cuda() for v in (z, a, G))
        out = torch.empty((n, n_out), dtype=torch.float32).cuda()
        B.reuse_net_reinforce_dlogits(n, n_out, zd.data_ptr(), ad.data_ptr(), Gd.data_ptr(), out.data_ptr(),
                                      torch.cuda.current_stream().cuda_stream)
        want = oracle.reinforce_dlogits(z, a, G)
        err = np.abs(out.cpu().numpy() - want).max()
        assert err <= 1e-6 * max(1.0, np.abs(want).max()), (n, n_out, err)


def test_sgd_step_equals_net_with_updated_weights(torch):
    # A rollout, a backward, an SGD step on the device; a second net created
    # with the host-updated weights fl(w - fl(lr g)) must give the same logits,
    # masks (the first step after the update recomputes everything) and next
    # gradients, bit for bit, on both heads.
    for base, h, w, n, head in (("atari-ds2-256x64", 40, 32, 3, "tiles"), ("fullres-1024x32", 42, 32, 2, "full")):
        wl = _wl(base, h, w, n)
        F = 6
        u8, _ = _inputs(wl, n, F)
        weights = synth.net_weights(wl, bias_std=0.05)
        dev = torch.from_numpy(u8).cuda()
        a = _net(wl, n, weights, head)
        for t in range(3):
            a.step(dev[t][:, None].contiguous())
        g = torch.from_numpy(np.random.default_rng(1).normal(0, 1, (n, wl.n_out)).astype(np.float32)).cuda()
        grads = a.new_grads()
        a.backward(g, grads)
        lr = 0.05
        a.sgd_step(grads, lr)
        gh = [v.cpu().numpy() for v in (*a.split_grads(grads)[0], *a.split_grads(grads)[1],
                                         a.split_grads(grads)[2], a.split_grads(grads)[3])]
        L = len(wl.convs)
        lr32 = np.float32(lr)
        cw = [weights[0][l] - lr32 * gh[l] for l in range(L)]
        cb = [weights[1][l] - lr32 * gh[L + l] for l in range(L)]
        dw = weights[2] - lr32 * gh[2 * L].reshape(weights[2].shape)
        db = weights[3] - lr32 * gh[2 * L + 1]
        b = _net(wl, n, (cw, cb, dw, db), head)
        for t in range(3, F):
            la = a.step(dev[t][:, None].contiguous()).cpu().numpy()
            lb = b.step(dev[t][:, None].contiguous()).cpu().numpy()
            assert np.array_equal(la.view(np.uint32), lb.view(np.uint32)), (base, t)
            if t == 3:                                         # unprimed by the update: all dirty
                assert all(a.tile_mask_u8(L, i).all() for i in range(n))
            for l in range(1, L + 1):
                assert np.array_equal(a.worklist(l), b.worklist(l))
        ga, gb = a.new_grads(), b.new_grads()
        a.backward(g, ga)
        b.backward(g, gb)
        assert np.array_equal(ga.cpu().numpy().view(np.uint32), gb.cpu().numpy().view(np.uint32)), base
        a.close()
        b.close()


def test_set_weights_device_equals_created_nets(torch):
    # reuse_net_set_weights_device rewrites every packed copy on the device from
    # a flat parameter buffer: the net must then compute exactly as one created
    # with those weights (logits, masks, work lists and gradients bit for bit),
    # and exactly as one whose weights came through the host path
    # (reuse_net_set_weights), on the epilogue tile head, the float32 tile
    # partials of a staged last layer (128 -> 128) and the full-read head.
    for base, h, w, n, head in (("atari-ds2-256x64", 40, 32, 3, "tiles"), ("fullres-1024x32", 42, 32, 2, "tiles"),
                                ("fullres-1024x32", 42, 32, 2, "full")):
        wl = _wl(base, h, w, n)
        F = 7
        u8, _ = _inputs(wl, n, F)
        w0 = synth.net_weights(wl, bias_std=0.05)
        w1 = synth.net_weights(wl, bias_std=0.05, seed_extra=3)
        dev = torch.from_numpy(u8).cuda()
        a = _net(wl, n, w0, head)
        for t in range(2):
            a.step(dev[t][:, None].contiguous())
        a.set_weights_device(a.pack_params(w1))
        b = _net(wl, n, w1, head)
        L = len(wl.convs)
        g = torch.from_numpy(np.random.default_rng(2).normal(0, 1, (n, wl.n_out)).astype(np.float32)).cuda()

        def same(t0, t1, label):
            for t in range(t0, t1):
                la = a.step(dev[t][:, None].contiguous()).cpu().numpy()
                lb = b.step(dev[t][:, None].contiguous()).cpu().numpy()
                assert np.array_equal(la.view(np.uint32), lb.view(np.uint32)), (base, head, label, t)
                if t == t0:                                    # unprimed by the update: all dirty
                    assert all(a.tile_mask_u8(L, i).all() for i in range(n))
                for l in range(1, L + 1):
                    assert np.array_equal(a.worklist(l), b.worklist(l)), (base, head, label, t, l)
            ga, gb = a.new_grads(), b.new_grads()
            a.backward(g, ga)
            b.backward(g, gb)
            assert np.array_equal(ga.cpu().numpy().view(np.uint32), gb.cpu().numpy().view(np.uint32)), \
                (base, head, label)

        same(2, 5, "device vs created")
        # Back to w0: device path on a, host path on b.
        a.set_weights_device(a.pack_params(w0))
        b.set_weights(w0)
        same(5, F, "device vs host")
        a.close()
        b.close()


def test_set_weights_device_unsupported_net(torch):
    # A net the training calls do not support (general-layer DQN trunk) refuses
    # the device update before reading the buffer, and keeps its weights.
    from paper_1909_05632_amd import binding as B
    wl = synth.WORKLOADS["dqn-84x84-256x64"]
    weights = synth.net_weights(wl)
    from paper_1909_05632_amd import ReuseNet
    net = ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, 2, weights, stack=wl.stack)
    assert net.grad_elems() == 0
    buf = torch.zeros(16, dtype=torch.float32, device="cuda")
    rc = B.load_library().reuse_net_set_weights_device(net.handle, buf.data_ptr(), None)
    assert rc == B.RN_EUNSUPPORTED
    with pytest.raises(RuntimeError):
        net.pack_params(weights)
    net.close()
