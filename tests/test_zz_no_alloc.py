"""reuse_net_variants_static (the library's static per-GPU scratch, no
allocation) against reuse_net_variants (caller scratch) through the C ABI:
the same kernels on the same inputs, so logits, masks and work lists must be
the same bits.  Two calls in a row, the second with fewer variants (the static
scratch keeps the first call's contents), then a request beyond the static
limit, which must be refused before any launch.  The logits of both are also
checked against the oracle's full recompute of each variant's input (float32,
max abs 1e-4)."""
import numpy as np
import pytest

import oracle
from paper_1909_05632_amd import binding as B
from synth import frames as synth
from tests.conftest import gpu_available
from tests.gpu_util import ATOL_F32, oracle_net

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X GPU")]


def _case(rng, n, h, w, P=8):
    """n variants: an 8x8 zero patch at a random corner, some with a second box."""
    boxes, off = [], [0]
    for i in range(n):
        y, x = int(rng.integers(-3, h - 4)), int(rng.integers(-3, w - 4))
        boxes.append((y, x, y + P, x + P))
        if i % 3 == 0:
            y2, x2 = int(rng.integers(0, h)), int(rng.integers(0, w))
            boxes.append((y2, x2, y2 + 3, x2 + 5))
        off.append(len(boxes))
    return np.asarray(boxes, np.int32), np.asarray(off, np.int32)


def test_static_scratch_variants_match_caller_scratch():
    import torch
    from paper_1909_05632_amd import ReuseNet
    wl = synth.WORKLOADS["occlusion-105x80-4096"]
    weights = synth.net_weights(wl, bias_std=0.05)
    base = synth.to_f32(synth.occlusion_base(wl))[None]              # [1][H][W]
    net = ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, 2, weights)
    net.full(torch.from_numpy(base[None]).cuda(), stream_ids=torch.tensor([1], dtype=torch.int32).cuda())
    zero = torch.zeros((1, 1, wl.h, wl.w), dtype=torch.float32).cuda()
    onet = oracle_net(wl)
    rng = np.random.default_rng(3)
    for n, max_tiles in ((1500, 16), (37, 0)):                        # the second call smaller
        boxes, off = _case(rng, n, wl.h, wl.w)
        db, do = torch.from_numpy(boxes).cuda(), torch.from_numpy(off).cuda()
        want = net.variants(1, db, do, zero, max_tiles=max_tiles).cpu().numpy()
        wl_want = [net.worklist(l) for l in (1, 2)]
        tm_want = [net.tile_mask_u8(2, i) for i in (0, n - 1)]
        got = net.variants_static(1, db, do, zero, max_tiles=max_tiles).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), f"n={n}"
        for l, w in zip((1, 2), wl_want):
            assert np.array_equal(net.worklist(l), w), f"n={n} layer {l}"
        for i, m in zip((0, n - 1), tm_want):
            assert np.array_equal(net.tile_mask_u8(2, i), m)
        # Variants over the tile limit are left out with NaN logits (the same
        # ones on both paths); the others against the oracle.
        finite = np.flatnonzero(np.isfinite(got).all(axis=1))
        assert len(finite) > n // 2
        pick = [int(finite[0]), int(finite[len(finite) // 2]), int(finite[-1])]
        xs = np.stack([oracle.variant_input(base, np.zeros_like(base), boxes[off[i]:off[i + 1]]) for i in pick])
        ref, _ = oracle.forward(onet, *weights, xs)
        assert np.abs(got[pick] - ref).max() <= ATOL_F32, f"n={n}"
    # Beyond the static limit (every tile of every layer for 65535 variants):
    # refused with RN_ENOSPACE, nothing launched.
    n = 65535
    assert B.reuse_net_variant_scratch_bytes(net.handle, n, 0) > B.RN_STATIC_SCRATCH_BYTES
    boxes = torch.zeros((1, 4), dtype=torch.int32).cuda()
    off = torch.zeros(n + 1, dtype=torch.int32).cuda()
    out = torch.empty((n, wl.n_out), dtype=torch.float32).cuda()
    with pytest.raises(B.ReuseNetError) as e:
        net.variants_static(1, boxes, off, zero, max_tiles=0, out=out)
    assert e.value.status == B.RN_ENOSPACE and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    net.close()
