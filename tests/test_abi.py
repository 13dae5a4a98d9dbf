"""The C-ABI library loads, exports every declared entry point, and rejects bad
arguments with status codes (host-side validation only: no GPU needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_1909_05632_amd as pkg
from paper_1909_05632_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "reuse_net.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(reuse_net_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(B.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = pkg.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def _cfg(convs=((1, 40), (40, 80)), h=105, w=80, stack=1, n_out=6, tile=4, streams=8,
         k=3, s=1, p=1, dtype=B.RN_F32, in_c=1, head=B.RN_HEAD_TILES, options=0):
    specs = (B.rn_conv_spec * len(convs))(*[B.rn_conv_spec(ci, co, k, s, p) for ci, co in convs])
    cfg = B.rn_config(in_c, h, w, stack, len(convs), specs, n_out, tile, tile, streams, dtype, head,
                      options)
    cfg._keep = specs
    return cfg


def test_head_modes_size_the_workspace():
    tiles = B.reuse_net_workspace_bytes(_cfg(head=B.RN_HEAD_TILES))
    full = B.reuse_net_workspace_bytes(_cfg(head=B.RN_HEAD_FULL))
    assert tiles > 0 and full > 0 and tiles != full
    assert B.reuse_net_workspace_bytes(_cfg(head=7)) == 0


def test_bf16_configs():
    full = ((1, 64), (64, 128), (128, 128))
    assert B.reuse_net_workspace_bytes(_cfg(full, h=210, w=160, n_out=18, dtype=B.RN_BF16)) > 0
    # bf16 caches are half the size of float32 ones.
    f32 = B.reuse_net_workspace_bytes(_cfg(full, h=210, w=160, n_out=18, streams=64))
    b16 = B.reuse_net_workspace_bytes(_cfg(full, h=210, w=160, n_out=18, streams=64, dtype=B.RN_BF16))
    assert b16 < 0.6 * f32
    # 40 input channels have no bf16 MFMA kernel (K blocks of 32 channels).
    assert B.reuse_net_workspace_bytes(_cfg(dtype=B.RN_BF16)) == 0
    st, h, msg = _create(_cfg(dtype=B.RN_BF16))
    assert st == B.RN_EUNSUPPORTED and "bf16" in msg


def test_separate_first_layer_option_is_accepted():
    assert B.reuse_net_workspace_bytes(_cfg(options=B.RN_OPT_SEPARATE_FIRST)) > 0


def test_workspace_bytes_valid_configs():
    n1 = B.reuse_net_workspace_bytes(_cfg(streams=1))
    n8 = B.reuse_net_workspace_bytes(_cfg(streams=8))
    assert n1 > 0 and n8 > n1
    # The caches dominate: 8 streams of 105x80 fp32 caches at 40 + 80 channels.
    assert n8 > 8 * (27 * 20 * 16) * 120 * 4
    assert B.reuse_net_workspace_bytes(_cfg(((4, 40), (40, 80)), stack=4)) > 0
    assert B.reuse_net_workspace_bytes(
        _cfg(((1, 64), (64, 128), (128, 128)), h=210, w=160, n_out=18)) > 0


def test_general_layer_configs():
    # DQN-style trunk: 8x8 stride 4, 4x4 stride 2, 3x3 stride 1, no padding, 4 stacked frames.
    specs = (B.rn_conv_spec * 3)(B.rn_conv_spec(4, 32, 8, 4, 0), B.rn_conv_spec(32, 64, 4, 2, 0),
                                 B.rn_conv_spec(64, 64, 3, 1, 0))
    def cfg(dtype=B.RN_F32, spec=specs, h=84, w=84):
        c = B.rn_config(1, h, w, 4, 3, spec, 6, 4, 4, 8, dtype, B.RN_HEAD_TILES, 0)
        c._keep = spec
        return c
    n = B.reuse_net_workspace_bytes(cfg())
    # the caches follow the shrinking grids: 20x20x32 + 9x9x64 + 7x7x64 (tiled) per stream
    assert n > 8 * (25 * 16 * 32 + 9 * 16 * 64 + 4 * 16 * 64) * 4
    assert B.reuse_net_workspace_bytes(cfg(B.RN_BF16)) == 0             # general layers: float32 only
    bad = (B.rn_conv_spec * 3)(B.rn_conv_spec(4, 32, 8, 3, 0), B.rn_conv_spec(32, 64, 4, 2, 0),
                               B.rn_conv_spec(64, 64, 3, 1, 0))
    assert B.reuse_net_workspace_bytes(cfg(spec=bad)) == 0              # stride 3
    assert B.reuse_net_workspace_bytes(cfg(h=12, w=12)) == 0            # no output pixels left


def test_frame_size_limit_of_the_mask_kernel():
    # Two bit planes of the frame in LDS: 640 x 448 (4480 words, more than the
    # default 64 KiB of dynamic LDS) is accepted, 1024 x 1024 is not.
    assert B.reuse_net_workspace_bytes(_cfg(h=640, w=448, streams=1)) > 0
    assert B.reuse_net_workspace_bytes(_cfg(h=1024, w=1024, streams=1)) == 0


@pytest.mark.parametrize("bad", [
    dict(k=2, p=0),                   # 2x2 kernel: no kernel for these shapes
    dict(p=0),                        # 3x3 without padding: no kernel for 1->40
    dict(p=2),                        # pad > (k-1)/2
    dict(s=0),                        # stride 0
    dict(convs=((1, 40), (32, 80))),  # broken channel chain
    dict(convs=()),                   # no layers
    dict(stack=3),
    dict(streams=0),
    dict(n_out=0),
    dict(tile=8),                     # valid but unsupported tile
    dict(w=78),                       # width not a multiple of 4
    dict(k=5, p=2),                   # valid but unsupported kernel size
    dict(convs=((1, 40), (40, 72))),  # no MFMA kernel for this shape
    dict(convs=((1, 20), (20, 40))),  # 40 output channels: not a multiple of 16
    dict(options=6),                  # unknown option bits
])
def test_workspace_bytes_rejects_bad_configs(bad):
    assert B.reuse_net_workspace_bytes(_cfg(**bad)) == 0


def _create(cfg, weights=True, ptr=256, nbytes=None):
    lib = pkg.load_library()
    h = ctypes.c_void_p()
    keep = []
    w = None
    if weights:
        L = cfg.n_conv
        arrs = [np.zeros(1 << 16, np.float32) for _ in range(2 * L + 2)]
        keep.append(arrs)
        cw = (ctypes.c_void_p * max(L, 1))(*[a.ctypes.data for a in arrs[:L]])
        cb = (ctypes.c_void_p * max(L, 1))(*[a.ctypes.data for a in arrs[L:2 * L]])
        w = B.rn_weights(cw, cb, arrs[-2].ctypes.data, arrs[-1].ctypes.data)
        keep += [cw, cb]
    need = B.reuse_net_workspace_bytes(cfg)
    st = lib.reuse_net_create(ctypes.byref(cfg), ctypes.byref(w) if w else None, ptr,
                              need if nbytes is None else nbytes, None, ctypes.byref(h))
    return st, h.value, B.reuse_net_last_error(None)


def test_create_reports_argument_errors_without_touching_the_gpu():
    st, h, msg = _create(_cfg(p=2))
    assert st == B.RN_EINVAL and h is None and "pad" in msg
    st, h, msg = _create(_cfg(k=2, p=0))
    assert st == B.RN_EUNSUPPORTED and h is None and "kernel" in msg
    st, h, msg = _create(_cfg(tile=8))
    assert st == B.RN_EUNSUPPORTED and "tile" in msg
    st, h, msg = _create(_cfg(h=1024, w=1024))
    assert st == B.RN_EUNSUPPORTED and "frame too large" in msg
    st, h, msg = _create(_cfg(), weights=False)
    assert st == B.RN_EINVAL and "weights" in msg
    st, h, msg = _create(_cfg(), nbytes=1024)
    assert st == B.RN_ENOSPACE and "too small" in msg
    st, h, msg = _create(_cfg(), ptr=256 + 4)
    assert st == B.RN_EINVAL and "aligned" in msg
    st, h, msg = _create(_cfg(), ptr=None)
    assert st == B.RN_EINVAL
    lib = pkg.load_library()
    assert lib.reuse_net_create(None, None, None, 0, None, None) == B.RN_EINVAL


def test_null_net_calls_return_einval():
    lib = pkg.load_library()
    assert lib.reuse_net_step(None, 1, None, None, 0, None, None, None, None) == B.RN_EINVAL
    assert lib.reuse_net_full(None, 1, None, None, 0, None, None) == B.RN_EINVAL
    assert lib.reuse_net_reset(None, -1) == B.RN_EINVAL
    assert lib.reuse_net_get_stats(None, None) == B.RN_EINVAL
    assert lib.reuse_net_get_profile(None, None) == B.RN_EINVAL
    assert lib.reuse_net_set_weights(None, None, None) == B.RN_EINVAL
    assert lib.reuse_net_set_weights_device(None, None, None) == B.RN_EINVAL
    assert lib.reuse_net_sgd_step(None, None, 0.0, None) == B.RN_EINVAL
    assert lib.reuse_net_variant_scratch_bytes(None, 4, 0) == 0
    assert lib.reuse_net_variants(None, 0, 4, None, 0, 1, None, None, 0, None, 0, None, None) == B.RN_EINVAL
    lib.reuse_net_destroy(None)


def _bare_net(in_c=1, h=16, w=12, n_out=6, max_streams=8):
    """A ReuseNet shell with the fields the binding's argument checks read, on
    the CPU device (no library handle: every case below must fail before a
    call reaches the library)."""
    import torch
    net = B.ReuseNet.__new__(B.ReuseNet)
    net.torch = torch
    net.device = torch.device("cpu")
    net.in_c, net.h, net.w, net.n_out, net.max_streams = in_c, h, w, n_out, max_streams
    net.handle = None
    return net


def test_binding_rejects_bad_tensors_before_any_launch():
    import torch
    net = _bare_net()
    f = torch.zeros((3, 1, 16, 12), dtype=torch.float32)
    ok_ids = torch.arange(3, dtype=torch.int32)
    ok_out = torch.zeros((3, 6), dtype=torch.float32)
    bad = [
        # int64 ids (torch's default integer) would be read as int32 pairs
        dict(stream_ids=torch.arange(3)),
        dict(stream_ids=torch.arange(4, dtype=torch.int32)),                 # wrong length
        dict(stream_ids=torch.arange(6, dtype=torch.int32)[::2]),            # not contiguous
        dict(out=torch.zeros((3, 5), dtype=torch.float32)),                  # undersized logits
        dict(out=torch.zeros((3, 6), dtype=torch.float64)),
        dict(out=torch.zeros((6, 3), dtype=torch.float32).t()),              # not contiguous
        dict(boxes=torch.zeros((2, 4), dtype=torch.int64), box_off=torch.tensor([0, 1, 2, 2], dtype=torch.int32)),
        dict(boxes=torch.zeros((2, 4), dtype=torch.int32), box_off=torch.tensor([0, 1, 2], dtype=torch.int32)),
        dict(boxes=torch.zeros((2, 3), dtype=torch.int32), box_off=torch.tensor([0, 1, 2, 2], dtype=torch.int32)),
        dict(boxes=torch.zeros((2, 4), dtype=torch.int32)),                  # boxes without offsets
    ]
    for kw in bad:
        args = dict(stream_ids=ok_ids, out=ok_out)
        args.update(kw)
        with pytest.raises((TypeError, ValueError)):
            net.step(f, **args)
    for frames in (torch.zeros((3, 1, 16, 8)),                                # wrong frame shape
                   torch.zeros((3, 2, 16, 12)),                               # wrong channel count
                   torch.zeros((3, 16, 12)),                                  # missing channel axis
                   torch.zeros((3, 1, 16, 12), dtype=torch.float16),          # unsupported dtype
                   torch.zeros((9, 1, 16, 12)),                               # more streams than slots
                   torch.zeros((3, 1, 12, 16)).transpose(2, 3)):              # not contiguous
        with pytest.raises((TypeError, ValueError)):
            net.step(frames)
        with pytest.raises((TypeError, ValueError)):
            net.full(frames)
    # variants: 1 or n frames, int32 boxes and n + 1 offsets
    boxes = torch.zeros((2, 4), dtype=torch.int32)
    off = torch.tensor([0, 1, 2], dtype=torch.int32)
    with pytest.raises(ValueError):
        net.variants(0, boxes, off, torch.zeros((3, 1, 16, 12)))
    with pytest.raises((TypeError, ValueError)):
        net.variants(0, boxes, off.long(), torch.zeros((1, 1, 16, 12)))
    with pytest.raises((TypeError, ValueError)):
        net.variants(0, boxes, off, torch.zeros((2, 1, 16, 12)), out=torch.zeros((2, 5)))
