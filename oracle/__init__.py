"""CPU oracle for frame-to-frame convolutional activation reuse.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg use it; the product library never does.  It shares no code
with the HIP path.  The arithmetic lives in ``oracle.c`` (plain C, double
accumulation); this module only marshals numpy arrays through ctypes and
composes the per-frame steps in the order the method takes them:

  change set (diff or boxes) -> per-layer growth -> tile masks -> work list
  -> full recompute of every layer -> dense head.

The reuse method must reach the full recompute's result exactly (Abstract;
Sec. 1), so the full recompute is the expected activations and logits.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
MAX_LAYERS = 8


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, OpenMP, no fast-math)."""
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


class _Net(ctypes.Structure):
    _fields_ = [("in_c", ctypes.c_int), ("h", ctypes.c_int), ("w", ctypes.c_int),
                ("n_conv", ctypes.c_int),
                ("cin", ctypes.c_int * MAX_LAYERS), ("cout", ctypes.c_int * MAX_LAYERS),
                ("k", ctypes.c_int * MAX_LAYERS), ("s", ctypes.c_int * MAX_LAYERS),
                ("p", ctypes.c_int * MAX_LAYERS),
                ("n_out", ctypes.c_int), ("tile_h", ctypes.c_int), ("tile_w", ctypes.c_int),
                ("bf16", ctypes.c_int)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        I = ctypes.c_int
        L.orc_level_to_f32.restype = ctypes.c_float
        L.orc_level_to_f32.argtypes = [ctypes.c_uint8]
        L.orc_levels_to_f32.argtypes = [P, ctypes.c_size_t, P]
        L.orc_bf16_rne.restype = ctypes.c_float
        L.orc_bf16_rne.argtypes = [ctypes.c_float]
        L.orc_bf16_rne_array.argtypes = [P, ctypes.c_size_t, P]
        L.orc_out_size.argtypes = [I, I, I, I]
        L.orc_diff.argtypes = [I, I, I, P, P, P]
        L.orc_box_mask.argtypes = [I, I, I, P, P]
        L.orc_dilate.argtypes = [I, I, P, I, I, I, P]
        L.orc_tile_mask.argtypes = [I, I, P, I, I, P]
        L.orc_worklist.argtypes = [I, I, I, P, P]
        L.orc_conv2d_relu.argtypes = [I, I, I, P, I, I, I, I, P, P, I, P]
        L.orc_conv2d_relu_tiles.argtypes = [I, I, I, P, I, I, I, I, P, P, I, P, I, I, P]
        L.orc_dense.argtypes = [I, P, I, P, P, P]
        L.orc_forward.argtypes = [ctypes.POINTER(_Net), P, P, P, P, I, P, P, P]
        L.orc_masks.argtypes = [ctypes.POINTER(_Net), I, P, P, P]
        L.orc_reuse_step.argtypes = [ctypes.POINTER(_Net), P, P, P, P, P, P, I, P, P]
        L.orc_reinforce_dlogits.argtypes = [I, I, P, P, P, P]
        L.orc_forward_preact.argtypes = [ctypes.POINTER(_Net), P, P, P, P]
        L.orc_backward.argtypes = [ctypes.POINTER(_Net), P, P, P, P, I, P, P, P, P, P, P]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _u8(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint8)


def _ptr_array(arrs):
    return (ctypes.c_void_p * len(arrs))(*[a.ctypes.data if a is not None else None for a in arrs])


# ------------------------------------------------------------ single ops

def level_to_f32(k: np.ndarray) -> np.ndarray:
    k = _u8(k)
    out = np.empty(k.shape, np.float32)
    lib().orc_levels_to_f32(_p(k), k.size, _p(out))
    return out


def bf16_rne(x: np.ndarray) -> np.ndarray:
    x = _f32(x)
    out = np.empty_like(x)
    lib().orc_bf16_rne_array(_p(x), x.size, _p(out))
    return out


def out_size(n: int, k: int, s: int, p: int) -> int:
    return lib().orc_out_size(n, k, s, p)


def diff(prev: np.ndarray, cur: np.ndarray) -> np.ndarray:
    """[C][H][W] x2 -> uint8 [H][W] change mask."""
    prev, cur = _f32(prev), _f32(cur)
    c, h, w = prev.shape
    d0 = np.empty((h, w), np.uint8)
    lib().orc_diff(c, h, w, _p(prev), _p(cur), _p(d0))
    return d0


def box_mask(h: int, w: int, boxes) -> np.ndarray:
    b = np.ascontiguousarray(np.asarray(boxes, dtype=np.int32).reshape(-1, 4))
    d0 = np.empty((h, w), np.uint8)
    lib().orc_box_mask(h, w, len(b), _p(b), _p(d0))
    return d0


def variant_input(base: np.ndarray, frame: np.ndarray, boxes) -> np.ndarray:
    """Input [C][H][W] of a known-change variant (Sec. 1, occlusion use): the
    base input with the pixels inside the boxes (half-open, clipped, union)
    taken from `frame`; every other pixel keeps the base value."""
    base = _f32(base)
    inside = box_mask(base.shape[1], base.shape[2], boxes).astype(bool)
    x = base.copy()
    x[:, inside] = _f32(frame)[:, inside]
    return x


def dilate(d: np.ndarray, k: int, s: int, p: int) -> np.ndarray:
    d = _u8(d)
    h, w = d.shape
    out = np.empty((out_size(h, k, s, p), out_size(w, k, s, p)), np.uint8)
    lib().orc_dilate(h, w, _p(d), k, s, p, _p(out))
    return out


def tile_mask(d: np.ndarray, tile_h: int, tile_w: int) -> np.ndarray:
    d = _u8(d)
    h, w = d.shape
    m = np.empty((-(-h // tile_h), -(-w // tile_w)), np.uint8)
    lib().orc_tile_mask(h, w, _p(d), tile_h, tile_w, _p(m))
    return m


def worklist(masks: np.ndarray) -> np.ndarray:
    """uint8 [n][th][tw] -> uint32 entries s<<16 | ty<<8 | tx in (ty, tx, s) order."""
    masks = _u8(masks)
    n, th, tw = masks.shape
    out = np.empty(max(1, masks.size), np.uint32)
    cnt = lib().orc_worklist(n, th, tw, _p(masks), _p(out))
    return out[:cnt].copy()


def conv2d_relu(x: np.ndarray, wt: np.ndarray, b: np.ndarray, stride: int = 1,
                pad: int | None = None, bf16: bool = False) -> np.ndarray:
    x, wt, b = _f32(x), _f32(wt), _f32(b)
    cin, h, w = x.shape
    cout, cin2, k, k2 = wt.shape
    assert cin == cin2 and k == k2
    p = (k - 1) // 2 if pad is None else pad
    y = np.empty((cout, out_size(h, k, stride, p), out_size(w, k, stride, p)), np.float32)
    lib().orc_conv2d_relu(cin, h, w, _p(x), cout, k, stride, p, _p(wt), _p(b), int(bf16), _p(y))
    return y


def conv2d_relu_tiles(x, wt, b, tmask, tile_h, tile_w, y_inout, stride=1, pad=None, bf16=False):
    x, wt, b, tmask = _f32(x), _f32(wt), _f32(b), _u8(tmask)
    assert y_inout.dtype == np.float32 and y_inout.flags.c_contiguous
    cin, h, w = x.shape
    cout, _, k, _ = wt.shape
    p = (k - 1) // 2 if pad is None else pad
    lib().orc_conv2d_relu_tiles(cin, h, w, _p(x), cout, k, stride, p, _p(wt), _p(b), int(bf16),
                                _p(tmask), tile_h, tile_w, _p(y_inout))
    return y_inout


def dense(a: np.ndarray, wd: np.ndarray, bd: np.ndarray) -> np.ndarray:
    a, wd, bd = _f32(a).reshape(-1), _f32(wd), _f32(bd)
    n, kdim = wd.shape
    assert a.size == kdim
    out = np.empty(n, np.float32)
    lib().orc_dense(kdim, _p(a), n, _p(wd), _p(bd), _p(out))
    return out


# ------------------------------------------------------------ networks

@dataclass
class Net:
    """Network description: input shape, conv stack (cin, cout, k, s, p), logits, tile."""

    in_c: int
    h: int
    w: int
    convs: Sequence[tuple]
    n_out: int
    tile_h: int = 4
    tile_w: int = 4
    bf16: bool = False

    def c_struct(self) -> _Net:
        s = _Net()
        s.in_c, s.h, s.w = self.in_c, self.h, self.w
        s.n_conv = len(self.convs)
        for i, (ci, co, k, st, p) in enumerate(self.convs):
            s.cin[i], s.cout[i], s.k[i], s.s[i], s.p[i] = ci, co, k, st, p
        s.n_out, s.tile_h, s.tile_w, s.bf16 = self.n_out, self.tile_h, self.tile_w, int(self.bf16)
        return s

    def layer_shape(self, l: int):
        c, h, w = self.in_c, self.h, self.w
        for (ci, co, k, st, p) in list(self.convs)[:l]:
            h, w, c = out_size(h, k, st, p), out_size(w, k, st, p), co
        return c, h, w

    def tile_grid(self, l: int):
        _, h, w = self.layer_shape(l)
        return -(-h // self.tile_h), -(-w // self.tile_w)


def forward(net: Net, conv_w, conv_b, dense_w, dense_b, x: np.ndarray, want_acts: bool = False):
    """Full recompute of n inputs x [n][in_c][h][w] -> (logits [n][n_out], acts or None)."""
    x = _f32(x)
    n = x.shape[0]
    cw = [_f32(w) for w in conv_w]
    cb = [_f32(b) for b in conv_b]
    dw, db = _f32(dense_w), _f32(dense_b)
    logits = np.empty((n, net.n_out), np.float32)
    acts = None
    if want_acts:
        acts = [np.empty((n,) + net.layer_shape(l + 1), np.float32) for l in range(len(net.convs))]
    st = net.c_struct()
    rc = lib().orc_forward(ctypes.byref(st), _ptr_array(cw), _ptr_array(cb), _p(dw), _p(db), n,
                           _p(x), _ptr_array(acts) if acts else None, _p(logits))
    if rc != 0:
        raise ValueError("oracle: bad net description")
    return logits, acts


def masks(net: Net, d0: np.ndarray, want_pixels: bool = True):
    """Change masks of one step for n streams.

    d0 uint8 [n][h][w] -> (pixel masks [L+1] of [n][H_l][W_l] or None,
                            tile masks [L+1] of [n][TH_l][TW_l])."""
    d0 = _u8(d0)
    n = d0.shape[0]
    L = len(net.convs)
    d = [np.empty((n,) + net.layer_shape(l)[1:], np.uint8) for l in range(L + 1)] \
        if want_pixels else None
    m = [np.empty((n,) + net.tile_grid(l), np.uint8) for l in range(L + 1)]
    st = net.c_struct()
    rc = lib().orc_masks(ctypes.byref(st), n, _p(d0), _ptr_array(d) if d else None, _ptr_array(m))
    if rc != 0:
        raise ValueError("oracle: bad net description")
    return d, m


def worklists(tile_masks) -> list:
    """Work lists of layers 1..L from the tile masks of one step (index 0 unused -> None)."""
    return [None] + [worklist(m) for m in tile_masks[1:]]


class ReuseStream:
    """Plain reuse of one stream, kept on the CPU (Sec. 1): the caches hold the
    previous frame's activations and each step recomputes only dirty tiles.
    Used to check that recomputing on the dirty tiles alone reproduces the full
    recompute bit for bit."""

    def __init__(self, net: Net, conv_w, conv_b, dense_w, dense_b):
        self.net = net
        self.st = net.c_struct()
        if net.bf16:
            conv_w = [bf16_rne(w) for w in conv_w]
            dense_w = bf16_rne(dense_w)
        self.cw = [_f32(w) for w in conv_w]
        self.cb = [_f32(b) for b in conv_b]
        self.dw, self.db = _f32(dense_w), _f32(dense_b)
        self.cache = [np.zeros(net.layer_shape(l), np.float32) for l in range(len(net.convs) + 1)]
        self.primed = False

    def reset(self):
        self.primed = False

    def step(self, x: np.ndarray, d0: np.ndarray | None = None) -> np.ndarray:
        x = _f32(x)
        logits = np.empty(self.net.n_out, np.float32)
        rc = lib().orc_reuse_step(ctypes.byref(self.st), _ptr_array(self.cw), _ptr_array(self.cb),
                                  _p(self.dw), _p(self.db), _p(x),
                                  _p(_u8(d0)) if d0 is not None else None, int(self.primed),
                                  _ptr_array(self.cache), _p(logits))
        if rc != 0:
            raise ValueError("oracle: bad net description")
        self.primed = True
        return logits


# ------------------------------------------------------------ training

def reinforce_dlogits(logits: np.ndarray, actions: np.ndarray, returns: np.ndarray) -> np.ndarray:
    """dJ/dlogits [n][n_out] of the REINFORCE loss (Sec. 2) J = sum_i -G_i log softmax(z_i)[a_i]."""
    z = _f32(logits)
    n, n_out = z.shape
    a = np.ascontiguousarray(actions, dtype=np.int32)
    g = _f32(returns)
    out = np.empty((n, n_out), np.float32)
    lib().orc_reinforce_dlogits(n, n_out, _p(z), _p(a), _p(g), _p(out))
    return out


def forward_preact(net: Net, conv_w, conv_b, x: np.ndarray) -> list:
    """Pre-activations (before the ReLU) of every layer for one input x [in_c][h][w]."""
    x = _f32(x)
    cw = [_f32(w) for w in conv_w]
    cb = [_f32(b) for b in conv_b]
    z = [np.empty(net.layer_shape(l + 1), np.float32) for l in range(len(net.convs))]
    rc = lib().orc_forward_preact(ctypes.byref(net.c_struct()), _ptr_array(cw), _ptr_array(cb), _p(x),
                                  _ptr_array(z))
    if rc != 0:
        raise ValueError("oracle: bad net description (float32 nets only)")
    return z


def backward(net: Net, conv_w, conv_b, dense_w, dense_b, x: np.ndarray, g: np.ndarray):
    """Gradients of sum_i sum_o g[i][o] logits[i][o] over n inputs x [n][in_c][h][w]
    -> (dconv_w list OIHW, dconv_b list, ddense_w [n_out][C_L H_L W_L], ddense_b)."""
    x, g = _f32(x), _f32(g)
    n = x.shape[0]
    assert g.shape == (n, net.n_out)
    cw = [_f32(w) for w in conv_w]
    cb = [_f32(b) for b in conv_b]
    dw, db = _f32(dense_w), _f32(dense_b)
    gw = [np.empty_like(w) for w in cw]
    gb = [np.empty_like(b) for b in cb]
    gdw, gdb = np.empty_like(dw), np.empty_like(db)
    rc = lib().orc_backward(ctypes.byref(net.c_struct()), _ptr_array(cw), _ptr_array(cb), _p(dw), _p(db),
                            n, _p(x), _p(g), _ptr_array(gw), _ptr_array(gb), _p(gdw), _p(gdb))
    if rc != 0:
        raise ValueError("oracle: bad net description (float32 nets only)")
    return gw, gb, gdw, gdb
