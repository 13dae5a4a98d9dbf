"""ctypes binding of libreuse_net.so (include/reuse_net.h).

The module-level functions carry the C names and only marshal arguments:
every step of the reuse path runs in the library's HIP kernels.  ``ReuseNet``
is a convenience wrapper that uses torch for device memory and streams.
There is no fallback: if the library is not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libreuse_net.so")

RN_MAX_CONV = 8
RN_PHASES = 9
RN_OK, RN_EINVAL, RN_EUNSUPPORTED, RN_ENOSPACE, RN_EHIP, RN_ESTATE = 0, -1, -2, -3, -4, -5
RN_F32, RN_BF16, RN_U8 = 0, 1, 2
RN_HEAD_TILES, RN_HEAD_FULL = 0, 1
RN_OPT_SEPARATE_FIRST = 1
PHASES = ("masks", "compact", "conv1", "convN", "head", "bwd_head", "bwd_dw", "bwd_dx", "sgd")
STATUS_NAMES = {0: "RN_OK", -1: "RN_EINVAL", -2: "RN_EUNSUPPORTED", -3: "RN_ENOSPACE",
                -4: "RN_EHIP", -5: "RN_ESTATE"}

# Every entry point include/reuse_net.h declares.
EXPORTS = (
    "reuse_net_workspace_bytes", "reuse_net_create", "reuse_net_step", "reuse_net_full",
    "reuse_net_reset", "reuse_net_get_pixel_mask", "reuse_net_get_tile_mask",
    "reuse_net_get_worklist", "reuse_net_read_activation", "reuse_net_get_stats",
    "reuse_net_set_profiling", "reuse_net_get_profile", "reuse_net_last_error",
    "reuse_net_destroy", "reuse_net_variant_scratch_bytes", "reuse_net_variants",
    "reuse_net_set_weights", "reuse_net_variants_static", "reuse_net_grad_elems",
    "reuse_net_backward_scratch_bytes", "reuse_net_reinforce_dlogits", "reuse_net_backward",
    "reuse_net_sgd_step", "reuse_net_set_weights_device",
)
RN_STATIC_SCRATCH_BYTES = 64 << 20


class rn_conv_spec(ctypes.Structure):
    _fields_ = [("cin", ctypes.c_int32), ("cout", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32)]


class rn_config(ctypes.Structure):
    _fields_ = [("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32), ("in_w", ctypes.c_int32),
                ("stack", ctypes.c_int32), ("n_conv", ctypes.c_int32),
                ("conv", ctypes.POINTER(rn_conv_spec)), ("n_out", ctypes.c_int32),
                ("tile_h", ctypes.c_int32), ("tile_w", ctypes.c_int32),
                ("max_streams", ctypes.c_int32), ("act_dtype", ctypes.c_int),
                ("head_mode", ctypes.c_int), ("options", ctypes.c_int32)]


class rn_weights(ctypes.Structure):
    _fields_ = [("conv_w", ctypes.POINTER(ctypes.c_void_p)),
                ("conv_b", ctypes.POINTER(ctypes.c_void_p)),
                ("dense_w", ctypes.c_void_p), ("dense_b", ctypes.c_void_p)]


class rn_stats(ctypes.Structure):
    _fields_ = [("streams", ctypes.c_int64), ("changed_px", ctypes.c_int64),
                ("dirty_tiles", ctypes.c_int64 * (RN_MAX_CONV + 1)),
                ("useful_mac", ctypes.c_int64), ("issued_mac", ctypes.c_int64),
                ("dense_mac", ctypes.c_int64)]


class rn_profile(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * RN_PHASES), ("launches", ctypes.c_int64 * RN_PHASES),
                ("layer_ms", ctypes.c_double * (RN_MAX_CONV + 1)),
                ("layer_launches", ctypes.c_int64 * (RN_MAX_CONV + 1))]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the HIP library and declare the C signatures.  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_1909_05632_amd.build`")
    L = ctypes.CDLL(path)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    st = ctypes.c_int
    L.reuse_net_workspace_bytes.restype = SZ
    L.reuse_net_workspace_bytes.argtypes = [ctypes.POINTER(rn_config)]
    L.reuse_net_create.restype = st
    L.reuse_net_create.argtypes = [ctypes.POINTER(rn_config), ctypes.POINTER(rn_weights), P, SZ, P,
                                   ctypes.POINTER(P)]
    L.reuse_net_step.restype = st
    L.reuse_net_step.argtypes = [P, I32, P, P, ctypes.c_int, P, P, P, P]
    L.reuse_net_full.restype = st
    L.reuse_net_full.argtypes = [P, I32, P, P, ctypes.c_int, P, P]
    L.reuse_net_reset.restype = st
    L.reuse_net_reset.argtypes = [P, I32]
    L.reuse_net_set_weights.restype = st
    L.reuse_net_set_weights.argtypes = [P, ctypes.POINTER(rn_weights), P]
    L.reuse_net_variant_scratch_bytes.restype = SZ
    L.reuse_net_variant_scratch_bytes.argtypes = [P, I32, I32]
    L.reuse_net_variants.restype = st
    L.reuse_net_variants.argtypes = [P, I32, I32, P, ctypes.c_int, I32, P, P, I32, P, SZ, P, P]
    L.reuse_net_grad_elems.restype = SZ
    L.reuse_net_grad_elems.argtypes = [P]
    L.reuse_net_backward_scratch_bytes.restype = SZ
    L.reuse_net_backward_scratch_bytes.argtypes = [P, I32]
    L.reuse_net_reinforce_dlogits.restype = st
    L.reuse_net_reinforce_dlogits.argtypes = [I32, I32, P, P, P, P, P]
    L.reuse_net_backward.restype = st
    L.reuse_net_backward.argtypes = [P, I32, P, P, P, I32, P, SZ, P]
    L.reuse_net_sgd_step.restype = st
    L.reuse_net_sgd_step.argtypes = [P, P, ctypes.c_float, P]
    L.reuse_net_set_weights_device.restype = st
    L.reuse_net_set_weights_device.argtypes = [P, P, P]
    L.reuse_net_variants_static.restype = st
    L.reuse_net_variants_static.argtypes = [P, I32, I32, P, ctypes.c_int, I32, P, P, I32, P, P]
    for name in ("reuse_net_get_pixel_mask", "reuse_net_get_tile_mask"):
        getattr(L, name).restype = st
        getattr(L, name).argtypes = [P, I32, I32, P, SZ]
    L.reuse_net_get_worklist.restype = st
    L.reuse_net_get_worklist.argtypes = [P, I32, P, SZ, ctypes.POINTER(I32)]
    L.reuse_net_read_activation.restype = st
    L.reuse_net_read_activation.argtypes = [P, I32, I32, P]
    L.reuse_net_get_stats.restype = st
    L.reuse_net_get_stats.argtypes = [P, ctypes.POINTER(rn_stats)]
    L.reuse_net_set_profiling.restype = st
    L.reuse_net_set_profiling.argtypes = [P, I32]
    L.reuse_net_get_profile.restype = st
    L.reuse_net_get_profile.argtypes = [P, ctypes.POINTER(rn_profile)]
    L.reuse_net_last_error.restype = ctypes.c_char_p
    L.reuse_net_last_error.argtypes = [P]
    L.reuse_net_destroy.restype = None
    L.reuse_net_destroy.argtypes = [P]
    _lib = L
    return L


class ReuseNetError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _check(status: int, net_handle=None):
    if status != RN_OK:
        msg = load_library().reuse_net_last_error(net_handle).decode()
        raise ReuseNetError(status, msg)


# ------------------------------------------------------- C-named wrappers

def reuse_net_workspace_bytes(cfg: rn_config) -> int:
    return load_library().reuse_net_workspace_bytes(ctypes.byref(cfg))


def reuse_net_create(cfg: rn_config, weights: rn_weights, dev_workspace: int, nbytes: int,
                     hip_stream: int) -> int:
    h = ctypes.c_void_p()
    _check(load_library().reuse_net_create(ctypes.byref(cfg), ctypes.byref(weights), dev_workspace,
                                           nbytes, hip_stream, ctypes.byref(h)))
    return h.value


def reuse_net_step(net: int, n: int, dev_stream_ids: int, dev_frames: int, frame_dtype: int,
                   dev_boxes: int, dev_box_off: int, dev_logits: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_step(net, n, dev_stream_ids, dev_frames, frame_dtype, dev_boxes,
                                         dev_box_off, dev_logits, hip_stream), net)


def reuse_net_full(net: int, n: int, dev_stream_ids: int, dev_frames: int, frame_dtype: int,
                   dev_logits: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_full(net, n, dev_stream_ids, dev_frames, frame_dtype,
                                         dev_logits, hip_stream), net)


def reuse_net_reset(net: int, stream_id: int) -> None:
    _check(load_library().reuse_net_reset(net, stream_id), net)


def reuse_net_set_weights(net: int, weights: rn_weights, hip_stream: int) -> None:
    _check(load_library().reuse_net_set_weights(net, ctypes.byref(weights), hip_stream), net)


def reuse_net_variant_scratch_bytes(net: int, n: int, max_tiles: int) -> int:
    return load_library().reuse_net_variant_scratch_bytes(net, n, max_tiles)


def reuse_net_variants(net: int, base_stream: int, n: int, dev_frames: int, frame_dtype: int,
                       frame_count: int, dev_boxes: int, dev_box_off: int, max_tiles: int,
                       dev_scratch: int, scratch_bytes: int, dev_logits: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_variants(net, base_stream, n, dev_frames, frame_dtype, frame_count,
                                             dev_boxes, dev_box_off, max_tiles, dev_scratch,
                                             scratch_bytes, dev_logits, hip_stream), net)


def reuse_net_variants_static(net: int, base_stream: int, n: int, dev_frames: int, frame_dtype: int,
                              frame_count: int, dev_boxes: int, dev_box_off: int, max_tiles: int,
                              dev_logits: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_variants_static(net, base_stream, n, dev_frames, frame_dtype, frame_count,
                                                    dev_boxes, dev_box_off, max_tiles, dev_logits, hip_stream),
           net)


def reuse_net_grad_elems(net: int) -> int:
    return load_library().reuse_net_grad_elems(net)


def reuse_net_backward_scratch_bytes(net: int, n: int) -> int:
    return load_library().reuse_net_backward_scratch_bytes(net, n)


def reuse_net_reinforce_dlogits(n: int, n_out: int, dev_logits: int, dev_actions: int, dev_returns: int,
                                dev_dlogits: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_reinforce_dlogits(n, n_out, dev_logits, dev_actions, dev_returns,
                                                      dev_dlogits, hip_stream))


def reuse_net_backward(net: int, n: int, dev_stream_ids: int, dev_dlogits: int, dev_grads: int,
                       accumulate: bool, dev_scratch: int, scratch_bytes: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_backward(net, n, dev_stream_ids, dev_dlogits, dev_grads, int(accumulate),
                                             dev_scratch, scratch_bytes, hip_stream), net)


def reuse_net_sgd_step(net: int, dev_grads: int, lr: float, hip_stream: int) -> None:
    _check(load_library().reuse_net_sgd_step(net, dev_grads, lr, hip_stream), net)


def reuse_net_set_weights_device(net: int, dev_params: int, hip_stream: int) -> None:
    _check(load_library().reuse_net_set_weights_device(net, dev_params, hip_stream), net)


def reuse_net_get_pixel_mask(net: int, layer: int, stream_id: int, words: int) -> np.ndarray:
    out = np.zeros(words, np.uint64)
    _check(load_library().reuse_net_get_pixel_mask(net, layer, stream_id, out.ctypes.data, words), net)
    return out


def reuse_net_get_tile_mask(net: int, layer: int, stream_id: int, words: int) -> np.ndarray:
    out = np.zeros(words, np.uint64)
    _check(load_library().reuse_net_get_tile_mask(net, layer, stream_id, out.ctypes.data, words), net)
    return out


def reuse_net_get_worklist(net: int, layer: int, cap: int) -> np.ndarray:
    out = np.zeros(max(cap, 1), np.uint32)
    cnt = ctypes.c_int32()
    _check(load_library().reuse_net_get_worklist(net, layer, out.ctypes.data, cap, ctypes.byref(cnt)), net)
    return out[:cnt.value].copy()


def reuse_net_read_activation(net: int, stream_id: int, layer: int, shape) -> np.ndarray:
    out = np.zeros(shape, np.float32)
    _check(load_library().reuse_net_read_activation(net, stream_id, layer, out.ctypes.data), net)
    return out


def reuse_net_get_stats(net: int) -> dict:
    s = rn_stats()
    _check(load_library().reuse_net_get_stats(net, ctypes.byref(s)), net)
    return {"streams": s.streams, "changed_px": s.changed_px, "dirty_tiles": list(s.dirty_tiles),
            "useful_mac": s.useful_mac, "issued_mac": s.issued_mac, "dense_mac": s.dense_mac}


def reuse_net_set_profiling(net: int, enable: bool) -> None:
    _check(load_library().reuse_net_set_profiling(net, int(enable)), net)


def reuse_net_get_profile(net: int) -> dict:
    p = rn_profile()
    _check(load_library().reuse_net_get_profile(net, ctypes.byref(p)), net)
    out = {name: {"ms": p.ms[i], "launches": p.launches[i]} for i, name in enumerate(PHASES)}
    out["layers"] = [{"ms": p.layer_ms[l], "launches": p.layer_launches[l]} for l in range(RN_MAX_CONV + 1)]
    return out


def reuse_net_last_error(net: Optional[int]) -> str:
    return load_library().reuse_net_last_error(net).decode()


def reuse_net_destroy(net: int) -> None:
    load_library().reuse_net_destroy(net)


# ------------------------------------------------------- torch convenience

def _dtype_code(name: str) -> int:
    return {"f32": RN_F32, "fp32": RN_F32, "float32": RN_F32, "bf16": RN_BF16,
            "bfloat16": RN_BF16}[name]


class ReuseNet:
    """One reuse net on a CUDA (HIP) device, workspace held in a torch tensor.

    convs: per layer either an output channel count (3x3, stride 1, pad 1) or a
    tuple (cout, k, stride, pad).
    weights: (conv_w list of OIHW float32, conv_b list, dense_w [n_out][C_L*H*W], dense_b).
    """

    def __init__(self, in_c: int, h: int, w: int, convs: Sequence[int], n_out: int,
                 max_streams: int, weights, act_dtype: str = "f32", stack: int = 1,
                 device="cuda", tile: int = 4, head: str = "tiles", fuse_first: bool = True):
        import torch
        self.torch = torch
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev                         # with its index: tensors are compared against it
        self.in_c, self.h, self.w, self.stack = in_c, h, w, stack
        self.convs = list(convs)
        self.n_out, self.max_streams = n_out, max_streams
        specs = []
        c = in_c * stack
        self.grids = [(h, w)]                     # output grid of each layer (0: the input)
        for co in self.convs:
            cout, k, st, pd = (tuple(co) if isinstance(co, (tuple, list)) else (co, 3, 1, 1))
            specs.append((c, cout, k, st, pd))
            gh, gw = self.grids[-1]
            self.grids.append((max(0, (gh + 2 * pd - k) // st + 1), max(0, (gw + 2 * pd - k) // st + 1)))
            c = cout
        self.specs = specs
        self.channels = [in_c] + [sp[1] for sp in specs]
        self._spec_arr = (rn_conv_spec * len(specs))(*[rn_conv_spec(*s) for s in specs])
        self.cfg = rn_config(in_c, h, w, stack, len(specs), self._spec_arr, n_out, tile, tile,
                             max_streams, _dtype_code(act_dtype),
                             {"tiles": RN_HEAD_TILES, "full": RN_HEAD_FULL}[head],
                             0 if fuse_first else RN_OPT_SEPARATE_FIRST)
        nbytes = reuse_net_workspace_bytes(self.cfg)
        if nbytes == 0:
            # Re-run create's validation to report why.
            _check(load_library().reuse_net_create(ctypes.byref(self.cfg), None, None, 0, None,
                                                   ctypes.byref(ctypes.c_void_p())))
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        keep, wts = self._weights(weights)
        stream = torch.cuda.current_stream(self.device).cuda_stream
        self.handle = reuse_net_create(self.cfg, wts, self.workspace.data_ptr(), nbytes, stream)
        del keep
        self.words_per_row = -(-w // 64)
        self.tiles = (-(-h // tile), -(-w // tile))
        self.tile_words = -(-(self.tiles[0] * self.tiles[1]) // 64)
        self.layer_tiles = [(-(-gh // tile), -(-gw // tile)) for gh, gw in self.grids]

    def _weights(self, weights):
        """rn_weights over contiguous float32 host copies (kept alive by the returned list)."""
        conv_w, conv_b, dense_w, dense_b = weights
        host = [np.ascontiguousarray(a, dtype=np.float32) for a in (*conv_w, *conv_b, dense_w, dense_b)]
        L = len(self.specs)
        cw = (ctypes.c_void_p * L)(*[a.ctypes.data for a in host[:L]])
        cb = (ctypes.c_void_p * L)(*[a.ctypes.data for a in host[L:2 * L]])
        return [host, cw, cb], rn_weights(cw, cb, host[2 * L].ctypes.data, host[2 * L + 1].ctypes.data)

    def set_weights(self, weights, stream=None):
        """New weights (same shapes); every slot recomputes everything on its next step."""
        keep, wts = self._weights(weights)
        s = (stream or self.torch.cuda.current_stream(self.device)).cuda_stream
        reuse_net_set_weights(self.handle, wts, s)
        del keep

    # -- hot path
    # Every tensor handed to the library is checked here, before any launch:
    # the C ABI takes raw pointers and sizes, so a wrong dtype, device, layout
    # or length would otherwise be read or written out of bounds on the GPU.
    def _check_dev(self, x, what: str, dtype, shape):
        t = self.torch
        if not isinstance(x, t.Tensor):
            raise TypeError(f"{what} must be a torch tensor")
        if x.dtype != dtype:
            raise TypeError(f"{what} must be {dtype}, got {x.dtype}")
        if x.device != self.device:
            raise ValueError(f"{what} must be on {self.device}, got {x.device}")
        if not x.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        if tuple(x.shape) != tuple(shape):
            raise ValueError(f"{what} must have shape {tuple(shape)}, got {tuple(x.shape)}")
        return x

    def _frames(self, frames):
        """(frames, dtype code); frames [n][in_c][h][w] uint8 or float32 on the net's device."""
        t = self.torch
        if not isinstance(frames, t.Tensor):
            raise TypeError("frames must be a torch tensor")
        if frames.dtype == t.uint8:
            code = RN_U8
        elif frames.dtype == t.float32:
            code = RN_F32
        else:
            raise TypeError("frames must be uint8 or float32")
        if frames.dim() != 4 or tuple(frames.shape[1:]) != (self.in_c, self.h, self.w):
            raise ValueError(f"frames must have shape (n, {self.in_c}, {self.h}, {self.w}), "
                             f"got {tuple(frames.shape)}")
        self._check_dev(frames, "frames", frames.dtype, (frames.shape[0], self.in_c, self.h, self.w))
        return frames, code

    def _batch(self, frames, stream_ids, out):
        """Checked batch size, id pointer and logits tensor of a step or full call."""
        t = self.torch
        frames, code = self._frames(frames)
        n = frames.shape[0]
        if not 1 <= n <= self.max_streams:
            raise ValueError(f"batch of {n} streams: must be 1..{self.max_streams}")
        ids = None
        if stream_ids is not None:
            ids = self._check_dev(stream_ids, "stream_ids", t.int32, (n,)).data_ptr()
        if out is None:
            out = t.empty((n, self.n_out), dtype=t.float32, device=self.device)
        self._check_dev(out, "out", t.float32, (n, self.n_out))
        return frames, code, n, ids, out

    def _boxes(self, boxes, box_off, n):
        t = self.torch
        if boxes is None or box_off is None:
            raise ValueError("boxes and box_off go together")
        if boxes.dim() != 2:
            raise ValueError("boxes must have shape (nb, 4)")
        self._check_dev(boxes, "boxes", t.int32, (boxes.shape[0], 4))
        self._check_dev(box_off, "box_off", t.int32, (n + 1,))
        if boxes.shape[0] == 0:
            # No boxes at all (no change): still a valid pointer, never read.
            boxes = t.zeros((1, 4), dtype=t.int32, device=self.device)
            self._empty_boxes = boxes
        return boxes.data_ptr(), box_off.data_ptr()

    def step(self, frames, stream_ids=None, boxes=None, box_off=None, out=None, stream=None):
        t = self.torch
        frames, code, n, ids, out = self._batch(frames, stream_ids, out)
        bx = bo = None
        if boxes is not None or box_off is not None:
            bx, bo = self._boxes(boxes, box_off, n)
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_step(self.handle, n, ids, frames.data_ptr(), code, bx, bo, out.data_ptr(), s)
        return out

    def full(self, frames, stream_ids=None, out=None, stream=None):
        t = self.torch
        frames, code, n, ids, out = self._batch(frames, stream_ids, out)
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_full(self.handle, n, ids, frames.data_ptr(), code, out.data_ptr(), s)
        return out

    def reset(self, stream_id: int = -1):
        reuse_net_reset(self.handle, stream_id)

    def variants(self, base_stream: int, boxes, box_off, frames, max_tiles: int = 0, out=None,
                 stream=None):
        """Logits of n variants of slot base_stream (reuse_net_variants): variant i
        takes the pixels of its boxes [box_off[i], box_off[i+1]) from frames[i]
        (frames of length n) or frames[0] (length 1).  The scratch is a torch
        tensor kept on this object and grown as needed."""
        t = self.torch
        frames, code = self._frames(frames)
        if not isinstance(box_off, t.Tensor) or box_off.dim() != 1 or box_off.shape[0] < 2:
            raise ValueError("box_off must be a 1-D int32 tensor of n + 1 entries")
        n = box_off.shape[0] - 1
        if frames.shape[0] not in (1, n):
            raise ValueError(f"frames must hold 1 or n = {n} frames, got {frames.shape[0]}")
        bx, bo = self._boxes(boxes, box_off, n)
        if out is None:
            out = t.empty((n, self.n_out), dtype=t.float32, device=self.device)
        self._check_dev(out, "out", t.float32, (n, self.n_out))
        need = reuse_net_variant_scratch_bytes(self.handle, n, max_tiles)
        if need == 0:
            _check(load_library().reuse_net_variants(self.handle, base_stream, n, None, 0, 0, None,
                                                     None, max_tiles, None, 0, None, None),
                   self.handle)
        if getattr(self, "_scratch", None) is None or self._scratch.numel() < need:
            self._scratch = t.empty(need, dtype=t.uint8, device=self.device)
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_variants(self.handle, base_stream, n, frames.data_ptr(), code, frames.shape[0],
                           bx, bo, max_tiles, self._scratch.data_ptr(),
                           self._scratch.numel(), out.data_ptr(), s)
        self._last_batch = n
        return out

    def variants_static(self, base_stream: int, boxes, box_off, frames, max_tiles: int = 0, out=None,
                        stream=None):
        """As variants(), through reuse_net_variants_static: the library's static
        per-GPU scratch, no allocation by the library (out is allocated here
        only when not given)."""
        t = self.torch
        frames, code = self._frames(frames)
        if not isinstance(box_off, t.Tensor) or box_off.dim() != 1 or box_off.shape[0] < 2:
            raise ValueError("box_off must be a 1-D int32 tensor of n + 1 entries")
        n = box_off.shape[0] - 1
        if frames.shape[0] not in (1, n):
            raise ValueError(f"frames must hold 1 or n = {n} frames, got {frames.shape[0]}")
        bx, bo = self._boxes(boxes, box_off, n)
        if out is None:
            out = t.empty((n, self.n_out), dtype=t.float32, device=self.device)
        self._check_dev(out, "out", t.float32, (n, self.n_out))
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_variants_static(self.handle, base_stream, n, frames.data_ptr(), code, frames.shape[0],
                                  bx, bo, max_tiles, out.data_ptr(), s)
        self._last_batch = n
        return out

    # -- training
    def grad_elems(self) -> int:
        return reuse_net_grad_elems(self.handle)

    def new_grads(self):
        """A zeroed float32 gradient buffer (layout of reuse_net_backward)."""
        n = self.grad_elems()
        if n == 0:
            _check(load_library().reuse_net_sgd_step(self.handle, None, 0.0, None), self.handle)
        return self.torch.zeros(n, dtype=self.torch.float32, device=self.device)

    def split_grads(self, grads):
        """Views of a gradient buffer: (conv_w list OIHW, conv_b list, dense_w, dense_b)."""
        off, cw, cb = 0, [], []
        for (ci, co, k, _s, _p) in self.specs:
            cw.append(grads[off:off + co * ci * k * k].view(co, ci, k, k))
            off += co * ci * k * k
            cb.append(grads[off:off + co])
            off += co
        gh, gw = self.grids[-1]
        nd = self.n_out * self.channels[-1] * gh * gw
        return cw, cb, grads[off:off + nd].view(self.n_out, -1), grads[off + nd:off + nd + self.n_out]

    def reinforce_dlogits(self, logits, actions, returns, out=None, stream=None):
        """dJ/dlogits of REINFORCE (reuse_net_reinforce_dlogits) for [n][n_out] logits."""
        t = self.torch
        n = logits.shape[0] if logits.dim() == 2 else -1
        self._check_dev(logits, "logits", t.float32, (n, self.n_out))
        self._check_dev(actions, "actions", t.int32, (n,))
        self._check_dev(returns, "returns", t.float32, (n,))
        if out is None:
            out = t.empty((n, self.n_out), dtype=t.float32, device=self.device)
        self._check_dev(out, "out", t.float32, (n, self.n_out))
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_reinforce_dlogits(n, self.n_out, logits.data_ptr(), actions.data_ptr(), returns.data_ptr(),
                                    out.data_ptr(), s)
        return out

    def backward(self, dlogits, grads, stream_ids=None, accumulate=False, stream=None):
        """Add (accumulate) or write the gradient of sum(dlogits * logits) for the
        streams' cached inputs into grads (reuse_net_backward)."""
        t = self.torch
        n = dlogits.shape[0] if dlogits.dim() == 2 else -1
        self._check_dev(dlogits, "dlogits", t.float32, (n, self.n_out))
        self._check_dev(grads, "grads", t.float32, (self.grad_elems(),))
        ids = None
        if stream_ids is not None:
            ids = self._check_dev(stream_ids, "stream_ids", t.int32, (n,)).data_ptr()
        need = reuse_net_backward_scratch_bytes(self.handle, n)
        if need == 0:
            _check(load_library().reuse_net_backward(self.handle, n, None, None, None, 0, None, 0, None),
                   self.handle)
        if getattr(self, "_bwd_scratch", None) is None or self._bwd_scratch.numel() < need:
            self._bwd_scratch = t.empty(need, dtype=t.uint8, device=self.device)
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_backward(self.handle, n, ids, dlogits.data_ptr(), grads.data_ptr(), accumulate,
                           self._bwd_scratch.data_ptr(), self._bwd_scratch.numel(), s)
        return grads

    def sgd_step(self, grads, lr: float, stream=None):
        """W <- W - lr * grads on the device; every slot recomputes on its next step."""
        t = self.torch
        self._check_dev(grads, "grads", t.float32, (self.grad_elems(),))
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_sgd_step(self.handle, grads.data_ptr(), lr, s)

    def set_weights_device(self, params, stream=None):
        """New weights from a device buffer in the gradient layout (see pack_params);
        every slot recomputes everything on its next step."""
        t = self.torch
        self._check_dev(params, "params", t.float32, (self.grad_elems(),))
        s = (stream or t.cuda.current_stream(self.device)).cuda_stream
        reuse_net_set_weights_device(self.handle, params.data_ptr(), s)

    def pack_params(self, weights):
        """(conv_w, conv_b, dense_w, dense_b) as one float32 device buffer in the
        gradient layout: each layer's OIHW weights then its bias, then the dense
        weights and bias (argument marshalling: a concatenation, no arithmetic)."""
        conv_w, conv_b, dense_w, dense_b = weights
        parts = []
        for w, b in zip(conv_w, conv_b):
            parts += [np.asarray(w, dtype=np.float32).ravel(), np.asarray(b, dtype=np.float32).ravel()]
        parts += [np.asarray(dense_w, dtype=np.float32).ravel(), np.asarray(dense_b, dtype=np.float32).ravel()]
        flat = np.concatenate(parts)
        n = self.grad_elems()
        if n == 0:
            raise RuntimeError("this net has no device weight layout (training calls unsupported)")
        if flat.size != n:
            raise ValueError(f"weights hold {flat.size} floats, the net needs {n}")
        return self.torch.from_numpy(flat).to(self.device)

    # -- introspection
    def pixel_mask(self, layer: int, stream_id: int) -> np.ndarray:
        """uint64 [H_l][words_per_row_l] bit rows of layer l's grid."""
        gh, gw = self.grids[layer]
        wpr = -(-gw // 64)
        return reuse_net_get_pixel_mask(self.handle, layer, stream_id, gh * wpr).reshape(gh, wpr)

    def pixel_mask_u8(self, layer: int, stream_id: int) -> np.ndarray:
        """uint8 [H_l][W_l], 1 = dirty (unpacked from the bit rows)."""
        gh, gw = self.grids[layer]
        m = self.pixel_mask(layer, stream_id)
        bits = np.unpackbits(m.view(np.uint8).reshape(gh, -1), axis=1, bitorder="little")
        return bits[:, :gw]

    def tile_mask_u8(self, layer: int, stream_id: int) -> np.ndarray:
        th, tw = self.layer_tiles[layer]
        m = reuse_net_get_tile_mask(self.handle, layer, stream_id, -(-(th * tw) // 64))
        bits = np.unpackbits(m.view(np.uint8), bitorder="little")
        return bits[:th * tw].reshape(th, tw)

    def worklist(self, layer: int, cap: Optional[int] = None) -> np.ndarray:
        batch = max(self.max_streams, getattr(self, "_last_batch", 0))
        th, tw = self.layer_tiles[layer]
        cap = cap if cap is not None else batch * th * tw
        return reuse_net_get_worklist(self.handle, layer, cap)

    def activation(self, stream_id: int, layer: int) -> np.ndarray:
        gh, gw = self.grids[layer]
        return reuse_net_read_activation(self.handle, stream_id, layer, (self.channels[layer], gh, gw))

    def stats(self) -> dict:
        return reuse_net_get_stats(self.handle)

    def set_profiling(self, on: bool):
        reuse_net_set_profiling(self.handle, on)

    def profile(self) -> dict:
        return reuse_net_get_profile(self.handle)

    def close(self):
        if getattr(self, "handle", None):
            reuse_net_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
