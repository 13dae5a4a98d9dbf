"""Seeded generators for the Atari-like sprite workloads.

The paper times a two-conv + dense policy on grayscale Atari frames downsampled
by 2 or 4 per side (Sec. 2; appendix tables).  The emulator and its ROMs are not
available, so these generators stand in for the game frames: a static uint8
background with a few constant-valued square sprites that move a few pixels per
frame, which keeps the property the paper's Fig. 3 discussion relies on (most
pixels stay the same from frame to frame).

Every random draw uses numpy's PCG64 with a fixed seed list:
  frames of stream ``s`` of workload ``cid``: ``default_rng([cid, s, 0])``
  weights of workload ``cid``:                ``default_rng([cid, 1])``
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Sequence

import numpy as np


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: stream count, frame count, frame shape and net."""

    cid: int                      # seed id
    streams: int
    frames: int
    h: int
    w: int
    convs: tuple                  # per conv layer: output channels (3x3, stride 1, pad 1)
                                  # or (cout, k, stride, pad)
    n_out: int                    # logits
    n_sprites: int = 3
    smin: int = 4
    smax: int = 4
    vmin: int = 1
    vmax: int = 2
    stack: int = 1                # frames stacked as input channels
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def in_c(self) -> int:
        return self.stack

    def conv_specs(self):
        """(cin, cout, k, stride, pad) per conv layer."""
        specs = []
        cin = self.in_c
        for c in self.convs:
            cout, k, s, p = tuple(c) if isinstance(c, (tuple, list)) else (c, 3, 1, 1)
            specs.append((cin, cout, k, s, p))
            cin = cout
        return specs

    def grids(self):
        """(h, w) of the input and of each conv layer's output."""
        g = [(self.h, self.w)]
        for (_ci, _co, k, s, p) in self.conv_specs():
            gh, gw = g[-1]
            g.append(((gh + 2 * p - k) // s + 1, (gw + 2 * p - k) // s + 1))
        return g

    def channels(self):
        return [self.in_c] + [sp[1] for sp in self.conv_specs()]

    def dense_in(self) -> int:
        gh, gw = self.grids()[-1]
        return self.conv_specs()[-1][1] * gh * gw

    def dense_macs_per_frame(self) -> int:
        m = 0
        for (ci, co, k, _s, _p), (gh, gw) in zip(self.conv_specs(), self.grids()[1:]):
            m += gh * gw * co * ci * k * k
        return m + self.n_out * self.dense_in()


WORKLOADS = {
    "atari-ds4-1x16": Workload(
        cid=1, streams=1, frames=16, h=53, w=40, convs=(40, 80), n_out=6,
        n_sprites=3, smin=4, smax=4, vmin=1, vmax=2,
        description="1 stream x 16 frames, 53x40, conv 1->40->80, dense->6"),
    "atari-ds2-256x64": Workload(
        cid=2, streams=256, frames=64, h=105, w=80, convs=(40, 80), n_out=6,
        n_sprites=6, smin=4, smax=8, vmin=1, vmax=3,
        description="256 streams x 64 frames, 105x80, conv 1->40->80, dense->6"),
    "occlusion-105x80-4096": Workload(
        cid=3, streams=64, frames=64, h=105, w=80, convs=(40, 80), n_out=6,
        n_sprites=6, smin=4, smax=8, vmin=1, vmax=3,
        description="4096 occlusion variants (8x8 zero patch, 64x64 top-left grid) "
                    "of one 105x80 base, evaluated together against the base's caches",
        extra={"patch": 8, "grid": 64}),
    "dqn-84x84-256x64": Workload(
        cid=6, streams=256, frames=64, h=84, w=84,
        convs=((32, 8, 4, 0), (64, 4, 2, 0), (64, 3, 1, 0)), n_out=6,
        n_sprites=5, smin=3, smax=6, vmin=1, vmax=2, stack=4,
        description="256 streams x 64 frames, 84x84, the last 4 frames stacked, conv 8x8/4 4->32, "
                    "4x4/2 32->64, 3x3/1 64->64 (no padding), dense->6"),
    "stack4-512x64": Workload(
        cid=4, streams=512, frames=64, h=105, w=80, convs=(40, 80), n_out=6,
        n_sprites=6, smin=4, smax=8, vmin=1, vmax=3, stack=4,
        description="512 streams x 64 frames, 105x80, last 4 frames stacked, "
                    "conv 4->40->80, dense->6"),
    "fullres-1024x32": Workload(
        cid=5, streams=1024, frames=32, h=210, w=160, convs=(64, 128, 128), n_out=18,
        n_sprites=6, smin=4, smax=8, vmin=1, vmax=3,
        description="1024 streams x 32 frames, 210x160, conv 1->64->128->128, dense->18"),
}

# Sprite presets for the full-resolution change-fraction sweep (210x160).
# The measured fraction is what gets reported; these only aim near the target.
FRACTION_PRESETS = {
    0.001: dict(n_sprites=2, smin=4, smax=4, vmin=1, vmax=1),
    0.01: dict(n_sprites=10, smin=6, smax=8, vmin=1, vmax=2),
    0.05: dict(n_sprites=26, smin=10, smax=14, vmin=2, vmax=3),
    0.20: dict(n_sprites=60, smin=14, smax=20, vmin=3, vmax=5),
}


def to_f32(frames_u8: np.ndarray) -> np.ndarray:
    """uint8 level k -> float32 k/255, IEEE single division (correctly rounded)."""
    return frames_u8.astype(np.float32) / np.float32(255.0)


def _moves(vmin: int, vmax: int) -> np.ndarray:
    """All integer (dy, dx) with vmin <= max(|dy|, |dx|) <= vmax."""
    out = []
    for dy in range(-vmax, vmax + 1):
        for dx in range(-vmax, vmax + 1):
            if vmin <= max(abs(dy), abs(dx)) <= vmax:
                out.append((dy, dx))
    return np.asarray(out, dtype=np.int64)


def _reflect(p: int, hi: int) -> int:
    """Reflect a top-left coordinate into [0, hi]."""
    if hi <= 0:
        return 0
    while p < 0 or p > hi:
        if p < 0:
            p = -p
        if p > hi:
            p = 2 * hi - p
    return p


def sprite_sequence(cid: int, stream: int, frames: int, h: int, w: int,
                    n_sprites: int, smin: int, smax: int, vmin: int, vmax: int) -> np.ndarray:
    """uint8 [frames][h][w]: static random background plus moving 255-valued squares."""
    rng = np.random.default_rng([cid, stream, 0])
    bg = rng.integers(0, 256, size=(h, w), dtype=np.uint8)
    sizes = rng.integers(smin, smax + 1, size=n_sprites)
    ys = [int(rng.integers(0, h - s + 1)) for s in sizes]
    xs = [int(rng.integers(0, w - s + 1)) for s in sizes]
    moves = _moves(vmin, vmax)
    out = np.empty((frames, h, w), dtype=np.uint8)
    for t in range(frames):
        if t > 0:
            pick = rng.integers(0, len(moves), size=n_sprites)
            for i in range(n_sprites):
                dy, dx = moves[pick[i]]
                ys[i] = _reflect(ys[i] + int(dy), h - int(sizes[i]))
                xs[i] = _reflect(xs[i] + int(dx), w - int(sizes[i]))
        f = bg.copy()
        for i in range(n_sprites):
            s = int(sizes[i])
            f[ys[i]:ys[i] + s, xs[i]:xs[i] + s] = 255
        out[t] = f
    return out


def full_change_sequence(cid: int, stream: int, frames: int, h: int, w: int) -> np.ndarray:
    """uint8 [frames][h][w] where every pixel changes every frame: k <- (k + 1 + U{0..254}) mod 256."""
    rng = np.random.default_rng([cid, stream, 0])
    out = np.empty((frames, h, w), dtype=np.uint8)
    cur = rng.integers(0, 256, size=(h, w), dtype=np.int64)
    out[0] = cur
    for t in range(1, frames):
        cur = (cur + 1 + rng.integers(0, 255, size=(h, w))) % 256
        out[t] = cur
    return out


def sprite_batch(wl: Workload, streams: Sequence[int] | None = None, frames: int | None = None,
                 **override) -> np.ndarray:
    """uint8 [frames][len(streams)][h][w] for a workload (frame-major, ready for per-step batches)."""
    if streams is None:
        streams = range(wl.streams)
    streams = list(streams)
    f = wl.frames if frames is None else frames
    p = dict(n_sprites=wl.n_sprites, smin=wl.smin, smax=wl.smax, vmin=wl.vmin, vmax=wl.vmax)
    p.update(override)
    out = np.empty((f, len(streams), wl.h, wl.w), dtype=np.uint8)
    for j, s in enumerate(streams):
        if p.get("full_change"):
            out[:, j] = full_change_sequence(wl.cid, s, f, wl.h, wl.w)
        else:
            out[:, j] = sprite_sequence(wl.cid, s, f, wl.h, wl.w, p["n_sprites"], p["smin"],
                                        p["smax"], p["vmin"], p["vmax"])
    return out


def stacked_view(seq: np.ndarray, t: int, depth: int = 4) -> np.ndarray:
    """Input of step t when the last ``depth`` frames are stacked as channels, oldest first.

    seq: [frames][...]; before enough frames exist, frame 0 repeats.  Returns [depth][...].
    """
    idx = [max(0, t - depth + 1 + j) for j in range(depth)]
    return np.stack([seq[i] for i in idx], axis=0)


def occlusion_base(wl: Workload) -> np.ndarray:
    """uint8 [h][w] base image: frame 0 of the sprite generator for stream 0."""
    return sprite_sequence(wl.cid, 0, 1, wl.h, wl.w, wl.n_sprites, wl.smin, wl.smax,
                           wl.vmin, wl.vmax)[0]


def occlusion_variant_frame(base_f32: np.ndarray, y: int, x: int, patch: int) -> np.ndarray:
    """float32 [h][w]: base with a zero patch whose top-left corner is (y, x)."""
    f = base_f32.copy()
    f[y:y + patch, x:x + patch] = 0.0
    return f


def occlusion_boxes(y: int, x: int, patch: int) -> list:
    """Change boxes (y0, x0, y1, x1), half-open, of occlusion step x on row y.

    Step x moves the patch from (y, x-1) to (y, x); step 0 only places it.
    """
    boxes = []
    if x > 0:
        boxes.append((y, x - 1, y + patch, x - 1 + patch))
    boxes.append((y, x, y + patch, x + patch))
    return boxes


def net_weights(wl: Workload, bias_std: float = 0.0, seed_extra: int | None = None):
    """float32 weights: conv OIHW per layer, conv bias, dense [n_out][C_L*H*W] (c,y,x order), dense bias.

    Weights ~ N(0, 0.05).  Biases are zero unless ``bias_std`` is given (tests use
    non-zero biases so that the bias path is exercised).
    """
    seeds = [wl.cid, 1] if seed_extra is None else [wl.cid, 1, seed_extra]
    rng = np.random.default_rng(seeds)
    conv_w, conv_b = [], []
    for (cin, cout, k, _s, _p) in wl.conv_specs():
        conv_w.append(rng.normal(0.0, 0.05, size=(cout, cin, k, k)).astype(np.float32))
        conv_b.append((rng.normal(0.0, bias_std, size=cout) if bias_std else
                       np.zeros(cout)).astype(np.float32))
    dense_w = rng.normal(0.0, 0.05, size=(wl.n_out, wl.dense_in())).astype(np.float32)
    dense_b = (rng.normal(0.0, bias_std, size=wl.n_out) if bias_std else
               np.zeros(wl.n_out)).astype(np.float32)
    return conv_w, conv_b, dense_w, dense_b
