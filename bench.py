"""Benchmark of frame-to-frame convolutional activation reuse on one MI355X.

A step is one pass of the whole hot path over one frame of every stream:
diff (or explicit change boxes) -> change growth and dirty-tile masks -> work
lists -> dirty-tile conv layers (bias, ReLU, scatter into the caches) -> dense
head.  Inputs are synthetic and resident in HBM before timing starts.  The
dense recompute path of the same library (`reuse_net_full`) and the CPU
oracle are timed in the same run.

Workloads (synth.WORKLOADS):
  fullres-1024x32 (default)   1024 streams x 32 frames, 210x160, 1->64->128->128, dense->18
                              (--change-frac picks the sprite preset of the sweep; default 0.01)
  atari-ds2-256x64            256 streams x 64 frames, 105x80, 1->40->80, dense->6
  atari-ds4-1x16              1 stream x 16 frames, 53x40
  stack4-512x64               512 streams, the last 4 frames stacked as input channels
  dqn-84x84-256x64            256 streams x 64 frames, 84x84, 4 stacked frames, DQN-style trunk
                              (8x8/4 4->32, 4x4/2 32->64, 3x3/1 64->64, no padding), dense->6
  occlusion-105x80-4096       4096 occlusion variants of one base image, one
                              reuse_net_variants call (copy-on-write overlays) per step
The frame order runs 1..F-1 and then back and forth, so every transition is
an ordinary sprite move.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_MFMA_F32_TFLOPS = 157.3
PEAK_MFMA_BF16_TFLOPS = 2500.0
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_1909_05632_amd", "csrc")
DEFAULT_WORKLOAD = "fullres-1024x32"
DEFAULT_CHANGE_FRAC = 0.01          # the full-resolution workload's 1% change preset


def kernel_source_hash(source: str) -> str:
    """Hash of a kernel source file together with the device headers it includes."""
    import hashlib
    h = hashlib.sha256()
    for f in (source, "rn_device.hpp", "rn_internal.hpp"):
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(key: dict):
    """HBM bytes per launch of one conv layer's kernel from the committed counter
    runs (profiles/traffic_*.json) whose workload key equals `key`, or None when
    there is none or it was taken on a different kernel source."""
    import glob
    for path in sorted(glob.glob(os.path.join(PROFILES, "traffic_*.json"))):
        try:
            rec = json.load(open(path))
        except (OSError, ValueError):
            continue
        if rec.get("key") != key:
            continue
        if rec.get("source_sha256_16") != kernel_source_hash(rec.get("source", "")):
            return None
        return rec.get("bytes_per_launch")
    return None


def layer_kernel(specs, l, dtype, folded):
    """Name of the kernel that computes conv layer l (1-based) in the library."""
    ci, co, k, st, pd = specs[l - 1]
    if not (k == 3 and st == 1 and pd == 1):
        return f"k_conv_gen<{k}, {st}, {ci}, {co}>"
    if dtype == "bf16":
        return f"k_conv_first_bf16<{ci}, {co}>" if l == 1 else f"k_conv_bf16_grp<{ci}, {co}>"
    if l == 1:
        return f"k_conv_first4_mfma<{co}>" if ci == 4 else f"k_conv_first_f32<{ci}, {co}>"
    if (ci, co) == (40, 80):                                     # weights resident in LDS
        return "k_conv_mfma_res<40, 80>" + (" (layer 1 folded in)" if folded else "")
    return f"k_conv_mfma_staged<{ci}, {co}>"


def schedule(frames: int, length: int):
    """Frame indices for `length` steps after priming on frame 0: 1..F-1, then back and forth."""
    seq = []
    t, d = 0, 1
    while len(seq) < length:
        if not 0 <= t + d < frames:
            d = -d
        t += d
        seq.append(t)
    return seq


# ------------------------------------------------------------------ drivers

class SpriteDriver:
    """Independent streams of sprite frames (optionally stacked 4 deep)."""

    unit = "frames/s"
    metric = "frames/sec (all streams)"

    def __init__(self, torch, wl, length, preset=None):
        from synth import frames as synth
        self.wl = wl
        self.S = wl.streams
        self.max_streams = wl.streams
        self.preset = preset or {}
        self.u8 = synth.sprite_batch(wl, **self.preset)            # [F][S][H][W]
        self.frames = torch.from_numpy(synth.to_f32(self.u8)).cuda().unsqueeze(2).contiguous()
        self.seq = schedule(wl.frames, length)

    def prime(self, net, out):
        net.full(self.frames[0], out=out)

    def reuse_step(self, net, k, out):
        net.step(self.frames[self.seq[k]], out=out)

    def dense_step(self, net, k, out):
        net.full(self.frames[self.seq[k]], out=out)

    def mask_bytes(self):
        # frame + cached input, read once per step
        wl = self.wl
        return 2 * self.S * wl.h * wl.w * 4 * wl.in_c

    def cpu_sample(self, oracle, weights, budget_s):
        from synth import frames as synth
        wl = self.wl
        onet = oracle.Net(wl.in_c, wl.h, wl.w, wl.conv_specs(), wl.n_out)
        n = min(16 if wl.h * wl.w < 20000 else 4, self.S)
        x = synth.to_f32(self.u8[:, :n])
        done, t0, t, frames = 0, time.perf_counter(), 0, 0
        while True:
            t = t % (x.shape[0] - 1) + 1
            if wl.stack > 1:
                cur = np.stack([synth.stacked_view(x[:, i], t) for i in range(n)])
                prev = np.stack([synth.stacked_view(x[:, i], t - 1) for i in range(n)])
            else:
                cur, prev = x[t][:, None], x[t - 1][:, None]
            d0 = np.stack([oracle.diff(prev[i], cur[i]) for i in range(n)])
            _, m = oracle.masks(onet, d0, want_pixels=False)
            oracle.worklists(m)
            oracle.forward(onet, *weights, cur)
            done += n
            frames += 1
            el = time.perf_counter() - t0
            if el >= budget_s:
                break
        return done / el, f"{n} streams x {frames} frames of {wl.h}x{wl.w}" + \
            (" (4 stacked)" if wl.stack > 1 else "")


class OcclusionDriver:
    """Occlusion map of one base image: 4096 variants, each the base with an
    8x8 zero patch at one corner of a 64x64 grid.  A step evaluates all of them
    in one reuse_net_variants call against the primed base slot (no per-variant
    caches; at most 16 dirty tiles per variant and layer).  The dense path runs
    the same 4096 variant frames through reuse_net_full, 512 at a time."""

    unit = "variants/s"
    metric = "occlusion variants/sec"
    DENSE_BATCH = 512
    MAX_TILES = 16

    def __init__(self, torch, wl, length):
        from synth import frames as synth
        self.wl = wl
        P, G = wl.extra["patch"], wl.extra["grid"]
        self.S = G * G
        self.max_streams = self.DENSE_BATCH
        self.base = synth.to_f32(synth.occlusion_base(wl))
        self.base_dev = torch.from_numpy(self.base[None, None]).cuda().contiguous()
        var = np.stack([synth.occlusion_variant_frame(self.base, i // G, i % G, P)[None]
                        for i in range(self.S)])                   # [4096][1][H][W]
        self.frames = torch.from_numpy(var).cuda().contiguous()
        boxes = np.asarray([(y, x, y + P, x + P) for y in range(G) for x in range(G)], np.int32)
        self.boxes = torch.from_numpy(boxes).cuda()
        self.box_off = torch.arange(0, self.S + 1, dtype=torch.int32).cuda()
        self.zero = torch.zeros((1, 1, wl.h, wl.w), dtype=torch.float32).cuda()
        self.P, self.G = P, G

    def prime(self, net, out):
        net.full(self.base_dev, out=out[:1])

    def reuse_step(self, net, k, out):
        net.variants(0, self.boxes, self.box_off, self.zero, max_tiles=self.MAX_TILES, out=out)

    def dense_step(self, net, k, out):
        B = self.DENSE_BATCH
        for j in range(0, self.S, B):
            net.full(self.frames[j:j + B], out=out[j:j + B])

    def mask_bytes(self):
        # pixel and tile masks of every layer written per variant (no frame is read)
        wl = self.wl
        L, th, tw = len(wl.convs), -(-wl.h // 4), -(-wl.w // 4)
        return self.S * (L + 1) * (wl.h * -(-wl.w // 64) + -(-th * tw // 64)) * 8

    def cpu_sample(self, oracle, weights, budget_s):
        from synth import frames as synth
        wl = self.wl
        onet = oracle.Net(1, wl.h, wl.w, wl.conv_specs(), wl.n_out)
        P, G, n = self.P, self.G, 16
        done, t0, i0 = 0, time.perf_counter(), 0
        while True:
            idx = [(i0 + j) % self.S for j in range(n)]
            var = np.stack([synth.occlusion_variant_frame(self.base, i // G, i % G, P)[None] for i in idx])
            d0 = np.stack([oracle.box_mask(wl.h, wl.w, [(i // G, i % G, i // G + P, i % G + P)])
                           for i in idx])
            _, m = oracle.masks(onet, d0, want_pixels=False)
            oracle.worklists(m)
            oracle.forward(onet, *weights, var)
            done += n
            i0 = (i0 + n) % self.S
            el = time.perf_counter() - t0
            if el >= budget_s:
                break
        return done / el, f"{done} variants (16 per batch) of {wl.h}x{wl.w}"


def train_bench(args, torch):
    """REINFORCE training with activation reuse (Sec. 2: the policy is trained
    with REINFORCE; the weights stay fixed within an episode).  One episode of
    T frames for every stream: a rollout of T reuse steps, then a replay of the
    same frames as reuse steps, each followed by the REINFORCE logit gradient
    (synthetic seeded actions and discounted returns) and a backward pass
    accumulating the episode's gradient, then one SGD step on the device (which
    unprimes every slot).  The dense comparison runs the same loop with
    reuse_net_full for every forward pass.  Frames/s = streams x T per episode
    time."""
    from paper_1909_05632_amd import ReuseNet
    from synth import frames as synth

    wl = synth.WORKLOADS[args.workload]
    T, S, F = args.episode, wl.streams, wl.frames
    preset = {}
    if args.change_frac is not None:
        preset = ({"full_change": True} if args.change_frac >= 1.0 else dict(synth.FRACTION_PRESETS[args.change_frac]))
    u8 = synth.sprite_batch(wl, **preset)
    frames = torch.from_numpy(synth.to_f32(u8)).cuda().unsqueeze(2).contiguous()
    weights = synth.net_weights(wl)
    # Training keeps layer 1 in its own cache unless --fold-first: the backward
    # needs layer 1's activations, which a folded net recomputes densely for
    # every backward call (1.98 ms per 16-frame episode against 0.47 ms for
    # layer 1's own kernel on the dirty tiles of the forward steps).
    net = ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, S, weights, stack=wl.stack, head=args.head,
                   fuse_first=args.fold_first)
    grads = net.new_grads()
    rng = np.random.default_rng([wl.cid, 7])
    actions = torch.from_numpy(rng.integers(0, wl.n_out, (T, S)).astype(np.int32)).cuda()
    rewards = rng.uniform(-1.0, 1.0, (T, S))
    G = np.zeros_like(rewards)
    acc = np.zeros(S)
    for t in range(T - 1, -1, -1):                          # discounted returns, gamma 0.99
        acc = rewards[t] + 0.99 * acc
        G[t] = acc
    returns = torch.from_numpy(G.astype(np.float32)).cuda()
    out = torch.empty((T, S, wl.n_out), dtype=torch.float32, device="cuda")
    dl = torch.empty((S, wl.n_out), dtype=torch.float32, device="cuda")
    lr = 1e-3
    stream = torch.cuda.current_stream()

    def episode(e, dense):
        f0 = (e * T) % max(1, F - T)
        fwd = net.full if dense else net.step
        for t in range(T):                                  # rollout
            fwd(frames[f0 + t], out=out[t])
        for t in range(T):                                  # replay with the episode's returns
            fwd(frames[f0 + t], out=out[t])
            net.reinforce_dlogits(out[t], actions[t], returns[t], out=dl)
            net.backward(dl, grads, accumulate=t > 0)
        net.sgd_step(grads, lr)

    def timed(dense, episodes, profile=False):
        for e in range(args.warmup):
            episode(e, dense)
        torch.cuda.synchronize()
        net.set_profiling(profile)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for e in range(episodes):
            episode(args.warmup + e, dense)
        e1.record(stream)
        torch.cuda.synchronize()
        prof = net.profile() if profile else None
        net.set_profiling(False)
        return e0.elapsed_time(e1) / episodes, prof

    K = args.steps
    ms_ep, _ = timed(False, K)
    _, prof = timed(False, 1, profile=True)
    ms_dense, _ = timed(True, max(1, K // 2))
    fps = S * T / (ms_ep / 1e3)
    fps_dense = S * T / (ms_dense / 1e3)

    specs = wl.conv_specs()
    grids = wl.grids()
    tiles = [-(-gh // 4) * -(-gw // 4) for gh, gw in grids]
    # algorithmic flops of one backward call over S streams (padded tile pixels included)
    f_dw = sum(2 * S * tiles[l + 1] * 16 * co * (k * k * ci + 1) for l, (ci, co, k, _s, _p) in enumerate(specs))
    f_dx = sum(2 * S * tiles[l + 1] * 16 * ci * k * k * co for l, (ci, co, k, _s, _p) in enumerate(specs) if l > 0)
    kern = {name: {"ms_per_episode": prof[name]["ms"], "launches": prof[name]["launches"]}
            for name in ("masks", "compact", "conv1", "convN", "head", "bwd_head", "bwd_dw", "bwd_dx", "sgd")}
    kern["bwd_dw"]["tflops"] = f_dw * T / (prof["bwd_dw"]["ms"] / 1e3) / 1e12
    if f_dx:
        kern["bwd_dx"]["tflops"] = f_dx * T / (prof["bwd_dx"]["ms"] / 1e3) / 1e12
    dom = max(("bwd_dw", "bwd_dx"), key=lambda k: prof[k]["ms"])
    ach = kern[dom]["tflops"]
    roof = {"bound": "mfma", "kernel": {"bwd_dw": "k_bwd_dw8 / k_bwd_dw2 + k_bwd_dw_first (weight gradients, teams of tiles on MFMA)",
                                        "bwd_dx": "k_bwd_dx (input gradients, transposed conv on MFMA)"}[dom],
            "achieved": ach, "peak": PEAK_MFMA_F32_TFLOPS, "unit": "TFLOP/s", "frac": ach / PEAK_MFMA_F32_TFLOPS,
            "traffic": None}
    cpu = None
    if not args.no_cpu:
        import oracle
        onet = oracle.Net(wl.in_c, wl.h, wl.w, specs, wl.n_out)
        x = synth.to_f32(u8[:T, :2])
        done, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_budget:
            t = done % T
            cur = x[t][:, None] if wl.stack == 1 else np.stack([synth.stacked_view(x[:, i], t) for i in range(2)])
            z, _ = oracle.forward(onet, *weights, cur)
            g = oracle.reinforce_dlogits(z, actions[t, :2].cpu().numpy(), returns[t, :2].cpu().numpy())
            oracle.backward(onet, *weights, cur, g)
            done += 1
        el = time.perf_counter() - t0
        cpu = {"value": 2 * done / el, "unit": "frames/s", "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
               "sample": f"2 streams x {done} frames: full forward, REINFORCE logit gradient and backpropagation "
                         "in double (one forward pass per frame, no rollout/replay split)"}
    line = {
        "metric": "training frames/sec (REINFORCE: reuse rollout + replay with backward + SGD step, all streams)",
        "value": fps, "unit": "frames/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms_ep, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "streams": S, "episode_frames": T, "h": wl.h, "w": wl.w,
                   "convs": list(wl.convs), "n_out": wl.n_out, "head": args.head, "lr": lr,
                   "first_layer": "folded into layer 2 where it applies" if args.fold_first else "own kernel and cache",
                   "step": "one episode: T rollout steps, T replay steps with backward, one SGD step"},
        "dense_path": {"value": fps_dense, "unit": "frames/s", "ms_per_step": ms_dense},
        "speedup_vs_dense": fps / fps_dense,
        "kernels": kern, "roofline": roof, "cpu_baseline": cpu,
    }
    print(json.dumps(line))
    net.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=120)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--change-frac", type=float, default=None,
                    help="full-resolution sweep preset: 0.001, 0.01, 0.05, 0.2 or 1.0 "
                         f"(default {DEFAULT_CHANGE_FRAC} for {DEFAULT_WORKLOAD})")
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--dense-steps", type=int, default=None)
    ap.add_argument("--head", default="tiles", choices=["tiles", "full"])
    ap.add_argument("--update-every", type=int, default=0,
                    help="training rollouts: replace the weights every N steps (inside the timed "
                         "region; every slot then recomputes everything on its next step)")
    ap.add_argument("--host-weight-update", action="store_true",
                    help="with --update-every: replace the weights through the host repack and upload "
                         "(reuse_net_set_weights) even where the device path applies")
    ap.add_argument("--separate-first", action="store_true",
                    help="run layer 1 as its own kernel instead of inside layer 2 (inference; "
                         "training always does unless --fold-first)")
    ap.add_argument("--fold-first", action="store_true",
                    help="--train: compute layer 1 inside layer 2 (no layer-1 cache; the backward "
                         "then recomputes layer 1)")
    ap.add_argument("--graph", action="store_true",
                    help="replay each reuse step from a HIP graph captured once per frame buffer "
                         "(one launch per step instead of one per kernel; the profiled pass stays eager)")
    ap.add_argument("--train", action="store_true",
                    help="time REINFORCE training episodes (rollout, replay with backward, SGD step) "
                         "instead of inference steps; --steps counts episodes")
    ap.add_argument("--episode", type=int, default=16, help="frames per training episode (--train)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy, 3 times (scales the "
                         "FETCH_SIZE / WRITE_SIZE counters to bytes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
              "(streams would shard across GPUs, one process each, with no exchange between them)", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = 1 << 28                                             # 1 GiB of float32
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"bytes_read": 4 * n, "bytes_written": 4 * n,
                                               "launches": 3}}))
        return

    from paper_1909_05632_amd import ReuseNet
    from synth import frames as synth

    if args.train:
        if args.workload == DEFAULT_WORKLOAD and "--workload" not in sys.argv:
            args.workload = "atari-ds2-256x64"              # the paper's training net (2 conv + dense)
        if args.steps == 120 and "--steps" not in sys.argv:
            args.steps = 4
        return train_bench(args, torch)
    if args.change_frac is None and args.workload == DEFAULT_WORKLOAD:
        args.change_frac = DEFAULT_CHANGE_FRAC
    wl = synth.WORKLOADS[args.workload]
    length = args.warmup + args.steps
    if args.workload.startswith("occlusion"):
        drv = OcclusionDriver(torch, wl, length)
    else:
        preset = None
        if args.change_frac is not None:
            preset = ({"full_change": True} if args.change_frac >= 1.0
                      else dict(synth.FRACTION_PRESETS[args.change_frac]))
        drv = SpriteDriver(torch, wl, length, preset)
    S = drv.S
    weights = synth.net_weights(wl)
    net = ReuseNet(1, wl.h, wl.w, wl.convs, wl.n_out, drv.max_streams, weights, act_dtype=args.dtype,
                   stack=wl.stack, head=args.head, fuse_first=not args.separate_first)
    out = torch.empty((S, wl.n_out), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    alt_weights = [weights, synth.net_weights(wl, seed_extra=1)] if args.update_every else None
    # Weight updates come from device buffers (reuse_net_set_weights_device) on
    # nets the training calls support, else through the host repack.
    dev_params = None
    if args.update_every and net.grad_elems() > 0 and not args.host_weight_update:
        dev_params = [net.pack_params(w) for w in alt_weights]

    def set_weights(i):
        if dev_params is not None:
            net.set_weights_device(dev_params[i])
        else:
            net.set_weights(alt_weights[i])

    graphs = {}
    if args.graph:
        if not isinstance(drv, SpriteDriver) or args.update_every:
            print("bench.py: --graph applies to the sprite workloads without weight updates", file=sys.stderr)
            sys.exit(2)
        # One eager step first, so one-time set-up happens outside the capture.
        drv.prime(net, out)
        drv.reuse_step(net, 0, out)
        torch.cuda.synchronize()
        for t in sorted(set(drv.seq)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                net.step(drv.frames[t], out=out)
            graphs[t] = g
        torch.cuda.synchronize()

    def do_step(k, eager=False):
        if args.update_every and k % args.update_every == 0 and k > 0:
            set_weights((k // args.update_every) % 2)
        if graphs and not eager:
            graphs[drv.seq[k]].replay()
        else:
            drv.reuse_step(net, k, out)

    def restart():
        # every pass starts from the first weight set, primed on the first frames
        if args.update_every:
            set_weights(0)
        drv.prime(net, out)

    # Stats pass: dirty tiles of exactly the steps the timed pass will run.
    restart()
    stats = []
    for k in range(length):
        do_step(k)
        if graphs:
            torch.cuda.synchronize()                            # the replay's stream, not the capture's
        stats.append(net.stats())
    timed_stats = stats[args.warmup:]

    def run_reuse(profile: bool):
        restart()
        for k in range(args.warmup):
            do_step(k, eager=profile)
        torch.cuda.synchronize()
        net.set_profiling(profile)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for k in range(args.warmup, length):
            do_step(k, eager=profile)
        e1.record(stream)
        torch.cuda.synchronize()
        prof = net.profile() if profile else None
        net.set_profiling(False)
        return e0.elapsed_time(e1), prof

    run_reuse(False)                                            # warm the caches and clocks
    ms_clean, _ = run_reuse(False)
    ms_prof, prof = run_reuse(True)

    # Dense recompute path of the same library on the same frames.
    dsteps = args.dense_steps or max(10, args.steps // 2)
    for k in range(args.warmup):
        drv.dense_step(net, k, out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for k in range(args.warmup, args.warmup + dsteps):
        drv.dense_step(net, k, out)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_dense = e0.elapsed_time(e1) / dsteps

    K = args.steps
    ms_step = ms_clean / K
    fps = S / (ms_step / 1e3)
    fps_dense = S / (ms_dense / 1e3)
    L = len(wl.convs)
    specs = wl.conv_specs()
    chans = wl.channels()
    ltiles = [-(-gh // 4) * -(-gw // 4) for gh, gw in wl.grids()]   # 4x4 tiles per layer grid
    general = [not (k == 3 and st == 1 and pd == 1) for (_ci, _co, k, st, pd) in specs]
    # algorithmic flops per dirty tile of layer l: 16 px x cout x k k cin x 2
    fpt = [0] + [16 * co * k * k * ci * 2 for (ci, co, k, _st, _pd) in specs]
    dirty = np.array([[s["dirty_tiles"][l] for l in range(L + 1)] for s in timed_stats], float)
    changed = np.mean([s["changed_px"] for s in timed_stats]) / (S * wl.h * wl.w)
    useful = np.mean([s["useful_mac"] for s in timed_stats])
    dense_mac = wl.dense_macs_per_frame()

    # Per-kernel figures from the HIP events of the profiled pass.
    kern = {}
    for name in ("masks", "compact", "conv1", "convN", "head"):
        kern[name] = {"ms_per_step": prof[name]["ms"] / K, "launches": prof[name]["launches"]}
    # MFMA conv layers 2..L (and a general first layer): flops of the dirty tiles
    flops_convn = sum(dirty[:, l].sum() * fpt[l] for l in range(2, L + 1))
    if prof["convN"]["ms"] > 0:
        kern["convN"]["tflops"] = flops_convn / (prof["convN"]["ms"] / 1e3) / 1e12
    if general[0] and prof["conv1"]["ms"] > 0:
        kern["conv1"]["tflops"] = dirty[:, 1].sum() * fpt[1] / (prof["conv1"]["ms"] / 1e3) / 1e12
    K_el = ltiles[L] * 16 * chans[L]
    esz = 2 if args.dtype == "bf16" else 4
    if args.head == "full":
        head_bytes = (S * K_el * esz + wl.n_out * K_el * 4) * K  # whole last-layer caches + weights
    else:
        head_bytes = S * ltiles[L] * wl.n_out * 4 * K           # per-tile partials
    kern["head"]["gbs"] = head_bytes / (prof["head"]["ms"] / 1e3) / 1e9
    mask_bytes = drv.mask_bytes() * K
    kern["masks"]["gbs"] = mask_bytes / (prof["masks"]["ms"] / 1e3) / 1e9
    k1, s1 = specs[0][2], specs[0][3]
    conv1_bytes = dirty[:, 1].sum() * (16 * chans[1] * esz + (3 * s1 + k1) ** 2 * chans[0] * 4)
    if prof["conv1"]["ms"] > 0:
        kern["conv1"]["gbs"] = conv1_bytes / (prof["conv1"]["ms"] / 1e3) / 1e9

    # Per conv layer: one kernel per layer and step, so its average launch is
    # the layer's summed event time over its launches.
    folded = (not args.separate_first) and chans[0] == 1 and L >= 2 and chans[1] == 40 and not any(general[:2])
    mfma_layer = [False] + [l >= 2 or general[0] or chans[0] == 4 for l in range(1, L + 1)]
    layers = {}
    for l in range(1, L + 1):
        rec = prof["layers"][l]
        if rec["launches"] == 0:
            continue                                            # layer 1 folded into layer 2
        ent = {"kernel": layer_kernel(specs, l, args.dtype, folded and l == 2), "launches": rec["launches"],
               "ms_per_step": rec["ms"] / K, "us_per_launch": 1e3 * rec["ms"] / rec["launches"],
               "dirty_tiles_per_launch": float(dirty[:, l].sum() / rec["launches"])}
        if mfma_layer[l]:
            ent["tflops"] = dirty[:, l].sum() * fpt[l] / (rec["ms"] / 1e3) / 1e12
        else:
            ent["gbs"] = conv1_bytes / (rec["ms"] / 1e3) / 1e9
        layers[str(l)] = ent
    kern["layers"] = layers

    # The roofline object reports the single kernel with the most time.
    cands = {("layer", l): layers[str(l)]["ms_per_step"] for l in range(1, L + 1) if str(l) in layers}
    for name in ("masks", "compact", "head"):
        cands[("phase", name)] = kern[name]["ms_per_step"]
    dom = max(cands, key=cands.get)
    if dom[0] == "layer":
        l = dom[1]
        ent = layers[str(l)]
        desc = f"{ent['kernel']}: dirty-tile conv layer {l} ({chans[l - 1]}->{chans[l]})"
        key = {"workload": args.workload, "change_preset": args.change_frac, "dtype": args.dtype,
               "head": args.head, "layer": l, "folded": bool(folded and l == 2)}
        traffic = measured_traffic(key)
        if mfma_layer[l]:
            peak = PEAK_MFMA_BF16_TFLOPS if args.dtype == "bf16" else PEAK_MFMA_F32_TFLOPS
            roof = {"bound": "mfma", "kernel": desc, "achieved": ent["tflops"], "peak": peak, "unit": "TFLOP/s",
                    "frac": ent["tflops"] / peak, "traffic": traffic}
        else:
            roof = {"bound": "hbm", "kernel": desc, "achieved": ent["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": ent["gbs"] / PEAK_HBM_GBS, "traffic": traffic}
        roof["us_per_launch"] = ent["us_per_launch"]
        roof["work_per_launch"] = (f"{ent['dirty_tiles_per_launch']:.0f} dirty tiles x "
                                   f"{fpt[l] / 1e6:.4f} MFLOP (2 x 16 px x {chans[l]} x "
                                   f"{specs[l - 1][2] ** 2 * chans[l - 1]})")
    else:
        name = dom[1]
        ach = kern[name].get("gbs", 0.0)
        roof = {"bound": "hbm", "kernel": name, "achieved": ach, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": ach / PEAK_HBM_GBS, "traffic": None}

    cpu = None
    if not args.no_cpu:
        import oracle
        v, sample = drv.cpu_sample(oracle, weights, args.cpu_budget)
        cpu = {"value": v, "unit": drv.unit, "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
               "sample": sample + " (full recompute in double + change masks and work lists, "
                                  "OpenMP over streams)"}

    cfg = {"workload": args.workload, "streams": S, "frames": wl.frames, "h": wl.h, "w": wl.w,
           "convs": list(wl.convs), "n_out": wl.n_out, "tile": "4x4", "head": args.head,
           "stack": wl.stack, "description": wl.description}
    if args.change_frac is not None:
        cfg["change_preset"] = args.change_frac
    if args.update_every:
        cfg["weight_update_every"] = args.update_every
        cfg["weight_update"] = "device" if dev_params is not None else "host"
    if graphs:
        cfg["launch"] = "graph replay per step"
    line = {
        "metric": drv.metric,
        "value": fps,
        "unit": drv.unit,
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": cfg,
        "dense_path": {"value": fps_dense, "unit": drv.unit, "ms_per_step": ms_dense},
        "speedup_vs_dense": fps / fps_dense,
        "changed_px_frac": changed,
        "dirty_tile_frac": [float(dirty[:, l].mean() / (S * ltiles[l])) for l in range(L + 1)],
        "effective_gmacs": dense_mac * fps / 1e9,
        "useful_gmacs": useful / (ms_step / 1e3) / 1e9,
        "ms_per_step_profiled": ms_prof / K,
        "kernels": kern,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))
    net.close()


if __name__ == "__main__":
    main()
