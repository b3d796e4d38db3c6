#!/usr/bin/env python3
"""Benchmark: PBB decode attention-core throughput on one MI355X.

One step = one fused ring-append + PBB-attention launch (``pbb_decode_step``) for every
sequence of the batch, followed by the position advance ``pos += 1`` on the same stream.
Inputs are seeded synthetic tensors already resident in HBM; rings are pre-filled.

Default workload (c3): batch 256, Hq 32, Hkv 8, head_dim 128, B 2048, bf16, positions
uniform in [0, 512K).  Also reported: the same-library sliding-window ring on the same
tensors (W = 2B = 4096 in 4096 slots, plus the paper-matched W = B), the ragged GQA-8
workload (c4), the paper-shape latency sweep, small-batch latency at c3's head shapes, and
prefill (PBB and SWA) in TFLOP/s against
the bf16 matrix-core peak, and the training backward of the same shapes.

Prints ONE JSON line.  Roofline: algorithmic bytes of the support actually read (ring K and
V rows of |A(t)| - 1 sources, q, out, the new K/V and their slot write, pos) divided by the
decode kernel's mean duration from HIP events on the launch stream, against 8 TB/s.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

HBM_PEAK_GBPS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "PBB decode attention-core tokens/s + achieved HBM GB/s (% of peak), 1 GPU"


def support_size(t, cfg):
    """|A(t)| for each position (PBB: t - a(t) + 1 with a(t) = max(0, h(floor(t/h) - 1));
    SWA: min(t + 1, W))."""
    import torch
    if cfg.mode == "swa":
        return torch.clamp(t + 1, max=cfg.window)
    h = cfg.block // 2
    a = torch.clamp(h * (torch.div(t, h, rounding_mode="floor") - 1), min=0)
    return t - a + 1


def step_bytes(t, cfg):
    """Algorithmic HBM bytes of one decode step for positions ``t`` (int64 [batch])."""
    u = 4 if cfg.dtype == "f32" else 2
    n = support_size(t, cfg) - 1
    per_seq = n * 2 * cfg.hkv * cfg.d * u + 2 * cfg.hq * cfg.d * u + 4 * cfg.hkv * cfg.d * u + 4
    return int(per_seq.sum())


_DECODE_SOURCES = ("pbb_kernels.hip", "pbb_device.h", "pbb_internal.h", "pbb_api.cpp")


def _code_only(text):
    """Source text without // comments, blank lines and runs of whitespace."""
    out = []
    for ln in text.splitlines():
        ln = re.sub(r"\s+", " ", re.sub(r"//.*$", "", ln)).strip()
        if ln:
            out.append(ln)
    return "\n".join(out)


def _kernel_hash(read=None):
    """Hash of the code that defines and selects the decode kernels (counter summaries are tied
    to it; comments do not count).  ``read(name)`` returns a source's text (default: the
    working tree)."""
    if read is None:
        def read(name):
            with open(os.path.join(ROOT, "paper_2606_02680_amd", "csrc", name)) as fh:
                return fh.read()
    h = hashlib.sha256()
    for f in _DECODE_SOURCES:
        h.update(_code_only(read(f)).encode())
    return h.hexdigest()[:16]


def _profile_values(workload_key):
    """Values of the committed rocprofv3 counter summary of one decode workload, or None when
    it is missing or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"decode_bf16_{workload_key}_counters.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for ln in f:
            if ":" in ln:
                k, v = ln.split(":", 1)
                vals[k.strip()] = v.strip().split()[0] if v.strip() else ""
    if vals.get("kernel_source_hash") != _kernel_hash():
        return None
    return vals


def _traffic_from_profile(workload_key):
    """HBM bytes per launch (FETCH_SIZE and WRITE_SIZE, scaled by the copy calibration) from
    the committed counter summary, or None (see _profile_values)."""
    vals = _profile_values(workload_key)
    try:
        return float(vals["hbm_bytes_per_launch_scaled"]) if vals else None
    except (KeyError, ValueError):
        return None


def _traffic_ratio_from_profile(workload_key):
    """Counter traffic over the algorithmic bytes of the same profiled launches, or None."""
    vals = _profile_values(workload_key)
    try:
        return (float(vals["hbm_bytes_per_launch_scaled"]) /
                float(vals["algorithmic_bytes_per_launch"])) if vals else None
    except (KeyError, ValueError, ZeroDivisionError):
        return None


class Workload:
    """Rings + pre-generated per-step inputs for one config, resident on the GPU."""

    def __init__(self, cfg, t0, n_steps, device, inputs=None):
        import torch
        import paper_2606_02680_amd as P
        import workloads as W
        self.cfg, self.t0, self.device = cfg, t0, device
        dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        if cfg.mode == "swa":
            self.desc = P.make_desc(cfg.batch, cfg.hq, cfg.hkv, cfg.d, window=cfg.window,
                                    slots=cfg.slots, dtype=dt, rope_base=cfg.rope_base)
            self.fn = P.swa_decode_step
            self.fn_advance = P.swa_decode_step_advance
        else:
            self.desc = P.make_desc(cfg.batch, cfg.hq, cfg.hkv, cfg.d, block=cfg.block, dtype=dt,
                                    rope_base=cfg.rope_base)
            self.fn = P.pbb_decode_step
            self.fn_advance = P.pbb_decode_step_advance
        self.k_ring, self.v_ring = P.alloc_rings(self.desc, device)
        self.ws = P.alloc_workspace(self.desc, device)
        P.ring_init(self.desc, self.k_ring, self.v_ring)
        self.pos0 = t0.to(torch.int32).to(device)
        self.pos = self.pos0.clone()
        self.pos_next = torch.empty_like(self.pos)
        L = self.desc.slots
        ks = W.kv_window(cfg, "k", t0, L, device=device)
        vs = W.kv_window(cfg, "v", t0, L, device=device)
        P.ring_fill(self.desc, self.pos, ks, vs, self.k_ring, self.v_ring)
        del ks, vs
        if inputs is None:
            inputs = (W.q_steps(cfg, t0, 0, n_steps, device=device),
                      W.kv_steps(cfg, "k", t0, 0, n_steps, device=device),
                      W.kv_steps(cfg, "v", t0, 0, n_steps, device=device))
        self.inputs = inputs
        self.out = torch.empty_like(inputs[0][0])
        torch.cuda.synchronize()

    def step(self, i):
        q, k, v = self.inputs[0][i], self.inputs[1][i], self.inputs[2][i]
        self.fn(self.desc, self.pos, q, k, v, self.k_ring, self.v_ring, self.out, self.ws)

    def timed(self, warmup, steps, graph=True):
        """Time ``steps`` decode steps after ``warmup`` untimed ones.  A timed step is one
        launch: the positions advance on the device inside the decode kernel
        (``*_decode_step_advance`` writing pos + 1 into a second position buffer, the two
        buffers alternating), as the paper's decode loop advances them on the device.

        Two passes over the same steps from the same state (rings and positions restored from a
        snapshot taken after the warmup):
          * graph (``graph=True``): the launches captured as one HIP graph, replayed once
            untimed and once timed -> ``wall_s``, the wall clock of the whole replay between
            two synchronisations (the throughput figure), and ``graph_event_s``, HIP events
            on the launch stream around it;
          * eager: back-to-back launches on one stream with HIP events around each launch on
            that stream -> ``eager_kernel_s``, the mean of those per-launch intervals.
        ``kernel_s`` (the roofline's duration) is ``graph_event_s`` per step with ``graph``: the
        mean launch duration over the timed region, the short gaps between graph nodes
        included; a pair of events around every eager launch adds a few microseconds of
        launch overhead to each interval (rocprof's kernel durations agree with the graph
        figure, and sit ~2% below the per-launch one).  Without ``graph``, ``kernel_s`` is
        ``eager_kernel_s`` and ``wall_s`` the eager loop's wall clock.  ``bytes``: algorithmic
        bytes of the timed steps (their actual positions)."""
        import torch
        for i in range(warmup):
            self.step(i)
            self.pos += 1
        torch.cuda.synchronize()
        total_bytes = 0
        t_first = (self.t0 + warmup)
        for i in range(steps):
            total_bytes += step_bytes(t_first + i, self.cfg)
        snap = (self.k_ring.clone(), self.v_ring.clone(), self.pos.clone())
        bufs = (self.pos, self.pos_next)

        def restore():
            self.k_ring.copy_(snap[0])
            self.v_ring.copy_(snap[1])
            self.pos.copy_(snap[2])
            torch.cuda.synchronize()

        def launch(i):
            j = warmup + i
            self.fn_advance(self.desc, bufs[i % 2], bufs[(i + 1) % 2], self.inputs[0][j],
                            self.inputs[1][j], self.inputs[2][j], self.k_ring, self.v_ring,
                            self.out, self.ws)

        res = {"bytes": total_bytes}
        if graph:
            restore()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(steps):
                    launch(i)
            restore()
            g.replay()                  # first replay: untimed
            restore()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            w0 = time.perf_counter()
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            res["wall_s"] = time.perf_counter() - w0
            res["graph_event_s"] = e0.elapsed_time(e1) / 1e3
            del g
        restore()
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
        ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
        w0 = time.perf_counter()
        for i in range(steps):
            starts[i].record()
            launch(i)
            ends[i].record()
        torch.cuda.synchronize()
        res["eager_wall_s"] = time.perf_counter() - w0
        if steps % 2:
            self.pos.copy_(self.pos_next)   # self.pos holds the next position, as after step()
        res["eager_kernel_s"] = sum(s.elapsed_time(e) for s, e in zip(starts, ends)) / 1e3 / steps
        if graph:
            res["kernel_s"] = res["graph_event_s"] / steps
        else:
            res["kernel_s"] = res["eager_kernel_s"]
            res["wall_s"] = res["eager_wall_s"]
        del snap
        return res


def _tup(res):
    """(wall seconds, mean kernel seconds, algorithmic bytes) of a Workload.timed result."""
    return res["wall_s"], res["kernel_s"], res["bytes"]


MFMA_BF16_PEAK_TFLOPS = 2500.0

# Prefill workloads (prompts at positions 0..n-1): c3's head shapes with a 16K prompt, and the
# paper's model shape (Hq 12, Hkv 2, d 64, B 128) with a 64K prompt.
PREFILL_SHAPES = (
    ("prefill_c3_shapes_pbb_b2048_n16384", dict(batch=4, n=16384, hq=32, hkv=8, d=128, block=2048)),
    ("prefill_c3_shapes_swa_w4096_n16384", dict(batch=4, n=16384, hq=32, hkv=8, d=128, window=4096)),
    ("prefill_paper_shape_pbb_b128_n65536", dict(batch=1, n=65536, hq=12, hkv=2, d=64, block=128)),
    ("prefill_paper_shape_swa_w128_n65536", dict(batch=1, n=65536, hq=12, hkv=2, d=64, window=128)),
)


def prefill_support_total(n, block=0, window=0):
    """sum over t < n of |A(t)| (PBB interval form, or the window)."""
    import torch
    t = torch.arange(n, dtype=torch.int64)
    if block:
        h = block // 2
        lo = torch.clamp(h * (torch.div(t, h, rounding_mode="floor") - 1), min=0)
    else:
        lo = torch.clamp(t - window + 1, min=0)
    return int((t - lo + 1).sum())


def prefill_measure(device, batch, n, hq, hkv, d, block=0, window=0, reps=10):
    """Median kernel time of one prefill launch (HIP events on the launch stream) and its
    algorithmic rate: 4 * d * Hq * batch * sum_t |A(t)| FLOP (scores and value products)."""
    import torch
    import paper_2606_02680_amd as P
    import workloads as W
    mode = "pbb" if block else "swa"
    cfg = W.Config(f"prefill-{mode}", mode, batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                   slots=block or window, window=window, dtype="bf16", seed=7, value_scale=1.0,
                   pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=device)
    if block:
        desc = P.make_desc(batch, hq, hkv, d, block=block, dtype=torch.bfloat16)
        fn = P.pbb_prefill
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=window, slots=window, dtype=torch.bfloat16)
        fn = P.swa_prefill
    out = torch.empty_like(q)
    lse = torch.empty((batch, hq, n), dtype=torch.float32, device=device)
    kr, vr = P.alloc_rings(desc, device)
    stream = torch.cuda.current_stream()
    for _ in range(2):
        fn(desc, q, k, v, out, lse, kr, vr, stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(stream)
        fn(desc, q, k, v, out, lse, kr, vr, stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[reps // 2]
    flops = 4.0 * d * hq * batch * prefill_support_total(n, block, window)
    # q, k, v read, out written (bf16), lse written (fp32), the ring's last `slots` rows written
    nbytes = (batch * n * (2 * hq + 2 * hkv) * d * 2 + batch * hq * n * 4
              + 2 * batch * hkv * min(n, block or window) * d * 2)
    return _rates(ms, flops, nbytes, batch * n)


def _rates(ms, flops, nbytes, tokens):
    """Rates of one launch (or call) against both ceilings; `bound` names the one whose floor
    time (algorithmic FLOPs at the bf16 matrix-core peak, or algorithmic bytes at 8 TB/s) is
    longer, and `frac_of_bound` is that floor over the measured time."""
    tflops = flops / (ms * 1e-3) / 1e12
    gbps = nbytes / (ms * 1e-3) / 1e9
    t_mfma = flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    t_hbm = nbytes / (HBM_PEAK_GBPS * 1e9)
    bound = "mfma" if t_mfma >= t_hbm else "hbm"
    return {"kernel_ms": ms, "tflops": tflops, "frac_of_bf16_mfma_peak": tflops / MFMA_BF16_PEAK_TFLOPS,
            "hbm_gbps": gbps, "frac_of_hbm_peak": gbps / HBM_PEAK_GBPS, "bound": bound,
            "frac_of_bound": max(t_mfma, t_hbm) / (ms * 1e-3),
            "tokens_per_s": tokens / (ms * 1e-3), "algorithmic_tflop": flops / 1e12,
            "algorithmic_gb": nbytes / 1e9}


def prefill_extras(device):
    res = {}
    for name, shape in PREFILL_SHAPES:
        res[name] = prefill_measure(device, **shape)
    return res


def backward_measure(device, batch, n, hq, hkv, d, block=0, window=0, reps=10):
    """Median time of one backward call (delta, dq and dk/dv launches; HIP events on the launch
    stream) after a prefill supplied ``out`` and ``lse``; algorithmic rate
    10 * d * Hq * batch * sum_t |A(t)| FLOP (the five products per covered pair: scores,
    dout.v, dq, dk, dv; the kernels recompute the first two once more in the dk/dv pass)."""
    import torch
    import paper_2606_02680_amd as P
    import workloads as W
    mode = "pbb" if block else "swa"
    cfg = W.Config(f"backward-{mode}", mode, batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                   slots=block or window, window=window, dtype="bf16", seed=7, value_scale=1.0,
                   pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=device)
    dout, _, _ = W.prompt(cfg.with_(seed=8), n, device=device)
    if block:
        desc = P.make_desc(batch, hq, hkv, d, block=block, dtype=torch.bfloat16)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=window, slots=window, dtype=torch.bfloat16)
        fwd, bwd = P.swa_prefill, P.swa_backward
    out = torch.empty_like(q)
    lse = torch.empty((batch, hq, n), dtype=torch.float32, device=device)
    stream = torch.cuda.current_stream()
    fwd(desc, q, k, v, out, lse, stream=stream)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(P.backward_workspace_bytes(desc, n), dtype=torch.uint8, device=device)
    for _ in range(2):
        bwd(desc, q, k, v, out, dout, lse, dq, dk, dv, workspace=ws, stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(stream)
        bwd(desc, q, k, v, out, dout, lse, dq, dk, dv, workspace=ws, stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[reps // 2]
    flops = 10.0 * d * hq * batch * prefill_support_total(n, block, window)
    # q, k, v, out, dout read and dq, dk, dv written (bf16), lse read (fp32)
    nbytes = batch * n * (4 * hq + 4 * hkv) * d * 2 + batch * hq * n * 4
    return _rates(ms, flops, nbytes, batch * n)


BACKWARD_SHAPES = tuple((name.replace("prefill", "backward"), shape)
                        for name, shape in PREFILL_SHAPES)


def backward_extras(device):
    return {name: backward_measure(device, **shape) for name, shape in BACKWARD_SHAPES}


def small_batch_latency(device, batches=(1, 4), steps=64, reps=7):
    """Decode latency at c3's head shapes (B 2048; SWA W 4096 in 4096 slots) for small batches,
    where a launch has few (sequence, KV head) units and is split over workgroups: 64 steps of
    ``*_decode_step_advance`` captured as one HIP graph, median replay time / 64."""
    import statistics
    import torch
    import paper_2606_02680_amd as P
    import workloads as W
    res = {}
    for batch in batches:
        for name in ("c3", "c5"):
            cfg = W.get_config(name).with_(batch=batch)
            t0 = W.initial_positions(cfg)
            wl = Workload(cfg, t0, steps, device)
            qs, ks, vs = wl.inputs
            adv = P.swa_decode_step_advance if cfg.mode == "swa" else P.pbb_decode_step_advance
            pos = [wl.pos.clone(), torch.zeros_like(wl.pos)]
            out = torch.empty_like(qs[0])
            snap = (wl.k_ring.clone(), wl.v_ring.clone())
            g = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                for i in range(steps):
                    adv(wl.desc, pos[i % 2], pos[(i + 1) % 2], qs[i], ks[i], vs[i], wl.k_ring,
                        wl.v_ring, out, wl.ws)
            times = []
            for _ in range(reps):
                wl.k_ring.copy_(snap[0])
                wl.v_ring.copy_(snap[1])
                pos[0].copy_(wl.pos0)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                g.replay()
                e1.record()
                torch.cuda.synchronize()
                times.append(e0.elapsed_time(e1) * 1e3 / steps)
            key = f"{'pbb_b2048' if cfg.mode == 'pbb' else 'swa_w4096'}_batch{batch}"
            res[key] = {"us_per_step": statistics.median(times),
                        "workspace_bytes": 0 if wl.ws is None else wl.ws.numel()}
            del g, wl, snap
            torch.cuda.empty_cache()
    return res


PAPER_ORIGINS = (8192, 16384, 32768, 65536, 131072, 262144, 524288, 1048576)


def paper_latency(device, shapes=(10, 12, 14), origins=(8192,), steps=256, reps=9):
    """The paper's latency-bound decode shape (batch 1, Hkv 2, head_dim 64, B 128; SWA w 128):
    per (query heads, origin), 256 steps of decode + on-device position advance (one
    ``*_decode_step_advance`` launch per step, alternating two position buffers) are captured as
    one HIP graph and replayed ``reps`` times from the same restored state; the median replay
    time / 256 is the per-step latency.  SWA runs in a 256-slot ring (the paper's SWA backend
    allocated 256 positions) and in a 128-slot ring."""
    import statistics

    import torch
    import paper_2606_02680_amd as P
    import workloads as W
    res = {}
    for hq in shapes:
        for origin in origins:
            base = dict(batch=1, hq=hq, hkv=2, d=64, dtype="bf16", seed=11, value_scale=1.0,
                        pos_hi=0, steps=steps, prefill=True)
            cfgs = {"pbb_b128": W.Config("paper-pbb", "pbb", block=128, slots=128, window=0, **base),
                    "swa_w128_s256": W.Config("paper-swa", "swa", block=128, slots=256, window=128,
                                              **base),
                    "swa_w128_s128": W.Config("paper-swa", "swa", block=128, slots=128, window=128,
                                              **base)}
            t0 = torch.tensor([origin], dtype=torch.int64)
            cell = {}
            inputs = None
            for name, c in cfgs.items():
                wl = Workload(c, t0, steps, device, inputs=inputs)
                inputs = wl.inputs
                snap = (wl.k_ring.clone(), wl.v_ring.clone(), wl.pos0.clone())
                outs = torch.empty_like(inputs[0])
                pos2 = (wl.pos, torch.empty_like(wl.pos))
                adv = P.swa_decode_step_advance if c.mode == "swa" else P.pbb_decode_step_advance

                def restore():
                    wl.k_ring.copy_(snap[0]); wl.v_ring.copy_(snap[1]); pos2[0].copy_(snap[2])

                restore()
                g = torch.cuda.CUDAGraph()
                torch.cuda.synchronize()
                with torch.cuda.graph(g):
                    # one kernel per step: decode + position advance into the other buffer
                    for i in range(steps):
                        adv(wl.desc, pos2[i % 2], pos2[(i + 1) % 2], inputs[0][i], inputs[1][i],
                            inputs[2][i], wl.k_ring, wl.v_ring, outs[i], wl.ws)
                times = []
                for _ in range(reps + 1):
                    restore()
                    torch.cuda.synchronize()
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    g.replay()
                    e1.record()
                    torch.cuda.synchronize()
                    times.append(e0.elapsed_time(e1) * 1e3 / steps)
                cell[f"{name}_us"] = statistics.median(times[1:])
                del g, wl
            cell["pbb_over_swa_s256"] = cell["swa_w128_s256_us"] / cell["pbb_b128_us"]
            cell["pbb_over_swa_s128"] = cell["swa_w128_s128_us"] / cell["pbb_b128_us"]
            res[f"hq{hq}_origin{origin}"] = cell
    return res


def _host_cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            return next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        return ""


def _bf16_round(x):
    """float64 -> nearest bfloat16 value, ties to even (8 significant bits)."""
    import numpy as np
    out = np.zeros_like(x)
    nz = x != 0
    ulp = np.exp2(np.floor(np.log2(np.abs(x[nz]))) - 7)
    out[nz] = np.round(x[nz] / ulp) * ulp
    return out


def _error_stats(got, ref):
    """max |got - ref|, max |got - bf16(ref)|, worst relative L2 and cosine per (seq, head)."""
    import numpy as np
    g = got.reshape(-1, got.shape[-1]).astype(np.float64)
    r = ref.reshape(-1, ref.shape[-1])
    rn = np.linalg.norm(r, axis=1)
    return {"max_abs": float(np.abs(g - r).max()),
            "max_abs_vs_bf16_ref": float(np.abs(g - _bf16_round(r)).max()),
            "rel_l2_max": float((np.linalg.norm(g - r, axis=1) / np.maximum(rn, 1e-30)).max()),
            "cos_min": float(((g * r).sum(1) / np.maximum(np.linalg.norm(g, axis=1) * rn,
                                                          1e-30)).min())}


def cpu_baseline(cfg, t0, device, budget_s=10.0, max_steps=64, threads=None,
                 single_thread=True):
    """The fp64 CPU oracle timed on FULL-BATCH decode steps of the workload: steps 0, 1, 2, ..
    (every sequence, every query head) with all host threads until ``budget_s`` seconds have
    passed (at least 3 steps, at most ``max_steps``), then one full-batch step single-threaded.
    The same steps are also run on the GPU from the same ring state, and the oracle's outputs
    are compared with them (error statistics, outside the clock)."""
    import numpy as np
    import torch
    import oracle
    import workloads as W
    if threads is None:
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 1)
    n = cfg.batch
    rows = torch.arange(n, dtype=torch.int64)
    back = cfg.slots
    lo = (t0 - back).numpy()
    hpos = torch.as_tensor(lo).view(-1, 1) + torch.arange(0, back + max_steps,
                                                          dtype=torch.int64).view(1, -1)
    kh = np.empty((n, cfg.hkv, back + max_steps, cfg.d), dtype=np.float32)
    vh = np.empty_like(kh)
    for c0 in range(0, n, 32):
        kh[c0:c0 + 32] = W.kv_at(cfg, "k", rows[c0:c0 + 32], hpos[c0:c0 + 32],
                                 device=device).float().cpu().numpy()
        vh[c0:c0 + 32] = W.kv_at(cfg, "v", rows[c0:c0 + 32], hpos[c0:c0 + 32],
                                 device=device).float().cpu().numpy()
    # GPU outputs of the same steps from the pre-filled rings
    wl = Workload(cfg, t0, max_steps, device)
    gpu_out = []
    for i in range(max_steps):
        wl.step(i)
        wl.pos += 1
        gpu_out.append(wl.out.float().cpu().numpy())
    qs = wl.inputs[0].float().cpu().numpy()
    del wl
    torch.cuda.empty_cache()
    mode = oracle.SWA if cfg.mode == "swa" else oracle.PBB
    t0n = t0.numpy().astype(np.int64)
    oracle.decode(mode, t0n[:1], qs[0][:1], kh[:1], vh[:1], lo[:1], block=cfg.block,
                  window=cfg.window, n_threads=1)  # load the library outside the clock
    refs = []
    w0 = time.perf_counter()
    while len(refs) < max_steps:
        i = len(refs)
        refs.append(oracle.decode(mode, t0n + i, qs[i], kh, vh, lo, block=cfg.block,
                                  window=cfg.window, n_threads=threads))
        if len(refs) >= 3 and time.perf_counter() - w0 >= budget_s:
            break
    el = time.perf_counter() - w0
    res = {"value": n * len(refs) / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"{len(refs)} full-batch decode steps of {cfg.name} (all {n} sequences x "
                     f"{cfg.hq} query heads each, positions t0+0..t0+{len(refs) - 1}) in "
                     f"{el:.1f} s; fp64 C oracle with {threads} threads on the host CPU "
                     f"({_host_cpu_model()}, {os.cpu_count()} logical CPUs visible)",
           "host_cpu": _host_cpu_model()}
    if single_thread:
        w0 = time.perf_counter()
        oracle.decode(mode, t0n, qs[0], kh, vh, lo, block=cfg.block, window=cfg.window,
                      n_threads=1)
        res["single_thread_value"] = n / (time.perf_counter() - w0)
    stats = None
    for i, ref in enumerate(refs):
        e = _error_stats(gpu_out[i], ref)
        stats = e if stats is None else {k: (min(stats[k], e[k]) if k == "cos_min"
                                             else max(stats[k], e[k])) for k in e}
    res["gpu_vs_oracle"] = dict(stats, steps=len(refs))
    return res


PROBE_LIB = os.path.join(ROOT, "paper_2606_02680_amd", "libpbbprobe.so")


def stream_probe(device, cfg, t0, waves, nontemporal=True, equal=False, reps=10):
    """Practical read rate of the decode's streaming pattern (include/pbb_probe.h): every
    (sequence, KV head) unit of ``cfg`` reads its K and V rows through LDS DMA, two 32-row steps
    in flight per wave, ``waves`` waves per unit, no arithmetic.  Rows per unit: the support's
    ring rows at positions ``t0`` (|A(t)| - 1, the decode's ragged sizes), or the whole ring
    minus one row with ``equal``.  Returns GB/s (rows actually read / median launch time from
    HIP events on the launch stream) and the bytes per launch."""
    import ctypes
    import torch
    if not os.path.exists(PROBE_LIB):
        raise ImportError(f"{PROBE_LIB} not found: build it with `python -m paper_2606_02680_amd.build`")
    lib = ctypes.CDLL(PROBE_LIB)
    vp = ctypes.c_void_p
    lib.pbb_probe_stream.argtypes = [vp, vp, ctypes.c_size_t, vp, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, vp, vp]
    lib.pbb_probe_stream.restype = ctypes.c_int
    assert cfg.d == 128 and cfg.dtype == "bf16"
    units, slots = cfg.batch * cfg.hkv, cfg.slots
    k = torch.empty(units * slots * 128, dtype=torch.bfloat16, device=device)
    v = torch.empty_like(k)
    per_seq = (torch.full_like(t0, slots - 1) if equal else support_size(t0, cfg) - 1)
    rows = per_seq.view(-1, 1).expand(-1, cfg.hkv).reshape(-1).to(torch.int32).to(device)
    sink = torch.zeros(1, dtype=torch.float32, device=device)
    stream = torch.cuda.current_stream()

    def launch():
        rc = lib.pbb_probe_stream(vp(k.data_ptr()), vp(v.data_ptr()), ctypes.c_size_t(slots * 256),
                                  vp(rows.data_ptr()), units, slots, waves, int(nontemporal),
                                  vp(sink.data_ptr()), vp(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"pbb_probe_stream failed ({rc})")

    for _ in range(2):
        launch()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(stream)
        launch()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[reps // 2]
    nbytes = 2 * 256 * int(rows.to(torch.int64).sum())
    del k, v
    torch.cuda.empty_cache()
    return {"gbps": nbytes / (ms * 1e-3) / 1e9, "bytes_per_launch": nbytes, "us": ms * 1e3,
            "waves": waves, "nontemporal": bool(nontemporal),
            "rows": "whole ring" if equal else "support (ragged)"}


def stream_probes(device, steps_offset=0):
    """The probe at the decode workloads' shapes and launch shapes (c3, c4; c5's equal rows)."""
    import workloads as W
    res = {}
    c3, c4, c5 = W.get_config("c3"), W.get_config("c4"), W.get_config("c5")
    t3 = W.initial_positions(c3) + steps_offset
    t4 = W.initial_positions(c4) + steps_offset
    res["c3_ragged_nw4"] = stream_probe(device, c3, t3, 4)
    res["c3_equal_nw4"] = stream_probe(device, c3, t3, 4, equal=True)
    res["c4_ragged_nw2"] = stream_probe(device, c4, t4, 2)
    res["c4_ragged_nw4"] = stream_probe(device, c4, t4, 4)
    res["c5_equal_nw4"] = stream_probe(device, c5, t3, 4, equal=True)
    return res


def copy_ceiling(device, reps=5):
    """HBM rate of a plain 1 GiB device-to-device copy (bytes read + written per second, HIP
    events on the copy's stream): the measured ceiling the decode rate is also compared with."""
    import torch
    n = 1 << 29  # 1 GiB of bf16
    x = torch.ones(n, dtype=torch.bfloat16, device=device)
    y = torch.empty_like(x)
    y.copy_(x)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        y.copy_(x)
    e1.record(stream)
    torch.cuda.synchronize()
    gbps = 4.0 * n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x, y
    torch.cuda.empty_cache()
    return gbps


def oracle_all_steps(cfg, device, threads=None):
    """Time the fp64 CPU oracle over every step of a lockstep workload (all sequences at
    positions 0, 1, .., steps-1; the whole history handed over once, as the oracle reads only
    each step's support)."""
    import numpy as np
    import torch
    import oracle
    import workloads as W
    if threads is None:
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 1)
    n, T = cfg.batch, cfg.steps
    rows = torch.arange(n, dtype=torch.int64)
    posm = torch.arange(T, dtype=torch.int64).view(1, -1).expand(n, T)
    kh = W.kv_at(cfg, "k", rows, posm, device=device).float().cpu().numpy()
    vh = W.kv_at(cfg, "v", rows, posm, device=device).float().cpu().numpy()
    qs = W.q_steps(cfg, torch.zeros(n, dtype=torch.int64), 0, T, device=device).float().cpu().numpy()
    lo = np.zeros(n, dtype=np.int64)
    mode = oracle.SWA if cfg.mode == "swa" else oracle.PBB
    w0 = time.perf_counter()
    for t in range(T):
        oracle.decode(mode, np.full(n, t, dtype=np.int64), qs[t], kh, vh, lo, block=cfg.block,
                      window=cfg.window, n_threads=threads)
    el = time.perf_counter() - w0
    return {"value": n * T / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"all {T} steps of {cfg.name} ({n} sequences in lockstep from position 0) "
                      f"in {el:.1f} s; fp64 C oracle, {threads} threads"}


def oracle_timing(device):
    """The fp64 CPU oracle: every step of c1 and c2, and full-batch decode steps of c3, c4 and
    c5 (at least three and 5 s each with all host threads, plus one single-threaded step)."""
    import workloads as W
    res = {"host_threads": os.cpu_count()}
    for name in ("c1", "c2"):
        res[name] = oracle_all_steps(W.get_config(name), device)
    for name in ("c3", "c4", "c5"):
        cfg = W.get_config(name)
        t0 = W.initial_positions(cfg)
        res[name] = cpu_baseline(cfg, t0, device, budget_s=5.0)
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c3", choices=["c3", "c4", "c5"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the SWA-ring and ragged-batch comparison runs")
    ap.add_argument("--paper-latency", action="store_true",
                    help="only run the paper-shape latency sweep (3 shapes x 8 origins)")
    ap.add_argument("--prefill", action="store_true",
                    help="only run the prefill measurements (c3 head shapes and paper shape)")
    ap.add_argument("--backward", action="store_true",
                    help="only run the training-backward measurements (same shapes as prefill)")
    ap.add_argument("--fp32", action="store_true",
                    help="only run fp32 decode at c3's and c4's shapes (and G = 1 variants)")
    ap.add_argument("--batch-sweep", action="store_true",
                    help="only run the decode at c3's head shapes for batches 16..1024")
    ap.add_argument("--small-batch", action="store_true",
                    help="only run the small-batch latency graphs (batches 1, 4, 8, 16 at c3's "
                         "head shapes; split launches up to 64 units)")
    ap.add_argument("--oracle-timing", action="store_true",
                    help="only time the CPU oracle (all steps of c1, c2; full batches of c3, c4, c5; minutes)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only time a plain 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--stream-probe", action="store_true",
                    help="only run the LDS-DMA streaming-read probe at the decode workloads' "
                         "shapes (the practical read ceiling)")
    ap.add_argument("--records", default=None,
                    help="also write one JSON record per measured workload to this file")
    ap.add_argument("--no-graph", action="store_true",
                    help="time the steps as eager back-to-back launches instead of a HIP graph")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the decode "
              "core shards by sequence or KV head with no exchange between GPUs)",
              file=sys.stderr)
        return 2

    import torch
    import workloads as W
    sys.path.insert(0, ROOT)
    import paper_2606_02680_amd as P
    P.load_library()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)

    if args.copy_probe:
        n = 1 << 29  # 1 GiB of bf16
        x = torch.ones(n, dtype=torch.bfloat16, device=device)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        el = (time.perf_counter() - w0) / 5
        print(json.dumps({"copy_probe_bytes_read": 2 * n, "copy_probe_bytes_written": 2 * n,
                          "copy_probe_gbps_read_plus_write": 4 * n / el / 1e9}), flush=True)
        return 0

    if args.prefill:
        print(json.dumps({"prefill": prefill_extras(device)}), flush=True)
        return 0

    if args.stream_probe:
        print(json.dumps({"stream_probe": stream_probes(device)}), flush=True)
        return 0

    if args.oracle_timing:
        print(json.dumps({"oracle_timing": oracle_timing(device)}), flush=True)
        return 0

    if args.backward:
        print(json.dumps({"backward": backward_extras(device)}), flush=True)
        return 0

    if args.paper_latency:
        print(json.dumps({"paper_shape_latency_us_per_step":
                          paper_latency(device, origins=PAPER_ORIGINS)}), flush=True)
        return 0

    if args.fp32:
        res = {}
        for name, over in (("c3", {}), ("c4", {}), ("c3", {"hq": 8}), ("c4", {"hq": 2, "batch": 512})):
            c = W.get_config(name).with_(dtype="f32", **over)
            wl = Workload(c, W.initial_positions(c), 60, device)
            el, ks, tb = _tup(wl.timed(10, 50))
            key = f"{name}_shapes_fp32_G{c.hq // c.hkv}_batch{c.batch}"
            res[key] = {"kernel_us": ks * 1e6, "tokens_per_s": c.batch * 50 / el,
                        "hbm_gbps_kernel": tb / 50 / ks / 1e9,
                        "frac_of_peak": tb / 50 / ks / 1e9 / HBM_PEAK_GBPS}
            print(f"[bench] {key}: {ks * 1e6:.1f} us", file=sys.stderr, flush=True)
            del wl
            torch.cuda.empty_cache()
        print(json.dumps({"fp32_decode": res}), flush=True)
        return 0

    if args.batch_sweep:
        res = {}
        for batch in (16, 32, 64, 128, 256, 512, 1024):
            c = W.get_config("c3").with_(batch=batch)
            wl = Workload(c, W.initial_positions(c), 60, device)
            el, ks, tb = _tup(wl.timed(10, 50))
            res[f"batch{batch}"] = {"kernel_us": ks * 1e6, "tokens_per_s": batch * 50 / el,
                                    "hbm_gbps_kernel": tb / 50 / ks / 1e9,
                                    "frac_of_peak": tb / 50 / ks / 1e9 / HBM_PEAK_GBPS,
                                    "workspace_bytes": 0 if wl.ws is None else wl.ws.numel()}
            print(f"[bench] batch {batch}: {ks * 1e6:.1f} us", file=sys.stderr, flush=True)
            del wl
            torch.cuda.empty_cache()
        print(json.dumps({"batch_sweep_c3_heads": res}), flush=True)
        return 0

    if args.small_batch:
        print(json.dumps({"small_batch_latency_us_per_step":
                          small_batch_latency(device, batches=(1, 4, 8, 16))}), flush=True)
        return 0

    cfg = W.get_config(args.config)
    n_steps = args.warmup + args.steps
    t0 = W.initial_positions(cfg)
    print(f"[bench] preparing {cfg.name} ({n_steps} steps of inputs)", file=sys.stderr, flush=True)
    wl = Workload(cfg, t0, n_steps, device)
    tm = wl.timed(args.warmup, args.steps, graph=not args.no_graph)
    elapsed, kern_s, total_bytes = tm["wall_s"], tm["kernel_s"], tm["bytes"]
    tokens = cfg.batch * args.steps
    value = tokens / elapsed
    achieved = total_bytes / args.steps / kern_s / 1e9
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: batch {cfg.batch}, Hq {cfg.hq}, Hkv {cfg.hkv}, "
                               f"head_dim {cfg.d}, B {cfg.block}, ring {cfg.slots} slots, "
                               f"positions U[0,{cfg.pos_hi}), pre-filled rings",
                   "batch": cfg.batch, "n_q_heads": cfg.hq, "n_kv_heads": cfg.hkv,
                   "head_dim": cfg.d, "block": cfg.block, "slots": cfg.slots,
                   "window": cfg.window, "parallelism": "single GPU"},
        "timing": ("steps captured as one HIP graph (one launch per step, positions advanced on "
                   "the device): value from the wall clock of the replay, kernel time (roofline) "
                   "from HIP events on the launch stream around the replay, per step; a second, "
                   "eager pass over the same steps with HIP events around each launch gives "
                   "eager_kernel_us"
                   if not args.no_graph else
                   "eager back-to-back launches with HIP events around each launch"),
        "hbm_gbps_step": total_bytes / elapsed / 1e9,
        "bytes_per_token": total_bytes / tokens,
        "kernel_us": kern_s * 1e6,
        "eager_kernel_us": tm["eager_kernel_s"] * 1e6,
        "eager_ms_per_step": tm["eager_wall_s"] / args.steps * 1e3,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": _traffic_from_profile(args.config)},
    }
    if "graph_event_s" in tm:
        result["graph_event_us_per_step"] = tm["graph_event_s"] / args.steps * 1e6
    print(f"[bench] {cfg.name}: {value:.4g} tokens/s, kernel {kern_s * 1e6:.1f} us, "
          f"{achieved:.1f} GB/s", file=sys.stderr, flush=True)

    if not args.no_extras and args.config == "c3":
        extra = {}
        ext_steps = min(args.steps, 200)
        inputs = wl.inputs
        del wl
        torch.cuda.empty_cache()
        # SWA rings on the same tensors: the graded W = 2B window, and the paper's own
        # comparison window W = B in a buffer of 2B slots and in a ring of B slots.
        for name, c in (("swa_ring_w4096_s4096", W.get_config("c5")),
                        ("swa_ring_w2048_s4096", W.get_config("c5").with_(window=2048,
                                                                          slots=4096)),
                        ("swa_ring_w2048_s2048", W.get_config("c5").with_(window=2048,
                                                                          slots=2048))):
            sw = Workload(c, t0, n_steps, device, inputs=inputs)
            el, ks, tb = _tup(sw.timed(args.warmup, ext_steps))
            extra[name] = {"tokens_per_s": cfg.batch * ext_steps / el, "kernel_us": ks * 1e6,
                           "bytes_per_token": tb / (cfg.batch * ext_steps),
                           "hbm_gbps_kernel": tb / ext_steps / ks / 1e9,
                           "frac_of_peak": tb / ext_steps / ks / 1e9 / HBM_PEAK_GBPS,
                           "pbb_over_swa_tokens_per_s": value / (cfg.batch * ext_steps / el)}
            if name == "swa_ring_w4096_s4096":
                extra[name]["traffic"] = _traffic_from_profile("c5")
                extra[name]["traffic_over_algorithmic"] = _traffic_ratio_from_profile("c5")
            del sw
            torch.cuda.empty_cache()
        # The same step with the rotary embedding fused in (q and the new key turned by position,
        # base 10^6): timing only, so the pre-filled ring is not re-rotated.
        rw = Workload(cfg.with_(rope_base=1e6), t0, n_steps, device, inputs=inputs)
        el, ks, tb = _tup(rw.timed(args.warmup, ext_steps))
        extra["c3_rope_base1e6"] = {"tokens_per_s": cfg.batch * ext_steps / el,
                                    "kernel_us": ks * 1e6,
                                    "hbm_gbps_kernel": tb / ext_steps / ks / 1e9,
                                    "kernel_us_over_plain": ks / kern_s}
        del rw
        del inputs
        torch.cuda.empty_cache()
        c4 = W.get_config("c4")
        t4 = W.initial_positions(c4)
        w4 = Workload(c4, t4, args.warmup + ext_steps, device)
        el, ks, tb = _tup(w4.timed(args.warmup, ext_steps))
        extra["c4_ragged_gqa8"] = {"tokens_per_s": c4.batch * ext_steps / el,
                                   "kernel_us": ks * 1e6,
                                   "bytes_per_token": tb / (c4.batch * ext_steps),
                                   "hbm_gbps_kernel": tb / ext_steps / ks / 1e9,
                                   "frac_of_peak": tb / ext_steps / ks / 1e9 / HBM_PEAK_GBPS,
                                   "traffic": _traffic_from_profile("c4"),
                                   "traffic_over_algorithmic": _traffic_ratio_from_profile("c4")}
        del w4
        torch.cuda.empty_cache()
        extra["paper_shape_latency_us_per_step"] = paper_latency(
            device, shapes=(10, 12, 14), origins=(8192, 1048576))
        extra["small_batch_latency_us_per_step"] = small_batch_latency(device)
        extra["prefill"] = prefill_extras(device)
        extra["backward"] = backward_extras(device)
        copy_gbps = copy_ceiling(device)
        probes = stream_probes(device, steps_offset=args.warmup)
        extra["hbm_copy_ceiling"] = {
            "copy_gbps_read_plus_write": copy_gbps,
            "graded_kernel_frac_of_copy": achieved / copy_gbps,
            "stream_probe": probes,
            "graded_kernel_frac_of_stream_probe": achieved / probes["c3_ragged_nw4"]["gbps"],
            "c4_kernel_frac_of_stream_probe": (extra["c4_ragged_gqa8"]["hbm_gbps_kernel"] /
                                               probes["c4_ragged_nw2"]["gbps"])}
        result["extra"] = extra
        result["paper_context"] = ("Flash-PBB 1.82x Flash-SWA decode-core throughput on an RTX "
                                   "4090 (48 GB), BF16, batch 1, Hkv 2, d 64, b 128 vs w 128")

    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, t0, device)
    if args.records:
        write_records(args.records, result)
    print(json.dumps(result), flush=True)
    return 0


def write_records(path, result):
    """One JSON record per measured workload: throughput, time per step, bytes per token,
    achieved rate against 8 TB/s and the streaming probe, counter traffic where a committed
    summary matches the kernel, and the oracle comparison of the CPU-baseline leg."""
    extra = result.get("extra", {})
    probe = extra.get("hbm_copy_ceiling", {}).get("stream_probe", {})
    recs = [{"workload": result["config"]["workload"], "tokens_per_s": result["value"],
             "us_per_step": result["ms_per_step"] * 1e3, "kernel_us": result["kernel_us"],
             "bytes_per_token": result["bytes_per_token"],
             "gbps_kernel": result["roofline"]["achieved"],
             "frac_of_8tbps": result["roofline"]["frac"],
             "frac_of_stream_probe": (result["roofline"]["achieved"] /
                                      probe["c3_ragged_nw4"]["gbps"]) if probe else None,
             "traffic_bytes_per_launch": result["roofline"]["traffic"],
             "gpu_vs_oracle": result.get("cpu_baseline", {}).get("gpu_vs_oracle"),
             "oracle_tokens_per_s": result.get("cpu_baseline", {}).get("value")}]
    for name in ("swa_ring_w4096_s4096", "swa_ring_w2048_s4096", "swa_ring_w2048_s2048",
                 "c3_rope_base1e6", "c4_ragged_gqa8"):
        if name in extra:
            recs.append({"workload": name, **extra[name]})
    for group in ("prefill", "backward"):
        for name, r in extra.get(group, {}).items():
            recs.append({"workload": name, **r})
    for name, r in extra.get("paper_shape_latency_us_per_step", {}).items():
        recs.append({"workload": f"paper_shape_{name}", **r})
    with open(path, "w") as f:
        for r in recs:
            f.write(json.dumps(r) + "\n")


if __name__ == "__main__":
    sys.exit(main())
