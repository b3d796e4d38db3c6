"""Decode-run harness shared by the GPU parity tests.

Runs the HIP library through its C ABI on seeded inputs from :mod:`workloads` and compares
against the CPU oracle on the same inputs.  The oracle reads absolute-position history that
the generator produces independently of the ring.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W


def desc_for(cfg: W.Config, batch: int | None = None) -> P.PbbDesc:
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    b = cfg.batch if batch is None else batch
    if cfg.mode == "swa":
        return P.make_desc(b, cfg.hq, cfg.hkv, cfg.d, window=cfg.window, slots=cfg.slots, dtype=dt,
                           rope_base=cfg.rope_base)
    return P.make_desc(b, cfg.hq, cfg.hkv, cfg.d, block=cfg.block, dtype=dt,
                       rope_base=cfg.rope_base)


def bf16_tolerance_ok(got: np.ndarray, ref: np.ndarray):
    """Elementwise |got - ref| <= 2e-2 + 2^-8 |ref| (2e-2 plus one bf16 rounding half-ulp)."""
    return np.abs(got - ref) <= 2e-2 + np.abs(ref) * 2.0 ** -8


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits), ties to even,
    directly from float64 (no intermediate float32 rounding)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = x != 0
    e = np.floor(np.log2(np.abs(x[nz])))
    ulp = np.exp2(e - 7)
    out[nz] = np.round(x[nz] / ulp) * ulp   # np.round: half to even; the scaling is exact
    return out


def error_stats(got: np.ndarray, ref: np.ndarray) -> dict:
    """Secondary error metrics of a comparison (the paper reports max abs, relative L2 and
    cosine): strict max |got - ref|, max |got - bf16(ref)|, the largest |ref|, and the worst
    relative L2 and cosine over (sequence, head) rows."""
    got = got.astype(np.float64)
    g = got.reshape(-1, got.shape[-1])
    r = ref.reshape(-1, ref.shape[-1])
    rn = np.linalg.norm(r, axis=1)
    rel = np.linalg.norm(g - r, axis=1) / np.maximum(rn, 1e-30)
    cos = (g * r).sum(1) / np.maximum(np.linalg.norm(g, axis=1) * rn, 1e-30)
    err = np.abs(got - ref)
    return {"max_abs": float(err.max()),
            "argmax": [int(x) for x in np.unravel_index(np.argmax(err), err.shape)],
            "max_abs_vs_bf16_ref": float(np.abs(got - bf16_round(ref)).max()),
            "max_ref": float(np.abs(ref).max()),
            "rel_l2_max": float(rel.max()), "cos_min": float(cos.min())}


def merge_stats(a: dict | None, b: dict, where=None) -> dict:
    """Worst-case merge of two error_stats results; ``argmax`` follows the larger max_abs and
    is prefixed with ``where`` (e.g. step and first sequence of the chunk) when given."""
    b = dict(b)
    if where is not None and "argmax" in b:
        b["argmax"] = list(where) + b["argmax"]
    if a is None:
        return b
    out = {k: (min(a[k], b[k]) if k == "cos_min" else max(a[k], b[k]))
           for k in b if k != "argmax"}
    if "argmax" in b:
        out["argmax"] = b["argmax"] if b["max_abs"] > a["max_abs"] else a["argmax"]
    return out


def record_stats(name: str, stats: dict):
    """Print a parity record and append it to the JSON-lines file named by the environment
    variable PBB_PARITY_RECORD, if set."""
    import json
    import os
    line = json.dumps({"case": name, **stats})
    print(f"[parity-stats] {line}", flush=True)
    path = os.environ.get("PBB_PARITY_RECORD")
    if path:
        with open(path, "a") as f:
            f.write(line + "\n")


def compare(cfg: W.Config, got: np.ndarray, ref: np.ndarray, what: str = ""):
    """Assert the tolerance for the workload dtype; returns a metrics dict."""
    got = got.astype(np.float64)
    diff = np.abs(got - ref)
    metrics = {"max_abs": float(diff.max()) if diff.size else 0.0}
    if cfg.dtype == "f32":
        assert metrics["max_abs"] <= 1e-5, f"{what}: fp32 max abs {metrics['max_abs']:.3e} > 1e-5"
        return metrics
    ok = bf16_tolerance_ok(got, ref)
    if not ok.all():
        idx = np.unravel_index(np.argmax(diff - (2e-2 + np.abs(ref) * 2.0 ** -8)), diff.shape)
        raise AssertionError(f"{what}: bf16 tolerance violated at {idx}: got {got[idx]}, "
                             f"ref {ref[idx]}")
    g = got.reshape(-1, got.shape[-1])
    r = ref.reshape(-1, ref.shape[-1])
    rn = np.linalg.norm(r, axis=1)
    rel = np.linalg.norm(g - r, axis=1) / np.maximum(rn, 1e-30)
    cos = (g * r).sum(1) / np.maximum(np.linalg.norm(g, axis=1) * rn, 1e-30)
    metrics["rel_l2_max"] = float(rel.max())
    metrics["cos_min"] = float(cos.min())
    # Rotary decode rounds the turned query and keys to bf16 (its matrix-core operands and ring
    # entries), which moves every score by up to scale * 2^-8 * sum_c |q_c k_c|; rows whose
    # output nearly cancels then take the paper's own row check (App. F.4: relative L2 0.02).
    rel_limit = 2e-2 if getattr(cfg, "rope_base", 0.0) else 1e-2
    assert metrics["rel_l2_max"] <= rel_limit, f"{what}: relative L2 {metrics['rel_l2_max']:.3e}"
    assert metrics["cos_min"] >= 0.9998, f"{what}: cosine {metrics['cos_min']:.6f}"
    return metrics


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float32).numpy()


def bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)).numpy()


@dataclass
class Run:
    """A decode run of ``steps`` steps for the sequences of ``cfg`` starting at ``t0``."""
    cfg: W.Config
    t0: torch.Tensor                    # int64 [batch]
    steps: int
    device: torch.device
    desc: P.PbbDesc = None
    hist_len: int = 0                   # prefill window length (0: empty rings)
    k_ring: torch.Tensor = None
    v_ring: torch.Tensor = None
    pos: torch.Tensor = None            # int32 [batch] on device
    step_index: int = 0
    metrics: list = field(default_factory=list)

    def __post_init__(self):
        self.desc = desc_for(self.cfg, batch=self.t0.numel())
        self.k_ring, self.v_ring = P.alloc_rings(self.desc, self.device)
        self.ws = P.alloc_workspace(self.desc, self.device)
        P.ring_init(self.desc, self.k_ring, self.v_ring)
        self.pos = self.t0.to(torch.int32).to(self.device)
        if self.cfg.prefill:
            self.hist_len = self.desc.slots
            ks = W.kv_window(self.cfg, "k", self.t0, self.hist_len, device=self.device)
            vs = W.kv_window(self.cfg, "v", self.t0, self.hist_len, device=self.device)
            if self.cfg.rope_base:
                # A rotary decode leaves rotated keys in the ring: fill it with the prefix keys
                # turned by their positions (fp64 rotation, rounded to bf16).
                posm = self.t0.view(-1, 1, 1) + torch.arange(-self.hist_len, 0).view(1, 1, -1)
                rot = oracle.rope_rows(to_np(ks), posm.numpy(), self.cfg.rope_base)
                ks = torch.from_numpy(rot).to(ks.dtype).to(self.device)
            P.ring_fill(self.desc, self.pos, ks, vs, self.k_ring, self.v_ring)
            del ks, vs
        self.seq = torch.arange(self.t0.numel(), dtype=torch.int64)

    # ---- inputs -----------------------------------------------------------------------
    def positions(self, i: int) -> torch.Tensor:
        return self.t0 + i

    def step_inputs(self, i: int):
        p = self.positions(i)
        q = W.q_at(self.cfg, p, device=self.device)
        k = W.kv_at(self.cfg, "k", self.seq, p.view(-1, 1), device=self.device)[:, :, 0, :]
        v = W.kv_at(self.cfg, "v", self.seq, p.view(-1, 1), device=self.device)[:, :, 0, :]
        return q.contiguous(), k.contiguous(), v.contiguous()

    def history(self, rows: np.ndarray, upto_step: int, back: int | None = None):
        """History [n][Hkv][L][d] (workload dtype) for sequences ``rows`` covering positions
        t0 - back .. t0 + upto_step (``back`` defaults to the pre-fill length), plus its first
        position per sequence."""
        back = self.hist_len if back is None else back
        rows_t = torch.as_tensor(rows, dtype=torch.int64)
        lo = self.t0[rows_t] - back
        offs = torch.arange(0, back + upto_step + 1, dtype=torch.int64)
        posm = lo.view(-1, 1) + offs.view(1, -1)
        kh = W.kv_at(self.cfg, "k", rows_t, posm, device=self.device)
        vh = W.kv_at(self.cfg, "v", rows_t, posm, device=self.device)
        return kh, vh, lo.numpy()

    # ---- one step ---------------------------------------------------------------------
    def step(self, inputs=None):
        q, k, v = self.step_inputs(self.step_index) if inputs is None else inputs
        out = torch.empty_like(q)
        fn = P.swa_decode_step if self.cfg.mode == "swa" else P.pbb_decode_step
        fn(self.desc, self.pos, q, k, v, self.k_ring, self.v_ring, out, self.ws)
        self.pos += 1
        self.step_index += 1
        return q, out

    def oracle_out(self, rows: np.ndarray, step: int, q: torch.Tensor, hist=None):
        """fp64 oracle output [n][Hq][d] of step ``step`` for sequences ``rows``."""
        kh, vh, lo = self.history(rows, step) if hist is None else hist
        pos = (self.t0.numpy()[rows] + step).astype(np.int64)
        mode = oracle.SWA if self.cfg.mode == "swa" else oracle.PBB
        return oracle.decode(mode, pos, to_np(q[torch.as_tensor(rows, device=q.device)]), to_np(kh), to_np(vh), lo,
                             block=self.cfg.block, window=self.cfg.window,
                             rope_base=self.cfg.rope_base)

    def expected_ring(self, rows: np.ndarray, step: int, which: str, hist=None):
        """Bit pattern the ring must hold after ``step`` (0-based) has run."""
        kh, vh, lo = self.history(rows, step) if hist is None else hist
        h = kh if which == "k" else vh
        t_last = self.t0.numpy()[rows] + step
        first = np.maximum(0, self.t0.numpy()[rows] - self.hist_len)
        return oracle.expected_ring(self._bits_of(h), lo, t_last, first, self.desc.slots)

    def _bits_of(self, h: torch.Tensor) -> np.ndarray:
        """bits(h), kept for the last two history tensors (a run checked every step reuses its
        K and V histories; copying them to the host each time would dominate)."""
        cache = self.__dict__.setdefault("_bits_cache", [])
        for t, val in cache:
            if t is h:          # the cache holds h itself, so its storage cannot be reused
                return val
        val = bits(h)
        cache.append((h, val))
        del cache[:-2]
        return val

    def expected_rotated_keys(self, rows: np.ndarray, step: int, hist=None) -> np.ndarray:
        """fp64 image of the K ring of a rotary run after ``step``: every slot holds the exact
        rotation of its key (or the initial zeros)."""
        kh, vh, lo = self.history(rows, step) if hist is None else hist
        posm = lo.reshape(-1, 1, 1) + np.arange(kh.shape[2]).reshape(1, 1, -1)
        rot = oracle.rope_rows(to_np(kh), posm, self.cfg.rope_base)
        t_last = self.t0.numpy()[rows] + step
        first = np.maximum(0, self.t0.numpy()[rows] - self.hist_len)
        return oracle.expected_ring(rot, lo, t_last, first, self.desc.slots,
                                    initial=np.zeros((len(rows),) + rot.shape[1:2] +
                                                     (self.desc.slots, rot.shape[3])))

    def ring_rows(self, rows: np.ndarray, which: str) -> np.ndarray:
        r = self.k_ring if which == "k" else self.v_ring
        return bits(r[torch.as_tensor(rows, device=self.device)])
