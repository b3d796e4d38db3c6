"""GPU parity of the training backward (``pbb_backward``, ``swa_backward``) against the fp64
oracle, through the C ABI.

The GPU forward (``pbb_prefill``) supplies ``out`` and ``lse``; the backward's dq, dk, dv are
compared with the oracle's exact gradients of the same inputs by the paper's own criteria for
its grouped backward check (Appendix F.4): relative L2 error <= 0.02 and cosine similarity >=
0.9998, here per (sequence, head) slice and for the whole tensor, plus an elementwise bound of
5e-2 times the slice's largest reference magnitude.  Shapes cover group sizes 1..16 (including
5 and 6), both head dims, blocks 2..2048, a single position, ragged tails and the window.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W
from tests.harness import to_np

pytestmark = pytest.mark.gpu


def _grad_ok(name, got, ref, heads_axis=2):
    """The paper's grouped-backward criteria (relative L2 <= 0.02, cosine >= 0.9998, App. F.4)
    for the whole tensor and for every (sequence, head) slice that carries at least a tenth of
    the largest slice's norm; elementwise, |got - ref| <= 5e-2 of the slice's largest magnitude
    for those slices, and of the tensor's for the rest: delta = dout . out uses the bf16
    forward output (reading of the kernel), which leaves an absolute error of that order even
    where the exact gradient nearly vanishes (one key taking almost all the weight)."""
    got = got.astype(np.float64)
    assert np.isfinite(got).all(), name
    rmax = float(np.abs(ref).max())
    if rmax == 0.0:
        assert np.abs(got).max() <= 1e-4, f"{name}: zero gradient"
        return
    tot = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    cos_t = float((got * ref).sum() / max(np.linalg.norm(got) * np.linalg.norm(ref), 1e-30))
    assert tot <= 2e-2, f"{name}: total relative L2 {tot:.3e}"
    assert cos_t >= 0.9998, f"{name}: total cosine {cos_t:.6f}"
    g = np.moveaxis(got, heads_axis, 1).reshape(got.shape[0] * got.shape[heads_axis], -1)
    r = np.moveaxis(ref, heads_axis, 1).reshape(ref.shape[0] * ref.shape[heads_axis], -1)
    rn = np.linalg.norm(r, axis=1)
    big = rn >= 0.1 * rn.max()
    gb, rb, rnb = g[big], r[big], rn[big]
    rel = np.linalg.norm(gb - rb, axis=1) / rnb
    cos = (gb * rb).sum(1) / np.maximum(np.linalg.norm(gb, axis=1) * rnb, 1e-30)
    assert rel.max() <= 2e-2, f"{name}: relative L2 {rel.max():.3e}"
    assert cos.min() >= 0.9998, f"{name}: cosine {cos.min():.6f}"
    scale = np.abs(rb).max(axis=1, keepdims=True)
    assert (np.abs(gb - rb) <= 5e-2 * scale).all(), f"{name}: elementwise"
    assert (np.abs(g[~big] - r[~big]) <= 5e-2 * rmax).all(), f"{name}: elementwise (small slices)"


def _run(mode, batch, n, hq, hkv, d, block=0, window=0, device="cuda"):
    cfg = W.Config(f"bwd-{mode}-{batch}-{n}-{hq}-{hkv}-{d}-{block}-{window}", mode, batch=batch,
                   hq=hq, hkv=hkv, d=d, block=block, slots=block or window, window=window,
                   dtype="bf16", seed=51, value_scale=1.0, pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=device)
    dout, _, _ = W.prompt(cfg.with_(seed=52), n, device=device)
    if mode == "pbb":
        desc = P.make_desc(batch, hq, hkv, d, block=block, dtype=torch.bfloat16)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=window, slots=window, dtype=torch.bfloat16)
        fwd, bwd = P.swa_prefill, P.swa_backward
    out = torch.empty_like(q)
    lse = torch.empty((batch, hq, n), dtype=torch.float32, device=device)
    fwd(desc, q, k, v, out, lse)
    dq = torch.full_like(q, float("nan"))
    dk = torch.full_like(k, float("nan"))
    dv = torch.full_like(v, float("nan"))
    print(f"[backward] {cfg.name}", flush=True)
    bwd(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    om = oracle.PBB if mode == "pbb" else oracle.SWA
    rq, rk, rv = oracle.backward(om, to_np(q), to_np(k), to_np(v), to_np(dout), block=block,
                                 window=window)
    return (to_np(dq), to_np(dk), to_np(dv)), (rq, rk, rv)


@pytest.mark.parametrize("mode,batch,n,hq,hkv,d,block,window", [
    ("pbb", 2, 300, 8, 2, 64, 64, 0),
    ("pbb", 1, 257, 12, 2, 64, 128, 0),      # G = 6, paper shape
    ("pbb", 1, 200, 10, 2, 64, 128, 0),      # G = 5
    ("pbb", 1, 200, 16, 1, 128, 32, 0),      # G = 16
    ("pbb", 2, 333, 32, 8, 128, 256, 0),
    ("pbb", 1, 77, 4, 4, 64, 2, 0),          # G = 1, B = 2
    ("pbb", 1, 3000, 8, 2, 128, 2048, 0),    # bridge rectangles of 1024
    ("pbb", 3, 1, 4, 2, 128, 64, 0),         # a single position
    ("swa", 2, 300, 8, 2, 128, 0, 100),
    ("swa", 1, 150, 6, 3, 64, 0, 1),
])
def test_backward_matches_oracle(cuda, mode, batch, n, hq, hkv, d, block, window):
    got, ref = _run(mode, batch, n, hq, hkv, d, block, window, cuda)
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        _grad_ok(name, g, r)


def test_backward_is_deterministic(cuda):
    a, _ = _run("pbb", 1, 260, 12, 2, 64, 128, 0, cuda)
    b, _ = _run("pbb", 1, 260, 12, 2, 64, 128, 0, cuda)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))


@pytest.mark.parametrize("name,shape", __import__("bench").BACKWARD_SHAPES,
                         ids=[nm for nm, _ in __import__("bench").BACKWARD_SHAPES])
def test_backward_bench_shapes(cuda, name, shape):
    """The bench's backward launches at full size.  The upstream gradient is nonzero only on a
    prefix [0, npre) and on the targets t >= t1 = lo + span of a tail window [lo, n) (lo a
    multiple of B for PBB, so those targets keep their full-prompt supports): the gradients there
    match the oracle on the prefix and on the tail sub-prompt, for two (sequence, KV-head group)
    slices, and every other gradient row is exactly zero."""
    from tests.test_prefill import _window_plan
    mode = "pbb" if shape.get("block") else "swa"
    block, window = shape.get("block", 0), shape.get("window", 0)
    batch, n, hq, hkv, d = shape["batch"], shape["n"], shape["hq"], shape["hkv"], shape["d"]
    G = hq // hkv
    cfg = W.Config(f"bwd-bench-{name}", mode, batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                   slots=block or window, window=window, dtype="bf16", seed=7, value_scale=1.0,
                   pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=cuda)
    dfull, _, _ = W.prompt(cfg.with_(seed=8), n, device=cuda)
    npre, lo, t1 = _window_plan(n, block or window, mode)
    keep = torch.zeros(n, dtype=dfull.dtype, device=cuda)
    keep[:npre] = 1
    keep[t1:] = 1
    dout = (dfull * keep.view(1, n, 1, 1)).contiguous()
    if mode == "pbb":
        desc = P.make_desc(batch, hq, hkv, d, block=block, dtype=torch.bfloat16)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=window, slots=window, dtype=torch.bfloat16)
        fwd, bwd = P.swa_prefill, P.swa_backward
    out = torch.empty_like(q)
    lse = torch.empty((batch, hq, n), dtype=torch.float32, device=cuda)
    fwd(desc, q, k, v, out, lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    print(f"[backward] {name} npre={npre} lo={lo} t1={t1}", flush=True)
    bwd(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    # rows no nonzero upstream gradient reaches are exactly zero
    assert not dq[:, npre:t1].any().item() and not dk[:, npre:lo].any().item()
    assert not dv[:, npre:lo].any().item()
    om = oracle.SWA if mode == "swa" else oracle.PBB
    for b, g in ((0, 0), (batch - 1, hkv - 1)):
        hs = slice(g * G, (g + 1) * G)
        for a0, a1 in ((0, npre), (lo, n)):
            sl = lambda x, h: to_np(x[b:b + 1, a0:a1, h])
            rq, rk, rv = oracle.backward(om, sl(q, hs), sl(k, slice(g, g + 1)),
                                         sl(v, slice(g, g + 1)), sl(dout, hs), block=block,
                                         window=window)
            _grad_ok(f"{name} dq seq {b} group {g} [{a0}, {a1})", sl(dq, hs), rq)
            _grad_ok(f"{name} dk seq {b} group {g} [{a0}, {a1})", sl(dk, slice(g, g + 1)), rk)
            _grad_ok(f"{name} dv seq {b} group {g} [{a0}, {a1})", sl(dv, slice(g, g + 1)), rv)


@pytest.mark.parametrize("mode,hq,hkv,block,window", [
    ("pbb", 16, 1, 65536, 0),
    ("swa", 4, 2, 0, 65536),
])
def test_backward_largest_ring(cuda, mode, hq, hkv, block, window):
    """A 70000-position prompt with the largest block or window (65536), so that dk/dv
    workgroups of the first keys walk ~65536 targets for each of up to 16 heads.  The upstream
    gradient is nonzero on the prefix [0, 1024) only: there the gradients match the oracle on
    the prefix (whose supports lie inside it), and every other row is exactly zero."""
    n, npre, d = 70000, 1024, 64
    G = hq // hkv
    cfg = W.Config(f"bwd-largest-{mode}", mode, batch=1, hq=hq, hkv=hkv, d=d, block=block,
                   slots=block or window, window=window, dtype="bf16", seed=17, value_scale=1.0,
                   pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=cuda)
    dfull, _, _ = W.prompt(cfg.with_(seed=18), n, device=cuda)
    keep = torch.zeros(n, dtype=dfull.dtype, device=cuda)
    keep[:npre] = 1
    dout = (dfull * keep.view(1, n, 1, 1)).contiguous()
    if mode == "pbb":
        desc = P.make_desc(1, hq, hkv, d, block=block, dtype=torch.bfloat16)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(1, hq, hkv, d, window=window, slots=window, dtype=torch.bfloat16)
        fwd, bwd = P.swa_prefill, P.swa_backward
    out = torch.empty_like(q)
    lse = torch.empty((1, hq, n), dtype=torch.float32, device=cuda)
    fwd(desc, q, k, v, out, lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    print(f"[backward] largest ring {mode} n={n}", flush=True)
    bwd(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    assert not dq[:, npre:].any().item()
    assert not dk[:, npre:].any().item() and not dv[:, npre:].any().item()
    om = oracle.SWA if mode == "swa" else oracle.PBB
    sl = lambda x: to_np(x[:, :npre])
    rq, rk, rv = oracle.backward(om, sl(q), sl(k), sl(v), sl(dout), block=block, window=window)
    _grad_ok(f"largest {mode} dq", sl(dq), rq)
    _grad_ok(f"largest {mode} dk", sl(dk), rk)
    _grad_ok(f"largest {mode} dv", sl(dv), rv)
