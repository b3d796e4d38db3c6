"""GPU parity of the training backward (``pbb_backward``, ``swa_backward``) against the fp64
oracle, through the C ABI.

The GPU forward (``pbb_prefill``) supplies ``out`` and ``lse``; the backward's dq, dk, dv are
compared with the oracle's exact gradients of the same inputs by the paper's own criteria for
its grouped backward check (Appendix F.4): relative L2 error <= 0.02 and cosine similarity >=
0.9998, here per (sequence, head) slice and for the whole tensor, plus an elementwise bound
derived from the kernels' rounding points and evaluated on the data (:func:`grad_bounds`).  Shapes cover group sizes 1..16 (including
5 and 6), both head dims, blocks 2..2048, a single position, ragged tails and the window.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W
from tests.grad_bounds import U_BF16, grad_bounds
from tests.harness import record_stats, to_np

pytestmark = pytest.mark.gpu


def _grad_ok(name, got, ref, bound, heads_axis=2):
    """Elementwise |got - ref| <= 2 (bound + U |ref|) with ``bound`` from :func:`grad_bounds`
    (the factor 2 covers second-order terms and the fp32 accumulations); and the paper's
    grouped-backward criteria (relative L2 <= 0.02, cosine >= 0.9998, App. F.4) for the whole
    tensor and for every (sequence, head) slice carrying at least a tenth of the largest slice's
    norm.  Returns the largest error / allowance ratio."""
    got = got.astype(np.float64)
    assert np.isfinite(got).all(), name
    allow = 2.0 * (bound + U_BF16 * np.abs(ref))
    err = np.abs(got - ref)
    worst = float((err / np.maximum(allow, 1e-300)).max()) if err.size else 0.0
    if not (err <= allow).all():
        idx = np.unravel_index(np.argmax(err - allow), err.shape)
        raise AssertionError(f"{name}: |got - ref| {err[idx]:.3e} > derived bound "
                             f"{allow[idx]:.3e} at {idx} (ref {ref[idx]:.4e})")
    rmax = float(np.abs(ref).max())
    if rmax == 0.0:
        return worst
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
    record_stats(name, {"max_abs": float(err.max()), "max_ref": rmax,
                        "worst_error_over_derived_bound": worst, "rel_l2_total": float(tot),
                        "cos_total": cos_t, "rel_l2_max_slice": float(rel.max()),
                        "cos_min_slice": float(cos.min())})
    return worst


def _check_all(name, mode, inputs, got, ref, block, window, scale=None):
    """grad_bounds + _grad_ok for (dq, dk, dv); prints the worst error / allowance ratio."""
    q, k, v, dout, out, lse = inputs
    bounds = grad_bounds(mode, q, k, v, dout, out, lse, block=block, window=window, scale=scale)
    worst = max(_grad_ok(f"{name} {nm}", g, r, bd)
                for nm, g, r, bd in zip(("dq", "dk", "dv"), got, ref, bounds))
    print(f"[backward] {name}: largest error / derived allowance {worst:.3f}", flush=True)
    return worst


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
    inputs = (to_np(q), to_np(k), to_np(v), to_np(dout), to_np(out), lse.cpu().numpy())
    return (to_np(dq), to_np(dk), to_np(dv)), (rq, rk, rv), inputs


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
    got, ref, inputs = _run(mode, batch, n, hq, hkv, d, block, window, cuda)
    _check_all(f"{mode} n={n} hq={hq} hkv={hkv} d={d}", mode, inputs, got, ref, block, window)


def test_backward_is_deterministic(cuda):
    a, _, _ = _run("pbb", 1, 260, 12, 2, 64, 128, 0, cuda)
    b, _, _ = _run("pbb", 1, 260, 12, 2, 64, 128, 0, cuda)
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
        gs = slice(g, g + 1)
        for a0, a1 in ((0, npre), (lo, n)):
            sl = lambda x, h: to_np(x[b:b + 1, a0:a1, h])
            rq, rk, rv = oracle.backward(om, sl(q, hs), sl(k, gs), sl(v, gs), sl(dout, hs),
                                         block=block, window=window)
            inputs = (sl(q, hs), sl(k, gs), sl(v, gs), sl(dout, hs), sl(out, hs),
                      lse[b:b + 1, hs, a0:a1].cpu().numpy())
            _check_all(f"{name} seq {b} group {g} [{a0}, {a1})", mode, inputs,
                       (sl(dq, hs), sl(dk, gs), sl(dv, gs)), (rq, rk, rv), block, window)


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
    inputs = (sl(q), sl(k), sl(v), sl(dout), sl(out), lse[:, :, :npre].cpu().numpy())
    _check_all(f"largest {mode}", mode, inputs, (sl(dq), sl(dk), sl(dv)), (rq, rk, rv), block,
               window)


@pytest.mark.parametrize("hq,hkv,d,B,nblocks,blk", [
    (12, 2, 64, 128, 6, 3),      # the paper's model shape
    (32, 8, 128, 2048, 3, 2),    # c3's head shapes
])
def test_bridge_gradient_of_repaired_targets(cuda, hq, hkv, d, B, nblocks, blk):
    """Appendix F.4's bridge check: the upstream gradient is nonzero only on the repaired
    targets of one block (positions p .. p+h-1 of block `blk`, whose supports add the bridge
    [p-h, p)), so the previous block's tail keys and values receive gradient only through the
    bridge rectangle.  Their dk and dv, the block's own, and dq of the repaired targets match
    the oracle (on the window [p-B, p+h), which holds every support involved); every other
    gradient row is exactly zero, and the bridge keys' gradients are not."""
    n, p, h = nblocks * B, blk * B, B // 2
    cfg = W.Config(f"bwd-bridge-{hq}-{B}", "pbb", batch=1, hq=hq, hkv=hkv, d=d, block=B,
                   slots=B, window=0, dtype="bf16", seed=61, value_scale=1.0, pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=cuda)
    dfull, _, _ = W.prompt(cfg.with_(seed=62), n, device=cuda)
    keep = torch.zeros(n, dtype=dfull.dtype, device=cuda)
    keep[p:p + h] = 1
    dout = (dfull * keep.view(1, n, 1, 1)).contiguous()
    desc = P.make_desc(1, hq, hkv, d, block=B, dtype=torch.bfloat16)
    out = torch.empty_like(q)
    lse = torch.empty((1, hq, n), dtype=torch.float32, device=cuda)
    P.pbb_prefill(desc, q, k, v, out, lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    print(f"[backward] bridge check hq={hq} B={B} block {blk}", flush=True)
    P.pbb_backward(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    assert not dq[:, :p].any().item() and not dq[:, p + h:].any().item()
    for g in (dk, dv):
        assert not g[:, :p - h].any().item() and not g[:, p + h:].any().item()
    bridge = dk[:, p - h:p].float().norm().item()
    own = dk[:, p:p + h].float().norm().item()
    assert bridge > 0.05 * own, (bridge, own)
    a0, a1 = p - B, p + h
    sl = lambda x: to_np(x[:, a0:a1])
    rq, rk, rv = oracle.backward(oracle.PBB, sl(q), sl(k), sl(v), sl(dout), block=B)
    inputs = (sl(q), sl(k), sl(v), sl(dout), sl(out), lse[:, :, a0:a1].cpu().numpy())
    _check_all(f"bridge hq={hq} B={B}", "pbb", inputs, (sl(dq), sl(dk), sl(dv)), (rq, rk, rv),
               B, 0)
    assert np.abs(rk[:, B - h:B]).max() > 0     # the oracle agrees the bridge keys get gradient
