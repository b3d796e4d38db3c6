"""GPU parity with an explicit attention scale (descriptor field ``scale`` > 0 instead of the
default 1/sqrt(head_dim), Sec. 3 Eq.(attention)): decode (bf16 split and unsplit, fp32, SWA),
prefill outputs and log-partitions, and the backward, each against the fp64 oracle run with the
same scale.  Scales above and below the default change how peaked the softmax is, so a kernel
that ignored the field (or applied it twice, or only in one of the two products) fails.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W
from tests.harness import Run, compare, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode,dtype,batch,hq,hkv,d,B,scale", [
    ("pbb", "bf16", 4, 32, 8, 128, 2048, 0.25),    # 32 units: split launch
    ("pbb", "bf16", 48, 8, 2, 64, 256, 0.04),
    ("pbb", "f32", 3, 8, 2, 64, 128, 0.3),
    ("swa", "bf16", 40, 12, 4, 128, 300, 0.2),
])
def test_decode_with_explicit_scale(cuda, mode, dtype, batch, hq, hkv, d, B, scale):
    cfg = W.Config(f"scale-{mode}-{dtype}-{d}-{scale}", mode, batch=batch, hq=hq, hkv=hkv, d=d,
                   block=B if mode == "pbb" else 0, slots=B, window=B if mode == "swa" else 0,
                   dtype=dtype, seed=37, value_scale=1.0, pos_hi=20000, steps=3, prefill=True)
    run = Run(cfg, W.initial_positions(cfg), cfg.steps, cuda)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    run.desc = (P.make_desc(batch, hq, hkv, d, window=B, slots=B, dtype=tdt, scale=scale)
                if mode == "swa" else P.make_desc(batch, hq, hkv, d, block=B, dtype=tdt,
                                                  scale=scale))
    rows = np.arange(batch)
    kh, vh, lo = run.history(rows, cfg.steps - 1)
    m = oracle.SWA if mode == "swa" else oracle.PBB
    print(f"[scale] {cfg.name}", flush=True)
    for i in range(cfg.steps):
        q, out = run.step()
        pos = (run.t0.numpy() + i).astype(np.int64)
        ref = oracle.decode(m, pos, to_np(q), to_np(kh), to_np(vh), lo, block=cfg.block,
                            window=cfg.window, scale=scale)
        compare(cfg, to_np(out), ref, what=f"{cfg.name} step {i}")
        # and the default scale would not pass: the field is really used
        other = oracle.decode(m, pos, to_np(q), to_np(kh), to_np(vh), lo, block=cfg.block,
                              window=cfg.window)
        assert np.abs(other - ref).max() > 0.05


@pytest.mark.parametrize("mode,n,hq,hkv,d,B,scale", [
    ("pbb", 700, 12, 2, 64, 128, 0.3),
    ("swa", 500, 16, 4, 128, 200, 0.05),
])
def test_prefill_and_backward_with_explicit_scale(cuda, mode, n, hq, hkv, d, B, scale):
    cfg = W.Config(f"scale-prefill-{mode}", mode, batch=2, hq=hq, hkv=hkv, d=d,
                   block=B if mode == "pbb" else 0, slots=B, window=B if mode == "swa" else 0,
                   dtype="bf16", seed=39, value_scale=1.0, pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n, device=cuda)
    dout, _, _ = W.prompt(cfg.with_(seed=40), n, device=cuda)
    bf = torch.bfloat16
    if mode == "pbb":
        desc = P.make_desc(2, hq, hkv, d, block=B, dtype=bf, scale=scale)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(2, hq, hkv, d, window=B, slots=B, dtype=bf, scale=scale)
        fwd, bwd = P.swa_prefill, P.swa_backward
    out = torch.empty_like(q)
    lse = torch.empty((2, hq, n), dtype=torch.float32, device=cuda)
    print(f"[scale] prefill/backward {mode} scale={scale}", flush=True)
    fwd(desc, q, k, v, out, lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    bwd(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    m = oracle.SWA if mode == "swa" else oracle.PBB
    ref, ref_lse = oracle.prefill(m, to_np(q), to_np(k), to_np(v), block=cfg.block,
                                  window=cfg.window, scale=scale)
    compare(cfg, to_np(out), ref, what=f"prefill {mode} scale {scale}")
    assert np.abs(to_np(lse) - ref_lse).max() <= 2e-3
    rq, rk, rv = oracle.backward(m, to_np(q), to_np(k), to_np(v), to_np(dout), block=cfg.block,
                                 window=cfg.window, scale=scale)
    from tests.test_backward import _check_all
    inputs = (to_np(q), to_np(k), to_np(v), to_np(dout), to_np(out), lse.cpu().numpy())
    _check_all(f"{mode} scale {scale}", mode, inputs, (to_np(dq), to_np(dk), to_np(dv)),
               (rq, rk, rv), cfg.block, cfg.window, scale=scale)
