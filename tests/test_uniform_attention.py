"""Zero queries on the GPU (through the C ABI): every score is 0, so each weight is exactly 1
(bf16 and fp32 hold it exactly) and the output is the plain mean of the support's values.  Every
launch kind must then return that mean to within one rounding of the output to bf16 (plus fp32
summation of at most |A(t)| terms): one missing or doubled key among n moves the mean by about
|v - mean| / n, far outside that.  Cases: the stepped kernel (4 and 2 waves), split launches,
whole-ring launches (PBB and SWA rings, rings not a multiple of 32 slots, rotary), each over
consecutive steps that cross block starts, bridges and ring wraps.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads as WL
from tests.harness import Run, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,mode,batch,hq,hkv,d,B,W,slots,pos_hi,steps,rope", [
    ("stepped4", "pbb", 40, 32, 8, 128, 2048, 0, 2048, 300000, 3, 0.0),      # 320 units, 4 waves
    ("stepped2", "pbb", 300, 16, 2, 128, 1024, 0, 1024, 60000, 3, 0.0),      # 600 units, 2 waves
    ("split", "pbb", 2, 32, 8, 128, 2048, 0, 2048, 300000, 4, 0.0),          # 16 units, 8 splits
    ("split-swa", "swa", 2, 8, 2, 128, 0, 4096, 4096, 300000, 3, 0.0),
    ("whole-pbb", "pbb", 2, 12, 2, 64, 128, 0, 128, 0, 300, 0.0),            # from position 0
    ("whole-pbb-rope", "pbb", 2, 12, 2, 64, 128, 0, 128, 70000, 140, 1e6),
    ("whole-pbb-100", "pbb", 3, 8, 2, 128, 100, 0, 100, 5000, 210, 0.0),
    ("stepped-swa256", "swa", 2, 12, 2, 64, 0, 128, 256, 9000, 300, 0.0),
    ("whole-swa128", "swa", 2, 12, 2, 64, 0, 100, 128, 9000, 300, 0.0),
    ("whole-swa-40", "swa", 4, 6, 1, 128, 0, 33, 40, 0, 90, 0.0),
])
def test_zero_queries_give_the_support_mean(cuda, name, mode, batch, hq, hkv, d, B, W, slots,
                                            pos_hi, steps, rope):
    cfg = WL.Config(f"uniform-{name}", mode, batch=batch, hq=hq, hkv=hkv, d=d, block=B,
                    slots=slots, window=W, dtype="bf16", seed=89, value_scale=1.0, pos_hi=pos_hi,
                    steps=steps, prefill=pos_hi > 0, rope_base=rope)
    t0 = WL.initial_positions(cfg)
    run = Run(cfg, t0, steps, cuda)
    rows = np.arange(batch) if batch <= 8 else np.arange(0, batch, max(1, batch // 8))
    hist = run.history(rows, steps - 1)
    print(f"[uniform] {cfg.name} t0[:4]={t0[:4].tolist()}", flush=True)
    for i in range(steps):
        q, k, v = run.step_inputs(i)
        q = torch.zeros_like(q)
        _, out = run.step((q, k, v))
        got = to_np(out)[rows].astype(np.float64)
        ref = run.oracle_out(rows, i, q, hist=hist)
        err = np.abs(got - ref)
        assert (err <= 2.0 ** -8 * np.abs(ref) + 1e-5).all(), (
            f"{cfg.name} step {i}: max error {err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}")
