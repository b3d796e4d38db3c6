"""GPU parity of the whole-ring decode launches (through the C ABI).

bf16 launches with at most 256 (sequence, KV head) units over rings of at most 128 slots load
the whole ring at entry, one 32-slot chunk per wave, together with the positions, and mask
each chunk to the support once the position is known (the support always lies in the ring).
These cases cover rings that are not a multiple of 32 slots (the last chunk's rows past the
ring are clamped and masked), chunks wholly outside the support (skipped), the current token's
chunk, negative positions inside a batch (those workgroups drain their ring loads before they
end), and the largest unit count of the mode.  Every
sequence at every step against the fp64 oracle; rings bit for bit.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import workloads as WL
from tests.harness import Run, compare, to_np

pytestmark = pytest.mark.gpu


def _every_step(cfg, t0, steps, device, rows=None):
    run = Run(cfg, t0, steps, device)
    assert run.ws is None, "a whole-ring launch needs no workspace"
    rows = np.arange(t0.numel()) if rows is None else rows
    hist = run.history(rows, steps - 1)
    print(f"[whole] {cfg.name} batch={cfg.batch} t0[:6]={t0[:6].tolist()}", flush=True)
    for i in range(steps):
        q, out = run.step()
        o = to_np(out)
        assert np.isfinite(o).all(), f"{cfg.name} step {i}: non-finite output"
        compare(cfg, o[rows], run.oracle_out(rows, i, q, hist=hist), what=f"{cfg.name} step {i}")
    for which in ("k", "v"):
        assert np.array_equal(run.ring_rows(rows, which),
                              run.expected_ring(rows, steps - 1, which, hist=hist)), which
    return run


@pytest.mark.parametrize("mode,batch,hq,hkv,d,B,W,slots,pos_hi,steps", [
    ("pbb", 5, 12, 2, 128, 100, 0, 100, 5000, 210),   # 100 slots: last chunk 4 rows, clamped
    ("pbb", 3, 16, 2, 64, 128, 0, 128, 9000, 300),    # G 8, bridges of 64
    ("pbb", 4, 8, 1, 128, 64, 0, 64, 0, 140),         # from position 0: chunks outside t's block
    ("swa", 3, 16, 4, 64, 0, 100, 128, 7000, 270),    # window 100 in 128 slots
    ("swa", 6, 6, 1, 128, 0, 33, 40, 300, 90),        # 40 slots: a partial second chunk
    ("swa", 2, 12, 2, 64, 0, 128, 128, 0, 150),       # from position 0, the window fills up
])
def test_whole_ring_every_step(cuda, mode, batch, hq, hkv, d, B, W, slots, pos_hi, steps):
    cfg = WL.Config(f"whole-{mode}-{batch}-{hq}-{hkv}-{d}-{B or W}-{slots}", mode, batch=batch,
                    hq=hq, hkv=hkv, d=d, block=B, slots=slots, window=W, dtype="bf16", seed=73,
                    value_scale=1.0, pos_hi=pos_hi, steps=steps, prefill=pos_hi > 0)
    _every_step(cfg, WL.initial_positions(cfg), steps, cuda)


def test_whole_ring_negative_positions(cuda):
    """Sequences at negative positions (inert: zero output, ring untouched) between live ones;
    their workgroups wait for the ring loads they issued before the position was known."""
    cfg = WL.Config("whole-neg", "pbb", batch=6, hq=12, hkv=2, d=64, block=128, slots=128,
                    window=0, dtype="bf16", seed=79, value_scale=1.0, pos_hi=3000, steps=4,
                    prefill=True)
    t0 = WL.initial_positions(cfg)
    run = Run(cfg, t0, 4, cuda)
    run.pos[1] = -20           # stays negative over the 4 steps (each adds 1)
    run.pos[4] = -9
    live = np.array([0, 2, 3, 5])
    hist = run.history(live, 3)
    rings0 = (run.k_ring[[1, 4]].clone(), run.v_ring[[1, 4]].clone())
    for i in range(4):
        q, out = run.step()
        o = to_np(out)
        assert not o[[1, 4]].any(), f"step {i}: inert rows not zero"
        compare(cfg, o[live], run.oracle_out(live, i, q, hist=hist), what=f"whole-neg step {i}")
    assert torch.equal(run.k_ring[[1, 4]].view(torch.int16), rings0[0].view(torch.int16))
    assert torch.equal(run.v_ring[[1, 4]].view(torch.int16), rings0[1].view(torch.int16))


def test_whole_ring_largest_unit_count(cuda):
    """256 units (128 sequences x 2 KV heads, the mode's limit), paper head shapes: a sample of
    sequences at every step."""
    cfg = WL.Config("whole-256u", "pbb", batch=128, hq=12, hkv=2, d=64, block=128, slots=128,
                    window=0, dtype="bf16", seed=83, value_scale=1.0, pos_hi=1 << 20, steps=40,
                    prefill=True)
    _every_step(cfg, WL.initial_positions(cfg), 40, cuda, rows=np.arange(0, 128, 9))
