"""The allocation-free decode entry point against pbb_decode_step (GPU, through the C ABI).

pbb_decode_step_noalloc runs the same kernels as pbb_decode_step but takes the workspace of
split launches from the library's per-device scratch buffer.  Two calls in a row on the same
buffer, the second with a smaller batch (more splits per unit, fewer units), each compared bit
for bit with pbb_decode_step on identical inputs and rings, and against the fp64 oracle.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2606_02680_amd as P
import workloads as W
from tests.harness import Run, compare, to_np

pytestmark = pytest.mark.gpu


def _cfg(batch):
    # c3's head shapes (Hq 32, Hkv 8, d 128, B 2048) at a small batch: a split launch
    return W.Config(f"noalloc-b{batch}", "pbb", batch=batch, hq=32, hkv=8, d=128, block=2048,
                    slots=2048, window=0, dtype="bf16", seed=53 + batch, value_scale=1.0,
                    pos_hi=400000, steps=3, prefill=True)


def _compare_step(cfg, device, steps):
    t0 = W.initial_positions(cfg)
    t0[0] = 5 * cfg.block                      # a block start (bridge only) in the batch
    ref_run = Run(cfg, t0, steps, device)      # pbb_decode_step with a caller workspace
    new_run = Run(cfg, t0, steps, device)      # pbb_decode_step_noalloc
    assert ref_run.ws is not None, "expected a split launch"
    rows = np.arange(cfg.batch)
    hist = ref_run.history(rows, steps - 1)
    print(f"[noalloc] {cfg.name} t0={t0.tolist()}", flush=True)
    for i in range(steps):
        inputs = ref_run.step_inputs(i)
        q, out_ref = ref_run.step(inputs)
        out_new = torch.empty_like(out_ref)
        P.pbb_decode_step_noalloc(new_run.desc, new_run.pos, *inputs, new_run.k_ring,
                                  new_run.v_ring, out_new)
        new_run.pos += 1
        torch.cuda.synchronize()
        assert torch.equal(out_new.view(torch.int16), out_ref.view(torch.int16)), f"step {i}"
        compare(cfg, to_np(out_new), ref_run.oracle_out(rows, i, q, hist=hist),
                what=f"{cfg.name} step {i}")
    assert torch.equal(new_run.k_ring.view(torch.int16), ref_run.k_ring.view(torch.int16))
    assert torch.equal(new_run.v_ring.view(torch.int16), ref_run.v_ring.view(torch.int16))


def test_noalloc_two_calls_second_smaller(cuda):
    """Batch 8 (64 units, 4 workgroups each), then batch 1 (8 units, 8 workgroups each) on the
    same scratch buffer."""
    _compare_step(_cfg(8), cuda, steps=3)
    _compare_step(_cfg(1), cuda, steps=3)


def test_noalloc_unsplit_launch(cuda):
    """A launch that needs no workspace (128 units) goes through the same entry point."""
    cfg = _cfg(16)
    t0 = W.initial_positions(cfg)
    a = Run(cfg, t0, 1, cuda)
    b = Run(cfg, t0, 1, cuda)
    assert a.ws is None
    inputs = a.step_inputs(0)
    _, out_a = a.step(inputs)
    out_b = torch.empty_like(out_a)
    P.pbb_decode_step_noalloc(b.desc, b.pos, *inputs, b.k_ring, b.v_ring, out_b)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(a.k_ring.view(torch.int16), b.k_ring.view(torch.int16))
