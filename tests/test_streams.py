"""Calls on a stream other than torch's current one, with the binding allocating the workspace
(split decode launches, the backward).  The allocation and its zero fill are ordered on the
launch stream and the block stays tied to it, so the result is right even while torch's current
stream is still busy with earlier work (a workspace cleared there would still hold stale
counters when the launch reads them).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2606_02680_amd as P
import workloads as WL
from tests.harness import Run, compare, to_np

pytestmark = pytest.mark.gpu


def _busy(device):
    """A few milliseconds of matrix products queued on torch's current stream."""
    a = torch.randn(4096, 4096, device=device)
    for _ in range(6):
        a = (a @ a) * 1e-3
    return a


def test_split_decode_on_a_side_stream(cuda):
    cfg = WL.Config("side-stream-split", "pbb", batch=2, hq=32, hkv=8, d=128, block=2048,
                    slots=2048, window=0, dtype="bf16", seed=71, value_scale=1.0, pos_hi=300000,
                    steps=6, prefill=True)
    t0 = WL.initial_positions(cfg)
    run = Run(cfg, t0, 6, cuda)
    assert P.workspace_bytes(run.desc) > 0            # a split launch: it needs the workspace
    rows = np.arange(cfg.batch)
    hist = run.history(rows, 5)
    side = torch.cuda.Stream(device=cuda)
    cur = torch.cuda.current_stream()
    print(f"[streams] {cfg.name} t0={t0.tolist()}", flush=True)
    for i in range(6):
        q, k, v = run.step_inputs(i)
        out = torch.full_like(q, float("nan"))
        side.wait_stream(cur)                         # the inputs are ready
        busy = _busy(cuda)                            # the current stream stays busy meanwhile
        P.pbb_decode_step(run.desc, run.pos, q, k, v, run.k_ring, run.v_ring, out, None,
                          stream=side)
        cur.wait_stream(side)
        run.pos += 1
        torch.cuda.synchronize()
        del busy
        compare(cfg, to_np(out), run.oracle_out(rows, i, q, hist=hist),
                what=f"{cfg.name} step {i}")


def test_backward_on_a_side_stream(cuda):
    """The backward with the binding's workspace on a side stream returns exactly the gradients
    of the same call on torch's current stream (the backward is deterministic; its parity with
    the oracle is tested elsewhere)."""
    batch, n, hq, hkv, d, block = 1, 700, 8, 2, 128, 128
    cfg = WL.Config("side-stream-bwd", "pbb", batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                    slots=block, window=0, dtype="bf16", seed=73, value_scale=1.0, pos_hi=0,
                    steps=n)
    q, k, v = WL.prompt(cfg, n, device=cuda)
    dout, _, _ = WL.prompt(cfg.with_(seed=74), n, device=cuda)
    desc = P.make_desc(batch, hq, hkv, d, block=block, dtype=torch.bfloat16)
    out = torch.empty_like(q)
    lse = torch.empty((batch, hq, n), dtype=torch.float32, device=cuda)
    P.pbb_prefill(desc, q, k, v, out, lse)
    grads = []
    for on_side in (False, True):
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        if on_side:
            side = torch.cuda.Stream(device=cuda)
            side.wait_stream(torch.cuda.current_stream())
            busy = _busy(cuda)
            P.pbb_backward(desc, q, k, v, out, dout, lse, dq, dk, dv, stream=side)
            torch.cuda.current_stream().wait_stream(side)
        else:
            P.pbb_backward(desc, q, k, v, out, dout, lse, dq, dk, dv)
        torch.cuda.synchronize()
        grads.append((dq, dk, dv))
    for a, b in zip(*grads):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
