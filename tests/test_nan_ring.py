"""Decode over rings whose never-written slots hold NaN bits (GPU, through the C ABI).

The ring only has to hold the support's positions (Appendix F.1): a caller may skip
``pbb_ring_init`` when decoding starts at position 0, or load only the history the support
needs with ``pbb_ring_fill``.  Slots outside the support may then hold any bits, NaN included;
the outputs must still match the fp64 oracle and the untouched slots must keep their bits.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W
from tests.harness import Run, bits, compare, to_np

pytestmark = pytest.mark.gpu

NAN_BF16 = 0x7FC1          # a quiet NaN with a payload
NAN_F32 = 0x7FC00001


def _poison(t: torch.Tensor):
    if t.dtype == torch.bfloat16:
        t.view(torch.int16).fill_(NAN_BF16)
    else:
        t.view(torch.int32).fill_(NAN_F32)


def _run(cfg, t0, steps, fill_len, device):
    """Rings poisoned with NaN bits, then (if fill_len > 0) the last fill_len positions before
    t0 loaded; every step against the oracle, rings against the image whose unwritten slots
    keep the NaN bits."""
    run = Run(cfg.with_(prefill=False), t0, steps, device)
    _poison(run.k_ring)
    _poison(run.v_ring)
    if fill_len > 0:
        ks = W.kv_window(cfg, "k", t0, fill_len, device=device)
        vs = W.kv_window(cfg, "v", t0, fill_len, device=device)
        P.ring_fill(run.desc, run.pos, ks, vs, run.k_ring, run.v_ring)
    rows = np.arange(t0.numel())
    hist = run.history(rows, steps - 1, back=fill_len)
    print(f"[nan-ring] {cfg.name} t0={t0.tolist()} fill={fill_len}", flush=True)
    for i in range(steps):
        q, out = run.step()
        o = to_np(out)
        assert np.isfinite(o).all(), f"{cfg.name} step {i}: non-finite output"
        compare(cfg, o, run.oracle_out(rows, i, q, hist=hist), what=f"{cfg.name} step {i}")
    nan = NAN_BF16 if cfg.dtype == "bf16" else NAN_F32
    kh, vh, lo = hist
    first = np.maximum(0, t0.numpy() - fill_len)
    t_last = t0.numpy() + steps - 1
    for which, h in (("k", kh), ("v", vh)):
        hb = bits(h)
        init = np.full((len(rows), cfg.hkv, run.desc.slots, cfg.d), nan, dtype=hb.dtype)
        exp = oracle.expected_ring(hb, lo, t_last, first, run.desc.slots, initial=init)
        assert np.array_equal(run.ring_rows(rows, which), exp), f"{cfg.name} ring {which}"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("d,hq,hkv,B", [(128, 8, 2, 64), (64, 12, 2, 128), (128, 4, 4, 40)])
def test_from_position_zero_without_ring_init(cuda, dtype, d, hq, hkv, B):
    """Decoding from position 0 on rings that were never initialised: for t < B the support
    holds only appended positions, and the padded rows of each step read slots that still
    hold NaN bits."""
    cfg = W.Config(f"nan-zero-{dtype}-{d}-{hq}-{hkv}-{B}", "pbb", batch=2, hq=hq, hkv=hkv, d=d,
                   block=B, slots=B, window=0, dtype=dtype, seed=31, value_scale=1.0, pos_hi=0,
                   steps=2 * B + 5)
    _run(cfg, torch.zeros(2, dtype=torch.int64), cfg.steps, 0, cuda)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_bridge_half_only_filled(cuda, dtype):
    """Block starts (r = 0) with only the bridge half [p - h, p) loaded: slots [0, h) hold NaN
    bits until the block's own positions are appended."""
    B = 256
    cfg = W.Config(f"nan-bridge-{dtype}", "pbb", batch=3, hq=16, hkv=2, d=128, block=B, slots=B,
                   window=0, dtype=dtype, seed=37, value_scale=1.0, pos_hi=0, steps=B // 2 + 40)
    t0 = torch.tensor([5 * B, 9 * B, 1000 * B], dtype=torch.int64)
    _run(cfg, t0, cfg.steps, B // 2, cuda)


def test_split_launch_bridge_half_only(cuda):
    """The same with one sequence at c3's head shapes, a split launch (8 workgroups per unit
    merging through the workspace)."""
    B = 2048
    cfg = W.Config("nan-split", "pbb", batch=1, hq=32, hkv=8, d=128, block=B, slots=B, window=0,
                   dtype="bf16", seed=41, value_scale=1.0, pos_hi=0, steps=6)
    run_ws = P.workspace_bytes(P.make_desc(1, 32, 8, 128, block=B))
    assert run_ws > 0, "expected a split launch"
    _run(cfg, torch.tensor([7 * B], dtype=torch.int64), cfg.steps, B // 2, cuda)


def test_swa_window_only_filled(cuda):
    """SWA ring larger than the window with only the window's history loaded."""
    cfg = W.Config("nan-swa", "swa", batch=2, hq=8, hkv=2, d=64, block=0, slots=160, window=100,
                   dtype="bf16", seed=43, value_scale=1.0, pos_hi=0, steps=70)
    _run(cfg, torch.tensor([1000, 333], dtype=torch.int64), cfg.steps, 99, cuda)


def test_rotary_from_zero_without_ring_init(cuda):
    cfg = W.Config("nan-rope", "pbb", batch=2, hq=12, hkv=2, d=64, block=128, slots=128,
                   window=0, dtype="bf16", seed=47, value_scale=1.0, pos_hi=0, steps=140,
                   rope_base=1e6)
    t0 = torch.zeros(2, dtype=torch.int64)
    run = Run(cfg, t0, cfg.steps, cuda)
    _poison(run.k_ring)
    _poison(run.v_ring)
    rows = np.arange(2)
    hist = run.history(rows, cfg.steps - 1, back=0)
    for i in range(cfg.steps):
        q, out = run.step()
        o = to_np(out)
        assert np.isfinite(o).all(), f"rotary step {i}: non-finite output"
        compare(cfg, o, run.oracle_out(rows, i, q, hist=hist), what=f"rotary step {i}")
