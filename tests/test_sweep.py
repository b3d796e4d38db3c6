"""Seeded random sweeps of the GPU kernels against the fp64 oracle, through the C ABI.

Each case draws a shape the hand-written cases do not pin down: head dims 64/128, group sizes
1..16, even blocks (including non-powers of two) and windows with spare ring slots, batches on
both sides of the split-launch threshold, positions from 0 and from large pre-filled origins.
Decode: every sequence at every step, rings bit for bit.  Prefill: every position.  Backward:
every gradient by the paper's grouped-backward criteria.  The draws are fixed by the seed so a
failure names a reproducible case.
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

BLOCKS = [2, 4, 6, 10, 16, 34, 64, 96, 130, 256, 512, 1000, 2048]


def _decode_cases(n=24, seed=2024):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        mode = "pbb" if i % 3 else "swa"
        d = int(rng.choice([64, 128]))
        G = int(rng.integers(1, 17))
        hkv = int(rng.integers(1, 5))
        batch = int(rng.choice([1, 2, 3, 5, 9, 17, 40]))
        if mode == "pbb":
            block = int(rng.choice(BLOCKS))
            window, slots = 0, block
        else:
            block = 0
            window = int(rng.choice([1, 3, 33, 100, 513, 2000, 4096]))
            slots = window + int(rng.choice([0, 1, 31, 64]))
        far = bool(rng.integers(0, 2))
        cases.append((i, mode, d, G, hkv, batch, block, window, slots, far))
    return cases


@pytest.mark.parametrize("i,mode,d,G,hkv,batch,block,window,slots,far", _decode_cases())
def test_decode_sweep(cuda, i, mode, d, G, hkv, batch, block, window, slots, far):
    _decode_sweep_case(cuda, "bf16", i, mode, d, G, hkv, batch, block, window, slots, far)


@pytest.mark.parametrize("i,mode,d,G,hkv,batch,block,window,slots,far",
                         _decode_cases(12, seed=77))
def test_decode_sweep_f32(cuda, i, mode, d, G, hkv, batch, block, window, slots, far):
    _decode_sweep_case(cuda, "f32", i, mode, d, G, hkv, batch, block, window, slots, far)


@pytest.mark.parametrize("i,mode,d,G,hkv,batch,block,window,slots,far",
                         _decode_cases(8, seed=99))
def test_decode_sweep_rope(cuda, i, mode, d, G, hkv, batch, block, window, slots, far):
    _decode_sweep_case(cuda, "bf16", i, mode, d, G, hkv, batch, block, window, slots, far,
                       rope=(1e4, 1e6)[i % 2])


def _decode_sweep_case(cuda, dtype, i, mode, d, G, hkv, batch, block, window, slots, far,
                       rope=0.0):
    steps = 3
    cfg = W.Config(f"sweep{i}-{dtype}-{mode}-{d}-{G}x{hkv}-b{batch}-{block}-{window}-{slots}"
                   f"-rope{rope:g}", mode, batch=batch, hq=G * hkv, hkv=hkv, d=d, block=block,
                   slots=slots, window=window, dtype=dtype, seed=100 + i, value_scale=1.0,
                   rope_base=rope,
                   pos_hi=(1 << 20) if far else 3 * (block or window) + 5, steps=steps,
                   prefill=True)
    t0 = W.initial_positions(cfg)
    print(f"[sweep] {cfg.name} t0={t0.tolist()[:4]}", flush=True)
    run = Run(cfg, t0, steps, cuda)
    rows = np.arange(batch)
    hist = run.history(rows, steps - 1)
    for s in range(steps):
        q, out = run.step()
        compare(cfg, to_np(out), run.oracle_out(rows, s, q, hist=hist), what=f"{cfg.name} step {s}")
    for which in (("v",) if rope else ("k", "v")):
        exp = run.expected_ring(rows, steps - 1, which, hist=hist)
        assert np.array_equal(run.ring_rows(rows, which), exp), f"{cfg.name} ring {which}"
    if rope:
        # rotated keys: within one bf16 rounding of their exact rotation
        exact = run.expected_rotated_keys(rows, steps - 1, hist=hist)
        got = run.ring_rows(rows, "k").view(np.uint16).astype(np.uint32) << 16
        err = np.abs(got.view(np.float32).astype(np.float64) - exact)
        assert (err <= np.abs(exact) * 2.0 ** -8 + 1e-6).all(), f"{cfg.name} rotated keys"


def _prompt_cases(n=12, seed=7):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        mode = "pbb" if i % 3 else "swa"
        d = int(rng.choice([64, 128]))
        G = int(rng.integers(1, 17))
        hkv = int(rng.integers(1, 4))
        batch = int(rng.integers(1, 3))
        n_pos = int(rng.choice([1, 2, 31, 33, 130, 517, 1500]))
        block = int(rng.choice(BLOCKS)) if mode == "pbb" else 0
        window = 0 if mode == "pbb" else int(rng.choice([1, 7, 64, 300]))
        cases.append((i, mode, d, G, hkv, batch, n_pos, block, window))
    return cases


def _prompt(i, mode, d, G, hkv, batch, n_pos, block, window, cuda, seed):
    cfg = W.Config(f"psweep{i}", mode, batch=batch, hq=G * hkv, hkv=hkv, d=d, block=block,
                   slots=block or window, window=window, dtype="bf16", seed=seed,
                   value_scale=1.0, pos_hi=0, steps=1)
    q, k, v = W.prompt(cfg, n_pos, device=cuda)
    if mode == "pbb":
        desc = P.make_desc(batch, G * hkv, hkv, d, block=block, dtype=torch.bfloat16)
    else:
        desc = P.make_desc(batch, G * hkv, hkv, d, window=window, slots=window,
                           dtype=torch.bfloat16)
    return cfg, desc, q, k, v


@pytest.mark.parametrize("i,mode,d,G,hkv,batch,n_pos,block,window", _prompt_cases())
def test_prefill_sweep(cuda, i, mode, d, G, hkv, batch, n_pos, block, window):
    cfg, desc, q, k, v = _prompt(i, mode, d, G, hkv, batch, n_pos, block, window, cuda, 300 + i)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((batch, G * hkv, n_pos), float("nan"), dtype=torch.float32, device=cuda)
    print(f"[psweep] {i} {mode} d{d} G{G} hkv{hkv} b{batch} n{n_pos} B{block} W{window}", flush=True)
    (P.pbb_prefill if mode == "pbb" else P.swa_prefill)(desc, q, k, v, out, lse)
    torch.cuda.synchronize()
    m = oracle.PBB if mode == "pbb" else oracle.SWA
    ref, ref_lse = oracle.prefill(m, to_np(q), to_np(k), to_np(v), block=block, window=window)
    compare(cfg, to_np(out), ref, what=f"prefill sweep {i}")
    assert np.abs(lse.cpu().numpy() - ref_lse).max() <= 2e-3


@pytest.mark.parametrize("i,mode,d,G,hkv,batch,n_pos,block,window", _prompt_cases(8, seed=11))
def test_backward_sweep(cuda, i, mode, d, G, hkv, batch, n_pos, block, window):
    from tests.test_backward import _check_all
    cfg, desc, q, k, v = _prompt(i, mode, d, G, hkv, batch, n_pos, block, window, cuda, 500 + i)
    dout, _, _ = W.prompt(cfg.with_(seed=700 + i), n_pos, device=cuda)
    out = torch.empty_like(q)
    lse = torch.empty((batch, G * hkv, n_pos), dtype=torch.float32, device=cuda)
    fwd, bwd = (P.pbb_prefill, P.pbb_backward) if mode == "pbb" else (P.swa_prefill, P.swa_backward)
    fwd(desc, q, k, v, out, lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    print(f"[bsweep] {i} {mode} d{d} G{G} hkv{hkv} b{batch} n{n_pos} B{block} W{window}", flush=True)
    bwd(desc, q, k, v, out, dout, lse, dq, dk, dv)
    torch.cuda.synchronize()
    m = oracle.PBB if mode == "pbb" else oracle.SWA
    rq, rk, rv = oracle.backward(m, to_np(q), to_np(k), to_np(v), to_np(dout), block=block,
                                 window=window)
    inputs = (to_np(q), to_np(k), to_np(v), to_np(dout), to_np(out), lse.cpu().numpy())
    _check_all(f"backward sweep {i}", mode, inputs, (to_np(dq), to_np(dk), to_np(dv)),
               (rq, rk, rv), block, window)
