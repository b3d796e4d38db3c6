"""GPU parity of the rotary decode (``rope_base`` > 0): q and k_new turned by position inside
the decode launch, the ring receiving the turned key.

Outputs are compared with the fp64 oracle, which rotates q and every (unrotated) history key at
its own position exactly (bf16 tolerance as elsewhere: the kernel rounds the turned q and key
to bf16, as its matrix-core operands and the ring hold them).  The ring: values bit for bit;
keys within one bf16 rounding of their exact rotation (the rounding of a computed value is the
one thing two correct implementations may legitimately differ in).  Positions from 0 (empty
ring) and large origins (pre-filled ring of rotated keys), PBB and SWA, both head dims, bases
10^6 and 10^4, and graph replay against eager execution.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2606_02680_amd as P
import workloads as W
from tests.harness import Run, bits, compare, error_stats, merge_stats, record_stats, to_np

pytestmark = pytest.mark.gpu


def _cfg(mode, batch, hq, hkv, d, block=0, window=0, slots=0, pos_hi=0, steps=64,
         prefill=False, base=1e6, seed=41):
    return W.Config(f"rope-{mode}-{d}-{hq}-{hkv}-{block}-{window}-{pos_hi}-{base:g}", mode,
                    batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                    slots=slots or (block if mode == "pbb" else window), window=window,
                    dtype="bf16", seed=seed, value_scale=1.0, pos_hi=pos_hi, steps=steps,
                    prefill=prefill, rope_base=base)


def _check_keys(run, rows, step, hist):
    exact = run.expected_rotated_keys(rows, step, hist=hist)
    got = run.ring_rows(rows, "k").view(np.uint16).astype(np.uint32) << 16
    got = got.view(np.float32).astype(np.float64)
    err = np.abs(got - exact)
    # one bf16 rounding: half an ulp of the exact value (2^-9 relative), plus slack for the
    # float32 sine/cosine under it
    assert (err <= np.abs(exact) * 2.0 ** -8 + 1e-6).all(), float((err - np.abs(exact) * 2.0 ** -8).max())


def _run_and_check(cfg, device, check_every=1):
    t0 = W.initial_positions(cfg)
    run = Run(cfg, t0, cfg.steps, device)
    rows = np.arange(cfg.batch)
    hist = run.history(rows, cfg.steps - 1)
    print(f"[rope] {cfg.name} batch={cfg.batch} steps={cfg.steps}", flush=True)
    for i in range(cfg.steps):
        q, out = run.step()
        if i % check_every == 0 or i == cfg.steps - 1:
            ref = run.oracle_out(rows, i, q, hist=hist)
            compare(cfg, to_np(out), ref, what=f"{cfg.name} step {i}")
    exp_v = run.expected_ring(rows, cfg.steps - 1, "v", hist=hist)
    assert np.array_equal(run.ring_rows(rows, "v"), exp_v)
    _check_keys(run, rows, cfg.steps - 1, hist)


@pytest.mark.parametrize("mode,d,hq,hkv,block,window,slots", [
    ("pbb", 64, 8, 2, 32, 0, 0),
    ("pbb", 128, 16, 2, 64, 0, 0),
    ("swa", 128, 6, 3, 0, 40, 48),
])
def test_rope_from_position_zero(cuda, mode, d, hq, hkv, block, window, slots):
    """Empty ring, every step checked: every key in the ring was turned by the kernel."""
    cfg = _cfg(mode, 3, hq, hkv, d, block, window, slots, steps=3 * (block or slots) + 5)
    _run_and_check(cfg, cuda)


@pytest.mark.parametrize("base", [1e6, 1e4])
@pytest.mark.parametrize("mode,d,hq,hkv,block,window,slots", [
    ("pbb", 128, 32, 8, 2048, 0, 0),
    ("pbb", 64, 12, 2, 128, 0, 0),
    ("swa", 128, 8, 2, 0, 1000, 1024),
])
def test_rope_at_large_positions(cuda, base, mode, d, hq, hkv, block, window, slots):
    """Origins up to 2^20 with rings pre-filled with rotated keys: angles of ~10^6 turns for the
    fastest channel pair exercise the double-precision reduction."""
    cfg = _cfg(mode, 12, hq, hkv, d, block, window, slots, pos_hi=1 << 20, steps=4,
               prefill=True, base=base)
    _run_and_check(cfg, cuda)


def test_rope_graph_replay_matches_eager(cuda):
    cfg = _cfg("pbb", 4, 12, 2, 64, 128, pos_hi=100000, steps=40, prefill=True)
    t0 = W.initial_positions(cfg)
    run = Run(cfg, t0, cfg.steps, cuda)
    qs = W.q_steps(cfg, t0, 0, cfg.steps, device=cuda)
    ks = W.kv_steps(cfg, "k", t0, 0, cfg.steps, device=cuda)
    vs = W.kv_steps(cfg, "v", t0, 0, cfg.steps, device=cuda)
    snap = (run.k_ring.clone(), run.v_ring.clone())
    pos = [run.pos.clone(), torch.zeros_like(run.pos)]
    eager = torch.empty_like(qs)
    for i in range(cfg.steps):
        P.pbb_decode_step_advance(run.desc, pos[i % 2], pos[(i + 1) % 2], qs[i], ks[i], vs[i],
                                  run.k_ring, run.v_ring, eager[i])
    torch.cuda.synchronize()
    ref_k, ref_v = run.k_ring.clone(), run.v_ring.clone()
    outs = torch.zeros_like(qs)

    def restore():
        run.k_ring.copy_(snap[0])
        run.v_ring.copy_(snap[1])
        pos[0].copy_(run.t0.to(torch.int32).to(cuda))

    restore()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for i in range(cfg.steps):
            P.pbb_decode_step_advance(run.desc, pos[i % 2], pos[(i + 1) % 2], qs[i], ks[i], vs[i],
                                      run.k_ring, run.v_ring, outs[i])
    for rep in range(3):
        restore()
        outs.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs.view(torch.int16), eager.view(torch.int16)), rep
        assert torch.equal(run.k_ring.view(torch.int16), ref_k.view(torch.int16)), rep
        assert torch.equal(run.v_ring.view(torch.int16), ref_v.view(torch.int16)), rep
        _ = (qs[0].float() * 2).sum().item()


def test_rope_split_launch(cuda):
    """Rotary decode in a split launch (one sequence at c3's head shapes: each unit over eight
    workgroups): the workgroup that owns the current token's step patches the turned key, the
    first workgroup appends it."""
    cfg = _cfg("pbb", 1, 32, 8, 128, 2048, pos_hi=1 << 20, steps=5, prefill=True)
    desc = P.make_desc(1, 32, 8, 128, block=2048, dtype=torch.bfloat16, rope_base=1e6)
    assert P.workspace_bytes(desc) > 0
    _run_and_check(cfg, cuda)


def test_c3_rope_full_batch(cuda):
    """The bench's rotary launch at its full size (c3's batch of 256 and 2 GiB of pre-filled
    rings, so the non-temporal kernel variant the bench times): every sequence against the
    oracle at the first and last step of an 8-step run, taken 32 sequences at a time; the value
    ring bit for bit and the key ring within one bf16 rounding of the exact rotation."""
    cfg = W.get_config("c3").with_(rope_base=1e6, name="c3-rope-1e6")
    steps, checks, chunk = 8, (0, 7), 32
    t0 = W.initial_positions(cfg)
    print(f"[rope] {cfg.name} batch={cfg.batch} steps={steps}", flush=True)
    run = Run(cfg, t0, steps, cuda)
    kept = {}
    for i in range(steps):
        q, out = run.step()
        if i in checks:
            kept[i] = (q.clone(), out.clone())
    torch.cuda.synchronize()
    stats = None
    for c0 in range(0, cfg.batch, chunk):
        rows = np.arange(c0, min(cfg.batch, c0 + chunk))
        hist = run.history(rows, steps - 1)
        for i in checks:
            q, out = kept[i]
            ref = run.oracle_out(rows, i, q, hist=hist)
            got = to_np(out[torch.as_tensor(rows, device=cuda)])
            compare(cfg, got, ref, what=f"{cfg.name} step {i} sequences {c0}..")
            stats = merge_stats(stats, error_stats(got, ref), where=(i, c0))
        exp_v = run.expected_ring(rows, steps - 1, "v", hist=hist)
        assert np.array_equal(run.ring_rows(rows, "v"), exp_v), f"value ring, sequences {c0}.."
        _check_keys(run, rows, steps - 1, hist)
        del hist
        run.__dict__.pop("_bits_cache", None)
    stats.update(batch=cfg.batch, steps=steps, checked_steps=list(checks))
    record_stats(cfg.name, stats)
