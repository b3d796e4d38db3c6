"""GPU parity: the HIP library (through its C ABI) against the fp64 CPU oracle.

Outputs: fp32 within max-abs 1e-5; bf16 within |d| <= 2e-2 + 2^-8 |ref| elementwise plus
relative L2 <= 1e-2 and cosine >= 0.9998 per (sequence, head).  Rings: bit-exact against the
oracle's ring image (slot = position mod slots, Appendix F.1).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.harness import Run, bits, compare, error_stats, merge_stats, record_stats, to_np

pytestmark = pytest.mark.gpu


def _lockstep(cfg, device, check_out, check_ring, batch=None):
    """Run cfg from position 0 (or cfg's t0) for cfg.steps steps, checking selected steps."""
    b = cfg.batch if batch is None else batch
    t0 = W.initial_positions(cfg.with_(batch=b))
    run = Run(cfg, t0, cfg.steps, device)
    rows = np.arange(b)
    hist = run.history(rows, cfg.steps - 1)
    print(f"[lockstep] {cfg.name} batch={b} steps={cfg.steps}", flush=True)
    worst = 0.0
    for i in range(cfg.steps):
        q, out = run.step()
        if check_out(i):
            ref = run.oracle_out(rows, i, q, hist=hist)
            m = compare(cfg, to_np(out), ref, what=f"{cfg.name} step {i}")
            worst = max(worst, m["max_abs"])
        if check_ring(i):
            for which in ("k", "v"):
                exp = run.expected_ring(rows, i, which, hist=hist)
                got = run.ring_rows(rows, which)
                assert np.array_equal(got, exp), f"{cfg.name} ring {which} mismatch after step {i}"
    return worst


def test_c1_tiny_fp32_every_step(cuda):
    cfg = W.get_config("c1")
    worst = _lockstep(cfg, cuda, check_out=lambda i: True, check_ring=lambda i: True)
    print(f"c1 worst max-abs {worst:.3e}")


def test_c2_lockstep_bf16(cuda):
    """2048 steps from 0 with B = 512 (every phase r four times, the bridge in blocks 1-3):
    outputs and both rings checked after every step."""
    cfg = W.get_config("c2")
    worst = _lockstep(cfg, cuda, check_out=lambda i: True, check_ring=lambda i: True)
    print(f"c2 worst max-abs {worst:.3e}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d,hq,hkv,block", [(64, 1, 1, 2), (128, 2, 1, 4), (64, 16, 1, 16),
                                            (128, 8, 2, 32), (64, 6, 3, 8), (128, 16, 2, 64)])
def test_small_shapes_every_step(cuda, dtype, d, hq, hkv, block):
    """Group sizes 1..16, both head dims, tiny blocks (one to several 32-key tiles, ragged
    tails), every step over five blocks, ring checked every step."""
    cfg = W.Config(f"small-{dtype}-{d}-{hq}-{hkv}-{block}", "pbb", batch=3, hq=hq, hkv=hkv,
                   d=d, block=block, slots=block, window=0, dtype=dtype, seed=5,
                   value_scale=1.0, pos_hi=0, steps=5 * block + 3)
    _lockstep(cfg, cuda, check_out=lambda i: True, check_ring=lambda i: True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("window,slots", [(48, 64), (64, 64), (37, 40), (1, 1), (100, 160)])
def test_swa_small_every_step(cuda, dtype, window, slots):
    cfg = W.Config(f"swa-{dtype}-{window}-{slots}", "swa", batch=2, hq=4, hkv=2, d=64,
                   block=0, slots=slots, window=window, dtype=dtype, seed=6, value_scale=1.0,
                   pos_hi=0, steps=3 * slots + 5)
    _lockstep(cfg, cuda, check_out=lambda i: True, check_ring=lambda i: True)


def _edge_positions(cfg, n):
    """Initial positions covering the degenerate phases of a block of size B (or a window)."""
    B = cfg.block if cfg.mode == "pbb" else cfg.slots
    h = B // 2
    k = 37  # an arbitrary later block
    edges = [0, 1, h - 1, h, B - 1, B, B + 1, B + h - 1, B + h, k * B, k * B + 1,
             k * B + h - 1, k * B + h, k * B + B - 1, cfg.pos_hi - 1]
    return [e for e in edges if 0 <= e][:n]


def _sampled(cfg, device, steps, n_rows=24, seed=0):
    """Full-size batch with forced edge positions; checks sampled sequences at every step."""
    t0 = W.initial_positions(cfg)
    edges = _edge_positions(cfg, n_rows // 2)
    t0[:len(edges)] = torch.tensor(edges, dtype=torch.int64)
    print(f"[sampled] {cfg.name} batch={cfg.batch} steps={steps}", flush=True)
    run = Run(cfg, t0, steps, device)
    rng = np.random.default_rng(seed)
    rest = rng.choice(np.arange(len(edges), cfg.batch), size=n_rows - len(edges), replace=False)
    rows = np.concatenate([np.arange(len(edges)), np.sort(rest)])
    hist = run.history(rows, steps - 1)
    worst = {}
    for i in range(steps):
        q, out = run.step()
        ref = run.oracle_out(rows, i, q, hist=hist)
        got = to_np(out[torch.as_tensor(rows, device=device)])
        m = compare(cfg, got, ref, what=f"{cfg.name} step {i}")
        worst = {k: max(worst.get(k, -1e30), v) if k != "cos_min" else min(worst.get(k, 1e30), v)
                 for k, v in m.items()}
    for which in ("k", "v"):
        exp = run.expected_ring(rows, steps - 1, which, hist=hist)
        assert np.array_equal(run.ring_rows(rows, which), exp), f"{cfg.name} ring {which}"
    return run, rows, hist, worst


def _full_batch(cfg, device, steps=128, checks=(0, 64, 127), chunk=32, strict=None):
    """Every sequence of the full-size batch (forced edge positions in the first ones) against
    the oracle at the checked steps of a run of ``steps`` steps, and every ring bit for bit
    after the last step.  The oracle side is taken 32 sequences at a time, so host memory stays
    bounded.  ``strict``: also assert the plain max-abs bound max |got - ref| <= strict."""
    t0 = W.initial_positions(cfg)
    edges = _edge_positions(cfg, 12)
    t0[:len(edges)] = torch.tensor(edges, dtype=torch.int64)
    print(f"[full-batch] {cfg.name} batch={cfg.batch} steps={steps} checks={checks}", flush=True)
    run = Run(cfg, t0, steps, device)
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
            got = to_np(out[torch.as_tensor(rows, device=device)])
            compare(cfg, got, ref, what=f"{cfg.name} step {i} sequences {c0}..")
            stats = merge_stats(stats, error_stats(got, ref), where=(i, c0))
        for which in ("k", "v"):
            exp = run.expected_ring(rows, steps - 1, which, hist=hist)
            assert np.array_equal(run.ring_rows(rows, which), exp), \
                f"{cfg.name} ring {which}, sequences {c0}..{rows[-1]}"
        del hist
        run.__dict__.pop("_bits_cache", None)
    stats.update(batch=cfg.batch, steps=steps, checked_steps=list(checks),
                 argmax_fields="step, first sequence of chunk, row, head, channel")
    record_stats(cfg.name, stats)
    if strict is not None:
        assert stats["max_abs"] <= strict, f"{cfg.name}: strict max abs {stats['max_abs']:.3e}"
    return stats


def test_c3_full_batch(cuda):
    """c3 (batch 256, Hq 32, Hkv 8, d 128, B 2048): all 256 sequences at steps 0, 64, 127;
    outputs here are small (|o| < 2), so the plain 2e-2 max-abs bound is asserted too."""
    _full_batch(W.get_config("c3"), cuda, strict=2e-2)


def test_c4_ragged_spiked_full_batch(cuda):
    """c4 (batch 1024, GQA 8, B 1024, K/V x4 on 1% of positions): all sequences; the x4
    spikes push |o| past 8, where one bf16 rounding exceeds 2e-2 (reading 7's bound applies)."""
    _full_batch(W.get_config("c4"), cuda)


def test_c4_shapes_fp32_full_batch(cuda):
    """c4's shapes and tensors with fp32 rings and I/O (the matrix-core fp32 kernel at its full
    launch size, G = 8): every sequence within 1e-5 at steps 0, 64, 127."""
    _full_batch(W.get_config("c4").with_(dtype="f32", name="c4-shapes-fp32"), cuda)


def test_c5_swa_full_batch(cuda):
    """c5 (SWA W 4096 in 4096 slots on c3's tensors): all sequences, plain 2e-2 asserted."""
    _full_batch(W.get_config("c5"), cuda, strict=2e-2)


@pytest.mark.parametrize("slots", [4096, 2048])
def test_c5_paper_window_full_size_sampled(cuda, slots):
    """The bench's paper-matched SWA rows at full size: c3's tensors and positions with the
    window W = B = 2048 in 4096 slots (the paper's 2x buffer) and in 2048 slots (a B-slot ring);
    the edge sequences and a sample of others at every one of 3 steps, rings bit for bit."""
    cfg = W.get_config("c5").with_(window=2048, slots=slots, name=f"c5-w2048-s{slots}")
    _, _, _, worst = _sampled(cfg, cuda, steps=3)
    print(f"{cfg.name} {worst}")


def test_c3_edge_rows_every_step(cuda):
    """c3 with forced edge positions: the edge sequences and a sample of others at every one
    of 3 consecutive steps (the full-batch test checks every sequence at 3 steps of a run)."""
    cfg = W.get_config("c3")
    _, _, _, worst = _sampled(cfg, cuda, steps=3)
    print(f"c3 {worst}")


@pytest.mark.parametrize("mode,d,hq,hkv,block,window,slots", [
    ("pbb", 64, 8, 2, 2048, 0, 2048),
    ("pbb", 128, 16, 1, 4096, 0, 4096),
    ("swa", 64, 4, 4, 0, 2048, 2048),
    ("swa", 128, 6, 3, 0, 2500, 3000),
])
def test_long_support_shapes_sampled(cuda, mode, d, hq, hkv, block, window, slots):
    """Supports of >= 2048 keys (the 4-wave workgroup variant) for both head dims, PBB and SWA,
    pre-filled rings at edge and random positions."""
    cfg = W.Config(f"long-{mode}-{d}-{hq}-{hkv}-{block}-{window}", mode, batch=40, hq=hq,
                   hkv=hkv, d=d, block=block, slots=slots, window=window, dtype="bf16", seed=9,
                   value_scale=1.0, pos_hi=300000, steps=2, prefill=True)
    _, _, _, worst = _sampled(cfg, cuda, steps=2, n_rows=cfg.batch)
    print(f"{cfg.name} {worst}")


def _support_variant(kind, t, B):
    h = B // 2
    p, r = B * (t // B), t % B
    if kind == "no_bridge":
        return list(range(p, t + 1))
    if kind == "bridge_always":
        return list(range(max(0, p - h), t + 1))
    if kind == "start_off_by_one":
        lo = max(0, h * (t // h - 1))
        return list(range(max(0, lo + (1 if lo > 0 else 0)), t + 1))
    if kind == "swa_w_eq_b":
        return list(range(max(0, t - B + 1), t + 1))
    raise ValueError(kind)


def test_wrong_support_controls_are_detected(cuda):
    """The tolerance can see support mistakes: at c2's scale (N(0,1)/8, where an all-zero
    output would pass a plain 2e-2 max-abs bound), outputs computed on plausible wrong
    supports or a strided GQA mapping fail the same comparison the GPU output passes."""
    cfg = W.get_config("c2").with_(batch=4, steps=1)
    B, h = cfg.block, cfg.block // 2
    run_t0 = torch.tensor([B + 3, 3 * B + h + 5, 2 * B + 7, B + 1], dtype=torch.int64)
    run = Run(cfg.with_(prefill=True), run_t0, 1, cuda)
    rows = np.arange(4)
    hist = run.history(rows, 0, back=2 * B)
    q, out = run.step()
    ref = run.oracle_out(rows, 0, q, hist=hist)
    compare(cfg, to_np(out), ref, what="gpu vs oracle")
    kh, vh, lo = (to_np(hist[0]), to_np(hist[1]), hist[2])
    qn = to_np(q)
    G = cfg.group
    for kind in ("no_bridge", "bridge_always", "start_off_by_one", "swa_w_eq_b", "gqa_strided"):
        wrong = np.zeros_like(ref)
        for b in range(4):
            t = int(run_t0[b])
            if kind == "gqa_strided":
                sup = oracle.pbb_support(t, B)
            else:
                sup = _support_variant(kind, t, B)
            idx = np.array(sup) - lo[b]
            for i in range(cfg.hq):
                g = (i % cfg.hkv) if kind == "gqa_strided" else i // G
                wrong[b, i], _ = oracle.attend(qn[b, i], kh[b, g, idx], vh[b, g, idx])
        with pytest.raises(AssertionError):
            compare(cfg, to_np(out), wrong, what=kind)
    with pytest.raises(AssertionError):
        compare(cfg, np.zeros_like(ref), ref, what="all zeros")


def test_negative_position_is_inert(cuda):
    cfg = W.get_config("c2").with_(batch=2, steps=1)
    run = Run(cfg, torch.tensor([5, 7]), 1, cuda)
    run.pos[1] = -1
    before = bits(run.k_ring[1]).copy()
    q, out = run.step()
    assert not to_np(out[1]).any()
    assert np.array_equal(bits(run.k_ring[1]), before)


def test_repeat_is_bitwise_deterministic(cuda):
    cfg = W.get_config("c4").with_(batch=64)
    t0 = W.initial_positions(cfg)
    a = Run(cfg, t0, 1, cuda)
    b = Run(cfg, t0, 1, cuda)
    inputs = a.step_inputs(0)
    _, oa = a.step(inputs)
    _, ob = b.step(inputs)
    assert torch.equal(oa.view(torch.int16), ob.view(torch.int16))
    assert torch.equal(a.k_ring.view(torch.int16), b.k_ring.view(torch.int16))


def test_snapshot_restore_continues_bitwise(cuda):
    """Ring + positions are the whole decode state: restoring a snapshot and continuing
    reproduces an uninterrupted run bit for bit."""
    cfg = W.get_config("c2").with_(batch=8)
    t0 = W.initial_positions(cfg)
    run = Run(cfg, t0, 0, cuda)
    for _ in range(300):
        run.step()
    snap = (run.k_ring.clone(), run.v_ring.clone(), run.pos.clone(), run.step_index)
    outs_a = [run.step()[1].clone() for _ in range(300)]
    run.k_ring.copy_(snap[0]); run.v_ring.copy_(snap[1]); run.pos.copy_(snap[2])
    run.step_index = snap[3]
    outs_b = [run.step()[1].clone() for _ in range(300)]
    for x, y in zip(outs_a, outs_b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


@pytest.mark.parametrize("mode,batch,d,hq,hkv,block,window,slots,pos_hi,steps", [
    ("pbb", 1, 128, 32, 8, 2048, 0, 2048, 300000, 6),   # c3's heads, one sequence: 8 splits
    ("pbb", 1, 128, 32, 8, 2048, 0, 2048, 0, 40),       # from position 0: mostly empty splits
    ("pbb", 3, 64, 12, 2, 1024, 0, 1024, 5000, 8),      # 4 splits
    ("swa", 2, 128, 8, 2, 0, 4096, 4096, 300000, 4),    # 8 splits
    ("pbb", 8, 128, 32, 8, 2048, 0, 2048, 300000, 3),   # 64 units: 4 splits
    ("swa", 10, 64, 16, 4, 0, 1000, 1024, 90000, 3),    # 40 units: 4 splits
    ("pbb", 5, 128, 32, 8, 2048, 0, 2048, 300000, 3),   # 40 units: floor(256 / 40) = 6 splits
    ("swa", 6, 128, 32, 8, 0, 4096, 4096, 300000, 3),   # 48 units, full windows: 5 splits
])
def test_split_workgroups_small_batch(cuda, mode, batch, d, hq, hkv, block, window, slots,
                                      pos_hi, steps):
    """Launches with fewer (sequence, KV head) units than CUs spread each unit's steps over
    several workgroups, which merge their softmax states (Eq.(lse)) in the last to finish:
    every sequence at every step against the oracle, rings bit for bit."""
    cfg = W.Config(f"split-{mode}-{batch}-{d}-{hq}-{hkv}-{block}-{window}-{pos_hi}", mode,
                   batch=batch, hq=hq, hkv=hkv, d=d, block=block, slots=slots, window=window,
                   dtype="bf16", seed=13, value_scale=1.0, pos_hi=pos_hi, steps=steps,
                   prefill=pos_hi > 0)
    t0 = W.initial_positions(cfg)
    run = Run(cfg, t0, steps, cuda)
    assert run.ws is not None and run.ws.numel() > 0, "expected a split launch"
    rows = np.arange(batch)
    hist = run.history(rows, steps - 1)
    print(f"[split] {cfg.name} t0={t0.tolist()}", flush=True)
    for i in range(steps):
        q, out = run.step()
        compare(cfg, to_np(out), run.oracle_out(rows, i, q, hist=hist), what=f"{cfg.name} step {i}")
    for which in ("k", "v"):
        exp = run.expected_ring(rows, steps - 1, which, hist=hist)
        assert np.array_equal(run.ring_rows(rows, which), exp), f"{cfg.name} ring {which}"
    # the launches left every unit counter at zero
    units = batch * hkv
    assert not run.ws[: 4 * units].any().item()


def test_one_workspace_for_split_launches_of_two_descriptors(cuda):
    """One caller workspace, zero-filled once, serves split launches of two descriptors in turn
    (64 units in 4 splits, 16 units in 8): both keep their counters in the first 256 bytes, so
    the partial states of one never land on the other's counters."""
    base = W.get_config("c3")
    runs = []
    for batch in (8, 2):
        cfg = base.with_(batch=batch, name=f"shared-ws-{batch}")
        runs.append(Run(cfg, W.initial_positions(cfg), 4, cuda))
    assert all(r.ws is not None for r in runs)
    ws = torch.zeros(max(r.ws.numel() for r in runs), dtype=torch.uint8, device=cuda)
    for r in runs:
        r.ws = ws
    hists = [r.history(np.arange(r.cfg.batch), 3) for r in runs]
    for i in range(4):
        for r, hist in zip(runs, hists):
            q, out = r.step()
            rows = np.arange(r.cfg.batch)
            compare(r.cfg, to_np(out), r.oracle_out(rows, i, q, hist=hist),
                    what=f"{r.cfg.name} step {i}")
            assert not ws[:256].any().item(), f"{r.cfg.name} step {i}: counters not zero"


@pytest.mark.parametrize("mode,dtype,d,hq,hkv,block,window,slots,rope", [
    ("pbb", "bf16", 128, 32, 8, 2048, 0, 2048, 0.0),    # 32 units: a split launch
    ("pbb", "f32", 64, 4, 1, 64, 0, 64, 0.0),
    ("swa", "bf16", 128, 8, 2, 0, 4096, 4096, 0.0),
    ("pbb", "bf16", 64, 12, 2, 128, 0, 128, 1e6),
])
def test_positions_at_int32_limit(cuda, mode, dtype, d, hq, hkv, block, window, slots, rope):
    """Positions up to 2^31 - 2, the largest the boundary admits: the last block before 2^31
    entered, bridged and left, every output against the oracle and the rings bit for bit."""
    steps = 4
    top = (1 << 31) - 2                      # last admissible position
    B = block if mode == "pbb" else slots
    t0 = torch.tensor([top - steps + 1,      # ends on the last admissible position
                       (1 << 31) - B - 1,    # crosses into the final block
                       (1 << 31) - B + 5,    # inside the bridge of the final block
                       (1 << 31) - B // 2 - 2],  # leaves the bridge (r crosses h)
                      dtype=torch.int64)
    assert int(t0.max()) + steps - 1 <= top
    cfg = W.Config(f"int32-limit-{mode}-{dtype}-{d}", mode, batch=4, hq=hq, hkv=hkv, d=d,
                   block=block, slots=slots, window=window, dtype=dtype, seed=23,
                   value_scale=1.0, pos_hi=0, steps=steps, prefill=True, rope_base=rope)
    print(f"[int32-limit] {cfg.name}", flush=True)
    run = Run(cfg, t0, steps, cuda)
    rows = np.arange(4)
    hist = run.history(rows, steps - 1)
    for i in range(steps):
        q, out = run.step()
        compare(cfg, to_np(out), run.oracle_out(rows, i, q, hist=hist), what=f"{cfg.name} step {i}")
    assert np.array_equal(run.ring_rows(rows, "v"), run.expected_ring(rows, steps - 1, "v", hist=hist))
    if not rope:
        assert np.array_equal(run.ring_rows(rows, "k"),
                              run.expected_ring(rows, steps - 1, "k", hist=hist))
    else:
        # rotated keys: within one bf16 rounding of their exact rotation
        exact = run.expected_rotated_keys(rows, steps - 1, hist=hist)
        got = run.ring_rows(rows, "k").view(np.uint16).astype(np.uint32) << 16
        err = np.abs(got.view(np.float32).astype(np.float64) - exact)
        assert (err <= np.abs(exact) * 2.0 ** -8 + 1e-6).all()
    assert int(run.pos.max()) == top + 1


@pytest.mark.parametrize("mode,dtype,hq,hkv,B", [
    ("pbb", "bf16", 8, 1, 65536),   # one unit: a split launch over the longest supports
    ("pbb", "f32", 4, 1, 65536),
    ("swa", "bf16", 4, 2, 65536),
])
def test_largest_ring(cuda, mode, dtype, hq, hkv, B):
    """Rings of the largest admitted size (65536 slots) with supports of up to 65536 keys:
    the bridge at its longest (phase h - 1 after a full block), a block's first phase, its
    last phase, and an SWA window of 65536."""
    h = B // 2
    t0 = torch.tensor([B + h - 2, 2 * B, 2 * B - 1], dtype=torch.int64)  # phases h-2.., 0.., B-1..
    steps = 2
    window = B if mode == "swa" else 0
    cfg = W.Config(f"largest-ring-{mode}-{dtype}", mode, batch=3, hq=hq, hkv=hkv, d=64,
                   block=B if mode == "pbb" else 0, slots=B, window=window, dtype=dtype,
                   seed=29, value_scale=1.0, pos_hi=0, steps=steps, prefill=True)
    print(f"[largest-ring] {cfg.name}", flush=True)
    run = Run(cfg, t0, steps, cuda)
    rows = np.arange(3)
    hist = run.history(rows, steps - 1)
    for i in range(steps):
        q, out = run.step()
        compare(cfg, to_np(out), run.oracle_out(rows, i, q, hist=hist), what=f"{cfg.name} step {i}")
    for which in ("k", "v"):
        assert np.array_equal(run.ring_rows(rows, which),
                              run.expected_ring(rows, steps - 1, which, hist=hist)), which
