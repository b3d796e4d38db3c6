"""Paper-shape decode (batch 1, two KV heads, head_dim 64, B = 128) and HIP-graph replay.

The decode workload the paper times (Sec. 5; Appendix F.2): batch 1, two KV heads, head_dim 64,
10/12/14 query heads, block 128 (bridge 64), position origins from 8K to 1M.  Parity: 384
sequential steps against the oracle with the ring compared bit for bit (the paper's own
sequential check spans 384 steps).  Graph replay: a captured 256-step sequence (decode + position
advance on the device) reproduces eager execution bit for bit, on every replay, for the last
output, all outputs and the full ring contents.
"""
import numpy as np
import pytest
import torch

import paper_2606_02680_amd as P
import workloads as W
from tests.harness import Run, bits, compare, to_np

pytestmark = pytest.mark.gpu


def paper_cfg(hq, origin, mode="pbb"):
    if mode == "pbb":
        return W.Config(f"paper-{hq}", "pbb", batch=1, hq=hq, hkv=2, d=64, block=128, slots=128,
                        window=0, dtype="bf16", seed=11, value_scale=1.0, pos_hi=0, steps=384,
                        prefill=True)
    return W.Config(f"paper-swa-{hq}", "swa", batch=1, hq=hq, hkv=2, d=64, block=128, slots=256,
                    window=128, dtype="bf16", seed=11, value_scale=1.0, pos_hi=0, steps=384,
                    prefill=True)


@pytest.mark.parametrize("hq,origin", [(12, 8192), (10, 1 << 20), (14, 65536 + 37)])
@pytest.mark.parametrize("mode", ["pbb", "swa"])
def test_paper_shape_384_steps(cuda, hq, origin, mode):
    cfg = paper_cfg(hq, origin, mode)
    t0 = torch.tensor([origin], dtype=torch.int64)
    run = Run(cfg, t0, cfg.steps, cuda)
    rows = np.array([0])
    hist = run.history(rows, cfg.steps - 1)
    print(f"[paper] {cfg.name} origin={origin}", flush=True)
    for i in range(cfg.steps):
        q, out = run.step()
        ref = run.oracle_out(rows, i, q, hist=hist)
        compare(cfg, to_np(out), ref, what=f"{cfg.name} step {i}")
        if i % 64 == 0 or i == cfg.steps - 1:
            for which in ("k", "v"):
                exp = run.expected_ring(rows, i, which, hist=hist)
                assert np.array_equal(run.ring_rows(rows, which), exp), (cfg.name, i, which)


def _captured_sequence(desc, fn, pos, k_ring, v_ring, qs, ks, vs, outs):
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for i in range(qs.shape[0]):
            fn(desc, pos, qs[i], ks[i], vs[i], k_ring, v_ring, outs[i])
            pos.add_(1)
    return g


@pytest.mark.parametrize("mode", ["pbb", "swa"])
def test_graph_replay_matches_eager_bitwise(cuda, mode):
    steps = 256
    cfg = paper_cfg(12, 8192, mode)
    t0 = torch.tensor([8192], dtype=torch.int64)
    run = Run(cfg, t0, steps, cuda)
    qs = W.q_steps(cfg, t0, 0, steps, device=cuda)
    ks = W.kv_steps(cfg, "k", t0, 0, steps, device=cuda)
    vs = W.kv_steps(cfg, "v", t0, 0, steps, device=cuda)
    snap = (run.k_ring.clone(), run.v_ring.clone(), run.pos.clone())
    fn = P.swa_decode_step if mode == "swa" else P.pbb_decode_step

    eager = torch.empty_like(qs)
    for i in range(steps):
        fn(run.desc, run.pos, qs[i], ks[i], vs[i], run.k_ring, run.v_ring, eager[i])
        run.pos += 1
    torch.cuda.synchronize()
    eager_k, eager_v, eager_pos = run.k_ring.clone(), run.v_ring.clone(), run.pos.clone()

    def restore():
        run.k_ring.copy_(snap[0])
        run.v_ring.copy_(snap[1])
        run.pos.copy_(snap[2])

    outs = torch.zeros_like(qs)
    restore()
    g = _captured_sequence(run.desc, fn, run.pos, run.k_ring, run.v_ring, qs, ks, vs, outs)
    for rep in range(3):
        restore()
        outs.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs.view(torch.int16), eager.view(torch.int16)), f"replay {rep} outputs"
        assert torch.equal(outs[-1].view(torch.int16), eager[-1].view(torch.int16))
        assert torch.equal(run.k_ring.view(torch.int16), eager_k.view(torch.int16)), f"replay {rep} K"
        assert torch.equal(run.v_ring.view(torch.int16), eager_v.view(torch.int16)), f"replay {rep} V"
        assert torch.equal(run.pos, eager_pos)
        # eager work between replays
        _ = (qs[0].float() * 2).sum().item()


@pytest.mark.parametrize("mode", ["pbb", "swa"])
def test_advance_variant_matches_plain_steps(cuda, mode):
    """decode_step_advance with two alternating position buffers gives the same outputs, rings
    and positions as decode_step followed by pos += 1; eager and captured-graph replays agree
    bit for bit."""
    steps = 130
    cfg = paper_cfg(14, 65536 + 5, mode)
    t0 = torch.tensor([65536 + 5], dtype=torch.int64)
    run = Run(cfg, t0, steps, cuda)
    qs = W.q_steps(cfg, t0, 0, steps, device=cuda)
    ks = W.kv_steps(cfg, "k", t0, 0, steps, device=cuda)
    vs = W.kv_steps(cfg, "v", t0, 0, steps, device=cuda)
    snap = (run.k_ring.clone(), run.v_ring.clone(), run.pos.clone())
    plain = P.swa_decode_step if mode == "swa" else P.pbb_decode_step
    adv = P.swa_decode_step_advance if mode == "swa" else P.pbb_decode_step_advance

    ref = torch.empty_like(qs)
    for i in range(steps):
        plain(run.desc, run.pos, qs[i], ks[i], vs[i], run.k_ring, run.v_ring, ref[i])
        run.pos += 1
    torch.cuda.synchronize()
    ref_k, ref_v, ref_pos = run.k_ring.clone(), run.v_ring.clone(), run.pos.clone()

    pos2 = [snap[2].clone(), torch.full_like(snap[2], -7)]

    def restore():
        run.k_ring.copy_(snap[0])
        run.v_ring.copy_(snap[1])
        pos2[0].copy_(snap[2])
        pos2[1].fill_(-7)

    def body(outs):
        for i in range(steps):
            adv(run.desc, pos2[i % 2], pos2[(i + 1) % 2], qs[i], ks[i], vs[i], run.k_ring,
                run.v_ring, outs[i])

    outs = torch.zeros_like(qs)
    restore()
    body(outs)
    torch.cuda.synchronize()

    def check(tag):
        assert torch.equal(outs.view(torch.int16), ref.view(torch.int16)), tag
        assert torch.equal(run.k_ring.view(torch.int16), ref_k.view(torch.int16)), tag
        assert torch.equal(run.v_ring.view(torch.int16), ref_v.view(torch.int16)), tag
        assert torch.equal(pos2[steps % 2], ref_pos), tag
        assert torch.equal(pos2[1 - steps % 2], ref_pos - 1), tag

    check("eager")
    restore()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        body(outs)
    for rep in range(3):
        restore()
        outs.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check(f"replay {rep}")


def test_graph_replay_with_split_workgroups(cuda):
    """A split launch (one sequence at c3's head shapes: each unit over 8 workgroups that merge
    through the workspace, whose counters every launch leaves at zero) captured as a 48-step
    graph with on-device position advance: every replay reproduces eager execution bit for
    bit."""
    steps = 48
    cfg = W.Config("split-graph", "pbb", batch=1, hq=32, hkv=8, d=128, block=2048, slots=2048,
                   window=0, dtype="bf16", seed=17, value_scale=1.0, pos_hi=200000, steps=steps,
                   prefill=True)
    t0 = W.initial_positions(cfg)
    run = Run(cfg, t0, steps, cuda)
    ws = run.ws
    assert ws is not None and ws.numel() > 0
    qs = W.q_steps(cfg, t0, 0, steps, device=cuda)
    ks = W.kv_steps(cfg, "k", t0, 0, steps, device=cuda)
    vs = W.kv_steps(cfg, "v", t0, 0, steps, device=cuda)
    snap = (run.k_ring.clone(), run.v_ring.clone())
    pos = [run.pos.clone(), torch.zeros_like(run.pos)]
    eager = torch.empty_like(qs)
    for i in range(steps):
        P.pbb_decode_step_advance(run.desc, pos[i % 2], pos[(i + 1) % 2], qs[i], ks[i], vs[i],
                                  run.k_ring, run.v_ring, eager[i], workspace=ws)
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
        for i in range(steps):
            P.pbb_decode_step_advance(run.desc, pos[i % 2], pos[(i + 1) % 2], qs[i], ks[i], vs[i],
                                      run.k_ring, run.v_ring, outs[i], workspace=ws)
    for rep in range(3):
        restore()
        outs.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(outs.view(torch.int16), eager.view(torch.int16)), rep
        assert torch.equal(run.k_ring.view(torch.int16), ref_k.view(torch.int16)), rep
        assert torch.equal(run.v_ring.view(torch.int16), ref_v.view(torch.int16)), rep
        assert not ws[: 4 * cfg.batch * cfg.hkv].any().item()
        _ = (qs[0].float() * 2).sum().item()
