"""GPU parity of the prefill entry points (``pbb_prefill``, ``swa_prefill``) against the fp64
oracle, through the C ABI.

Every position of every sequence is compared: outputs at the bf16 tolerance of the decode
tests, log-partitions within 2e-3 (fp32 running sums of the same bf16 inputs); ring state
after the prompt bit for bit (slot s mod slots holds the last prompt position s); and
decoding continued from that ring at position n matches the oracle over prompt plus new
tokens.  Shapes cover group sizes 1..16 including ones that do not divide the 128-column tile
(5, 6, 7), both head dims, blocks from 2 to 2048, prompts shorter than one tile and ragged
tails, and the sliding window.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as W
from tests.harness import bits, compare, error_stats, record_stats, to_np

pytestmark = pytest.mark.gpu


def _cfg(mode, batch, n, hq, hkv, d, block=0, window=0, slots=0, seed=31, scale=1.0):
    return W.Config(f"prefill-{mode}-{batch}-{n}-{hq}-{hkv}-{d}-{block}-{window}", mode,
                    batch=batch, hq=hq, hkv=hkv, d=d, block=block,
                    slots=slots or (block if mode == "pbb" else window), window=window,
                    dtype="bf16", seed=seed, value_scale=scale, pos_hi=0, steps=n)


def _desc(cfg):
    if cfg.mode == "swa":
        return P.make_desc(cfg.batch, cfg.hq, cfg.hkv, cfg.d, window=cfg.window, slots=cfg.slots,
                           dtype=torch.bfloat16)
    return P.make_desc(cfg.batch, cfg.hq, cfg.hkv, cfg.d, block=cfg.block, dtype=torch.bfloat16)


def _run(cfg, n, device, rings=True):
    q, k, v = W.prompt(cfg, n, device=device)
    desc = _desc(cfg)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((cfg.batch, cfg.hq, n), float("nan"), dtype=torch.float32, device=device)
    kr = vr = None
    if rings:
        kr, vr = P.alloc_rings(desc, device)
        P.ring_init(desc, kr, vr)
    fn = P.swa_prefill if cfg.mode == "swa" else P.pbb_prefill
    print(f"[prefill] {cfg.name}", flush=True)
    fn(desc, q, k, v, out, lse, kr, vr)
    torch.cuda.synchronize()
    return desc, (q, k, v), out, lse, kr, vr


def _check(cfg, n, device, rings=True):
    desc, (q, k, v), out, lse, kr, vr = _run(cfg, n, device, rings)
    mode = oracle.SWA if cfg.mode == "swa" else oracle.PBB
    ref, ref_lse = oracle.prefill(mode, to_np(q), to_np(k), to_np(v), block=cfg.block,
                                  window=cfg.window)
    compare(cfg, to_np(out), ref, what=cfg.name)
    got_lse = lse.cpu().numpy().astype(np.float64)
    assert np.isfinite(got_lse).all()
    assert np.abs(got_lse - ref_lse).max() <= 2e-3, np.abs(got_lse - ref_lse).max()
    record_stats(cfg.name, {**error_stats(to_np(out), ref),
                            "lse_max_abs": float(np.abs(got_lse - ref_lse).max())})
    if rings:
        kh = k.permute(0, 2, 1, 3).contiguous().cpu()
        vh = v.permute(0, 2, 1, 3).contiguous().cpu()
        zeros = np.zeros(kr.shape, dtype=np.int16)
        for name, hist, ring in (("k", kh, kr), ("v", vh, vr)):
            exp = oracle.expected_ring(bits(hist), np.zeros(cfg.batch), np.full(cfg.batch, n - 1),
                                       np.zeros(cfg.batch), desc.slots, initial=zeros)
            assert np.array_equal(bits(ring), exp), f"{cfg.name} ring {name}"
    return desc, (q, k, v), out, lse, kr, vr


@pytest.mark.parametrize("mode,batch,n,hq,hkv,d,block,window,slots", [
    ("pbb", 2, 300, 8, 2, 64, 64, 0, 0),         # G = 4, several blocks, ragged tail
    ("pbb", 1, 600, 12, 2, 64, 128, 0, 0),       # paper shape, G = 6 (21 positions / tile)
    ("pbb", 1, 257, 10, 2, 64, 128, 0, 0),       # G = 5
    ("pbb", 1, 200, 14, 2, 64, 128, 0, 0),       # G = 7
    ("pbb", 2, 333, 32, 8, 128, 256, 0, 0),      # G = 4, head_dim 128
    ("pbb", 1, 150, 16, 1, 128, 32, 0, 0),       # G = 16: 8 positions per tile
    ("pbb", 1, 77, 4, 4, 64, 2, 0, 0),           # G = 1, B = 2 (h = 1)
    ("pbb", 1, 5000, 8, 2, 128, 2048, 0, 0),     # long block, bridge rectangles of 1024
    ("pbb", 3, 17, 6, 3, 64, 16, 0, 0),          # prompt shorter than one tile
    ("pbb", 1, 1, 4, 1, 128, 64, 0, 0),          # a single position
    ("swa", 2, 300, 8, 2, 128, 0, 100, 128),     # window 100 in 128 slots
    ("swa", 1, 400, 6, 2, 64, 0, 37, 40),
    ("swa", 1, 90, 4, 1, 64, 0, 1, 1),           # window 1: each position attends to itself
])
def test_prefill_matches_oracle(cuda, mode, batch, n, hq, hkv, d, block, window, slots):
    cfg = _cfg(mode, batch, n, hq, hkv, d, block, window, slots)
    _check(cfg, n, cuda)


def test_prefill_without_optional_outputs(cuda):
    cfg = _cfg("pbb", 1, 130, 8, 2, 64, 64)
    q, k, v = W.prompt(cfg, 130, device=cuda)
    desc = _desc(cfg)
    out = torch.empty_like(q)
    P.pbb_prefill(desc, q, k, v, out)
    torch.cuda.synchronize()
    ref, _ = oracle.prefill(oracle.PBB, to_np(q), to_np(k), to_np(v), block=64)
    compare(cfg, to_np(out), ref, what="no lse, no rings")


@pytest.mark.parametrize("mode,batch,n,hq,hkv,d,block,window,slots", [
    ("pbb", 1, 600, 12, 2, 64, 128, 0, 0),       # paper shape
    ("pbb", 2, 700, 8, 2, 128, 256, 0, 0),
    ("swa", 1, 500, 8, 2, 128, 0, 100, 128),
])
def test_prefill_rising_scores(cuda, mode, batch, n, hq, hkv, d, block, window, slots):
    """Scores that jump above everything the walk has seen: every query carries 8 in channel 0
    and a few keys carry a boost there worth about 4 or about 40 log2 units of score (3 % and
    2 % of keys), so within most tiles the softmax's dominant keys first appear after the first
    key step.  Small rises keep the softmax reference (weights up to ~2^4); large ones move it
    mid-walk, the dominant key becoming the reference.  Outputs (dominated by the boosted keys'
    values) and log-partitions (up to ~30 in natural-log units) against the oracle on the same
    bf16 inputs."""
    cfg = _cfg(mode, batch, n, hq, hkv, d, block, window, slots, seed=53)
    q, k, v = W.prompt(cfg, n, device=cuda)
    c = np.log2(np.e) / np.sqrt(d)                      # log2 units per unit of q.k
    b4, b40 = float(round(4 / (8 * c))), float(round(40 / (8 * c)))
    g = torch.Generator().manual_seed(1234)
    u = torch.rand((batch, n, hkv), generator=g)
    boost = torch.where(u < 0.03, b4, torch.where(u < 0.05, b40, 0.0))
    q[..., 0] = 8.0
    k[..., 0] = boost.to(device=cuda, dtype=k.dtype)
    desc = _desc(cfg)
    out = torch.full_like(q, float("nan"))
    lse = torch.full((batch, hq, n), float("nan"), dtype=torch.float32, device=cuda)
    fn = P.swa_prefill if mode == "swa" else P.pbb_prefill
    print(f"[prefill] rising scores {cfg.name}", flush=True)
    fn(desc, q, k, v, out, lse)
    torch.cuda.synchronize()
    m = oracle.SWA if mode == "swa" else oracle.PBB
    ref, ref_lse = oracle.prefill(m, to_np(q), to_np(k), to_np(v), block=block, window=window)
    assert ref_lse.max() > 25.0                         # the boosts dominate where present
    compare(cfg, to_np(out), ref, what=f"rising scores {cfg.name}")
    got_lse = lse.cpu().numpy().astype(np.float64)
    assert np.isfinite(got_lse).all()
    assert np.abs(got_lse - ref_lse).max() <= 2e-3, np.abs(got_lse - ref_lse).max()
    record_stats(f"rising scores {cfg.name}", {**error_stats(to_np(out), ref),
                 "lse_max_abs": float(np.abs(got_lse - ref_lse).max())})


@pytest.mark.parametrize("mode,batch,hq,hkv,d,block,window,slots,n,steps", [
    ("pbb", 2, 8, 2, 128, 128, 0, 128, 700, 70),
    ("swa", 2, 8, 2, 64, 0, 100, 128, 700, 70),          # ring larger than the window
    ("pbb", 1, 32, 8, 128, 2048, 0, 2048, 3000, 20),     # decode as a split launch
])
def test_prefill_then_decode_continues(cuda, mode, batch, hq, hkv, d, block, window, slots, n,
                                       steps):
    """Rings written by prefill are the state decode needs: steps at positions n, n+1, ...
    match the oracle over prompt plus appended tokens."""
    cfg = _cfg(mode, batch, n + steps, hq, hkv, d, block, window, slots)
    desc, (q, k, v), out, lse, kr, vr = _run(cfg, n, cuda)
    qa, ka, va = W.prompt(cfg, n + steps, device=cuda)   # positions 0 .. n+steps-1
    pos = torch.full((cfg.batch,), n, dtype=torch.int32, device=cuda)
    kh = ka.permute(0, 2, 1, 3).contiguous()
    vh = va.permute(0, 2, 1, 3).contiguous()
    step = P.swa_decode_step if mode == "swa" else P.pbb_decode_step
    m = oracle.SWA if mode == "swa" else oracle.PBB
    for i in range(steps):
        t = n + i
        qd = qa[:, t].contiguous()
        o = torch.empty_like(qd)
        step(desc, pos, qd, ka[:, t].contiguous(), va[:, t].contiguous(), kr, vr, o)
        pos += 1
        if i % 7 == 0 or i == steps - 1:
            ref = oracle.decode(m, np.full(cfg.batch, t), to_np(qd), to_np(kh[:, :, :t + 1]),
                                to_np(vh[:, :, :t + 1]), np.zeros(cfg.batch, np.int64),
                                block=block, window=window)
            compare(cfg, to_np(o), ref, what=f"{mode} decode after prefill, t={t}")


def test_prefill_is_deterministic_and_leaves_inputs(cuda):
    cfg = _cfg("pbb", 2, 260, 12, 2, 64, 128)
    q, k, v = W.prompt(cfg, 260, device=cuda)
    copies = [x.clone() for x in (q, k, v)]
    desc = _desc(cfg)
    o1, o2 = torch.empty_like(q), torch.empty_like(q)
    P.pbb_prefill(desc, q, k, v, o1)
    P.pbb_prefill(desc, q, k, v, o2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    for x, c in zip((q, k, v), copies):
        assert torch.equal(x.view(torch.int16), c.view(torch.int16))


def _window_plan(n, span, mode, tail=512, npre=1024):
    """Prefix [0, npre) and a tail sub-prompt [lo, n) whose targets t >= t1 = lo + span have the
    same support as in the full prompt (lo a multiple of B for PBB: the supports are
    shift-invariant by whole blocks once the max(0, .) of a(t) is inactive)."""
    npre = min(npre, n)
    lo = n - span - tail
    if mode == "pbb":
        lo = (lo // span) * span
    return npre, max(lo, npre), max(lo, npre) + span


@pytest.mark.parametrize("name,shape", __import__("bench").PREFILL_SHAPES,
                         ids=[nm for nm, _ in __import__("bench").PREFILL_SHAPES])
def test_prefill_bench_shapes(cuda, name, shape):
    """The bench's prefill launches at full size (its grid, tiles and head shapes): a prefix and
    a block-aligned tail window of two (sequence, KV-head group) slices against the oracle."""
    mode = "pbb" if shape.get("block") else "swa"
    block, window = shape.get("block", 0), shape.get("window", 0)
    cfg = _cfg(mode, shape["batch"], shape["n"], shape["hq"], shape["hkv"], shape["d"],
               block=block, window=window, seed=7)
    n, G = shape["n"], shape["hq"] // shape["hkv"]
    desc, (q, k, v), out, lse, _, _ = _run(cfg, n, cuda, rings=False)
    npre, lo, t1 = _window_plan(n, block or window, mode)
    m = oracle.SWA if mode == "swa" else oracle.PBB
    for b, g in ((0, 0), (shape["batch"] - 1, shape["hkv"] - 1)):
        hs = slice(g * G, (g + 1) * G)
        for a0, a1, first in ((0, npre, 0), (lo, n, t1 - lo)):
            qs = to_np(q[b:b + 1, a0:a1, hs])
            ks = to_np(k[b:b + 1, a0:a1, g:g + 1])
            vs = to_np(v[b:b + 1, a0:a1, g:g + 1])
            ref, ref_lse = oracle.prefill(m, qs, ks, vs, block=block, window=window)
            got = to_np(out[b:b + 1, a0 + first:a1, hs])
            compare(cfg, got, ref[:, first:], what=f"{name} seq {b} group {g} [{a0 + first}, {a1})")
            gl = lse[b:b + 1, hs, a0 + first:a1].cpu().numpy().astype(np.float64)
            assert np.abs(gl - ref_lse[:, :, first:]).max() <= 2e-3
            record_stats(f"{name} seq {b} group {g} [{a0 + first}, {a1})",
                         {**error_stats(got, ref[:, first:]),
                          "lse_max_abs": float(np.abs(gl - ref_lse[:, :, first:]).max())})


@pytest.mark.parametrize("mode,hq,hkv,block,window", [
    ("pbb", 16, 1, 65536, 0),     # group of 16, supports up to 65536 keys
    ("swa", 4, 2, 0, 65536),
])
def test_prefill_largest_ring_sampled(cuda, mode, hq, hkv, block, window):
    """A 70000-position prompt with the largest admitted block or window (65536): outputs and
    log-partitions of sampled positions (block and bridge edges, the longest supports, the
    last position) against the decode oracle at each position over the prompt's history, and
    the ring state bit for bit."""
    n = 70000
    cfg = _cfg(mode, 1, n, hq, hkv, 64, block=block, window=window)
    desc, (q, k, v), out, lse, kr, vr = _run(cfg, n, cuda)
    B = block or window
    h = B // 2
    picks = {0, 1, 31, 32, h - 1, h, h + 1, B - 1, B, B + 1, B + h - 2, B + h - 1, B + h,
             n - 2, n - 1} | set(np.random.default_rng(5).integers(0, n, 24).tolist())
    t = np.array(sorted(p for p in picks if 0 <= p < n), dtype=np.int64)
    assert t.min() >= 0 and t.max() < n   # indices into the prompt, checked on the host
    kh = to_np(k[0].permute(1, 0, 2).contiguous())[None]   # [1][Hkv][n][d]
    vh = to_np(v[0].permute(1, 0, 2).contiguous())[None]
    m = oracle.SWA if mode == "swa" else oracle.PBB
    qs = to_np(q[0, torch.as_tensor(t, device=cuda)])     # [len(t)][Hq][d]
    ref = np.stack([oracle.decode(m, np.array([tt]), qs[i:i + 1], kh, vh, np.zeros(1, np.int64),
                                  block=block, window=window)[0] for i, tt in enumerate(t)])
    got = to_np(out[0, torch.as_tensor(t, device=cuda)])
    compare(cfg, got, ref, what=f"{cfg.name} sampled positions")
    # log-partitions in fp64 over each sampled position's support as the oracle's two-case
    # membership test (Eq.(pbb), Prop. 2) gives it
    scale = 1.0 / np.sqrt(64.0)
    G = hq // hkv
    for i, tt in enumerate(t):
        tt = int(tt)
        sup = np.array(oracle.pbb_support(tt, block) if mode == "pbb"
                       else oracle.swa_support(tt, window), dtype=np.int64)
        for hd in range(hq):
            z = kh[0, hd // G, sup].astype(np.float64) @ qs[i, hd].astype(np.float64) * scale
            ref_lse = z.max() + np.log(np.exp(z - z.max()).sum())
            assert abs(float(lse[0, hd, tt]) - ref_lse) <= 2e-3, (tt, hd)
    # ring: slot s mod slots holds the last prompt position s
    kb = bits(kr[0])
    for s in (n - 1, n - 2, n - B if n - B >= 0 else 0, n - 40000):
        assert np.array_equal(kb[:, s % desc.slots], bits(k[0, s]).reshape(hkv, -1)), s


@pytest.mark.parametrize("mode,block,window,slots", [
    ("pbb", 128, 0, 128),
    ("swa", 0, 128, 256),
])
def test_rotary_prompt_prefill_then_rotary_decode(cuda, mode, block, window, slots):
    """The paper's inference path at its head shape (Hq 12, Hkv 2, head_dim 64, B 128; RoPE
    base 10^6, App. C; cached prefill then sequential decoding, App. F.7): the prompt's q and k
    are turned by position (the oracle's exact rotation, rounded to bf16) and go through
    prefill, whose ring -- rotated keys -- then feeds decode steps that turn q and the new key
    themselves.  Prefill outputs match the oracle prefill of the turned prompt; every decode
    step matches the oracle, which turns the raw history keys exactly at their positions."""
    base, n, steps = 1e6, 700, 40
    cfg = _cfg(mode, 1, n + steps, 12, 2, 64, block, window, slots).with_(rope_base=base)
    qa, ka, va = W.prompt(cfg.with_(rope_base=0.0), n + steps, device=cuda)  # raw q, k, v
    idx = np.arange(n)[None, :, None]                                      # position of each row
    qr = torch.from_numpy(oracle.rope_rows(to_np(qa[:, :n]), idx, base)).to(cuda, torch.bfloat16)
    kr_ = torch.from_numpy(oracle.rope_rows(to_np(ka[:, :n]), idx, base)).to(cuda, torch.bfloat16)
    vp = va[:, :n].contiguous()
    plain = (P.make_desc(1, 12, 2, 64, window=window, slots=slots, dtype=torch.bfloat16)
             if mode == "swa" else P.make_desc(1, 12, 2, 64, block=block, dtype=torch.bfloat16))
    rot = (P.make_desc(1, 12, 2, 64, window=window, slots=slots, dtype=torch.bfloat16,
                       rope_base=base)
           if mode == "swa" else P.make_desc(1, 12, 2, 64, block=block, dtype=torch.bfloat16,
                                             rope_base=base))
    kring, vring = P.alloc_rings(plain, cuda)
    P.ring_init(plain, kring, vring)
    out = torch.empty_like(qr)
    lse = torch.empty((1, 12, n), dtype=torch.float32, device=cuda)
    print(f"[prefill] rotary prompt then rotary decode, {mode}", flush=True)
    (P.swa_prefill if mode == "swa" else P.pbb_prefill)(plain, qr, kr_, vp, out, lse, kring, vring)
    torch.cuda.synchronize()
    m = oracle.SWA if mode == "swa" else oracle.PBB
    ref, ref_lse = oracle.prefill(m, to_np(qr), to_np(kr_), to_np(vp), block=block, window=window)
    compare(cfg.with_(rope_base=0.0), to_np(out), ref, what=f"{mode} rotary-prompt prefill")
    assert np.abs(lse.cpu().numpy().astype(np.float64) - ref_lse).max() <= 2e-3
    kh = to_np(ka.permute(0, 2, 1, 3).contiguous())     # raw history [1][Hkv][n+steps][d]
    vh = to_np(va.permute(0, 2, 1, 3).contiguous())
    pos = torch.full((1,), n, dtype=torch.int32, device=cuda)
    step = P.swa_decode_step if mode == "swa" else P.pbb_decode_step
    for i in range(steps):
        t = n + i
        qd = qa[:, t].contiguous()
        o = torch.empty_like(qd)
        step(rot, pos, qd, ka[:, t].contiguous(), va[:, t].contiguous(), kring, vring, o)
        pos += 1
        ref = oracle.decode(m, np.array([t]), to_np(qd), kh[:, :, :t + 1], vh[:, :, :t + 1],
                            np.zeros(1, np.int64), block=block, window=window, rope_base=base)
        compare(cfg, to_np(o), ref, what=f"{mode} rotary decode after rotary prefill, t={t}")
