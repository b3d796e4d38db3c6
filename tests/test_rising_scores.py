"""Decode over supports whose scores jump far above what a wave has seen (through the C ABI,
against the fp64 oracle): every query carries 8 in channel 0 and a few keys carry a boost there
worth about 4 or about 40 log2 units of score (3 % and 2 % of positions), so the dominant keys of
a support often sit in a later key step than a wave's first one.  Small rises keep the softmax
reference; large ones move it mid-walk, the dominant key becoming the reference (Eq.(lse)
rescaling).  Cases: the stepped kernel (4 and 2 waves), split launches and whole-ring launches,
each decoding from position 0 across block starts and bridges.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2606_02680_amd as P
import workloads as WL
from tests.harness import compare, desc_for, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,batch,hq,hkv,d,B,steps", [
    ("stepped4", 20, 32, 8, 128, 256, 300),     # 160 units: 4-wave workgroups, unsplit
    ("stepped2", 160, 16, 2, 128, 256, 300),    # 320 units, groups of 8: 2-wave workgroups
    ("split", 2, 32, 8, 128, 2048, 300),        # 16 units: split over workgroups
    ("whole", 2, 12, 2, 64, 128, 300),          # whole-ring launches (paper shape)
])
def test_decode_rising_scores(cuda, name, batch, hq, hkv, d, B, steps):
    cfg = WL.Config(f"rising-{name}", "pbb", batch=batch, hq=hq, hkv=hkv, d=d, block=B,
                    slots=B, window=0, dtype="bf16", seed=97, value_scale=1.0, pos_hi=0,
                    steps=steps)
    desc = desc_for(cfg, batch=batch)
    kr, vr = P.alloc_rings(desc, cuda)
    P.ring_init(desc, kr, vr)
    ws = P.alloc_workspace(desc, cuda)
    pos = torch.zeros(batch, dtype=torch.int32, device=cuda)
    c = np.log2(np.e) / np.sqrt(d)                      # log2 units per unit of q.k
    b4, b40 = float(round(4 / (8 * c))), float(round(40 / (8 * c)))
    g = torch.Generator().manual_seed(4321)
    u = torch.rand((batch, hkv, steps), generator=g)
    boost = torch.where(u < 0.03, b4, torch.where(u < 0.05, b40, 0.0)).to(torch.bfloat16)
    seq = torch.arange(batch, dtype=torch.int64)
    rows = np.arange(batch) if batch <= 8 else np.arange(0, batch, batch // 8)
    kh = torch.empty((len(rows), hkv, steps, d), dtype=torch.bfloat16)
    vh = torch.empty_like(kh)
    print(f"[rising] {cfg.name}", flush=True)
    for t in range(steps):
        p = torch.full((batch,), t, dtype=torch.int64)
        q = WL.q_at(cfg, p, device=cuda).contiguous()
        k = WL.kv_at(cfg, "k", seq, p.view(-1, 1), device=cuda)[:, :, 0, :].contiguous()
        v = WL.kv_at(cfg, "v", seq, p.view(-1, 1), device=cuda)[:, :, 0, :].contiguous()
        q[..., 0] = 8.0
        k[..., 0] = boost[:, :, t].to(cuda)
        kh[:, :, t] = k[torch.as_tensor(rows, device=cuda)].cpu()
        vh[:, :, t] = v[torch.as_tensor(rows, device=cuda)].cpu()
        out = torch.empty_like(q)
        P.pbb_decode_step(desc, pos, q, k, v, kr, vr, out, ws)
        pos += 1
        if t % 10 == 9 or t == steps - 1:
            ref = oracle.decode(oracle.PBB, np.full(len(rows), t), to_np(q)[rows],
                                to_np(kh[:, :, :t + 1]), to_np(vh[:, :, :t + 1]),
                                np.zeros(len(rows), np.int64), block=B)
            compare(cfg, to_np(out)[rows], ref, what=f"{cfg.name} t={t}")
