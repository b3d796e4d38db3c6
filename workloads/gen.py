"""Counter-based synthetic tensors.

Every value is a pure function of (seed, stream, sequence, head, absolute position, channel),
so a key written at position ``s`` is the same number whether it reaches the ring through a
pre-fill window or through a decode-step append, and any window of history can be produced
on demand without materialising the whole sequence.

Generator: a 64-bit counter ``((seq*H + head) * 2^23 + pos) * 256 + channel`` is hashed with
the 32-bit "lowbias32" integer mixer (C. Wellons, "Prospecting for Hash Functions", 2018)
keyed by (seed, stream); two hashes feed a Box-Muller transform (Box and Muller, 1958) that
gives one N(0, 1) sample, evaluated in float64 and rounded to the target dtype by PyTorch's
round-to-nearest-even conversion.  All integer steps are exact in int64 on any device.
"""
from __future__ import annotations

import math

import torch

_M32 = 0xFFFFFFFF
POS_BITS = 23          # positions must stay below 2^23 (8M)
CH_BITS = 8            # channels below 256

STREAM_Q, STREAM_K, STREAM_V, STREAM_SPIKE = 11, 22, 33, 44


def _mix32(x: torch.Tensor) -> torch.Tensor:
    x = x & _M32
    x = x ^ (x >> 16)
    x = (x * 0x7FEB352D) & _M32
    x = x ^ (x >> 15)
    x = (x * 0x846CA68B) & _M32
    x = x ^ (x >> 16)
    return x


def _hash(counter: torch.Tensor, seed: int, stream: int, lane: int) -> torch.Tensor:
    key = ((seed * 0x9E3779B1) ^ (stream * 0x85EBCA77) ^ (lane * 0xC2B2AE3D)) & _M32
    hi = (counter >> 32) & _M32
    lo = counter & _M32
    h = _mix32(hi ^ key)
    h = _mix32(lo ^ h)
    return _mix32(h ^ key)


def hash_normal(counter: torch.Tensor, seed: int, stream: int) -> torch.Tensor:
    """float64 N(0,1) sample for every int64 counter (same shape and device)."""
    h1 = _hash(counter, seed, stream, 1)
    h2 = _hash(counter, seed, stream, 2)
    u1 = ((h1 >> 8).to(torch.float64) + 0.5) * (1.0 / 16777216.0)   # (0, 1)
    u2 = (h2 >> 8).to(torch.float64) * (1.0 / 16777216.0)           # [0, 1)
    return torch.sqrt(-2.0 * torch.log(u1)) * torch.cos((2.0 * math.pi) * u2)


def _dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def _counter(seq: torch.Tensor, heads: int, pos: torch.Tensor, d: int, device) -> torch.Tensor:
    """Counters [n_seq][heads][n_pos][d] for sequences ``seq`` [n_seq] and positions
    ``pos`` [n_seq][n_pos] (int64)."""
    seq = seq.to(device=device, dtype=torch.int64).view(-1, 1, 1, 1)
    h = torch.arange(heads, device=device, dtype=torch.int64).view(1, -1, 1, 1)
    p = pos.to(device=device, dtype=torch.int64).unsqueeze(1).unsqueeze(-1)
    c = torch.arange(d, device=device, dtype=torch.int64).view(1, 1, 1, -1)
    return (((seq * heads + h) << POS_BITS) + p) << CH_BITS | c


def spike_mask(cfg, seq: torch.Tensor, pos: torch.Tensor) -> torch.Tensor:
    """Bool [n_seq][n_pos]: (sequence, position) pairs whose K and V are scaled."""
    if cfg.spike_prob <= 0.0:
        return torch.zeros(pos.shape, dtype=torch.bool, device=pos.device)
    ctr = (seq.to(pos.device, torch.int64).view(-1, 1) << POS_BITS) + pos.to(torch.int64)
    h = _hash(ctr, cfg.seed, STREAM_SPIKE, 3)
    return h < int(cfg.spike_prob * 4294967296.0)


def _normal_block(cfg, stream: int, seq: torch.Tensor, heads: int, pos: torch.Tensor, device,
                  spike: bool, chunk: int) -> torch.Tensor:
    """N(0,1)*value_scale values [n_seq][heads][n_pos][d] (workload dtype) for sequences
    ``seq`` and absolute positions ``pos`` [n_seq][n_pos]; negative positions give zeros."""
    n_seq, n_pos = pos.shape
    out = torch.empty((n_seq, heads, n_pos, cfg.d), dtype=_dtype(cfg.dtype), device=device)
    per = max(1, chunk // max(1, heads * n_pos * cfg.d))
    for i in range(0, n_seq, per):
        sq = seq[i:i + per].to(device)
        ps = pos[i:i + per].to(device)
        valid = ps >= 0
        ctr = _counter(sq, heads, ps.clamp(min=0), cfg.d, device)
        x = hash_normal(ctr, cfg.seed, stream) * cfg.value_scale
        if spike and cfg.spike_prob > 0.0:
            m = spike_mask(cfg, sq, ps.clamp(min=0))
            x = torch.where(m.unsqueeze(1).unsqueeze(-1), x * cfg.spike_scale, x)
        x = torch.where(valid.unsqueeze(1).unsqueeze(-1), x, torch.zeros((), dtype=x.dtype,
                                                                          device=x.device))
        out[i:i + per] = x.to(out.dtype)
    return out


def kv_at(cfg, which: str, seq: torch.Tensor, pos: torch.Tensor, device="cpu",
          chunk: int = 1 << 24) -> torch.Tensor:
    """Keys (``which='k'``) or values (``'v'``) at absolute positions.

    ``seq``: int [n_seq] sequence ids; ``pos``: int [n_seq][n_pos] absolute positions
    (entries < 0 give zeros).  Returns [n_seq][Hkv][n_pos][d] in the workload dtype.
    """
    stream = {"k": STREAM_K, "v": STREAM_V}[which]
    seq = torch.as_tensor(seq, dtype=torch.int64).view(-1)
    pos = torch.as_tensor(pos, dtype=torch.int64).view(seq.numel(), -1)
    return _normal_block(cfg, stream, seq, cfg.hkv, pos, device, True, chunk)


def kv_steps(cfg, which: str, t0: torch.Tensor, first: int, n: int, device="cpu") -> torch.Tensor:
    """New keys/values of ``n`` consecutive decode steps: [n][batch][Hkv][d], step ``i``
    holding position ``t0[b] + first + i``."""
    t0 = torch.as_tensor(t0, dtype=torch.int64).view(-1)
    pos = t0.view(-1, 1) + first + torch.arange(n, dtype=torch.int64).view(1, -1)
    x = kv_at(cfg, which, torch.arange(t0.numel(), dtype=torch.int64), pos, device=device)
    return x.permute(2, 0, 1, 3).contiguous()


def q_steps(cfg, t0: torch.Tensor, first: int, n: int, device="cpu") -> torch.Tensor:
    """Queries of ``n`` consecutive decode steps: [n][batch][Hq][d]."""
    t0 = torch.as_tensor(t0, dtype=torch.int64).view(-1)
    pos = t0.view(-1, 1) + first + torch.arange(n, dtype=torch.int64).view(1, -1)
    seq = torch.arange(t0.numel(), dtype=torch.int64)
    x = _normal_block(cfg, STREAM_Q, seq, cfg.hq, pos, device, False, 1 << 24)
    return x.permute(2, 0, 1, 3).contiguous()


def kv_window(cfg, which: str, t0: torch.Tensor, length: int, device="cpu") -> torch.Tensor:
    """History window [batch][Hkv][length][d]: positions ``t0[b]-length .. t0[b]-1``
    (negative positions give zeros)."""
    t0 = torch.as_tensor(t0, dtype=torch.int64).view(-1)
    offs = torch.arange(-length, 0, dtype=torch.int64)
    pos = t0.view(-1, 1) + offs.view(1, -1)
    seq = torch.arange(t0.numel(), dtype=torch.int64)
    return kv_at(cfg, which, seq, pos, device=device)


def q_at(cfg, pos: torch.Tensor, device="cpu") -> torch.Tensor:
    """Queries [batch][Hq][d] of every sequence decoding absolute position ``pos[b]``."""
    pos = torch.as_tensor(pos, dtype=torch.int64).view(-1)
    seq = torch.arange(pos.numel(), dtype=torch.int64)
    x = _normal_block(cfg, STREAM_Q, seq, cfg.hq, pos.view(-1, 1), device, False, 1 << 24)
    return x[:, :, 0, :].contiguous()


def prompt(cfg, n: int, device="cpu"):
    """Prompt tensors for positions ``0 .. n-1`` of every sequence, token-major:
    ``q`` [batch][n][Hq][d] and ``k``, ``v`` [batch][n][Hkv][d].  Position ``s`` carries the
    same values as decoding position ``s`` (``q_at``, ``kv_at``)."""
    seq = torch.arange(cfg.batch, dtype=torch.int64)
    pos = torch.arange(n, dtype=torch.int64).view(1, -1).expand(cfg.batch, n)
    q = _normal_block(cfg, STREAM_Q, seq, cfg.hq, pos, device, False, 1 << 24)
    k = kv_at(cfg, "k", seq, pos, device=device)
    v = kv_at(cfg, "v", seq, pos, device=device)
    return (q.permute(0, 2, 1, 3).contiguous(), k.permute(0, 2, 1, 3).contiguous(),
            v.permute(0, 2, 1, 3).contiguous())


def initial_positions(cfg) -> torch.Tensor:
    """int64 [batch] first decode position of every sequence (zeros, or U[0, pos_hi))."""
    if cfg.pos_hi <= 0:
        return torch.zeros(cfg.batch, dtype=torch.int64)
    g = torch.Generator().manual_seed(cfg.seed * 1000003 + 17)
    return torch.randint(0, cfg.pos_hi, (cfg.batch,), generator=g, dtype=torch.int64)
