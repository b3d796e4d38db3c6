"""Decode workload presets.

Each preset names the shapes, dtype, seed, value distribution and position recipe of one
synthetic workload.  The sizes follow the paper's decode setting scaled to one MI355X:
batched sequences, grouped-query heads sharing KV heads, and block/ring sizes B.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Config:
    name: str
    mode: str            # "pbb" or "swa"
    batch: int
    hq: int              # query heads
    hkv: int             # KV heads
    d: int               # head dimension
    block: int           # PBB block size B (ring slots for PBB)
    slots: int           # ring slots actually allocated
    window: int          # SWA window W (0 for PBB)
    dtype: str           # "f32" or "bf16"
    seed: int
    value_scale: float   # q, k, v ~ N(0, 1) * value_scale
    pos_hi: int          # initial positions ~ U[0, pos_hi); 0 means every sequence starts at 0
    steps: int           # decode steps of the workload
    spike_prob: float = 0.0   # probability that a (sequence, position) has K and V scaled
    spike_scale: float = 1.0  # the scale applied to spiked positions
    prefill: bool = False     # rings hold the history before the first position
    rope_base: float = 0.0    # > 0: decode applies rotary positions with this base

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS = {
    # Tiny fp32: 256 steps from an empty ring with B = 64 (blocks 0..3).
    "c1": Config("c1-tiny-fp32", "pbb", batch=1, hq=4, hkv=1, d=64, block=64, slots=64,
                 window=0, dtype="f32", seed=1, value_scale=1.0, pos_hi=0, steps=256),
    # bf16, GQA 4:1, lockstep from position 0 for 2048 steps (every phase r hit 4 times).
    "c2": Config("c2-lockstep-bf16", "pbb", batch=32, hq=16, hkv=4, d=64, block=512, slots=512,
                 window=0, dtype="bf16", seed=2, value_scale=0.125, pos_hi=0, steps=2048),
    # bf16 throughput: 256 sequences at mixed positions in [0, 512K), pre-filled rings.
    "c3": Config("c3-throughput-bf16", "pbb", batch=256, hq=32, hkv=8, d=128, block=2048,
                 slots=2048, window=0, dtype="bf16", seed=3, value_scale=1.0, pos_hi=524288,
                 steps=1000, prefill=True),
    # bf16 ragged GQA 8:1: 1024 sequences at positions in [0, 64K), 1% of tokens with K,V x4.
    "c4": Config("c4-ragged-gqa8-bf16", "pbb", batch=1024, hq=16, hkv=2, d=128, block=1024,
                 slots=1024, window=0, dtype="bf16", seed=4, value_scale=1.0, pos_hi=65536,
                 steps=1000, spike_prob=0.01, spike_scale=4.0, prefill=True),
    # Sliding-window ring baseline on c3's shapes and tensors: W = 2B = 4096 in 4096 slots.
    "c5": Config("c5-swa-ring-bf16", "swa", batch=256, hq=32, hkv=8, d=128, block=2048,
                 slots=4096, window=4096, dtype="bf16", seed=3, value_scale=1.0, pos_hi=524288,
                 steps=1000, prefill=True),
}


def get_config(name: str) -> Config:
    return CONFIGS[name]
