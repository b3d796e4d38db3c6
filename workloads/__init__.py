"""Seeded synthetic decode workloads shared by the tests, the benchmark and the smoke check.

This package holds shapes, seeds and random-number generation only: none of the attention
method's arithmetic (no supports, no slot mapping, no softmax).  Both the CPU oracle and the
HIP library consume the tensors it produces; neither of them imports it.
"""
from .configs import CONFIGS, Config, get_config  # noqa: F401
from .gen import (  # noqa: F401
    hash_normal, kv_at, kv_steps, kv_window, prompt, q_at, q_steps, initial_positions,
    spike_mask)
