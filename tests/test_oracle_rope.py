"""Pins for the oracle's rotary position embedding and RoPE decode (CPU only).

RoPE (base 10^6 in the paper's models, Appendix C) with half-split pairs (channel c with
c + d/2, as in the Qwen2.5 decoders the paper trains).  Pinned by hand-computed values (d = 4,
position 1), the identity at position 0, composition of rotations, the relative-position
property of scores, per-pair norm preservation, and decode with rotation equal to the dense
masked softmax over pre-rotated queries and keys.  Planted mistakes in a copy of the rotation
routine are rejected.
"""
import ctypes
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from tests.brute import coverage_mask, coverage_mask_window

SRC = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle", "pbb_oracle.c")
BASE = 1e6


def test_hand_computed_values():
    """d = 4, position 1: channel 0 pairs with channel 2 at angle 1, channel 1 with channel 3 at
    angle 1e6^(-1/2) = 1e-3."""
    np.testing.assert_allclose(oracle.rope([1.0, 0, 0, 0], 1, BASE),
                               [math.cos(1.0), 0, math.sin(1.0), 0], atol=1e-15)
    np.testing.assert_allclose(oracle.rope([0, 1.0, 0, 0], 1, BASE),
                               [0, math.cos(1e-3), 0, math.sin(1e-3)], atol=1e-15)
    np.testing.assert_allclose(oracle.rope([0, 0, 1.0, 0], 1, BASE),
                               [-math.sin(1.0), 0, math.cos(1.0), 0], atol=1e-15)
    # position 7, base 10000, d = 8: channel 3 turns by 7 * 10000^(-6/8) = 7e-3
    x = np.zeros(8)
    x[3] = 1.0
    np.testing.assert_allclose(oracle.rope(x, 7, 1e4)[[3, 7]], [math.cos(7e-3), math.sin(7e-3)],
                               atol=1e-15)


def test_identity_composition_and_norms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(64)
    np.testing.assert_allclose(oracle.rope(x, 0, BASE), x, atol=1e-15)
    a, b = 12345, 987654
    np.testing.assert_allclose(oracle.rope(oracle.rope(x, a, BASE), b, BASE),
                               oracle.rope(x, a + b, BASE), atol=1e-9)
    y = oracle.rope(x, 424242, BASE)
    np.testing.assert_allclose(y[:32] ** 2 + y[32:] ** 2, x[:32] ** 2 + x[32:] ** 2, atol=1e-12)


@pytest.mark.parametrize("t,s", [(5, 3), (1 << 20, (1 << 20) - 77), (300000, 299000)])
def test_scores_depend_on_distance_only(t, s):
    rng = np.random.default_rng(t)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    lhs = oracle.rope(q, t, BASE) @ oracle.rope(k, s, BASE)
    rhs = oracle.rope(q, t - s, BASE) @ k
    assert abs(lhs - rhs) < 1e-9 * (1 + abs(rhs))


@pytest.mark.parametrize("t0", [0, 100000, 100003])
def test_rope_decode_matches_dense_mask_on_rotated_inputs(t0):
    """Queries at t0 .. t0+n-1 over history from max(0, t0 - b): decode with rotation equals the
    dense masked softmax of rotated queries and keys (mask from the coverage form)."""
    rng = np.random.default_rng(3 + t0)
    n, b, hq, hkv, d = 80, 16, 4, 2, 8
    lo = max(0, t0 - b)
    L = t0 + n - lo
    q = rng.standard_normal((n, hq, d)).astype(np.float32)
    k = rng.standard_normal((L, hkv, d)).astype(np.float32)
    v = rng.standard_normal((L, hkv, d)).astype(np.float32)
    pos = t0 + np.arange(n, dtype=np.int64)
    kh = np.ascontiguousarray(np.broadcast_to(np.transpose(k, (1, 0, 2))[None], (n, hkv, L, d)))
    vh = np.ascontiguousarray(np.broadcast_to(np.transpose(v, (1, 0, 2))[None], (n, hkv, L, d)))
    out = oracle.decode(oracle.PBB, pos, q, kh, vh, np.full(n, lo), block=b, rope_base=BASE)
    qr = np.stack([oracle.rope(q[i], t0 + i, BASE) for i in range(n)])
    kr = np.stack([oracle.rope(k[r], lo + r, BASE) for r in range(L)])
    mask = coverage_mask_window(t0, n, lo, L, b)
    g = hq // hkv
    for i in range(hq):
        z = (qr[:, i] @ kr[:, i // g].T) / np.sqrt(d)
        z = np.where(mask, z, -np.inf)
        w = np.exp(z - z.max(axis=1, keepdims=True))
        ref = (w / w.sum(axis=1, keepdims=True)) @ v[:, i // g].astype(np.float64)
        np.testing.assert_allclose(out[:, i], ref, atol=1e-12)


ROPE_MUTATIONS = {
    "sign_flipped": ("out[c] = a * cs - b * sn;", "out[c] = a * cs + b * sn;"),
    "interleaved_pairs": ("const double a = x[c], b = x[c + half];",
                          "const double a = x[(2 * c) % d], b = x[(2 * c + 1) % d];"),
    "exponent_off": ("pow(base, -2.0 * (double)c / (double)d)", "pow(base, -1.0 * (double)c / (double)d)"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(ROPE_MUTATIONS))
def test_planted_rope_mistakes_are_caught(tmp_path, name):
    old, new = ROPE_MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", str(path), "-o", str(so),
                           "-lm", "-lpthread"])
    lib = ctypes.CDLL(str(so))
    lib.oracle_rope.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p,
                                ctypes.c_void_p]

    def rope(x, pos, base):
        x = np.ascontiguousarray(x, dtype=np.float64)
        out = np.empty_like(x)
        lib.oracle_rope(x.shape[0], pos, base, x.ctypes.data_as(ctypes.c_void_p),
                        out.ctypes.data_as(ctypes.c_void_p))
        return out

    ok = np.allclose(rope([1.0, 0, 0, 0], 1, BASE), [math.cos(1.0), 0, math.sin(1.0), 0], atol=1e-15)
    ok &= np.allclose(rope([0, 0, 1.0, 0], 1, BASE), [-math.sin(1.0), 0, math.cos(1.0), 0], atol=1e-15)
    ok &= np.allclose(rope([0, 1.0, 0, 0], 1, BASE), [0, math.cos(1e-3), 0, math.sin(1e-3)], atol=1e-15)
    assert not ok, f"mutation {name} was not detected"
