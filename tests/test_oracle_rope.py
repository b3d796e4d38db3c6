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


# ----------------------------------------------------------------------------------------
# oracle_rope_rows: many rows, each at its own position (the rotated ring images and pre-fills
# of the rotary decode tests are built with it).

def _rope_rows_pins_pass(rope_rows) -> bool:
    """The pins of the row-wise rotation, as one predicate so that planted mistakes can be run
    through the same checks.  ``rope_rows(x [n][d] float32, pos [n] int64, base)`` -> fp64."""
    ok = True
    # Closed form, independent of the single-row routine: unit vector e_0 (d = 4) at position
    # p turns by angle p in the (0, 2) plane; e_1 by p * 1e-3 in the (1, 3) plane.
    pos = np.array([0, 1, 2, 5, 1000, 123457], dtype=np.int64)
    e0 = np.zeros((pos.size, 4), dtype=np.float32)
    e0[:, 0] = 1.0
    got = rope_rows(e0, pos, BASE)
    exp = np.stack([np.cos(pos), np.zeros(pos.size), np.sin(pos), np.zeros(pos.size)], axis=1)
    ok &= np.allclose(got, exp, atol=1e-9, rtol=0)
    e1 = np.zeros((pos.size, 4), dtype=np.float32)
    e1[:, 1] = 1.0
    a = pos * 1e-3
    exp = np.stack([np.zeros(pos.size), np.cos(a), np.zeros(pos.size), np.sin(a)], axis=1)
    ok &= np.allclose(rope_rows(e1, pos, BASE), exp, atol=1e-9, rtol=0)
    # Distinct random rows at distinct positions agree with the (separately pinned) single-row
    # rotation, row by row.
    rng = np.random.default_rng(11)
    x = rng.standard_normal((37, 64)).astype(np.float32)
    p = rng.integers(0, 1 << 22, size=37).astype(np.int64)
    got = rope_rows(x, p, BASE)
    exp = np.stack([oracle.rope(x[r].astype(np.float64), int(p[r]), BASE) for r in range(37)])
    ok &= np.allclose(got, exp, atol=1e-12, rtol=0)
    # Relative positions: dot products of rows rotated at t_r and s_r depend on t_r - s_r only.
    q = rng.standard_normal((9, 64)).astype(np.float32)
    k = rng.standard_normal((9, 64)).astype(np.float32)
    t = np.arange(9, dtype=np.int64) * 1000 + 50000
    s = t - (np.arange(9, dtype=np.int64) * 7 + 3)
    lhs = np.einsum("rc,rc->r", rope_rows(q, t, BASE), rope_rows(k, s, BASE))
    rhs = np.einsum("rc,rc->r", rope_rows(q, t - s, BASE), k.astype(np.float64))
    ok &= np.allclose(lhs, rhs, atol=1e-9, rtol=1e-9)
    return bool(ok)


def test_rope_rows_pins():
    assert _rope_rows_pins_pass(lambda x, p, base: oracle.rope_rows(x, p, base))


def test_rope_rows_broadcast_positions():
    """The wrapper's position broadcast ([..., L] positions for [..., L, d] rows) lines up with
    the row order."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 3, 4, 64)).astype(np.float32)
    pos = np.arange(2 * 3 * 4, dtype=np.int64).reshape(2, 3, 4) * 977 + 13
    got = oracle.rope_rows(x, pos, BASE)
    for idx in np.ndindex(2, 3, 4):
        np.testing.assert_allclose(got[idx], oracle.rope(x[idx].astype(np.float64),
                                                         int(pos[idx]), BASE), atol=1e-12)


ROPE_ROWS_MUTATIONS = {
    "every_row_at_first_position": ("rope_apply(d, pos[r], freq, row, out + r * d);",
                                    "rope_apply(d, pos[0], freq, row, out + r * d);"),
    "row_stride_dropped": ("row[c] = (double)x[r * d + c];", "row[c] = (double)x[c];"),
    "output_rows_overlap": ("rope_apply(d, pos[r], freq, row, out + r * d);",
                            "rope_apply(d, pos[r], freq, row, out + r * (d / 2));"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(ROPE_ROWS_MUTATIONS) + ["unmutated"])
def test_planted_rope_rows_mistakes_are_caught(tmp_path, name):
    src = open(SRC).read()
    if name != "unmutated":
        old, new = ROPE_ROWS_MUTATIONS[name]
        assert src.count(old) == 1, name
        src = src.replace(old, new)
    path = tmp_path / f"{name}.c"
    path.write_text(src)
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", str(path), "-o", str(so),
                           "-lm", "-lpthread"])
    lib = ctypes.CDLL(str(so))
    vp = ctypes.c_void_p
    lib.oracle_rope_rows.argtypes = [ctypes.c_int64, ctypes.c_int64, vp, ctypes.c_double, vp, vp]
    lib.oracle_rope_rows.restype = None

    def rope_rows(x, pos, base):
        x = np.ascontiguousarray(x, dtype=np.float32)
        pos = np.ascontiguousarray(pos, dtype=np.int64)
        out = np.zeros(x.shape, dtype=np.float64)
        lib.oracle_rope_rows(x.shape[1], x.shape[0], pos.ctypes.data_as(vp), float(base),
                             x.ctypes.data_as(vp), out.ctypes.data_as(vp))
        return out

    passed = _rope_rows_pins_pass(rope_rows)
    if name == "unmutated":
        assert passed
    else:
        assert not passed, f"mutation {name} was not detected"
