"""Pins for the oracle's prefill (every prompt position over its own support; CPU only).

Pinned by: the dense masked softmax of ``tests/brute.py`` (mask from the direct-coverage
form, Sec. 3 "Coverage and arithmetic"), for outputs and log-partitions; the paper's printed
score count at n = 8192 (Appendix A.5), recovered from the log-partitions of zero queries
(``lse = log |A(t)|``); the interval form of the support through position-coded values
(mean position ``(a(t) + t) / 2``, Sec. 3 "Flash-PBB"); reductions to full causal attention
(``B >= n``, ``W >= n``); the first position (``o_0 = v_0``); and the disjoint-support LSE
identity (Appendix A.4, Eq.(lse)).  Planted mistakes in a copy of the prefill routine are
rejected by these pins.
"""
import ctypes
import json
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from tests.brute import coverage_mask, interval_start, masked_attention, window_mask

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "score_counts.json")
SRC = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle", "pbb_oracle.c")


def _rand(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


def _dense(q, k, v, mask, scale):
    """Dense reference for one head: (out [n][d], lse [n]) in fp64."""
    z = (q.astype(np.float64) @ k.astype(np.float64).T) * scale
    z = np.where(mask, z, -np.inf)
    m = z.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    return masked_attention(q, k, v, mask, scale), lse


@pytest.mark.parametrize("mode,batch,n,b,w,hq,hkv,d", [
    ("pbb", 2, 200, 16, 0, 8, 2, 16),
    ("pbb", 1, 97, 8, 0, 6, 3, 8),
    ("pbb", 1, 40, 2, 0, 2, 1, 4),
    ("pbb", 1, 300, 64, 0, 4, 4, 32),
    ("swa", 2, 150, 0, 37, 4, 2, 16),
    ("swa", 1, 64, 0, 1, 2, 1, 8),
])
def test_prefill_matches_dense_mask(mode, batch, n, b, w, hq, hkv, d):
    rng = np.random.default_rng(n + b + w)
    q, k, v = _rand(rng, batch, n, hq, d), _rand(rng, batch, n, hkv, d), _rand(rng, batch, n, hkv, d)
    m = oracle.PBB if mode == "pbb" else oracle.SWA
    out, lse = oracle.prefill(m, q, k, v, block=b, window=w)
    mask = coverage_mask(n, b) if mode == "pbb" else window_mask(n, w)
    g = hq // hkv
    for bb in range(batch):
        for i in range(hq):
            ref, ref_lse = _dense(q[bb, :, i], k[bb, :, i // g], v[bb, :, i // g], mask,
                                  1 / np.sqrt(d))
            np.testing.assert_allclose(out[bb, :, i], ref, rtol=0, atol=1e-12)
            np.testing.assert_allclose(lse[bb, i], ref_lse, rtol=0, atol=1e-12)


def test_printed_score_count_from_log_partitions():
    """With q = 0 every score is 0, so exp(lse) = |A(t)|; summed over n = 8192 positions at
    B = 128 this is the paper's printed PBB count (Appendix A.5)."""
    g = json.load(open(GOLDEN))
    n, b = g["n"], g["block"]
    q = np.zeros((1, n, 1, 4), np.float32)
    k = np.ones((1, n, 1, 4), np.float32)
    _, lse = oracle.prefill(oracle.PBB, q, k, k, block=b)
    sizes = np.exp(lse[0, 0])
    assert np.allclose(sizes, np.round(sizes), atol=1e-9)
    assert int(np.round(sizes).sum()) == g["scores_per_head_per_local_layer"]["PBB-128/64"]
    _, lse_w = oracle.prefill(oracle.SWA, q, k, k, window=g["window"])
    assert int(np.round(np.exp(lse_w[0, 0])).sum()) == g["scores_per_head_per_local_layer"]["SWA-128"]


@pytest.mark.parametrize("b", [2, 8, 64])
def test_position_coded_values_give_interval_midpoints(b):
    """q = 0 and v_s = s: o_t is the mean position of the support, (a(t) + t) / 2 with the
    interval start a(t) = max(0, h (floor(t/h) - 1)) (Sec. 3 "Flash-PBB")."""
    n = 5 * b + 3
    q = np.zeros((1, n, 2, 2), np.float32)
    k = _rand(np.random.default_rng(1), 1, n, 1, 2)
    v = np.repeat(np.arange(n, dtype=np.float32).reshape(1, n, 1, 1), 2, axis=3)
    out, _ = oracle.prefill(oracle.PBB, q, k, v, block=b)
    want = np.array([(interval_start(t, b) + t) / 2 for t in range(n)])
    for i in range(2):
        np.testing.assert_allclose(out[0, :, i, 0], want, rtol=0, atol=1e-9)


def test_reductions_to_full_causal():
    rng = np.random.default_rng(4)
    n, d = 50, 8
    q, k, v = _rand(rng, 1, n, 2, d), _rand(rng, 1, n, 1, d), _rand(rng, 1, n, 1, d)
    causal = np.tril(np.ones((n, n), bool))
    for mode, kw in ((oracle.PBB, dict(block=64)), (oracle.PBB, dict(block=200)),
                     (oracle.SWA, dict(window=n))):
        out, lse = oracle.prefill(mode, q, k, v, **kw)
        for i in range(2):
            ref, ref_lse = _dense(q[0, :, i], k[0, :, 0], v[0, :, 0], causal, 1 / np.sqrt(d))
            np.testing.assert_allclose(out[0, :, i], ref, atol=1e-12)
            np.testing.assert_allclose(lse[0, i], ref_lse, atol=1e-12)


def test_first_position_and_scale():
    rng = np.random.default_rng(6)
    q, k, v = _rand(rng, 1, 3, 1, 4), _rand(rng, 1, 3, 1, 4), _rand(rng, 1, 3, 1, 4)
    out, lse = oracle.prefill(oracle.PBB, q, k, v, block=4, scale=0.3)
    np.testing.assert_allclose(out[0, 0, 0], v[0, 0, 0], atol=1e-15)
    assert abs(lse[0, 0, 0] - 0.3 * float(q[0, 0, 0].astype(np.float64) @ k[0, 0, 0])) < 1e-12


def test_lse_identity_over_block_prefix_and_bridge():
    """Eq.(lse): the log-partition of A(t) is the log-sum-exp of its disjoint parts, the block
    prefix {p..t} and the bridge {p-h..p-1}, each from a single-head attention."""
    rng = np.random.default_rng(8)
    n, b, d = 70, 16, 8
    q, k, v = _rand(rng, 1, n, 1, d), _rand(rng, 1, n, 1, d), _rand(rng, 1, n, 1, d)
    out, lse = oracle.prefill(oracle.PBB, q, k, v, block=b)
    h = b // 2
    for t in range(b, n):
        p, r = b * (t // b), t % b
        if r >= h:
            continue
        o1, l1 = oracle.attend(q[0, t, 0], k[0, p:t + 1, 0], v[0, p:t + 1, 0])
        o2, l2 = oracle.attend(q[0, t, 0], k[0, p - h:p, 0], v[0, p - h:p, 0])
        mx = max(l1, l2)
        want = mx + np.log(np.exp(l1 - mx) + np.exp(l2 - mx))
        assert abs(lse[0, 0, t] - want) < 1e-12
        wt1, wt2 = np.exp(l1 - lse[0, 0, t]), np.exp(l2 - lse[0, 0, t])
        np.testing.assert_allclose(out[0, t, 0], wt1 * o1 + wt2 * o2, atol=1e-12)


def test_prefill_agrees_with_decode_oracle():
    rng = np.random.default_rng(10)
    n, b, hq, hkv, d = 90, 16, 4, 2, 8
    q, k, v = _rand(rng, 1, n, hq, d), _rand(rng, 1, n, hkv, d), _rand(rng, 1, n, hkv, d)
    out, _ = oracle.prefill(oracle.PBB, q, k, v, block=b)
    kh = np.ascontiguousarray(np.broadcast_to(np.transpose(k[0], (1, 0, 2))[None], (n, hkv, n, d)))
    vh = np.ascontiguousarray(np.broadcast_to(np.transpose(v[0], (1, 0, 2))[None], (n, hkv, n, d)))
    dec = oracle.decode(oracle.PBB, np.arange(n), q[0], kh, vh, np.zeros(n, np.int64), block=b)
    np.testing.assert_allclose(out[0], dec, atol=1e-13)


PREFILL_MUTATIONS = {
    "scale_dropped": ("        z[s - lo] = acc * j->scale;\n        if (z[s - lo] > m) m = z[s - lo];\n    }\n    double den = 0.0;\n    for (int64_t s = lo; s <= t; ++s) {\n        if (!prefill_member",
                      "        z[s - lo] = acc;\n        if (z[s - lo] > m) m = z[s - lo];\n    }\n    double den = 0.0;\n    for (int64_t s = lo; s <= t; ++s) {\n        if (!prefill_member"),
    "lse_without_max": ("j->lse[(b * hq + i) * n + t] = m + log(den);",
                        "j->lse[(b * hq + i) * n + t] = log(den);"),
    "gqa_strided": ("    const int64_t g = i / G; /* query head i reads KV head floor(i/G) */\n    double *o = j->out + ((b * n + t)",
                    "    const int64_t g = i % hkv;\n    double *o = j->out + ((b * n + t)"),
    "bridge_dropped": ("if (j->mode == 0) return oracle_pbb_member(t, s, j->block, j->block / 2);\n    return oracle_swa_member(t, s, j->window);\n}\n\n/* One (sequence, position",
                       "if (j->mode == 0) return oracle_pbb_member(t, s, j->block, 0);\n    return oracle_swa_member(t, s, j->window);\n}\n\n/* One (sequence, position"),
    "value_row_off_by_one": ("const float *vs = j->v + ((b * n + s) * hkv + g) * d;\n        double w = exp",
                             "const float *vs = j->v + ((b * n + (s > 0 ? s - 1 : s)) * hkv + g) * d;\n        double w = exp"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(PREFILL_MUTATIONS))
def test_planted_prefill_mistakes_are_caught(tmp_path, name):
    old, new = PREFILL_MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", str(path), "-o", str(so),
                           "-lm", "-lpthread"])
    lib = ctypes.CDLL(str(so))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_prefill.argtypes = [ctypes.c_int, i64, i64, i64, i64, i64, i64, i64, vp, vp, vp,
                                   ctypes.c_double, vp, vp, ctypes.c_int]
    lib.oracle_prefill.restype = ctypes.c_int
    rng = np.random.default_rng(2)
    n, b, hq, hkv, d = 80, 16, 4, 2, 8
    q, k, v = _rand(rng, 1, n, hq, d), _rand(rng, 1, n, hkv, d), _rand(rng, 1, n, hkv, d)
    out = np.zeros((1, n, hq, d))
    lse = np.zeros((1, hq, n))
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    assert lib.oracle_prefill(0, 1, n, hq, hkv, d, b, 0, p(q), p(k), p(v), 1 / np.sqrt(d), p(out),
                              p(lse), 2) == 0
    mask = coverage_mask(n, b)
    ok = True
    for i in range(hq):
        ref, ref_lse = _dense(q[0, :, i], k[0, :, i // 2], v[0, :, i // 2], mask, 1 / np.sqrt(d))
        ok &= np.allclose(out[0, :, i], ref, atol=1e-12) and np.allclose(lse[0, i], ref_lse, atol=1e-12)
    assert not ok, f"mutation {name} was not detected"
