"""Pins for the oracle's backward (gradients of the prefill attention; CPU only).

Pinned by: reverse-mode automatic differentiation (torch, float64) of the dense masked softmax
whose mask comes from the direct-coverage form — an independent implementation of the same
derivative; central finite differences of L = sum(dout * out) computed with the oracle's own
forward (an independent route through the definition of a derivative); and planted mistakes in
a copy of the routine (a dropped softmax-normalisation term, a missing scale, the wrong weights
for dv, strided grouped-query accumulation), each rejected.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest
import torch

import oracle
from tests.brute import coverage_mask, window_mask

SRC = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle", "pbb_oracle.c")


def _inputs(rng, batch, n, hq, hkv, d, grid=True):
    def r(*s):
        x = rng.standard_normal(s)
        if grid:  # multiples of 2^-8: x +- 2^-10 stays exact in float32
            x = np.round(x * 256) / 256
        return x.astype(np.float32)
    return r(batch, n, hq, d), r(batch, n, hkv, d), r(batch, n, hkv, d), r(batch, n, hq, d)


def _autograd(mode, q, k, v, dout, block=0, window=0):
    """float64 autograd of the dense masked softmax (mask from tests/brute.py)."""
    batch, n, hq, d = q.shape
    hkv = k.shape[2]
    g = hq // hkv
    mask = torch.from_numpy(coverage_mask(n, block) if mode == oracle.PBB else window_mask(n, window))
    qt, kt, vt = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    idx = torch.arange(hq) // g
    kk = kt[:, :, idx].permute(0, 2, 1, 3)                     # [b][hq][n][d]
    vv = vt[:, :, idx].permute(0, 2, 1, 3)
    qq = qt.permute(0, 2, 1, 3)
    z = (qq @ kk.transpose(-1, -2)) / np.sqrt(d)
    z = z.masked_fill(~mask, float("-inf"))
    o = torch.softmax(z, dim=-1) @ vv                            # [b][hq][n][d]
    loss = (o.permute(0, 2, 1, 3) * torch.from_numpy(dout.astype(np.float64))).sum()
    loss.backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


@pytest.mark.parametrize("mode,batch,n,hq,hkv,d,block,window", [
    (oracle.PBB, 2, 70, 4, 2, 8, 16, 0),
    (oracle.PBB, 1, 45, 6, 3, 4, 8, 0),
    (oracle.PBB, 1, 33, 2, 1, 16, 2, 0),
    (oracle.SWA, 2, 50, 4, 1, 8, 0, 9),
])
def test_backward_matches_autograd_of_dense_mask(mode, batch, n, hq, hkv, d, block, window):
    rng = np.random.default_rng(n + hq)
    q, k, v, dout = _inputs(rng, batch, n, hq, hkv, d, grid=False)
    got = oracle.backward(mode, q, k, v, dout, block=block, window=window)
    ref = _autograd(mode, q, k, v, dout, block, window)
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-11, err_msg=name)


def test_backward_matches_finite_differences():
    rng = np.random.default_rng(5)
    batch, n, hq, hkv, d, b = 1, 24, 4, 2, 4, 8
    q, k, v, dout = _inputs(rng, batch, n, hq, hkv, d)
    dq, dk, dv = oracle.backward(oracle.PBB, q, k, v, dout, block=b)
    eps = 2.0 ** -10

    def loss(q_, k_, v_):
        out, _ = oracle.prefill(oracle.PBB, q_, k_, v_, block=b)
        return float((out * dout.astype(np.float64)).sum())

    for which, grad in (("q", dq), ("k", dk), ("v", dv)):
        for flat in rng.choice(grad.size, size=12, replace=False):
            idx = np.unravel_index(flat, grad.shape)
            args = {"q": q, "k": k, "v": v}
            plus = {n_: a.copy() for n_, a in args.items()}
            minus = {n_: a.copy() for n_, a in args.items()}
            plus[which][idx] += eps
            minus[which][idx] -= eps
            fd = (loss(plus["q"], plus["k"], plus["v"]) - loss(minus["q"], minus["k"], minus["v"])) / (2 * eps)
            assert abs(fd - grad[idx]) <= 2e-5 * (1 + abs(grad[idx])), (which, idx, fd, grad[idx])


BACKWARD_MUTATIONS = {
    "normalisation_term_dropped": ("const double dz = p * (gv - go);", "const double dz = p * gv;"),
    "dk_scale_dropped": ("dks[c] += j->scale * dz * qd[c];", "dks[c] += dz * qd[c];"),
    "dv_weights_wrong": ("dvs[c] += p * gd[c];", "dvs[c] += dz * gd[c];"),
    "gqa_strided": ("for (int64_t i = g * G; i < (g + 1) * G; ++i) {",
                    "for (int64_t i = g; i < hq; i += hkv) {"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(BACKWARD_MUTATIONS))
def test_planted_backward_mistakes_are_caught(tmp_path, name):
    old, new = BACKWARD_MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", str(path), "-o", str(so),
                           "-lm", "-lpthread"])
    lib = ctypes.CDLL(str(so))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_backward.argtypes = [ctypes.c_int, i64, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp,
                                    ctypes.c_double, vp, vp, vp, ctypes.c_int]
    lib.oracle_backward.restype = ctypes.c_int
    rng = np.random.default_rng(9)
    batch, n, hq, hkv, d, b = 1, 40, 4, 2, 8, 16
    q, k, v, dout = _inputs(rng, batch, n, hq, hkv, d, grid=False)
    dq, dk, dv = (np.zeros(x.shape) for x in (q, k, v))
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    assert lib.oracle_backward(0, batch, n, hq, hkv, d, b, 0, p(q), p(k), p(v), p(dout),
                               1 / np.sqrt(d), p(dq), p(dk), p(dv), 2) == 0
    ref = _autograd(oracle.PBB, q, k, v, dout, b)
    ok = all(np.allclose(a, r, atol=1e-11) for a, r in zip((dq, dk, dv), ref))
    assert not ok, f"mutation {name} was not detected"
