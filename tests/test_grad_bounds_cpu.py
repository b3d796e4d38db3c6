"""CPU check of the backward's derived error bound (tests/grad_bounds.py).

An fp64 numpy emulation of the kernels' arithmetic -- the forward output rounded to bf16, dP and
delta as fp32 dot products summed in different orders (so that a target whose exact gradient
vanishes, e.g. position 0, gets a rounding-level nonzero one), the softmax weights P rounded to
bf16 before dv = P^T dout, dS = P (dP - delta) rounded to bf16
before dq = scale dS K and dk = scale dS^T Q, gradients rounded to bf16 -- must stay inside
2 (bound + U |exact|); a planted mistake (delta from a 1 % perturbed output, or P without
rounding but scaled by 1 + 2^-6) must leave it, so the bound is tight enough to notice such
errors.  Exact gradients come from the fp64 oracle.
"""
import numpy as np
import pytest

import oracle
from tests.brute import coverage_mask, window_mask
from tests.grad_bounds import U_BF16, grad_bounds
from tests.harness import bf16_round


def _emulate(mode, q, k, v, dout, block, window, out_err=0.0, p_scale=None):
    batch, n, hq, d = q.shape
    hkv = k.shape[2]
    G = hq // hkv
    scale = 1.0 / np.sqrt(d)
    mask = coverage_mask(n, block) if mode == "pbb" else window_mask(n, window)
    dq, dk, dv = np.zeros(q.shape), np.zeros(k.shape), np.zeros(v.shape)
    out = np.zeros(q.shape)
    lse_all = np.zeros((batch, hq, n))
    for b in range(batch):
        for i in range(hq):
            g = i // G
            Q, K, V, dO = q[b, :, i], k[b, :, g], v[b, :, g], dout[b, :, i]
            Z = np.where(mask, scale * (Q @ K.T), -np.inf)
            zmax = Z.max(axis=1, keepdims=True)
            lse = zmax[:, 0] + np.log(np.exp(Z - zmax).sum(axis=1))
            P = np.exp(Z - lse[:, None])
            O = bf16_round(P @ V) * (1.0 + out_err)       # the forward's bf16 output
            out[b, :, i] = O
            lse_all[b, i] = lse
            # dP and delta as fp32 dot products summed in different orders (the kernels take
            # them on the matrix cores and in a vector loop respectively)
            f32 = np.float32
            dP = (dO.astype(f32) @ V.T.astype(f32)).astype(np.float64)
            delta = np.zeros(n, dtype=f32)
            for c in range(d - 1, -1, -1):
                delta = (delta + (dO[:, c] * O[:, c]).astype(f32)).astype(f32)
            delta = delta.astype(np.float64)
            Pr = bf16_round(P) if p_scale is None else P * p_scale
            dv[b, :, g] += Pr.T @ dO
            dS = bf16_round(P * (dP - delta[:, None]))
            dq[b, :, i] = scale * (dS @ K)
            dk[b, :, g] += scale * (dS.T @ Q)
    return (bf16_round(dq), bf16_round(dk), bf16_round(dv)), out, lse_all


def _inputs(mode, n, hq, hkv, d, seed):
    rng = np.random.default_rng(seed)
    r = lambda *s: bf16_round(rng.standard_normal(s))
    q, k, v, dout = r(1, n, hq, d), r(1, n, hkv, d), r(1, n, hkv, d), r(1, n, hq, d)
    # a few large keys so that some targets put almost all their weight on one key (the
    # gradients of those rows nearly cancel)
    k[0, rng.integers(0, n, 6)] *= 4.0
    return q, k, v, dout


def _within(got, exact, bounds):
    return all((np.abs(g - e) <= 2.0 * (bd + U_BF16 * np.abs(e))).all()
               for g, e, bd in zip(got, exact, bounds))


@pytest.mark.parametrize("mode,n,hq,hkv,d,block,window", [
    ("pbb", 200, 4, 2, 32, 32, 0), ("pbb", 150, 6, 1, 64, 64, 0), ("swa", 180, 4, 2, 32, 0, 40)])
def test_emulated_kernel_arithmetic_stays_inside_the_bound(mode, n, hq, hkv, d, block, window):
    q, k, v, dout = _inputs(mode, n, hq, hkv, d, seed=n)
    om = oracle.PBB if mode == "pbb" else oracle.SWA
    exact = oracle.backward(om, q, k, v, dout, block=block, window=window)
    got, out, lse = _emulate(mode, q, k, v, dout, block, window)
    bounds = grad_bounds(mode, q, k, v, dout, out, lse.astype(np.float32), block=block,
                         window=window)
    assert _within(got, exact, bounds)


@pytest.mark.parametrize("kind", ["output_off_by_1pct", "weights_scaled"])
def test_planted_mistakes_leave_the_bound(kind):
    mode, n, hq, hkv, d, block = "pbb", 200, 4, 2, 32, 32
    q, k, v, dout = _inputs(mode, n, hq, hkv, d, seed=7)
    exact = oracle.backward(oracle.PBB, q, k, v, dout, block=block)
    _, out_ok, lse = _emulate(mode, q, k, v, dout, block, 0)
    if kind == "output_off_by_1pct":
        # delta from an output 1 % off, while the bound is given the correct output
        got, _, _ = _emulate(mode, q, k, v, dout, block, 0, out_err=0.01)
    else:
        got, _, _ = _emulate(mode, q, k, v, dout, block, 0, p_scale=1.0 + 2.0 ** -6)
    bounds = grad_bounds(mode, q, k, v, dout, out_ok, lse.astype(np.float32), block=block)
    assert not _within(got, exact, bounds)
