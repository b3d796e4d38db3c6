"""Elementwise error bounds of the training backward, derived from where its kernels round.

Used by the GPU parity tests of the backward (``tests/test_backward.py``) and checked on the CPU
against a numpy emulation of those rounding points (``tests/test_grad_bounds_cpu.py``).
"""
from __future__ import annotations

import numpy as np

U_BF16 = 2.0 ** -9      # unit roundoff of bf16 round-to-nearest-even


def grad_bounds(mode, q, k, v, dout, out_gpu, lse_gpu, block=0, window=0, scale=None):
    """Elementwise bounds on |GPU gradient - exact gradient| derived from where the kernels
    round (fp64, dense masks; test-sized inputs only).  With P the exact softmax weights,
    dP = dout . v, delta = dout . out_exact and dS = P (dP - delta):
      * scores, dP and delta are fp32 dot products of d terms (error <= g_d times the sum of
        the absolute products, g_d = d 2^-24);
      * P is built from fp32 scores and the forward's fp32 log-partition -- relative error
        eps = expm1(|lse_gpu - lse| + g_d scale |q|.|k|) -- and enters the dv product rounded
        to bf16 (relative U);
      * delta uses the forward's bf16 output: |delta_gpu - delta| <= sum_c |dout_c|
        |out_gpu_c - out_c| + g_d sum_c |dout_c out_gpu_c|;
      * dS is rounded to bf16 (relative U) before the dq and dk products;
      * dq, dk, dv are fp32 sums of at most n terms (error <= g_n times their absolute sum,
        g_n = n 2^-24).
    Per element |E_P| <= P (U + eps) and |E_dS| <= |dS| (2U + eps) + P (|E_dP| + |E_delta|), so
    dq <= scale (|E_dS| + g_n |dS|) |K|, dk <= scale sum_heads (|E_dS| + g_n |dS|)^T |Q| and
    dv <= sum_heads (|E_P| + g_n P)^T |dout|.  The stored gradient's own rounding and
    second-order terms come on top (the caller adds U |ref| and a factor 2).  Arrays: q, dout,
    out_gpu [b][n][Hq][d]; k, v [b][n][Hkv][d]; lse_gpu [b][Hq][n] (natural log)."""
    from tests.brute import coverage_mask, window_mask
    batch, n, hq, d = q.shape
    hkv = k.shape[2]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    g_d, g_n = d * 2.0 ** -24, n * 2.0 ** -24
    mask = coverage_mask(n, block) if mode == "pbb" else window_mask(n, window)
    bq = np.zeros(q.shape)
    bk = np.zeros(k.shape)
    bv = np.zeros(v.shape)
    for b in range(batch):
        for i in range(hq):
            g = i // G
            Q, K, V = (x.astype(np.float64) for x in (q[b, :, i], k[b, :, g], v[b, :, g]))
            dO, O = dout[b, :, i].astype(np.float64), out_gpu[b, :, i].astype(np.float64)
            aQ, aK, aV, adO = np.abs(Q), np.abs(K), np.abs(V), np.abs(dO)
            Z = np.where(mask, scale * (Q @ K.T), -np.inf)
            zmax = Z.max(axis=1, keepdims=True)
            lse = zmax[:, 0] + np.log(np.exp(Z - zmax).sum(axis=1))
            P = np.exp(Z - lse[:, None])
            Oex = P @ V
            delta = (dO * Oex).sum(axis=1)
            e_delta = (adO * np.abs(O - Oex)).sum(axis=1) + g_d * (adO * np.abs(O)).sum(axis=1)
            dlse = np.minimum(np.abs(lse_gpu[b, i].astype(np.float64) - lse), 30.0)[:, None]
            eps = np.expm1(dlse + g_d * scale * (aQ @ aK.T))
            dS = P * (dO @ V.T - delta[:, None])
            aS = np.abs(dS)
            EdS = aS * (2 * U_BF16 + eps) + P * (g_d * (adO @ aV.T) + e_delta[:, None]) + g_n * aS
            bq[b, :, i] = scale * (EdS @ aK)
            bk[b, :, g] += scale * (EdS.T @ aQ)
            bv[b, :, g] += (P * (U_BF16 + eps + g_n)).T @ adO
    return bq, bk, bv
