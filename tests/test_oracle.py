"""Pins for the oracle's attention output (CPU only).

The paper prints no attention values, so the softmax output is pinned by: a dense masked
softmax whose mask comes from the direct-coverage form; reductions to full-causal and
block-causal attention; closed forms; the disjoint-support LSE identity (Appendix A.4,
Eq.(lse)); the omitted-mass identity (Appendix B.3, Eq.(omitted_mass)); a negative control
against the legacy separately normalised branches (Appendix G.1); and key-order invariance.
"""
import numpy as np
import pytest

import oracle
from tests.brute import (block_causal_mask, coverage_mask, interval_start, masked_attention,
                         window_mask)


def _rand(rng, *shape):
    return rng.standard_normal(shape).astype(np.float32)


def _decode_all(mode, q, k, v, *, block=0, window=0, scale=None):
    """Decode every position t < n of one sequence: q [n][Hq][d], k/v [n][Hkv][d]."""
    n, hq, d = q.shape
    hkv = k.shape[1]
    pos = np.arange(n, dtype=np.int64)
    kh = np.broadcast_to(np.transpose(k, (1, 0, 2))[None], (n, hkv, n, d))
    vh = np.broadcast_to(np.transpose(v, (1, 0, 2))[None], (n, hkv, n, d))
    lo = np.zeros(n, dtype=np.int64)
    return oracle.decode(mode, pos, q, kh, vh, lo, block=block, window=window, scale=scale)


@pytest.mark.parametrize("n,b,hq,hkv,d", [(256, 64, 4, 1, 64), (200, 16, 8, 2, 16),
                                          (96, 8, 6, 3, 8), (130, 32, 4, 4, 32)])
def test_decode_matches_dense_mask(n, b, hq, hkv, d):
    rng = np.random.default_rng(n + b)
    q, k, v = _rand(rng, n, hq, d), _rand(rng, n, hkv, d), _rand(rng, n, hkv, d)
    out = _decode_all(oracle.PBB, q, k, v, block=b)
    mask = coverage_mask(n, b)
    g = hq // hkv
    for i in range(hq):
        ref = masked_attention(q[:, i], k[:, i // g], v[:, i // g], mask, 1 / np.sqrt(d))
        np.testing.assert_allclose(out[:, i], ref, rtol=0, atol=1e-12)


def test_gqa_mapping_is_contiguous():
    """Query head i reads KV head floor(i/G): a strided mapping would differ."""
    rng = np.random.default_rng(5)
    n, b, hq, hkv, d = 64, 16, 4, 2, 8
    q, k, v = _rand(rng, n, hq, d), _rand(rng, n, hkv, d), _rand(rng, n, hkv, d)
    out = _decode_all(oracle.PBB, q, k, v, block=b)
    mask = coverage_mask(n, b)
    strided = masked_attention(q[:, 1], k[:, 1], v[:, 1], mask, 1 / np.sqrt(d))
    contiguous = masked_attention(q[:, 1], k[:, 0], v[:, 0], mask, 1 / np.sqrt(d))
    np.testing.assert_allclose(out[:, 1], contiguous, atol=1e-12)
    assert np.abs(out[:, 1] - strided).max() > 0.1


def test_swa_matches_dense_mask():
    rng = np.random.default_rng(9)
    n, w, d = 300, 37, 16
    q, k, v = _rand(rng, n, 2, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    out = _decode_all(oracle.SWA, q, k, v, window=w)
    for i in range(2):
        ref = masked_attention(q[:, i], k[:, 0], v[:, 0], window_mask(n, w), 1 / np.sqrt(d))
        np.testing.assert_allclose(out[:, i], ref, atol=1e-12)


def test_large_block_is_full_causal():
    """B >= n: the first block covers the sequence, so PBB is full causal attention."""
    rng = np.random.default_rng(11)
    n, d = 100, 16
    q, k, v = _rand(rng, n, 1, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    out = _decode_all(oracle.PBB, q, k, v, block=128)
    causal = np.tril(np.ones((n, n), dtype=bool))
    ref = masked_attention(q[:, 0], k[:, 0], v[:, 0], causal, 1 / np.sqrt(d))
    np.testing.assert_allclose(out[:, 0], ref, atol=1e-12)


def test_second_half_phases_are_block_causal():
    """r >= h: no bridge, so PBB equals block-causal attention for those targets."""
    rng = np.random.default_rng(12)
    n, b, d = 256, 32, 16
    q, k, v = _rand(rng, n, 1, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    out = _decode_all(oracle.PBB, q, k, v, block=b)
    ref = masked_attention(q[:, 0], k[:, 0], v[:, 0], block_causal_mask(n, b), 1 / np.sqrt(d))
    rows = [t for t in range(n) if t % b >= b // 2 or t < b]
    np.testing.assert_allclose(out[rows, 0], ref[rows], atol=1e-12)
    bridged = [t for t in range(b, n) if t % b < b // 2]
    assert np.abs(out[bridged, 0] - ref[bridged]).max() > 1e-3


def test_closed_forms():
    rng = np.random.default_rng(13)
    n, b, d = 200, 16, 8
    q, k, v = _rand(rng, n, 1, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    # t = 0: the support is {0}, so o = v_0.
    out = _decode_all(oracle.PBB, q, k, v, block=b)
    np.testing.assert_allclose(out[0, 0], v[0, 0], atol=1e-15)
    # q = 0: uniform weights, o = mean of V over the support [a(t), t].
    out0 = _decode_all(oracle.PBB, np.zeros_like(q), k, v, block=b)
    for t in range(n):
        a = interval_start(t, b)
        np.testing.assert_allclose(out0[t, 0], v[a:t + 1, 0].astype(np.float64).mean(0),
                                   atol=1e-13)
    # Position-coded V (v_s[0] = s) with q = 0: o[0] = (a(t) + t) / 2 exactly.
    vp = np.zeros_like(v)
    vp[:, 0, 0] = np.arange(n)
    outp = _decode_all(oracle.PBB, np.zeros_like(q), k, vp, block=b)
    for t in range(n):
        assert abs(outp[t, 0, 0] - (interval_start(t, b) + t) / 2) < 1e-10


def test_lse_fusion_identity():
    """Disjoint supports merged by Eq.(lse) equal attention on their union; an empty part
    (Z = 0) returns the other part's output (Appendix A.4)."""
    rng = np.random.default_rng(14)
    d = 32
    for trial in range(20):
        n = int(rng.integers(2, 300))
        q, k, v = rng.standard_normal(d), rng.standard_normal((n, d)), rng.standard_normal((n, d))
        perm = rng.permutation(n)
        cut = int(rng.integers(1, n))
        s1, s2 = perm[:cut], perm[cut:]
        o1, l1 = oracle.attend(q, k[s1], v[s1])
        o2, l2 = oracle.attend(q, k[s2], v[s2])
        m = max(l1, l2)
        fused = (np.exp(l1 - m) * o1 + np.exp(l2 - m) * o2) / (np.exp(l1 - m) + np.exp(l2 - m))
        o, _ = oracle.attend(q, k, v)
        np.testing.assert_allclose(fused, o, atol=1e-13)
    o_empty, l_empty = oracle.attend(q, k[:0], v[:0])
    assert l_empty == -np.inf and not o_empty.any()
    m = max(l1, l_empty)
    fused = (np.exp(l1 - m) * o1 + np.exp(l_empty - m) * o_empty) / (np.exp(l1 - m) + 0.0)
    np.testing.assert_allclose(fused, o1, atol=1e-15)


def test_omitted_mass_identity():
    """SWA(w = b) output = (1 - mu) PBB + mu o_D with D = SWA minus PBB, and
    |o_SWA - o_PBB| <= 2 V mu (Appendix B.3, Eq.(omitted_mass))."""
    rng = np.random.default_rng(15)
    b, d = 32, 16
    n = 5 * b
    q, k, v = _rand(rng, n, 1, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    o_pbb = _decode_all(oracle.PBB, q, k, v, block=b)[:, 0]
    o_swa = _decode_all(oracle.SWA, q, k, v, window=b)[:, 0]
    checked = 0
    for t in range(n):
        A = oracle.swa_support(t, b)
        S = set(oracle.pbb_support(t, b))
        D = [s for s in A if s not in S]
        if not D:
            np.testing.assert_allclose(o_swa[t], o_pbb[t], atol=1e-13)
            continue
        z = (k[A, 0].astype(np.float64) @ q[t, 0].astype(np.float64)) / np.sqrt(d)
        a = np.exp(z - z.max())
        a /= a.sum()
        mu = sum(a[i] for i, s in enumerate(A) if s not in S)
        o_d, _ = oracle.attend(q[t, 0], k[D, 0], v[D, 0])
        np.testing.assert_allclose(o_swa[t], (1 - mu) * o_pbb[t] + mu * o_d, atol=1e-12)
        vmax = np.linalg.norm(v[A, 0].astype(np.float64), axis=1).max()
        assert np.linalg.norm(o_swa[t] - o_pbb[t]) <= 2 * vmax * mu + 1e-12
        checked += 1
    assert checked > n // 4


def test_legacy_two_branch_sum_differs():
    """Negative control: W_O(o1 + o2) with separately normalised block and bridge branches
    (Appendix G.1) is not the single-softmax output."""
    rng = np.random.default_rng(16)
    b, d = 32, 16
    n = 3 * b
    q, k, v = _rand(rng, n, 1, d), _rand(rng, n, 1, d), _rand(rng, n, 1, d)
    out = _decode_all(oracle.PBB, q, k, v, block=b)[:, 0]
    worst = 0.0
    for t in range(b, n):
        p, r = b * (t // b), t % b
        if r >= b // 2:
            continue
        o1, _ = oracle.attend(q[t, 0], k[p:t + 1, 0], v[p:t + 1, 0])
        o2, _ = oracle.attend(q[t, 0], k[p - b // 2:p, 0], v[p - b // 2:p, 0])
        worst = max(worst, np.abs((o1 + o2) - out[t]).max())
    assert worst > 0.1


def test_key_order_invariance():
    rng = np.random.default_rng(17)
    d, n = 64, 500
    q, k, v = rng.standard_normal(d), rng.standard_normal((n, d)), rng.standard_normal((n, d))
    perm = rng.permutation(n)
    o1, l1 = oracle.attend(q, k, v)
    o2, l2 = oracle.attend(q, k[perm], v[perm])
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    assert abs(l1 - l2) < 1e-12


def test_missing_history_raises():
    rng = np.random.default_rng(18)
    q = _rand(rng, 1, 1, 8)
    kh = _rand(rng, 1, 1, 4, 8)
    with pytest.raises(ValueError):
        oracle.decode(oracle.PBB, np.array([10]), q, kh, kh, np.array([0]), block=8)


def test_expected_ring_matches_sequential_writes():
    """The ring-image rule equals a literal simulation that writes each position into slot
    s mod S in order (Appendix F.1 proposition), starting from zeros."""
    rng = np.random.default_rng(19)
    for slots, first, last in [(8, 0, 5), (8, 0, 30), (16, 3, 50), (12, 40, 41), (4, 9, 8)]:
        hist = rng.standard_normal((1, 2, last + 1, 3)).astype(np.float32)
        sim = np.zeros((1, 2, slots, 3), dtype=np.float32)
        for s in range(first, last + 1):
            sim[0, :, s % slots] = hist[0, :, s]
        got = oracle.expected_ring(hist, [0], [last], [first], slots)
        np.testing.assert_array_equal(got, sim)
        # The PBB support of the last position is fully present in the ring (slots = b).
        if slots % 2 == 0 and last >= first and first == 0:
            for s in oracle.pbb_support(last, slots):
                np.testing.assert_array_equal(got[0, :, s % slots], hist[0, :, s])
