"""Pins for the oracle's PBB support (CPU only).

The oracle builds the support from the two-case Eq.(pbb).  These tests compare it with the
paper's printed score counts, its closed forms, and two other forms of the same support that
the paper states (the interval form and the direct-coverage form), all written here.
"""
import json
import os

import numpy as np
import pytest

import oracle
from tests.brute import coverage_mask, interval_start

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "score_counts.json")
BLOCKS = [2, 4, 8, 16, 64, 128, 512]


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_printed_counts_pbb(golden):
    n, b, h = golden["n"], golden["block"], golden["bridge"]
    total, cross = oracle.pbb_counts(n, b, h)
    assert total == golden["scores_per_head_per_local_layer"]["PBB-128/64"]
    assert cross == golden["cross_block_scores"]["PBB-128/64"]
    # Within-block scores are exactly the Block-128 count.
    assert total - cross == golden["scores_per_head_per_local_layer"]["Block-128"]


def test_printed_counts_swa(golden):
    n, w, b = golden["n"], golden["window"], golden["block"]
    total, cross = oracle.swa_counts(n, w, b)
    assert total == golden["scores_per_head_per_local_layer"]["SWA-128"]
    assert cross == golden["cross_block_scores"]["SWA-128"]


def test_printed_reduction(golden):
    n, b, h, w = golden["n"], golden["block"], golden["bridge"], golden["window"]
    pbb, _ = oracle.pbb_counts(n, b, h)
    swa, _ = oracle.swa_counts(n, w, b)
    assert round(100.0 * (1.0 - pbb / swa), 1) == golden["local_score_reduction_percent_vs_SWA"]


@pytest.mark.parametrize("n,b", [(1024, 64), (2048, 128), (4096, 512), (96, 8), (64, 4)])
def test_closed_form_counts(n, b):
    """E_PBB = n(b+1)/2 + (n/b - 1) h^2 and E_SWA = nw - w(w-1)/2 (Appendix A.5)."""
    h = b // 2
    total, cross = oracle.pbb_counts(n, b, h)
    assert total == n * (b + 1) // 2 + (n // b - 1) * h * h
    assert cross == (n // b - 1) * h * h
    w = b
    swa, _ = oracle.swa_counts(n, w, b)
    assert swa == n * w - w * (w - 1) // 2


@pytest.mark.parametrize("b", BLOCKS)
def test_three_forms_agree(b):
    """Two-case Eq.(pbb) == interval [a(t), t] == direct coverage C(d, r), t < 6b."""
    n = 6 * b
    cov = coverage_mask(n, b)
    for t in range(n):
        sup = oracle.pbb_support(t, b)
        a = interval_start(t, b)
        assert sup == list(range(a, t + 1)), (b, t)
        assert sup == list(np.nonzero(cov[t])[0]), (b, t)


@pytest.mark.parametrize("b", BLOCKS)
def test_support_size_closed_form(b):
    """|A(t)| = h + 1 + (t mod h) for t >= h (Appendix F.1, Eq.(pbb_cache_support))."""
    h = b // 2
    for t in range(h, 6 * b):
        assert len(oracle.pbb_support(t, b)) == h + 1 + (t % h) <= b


def test_phase_average(golden):
    b = golden["block"]
    h = b // 2
    sizes = [len(oracle.pbb_support(t, b)) for t in range(4 * b, 5 * b)]
    assert np.mean(sizes) == golden["support_phase_average_h64"] == (3 * h + 1) / 2


@pytest.mark.parametrize("b", BLOCKS)
def test_slot_layout(b):
    """Ring slots of the non-current sources: [h, b) in bridge phases, then [0, r)
    (Appendix F.1, the paragraph after the ring proposition)."""
    h = b // 2
    for t in range(6 * b):
        p, r = b * (t // b), t % b
        slots = sorted(s % b for s in oracle.pbb_support(t, b) if s != t)
        bridge = p > 0 and r < h
        expect = (list(range(h, b)) if bridge else []) + list(range(0, r))
        assert slots == sorted(expect), (b, t)


@pytest.mark.parametrize("b", BLOCKS)
def test_ring_proposition(b):
    """Writing slot t mod b at step t overwrites t - b, which lies before a(t); a(t) never
    decreases; the current sources occupy distinct slots (Appendix F.1, proposition)."""
    prev_a = 0
    for t in range(8 * b):
        sup = oracle.pbb_support(t, b)
        a = sup[0]
        assert a >= prev_a
        prev_a = a
        if t >= b:
            assert t - b < a
        assert len({s % b for s in sup}) == len(sup)


@pytest.mark.parametrize("b", BLOCKS)
def test_pbb_subset_of_swa(b):
    """With w = b = 2h every PBB edge is an SWA edge (Sec. 3; Appendix A.4)."""
    for t in range(6 * b):
        sup = set(oracle.pbb_support(t, b))
        assert sup <= set(oracle.swa_support(t, b))


def test_first_block_is_causal():
    """p = 0 adds no bridge (Eq.(pbb) second case): block 0 is plain causal."""
    for b in BLOCKS:
        for t in range(b):
            assert oracle.pbb_support(t, b) == list(range(0, t + 1))


def test_kv_bytes(golden):
    """Local KV storage 2 * batch * b * H_KV * d_h * u (Appendix F.1)."""
    batch, b, hkv, d, u = 1, 128, 2, 64, 2
    assert 2 * batch * b * hkv * d * u == golden["local_kv_bytes_batch1_b128_hkv2_d64_bf16"]


def test_windowed_coverage_mask_matches_full_mask():
    from tests.brute import coverage_mask_window
    full = coverage_mask(300, 16)
    np.testing.assert_array_equal(coverage_mask_window(100, 50, 60, 90, 16), full[100:150, 60:150])
    np.testing.assert_array_equal(coverage_mask_window(0, 40, 0, 40, 16), full[:40, :40])
