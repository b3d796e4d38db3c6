"""Bench sanity on the CPU: the algorithmic byte model of bench.py against the support sizes
of the brute-force coverage mask and the closed forms (mean support 1.5h + 0.5 over a block
period, Appendix F.1 Eq.(pbb_cache_support)), the committed HBM counter summary against the
model, and the one-GPU guard of the command line."""
from __future__ import annotations

import os
import re

import numpy as np
import pytest
import torch

import bench
import workloads as W
from tests.brute import coverage_mask, window_mask

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("block", [2, 8, 64, 128])
def test_support_size_matches_coverage_mask(block):
    n = 6 * block
    cfg = W.get_config("c3").with_(block=block, slots=block)
    got = bench.support_size(torch.arange(n, dtype=torch.int64), cfg).numpy()
    np.testing.assert_array_equal(got, coverage_mask(n, block).sum(axis=1))


@pytest.mark.parametrize("window", [1, 7, 128])
def test_swa_support_size_matches_window_mask(window):
    n = 5 * window + 3
    cfg = W.get_config("c5").with_(window=window, slots=window)
    got = bench.support_size(torch.arange(n, dtype=torch.int64), cfg).numpy()
    np.testing.assert_array_equal(got, window_mask(n, window).sum(axis=1))


def test_step_bytes_closed_form_c3_and_c4():
    # over one full block period past the first block the mean support is 1.5h + 0.5
    c3 = W.get_config("c3")
    t = torch.arange(2 * c3.block, 3 * c3.block, dtype=torch.int64)
    per_tok = bench.step_bytes(t, c3) / len(t)
    h = c3.block // 2
    mean_ring = 1.5 * h + 0.5 - 1
    exp = mean_ring * 2 * c3.hkv * c3.d * 2 + 2 * c3.hq * c3.d * 2 + 4 * c3.hkv * c3.d * 2 + 4
    assert per_tok == pytest.approx(exp, rel=0, abs=1e-6)
    assert round(per_tok) == 6_313_988
    c4 = W.get_config("c4")
    t = torch.arange(2 * c4.block, 3 * c4.block, dtype=torch.int64)
    assert bench.step_bytes(t, c4) / len(t) == pytest.approx(
        (0.75 * c4.block + 0.5 - 1) * 2 * c4.hkv * c4.d * 2 + 2 * c4.hq * c4.d * 2
        + 4 * c4.hkv * c4.d * 2 + 4)


@pytest.mark.parametrize("workload", ["c3", "c4", "c5"])
def test_committed_counters_match_the_byte_model(workload):
    """The committed FETCH_SIZE / WRITE_SIZE summaries of the decode (scaled by the copy
    calibration) agree with the byte model within 5 %, re-derived here from their own counter
    values; the bench uses them only while the kernel sources are the profiled ones."""
    path = os.path.join(ROOT, "profiles", f"decode_bf16_{workload}_counters.txt")
    txt = open(path).read()
    num = lambda key: float(re.search(key + r": ([\d.]+)", txt).group(1))
    ratio = num("traffic / algorithmic")
    assert 0.99 <= ratio <= 1.05, ratio
    scaled = (num("decode FETCH_SIZE_KiB") * 1024 * 1048576 / num("copy FETCH_SIZE_KiB")
              + num("decode WRITE_SIZE_KiB") * 1024 * 1048576 / num("copy WRITE_SIZE_KiB"))
    assert scaled == pytest.approx(num("hbm_bytes_per_launch_scaled"), rel=1e-6)
    assert scaled / num("algorithmic_bytes_per_launch") == pytest.approx(ratio, abs=1e-4)
    assert re.fullmatch(r"[0-9a-f]{16}", re.search(r"kernel_source_hash: (\S+)", txt).group(1))
    # the bench reports the committed figure while the kernel sources are the profiled ones,
    # and null (unmeasured) once they have changed
    got = bench._traffic_ratio_from_profile(workload)
    if re.search(r"kernel_source_hash: (\S+)", txt).group(1) == bench._kernel_hash():
        assert got == pytest.approx(ratio, abs=1e-4)
    else:
        assert got is None


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err
