"""Detection power of the oracle's pins (CPU only).

Each case plants one plausible mistake in a temporary copy of the oracle's C source
(a wrong bound, a dropped term, a flipped sign, a swapped operand), builds it, and checks
that the printed score counts or the dense-mask comparison reject it.  The real oracle is
never modified.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

from tests.brute import coverage_mask, masked_attention

SRC = os.path.join(os.path.dirname(os.path.dirname(__file__)), "oracle", "pbb_oracle.c")

MUTATIONS = {
    "bridge_phase_off_by_one": ("r < bridge && s >= p - bridge", "r <= bridge && s >= p - bridge"),
    "bridge_start_off_by_one": ("s >= p - bridge && s <= p - 1", "s > p - bridge && s <= p - 1"),
    "block_start_dropped": ("if (s >= p) return 1;", "if (s > p) return 1;"),
    "bridge_wrong_half": ("s >= p - bridge && s <= p - 1", "s >= p - 2 * bridge && s <= p - bridge - 1"),
    "scale_dropped": ("(double)kh[row * d + c];\n        }\n        z[s - lo] = acc * j->scale;",
                      "(double)kh[row * d + c];\n        }\n        z[s - lo] = acc;"),
    "exp_sign_flipped": ("int64_t row = s - j->hist_lo[b];\n        double w = exp(z[s - lo] - m);",
                         "int64_t row = s - j->hist_lo[b];\n        double w = exp(m - z[s - lo]);"),
    "gqa_strided": ("const int64_t g = i / G; /* query head i reads KV head floor(i/G) */\n    const int64_t t = j->pos[b];",
                    "const int64_t g = i % j->n_kv_heads;\n    const int64_t t = j->pos[b];"),
    "value_operand_swapped": ("o[c] += w * (double)vh[row * d + c];",
                              "o[c] += w * (double)kh[row * d + c];"),
    "normalisation_dropped": ("(void)cnt;\n    for (int64_t c = 0; c < d; ++c) o[c] /= den;",
                              "(void)cnt;"),
}


def _build(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / f"{name}.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", str(path), "-o",
                           str(so), "-lm", "-lpthread"])
    lib = ctypes.CDLL(str(so))
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_pbb_counts.argtypes = [i64, i64, i64, vp, vp]
    lib.oracle_decode.argtypes = [ctypes.c_int, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp,
                                  vp, i64, ctypes.c_double, vp, ctypes.c_int]
    lib.oracle_decode.restype = ctypes.c_int
    return lib


def _pins_pass(lib) -> bool:
    tot, cr = ctypes.c_int64(), ctypes.c_int64()
    lib.oracle_pbb_counts(8192, 128, 64, ctypes.byref(tot), ctypes.byref(cr))
    if (tot.value, cr.value) != (786432, 258048):
        return False
    rng = np.random.default_rng(3)
    n, b, hq, hkv, d = 96, 16, 4, 2, 8
    q = rng.standard_normal((n, hq, d)).astype(np.float32)
    k = rng.standard_normal((n, hkv, d)).astype(np.float32)
    v = rng.standard_normal((n, hkv, d)).astype(np.float32)
    pos = np.arange(n, dtype=np.int64)
    kh = np.ascontiguousarray(np.broadcast_to(np.transpose(k, (1, 0, 2))[None], (n, hkv, n, d)))
    vh = np.ascontiguousarray(np.broadcast_to(np.transpose(v, (1, 0, 2))[None], (n, hkv, n, d)))
    lo = np.zeros(n, dtype=np.int64)
    out = np.zeros((n, hq, d))
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    rc = lib.oracle_decode(0, n, hq, hkv, d, b, 0, p(pos), p(q), p(kh), p(vh), p(lo), n,
                           1 / np.sqrt(d), p(out), 2)
    if rc != 0:
        return False
    mask = coverage_mask(n, b)
    for i in range(hq):
        ref = masked_attention(q[:, i], k[:, i // 2], v[:, i // 2], mask, 1 / np.sqrt(d))
        if not np.allclose(out[:, i], ref, rtol=0, atol=1e-12):
            return False
    return True


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_unmutated_copy_passes(tmp_path):
    assert _pins_pass(_build(tmp_path, "identity", "#include <math.h>", "#include <math.h>"))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    assert not _pins_pass(_build(tmp_path, name, old, new))
