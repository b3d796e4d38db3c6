"""Plain fp64 CPU oracle for Post-Boundary Bridge (PBB) decode attention.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package.  The product path (the HIP library and its Python
binding) never imports, links or calls it, and the oracle imports nothing from the product.

What it follows (paper: "Post-Boundary Bridge: Must Local Attention Go Global Between Global
Layers?"):

* Sec. 2.2, Eq.(1) -- block start ``p(t) = b*floor(t/b)`` and phase ``r(t) = t - p(t)``.
* Sec. 3, Eq.(pbb) -- the PBB support in its two-case form (causal block prefix, plus the
  preceding ``h`` positions when ``p > 0`` and ``r < h``).  Decode uses ``h = b/2``, the width
  for which the paper's ring cache is defined (Sec. 3 "Flash-PBB", Appendix F.1).
* Prop. 2 (Sec. 2.2) -- the sliding-window support ``{max(0, t-w+1) .. t}``.
* Sec. 3, Eq.(attention) -- one softmax over the support with scores ``q.k / sqrt(d_h)``.
* Appendix F.1, Proposition "Relocation-free PBB cache" -- position ``s`` is stored at slot
  ``s mod b``; :func:`expected_ring` gives the ring image that sequential appends produce.
* Appendix C -- rotary positions with base 10^6 (RoPE); half-split channel pairs as in the
  Qwen2.5 decoders the paper trains (:func:`rope`, ``decode(..., rope_base=...)``).
* Sec. 3 (the fused kernel's backward propagation; Appendix F.4, grouped backward checks) --
  :func:`backward`, the gradients of the prefill attention with respect to q, k, v.
* Appendix A.4, Eq.(lse) -- the log-partition ``log sum_s e^{z_s}`` that :func:`prefill` also
  returns for every prompt position (the quantity a tiled prefill rescales with).

The arithmetic lives in ``pbb_oracle.c`` (fp64, plain loops, threads over (sequence, query
head)); this module is argument marshalling plus the ring-image rule.  Inputs are float32
arrays (bf16 inputs widen to float32 exactly) and every sum is formed in fp64.

Parity status: the mask and counts are pinned by the paper's printed score counts and
closed forms; the softmax output has no printed worked example and is pinned by brute force,
closed forms and identities (see ``tests/test_oracle.py``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pbb_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

PBB = 0
SWA = 1


def build(force: bool = True) -> str:
    """Compile ``pbb_oracle.c`` into ``liboracle.so`` with gcc (no HIP involved)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm", "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64, dbl, i32 = ctypes.c_int64, ctypes.c_double, ctypes.c_int
    vp = ctypes.c_void_p
    lib.oracle_pbb_member.argtypes = [i64, i64, i64, i64]
    lib.oracle_pbb_member.restype = i32
    lib.oracle_swa_member.argtypes = [i64, i64, i64]
    lib.oracle_swa_member.restype = i32
    lib.oracle_pbb_counts.argtypes = [i64, i64, i64, vp, vp]
    lib.oracle_pbb_counts.restype = None
    lib.oracle_swa_counts.argtypes = [i64, i64, i64, vp, vp]
    lib.oracle_swa_counts.restype = None
    lib.oracle_attend.argtypes = [i64, i64, vp, vp, vp, dbl, vp, vp]
    lib.oracle_attend.restype = None
    lib.oracle_decode.argtypes = [i32, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp, vp, i64,
                                  dbl, vp, i32]
    lib.oracle_decode.restype = i32
    lib.oracle_rope.argtypes = [i64, i64, dbl, vp, vp]
    lib.oracle_rope.restype = None
    lib.oracle_rope_rows.argtypes = [i64, i64, vp, dbl, vp, vp]
    lib.oracle_rope_rows.restype = None
    lib.oracle_decode_rope.argtypes = [i32, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp, vp,
                                       i64, dbl, dbl, vp, i32]
    lib.oracle_decode_rope.restype = i32
    lib.oracle_backward.argtypes = [i32, i64, i64, i64, i64, i64, i64, i64, vp, vp, vp, vp, dbl,
                                    vp, vp, vp, i32]
    lib.oracle_backward.restype = i32
    lib.oracle_prefill.argtypes = [i32, i64, i64, i64, i64, i64, i64, i64, vp, vp, vp, dbl, vp,
                                   vp, i32]
    lib.oracle_prefill.restype = i32
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ----------------------------------------------------------------------------------------
# Supports and counts

def pbb_member(t: int, s: int, block: int, bridge: int | None = None) -> bool:
    """``s in A_PBB(t)`` by the two-case Eq.(pbb); ``bridge`` defaults to ``block // 2``."""
    h = block // 2 if bridge is None else bridge
    return bool(_load().oracle_pbb_member(t, s, block, h))


def swa_member(t: int, s: int, window: int) -> bool:
    """``s in A_SWA(t) = {max(0, t-w+1) .. t}`` (Prop. 2)."""
    return bool(_load().oracle_swa_member(t, s, window))


def pbb_support(t: int, block: int, bridge: int | None = None) -> list[int]:
    """Sorted source positions of ``A_PBB(t)`` (candidate window, then membership test)."""
    h = block // 2 if bridge is None else bridge
    lo = max(0, t - block - h)
    return [s for s in range(lo, t + 1) if pbb_member(t, s, block, h)]


def swa_support(t: int, window: int) -> list[int]:
    lo = max(0, t - window)
    return [s for s in range(lo, t + 1) if swa_member(t, s, window)]


def pbb_counts(n: int, block: int, bridge: int | None = None) -> tuple[int, int]:
    """(total scores, cross-block scores) per head over a length-``n`` sequence."""
    h = block // 2 if bridge is None else bridge
    tot, cr = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_pbb_counts(n, block, h, ctypes.byref(tot), ctypes.byref(cr))
    return tot.value, cr.value


def swa_counts(n: int, window: int, block: int) -> tuple[int, int]:
    """(total scores, scores reaching an earlier ``block``-sized block) for SWA."""
    tot, cr = ctypes.c_int64(), ctypes.c_int64()
    _load().oracle_swa_counts(n, window, block, ctypes.byref(tot), ctypes.byref(cr))
    return tot.value, cr.value


# ----------------------------------------------------------------------------------------
# Attention

def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float | None = None):
    """Single-softmax attention of one query over explicit keys (Eq.(attention)).

    Returns ``(o, lse)`` with ``lse = log sum_s exp(z_s)``; an empty key set gives zeros and
    ``-inf`` (Appendix A.4, Eq.(lse): an empty part has ``Z = 0``).
    """
    q = np.ascontiguousarray(q, dtype=np.float64)
    d = q.shape[-1]
    k = np.ascontiguousarray(k, dtype=np.float64).reshape(-1, d)
    v = np.ascontiguousarray(v, dtype=np.float64).reshape(-1, d)
    assert k.shape == v.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    o = np.zeros(d, dtype=np.float64)
    lse = ctypes.c_double()
    _load().oracle_attend(k.shape[0], d, _ptr(q), _ptr(k), _ptr(v), float(scale), _ptr(o),
                          ctypes.byref(lse))
    return o, lse.value


def rope(x, pos: int, base: float) -> np.ndarray:
    """Rotary position embedding of head vector(s) ``x`` [..., d] at absolute position ``pos``
    (half-split pairs c, c + d/2; angle ``pos * base^(-2c/d)``), fp64."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    d = x.shape[-1]
    flat = x.reshape(-1, d)
    out = np.empty_like(flat)
    for r in range(flat.shape[0]):
        _load().oracle_rope(d, int(pos), float(base), _ptr(flat[r]), _ptr(out[r]))
    return out.reshape(x.shape)


def rope_rows(x, pos, base: float) -> np.ndarray:
    """:func:`rope` of every row of ``x`` [..., L, d] (float32 values) at its position ``pos``
    (int, broadcastable to ``x.shape[:-1]``); fp64 result of ``x``'s shape."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    d = x.shape[-1]
    p = np.ascontiguousarray(np.broadcast_to(np.asarray(pos, dtype=np.int64), x.shape[:-1]))
    flat = x.reshape(-1, d)
    out = np.empty(flat.shape, dtype=np.float64)
    _load().oracle_rope_rows(d, flat.shape[0], _ptr(p), float(base), _ptr(flat), _ptr(out))
    return out.reshape(x.shape)


def decode(mode: int, pos, q, k_hist, v_hist, hist_lo, *, block: int = 0, window: int = 0,
           scale: float | None = None, n_threads: int = 0, rope_base: float = 0.0) -> np.ndarray:
    """One batched decode step in fp64.

    ``pos``: int [batch] absolute positions t.  ``q``: [batch][Hq][d].
    ``k_hist``/``v_hist``: [batch][Hkv][hist_len][d] with absolute position ``s`` of sequence
    ``b`` stored at row ``s - hist_lo[b]``.  ``mode`` is :data:`PBB` (support Eq.(pbb) with
    ``h = block/2``) or :data:`SWA` (support of Prop. 2 with ``window``).  ``rope_base > 0``
    rotates q at ``pos`` and each (unrotated) history key at its own position (:func:`rope`).
    Returns float64 [batch][Hq][d].
    """
    pos = np.ascontiguousarray(pos, dtype=np.int64)
    q = np.ascontiguousarray(q, dtype=np.float32)
    k_hist = np.ascontiguousarray(k_hist, dtype=np.float32)
    v_hist = np.ascontiguousarray(v_hist, dtype=np.float32)
    hist_lo = np.ascontiguousarray(hist_lo, dtype=np.int64)
    batch, hq, d = q.shape
    assert k_hist.ndim == 4 and k_hist.shape == v_hist.shape
    assert k_hist.shape[0] == batch and k_hist.shape[3] == d
    hkv, hist_len = k_hist.shape[1], k_hist.shape[2]
    assert pos.shape == (batch,) and hist_lo.shape == (batch,)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((batch, hq, d), dtype=np.float64)
    if rope_base:
        rc = _load().oracle_decode_rope(int(mode), batch, hq, hkv, d, int(block), int(window),
                                        _ptr(pos), _ptr(q), _ptr(k_hist), _ptr(v_hist),
                                        _ptr(hist_lo), hist_len, float(scale), float(rope_base),
                                        _ptr(out), int(n_threads))
    else:
        rc = _load().oracle_decode(int(mode), batch, hq, hkv, d, int(block), int(window),
                                   _ptr(pos), _ptr(q), _ptr(k_hist), _ptr(v_hist), _ptr(hist_lo),
                                   hist_len, float(scale), _ptr(out), int(n_threads))
    if rc == 1:
        raise ValueError("oracle.decode: a support position is missing from the history")
    if rc != 0:
        raise ValueError("oracle.decode: invalid arguments")
    return out


def prefill(mode: int, q, k, v, *, block: int = 0, window: int = 0, scale: float | None = None,
            n_threads: int = 0):
    """Prefill of prompts at positions ``0 .. n-1`` in fp64: every position attends over its
    own support (Eq.(pbb) with ``h = block/2`` for :data:`PBB`, Prop. 2 for :data:`SWA`).

    ``q``: [batch][n][Hq][d]; ``k``/``v``: [batch][n][Hkv][d] (token-major).  Returns
    ``(out, lse)``: float64 [batch][n][Hq][d] and the log-partition ``log sum_s e^{z_s}``
    (Appendix A.4, Eq.(lse)) as float64 [batch][Hq][n].
    """
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    batch, n, hq, d = q.shape
    assert k.shape == v.shape and k.shape[:2] == (batch, n) and k.shape[3] == d
    hkv = k.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((batch, n, hq, d), dtype=np.float64)
    lse = np.zeros((batch, hq, n), dtype=np.float64)
    rc = _load().oracle_prefill(int(mode), batch, n, hq, hkv, d, int(block), int(window),
                                _ptr(q), _ptr(k), _ptr(v), float(scale), _ptr(out), _ptr(lse),
                                int(n_threads))
    if rc != 0:
        raise ValueError("oracle.prefill: invalid arguments")
    return out, lse


def backward(mode: int, q, k, v, dout, *, block: int = 0, window: int = 0,
             scale: float | None = None, n_threads: int = 0):
    """Gradients of :func:`prefill`'s output with respect to q, k, v for the upstream gradient
    ``dout`` ([batch][n][Hq][d]), fp64: returns ``(dq, dk, dv)`` shaped like q, k, v."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    dout = np.ascontiguousarray(dout, dtype=np.float32)
    batch, n, hq, d = q.shape
    assert dout.shape == q.shape and k.shape == v.shape and k.shape[:2] == (batch, n)
    hkv = k.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    dq = np.zeros(q.shape, dtype=np.float64)
    dk = np.zeros(k.shape, dtype=np.float64)
    dv = np.zeros(v.shape, dtype=np.float64)
    rc = _load().oracle_backward(int(mode), batch, n, hq, hkv, d, int(block), int(window),
                                 _ptr(q), _ptr(k), _ptr(v), _ptr(dout), float(scale), _ptr(dq),
                                 _ptr(dk), _ptr(dv), int(n_threads))
    if rc != 0:
        raise ValueError("oracle.backward: invalid arguments")
    return dq, dk, dv


# ----------------------------------------------------------------------------------------
# Ring image

def expected_ring(hist: np.ndarray, hist_lo, t_last, first_written, slots: int,
                  initial: np.ndarray | None = None) -> np.ndarray:
    """Ring contents after writing positions ``first_written[b] .. t_last[b]`` in order.

    Position ``s`` lives at slot ``s mod slots`` (Appendix F.1, Proposition "Relocation-free
    PBB cache"; the same rule with ``slots`` entries for the sliding-window ring).  Slot ``j``
    therefore holds the LAST written position congruent to ``j``:
    ``s* = t_last - ((t_last - j) mod slots)`` if ``s* >= first_written``, otherwise its
    initial content (zeros unless ``initial`` is given).

    ``hist``: [batch][Hkv][hist_len][d] (any dtype; values are copied bit for bit) holding
    position ``s`` at row ``s - hist_lo[b]``.  Returns [batch][Hkv][slots][d] of ``hist.dtype``.
    """
    batch, hkv, hist_len, d = hist.shape
    hist_lo = np.asarray(hist_lo, dtype=np.int64).reshape(batch)
    t_last = np.asarray(t_last, dtype=np.int64).reshape(batch)
    first_written = np.asarray(first_written, dtype=np.int64).reshape(batch)
    if initial is None:
        ring = np.zeros((batch, hkv, slots, d), dtype=hist.dtype)
    else:
        ring = np.array(initial, dtype=hist.dtype, copy=True).reshape(batch, hkv, slots, d)
    j = np.arange(slots, dtype=np.int64)
    for b in range(batch):
        s_star = t_last[b] - np.mod(t_last[b] - j, slots)
        ok = s_star >= first_written[b]
        if not ok.any():
            continue
        rows = s_star[ok] - hist_lo[b]
        if rows.min() < 0 or rows.max() >= hist_len:
            raise ValueError("expected_ring: a written position is missing from the history")
        ring[b, :, j[ok], :] = np.transpose(hist[b][:, rows, :], (1, 0, 2))
    return ring
