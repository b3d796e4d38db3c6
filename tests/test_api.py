"""C-ABI surface of libpbb.

CPU tests: the library loads, exports every function ``include/pbb.h`` declares, and each
invalid argument returns its documented status before anything is enqueued (fake, never
dereferenced device addresses are enough for that).  GPU tests: a failing call leaves every
buffer untouched, and the size queries agree with the paper's KV-bytes formula.
"""
import ctypes
import os
import re

import pytest
import torch

import paper_2606_02680_amd as P
from paper_2606_02680_amd import pbb as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "pbb.h")
A = 0x10000  # an aligned fake device address (never dereferenced: validation fails first)


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\S.*?\b((?:pbb|swa)_[a-z_]+)\s*\(", text, re.M)))


def test_header_symbols_exported():
    lib = B.load_library()
    names = _declared()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for code in range(7):
        assert B.lib_status_string(code).startswith(B.STATUS_NAMES[code])
    assert "UNKNOWN" in B.lib_status_string(99)


def _desc(**kw):
    base = dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=64, block=64, window=0, slots=64,
                dtype=B.DTYPE_BF16, scale=0.0)
    base.update(kw)
    return B.PbbDesc(**base)


def _decode(desc, fn="pbb_decode_step", **ptrs):
    args = dict(pos=A, q=A, k_new=A, v_new=A, k_ring=A, v_ring=A, out=A, ws=0)
    args.update(ptrs)
    lib = B.load_library()
    vp = ctypes.c_void_p
    d = None if desc is None else ctypes.byref(desc)
    return getattr(lib, fn)(d, vp(args["pos"]), vp(args["q"]), vp(args["k_new"]),
                            vp(args["v_new"]), vp(args["k_ring"]), vp(args["v_ring"]),
                            vp(args["out"]), vp(args["ws"]), ctypes.c_size_t(0), vp(0))


@pytest.mark.parametrize("fn", ["pbb_decode_step", "swa_decode_step"])
def test_null_arguments(fn):
    desc = _desc(window=32, slots=64) if fn == "swa_decode_step" else _desc()
    assert _decode(None, fn) == 1
    for name in ("pos", "q", "k_new", "v_new", "k_ring", "v_ring", "out"):
        assert _decode(desc, fn, **{name: 0}) == 1, name


@pytest.mark.parametrize("bad", [
    dict(batch=0), dict(n_kv_heads=0), dict(n_q_heads=6, n_kv_heads=4), dict(n_q_heads=34,
    n_kv_heads=2), dict(head_dim=96), dict(head_dim=256), dict(block=63, slots=63),
    dict(block=64, slots=128), dict(block=0, slots=0), dict(block=131072, slots=131072)])
def test_pbb_shape_errors(bad):
    assert _decode(_desc(**bad)) == 2


@pytest.mark.parametrize("bad", [dict(window=65, slots=64), dict(window=-1, slots=64),
                                 dict(window=8, slots=100000)])
def test_swa_shape_errors(bad):
    assert _decode(_desc(**bad), "swa_decode_step") == 2


def test_swa_descriptor_rejected_by_pbb_step():
    # slots != block under the PBB rules
    assert _decode(_desc(window=64, slots=128, block=64)) == 2


def test_dtype_error():
    assert _decode(_desc(dtype=7)) == 3


@pytest.mark.parametrize("name", ["q", "k_new", "v_new", "k_ring", "v_ring", "out"])
def test_alignment_errors(name):
    assert _decode(_desc(), **{name: A + 8}) == 4
    assert _decode(_desc(window=64, slots=64), "swa_decode_step", **{name: A + 2}) == 4


def _advance(desc, fn="pbb_decode_step_advance", **ptrs):
    args = dict(pos=A, pos_next=A + 4096, q=A, k_new=A, v_new=A, k_ring=A, v_ring=A, out=A)
    args.update(ptrs)
    vp = ctypes.c_void_p
    return getattr(B.load_library(), fn)(
        ctypes.byref(desc), vp(args["pos"]), vp(args["pos_next"]), vp(args["q"]),
        vp(args["k_new"]), vp(args["v_new"]), vp(args["k_ring"]), vp(args["v_ring"]),
        vp(args["out"]), vp(0), ctypes.c_size_t(0), vp(0))


@pytest.mark.parametrize("fn", ["pbb_decode_step_advance", "swa_decode_step_advance"])
def test_advance_argument_errors(fn):
    desc = _desc(window=32, slots=64) if fn.startswith("swa") else _desc()
    assert _advance(desc, fn, pos_next=0) == 1
    assert _advance(desc, fn, pos_next=A + 4098) == 4
    assert _advance(desc, fn, pos_next=A) == 2          # aliases pos
    assert _advance(desc, fn, pos_next=A + 4) == 2      # overlaps pos[1] (batch 2)
    assert _advance(desc, fn, q=A + 2) == 4


def test_pos_alignment():
    assert _decode(_desc(), pos=A + 2) == 4


def test_ring_bytes_and_workspace():
    desc = _desc()
    assert P.ring_bytes(desc) == 2 * 2 * 64 * 64 * 2
    assert P.workspace_bytes(desc) == 0
    swa = _desc(window=48, slots=64)
    assert P.ring_bytes(swa) == 2 * 2 * 64 * 64 * 2
    assert P.swa_workspace_bytes(swa) == 0
    # Paper's local KV storage 2*batch*b*H_KV*d_h*u = 65,536 B at (1, 128, 2, 64, bf16)
    paper = P.make_desc(1, 12, 2, 64, block=128)
    assert 2 * P.ring_bytes(paper) == 65536
    with pytest.raises(P.PbbError):
        P.ring_bytes(_desc(head_dim=80))


def test_ring_fill_and_init_errors():
    lib = B.load_library()
    vp = ctypes.c_void_p
    desc = _desc()
    assert lib.pbb_ring_init(None, vp(A), vp(A), vp(0)) == 1
    assert lib.pbb_ring_init(ctypes.byref(desc), vp(0), vp(A), vp(0)) == 1
    assert lib.pbb_ring_init(ctypes.byref(desc), vp(A + 4), vp(A), vp(0)) == 4
    fill = lambda n, **kw: lib.pbb_ring_fill(ctypes.byref(desc), vp(kw.get("pos", A)),
                                             vp(kw.get("ks", A)), vp(A), n, vp(A), vp(A), vp(0))
    assert fill(65) == 2          # longer than the ring
    assert fill(-1) == 2
    assert fill(8, ks=0) == 1
    assert fill(8, pos=0) == 1
    assert fill(8, ks=A + 8) == 4


# ---------------------------------------------------------------------------------------
# GPU: failing calls write nothing

@pytest.mark.gpu
def test_failed_calls_leave_buffers_untouched(cuda):
    desc = P.make_desc(2, 8, 2, 64, block=64)
    canary = 0x5A5A
    mk = lambda *s: torch.full(s, canary, dtype=torch.int16, device=cuda).view(torch.bfloat16)
    q, out = mk(2, 8, 64), mk(2, 8, 64)
    kn, vn = mk(2, 2, 64), mk(2, 2, 64)
    kr, vr = mk(2, 2, 64, 64), mk(2, 2, 64, 64)
    pos = torch.zeros(2, dtype=torch.int32, device=cuda)
    bad = P.make_desc(2, 8, 3, 64, block=64)  # 8 % 3 != 0
    ptr = lambda t: t.data_ptr()
    st = _decode(bad, pos=ptr(pos), q=ptr(q), k_new=ptr(kn), v_new=ptr(vn), k_ring=ptr(kr),
                 v_ring=ptr(vr), out=ptr(out))
    assert st == 2
    st = _decode(desc, pos=ptr(pos), q=ptr(q) + 2, k_new=ptr(kn), v_new=ptr(vn),
                 k_ring=ptr(kr), v_ring=ptr(vr), out=ptr(out))
    assert st == 4
    torch.cuda.synchronize()
    for t in (q, out, kn, vn, kr, vr):
        assert bool((t.view(torch.int16) == canary).all())
    # A valid call on the same buffers does write (sanity of the canary check).
    P.pbb_decode_step(desc, pos, q.zero_(), kn.zero_(), vn.zero_(), kr.zero_(), vr.zero_(), out)
    torch.cuda.synchronize()
    assert not bool((out.view(torch.int16) == canary).any())


def _prefill(desc, fn="pbb_prefill", n=64, **ptrs):
    args = dict(q=A, k=A, v=A, out=A, lse=0, kr=0, vr=0)
    args.update(ptrs)
    vp = ctypes.c_void_p
    return getattr(B.load_library(), fn)(
        ctypes.byref(desc), n, vp(args["q"]), vp(args["k"]), vp(args["v"]), vp(args["out"]),
        vp(args["lse"]), vp(args["kr"]), vp(args["vr"]), vp(0))


@pytest.mark.parametrize("fn", ["pbb_prefill", "swa_prefill"])
def test_prefill_argument_errors(fn):
    desc = _desc(window=32, slots=64) if fn == "swa_prefill" else _desc()
    lib = B.load_library()
    vp = ctypes.c_void_p
    assert getattr(lib, fn)(None, 8, vp(A), vp(A), vp(A), vp(A), vp(0), vp(0), vp(0), vp(0)) == 1
    for name in ("q", "k", "v", "out"):
        assert _prefill(desc, fn, **{name: 0}) == 1, name
    assert _prefill(desc, fn, kr=A) == 1                 # one ring without the other
    assert _prefill(desc, fn, vr=A) == 1
    assert _prefill(desc, fn, n=-1) == 2
    assert _prefill(desc, fn, n=(1 << 30) + 1) == 2
    for name in ("q", "k", "v", "out", "kr"):
        kw = {name: A + 8}
        if name == "kr":
            kw["vr"] = A
        assert _prefill(desc, fn, **kw) == 4, name
    assert _prefill(desc, fn, lse=A + 2) == 4
    f32 = _desc(window=32, slots=64, dtype=B.DTYPE_F32) if fn == "swa_prefill" else _desc(dtype=B.DTYPE_F32)
    assert _prefill(f32, fn) == 3                         # bf16 only
    bad = _desc(window=65, slots=64) if fn == "swa_prefill" else _desc(block=63, slots=63)
    assert _prefill(bad, fn) == 2
    assert _prefill(desc, fn, n=0) == 0                   # nothing to do, nothing launched


def test_rope_descriptor_rules():
    assert _decode(_desc(rope_base=0.5)) == 2                   # bases in (0, 1] are rejected
    assert _decode(_desc(rope_base=float("nan"))) == 2
    assert _decode(_desc(rope_base=-1.0)) == 2
    assert _decode(_desc(rope_base=1e6, dtype=B.DTYPE_F32)) == 3  # rotary decode is bf16 only
    assert _prefill(_desc(rope_base=1e6)) == 2                   # prefill takes rotated inputs
    assert _decode(_desc(rope_base=1e6), q=A + 2) == 4           # other checks unchanged


def _backward(desc, fn="pbb_backward", n=64, **ptrs):
    args = dict(q=A, k=A, v=A, out=A, dout=A, lse=A, dq=A, dk=A, dv=A, ws=A, ws_bytes=1 << 20)
    args.update(ptrs)
    vp = ctypes.c_void_p
    return getattr(B.load_library(), fn)(
        ctypes.byref(desc), n, vp(args["q"]), vp(args["k"]), vp(args["v"]), vp(args["out"]),
        vp(args["dout"]), vp(args["lse"]), vp(args["dq"]), vp(args["dk"]), vp(args["dv"]),
        vp(args["ws"]), ctypes.c_size_t(args["ws_bytes"]), vp(0))


@pytest.mark.parametrize("fn", ["pbb_backward", "swa_backward"])
def test_backward_argument_errors(fn):
    desc = _desc(window=32, slots=64) if fn == "swa_backward" else _desc()
    for name in ("q", "k", "v", "out", "dout", "lse", "dq", "dk", "dv"):
        assert _backward(desc, fn, **{name: 0}) == 1, name
    for name in ("q", "k", "v", "out", "dout", "dq", "dk", "dv"):
        assert _backward(desc, fn, **{name: A + 8}) == 4, name
    assert _backward(desc, fn, lse=A + 2) == 4
    need = P.backward_workspace_bytes(desc, 64)
    assert need == 2 * 8 * 64 * 8          # batch x Hq x n x 2 floats (256-byte multiple)
    assert _backward(desc, fn, ws=0) == 5
    assert _backward(desc, fn, ws_bytes=need - 1) == 5
    assert _backward(desc, fn, ws=A + 4, ws_bytes=need) == 4
    assert _backward(desc, fn, n=-1) == 2
    f32 = _desc(window=32, slots=64, dtype=B.DTYPE_F32) if fn == "swa_backward" else _desc(dtype=B.DTYPE_F32)
    assert _backward(f32, fn) == 3
    assert _backward(_desc(rope_base=1e6), "pbb_backward") == 2
    assert _backward(desc, fn, n=0, ws=0) == 0


def test_split_decode_workspace():
    """bf16 launches with at most 64 (sequence, KV head) units split each unit over up to eight
    workgroups and need a workspace: counters (256-byte aligned) plus partial states."""
    one = B.make_desc(1, 32, 8, 128, block=2048, dtype=torch.bfloat16)
    # 8 units -> min(floor(256 / 8), ceil(64 / 8), 8) = 8 workgroups per unit
    assert P.workspace_bytes(one) == 256 + 8 * 8 * 4 * (128 + 2) * 4
    swa = B.make_desc(2, 8, 2, 128, window=4096, slots=4096, dtype=torch.bfloat16)
    assert P.swa_workspace_bytes(swa) == 256 + 4 * min(64, 16, 8) * 4 * 130 * 4
    mid = B.make_desc(5, 32, 8, 128, block=2048, dtype=torch.bfloat16)    # 40 units
    assert P.workspace_bytes(mid) == 256 + 40 * 6 * 4 * 130 * 4           # floor(256 / 40) = 6
    many = B.make_desc(9, 32, 8, 128, block=2048, dtype=torch.bfloat16)   # 72 units
    assert P.workspace_bytes(many) == 0
    short = B.make_desc(1, 32, 8, 128, block=256, dtype=torch.bfloat16)   # 8 steps at most
    assert P.workspace_bytes(short) == 0
    f32 = B.make_desc(1, 32, 8, 128, block=2048, dtype=torch.float32)
    assert P.workspace_bytes(f32) == 0
    # a split launch without (or with too small) a workspace is refused before launching
    vp = ctypes.c_void_p
    lib = B.load_library()
    args = [ctypes.byref(one), vp(A), vp(A), vp(A), vp(A), vp(A), vp(A), vp(A)]
    assert lib.pbb_decode_step(*args, vp(0), ctypes.c_size_t(0), vp(0)) == 5
    assert lib.pbb_decode_step(*args, vp(A), ctypes.c_size_t(P.workspace_bytes(one) - 1), vp(0)) == 5
    assert lib.pbb_decode_step(*args, vp(A + 8), ctypes.c_size_t(1 << 24), vp(0)) == 4


def test_split_rule_over_random_descriptors():
    """The documented split rule, restated: bf16 launches with at most 64 (sequence, KV head)
    units split each unit over S = min(floor(256 / units), ceil(steps / 8), 8) workgroups
    (steps = ceil(B / 32) or ceil(W / 32)); S > 1 needs 256-byte-aligned counters plus
    units * S * G * (d + 2) floats."""
    import numpy as np
    rng = np.random.default_rng(3)
    for _ in range(400):
        batch = int(rng.integers(1, 80))
        hkv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.integers(1, 17))
        d = int(rng.choice([64, 128]))
        swa = bool(rng.integers(0, 2))
        span = int(rng.choice([2, 64, 256, 258, 300, 1024, 2048, 4096, 65536]))
        dt = torch.bfloat16 if rng.integers(0, 4) else torch.float32
        if swa:
            desc = B.make_desc(batch, G * hkv, hkv, d, window=span, slots=span, dtype=dt)
            got = P.swa_workspace_bytes(desc)
        else:
            desc = B.make_desc(batch, G * hkv, hkv, d, block=span, dtype=dt)
            got = P.workspace_bytes(desc)
        units = batch * hkv
        steps = -(-span // 32)
        S = min(256 // units, -(-steps // 8), 8) if units <= 64 else 1
        if dt != torch.bfloat16 or S <= 1:
            assert got == 0, (batch, hkv, G, d, swa, span, dt)
            continue
        counters = -(-(units * 4) // 256) * 256
        part = units * S * G * (d + 2) * 4
        assert got == counters + -(-part // 256) * 256, (batch, hkv, G, d, swa, span)


def _noalloc(desc, **ptrs):
    args = dict(pos=A, q=A, k_new=A, v_new=A, k_ring=A, v_ring=A, out=A)
    args.update(ptrs)
    vp = ctypes.c_void_p
    d = None if desc is None else ctypes.byref(desc)
    return B.load_library().pbb_decode_step_noalloc(
        d, vp(args["pos"]), vp(args["q"]), vp(args["k_new"]), vp(args["v_new"]),
        vp(args["k_ring"]), vp(args["v_ring"]), vp(args["out"]), vp(0))


def test_noalloc_argument_errors():
    """The allocation-free decode validates like pbb_decode_step before touching its scratch
    buffer (these calls fail before any HIP call, so they run without a GPU)."""
    assert _noalloc(None) == 1
    desc = _desc()
    for name in ("pos", "q", "k_new", "v_new", "k_ring", "v_ring", "out"):
        assert _noalloc(desc, **{name: 0}) == 1, name
    assert _noalloc(_desc(block=63, slots=63)) == 2
    assert _noalloc(_desc(window=64, slots=128, block=64)) == 2   # slots != block (PBB rules)
    assert _noalloc(_desc(dtype=7)) == 3
    assert _noalloc(_desc(dtype=B.DTYPE_F32, rope_base=1e6)) == 3
    assert _noalloc(desc, q=A + 8) == 4
    # the largest split launch the rules allow fits the library's buffer
    big = _desc(batch=4, n_q_heads=256, n_kv_heads=16, head_dim=128, block=65536, slots=65536)
    assert B.workspace_bytes(big) <= 4260096


def test_stream_probe_library_exports_and_validates():
    """The measurement helper libpbbprobe.so exports what include/pbb_probe.h declares and
    rejects bad arguments on the host (code 1) before any HIP call."""
    path = os.path.join(os.path.dirname(B._LIB_PATH), "libpbbprobe.so")
    lib = ctypes.CDLL(path)
    text = open(os.path.join(os.path.dirname(HEADER), "pbb_probe.h")).read()
    names = set(re.findall(r"^\S.*?\b(pbb_probe_[a-z_]+)\s*\(", text, re.M))
    assert names == {"pbb_probe_stream"}
    vp = ctypes.c_void_p
    f = lib.pbb_probe_stream
    f.argtypes = [vp, vp, ctypes.c_size_t, vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_int32, vp, vp]
    f.restype = ctypes.c_int
    ok = dict(k=A, v=A, stride=2048 * 256, rows=A, units=4, max_rows=2048, waves=4, nt=1, sink=A)

    def call(**kw):
        a = dict(ok, **kw)
        return f(vp(a["k"]), vp(a["v"]), ctypes.c_size_t(a["stride"]), vp(a["rows"]), a["units"],
                 a["max_rows"], a["waves"], a["nt"], vp(a["sink"]), vp(0))

    assert call(k=0) == 1 and call(rows=0) == 1 and call(sink=0) == 1
    assert call(units=0) == 1 and call(waves=3) == 1 and call(max_rows=0) == 1
    assert call(max_rows=2049) == 1          # rows would run past the unit's region
    assert call(k=A + 8) == 1 and call(stride=2048 * 256 + 8) == 1
