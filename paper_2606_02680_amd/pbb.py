"""ctypes binding of libpbb (``include/pbb.h``).

Argument marshalling only: every function checks that the tensors match the descriptor
(device, dtype, shape, contiguity), passes raw device pointers and the current HIP stream of
PyTorch to the C entry point of the same name, and raises :class:`PbbError` on a non-OK
status.  All computation happens in the library's HIP kernels; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpbb.so")

PBB_OK = 0
STATUS_NAMES = {0: "PBB_OK", 1: "PBB_ERR_NULL", 2: "PBB_ERR_SHAPE", 3: "PBB_ERR_DTYPE",
                4: "PBB_ERR_ALIGN", 5: "PBB_ERR_WORKSPACE", 6: "PBB_ERR_LAUNCH"}
DTYPE_F32 = 0
DTYPE_BF16 = 1
_TORCH_DTYPE = {DTYPE_F32: torch.float32, DTYPE_BF16: torch.bfloat16}

EXPORTS = ("pbb_status_string", "pbb_ring_bytes", "pbb_ring_init", "pbb_ring_fill",
           "pbb_workspace_bytes", "pbb_decode_step", "swa_workspace_bytes", "swa_decode_step",
           "pbb_decode_step_advance", "swa_decode_step_advance", "pbb_prefill", "swa_prefill",
           "pbb_backward_workspace_bytes", "pbb_backward", "swa_backward",
           "pbb_decode_step_noalloc")


class PbbError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)} ({lib_status_string(status)})")


class PbbDesc(ctypes.Structure):
    """Mirror of ``pbb_desc_t``."""
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block", ctypes.c_int32), ("window", ctypes.c_int32),
                ("slots", ctypes.c_int32), ("dtype", ctypes.c_int32), ("scale", ctypes.c_float),
                ("rope_base", ctypes.c_float)]

    @property
    def torch_dtype(self) -> torch.dtype:
        return _TORCH_DTYPE[self.dtype]

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


_lib = None


def load_library(path: str = _LIB_PATH):
    """Load libpbb.so; raises if it has not been built (no silent fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libpbb.so not found at {path}: build it with "
                          "`python -m paper_2606_02680_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    dp = ctypes.POINTER(PbbDesc)
    lib.pbb_status_string.argtypes = [ctypes.c_int]
    lib.pbb_status_string.restype = ctypes.c_char_p
    lib.pbb_ring_bytes.argtypes = [dp, ctypes.POINTER(sz)]
    lib.pbb_ring_init.argtypes = [dp, vp, vp, vp]
    lib.pbb_ring_fill.argtypes = [dp, vp, vp, vp, i32, vp, vp, vp]
    lib.pbb_workspace_bytes.argtypes = [dp, ctypes.POINTER(sz)]
    lib.swa_workspace_bytes.argtypes = [dp, ctypes.POINTER(sz)]
    for fn in ("pbb_decode_step", "swa_decode_step"):
        getattr(lib, fn).argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    for fn in ("pbb_decode_step_advance", "swa_decode_step_advance"):
        getattr(lib, fn).argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.pbb_decode_step_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp]
    for fn in ("pbb_prefill", "swa_prefill"):
        getattr(lib, fn).argtypes = [dp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.pbb_backward_workspace_bytes.argtypes = [dp, i32, ctypes.POINTER(sz)]
    for fn in ("pbb_backward", "swa_backward"):
        getattr(lib, fn).argtypes = [dp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    for fn in EXPORTS[1:]:
        getattr(lib, fn).restype = ctypes.c_int
    _lib = lib
    return lib


def lib_status_string(status: int) -> str:
    return load_library().pbb_status_string(int(status)).decode()


def make_desc(batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int, *, block: int = 0,
              window: int = 0, slots: int | None = None, dtype=torch.bfloat16,
              scale: float = 0.0, rope_base: float = 0.0) -> PbbDesc:
    """Descriptor for a PBB ring (``block`` = B, ``slots`` = B) or, with ``window`` > 0, an SWA
    ring (``slots`` >= ``window``, default ``window``).  ``rope_base`` > 1 makes the decode
    steps apply the rotary embedding to q and k_new themselves (see ``include/pbb.h``)."""
    if slots is None:
        slots = window if window > 0 else block
    code = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16}.get(dtype, dtype)
    return PbbDesc(batch, n_q_heads, n_kv_heads, head_dim, block, window, slots, int(code),
                   float(scale), float(rope_base))


def _torch_stream(stream):
    """The torch stream object of ``stream`` (None: torch's current stream; a raw hipStream_t
    handle is wrapped as an external stream)."""
    if stream is None:
        return torch.cuda.current_stream()
    if hasattr(stream, "cuda_stream"):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _stream(stream):
    return ctypes.c_void_p(_torch_stream(stream).cuda_stream)


def _scratch_on(stream, make):
    """Allocate a temporary buffer with ``make()`` for a launch on ``stream``: the allocation
    (and a zero fill, if ``make`` does one) is ordered on that stream, and the caching allocator
    ties the block to it, so the block is not handed to other work until the launch is done."""
    s = _torch_stream(stream)
    with torch.cuda.stream(s):
        return make()


def _ptr(t: torch.Tensor | None):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _check(fn: str, status: int):
    if status != PBB_OK:
        raise PbbError(fn, status)


def _expect(name: str, t: torch.Tensor, shape, dtype):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be a GPU tensor, got {t.device}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)} != {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype} != {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def ring_bytes(desc: PbbDesc) -> int:
    out = ctypes.c_size_t()
    _check("pbb_ring_bytes", load_library().pbb_ring_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def workspace_bytes(desc: PbbDesc) -> int:
    out = ctypes.c_size_t()
    _check("pbb_workspace_bytes",
           load_library().pbb_workspace_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def swa_workspace_bytes(desc: PbbDesc) -> int:
    out = ctypes.c_size_t()
    _check("swa_workspace_bytes",
           load_library().swa_workspace_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def alloc_workspace(desc: PbbDesc, device="cuda"):
    """Zero-filled workspace for the decode calls of ``desc`` (PBB or SWA rules by
    ``desc.window``), or None when they need none.  Launches leave its counters zeroed, so one
    allocation serves every later call on one stream (calls that may overlap need their own)."""
    n = swa_workspace_bytes(desc) if desc.window > 0 else workspace_bytes(desc)
    return torch.zeros(n, dtype=torch.uint8, device=device) if n > 0 else None


def ring_shape(desc: PbbDesc):
    return (desc.batch, desc.n_kv_heads, desc.slots, desc.head_dim)


def alloc_rings(desc: PbbDesc, device="cuda"):
    """Allocate (uninitialised) K and V rings for ``desc``."""
    shape = ring_shape(desc)
    return (torch.empty(shape, dtype=desc.torch_dtype, device=device),
            torch.empty(shape, dtype=desc.torch_dtype, device=device))


def ring_init(desc: PbbDesc, k_ring: torch.Tensor, v_ring: torch.Tensor, stream=None):
    for n, t in (("k_ring", k_ring), ("v_ring", v_ring)):
        _expect(n, t, ring_shape(desc), desc.torch_dtype)
    _check("pbb_ring_init", load_library().pbb_ring_init(
        ctypes.byref(desc), _ptr(k_ring), _ptr(v_ring), _stream(stream)))


def ring_fill(desc: PbbDesc, pos: torch.Tensor, k_src: torch.Tensor, v_src: torch.Tensor,
              k_ring: torch.Tensor, v_ring: torch.Tensor, stream=None):
    """Load history rows ``pos[b]-L .. pos[b]-1`` (``k_src`` [batch][Hkv][L][d]) into the rings."""
    src_len = k_src.shape[2]
    _expect("pos", pos, (desc.batch,), torch.int32)
    for n, t in (("k_src", k_src), ("v_src", v_src)):
        _expect(n, t, (desc.batch, desc.n_kv_heads, src_len, desc.head_dim), desc.torch_dtype)
    for n, t in (("k_ring", k_ring), ("v_ring", v_ring)):
        _expect(n, t, ring_shape(desc), desc.torch_dtype)
    _check("pbb_ring_fill", load_library().pbb_ring_fill(
        ctypes.byref(desc), _ptr(pos), _ptr(k_src), _ptr(v_src), int(src_len), _ptr(k_ring),
        _ptr(v_ring), _stream(stream)))


def _decode(fn: str, desc: PbbDesc, pos, q, k_new, v_new, k_ring, v_ring, out, workspace,
            stream, pos_next=None):
    _expect("pos", pos, (desc.batch,), torch.int32)
    if pos_next is not None:
        _expect("pos_next", pos_next, (desc.batch,), torch.int32)
    _expect("q", q, (desc.batch, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    _expect("out", out, (desc.batch, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    for n, t in (("k_new", k_new), ("v_new", v_new)):
        _expect(n, t, (desc.batch, desc.n_kv_heads, desc.head_dim), desc.torch_dtype)
    for n, t in (("k_ring", k_ring), ("v_ring", v_ring)):
        _expect(n, t, ring_shape(desc), desc.torch_dtype)
    if workspace is None:
        # a fresh zero-filled workspace when the launch needs one (split workgroups), allocated
        # and cleared on the launch stream; callers that capture graphs or step in a loop pass
        # their own from alloc_workspace
        workspace = _scratch_on(stream, lambda: alloc_workspace(desc, q.device))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    extra = () if pos_next is None else (_ptr(pos_next),)
    _check(fn, getattr(load_library(), fn)(
        ctypes.byref(desc), _ptr(pos), *extra, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_ring),
        _ptr(v_ring), _ptr(out), _ptr(workspace), ctypes.c_size_t(ws_bytes), _stream(stream)))
    return out


def pbb_decode_step(desc: PbbDesc, pos, q, k_new, v_new, k_ring, v_ring, out, workspace=None,
                    stream=None):
    """Fused ring append + PBB attention for every sequence (see ``include/pbb.h``)."""
    return _decode("pbb_decode_step", desc, pos, q, k_new, v_new, k_ring, v_ring, out, workspace,
                   stream)


def swa_decode_step(desc: PbbDesc, pos, q, k_new, v_new, k_ring, v_ring, out, workspace=None,
                    stream=None):
    """Fused ring append + sliding-window attention (baseline, same kernels)."""
    return _decode("swa_decode_step", desc, pos, q, k_new, v_new, k_ring, v_ring, out, workspace,
                   stream)


def pbb_decode_step_noalloc(desc: PbbDesc, pos, q, k_new, v_new, k_ring, v_ring, out, stream=None):
    """:func:`pbb_decode_step` without a workspace argument: split launches use the library's
    per-device scratch buffer (nothing is allocated; overlapping calls on one GPU race)."""
    _expect("pos", pos, (desc.batch,), torch.int32)
    _expect("q", q, (desc.batch, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    _expect("out", out, (desc.batch, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    for n, t in (("k_new", k_new), ("v_new", v_new)):
        _expect(n, t, (desc.batch, desc.n_kv_heads, desc.head_dim), desc.torch_dtype)
    for n, t in (("k_ring", k_ring), ("v_ring", v_ring)):
        _expect(n, t, ring_shape(desc), desc.torch_dtype)
    _check("pbb_decode_step_noalloc", load_library().pbb_decode_step_noalloc(
        ctypes.byref(desc), _ptr(pos), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_ring),
        _ptr(v_ring), _ptr(out), _stream(stream)))
    return out


def pbb_decode_step_advance(desc: PbbDesc, pos, pos_next, q, k_new, v_new, k_ring, v_ring, out,
                            workspace=None, stream=None):
    """:func:`pbb_decode_step` that also writes ``pos_next = pos + 1`` (``pos`` unchanged)."""
    return _decode("pbb_decode_step_advance", desc, pos, q, k_new, v_new, k_ring, v_ring, out,
                   workspace, stream, pos_next=pos_next)


def swa_decode_step_advance(desc: PbbDesc, pos, pos_next, q, k_new, v_new, k_ring, v_ring, out,
                            workspace=None, stream=None):
    """:func:`swa_decode_step` that also writes ``pos_next = pos + 1`` (``pos`` unchanged)."""
    return _decode("swa_decode_step_advance", desc, pos, q, k_new, v_new, k_ring, v_ring, out,
                   workspace, stream, pos_next=pos_next)


def _prefill(fn: str, desc: PbbDesc, q, k, v, out, lse, k_ring, v_ring, stream):
    if q.dim() != 4:
        raise ValueError(f"{fn}: q must be [batch][n][Hq][d], got {tuple(q.shape)}")
    n = q.shape[1]
    _expect("q", q, (desc.batch, n, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    _expect("out", out, (desc.batch, n, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    for name, t in (("k", k), ("v", v)):
        _expect(name, t, (desc.batch, n, desc.n_kv_heads, desc.head_dim), desc.torch_dtype)
    if lse is not None:
        _expect("lse", lse, (desc.batch, desc.n_q_heads, n), torch.float32)
    if (k_ring is None) != (v_ring is None):
        raise ValueError(f"{fn}: pass both rings or neither")
    if k_ring is not None:
        for name, t in (("k_ring", k_ring), ("v_ring", v_ring)):
            _expect(name, t, ring_shape(desc), desc.torch_dtype)
    _check(fn, getattr(load_library(), fn)(
        ctypes.byref(desc), int(n), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
        _ptr(k_ring), _ptr(v_ring), _stream(stream)))
    return out


def pbb_prefill(desc: PbbDesc, q, k, v, out, lse=None, k_ring=None, v_ring=None, stream=None):
    """PBB attention for every position of prompts at positions ``0 .. n-1`` (q, out
    [batch][n][Hq][d]; k, v [batch][n][Hkv][d]); optional log-partitions ``lse``
    [batch][Hq][n] (float32) and ring state for decoding from position ``n``."""
    return _prefill("pbb_prefill", desc, q, k, v, out, lse, k_ring, v_ring, stream)


def swa_prefill(desc: PbbDesc, q, k, v, out, lse=None, k_ring=None, v_ring=None, stream=None):
    """Sliding-window counterpart of :func:`pbb_prefill` (support of Prop. 2)."""
    return _prefill("swa_prefill", desc, q, k, v, out, lse, k_ring, v_ring, stream)


def backward_workspace_bytes(desc: PbbDesc, n: int) -> int:
    out = ctypes.c_size_t()
    _check("pbb_backward_workspace_bytes", load_library().pbb_backward_workspace_bytes(
        ctypes.byref(desc), int(n), ctypes.byref(out)))
    return out.value


def _backward(fn: str, desc: PbbDesc, q, k, v, out, dout, lse, dq, dk, dv, workspace, stream):
    n = q.shape[1]
    for name, t in (("q", q), ("out", out), ("dout", dout), ("dq", dq)):
        _expect(name, t, (desc.batch, n, desc.n_q_heads, desc.head_dim), desc.torch_dtype)
    for name, t in (("k", k), ("v", v), ("dk", dk), ("dv", dv)):
        _expect(name, t, (desc.batch, n, desc.n_kv_heads, desc.head_dim), desc.torch_dtype)
    _expect("lse", lse, (desc.batch, desc.n_q_heads, n), torch.float32)
    if workspace is None:
        nbytes = max(1, backward_workspace_bytes(desc, n))
        workspace = _scratch_on(stream, lambda: torch.empty(nbytes, dtype=torch.uint8,
                                                            device=q.device))
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(fn, getattr(load_library(), fn)(
        ctypes.byref(desc), int(n), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), ctypes.c_size_t(ws_bytes), _stream(stream)))
    return dq, dk, dv


def pbb_backward(desc: PbbDesc, q, k, v, out, dout, lse, dq, dk, dv, workspace=None, stream=None):
    """Gradients (dq, dk, dv) of :func:`pbb_prefill`'s output for the upstream gradient
    ``dout``; ``out`` and ``lse`` are the prefill's outputs.  Allocates the workspace when none
    is given."""
    return _backward("pbb_backward", desc, q, k, v, out, dout, lse, dq, dk, dv, workspace, stream)


def swa_backward(desc: PbbDesc, q, k, v, out, dout, lse, dq, dk, dv, workspace=None, stream=None):
    """Sliding-window counterpart of :func:`pbb_backward`."""
    return _backward("swa_backward", desc, q, k, v, out, dout, lse, dq, dk, dv, workspace, stream)

