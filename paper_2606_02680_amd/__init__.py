"""MI355X-native Post-Boundary Bridge (PBB) decode attention.

The product is ``libpbb.so`` (C ABI in ``include/pbb.h``, HIP kernels for gfx950 in
``csrc/``); :mod:`paper_2606_02680_amd.pbb` is its thin ctypes binding.
"""
from .pbb import (  # noqa: F401
    PbbDesc, PbbError, alloc_rings, alloc_workspace, backward_workspace_bytes, load_library,
    make_desc, pbb_backward, pbb_decode_step, pbb_decode_step_advance, pbb_decode_step_noalloc,
    pbb_prefill, ring_bytes,
    ring_fill, ring_init, ring_shape, swa_backward, swa_decode_step, swa_decode_step_advance, swa_prefill,
    swa_workspace_bytes, workspace_bytes)
