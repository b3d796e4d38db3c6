"""GPU bounds checks of successful calls: every buffer a call may write (outputs, rings,
log-partitions, gradients, workspaces) is carved out of a larger allocation between two 4 KiB
guard zones of a fixed byte pattern, and every input is compared before and after.  A call
must leave the guard zones and its inputs bit for bit unchanged (no write outside its
buffers, no write to read-only arguments).  Shapes pick the launch variants: split and unsplit
bf16 decode, fp32 decode, SWA with a wrapping window, rotary decode, a prefill whose last tile
is partly empty, and the backward's two launches.
"""
from __future__ import annotations

import pytest
import torch

import paper_2606_02680_amd as P

pytestmark = pytest.mark.gpu

GUARD = 4096          # bytes on each side
PATTERN = 0xA5


class Guarded:
    """A tensor of ``shape`` inside a byte buffer with guard zones on both sides."""

    def __init__(self, shape, dtype, device, fill=None, nbytes=None):
        if nbytes is None:
            n = 1
            for s in shape:
                n *= s
            nbytes = n * torch.empty((), dtype=dtype).element_size()
        else:
            shape = None
        self.nbytes = nbytes
        self.raw = torch.full((GUARD + self.nbytes + GUARD,), PATTERN, dtype=torch.uint8,
                              device=device)
        body = self.raw[GUARD:GUARD + self.nbytes]
        self.t = body.view(dtype).view(shape) if shape is not None else body
        if fill is not None:
            self.t.copy_(fill)

    def intact(self) -> bool:
        return bool((self.raw[:GUARD] == PATTERN).all()) and \
            bool((self.raw[GUARD + self.nbytes:] == PATTERN).all())


def _randn(shape, dtype, device, gen):
    return torch.randn(shape, generator=gen, device=device).to(dtype)


def _decode_case(device, mode, dtype, batch, hq, hkv, d, B, pos_hi, rope=0.0, seed=0):
    gen = torch.Generator(device=device).manual_seed(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    if mode == "pbb":
        desc = P.make_desc(batch, hq, hkv, d, block=B, dtype=tdt, rope_base=rope)
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=B - 3, slots=B, dtype=tdt, rope_base=rope)
    pos = torch.randint(0, pos_hi, (batch,), generator=gen, device=device, dtype=torch.int32)
    q = _randn((batch, hq, d), tdt, device, gen)
    kn = _randn((batch, hkv, d), tdt, device, gen)
    vn = _randn((batch, hkv, d), tdt, device, gen)
    rings = [Guarded(P.ring_shape(desc), tdt, device,
                     fill=_randn(P.ring_shape(desc), tdt, device, gen)) for _ in range(2)]
    out = Guarded((batch, hq, d), tdt, device, fill=torch.zeros((batch, hq, d), dtype=tdt))
    wsb = P.swa_workspace_bytes(desc) if mode == "swa" else P.workspace_bytes(desc)
    ws = Guarded(None, torch.uint8, device, nbytes=wsb) if wsb else None
    if ws is not None:
        ws.t.zero_()
    inputs = [pos, q, kn, vn]
    before = [x.clone() for x in inputs]
    fn = P.swa_decode_step if mode == "swa" else P.pbb_decode_step
    print(f"[guard] decode {mode} {dtype} batch={batch} hq={hq} hkv={hkv} d={d} B={B} "
          f"rope={rope} workspace={wsb}", flush=True)
    for _ in range(3):   # a few steps: positions advance, split counters reset and are reused
        fn(desc, pos, q, kn, vn, rings[0].t, rings[1].t, out.t, None if ws is None else ws.t)
        pos += 1
        before[0] += 1
    torch.cuda.synchronize()
    for g in rings + [out] + ([ws] if ws is not None else []):
        assert g.intact()
    for x, y in zip(inputs, before):
        assert torch.equal(x.view(torch.uint8) if x.dtype != torch.int32 else x,
                           y.view(torch.uint8) if y.dtype != torch.int32 else y)


@pytest.mark.parametrize("mode,dtype,batch,hq,hkv,d,B,pos_hi,rope", [
    ("pbb", "bf16", 2, 32, 8, 128, 2048, 300000, 0.0),   # 16 units: split launch
    ("pbb", "bf16", 64, 16, 4, 64, 256, 5000, 0.0),      # 256 units: two waves per workgroup
    ("pbb", "f32", 3, 12, 2, 64, 128, 9000, 0.0),
    ("swa", "bf16", 40, 8, 8, 128, 100, 100000, 0.0),    # window wraps the ring
    ("pbb", "bf16", 5, 12, 2, 64, 128, 70000, 1e6),      # rotary, split
])
def test_decode_writes_only_its_buffers(cuda, mode, dtype, batch, hq, hkv, d, B, pos_hi, rope):
    _decode_case(cuda, mode, dtype, batch, hq, hkv, d, B, pos_hi, rope)


@pytest.mark.parametrize("mode,batch,n,hq,hkv,d,B", [
    ("pbb", 2, 1000, 12, 2, 64, 128),     # G = 6: the last tile is partly empty
    ("swa", 1, 777, 32, 8, 128, 300),
])
def test_prefill_and_backward_write_only_their_buffers(cuda, mode, batch, n, hq, hkv, d, B):
    gen = torch.Generator(device=cuda).manual_seed(1)
    bf = torch.bfloat16
    if mode == "pbb":
        desc = P.make_desc(batch, hq, hkv, d, block=B, dtype=bf)
        fwd, bwd = P.pbb_prefill, P.pbb_backward
    else:
        desc = P.make_desc(batch, hq, hkv, d, window=B, slots=B, dtype=bf)
        fwd, bwd = P.swa_prefill, P.swa_backward
    q = _randn((batch, n, hq, d), bf, cuda, gen)
    k = _randn((batch, n, hkv, d), bf, cuda, gen)
    v = _randn((batch, n, hkv, d), bf, cuda, gen)
    dout = _randn((batch, n, hq, d), bf, cuda, gen)
    ins = [q, k, v, dout]
    before = [x.clone() for x in ins]
    out = Guarded((batch, n, hq, d), bf, cuda)
    lse = Guarded((batch, hq, n), torch.float32, cuda)
    rings = [Guarded(P.ring_shape(desc), bf, cuda) for _ in range(2)]
    P.ring_init(desc, rings[0].t, rings[1].t)
    print(f"[guard] prefill {mode} batch={batch} n={n} hq={hq} hkv={hkv} d={d} B={B}", flush=True)
    fwd(desc, q, k, v, out.t, lse.t, rings[0].t, rings[1].t)
    torch.cuda.synchronize()
    for g in [out, lse] + rings:
        assert g.intact()
    grads = [Guarded(tuple(x.shape), bf, cuda) for x in (q, k, v)]
    ws = Guarded(None, torch.uint8, cuda, nbytes=P.backward_workspace_bytes(desc, n))
    out_before, lse_before = out.t.clone(), lse.t.clone()
    print(f"[guard] backward {mode}", flush=True)
    bwd(desc, q, k, v, out.t, dout, lse.t, grads[0].t, grads[1].t, grads[2].t, ws.t)
    torch.cuda.synchronize()
    for g in grads + [ws]:
        assert g.intact()
    assert torch.equal(out.t.view(torch.int16), out_before.view(torch.int16))
    assert torch.equal(lse.t, lse_before)
    for x, y in zip(ins, before):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
