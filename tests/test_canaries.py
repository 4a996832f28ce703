"""GPU: no kernel writes outside the buffers it is given.

Every output (o, s_final, the decode state pool and output) and the workspace
sit inside a larger allocation whose guard zones before and after are filled
with a byte pattern; after the call the guards must be intact.  The cases
reach every launch path: the overlapped launch, the serialized four-wave walk,
the staged walk (more walks than CUs), the segment maps and segment walks
(bf16 and fp32 maps), fp32 with d = 64, the allocation-free entry point and
decode over a slot-addressed pool.
"""

import numpy as np
import pytest

from gpu_harness import say, to_device
from paper_2609_32114_amd.inputs import make_case, make_decode_case

pytestmark = pytest.mark.gpu

GUARD = 4096
PATTERN = 0xA5


def _guarded(nbytes, dtype, shape):
    """A tensor of `shape` inside a uint8 allocation with GUARD pattern bytes on both sides."""
    import torch
    raw = torch.full((GUARD + nbytes + GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
    body = raw[GUARD:GUARD + nbytes]
    t = body.view(dtype).view(shape) if shape is not None else body
    return raw, t


def _guards_intact(raw, nbytes):
    h = raw.cpu().numpy()
    return bool(np.all(h[:GUARD] == PATTERN) and np.all(h[GUARD + nbytes:] == PATTERN))


CASES = [
    # kind, lengths, Hqk, Hv, D, dtype, segment chunks (0: automatic), overlap forced where it can run
    ("gdn", (1000,), 4, 16, 128, "bf16", 0, True),          # overlapped launch
    ("gdn", (1000,), 4, 16, 128, "bf16", 0, False),         # serialized four-wave walk (too short to overlap)
    ("gdn", (300, 0, 1, 777), 12, 12, 128, "bf16", 0, True),  # staged walk: 384 walks
    ("kda", (1000,), 2, 8, 128, "bf16", 3, True),           # bf16 segment maps + segment walks
    ("gdn", (700, 65), 2, 6, 64, "f32", 4, True),           # fp32 maps, d = 64
    ("kda", (129,), 1, 3, 64, "f32", 0, True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-N{len(c[1])}-Hv{c[3]}-d{c[4]}-{c[5]}-L{c[6]}"
                         f"{'-ovl' if c[7] else ''}")
def test_prefill_writes_stay_inside_buffers(case):
    import torch
    import paper_2609_32114_amd as P
    kind, lengths, Hqk, Hv, D, dtype, L, ovl = case
    inp = make_case(kind, lengths, Hqk, Hv, D, D, dtype, with_s0=True, variant="s0", seed=5)
    d = to_device(inp)
    N, T = len(lengths), sum(lengths)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    esz = 2 if dtype == "bf16" else 4
    try:
        P.set_segment_chunks(L)
        P.set_overlap(True, force=ovl)
        code = P.HAGDN_BF16 if dtype == "bf16" else P.HAGDN_F32
        wsb = P.workspace_size(kind, N, T, Hqk, Hv, D, D, code)
        ws_raw, ws = _guarded(wsb, torch.uint8, None)
        o_raw, o = _guarded(T * Hv * D * esz, dt, (T, Hv, D))
        s_raw, sf = _guarded(N * Hv * D * D * 4, torch.float32, (N, Hv, D, D))
        fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
        say(f"canaries {case}")
        fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"], cu_seqlens=d["cu"],
           scale=inp.scale, workspace=ws, out=o, final_out=sf)
        torch.cuda.synchronize()
    finally:
        P.set_segment_chunks(0)
        P.set_overlap(True)
    assert _guards_intact(ws_raw, wsb), "workspace guard overwritten"
    assert _guards_intact(o_raw, T * Hv * D * esz), "output guard overwritten"
    assert _guards_intact(s_raw, N * Hv * D * D * 4), "final-state guard overwritten"
    assert P.device_status(ws) == P.DEV_OK


def test_noalloc_writes_stay_inside_outputs():
    import ctypes
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (900,), 4, 16, 128, 128, "bf16", with_s0=True, variant="s0", seed=6)
    d = to_device(inp)
    T, Hv = 900, 16
    o_raw, o = _guarded(T * Hv * 128 * 2, torch.bfloat16, (T, Hv, 128))
    s_raw, sf = _guarded(Hv * 128 * 128 * 4, torch.float32, (1, Hv, 128, 128))
    lib = P.load_library()
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.hagdn_prefill_noalloc(0, ptr(d["q"]), ptr(d["k"]), ptr(d["v"]), ptr(d["g"]), ptr(d["beta"]),
                                   ptr(d["s0"]), ptr(d["cu"]), 1, T, 4, Hv, 128, 128, ctypes.c_float(inp.scale),
                                   P.HAGDN_BF16, 0, ptr(o), ptr(sf), stream)
    assert rc == 0, P._err(lib)
    torch.cuda.synchronize()
    assert _guards_intact(o_raw, T * Hv * 128 * 2)
    assert _guards_intact(s_raw, Hv * 128 * 128 * 4)


def test_decode_writes_stay_inside_buffers():
    import torch
    import paper_2609_32114_amd as P
    dc = make_decode_case("gdn", N=9, Hqk=2, Hv=4, Dk=128, Dv=64, dtype="bf16", pool=20, pad=2, seed=7)
    t = lambda x, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(dt)
    q, k, v = t(dc.q, torch.bfloat16), t(dc.k, torch.bfloat16), t(dc.v, torch.bfloat16)
    pool_bytes = 20 * 4 * 128 * 64 * 4
    p_raw, pool = _guarded(pool_bytes, torch.float32, (20, 4, 128, 64))
    pool.copy_(t(dc.state))
    o_raw, o = _guarded(9 * 4 * 64 * 2, torch.bfloat16, (9, 4, 64))
    P.gdn_decode(q, k, v, t(dc.g), t(dc.beta), pool, slots=t(dc.slots, torch.int32), scale=1.0, out=o)
    torch.cuda.synchronize()
    assert _guards_intact(p_raw, pool_bytes)
    assert _guards_intact(o_raw, 9 * 4 * 64 * 2)
