"""GPU: the allocation-free entry point hagdn_prefill_noalloc (workspace in the
library's static device array) against the workspace entry points
gdn_prefill_ex / kda_prefill_ex, called through the C ABI: two calls in a
row, the second on a smaller input, must match the workspace calls bit for
bit (the same kernels on the same inputs), and a call too large for the
array is refused before anything runs."""

import ctypes

import numpy as np
import pytest

from gpu_harness import say, to_device
from paper_2609_32114_amd.inputs import make_case

pytestmark = pytest.mark.gpu


def _noalloc(lib, kind, d, inp, pre=0):
    import torch
    T, Hqk, Dk = inp.q.shape
    Hv, Dv = inp.v.shape[1:]
    N = inp.N
    dt = 1 if inp.dtype == "bf16" else 0
    o = torch.full((T, Hv, Dv), float("nan"), dtype=d["q"].dtype, device="cuda")
    sf = torch.full((N, Hv, Dk, Dv), float("nan"), dtype=torch.float32, device="cuda")
    p = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.hagdn_prefill_noalloc(int(kind == "kda"), p(d["q"]), p(d["k"]), p(d["v"]), p(d["g"]),
                                   p(d["beta"]), p(d["s0"]), p(d["cu"]), N, T, Hqk, Hv, Dk, Dv,
                                   float(inp.scale), dt, pre, p(o), p(sf), stream)
    torch.cuda.synchronize()
    return rc, o, sf


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_noalloc_matches_workspace_entry_point(kind):
    import torch
    import paper_2609_32114_amd as P
    lib = P.load_library()
    cases = [make_case(kind, (1000, 300, 777), 2, 4, 128, 128, "bf16", with_s0=True, variant="lm", seed=71),
             make_case(kind, (129, 5), 1, 2, 64, 128, "bf16", with_s0=True, variant="lm", seed=72)]
    for i, inp in enumerate(cases):   # the second call is smaller than the first
        say(f"[gpu] noalloc {kind} call {i}: lengths {inp.meta['lengths']} q {inp.q.shape} v {inp.v.shape}")
        d = to_device(inp)
        rc, o, sf = _noalloc(lib, kind, d, inp)
        assert rc == 0, lib.hagdn_last_error().decode()
        fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
        o_ref, s_ref = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                          cu_seqlens=d["cu"], scale=inp.scale)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(o.float().cpu().numpy(), o_ref.float().cpu().numpy())
        np.testing.assert_array_equal(sf.cpu().numpy(), s_ref.cpu().numpy())


def test_noalloc_refuses_calls_beyond_its_array():
    import paper_2609_32114_amd as P
    lib = P.load_library()
    cap = lib.hagdn_prefill_noalloc_capacity()
    assert cap == 128 << 20
    assert P.workspace_size("gdn", 1, 4096, 16, 16, 128, 128, P.HAGDN_BF16) <= cap
    big = P.workspace_size("gdn", 1, 8192, 16, 16, 128, 128, P.HAGDN_BF16)
    assert big > cap
    f = ctypes.c_void_p(0x100000)   # never dereferenced: the size check comes first
    rc = lib.hagdn_prefill_noalloc(0, f, f, f, f, f, None, f, 1, 8192, 16, 16, 128, 128, 1.0, 1, 0,
                                   f, None, None)
    assert rc == 3 and "workspace" in lib.hagdn_last_error().decode()
