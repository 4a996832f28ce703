"""GPU: calls captured in a HIP graph and replayed, as a serving loop would.

Each case captures one call on fixed device buffers, then replays the graph
several times with new inputs copied into those buffers, with eager calls and
synchronisations between the replays.  Every replay must match an eager call
on the same inputs bit for bit and leave a clean device status word: the
per-call state of a launch (the overlapped launch's queues and ready flags,
the chunk index tables, the status word) is set up by kernels inside the
graph, not by the host, so each replay starts from it afresh.
"""

import numpy as np
import pytest

from gpu_harness import say, to_device
from paper_2609_32114_amd.inputs import make_case, make_decode_case

pytestmark = pytest.mark.gpu

CASES = [
    # kind, lengths, Hqk, Hv, D, dtype, segment chunks (0: automatic), overlap forced where it can run
    ("gdn", (1000,), 4, 16, 128, "bf16", 0, True),             # the overlapped launch
    ("gdn", (1000,), 4, 16, 128, "bf16", 0, False),            # chunk-local kernel, then the walk
    ("gdn", (700, 0, 1, 299), 2, 6, 128, "bf16", 3, False),    # chunk index, segment maps and walks
    ("kda", (900,), 2, 8, 128, "bf16", 3, False),
    ("gdn", (300, 500), 2, 4, 64, "f32", 0, False),
]


def _ids(c):
    return f"{c[0]}-N{len(c[1])}-Hv{c[3]}-d{c[4]}-{c[5]}-L{c[6]}{'-ovl' if c[7] else ''}"


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_prefill_graph_replays_match_eager(case):
    import torch
    import paper_2609_32114_amd as P
    kind, lengths, Hqk, Hv, D, dtype, L, ovl = case
    N, T = len(lengths), sum(lengths)
    sets = [to_device(make_case(kind, lengths, Hqk, Hv, D, D, dtype, with_s0=True, variant="s0", seed=s))
            for s in (11, 12, 13)]
    scale = 0.5
    fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
    code = P.HAGDN_BF16 if dtype == "bf16" else P.HAGDN_F32
    dt = sets[0]["q"].dtype
    say(f"graph {_ids(case)}")
    try:
        P.set_segment_chunks(L)
        P.set_overlap(True, force=ovl)
        assert P.overlap_for(N, T, Hv, D, D, code, kind) == (ovl and kind == "gdn" and dtype == "bf16")
        wsb = P.workspace_size(kind, N, T, Hqk, Hv, D, D, code)

        def call(d, ws, o, sf):
            fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"], cu_seqlens=d["cu"],
               scale=scale, workspace=ws, out=o, final_out=sf)

        # eager references, on a workspace of their own
        ws_e = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        refs = []
        for d in sets:
            o = torch.empty((T, Hv, D), dtype=dt, device="cuda")
            sf = torch.empty((N, Hv, D, D), dtype=torch.float32, device="cuda")
            call(d, ws_e, o, sf)
            torch.cuda.synchronize()
            assert P.device_status(ws_e) == P.DEV_OK
            refs.append((o.float().cpu().numpy(), sf.cpu().numpy()))

        # fixed buffers the graph reads and writes
        static = {k: v.clone() for k, v in sets[0].items()}
        ws_g = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        o_g = torch.empty((T, Hv, D), dtype=dt, device="cuda")
        sf_g = torch.empty((N, Hv, D, D), dtype=torch.float32, device="cuda")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            call(static, ws_g, o_g, sf_g)  # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            call(static, ws_g, o_g, sf_g)
        torch.cuda.synchronize()

        for rep, i in enumerate((1, 0, 2, 1, 2)):
            for key in static:
                static[key].copy_(sets[i][key])
            o_g.fill_(float("nan"))
            sf_g.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(o_g.float().cpu().numpy(), refs[i][0], err_msg=f"replay {rep} o")
            np.testing.assert_array_equal(sf_g.cpu().numpy(), refs[i][1], err_msg=f"replay {rep} s_final")
            assert P.device_status(ws_g) == P.DEV_OK
            # eager work on another workspace between replays
            o = torch.empty((T, Hv, D), dtype=dt, device="cuda")
            sf = torch.empty((N, Hv, D, D), dtype=torch.float32, device="cuda")
            call(sets[(i + 1) % 3], ws_e, o, sf)
            torch.cuda.synchronize()
        del graph
    finally:
        P.set_segment_chunks(0)
        P.set_overlap(True)


def test_decode_graph_replays_match_eager():
    """Decode steps captured once and replayed: each replay advances the pool
    in place exactly as an eager step does."""
    import torch
    import paper_2609_32114_amd as P
    dcs = [make_decode_case("gdn", N=9, Hqk=2, Hv=4, Dk=128, Dv=64, dtype="bf16", pool=20, pad=2, seed=s)
           for s in (21, 22)]
    t = lambda x, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(dt)
    ins = [dict(q=t(dc.q, torch.bfloat16), k=t(dc.k, torch.bfloat16), v=t(dc.v, torch.bfloat16), g=t(dc.g),
                beta=t(dc.beta), slots=t(dc.slots, torch.int32)) for dc in dcs]
    pool0 = t(dcs[0].state)
    say("graph decode")

    def step(d, pool, o):
        P.gdn_decode(d["q"], d["k"], d["v"], d["g"], d["beta"], pool, slots=d["slots"], scale=1.0, out=o)

    # eager: two steps with input set 0, then two with set 1, from pool0
    pool_e = pool0.clone()
    o_e = torch.empty((9, 4, 64), dtype=torch.bfloat16, device="cuda")
    ref = []
    for i in (0, 0, 1, 1):
        step(ins[i], pool_e, o_e)
        torch.cuda.synchronize()
        ref.append((o_e.float().cpu().numpy(), pool_e.cpu().numpy()))

    static = {k: v.clone() for k, v in ins[0].items()}
    pool_g = pool0.clone()
    o_g = torch.empty((9, 4, 64), dtype=torch.bfloat16, device="cuda")
    warm = pool0.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(static, warm, o_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(static, pool_g, o_g)
    torch.cuda.synchronize()
    pool_g.copy_(pool0)  # the capture itself ran nothing
    for rep, i in enumerate((0, 0, 1, 1)):
        for key in static:
            static[key].copy_(ins[i][key])
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(o_g.float().cpu().numpy(), ref[rep][0], err_msg=f"replay {rep} o")
        np.testing.assert_array_equal(pool_g.cpu().numpy(), ref[rep][1], err_msg=f"replay {rep} pool")
    del graph


def test_noalloc_graph_replays_match_eager():
    """The allocation-free entry point (its workspace is a library-held device
    array) captured and replayed; eager calls of it run between the replays."""
    import ctypes
    import torch
    import paper_2609_32114_amd as P
    lib = P.load_library()
    T, Hqk, Hv = 900, 4, 16
    sets = [to_device(make_case("gdn", (T,), Hqk, Hv, 128, 128, "bf16", with_s0=True, variant="s0", seed=s))
            for s in (31, 32)]
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())
    say("graph noalloc")

    def call(d, o, sf):
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        rc = lib.hagdn_prefill_noalloc(0, ptr(d["q"]), ptr(d["k"]), ptr(d["v"]), ptr(d["g"]), ptr(d["beta"]),
                                       ptr(d["s0"]), ptr(d["cu"]), 1, T, Hqk, Hv, 128, 128, ctypes.c_float(0.25),
                                       P.HAGDN_BF16, 0, ptr(o), ptr(sf), stream)
        assert rc == 0, P._err(lib)

    new = lambda: (torch.empty((T, Hv, 128), dtype=torch.bfloat16, device="cuda"),
                   torch.empty((1, Hv, 128, 128), dtype=torch.float32, device="cuda"))
    refs = []
    for d in sets:
        o, sf = new()
        call(d, o, sf)
        torch.cuda.synchronize()
        refs.append((o.float().cpu().numpy(), sf.cpu().numpy()))
    static = {k: v.clone() for k, v in sets[0].items()}
    o_g, sf_g = new()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(static, o_g, sf_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(static, o_g, sf_g)
    torch.cuda.synchronize()
    for rep, i in enumerate((1, 0, 1)):
        for key in static:
            static[key].copy_(sets[i][key])
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(o_g.float().cpu().numpy(), refs[i][0], err_msg=f"replay {rep} o")
        np.testing.assert_array_equal(sf_g.cpu().numpy(), refs[i][1], err_msg=f"replay {rep} s_final")
        o, sf = new()
        call(sets[1 - i], o, sf)  # eager call of the same entry point between replays
        torch.cuda.synchronize()
    del graph
