"""GPU parity for in-kernel preprocessing and the decode step, through the C ABI.

Preprocessing: the kernels take raw projections (q, k unnormalised, raw gate
and beta values) with HAGDN_PRE_* flags; the oracle applies the same maps in
fp64 and runs the recurrence.  Decode: one token per sequence updates a state
pool in place; the oracle runs the same step in fp64.  Tolerances are the
prefill ones (max |gpu - ref| / max |ref| per tensor: 1e-4 for fp32 inputs,
2e-2 for bf16 inputs).
"""

import numpy as np
import pytest

import oracle
from gpu_harness import TOL, nmse, oracle_threads, relerr, say, to_device
from paper_2609_32114_amd import inputs

pytestmark = pytest.mark.gpu

ALL = 7  # every preprocessing flag


def _torch():
    import torch
    return torch


def _run_prefill_pre(inp, pre):
    torch = _torch()
    import paper_2609_32114_amd as P
    d = to_device(inp)
    fn = P.gdn_prefill if inp.kind == "gdn" else P.kda_prefill
    o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"], cu_seqlens=d["cu"],
               scale=inp.scale, preprocess=pre)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), sf.cpu().numpy().astype(np.float64)


def _check(name, got, ref, tol):
    e = relerr(got, ref)
    say(f"       {name}: max-rel {e:.3e} nmse {nmse(got, ref):.3e}")
    assert np.all(np.isfinite(got)), name
    assert e <= tol, f"{name}: max-rel {e:.3e} > {tol}"


PRE_CASES = [
    # kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0, pre
    ("gdn", (256,), 1, 1, 64, 64, "f32", False, ALL),
    ("gdn", (200,), 2, 2, 128, 128, "bf16", False, ALL),
    ("gdn", (130,), 1, 1, 128, 64, "bf16", True, 1),
    ("gdn", (130,), 1, 1, 64, 128, "bf16", True, 2),
    ("gdn", (130,), 1, 1, 128, 128, "f32", True, 4),
    ("kda", (150,), 1, 2, 128, 128, "bf16", True, ALL),
    ("kda", (97,), 1, 1, 64, 64, "f32", False, ALL),
    ("gdn", (70, 0, 129, 1, 64), 2, 4, 128, 128, "bf16", True, ALL),
]


@pytest.mark.parametrize("case", PRE_CASES, ids=[f"{c[0]}-{c[6]}-pre{c[8]}-{i}" for i, c in enumerate(PRE_CASES)])
def test_prefill_preprocessing_matches_oracle(case):
    kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0, pre = case
    # raw draws for the flagged inputs, finished inputs for the others
    raw = inputs.make_case(kind=kind, lengths=lengths, Hqk=Hqk, Hv=Hv, Dk=Dk, Dv=Dv, dtype=dtype,
                           with_s0=s0, seed=77, raw=True)
    fin = inputs.make_case(kind=kind, lengths=lengths, Hqk=Hqk, Hv=Hv, Dk=Dk, Dv=Dv, dtype=dtype,
                           with_s0=s0, seed=77)
    if not pre & 1:
        raw.q, raw.k = fin.q, fin.k
    if not pre & 2:
        raw.g = fin.g
    if not pre & 4:
        raw.beta = fin.beta
    say(f"[gpu] prefill pre={pre} kind={kind} dtype={dtype} lengths={lengths} Hqk={Hqk} Hv={Hv} Dk={Dk} Dv={Dv}")
    o, sf = _run_prefill_pre(raw, pre)
    ro, rs = oracle.run_inputs(raw, nthreads=oracle_threads(), pre=pre)
    _check("o", o, ro, TOL[dtype])
    _check("s_final", sf, rs, TOL[dtype])


# the flagged chunk-local instance feeding the other chain kernels: the bf16
# segment maps (forced short segments) and the staged walk (more walks than
# compute units: 3 sequences x 12 heads x 8 column tiles = 320 walks)
PRE_CHAIN_CASES = [
    # kind, lengths, Hqk, Hv, segment chunks (0: automatic)
    ("kda", (700,), 2, 4, 3),
    ("gdn", (400, 130), 2, 4, 2),
    ("gdn", (130, 257, 64), 4, 12, 0),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", PRE_CHAIN_CASES, ids=[f"{c[0]}-L{c[4]}-{i}" for i, c in enumerate(PRE_CHAIN_CASES)])
def test_prefill_preprocessing_through_segments_and_staged_walk(case):
    import paper_2609_32114_amd as P
    kind, lengths, Hqk, Hv, L = case
    raw = inputs.make_case(kind=kind, lengths=lengths, Hqk=Hqk, Hv=Hv, Dk=128, Dv=128, dtype="bf16",
                           with_s0=True, seed=78, raw=True)
    say(f"[gpu] prefill pre={ALL} kind={kind} lengths={lengths} Hqk={Hqk} Hv={Hv} segment_chunks={L}")
    P.set_segment_chunks(L)
    try:
        o, sf = _run_prefill_pre(raw, ALL)
    finally:
        P.set_segment_chunks(0)
    ro, rs = oracle.run_inputs(raw, nthreads=oracle_threads(), pre=ALL)
    _check("o", o, ro, TOL["bf16"])
    _check("s_final", sf, rs, TOL["bf16"])


def test_prefill_preprocessing_workload1_sampled_heads():
    """Workload 1 (T=4096, H=16, d=128, bf16) from raw projections, every flag,
    in the launch configuration the benchmark times; heads 0 and 11 checked."""
    from gpu_harness import sub_heads
    raw = inputs.make_workload(1, raw=True)
    say("[gpu] workload 1 raw projections, pre=7, heads [0, 11]")
    o, sf = _run_prefill_pre(raw, ALL)
    heads = [0, 11]
    ro, rs = oracle.run_inputs(sub_heads(raw, heads), nthreads=oracle_threads(), pre=ALL)
    _check("o", o[:, heads], ro, TOL["bf16"])
    _check("s_final", sf[:, heads], rs, TOL["bf16"])


def _run_decode(di, pre=0, state_dev=None):
    torch = _torch()
    import paper_2609_32114_amd as P
    dt = torch.bfloat16 if di.dtype == "bf16" else torch.float32
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).cuda().to(d)
    st = state_dev if state_dev is not None else t(di.state)
    slots = None if di.slots is None else torch.from_numpy(di.slots.astype(np.int32)).cuda()
    fn = P.gdn_decode if di.kind == "gdn" else P.kda_decode
    o = fn(t(di.q, dt), t(di.k, dt), t(di.v, dt), t(di.g), t(di.beta), st, slots=slots,
           scale=di.scale, preprocess=pre)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), st


DEC_CASES = [
    # kind, N, Hqk, Hv, Dk, Dv, dtype, pool, pad, raw
    ("gdn", 1, 1, 1, 64, 64, "f32", None, 0, False),
    ("gdn", 5, 1, 2, 128, 128, "f32", None, 0, False),
    ("gdn", 9, 2, 4, 128, 64, "bf16", 13, 3, False),
    ("gdn", 7, 1, 1, 64, 128, "bf16", 7, 0, True),
    ("kda", 6, 1, 2, 128, 128, "f32", 10, 2, False),
    ("kda", 4, 2, 2, 64, 64, "bf16", None, 0, True),
    ("kda", 3, 1, 3, 128, 128, "bf16", 5, 1, True),
]


@pytest.mark.parametrize("case", DEC_CASES, ids=[f"{c[0]}-{c[6]}-N{c[1]}-{i}" for i, c in enumerate(DEC_CASES)])
def test_decode_matches_oracle(case):
    kind, N, Hqk, Hv, Dk, Dv, dtype, pool, pad, raw = case
    di = inputs.make_decode_case(kind=kind, N=N, Hqk=Hqk, Hv=Hv, Dk=Dk, Dv=Dv, dtype=dtype, pool=pool,
                                 pad=pad, seed=91, scale=0.5, raw=raw)
    pre = ALL if raw else 0
    say(f"[gpu] decode kind={kind} dtype={dtype} N={N} Hqk={Hqk} Hv={Hv} Dk={Dk} Dv={Dv} pool={pool} pad={pad} pre={pre}")
    o, st = _run_decode(di, pre)
    ro, rstate = oracle.decode(kind, di.q, di.k, di.v, di.g, di.beta, di.state, di.scale,
                               slots=di.slots, pre=pre, nthreads=oracle_threads())
    _check("o", o, ro, TOL[dtype])
    _check("state", st.cpu().numpy(), rstate, TOL[dtype])
    if di.slots is not None:  # padding rows are zero; untouched slots unchanged bit for bit
        assert np.all(o[di.slots < 0] == 0.0)
        used = set(int(s) for s in di.slots if s >= 0)
        for s in range(di.state.shape[0]):
            if s not in used:
                assert np.array_equal(st[s].cpu().numpy(), di.state[s]), f"slot {s} changed"


def test_decode_workload_full():
    """The decode workload the benchmark times (256 sequences, H=16, d=128, bf16), every output."""
    w = inputs.DECODE_WORKLOAD
    di = inputs.make_decode_case(kind=w["kind"], N=w["N"], Hqk=w["Hqk"], Hv=w["Hv"], Dk=w["Dk"],
                                 Dv=w["Dv"], dtype=w["dtype"], seed=5)
    say(f"[gpu] decode workload {w}")
    o, st = _run_decode(di)
    ro, rstate = oracle.decode(w["kind"], di.q, di.k, di.v, di.g, di.beta, di.state, di.scale,
                               nthreads=oracle_threads())
    _check("o", o, ro, TOL["bf16"])
    _check("state", st.cpu().numpy(), rstate, TOL["bf16"])


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_prefill_then_decode_continues_the_sequence(kind):
    """GPU prefill of T tokens, then K GPU decode steps from its final state,
    equals the oracle's prefill of T + K tokens (decoded outputs and the state)."""
    torch = _torch()
    import paper_2609_32114_amd as P
    N, T, K, Hqk, Hv, D = 3, 150, 4, 1, 2, 128
    full = inputs.make_case(kind=kind, lengths=(T + K,) * N, Hqk=Hqk, Hv=Hv, Dk=D, Dv=D, dtype="bf16",
                            variant="lm", seed=13)
    say(f"[gpu] prefill {T} + decode {K} kind={kind} N={N}")
    idx = lambda a, z: np.concatenate([np.arange(n * (T + K) + a, n * (T + K) + z) for n in range(N)])
    pre_idx = idx(0, T)
    sub = inputs.Inputs(kind=kind, dtype="bf16", q=full.q[pre_idx], k=full.k[pre_idx], v=full.v[pre_idx],
                        g=full.g[pre_idx], beta=full.beta[pre_idx], s0=None,
                        cu_seqlens=(np.arange(N + 1) * T).astype(np.int32))
    d = to_device(sub)
    fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
    _, state = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], cu_seqlens=d["cu"])
    outs = []
    for t in range(T, T + K):
        rows = np.arange(N) * (T + K) + t
        di = inputs.DecodeInputs(kind=kind, dtype="bf16", q=full.q[rows], k=full.k[rows], v=full.v[rows],
                                 g=full.g[rows], beta=full.beta[rows], state=None, slots=None)
        o, state = _run_decode(di, state_dev=state)
        outs.append(o)
    ro, rs = oracle.run_inputs(full, nthreads=oracle_threads())
    ref = np.stack([ro[np.arange(N) * (T + K) + t] for t in range(T, T + K)])
    _check("decoded o", np.stack(outs), ref, TOL["bf16"])
    _check("state", state.cpu().numpy(), rs, TOL["bf16"])
