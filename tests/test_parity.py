"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small cases compare every element and span several 64-token chunks with
ragged tails; the full-size workloads run in the benchmark's launch
configuration and compare every head.  Tolerance: max|gpu - oracle| /
max|oracle| <= 1e-4 (fp32 inputs), <= 2e-2 (bf16 inputs).
"""

import numpy as np
import pytest

from gpu_harness import TOL, check_against_oracle, run_gpu, say, to_device
from paper_2609_32114_amd.inputs import make_case, make_workload

pytestmark = pytest.mark.gpu


def test_workload0_full():
    check_against_oracle(make_workload(0), label="workload0")


SMALL = [
    # kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0
    ("gdn", (1,), 1, 1, 64, 64, "f32", True),
    ("gdn", (63,), 1, 2, 64, 64, "f32", True),
    ("gdn", (65,), 2, 2, 128, 128, "f32", True),
    ("gdn", (200,), 2, 2, 128, 128, "bf16", True),
    ("gdn", (130,), 1, 1, 64, 128, "bf16", False),
    ("gdn", (130,), 1, 1, 128, 64, "f32", True),
    ("gdn", (129,), 2, 4, 128, 128, "bf16", True),
    ("kda", (1,), 1, 1, 64, 64, "f32", True),
    ("kda", (200,), 1, 2, 64, 64, "f32", True),
    ("kda", (200,), 2, 2, 128, 128, "bf16", True),
    ("kda", (130,), 1, 2, 128, 64, "bf16", False),
    ("kda", (97,), 2, 4, 64, 128, "f32", True),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"{c[0]}-T{sum(c[1])}-h{c[2]}x{c[3]}-d{c[4]}x{c[5]}-{c[6]}")
def test_small_shapes(case):
    kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0 = case
    inp = make_case(kind, lengths, Hqk, Hv, Dk, Dv, dtype, with_s0=s0, seed=7)
    check_against_oracle(inp, label="small")


@pytest.mark.parametrize("kind", ["gdn", "kda"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_varlen_small(kind, dtype):
    inp = make_case(kind, (0, 1, 64, 65, 130, 7, 0, 200), 2, 4, 128, 128, dtype, with_s0=True,
                    seed=11)
    check_against_oracle(inp, label="varlen")


@pytest.mark.parametrize("variant", ["lm", "dn", "ks", "s0", "lg", "fg"])
def test_stress_variants_small(variant):
    for kind in ("gdn", "kda"):
        inp = make_case(kind, (300,), 1, 2, 128, 128, "bf16", variant=variant, seed=21)
        check_against_oracle(inp, label=f"stress-{variant}")
        inp = make_case(kind, (300,), 1, 2, 64, 64, "f32", variant=variant, seed=22)
        check_against_oracle(inp, label=f"stress-{variant}")


FORGET = [
    # kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0
    ("kda", (200,), 1, 2, 128, 128, "bf16", True),
    ("kda", (200,), 1, 2, 128, 128, "f32", True),
    ("kda", (130, 1, 97), 2, 4, 64, 128, "bf16", True),
    ("kda", (150,), 1, 1, 128, 64, "f32", False),
    ("kda", (65,), 1, 1, 64, 64, "f32", True),
    ("gdn", (200,), 1, 2, 128, 128, "bf16", True),
    ("gdn", (130,), 1, 1, 64, 64, "f32", True),
]


@pytest.mark.parametrize("case", FORGET, ids=lambda c: f"{c[0]}-T{sum(c[1])}-d{c[4]}x{c[5]}-{c[6]}")
def test_forget_runs_small(case):
    """Runs of 8-24 tokens with g = -30 (a gate of ~1e-13) on a quarter of the
    key channels (KDA) or on the scalar gate (GDN): KDA's factored decay of
    operator #2 would overflow there; the exact path must match the oracle."""
    kind, lengths, Hqk, Hv, Dk, Dv, dtype, s0 = case
    inp = make_case(kind, lengths, Hqk, Hv, Dk, Dv, dtype, with_s0=s0, variant="fg", seed=23)
    check_against_oracle(inp, label="forget-runs")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_forget_runs_workload3_shape(dtype):
    """Workload 3's shape (KDA, 8192 tokens, 16 heads, d = 128; segments of 8
    chunks in bf16) with forget runs, every head."""
    inp = make_case("kda", (8192,), 16, 16, 128, 128, dtype, variant="fg", seed=1003)
    check_against_oracle(inp, label=f"workload3-fg-{dtype}")


def test_forget_runs_workload1_shape():
    inp = make_workload(1, variant="fg")
    check_against_oracle(inp, label="workload1-fg")


@pytest.mark.parametrize("case", [
    ("gdn", (1000, 700, 1300), 4, 12, 128, 128, "bf16", 2),   # 48 segments x 12 heads
    ("kda", (3000,), 4, 20, 128, 128, "bf16", 1),             # 47 segments x 20 heads
    ("gdn", (900, 0, 450), 2, 6, 128, 64, "bf16", 2),         # one workgroup per map (d_k != d_v)
    ("kda", (700, 300), 3, 9, 64, 64, "f32", 2),              # fp32 maps
], ids=lambda c: f"{c[0]}-N{len(c[1])}-Hv{c[3]}-d{c[4]}x{c[5]}-{c[6]}-L{c[7]}")
def test_inplace_state_on_segments(case):
    """s_final aliasing s0 on the segmented path, with more segment workgroups
    than CUs and Hv not a multiple of 8: the first segment's state walk must
    not see the last segment's s_final.  Bitwise equal to the call with a
    separate s_final, and within tolerance of the oracle."""
    import torch
    import paper_2609_32114_amd as P
    kind, lengths, Hqk, Hv, Dk, Dv, dtype, L = case
    inp = make_case(kind, lengths, Hqk, Hv, Dk, Dv, dtype, with_s0=True, variant="s0", seed=29)
    fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
    try:
        P.set_segment_chunks(L)
        check_against_oracle(inp, label=f"segments-L{L}")
        d = to_device(inp)
        o_ref, s_ref = run_gpu(inp, dev=d)
        state = d["s0"].clone()
        o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=state,
                   cu_seqlens=d["cu"], scale=inp.scale, final_out=state)
        torch.cuda.synchronize()
    finally:
        P.set_segment_chunks(0)
    assert sf.data_ptr() == state.data_ptr()
    np.testing.assert_array_equal(state.cpu().numpy(), s_ref.astype(np.float32))
    np.testing.assert_array_equal(o.float().cpu().numpy(), o_ref.astype(np.float32))


def test_binding_checks_caller_buffers():
    """Buffers the caller hands in are checked before their pointers reach a
    kernel: device, dtype, shape and layout."""
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (100,), 1, 2, 64, 64, "bf16", with_s0=True, seed=2)
    d = to_device(inp)
    args = (d["q"], d["k"], d["v"], d["g"], d["beta"])
    bad_out = [torch.empty((100, 2, 64), dtype=torch.bfloat16),                     # host memory
               torch.empty((100, 2, 64), dtype=torch.float32, device="cuda"),       # wrong dtype
               torch.empty((99, 2, 64), dtype=torch.bfloat16, device="cuda"),       # too small
               torch.empty((100, 64, 2), dtype=torch.bfloat16, device="cuda").transpose(1, 2)]
    for o in bad_out:
        with pytest.raises((ValueError, TypeError)):
            P.gdn_prefill(*args, initial_state=d["s0"], cu_seqlens=d["cu"], out=o)
    good = torch.empty((1, 2, 64, 64), dtype=torch.float32, device="cuda")
    for sf in [good.cpu(), good.to(torch.bfloat16), good[:, :1], good.transpose(2, 3)]:
        with pytest.raises((ValueError, TypeError)):
            P.gdn_prefill(*args, initial_state=d["s0"], cu_seqlens=d["cu"], final_out=sf)
    for s0 in [d["s0"].cpu(), d["s0"].to(torch.bfloat16), d["s0"][:, :1]]:
        with pytest.raises((ValueError, TypeError)):
            P.gdn_prefill(*args, initial_state=s0, cu_seqlens=d["cu"])
    with pytest.raises(ValueError):
        P.gdn_prefill(*args, cu_seqlens=d["cu"], workspace=torch.empty(1 << 24, dtype=torch.uint8))
    with pytest.raises((ValueError, TypeError)):
        P.gdn_prefill(*args, cu_seqlens=d["cu"].cpu())
    # decode: out checked like the prefill output
    dq = d["q"][:3].contiguous()
    pool = torch.zeros((3, 2, 64, 64), dtype=torch.float32, device="cuda")
    dargs = (dq, d["k"][:3].contiguous(), d["v"][:3].contiguous(), d["g"][:3].contiguous(),
             d["beta"][:3].contiguous(), pool)
    for o in [torch.empty((3, 2, 64), dtype=torch.bfloat16), torch.empty((3, 2, 64), device="cuda"),
              torch.empty((2, 2, 64), dtype=torch.bfloat16, device="cuda")]:
        with pytest.raises((ValueError, TypeError)):
            P.gdn_decode(*dargs, out=o)
    # the checks pass for well-formed buffers
    o = torch.empty((100, 2, 64), dtype=torch.bfloat16, device="cuda")
    P.gdn_prefill(*args, initial_state=d["s0"], cu_seqlens=d["cu"], out=o, final_out=good)
    torch.cuda.synchronize()


def test_scale_and_inplace_state():
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (150,), 1, 2, 128, 128, "bf16", with_s0=True, seed=3,
                    scale=128 ** -0.5)
    check_against_oracle(inp, label="scale")
    d = to_device(inp)
    o_ref, s_ref = run_gpu(inp)
    state = d["s0"].clone()
    o, sf = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=state,
                          cu_seqlens=d["cu"], scale=inp.scale, final_out=state)
    torch.cuda.synchronize()
    assert sf.data_ptr() == state.data_ptr()
    np.testing.assert_array_equal(state.cpu().numpy(), s_ref.astype(np.float32))
    np.testing.assert_array_equal(o.float().cpu().numpy(), o_ref.astype(np.float32))


def test_no_final_state_and_zero_state():
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("kda", (90,), 1, 1, 64, 64, "f32", seed=4)
    d = to_device(inp)
    o, sf = P.kda_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], cu_seqlens=d["cu"],
                          output_final_state=False)
    torch.cuda.synchronize()
    assert sf is None
    o_ref, _ = run_gpu(inp)
    np.testing.assert_array_equal(o.float().cpu().numpy(), o_ref.astype(np.float32))


def test_empty_batch_returns_initial_state():
    import torch
    import paper_2609_32114_amd as P
    for kind in ("gdn", "kda"):
        inp = make_case(kind, (0, 0), 1, 2, 64, 64, "bf16", with_s0=True, seed=5)
        d = to_device(inp)
        fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
        o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                   cu_seqlens=d["cu"])
        torch.cuda.synchronize()
        assert o.shape[0] == 0
        np.testing.assert_array_equal(sf.cpu().numpy(), inp.s0)


def test_bad_seqlens_are_reported_not_faulted():
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (100, 50), 1, 1, 64, 64, "f32", with_s0=True, seed=6)
    d = to_device(inp)
    ws = torch.zeros(P.workspace_size("gdn", 2, 150, 1, 1, 64, 64, P.HAGDN_F32),
                     dtype=torch.uint8, device="cuda")
    for bad in ([0, 120, 100], [5, 100, 150], [0, 100, 149]):   # decreasing, cu[0]!=0, cu[N]!=T
        cu = torch.tensor(bad, dtype=torch.int32, device="cuda")
        o = torch.full((150, 1, 64), 7.0, device="cuda")
        o, sf = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                              cu_seqlens=cu, workspace=ws, out=o)
        assert P.device_status(ws) == P.DEV_BAD_SEQLENS
        np.testing.assert_array_equal(sf.cpu().numpy(), inp.s0)
        assert torch.all(o == 7.0)
    o, sf = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                          cu_seqlens=d["cu"], workspace=ws)
    assert P.device_status(ws) == P.DEV_OK


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_bad_seqlens_single_sequence(kind):
    """One sequence with malformed cu_seqlens: the kernels take its chunk
    bounds from T, and the status word must still keep every write out."""
    import torch
    import paper_2609_32114_amd as P
    inp = make_case(kind, (300,), 1, 2, 128, 128, "bf16", with_s0=True, seed=16)
    d = to_device(inp)
    fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
    ws = torch.zeros(P.workspace_size(kind, 1, 300, 1, 2, 128, 128, P.HAGDN_BF16), dtype=torch.uint8,
                     device="cuda")
    for bad in ([0, 299], [3, 300]):
        cu = torch.tensor(bad, dtype=torch.int32, device="cuda")
        o = torch.full((300, 2, 128), 7.0, dtype=torch.bfloat16, device="cuda")
        o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"], cu_seqlens=cu,
                   workspace=ws, out=o)
        assert P.device_status(ws) == P.DEV_BAD_SEQLENS
        np.testing.assert_array_equal(sf.cpu().numpy(), inp.s0)
        assert torch.all(o == 7.0)
    check_against_oracle(inp, label="after bad seqlens")


@pytest.mark.parametrize("case", [
    ("gdn", (1000, 333), 2, 4),          # four-wave walk
    ("gdn", (300, 200, 150), 8, 16),     # staged walk, two tiles per workgroup
    ("kda", (130, 70, 200, 65), 8, 40),  # staged walk, four tiles per workgroup
], ids=lambda c: f"{c[0]}-N{len(c[1])}-Hv{c[3]}")
def test_bitwise_deterministic(case):
    kind, lengths, Hqk, Hv = case
    inp = make_case(kind, lengths, Hqk, Hv, 128, 128, "bf16", with_s0=True, seed=8)
    d = to_device(inp)
    a = run_gpu(inp, dev=d)
    b = run_gpu(inp, dev=d)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


# ------------------------------------------------------------ full-size workloads
# Every head of every full-size call is compared: the oracle runs the whole
# workload (a few seconds on the host's cores).

@pytest.mark.parametrize("idx", [1, 2, 3, 4])
def test_workload_full_size(idx):
    inp = make_workload(idx)
    check_against_oracle(inp, label=f"workload{idx}")


@pytest.mark.parametrize("variant", ["lm", "dn", "ks", "s0"])
def test_workload1_shape_stress(variant):
    inp = make_workload(1, variant=variant)
    check_against_oracle(inp, label=f"workload1-{variant}")


@pytest.mark.parametrize("variant", ["lm", "lg"])
def test_workload3_shape_stress(variant):
    inp = make_workload(3, variant=variant)
    check_against_oracle(inp, label=f"workload3-{variant}")


@pytest.mark.parametrize("variant", ["dn", "s0"])
def test_workload2_shape_stress(variant):
    inp = make_workload(2, variant=variant)
    check_against_oracle(inp, label=f"workload2-{variant}")


@pytest.mark.parametrize("variant", ["lm", "dn", "ks"])
def test_workload4_shape_stress(variant):
    """Workload 4's shape (2048 walks: the staged walk, four tiles per
    workgroup) with gates that carry the state across every chunk."""
    inp = make_workload(4, variant=variant)
    check_against_oracle(inp, label=f"workload4-{variant}")


# More walk workgroups than CUs (N x Hv x Dv/16 > 256): bf16 chains take the
# staged walk, two or four column tiles per workgroup.
# Long-memory gates so that the state carries across every chunk; the oracle
# checks every head.
MANY_WALKS = [
    # kind, lengths, Hqk, Hv, Dk, Dv
    ("gdn", (300, 200, 150), 8, 16, 128, 128),
    ("kda", (300, 200, 150), 8, 16, 128, 128),
    ("gdn", (130, 0, 260, 64, 1), 4, 16, 64, 64),
    ("kda", (200, 129), 2, 40, 128, 64),
    ("gdn", (129, 200), 8, 40, 64, 128),
    # a single sequence with more walks than CUs (its own kernel instances)
    ("gdn", (700,), 8, 48, 128, 128),
    ("kda", (300,), 4, 40, 128, 128),
    # more than twice as many walks as CUs: four tiles per walk workgroup
    ("kda", (130, 70, 200, 65), 8, 40, 128, 128),
    ("gdn", (300,), 8, 96, 128, 128),
    ("gdn", (100, 37), 4, 80, 64, 64),
    ("kda", (90, 40), 4, 96, 64, 64),
    ("kda", (150,), 2, 40, 64, 128),
    ("kda", (200,), 4, 80, 128, 128),
    # more than four walks per CU
    ("gdn", (150,), 8, 160, 128, 128),
    ("gdn", (90, 60), 4, 80, 64, 128),
]


@pytest.mark.parametrize("case", MANY_WALKS, ids=lambda c: f"{c[0]}-N{len(c[1])}-Hv{c[3]}-d{c[4]}x{c[5]}")
def test_many_walks(case):
    kind, lengths, Hqk, Hv, Dk, Dv = case
    assert len(lengths) * Hv * (Dv // 16) > 256
    inp = make_case(kind, lengths, Hqk, Hv, Dk, Dv, "bf16", with_s0=True, variant="lm", seed=31)
    check_against_oracle(inp, label="many-walks")


@pytest.mark.parametrize("forced", [0, 32])
def test_output_beyond_2gib(forced):
    """A single sequence whose output exceeds 2 GiB (T = 32832 tokens x 128
    value heads x d_v = 128, fp32).  The automatic choice would walk the chain
    whole (1024 walk workgroups), but the segment length is capped so that one
    segment's output rows stay below 2 GiB (511 chunks here): the call takes
    the segmented path with two segments and no byte offset overflows.  A
    forced L = 32 covers many segments at this size.  Inputs are drawn on the
    GPU (seeded); the oracle checks the last head and one in the middle."""
    import torch
    import oracle
    import paper_2609_32114_amd as P
    from gpu_harness import oracle_threads, relerr
    T, Hqk, Hv, D = 32832, 1, 128, 128
    assert T * Hv * D * 4 > 2 ** 31
    gen = torch.Generator(device="cuda").manual_seed(41)
    q = torch.nn.functional.normalize(torch.randn(T, Hqk, D, device="cuda", generator=gen), dim=-1)
    k = torch.nn.functional.normalize(torch.randn(T, Hqk, D, device="cuda", generator=gen), dim=-1)
    v = torch.randn(T, Hv, D, device="cuda", generator=gen)
    g = -0.01 * torch.nn.functional.softplus(torch.randn(T, Hv, device="cuda", generator=gen))
    beta = torch.sigmoid(torch.randn(T, Hv, device="cuda", generator=gen))
    try:
        P.set_segment_chunks(forced)
        L = P.segment_chunks(1, T, Hv, D, torch.float32)
        assert L == (forced or 511) and 64 * L * Hv * D * 4 < 2 ** 31
        say(f"[gpu] o beyond 2 GiB: T={T} Hv={Hv} fp32 forced={forced} L={L}")
        o, sf = P.gdn_prefill(q, k, v, g, beta)
        torch.cuda.synchronize()
    finally:
        P.set_segment_chunks(0)
    heads = [Hv // 2, Hv - 1]
    ro, rs = oracle.prefill("gdn", q.cpu().numpy(), k.cpu().numpy(), v[:, heads].cpu().numpy(),
                            g[:, heads].cpu().numpy(), beta[:, heads].cpu().numpy(),
                            nthreads=oracle_threads())
    eo = relerr(o[:, heads].cpu().numpy(), ro)
    es = relerr(sf[:, heads].cpu().numpy(), rs)
    say(f"       max-rel o={eo:.3e} s={es:.3e}")
    assert eo <= 1e-4 and es <= 1e-4


def test_accuracy_protocol_nmse():
    """The paper's accuracy protocol (Sec. 7.4, "Accuracy"): the maximum NMSE
    of outputs and of final states over many GDN instances against a CPU fp64
    reference.  96 seeded instances (lengths 1-700, 1-4 value heads, every
    (d_k, d_v) pair, with and without s0, base / long-memory / DeltaNet-limit
    gates), bf16 and fp32.  NMSE = sum (x - ref)^2 / sum ref^2 per tensor.
    Bounds: fp32 1e-9, bf16 1e-4 (the measured maxima are printed; bf16
    rounding alone gives about 1e-6 per element)."""
    import gpu_harness as H
    rng = np.random.Generator(np.random.PCG64(926))
    worst = {}
    for i in range(96):
        dtype = "bf16" if i % 2 else "f32"
        Dk, Dv = [(64, 64), (64, 128), (128, 64), (128, 128)][(i // 2) % 4]
        Hqk = int(rng.integers(1, 3))
        Hv = Hqk * int(rng.integers(1, 3))
        T = int(rng.integers(1, 700, endpoint=True))
        variant = ["base", "lm", "dn"][i % 3]
        inp = make_case("gdn", (T,), Hqk, Hv, Dk, Dv, dtype, with_s0=bool(i % 4 < 2),
                        variant=variant, seed=5000 + i)
        n0 = len(H.RESULTS)
        check_against_oracle(inp, label=f"nmse-{i}")
        _, _, _, _, _, no, ns = H.RESULTS[n0]
        w = worst.setdefault(dtype, [0.0, 0.0])
        w[0], w[1] = max(w[0], no), max(w[1], ns)
    summary = "  ".join(f"{dt}: max NMSE o {w[0]:.2e} s {w[1]:.2e}" for dt, w in sorted(worst.items()))
    say(f"[accuracy] 96 GDN instances vs fp64 oracle -- {summary} "
        f"(paper, FP16 on Ascend: o 5.23e-8, s 9.38e-12)")
    assert worst["f32"][0] <= 1e-9 and worst["f32"][1] <= 1e-9
    assert worst["bf16"][0] <= 1e-4 and worst["bf16"][1] <= 1e-4


def test_zz_parity_summary():
    """One line over every oracle comparison this process made (run last in
    this file): worst max-rel and NMSE per dtype, all within tolerance."""
    import gpu_harness as H
    if not H.RESULTS:
        pytest.skip("no comparisons in this process")
    by = {}
    for label, dt, kind, eo, es, no, ns in H.RESULTS:
        b = by.setdefault(dt, [0, 0.0, 0.0, 0.0, 0.0])
        b[0] += 1
        b[1], b[2] = max(b[1], eo), max(b[2], es)
        b[3], b[4] = max(b[3], no), max(b[4], ns)
    line = "; ".join(f"{dt}: {b[0]} cases, max-rel o {b[1]:.2e} s {b[2]:.2e}, max NMSE o {b[3]:.2e} "
                     f"s {b[4]:.2e}" for dt, b in sorted(by.items()))
    say(f"[parity summary] {line}")
    for dt, b in by.items():
        assert b[1] <= TOL[dt] and b[2] <= TOL[dt]
