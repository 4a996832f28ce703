"""GPU: the overlapped launch (chunk-local items and whole-chain walks in one
grid, per-XCD queues and ready flags) against the serialized kernels.

Both run the same arithmetic on every block, so o and s_final must match bit
for bit; each case is also checked against the oracle and reads back a clean
device status word (no walk timed out waiting for a chunk).  The small cases
force the overlapped launch (mode 2): by default it is used only where the
chunk-local work needs more than one round.
"""

import numpy as np
import pytest

from gpu_harness import check_against_oracle, run_gpu, say, to_device
from paper_2609_32114_amd.inputs import make_case, make_workload

pytestmark = pytest.mark.gpu

CASES = [
    # kind, lengths, Hqk, Hv, with_s0, variant, raw
    ("gdn", (4096,), 16, 16, False, "base", False),        # the timed workload's shape
    ("gdn", (1000,), 4, 16, True, "s0", False),            # grouped heads, ragged tail
    ("gdn", (65,), 1, 3, False, "base", False),            # 2 chunks; XCDs 3-7 serve no head
    ("gdn", (1500,), 12, 12, False, "base", True),         # raw projections; 1 or 2 heads per XCD
    ("gdn", (0, 1, 700, 64, 129), 2, 2, True, "s0", False),  # a batch: empty, 1-token, ragged
    ("gdn", (2048,), 8, 8, False, "lm", False),            # long memory
    ("gdn", (1200,), 16, 16, False, "fg", False),          # forgetting gates
]


def _ids(c):
    return f"{c[0]}-N{len(c[1])}-T{sum(c[1])}-Hv{c[3]}-{c[5]}{'-raw' if c[6] else ''}"


def _run(inp, d, pre, workspace=None):
    import torch
    import paper_2609_32114_amd as P
    fn = P.gdn_prefill if inp.kind == "gdn" else P.kda_prefill
    o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"], cu_seqlens=d["cu"],
               scale=inp.scale, preprocess=pre, workspace=workspace)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), sf.cpu().numpy()


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_overlap_matches_serialized(case):
    import torch
    import paper_2609_32114_amd as P
    kind, lengths, Hqk, Hv, with_s0, variant, raw = case
    inp = make_case(kind, lengths, Hqk, Hv, 128, 128, "bf16", with_s0=with_s0, variant=variant,
                    seed=41, raw=raw)
    pre = P.PRE_ALL if raw else 0
    N, T = len(lengths), sum(lengths)
    say(f"overlap {_ids(case)}")
    d = to_device(inp)
    ws = torch.empty(P.workspace_size(kind, N, T, Hqk, Hv, 128, 128, P.HAGDN_BF16), dtype=torch.uint8,
                     device="cuda")
    try:
        P.set_overlap(False)
        o_ser, s_ser = _run(inp, d, pre, ws)
        assert P.device_status(ws) == P.DEV_OK
        P.set_overlap(True, force=True)
        assert P.overlap_for(N, T, Hv, 128, 128, P.HAGDN_BF16, kind)
        for rep in range(2):  # a second call reuses the workspace: flags and queues start over
            o_ovl, s_ovl = _run(inp, d, pre, ws)
            assert P.device_status(ws) == P.DEV_OK
            np.testing.assert_array_equal(o_ovl, o_ser)
            np.testing.assert_array_equal(s_ovl, s_ser)
    finally:
        P.set_overlap(True)
    if not raw:
        check_against_oracle(inp, label=f"overlap-{_ids(case)}")


def test_overlap_bad_seqlens_reported():
    """A single sequence whose cu_seqlens is malformed: nothing is walked, the
    state comes back as s0 and the status word says why, also overlapped."""
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (300,), 2, 8, 128, 128, "bf16", with_s0=True, variant="s0", seed=3)
    d = to_device(inp)
    d["cu"] = torch.tensor([0, 299], dtype=torch.int32, device="cuda")
    ws = torch.empty(P.workspace_size("gdn", 1, 300, 2, 8, 128, 128, P.HAGDN_BF16), dtype=torch.uint8,
                     device="cuda")
    try:
        P.set_overlap(True, force=True)
        assert P.overlap_for(1, 300, 8, 128, 128, P.HAGDN_BF16)
        o, sf = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                              cu_seqlens=d["cu"], workspace=ws)
        torch.cuda.synchronize()
    finally:
        P.set_overlap(True)
    assert P.device_status(ws) == P.DEV_BAD_SEQLENS
    np.testing.assert_array_equal(sf.cpu().numpy(), d["s0"].cpu().numpy())


def test_overlap_workload1_every_head():
    """Workload 1 in the benchmark's configuration (overlapped by default)
    against the oracle on every head, and bitwise against the serialized path."""
    import paper_2609_32114_amd as P
    inp = make_workload(1)
    assert P.overlap_for(inp.N, inp.T, 16, 128, 128, P.HAGDN_BF16)
    check_against_oracle(inp, label="overlap-workload1")
    d = to_device(inp)
    o_ovl, s_ovl = run_gpu(inp, dev=d)
    try:
        P.set_overlap(False)
        o_ser, s_ser = run_gpu(inp, dev=d)
    finally:
        P.set_overlap(True)
    np.testing.assert_array_equal(o_ovl, o_ser)
    np.testing.assert_array_equal(s_ovl, s_ser)


def test_overlap_in_place_state():
    """s_final aliasing s0 on the overlapped launch: every walk reads its
    columns of s0 before it writes them, and no producer touches the state."""
    import torch
    import paper_2609_32114_amd as P
    inp = make_case("gdn", (777,), 4, 16, 128, 128, "bf16", with_s0=True, variant="s0", seed=43)
    d = to_device(inp)
    try:
        P.set_overlap(True, force=True)
        assert P.overlap_for(1, 777, 16, 128, 128, P.HAGDN_BF16)
        o_ref, s_ref = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
                                     cu_seqlens=d["cu"], scale=inp.scale)
        state = d["s0"].clone()
        o, sf = P.gdn_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=state,
                              cu_seqlens=d["cu"], scale=inp.scale, final_out=state)
        torch.cuda.synchronize()
    finally:
        P.set_overlap(True)
    assert sf.data_ptr() == state.data_ptr()
    np.testing.assert_array_equal(state.cpu().numpy(), s_ref.cpu().numpy())
    np.testing.assert_array_equal(o.float().cpu().numpy(), o_ref.float().cpu().numpy())


def test_kda_never_overlaps():
    """KDA has no overlapped instance (its chunk-local items are about twice as
    heavy; overlapped it measured slower), even in the forced mode."""
    import paper_2609_32114_amd as P
    try:
        P.set_overlap(True, force=True)
        assert not P.overlap_for(1, 4096, 16, 128, 128, P.HAGDN_BF16, "kda")
        assert P.overlap_for(1, 4096, 16, 128, 128, P.HAGDN_BF16, "gdn")
    finally:
        P.set_overlap(True)
