"""GPU parity of the segment-parallel state chain (paper Sec. 4, the
Chunk-Seg-Seg mapping) at forced segment lengths.

Small inputs are cut into many short segments, so every path of the two
segment kernels runs: segment maps with and without an initial state (the A
part is skipped when the chain starts from zero), prefixes of one or several
maps, last segments shorter than the rest, empty and one-token sequences in a
packed batch, fp32 maps (1e-4) and bf16 maps (2e-2).  Every case is compared
element by element with the fp64 oracle, whose result does not depend on the
segment length.
"""

import numpy as np
import pytest

from gpu_harness import check_against_oracle, run_gpu, to_device
from paper_2609_32114_amd.inputs import make_case

pytestmark = pytest.mark.gpu


@pytest.fixture
def seg():
    import paper_2609_32114_amd as P
    yield P.set_segment_chunks
    P.set_segment_chunks(0)


@pytest.mark.parametrize("L", [1, 2, 3, 5, 16])
@pytest.mark.parametrize("s0", [True, False])
def test_gdn_bf16_segment_lengths(seg, L, s0):
    seg(L)
    inp = make_case("gdn", (1000,), 2, 4, 128, 128, "bf16", with_s0=s0, seed=31)
    check_against_oracle(inp, label=f"seg L={L}")


@pytest.mark.parametrize("L", [1, 3])
@pytest.mark.parametrize("s0", [True, False])
def test_kda_bf16_segment_lengths(seg, L, s0):
    seg(L)
    inp = make_case("kda", (700,), 1, 2, 128, 128, "bf16", with_s0=s0, seed=32)
    check_against_oracle(inp, label=f"seg-kda L={L}")


@pytest.mark.parametrize("dims", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_f32_segments(seg, kind, dims):
    seg(2)
    inp = make_case(kind, (450,), 1, 2, dims[0], dims[1], "f32", with_s0=True, seed=33)
    check_against_oracle(inp, label=f"seg-f32 {kind} {dims}")


@pytest.mark.parametrize("dims", [(64, 64), (64, 128), (128, 64)])
@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_bf16_segment_dims(seg, kind, dims):
    seg(2)
    inp = make_case(kind, (450, 130), 2, 4, dims[0], dims[1], "bf16", with_s0=True, seed=36)
    check_against_oracle(inp, label=f"seg-bf16 {kind} {dims}")


@pytest.mark.parametrize("L", [1, 2])
@pytest.mark.parametrize("s0", [True, False])
def test_varlen_segments(seg, L, s0):
    seg(L)
    inp = make_case("gdn", (0, 1, 64, 65, 130, 7, 0, 200, 1000), 2, 4, 128, 128, "bf16",
                    with_s0=s0, seed=34)
    check_against_oracle(inp, label=f"seg-varlen L={L}")


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_segments_deterministic(seg, kind):
    seg(3)
    inp = make_case(kind, (900, 333), 2, 4, 128, 128, "bf16", with_s0=True, seed=35)
    d = to_device(inp)
    a = run_gpu(inp, dev=d)
    b = run_gpu(inp, dev=d)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
