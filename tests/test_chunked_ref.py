"""The chunkwise formulation agrees with the token-by-token oracle (fp64, tiny inputs).

Chunk sizes 1 (the recurrence itself), 2, 3, 4, 8, 16, 64; lengths that are
not multiples of the chunk; nonzero initial state; GDN and KDA; grouped heads
and varlen packing.  Both sides are fp64, so they must agree to rounding.
"""

import numpy as np
import pytest

import oracle
from chunked_ref import chunked_prefill


def _inputs(rng, T, Hqk, Hv, Dk, Dv, kind, gate_scale=1.0):
    q = rng.standard_normal((T, Hqk, Dk))
    k = rng.standard_normal((T, Hqk, Dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, Hv, Dv))
    gs = (T, Hv) if kind == "gdn" else (T, Hv, Dk)
    g = -np.logaddexp(0.0, gate_scale * rng.standard_normal(gs))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((T, Hv))))
    return q, k, v, g, beta


def _relerr(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


@pytest.mark.parametrize("kind", ["gdn", "kda"])
@pytest.mark.parametrize("T", [1, 7, 50, 130])
@pytest.mark.parametrize("chunk", [1, 2, 3, 4, 8, 16, 64])
def test_chunked_matches_oracle(kind, T, chunk, oracle_mod):
    rng = np.random.default_rng(100 + T * 7 + chunk)
    Hqk, Hv, Dk, Dv = 1, 2, 6, 5
    q, k, v, g, beta = _inputs(rng, T, Hqk, Hv, Dk, Dv, kind, gate_scale=0.5)
    s0 = 0.5 * rng.standard_normal((1, Hv, Dk, Dv))
    o, sf = oracle.prefill(kind, q, k, v, g, beta, s0, None, 1.0)
    oc, sc = chunked_prefill(kind, q, k, v, g, beta, s0, None, 1.0, chunk=chunk)
    assert _relerr(oc, o) < 1e-12
    assert _relerr(sc, sf) < 1e-12


@pytest.mark.parametrize("kind", ["gdn", "kda"])
def test_chunked_varlen_grouped(kind, oracle_mod):
    rng = np.random.default_rng(7)
    lens = [70, 3, 0, 129]
    cu = np.concatenate([[0], np.cumsum(lens)])
    q, k, v, g, beta = _inputs(rng, int(cu[-1]), 2, 4, 8, 8, kind)
    s0 = 0.1 * rng.standard_normal((4, 4, 8, 8))
    o, sf = oracle.prefill(kind, q, k, v, g, beta, s0, cu, 0.3)
    oc, sc = chunked_prefill(kind, q, k, v, g, beta, s0, cu, 0.3, chunk=64)
    assert _relerr(oc, o) < 1e-12
    assert _relerr(sc, sf) < 1e-12


def test_chunked_long_memory_and_deltanet_limit(oracle_mod):
    """alpha close to 1 and alpha = 1: inter-chunk propagation carries real signal."""
    rng = np.random.default_rng(8)
    for gscale in (0.01, 0.0):
        q, k, v, g, beta = _inputs(rng, 200, 1, 1, 16, 16, "gdn")
        g = g * gscale
        s0 = rng.standard_normal((1, 1, 16, 16))
        o, sf = oracle.prefill("gdn", q, k, v, g, beta, s0, None, 1.0)
        oc, sc = chunked_prefill("gdn", q, k, v, g, beta, s0, None, 1.0, chunk=64)
        assert _relerr(oc, o) < 1e-11
        assert _relerr(sc, sf) < 1e-11
