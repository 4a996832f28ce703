"""Pins for the oracle's preprocessing of raw projections and its decode step.

Preprocessing (oracle_preprocess in oracle.c) maps raw projections to the
recurrence's inputs: q and k L2-normalised per token and head with the norm
floored at 1e-6, the log-gate g = -softplus(x), the write strength
beta = sigmoid(x).  Its pins check the results against library routines
(numpy's logaddexp, scipy's expit, numpy's norm) and closed forms, and a
planted-mistake test builds copies of the oracle with plausible slips in that
code, each of which must fail a pin.

Decode (oracle.decode) is one token of the recurrence for each of N
sequences whose states live in a pool addressed through slots.  Its pins
check the handoff (prefill of T tokens then K decode steps equals prefill of
T + K tokens), the slot gather and scatter, and padding slots.
"""

import os
import shutil
import tempfile

import numpy as np
import pytest
import scipy.special

import oracle

PRE = (oracle.PRE_QK_L2NORM, oracle.PRE_GATE_SOFTPLUS, oracle.PRE_BETA_SIGMOID)


def _close(a, b, rtol=1e-13, atol=1e-15, what=""):
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= atol + rtol * scale, f"{what}: max err {err:.3e}"


def _raw(rng, T, Hqk, Hv, Dk, kind):
    q = 3.0 * rng.standard_normal((T, Hqk, Dk))
    k = 0.5 * rng.standard_normal((T, Hqk, Dk))
    gs = (T, Hv) if kind == "gdn" else (T, Hv, Dk)
    g = 4.0 * rng.standard_normal(gs)
    b = 4.0 * rng.standard_normal((T, Hv))
    return q, k, g, b


# ------------------------------------------------------------ preprocessing pins

def pin_pre_l2norm_unit_rows(pre):
    """Every q and k row gets unit norm and keeps its direction (a positive multiple)."""
    rng = np.random.default_rng(31)
    q, k, g, b = _raw(rng, 7, 3, 3, 5, "gdn")
    q2, k2, g2, b2 = pre("gdn", q, k, g, b, oracle.PRE_QK_L2NORM)
    for x, y, name in ((q, q2, "q"), (k, k2, "k")):
        _close(np.linalg.norm(y, axis=-1), np.ones(x.shape[:2]), what=f"{name} norm")
        ratio = x / y
        _close(ratio, np.repeat(np.linalg.norm(x, axis=-1)[..., None], x.shape[-1], axis=-1),
               rtol=1e-13, what=f"{name} direction")
    assert np.array_equal(g2, g) and np.array_equal(b2, b), "flag 1 touches only q and k"


def pin_pre_l2norm_floor(pre):
    """Rows with norm below 1e-6 are divided by 1e-6, not by their norm (a zero row stays zero)."""
    q = np.zeros((2, 1, 4))
    q[1, 0] = [3e-8, 0.0, -4e-8, 0.0]  # norm 5e-8
    k = np.ones((2, 1, 4))
    q2, k2, _, _ = pre("gdn", q, k, np.zeros((2, 1)), np.zeros((2, 1)), oracle.PRE_QK_L2NORM)
    assert np.array_equal(q2[0], q[0])
    _close(q2[1, 0], q[1, 0] / 1e-6, rtol=1e-15, what="floored row")
    _close(k2, np.full((2, 1, 4), 0.5), what="k = 1/2 per element")


def pin_pre_softplus_vs_library(pre):
    """-g equals numpy's logaddexp(0, x) (softplus), also far into both tails."""
    rng = np.random.default_rng(32)
    for kind in ("gdn", "kda"):
        q, k, g, b = _raw(rng, 6, 1, 2, 4, kind)
        g.flat[:6] = [0.0, 40.0, -40.0, 700.0, -700.0, 1e-9]
        _, _, g2, b2 = pre(kind, q, k, g, b, oracle.PRE_GATE_SOFTPLUS)
        _close(-g2, np.logaddexp(0.0, g), rtol=1e-15, atol=0.0, what=f"{kind} softplus")
        assert g2.flat[0] == -np.log(2.0), "softplus(0) = ln 2"
        assert np.array_equal(b2, b)


def pin_pre_softplus_identity(pre):
    """softplus(x) - softplus(-x) = x, for every element of a KDA gate tensor."""
    rng = np.random.default_rng(33)
    q, k, g, b = _raw(rng, 5, 1, 2, 6, "kda")
    _, _, gp, _ = pre("kda", q, k, g, b, oracle.PRE_GATE_SOFTPLUS)
    _, _, gm, _ = pre("kda", q, k, -g, b, oracle.PRE_GATE_SOFTPLUS)
    _close(-gp + gm, g, rtol=1e-14, what="softplus(x) - softplus(-x)")


def pin_pre_sigmoid_vs_library(pre):
    """beta equals scipy's expit; sigmoid(0) = 1/2 and sigmoid(x) + sigmoid(-x) = 1."""
    rng = np.random.default_rng(34)
    q, k, g, b = _raw(rng, 9, 1, 3, 4, "gdn")
    b.flat[:3] = [0.0, 50.0, -50.0]
    _, _, g2, b2 = pre("gdn", q, k, g, b, oracle.PRE_BETA_SIGMOID)
    _close(b2, scipy.special.expit(b), rtol=1e-15, atol=1e-300, what="sigmoid")
    assert b2.flat[0] == 0.5
    _, _, _, bm = pre("gdn", q, k, g, -b, oracle.PRE_BETA_SIGMOID)
    _close(b2 + bm, np.ones_like(b), rtol=1e-15, what="sigmoid symmetry")
    assert np.array_equal(g2, g)


def pin_pre_all_flags_compose(pre):
    """All three flags at once equal the three applied one after another."""
    rng = np.random.default_rng(35)
    q, k, g, b = _raw(rng, 4, 2, 4, 8, "kda")
    full = pre("kda", q, k, g, b, 7)
    step = (q, k, g, b)
    for f in PRE:
        step = pre("kda", *step, f)
    for x, y, name in zip(full, step, "qkgb"):
        _close(x, y, rtol=1e-15, what=name)


PRE_PINS = [v for n, v in sorted(globals().items()) if n.startswith("pin_pre_")]


@pytest.mark.parametrize("pin", PRE_PINS, ids=[p.__name__ for p in PRE_PINS])
def test_preprocess_pin(pin, oracle_mod):
    pin(oracle.preprocess)


def test_preprocess_rejects_bad_flags(oracle_mod):
    z = np.zeros((1, 1, 4))
    with pytest.raises(ValueError):
        oracle.preprocess("gdn", z, z, np.zeros((1, 1)), np.zeros((1, 1)), 8)


# Slips planted in a copy of the preprocessing code of oracle.c.
PRE_MUTANTS = [
    ("norm without the square root", "double nrm = sqrt(ss);", "double nrm = ss;"),
    ("no floor on the norm", "if (nrm < 1e-6) nrm = 1e-6;", ""),
    ("normalise q only", "for (int w = 0; w < 2; ++w) {", "for (int w = 0; w < 1; ++w) {"),
    ("softplus without the linear term", "g[e] = -((x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x))));",
     "g[e] = -log1p(exp(-fabs(x)));"),
    ("softplus sign", "g[e] = -((x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x))));",
     "g[e] = ((x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x))));"),
    ("kda gate: first channel only", "const size_t n = (size_t)T * Hv * (kda ? Dk : 1);",
     "const size_t n = (size_t)T * Hv;"),
    ("sigmoid sign", "beta[e] = 1.0 / (1.0 + exp(-beta[e]));", "beta[e] = 1.0 / (1.0 + exp(beta[e]));"),
]


def test_preprocess_planted_mistakes_are_caught(oracle_mod):
    src = open(oracle.SOURCE).read()
    tmp = tempfile.mkdtemp(prefix="oracle_pre_mut_")
    try:
        for i, (desc, old, new) in enumerate(PRE_MUTANTS):
            assert src.count(old) == 1, f"mutant '{desc}': anchor not unique in oracle.c"
            path = os.path.join(tmp, f"p{i}.c")
            with open(path, "w") as f:
                f.write(src.replace(old, new))
            lib = oracle.load_library(oracle.compile_source(path, os.path.join(tmp, f"p{i}.so")))

            def pre(kind, q, k, g, b, flags, _lib=lib):
                return oracle.preprocess(kind, q, k, g, b, flags, lib=_lib)

            failed = []
            for pin in PRE_PINS:
                try:
                    with np.errstate(all="ignore"):
                        pin(pre)
                except AssertionError:
                    failed.append(pin.__name__)
            assert failed, f"planted mistake '{desc}' passed every preprocessing pin"
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


# ---------------------------------------------------------------------- decode

def _seqs(rng, N, T, Hqk, Hv, Dk, Dv, kind):
    q = rng.standard_normal((N, T, Hqk, Dk))
    k = rng.standard_normal((N, T, Hqk, Dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((N, T, Hv, Dv))
    gs = (N, T, Hv) if kind == "gdn" else (N, T, Hv, Dk)
    g = -0.1 * np.logaddexp(0.0, rng.standard_normal(gs))
    b = scipy.special.expit(rng.standard_normal((N, T, Hv)))
    return q, k, v, g, b


def test_decode_continues_prefill(oracle_mod):
    """Prefill T tokens, then K decode steps (all sequences at once) = prefill of T + K tokens."""
    rng = np.random.default_rng(41)
    N, T, K, Hqk, Hv, Dk, Dv = 3, 9, 4, 1, 2, 5, 3
    for kind in ("gdn", "kda"):
        q, k, v, g, b = _seqs(rng, N, T + K, Hqk, Hv, Dk, Dv, kind)
        s0 = rng.standard_normal((N, Hv, Dk, Dv))
        pack = lambda x, a, z: np.concatenate([x[n, a:z] for n in range(N)])
        cu_full = np.arange(N + 1, dtype=np.int32) * (T + K)
        o_full, s_full = oracle.prefill(kind, *(pack(x, 0, T + K) for x in (q, k, v, g, b)), s0,
                                        cu_full, 0.5, nthreads=2)
        cu_pre = np.arange(N + 1, dtype=np.int32) * T
        _, state = oracle.prefill(kind, *(pack(x, 0, T) for x in (q, k, v, g, b)), s0, cu_pre,
                                  0.5, nthreads=2)
        for t in range(T, T + K):
            o_t, state = oracle.decode(kind, q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], state,
                                       0.5, nthreads=2)
            for n in range(N):
                _close(o_t[n], o_full[n * (T + K) + t], rtol=1e-12, what=f"{kind} o n={n} t={t}")
        _close(state, s_full, rtol=1e-12, what=f"{kind} state")


def test_decode_slots_gather_scatter(oracle_mod):
    """Sequence n updates pool slot slots[n] only; a slot out of range is padding."""
    rng = np.random.default_rng(42)
    N, S, Hqk, Hv, Dk, Dv = 4, 6, 2, 4, 4, 5
    q, k, v, g, b = (x[:, 0] for x in _seqs(rng, N, 1, Hqk, Hv, Dk, Dv, "gdn"))
    pool = rng.standard_normal((S, Hv, Dk, Dv))
    slots = np.array([5, -1, 0, 6])  # 6 is out of range: padding too
    o, pool2 = oracle.decode("gdn", q, k, v, g, b, pool, 1.0, slots=slots)
    for n in range(N):
        s = slots[n]
        if 0 <= s < S:
            on, sn = oracle.prefill("gdn", q[n:n + 1], k[n:n + 1], v[n:n + 1], g[n:n + 1],
                                    b[n:n + 1], pool[s:s + 1], None, 1.0)
            _close(o[n], on[0], rtol=1e-15, what=f"o {n}")
            _close(pool2[s], sn[0], rtol=1e-15, what=f"state {n}")
        else:
            assert np.all(o[n] == 0.0)
    for s in (1, 2, 3, 4):
        assert np.array_equal(pool2[s], pool[s]), f"untouched slot {s}"


def test_decode_t1_closed_form(oracle_mod):
    """One decode step from S: S' = a S (I - b k k^T) + b v k^T, o = scale S' q (S orientation)."""
    rng = np.random.default_rng(43)
    Dk, Dv = 6, 3
    q, k, v, g, b = (x[:, 0] for x in _seqs(rng, 2, 1, 1, 1, Dk, Dv, "gdn"))
    pool = rng.standard_normal((2, 1, Dk, Dv))
    o, pool2 = oracle.decode("gdn", q, k, v, g, b, pool, 0.25, slots=[1, 0])
    for n, s in ((0, 1), (1, 0)):
        S = pool[s, 0].T
        kk = k[n, 0]
        S1 = np.exp(g[n, 0]) * S @ (np.eye(Dk) - b[n, 0] * np.outer(kk, kk)) + b[n, 0] * np.outer(v[n, 0], kk)
        _close(pool2[s, 0], S1.T, rtol=1e-13, what="state")
        _close(o[n, 0], 0.25 * S1 @ q[n, 0], rtol=1e-13, what="o")
