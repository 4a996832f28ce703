"""Pins for the fp64 oracle: what the definition and the mathematics fix.

Every pin takes a ``run(kind, q, k, v, g, beta, s0, cu, scale) -> (o, s_final)``
callable so that the same checks also run against builds of the oracle with a
planted mistake (``test_planted_mistakes_are_caught``): each plausible slip
(a dropped term, a wrong sign, operand or index) must fail at least one pin.

The gated delta rule, in the state orientation S (d_v x d_k) of the Gated
DeltaNet definition, is S_t = a_t S_{t-1}(I - b_t k_t k_t^T) + b_t v_t k_t^T,
o_t = S_t q_t (the output reads the updated state, paper Sec. 2.1); KDA puts a
per-key-channel Diag(a_t) on the key side before the delta update.  The
oracle stores H = S^T.
"""

import os
import shutil
import tempfile

import numpy as np
import pytest
import scipy.linalg
import scipy.signal

import oracle

RTOL = 1e-12


def _close(a, b, rtol=RTOL, atol=1e-13, what=""):
    a = np.asarray(a)
    b = np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= atol + rtol * scale, f"{what}: max err {err:.3e}"


def _unit(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind="gdn", unit=True, s0=True):
    q = rng.standard_normal((T, Hqk, Dk))
    k = rng.standard_normal((T, Hqk, Dk))
    if unit:
        q, k = _unit(q), _unit(k)
    v = rng.standard_normal((T, Hv, Dv))
    gs = (T, Hv) if kind == "gdn" else (T, Hv, Dk)
    g = -np.logaddexp(0.0, rng.standard_normal(gs)) * 0.3
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((T, Hv))))
    S0 = 0.3 * rng.standard_normal((1, Hv, Dk, Dv)) if s0 else None
    return q, k, v, g, beta, S0


# ----------------------------------------------------------------------------- pins

def pin_t1_closed_form_gdn(run):
    """T=1: S_1 = a S_0 (I - b k k^T) + b v k^T, o_1 = S_1 q (d_k != d_v catches transposes)."""
    rng = np.random.default_rng(11)
    Dk, Dv = 5, 3
    q, k, v, g, beta, s0 = _one_seq(rng, 1, 1, 1, Dk, Dv, unit=False)
    o, sf = run("gdn", q, k, v, g, beta, s0, None, 1.0)
    S0 = s0[0, 0].T
    kk, vv, qq = k[0, 0], v[0, 0], q[0, 0]
    a, b = np.exp(g[0, 0]), beta[0, 0]
    S1 = a * S0 @ (np.eye(Dk) - b * np.outer(kk, kk)) + b * np.outer(vv, kk)
    _close(sf[0, 0], S1.T, what="state")
    _close(o[0, 0], S1 @ qq, what="output")
    # zero initial state: o_1 = b (k . q) v
    o, sf = run("gdn", q, k, v, g, beta, None, None, 1.0)
    _close(o[0, 0], b * np.dot(kk, qq) * vv, what="o from zero state")
    _close(sf[0, 0], b * np.outer(kk, vv), what="s from zero state")


def pin_t1_closed_form_kda(run):
    """KDA T=1: S_1 = S_0 Diag(a) (I - b k k^T) + b v k^T (decay before the delta update)."""
    rng = np.random.default_rng(12)
    Dk, Dv = 6, 4
    q, k, v, g, beta, s0 = _one_seq(rng, 1, 1, 1, Dk, Dv, kind="kda", unit=False)
    g = g * 5.0  # strongly channel-dependent decay
    o, sf = run("kda", q, k, v, g, beta, s0, None, 1.0)
    S0 = s0[0, 0].T
    kk, vv, qq = k[0, 0], v[0, 0], q[0, 0]
    b = beta[0, 0]
    S1 = S0 @ np.diag(np.exp(g[0, 0])) @ (np.eye(Dk) - b * np.outer(kk, kk)) + b * np.outer(vv, kk)
    _close(sf[0, 0], S1.T, what="state")
    _close(o[0, 0], S1 @ qq, what="output")


def pin_literal_matrix_form(run):
    """T=9, grouped heads: iterate the matrix form of the definition literally in S orientation."""
    rng = np.random.default_rng(13)
    T, Hqk, Hv, Dk, Dv = 9, 2, 4, 5, 7
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, s0 = _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind=kind, unit=False)
        o, sf = run(kind, q, k, v, g, beta, s0, None, 0.75)
        for h in range(Hv):
            hk = h // (Hv // Hqk)
            S = s0[0, h].T.copy()
            for t in range(T):
                kk = k[t, hk]
                D = np.diag(np.exp(g[t, h])) if kind == "kda" else np.exp(g[t, h]) * np.eye(Dk)
                S = S @ D @ (np.eye(Dk) - beta[t, h] * np.outer(kk, kk)) + beta[t, h] * np.outer(v[t, h], kk)
                _close(o[t, h], 0.75 * S @ q[t, hk], what=f"{kind} o t={t} h={h}")
            _close(sf[0, h], S.T, what=f"{kind} state h={h}")


def pin_identity_when_no_write_no_decay(run):
    """beta=0, a=1: the state is unchanged bit for bit and o_t = S_0 q_t."""
    rng = np.random.default_rng(14)
    T, Dk, Dv = 13, 6, 5
    q, k, v, g, beta, s0 = _one_seq(rng, T, 1, 2, Dk, Dv)
    for kind in ("gdn", "kda"):
        gz = np.zeros((T, 2)) if kind == "gdn" else np.zeros((T, 2, Dk))
        o, sf = run(kind, q, k, v, gz, np.zeros((T, 2)), s0, None, 1.0)
        assert np.array_equal(sf, s0), kind
        for h in range(2):
            _close(o[:, h], q[:, 0] @ s0[0, h], what=f"{kind} o")


def pin_pure_decay(run):
    """beta=0: the state only decays, H_t = Diag(exp(sum_{s<=t} g_s)) H_0 (scalar for GDN)."""
    rng = np.random.default_rng(15)
    T, Dk, Dv = 11, 4, 3
    q, k, v, g, beta, s0 = _one_seq(rng, T, 1, 1, Dk, Dv)
    o, sf = run("gdn", q, k, v, g, np.zeros((T, 1)), s0, None, 1.0)
    cum = np.cumsum(g[:, 0])
    _close(sf[0, 0], np.exp(cum[-1]) * s0[0, 0], what="gdn state")
    _close(o[:, 0], np.exp(cum)[:, None] * (q[:, 0] @ s0[0, 0]), what="gdn o")
    gk = -np.abs(rng.standard_normal((T, 1, Dk)))
    o, sf = run("kda", q, k, v, gk, np.zeros((T, 1)), s0, None, 1.0)
    cumk = np.cumsum(gk[:, 0], axis=0)
    _close(sf[0, 0], np.exp(cumk[-1])[:, None] * s0[0, 0], what="kda state")
    _close(o[:, 0], (q[:, 0] * np.exp(cumk)) @ s0[0, 0], what="kda o")


def pin_orthonormal_retrieval(run):
    """Orthonormal keys, a=1, b=1: S_T k_i = v_i for every written key; o_t = v_t when q_t = k_t."""
    rng = np.random.default_rng(16)
    Dk, Dv, T = 8, 5, 6
    Qm, _ = np.linalg.qr(rng.standard_normal((Dk, Dk)))
    k = Qm[:T][:, None, :]
    v = rng.standard_normal((T, 1, Dv))
    s0 = rng.standard_normal((1, 1, Dk, Dv))
    for kind in ("gdn", "kda"):
        gz = np.zeros((T, 1)) if kind == "gdn" else np.zeros((T, 1, Dk))
        o, sf = run(kind, k.copy(), k, v, gz, np.ones((T, 1)), s0, None, 1.0)
        for i in range(T):
            _close(sf[0, 0].T @ k[i, 0], v[i, 0], rtol=1e-12, what=f"{kind} retrieval {i}")
        _close(o[:, 0], v[:, 0], what=f"{kind} o_t = v_t")


def pin_linearity_in_v_and_s0(run):
    """(o, s_final) is linear in (v, s0) for fixed q, k, g, beta."""
    rng = np.random.default_rng(17)
    T, Hqk, Hv, Dk, Dv = 10, 1, 2, 6, 4
    for kind in ("gdn", "kda"):
        q, k, v1, g, beta, s01 = _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind=kind)
        v2 = rng.standard_normal(v1.shape)
        s02 = rng.standard_normal(s01.shape)
        o1, f1 = run(kind, q, k, v1, g, beta, s01, None, 1.0)
        o2, f2 = run(kind, q, k, v2, g, beta, s02, None, 1.0)
        o3, f3 = run(kind, q, k, v1 - 2.5 * v2, g, beta, s01 - 2.5 * s02, None, 1.0)
        _close(o3, o1 - 2.5 * o2, what=f"{kind} o")
        _close(f3, f1 - 2.5 * f2, what=f"{kind} s")


def pin_split_invariance(run):
    """prefill(x1 || x2) = prefill(x2; s0 = final(x1)), the prefill -> resume handoff."""
    rng = np.random.default_rng(18)
    T, cut, Hqk, Hv, Dk, Dv = 37, 20, 1, 2, 5, 6
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, s0 = _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind=kind)
        o, sf = run(kind, q, k, v, g, beta, s0, None, 1.0)
        oa, sa = run(kind, q[:cut], k[:cut], v[:cut], g[:cut], beta[:cut], s0, None, 1.0)
        ob, sb = run(kind, q[cut:], k[cut:], v[cut:], g[cut:], beta[cut:], sa, None, 1.0)
        _close(np.concatenate([oa, ob]), o, what=f"{kind} o")
        _close(sb, sf, what=f"{kind} s")


def pin_norm_bound(run):
    """Unit keys, b in [0,1], a <= 1: ||H_T||_F <= ||H_0||_F + sum_t b_t ||v_t||."""
    rng = np.random.default_rng(19)
    T, Dk, Dv = 40, 6, 6
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, s0 = _one_seq(rng, T, 1, 1, Dk, Dv, kind=kind)
        o, sf = run(kind, q, k, v, g, beta, s0, None, 1.0)
        bound = np.linalg.norm(s0) + np.sum(beta[:, 0] * np.linalg.norm(v[:, 0], axis=-1))
        assert np.linalg.norm(sf) <= bound * (1 + 1e-12), kind
        # and in the DeltaNet limit the write is an exact projection: ||H_T|| stays bounded
        gz = np.zeros_like(g)
        o, sf = run(kind, q, k, v, gz, np.ones_like(beta), s0, None, 1.0)
        assert np.linalg.norm(sf) <= np.linalg.norm(s0) + np.sum(np.linalg.norm(v[:, 0], axis=-1))


def pin_scalar_recurrence_vs_lfilter(run):
    """d_k=d_v=1 with constant a, b, k, q: h_t = a(1-b k^2) h_{t-1} + b k v_t is a
    first-order IIR filter; scipy.signal.lfilter computes it independently."""
    rng = np.random.default_rng(20)
    T = 50
    a, b, kk, qq = 0.93, 0.6, 0.8, -1.3
    v = rng.standard_normal((T, 1, 1))
    h0 = 0.4
    c = a * (1 - b * kk * kk)
    y, _ = scipy.signal.lfilter([b * kk], [1.0, -c], v[:, 0, 0], zi=[c * h0])
    for kind in ("gdn", "kda"):
        g = np.full((T, 1), np.log(a)) if kind == "gdn" else np.full((T, 1, 1), np.log(a))
        o, sf = run(kind, np.full((T, 1, 1), qq), np.full((T, 1, 1), kk), v, g,
                    np.full((T, 1), b), np.full((1, 1, 1, 1), h0), None, 1.0)
        _close(o[:, 0, 0], qq * y, rtol=1e-12, what=f"{kind} o")
        _close(sf[0, 0, 0, 0], y[-1], rtol=1e-12, what=f"{kind} s")


def pin_kda_uniform_equals_gdn(run):
    """KDA with a channel-uniform gate is GDN with that scalar gate."""
    rng = np.random.default_rng(21)
    T, Hqk, Hv, Dk, Dv = 23, 2, 4, 8, 5
    q, k, v, g, beta, s0 = _one_seq(rng, T, Hqk, Hv, Dk, Dv)
    o1, f1 = run("gdn", q, k, v, g, beta, s0, None, 1.0)
    o2, f2 = run("kda", q, k, v, np.repeat(g[:, :, None], Dk, axis=2), beta, s0, None, 1.0)
    _close(o2, o1, rtol=1e-14, what="o")
    _close(f2, f1, rtol=1e-14, what="s")


def pin_grouped_heads_equal_repeated(run):
    """Grouped q/k heads: value head h reads q/k head h // (Hv/Hqk) -- equal to repeating q, k."""
    rng = np.random.default_rng(22)
    T, Hqk, Hv, Dk, Dv = 17, 2, 6, 4, 3
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, s0 = _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind=kind)
        o1, f1 = run(kind, q, k, v, g, beta, s0, None, 1.0)
        rep = Hv // Hqk
        o2, f2 = run(kind, np.repeat(q, rep, axis=1), np.repeat(k, rep, axis=1), v, g, beta, s0,
                     None, 1.0)
        _close(o1, o2, rtol=1e-15, what=f"{kind} o")
        _close(f1, f2, rtol=1e-15, what=f"{kind} s")


def pin_varlen_is_concatenation(run):
    """Packed sequences (with an empty one) equal independent single-sequence runs."""
    rng = np.random.default_rng(23)
    lens = [5, 0, 11, 1]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T, Hqk, Hv, Dk, Dv = int(cu[-1]), 1, 2, 4, 4
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, _ = _one_seq(rng, T, Hqk, Hv, Dk, Dv, kind=kind)
        s0 = rng.standard_normal((len(lens), Hv, Dk, Dv))
        o, sf = run(kind, q, k, v, g, beta, s0, cu, 1.0)
        for n in range(len(lens)):
            a, b = cu[n], cu[n + 1]
            on, sn = run(kind, q[a:b], k[a:b], v[a:b], g[a:b], beta[a:b], s0[n:n + 1], None, 1.0)
            _close(o[a:b], on, what=f"{kind} o seq {n}")
            _close(sf[n:n + 1], sn, what=f"{kind} s seq {n}")
        assert np.array_equal(sf[1], s0[1]), "empty sequence must return its s0"


def pin_scale_only_scales_output(run):
    rng = np.random.default_rng(24)
    q, k, v, g, beta, s0 = _one_seq(rng, 12, 1, 1, 4, 4)
    o1, f1 = run("gdn", q, k, v, g, beta, s0, None, 1.0)
    o2, f2 = run("gdn", q, k, v, g, beta, s0, None, 0.125)
    _close(o2, 0.125 * o1, rtol=1e-15, what="o")
    assert np.array_equal(f1, f2)


def pin_chunked_formulation_agrees(run):
    """Brute force: the independent chunkwise fp64 formulation reaches the same result."""
    from chunked_ref import chunked_prefill
    rng = np.random.default_rng(25)
    for kind in ("gdn", "kda"):
        q, k, v, g, beta, s0 = _one_seq(rng, 50, 1, 2, 5, 3, kind=kind)
        o, sf = run(kind, q, k, v, g, beta, s0, None, 1.0)
        oc, sc = chunked_prefill(kind, q, k, v, g, beta, s0, None, 1.0, chunk=16)
        _close(o, oc, what=f"{kind} o")
        _close(sf, sc, what=f"{kind} s")


PINS = [v for n, v in sorted(globals().items()) if n.startswith("pin_")]


def _default_run(kind, q, k, v, g, beta, s0, cu, scale):
    return oracle.prefill(kind, q, k, v, g, beta, s0, cu, scale, nthreads=2)


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin, oracle_mod):
    pin(_default_run)


def test_oracle_rejects_bad_arguments(oracle_mod):
    rng = np.random.default_rng(0)
    q, k, v, g, beta, s0 = _one_seq(rng, 8, 2, 3, 4, 4)  # Hv % Hqk != 0
    with pytest.raises(ValueError):
        oracle.prefill("gdn", q, k, v, g, beta, None, None, 1.0)
    q, k, v, g, beta, s0 = _one_seq(rng, 8, 1, 1, 4, 4)
    with pytest.raises(ValueError):  # cu_seqlens not ending at T
        oracle.prefill("gdn", q, k, v, g, beta, None, np.array([0, 5]), 1.0)
    with pytest.raises(ValueError):  # decreasing cu_seqlens
        oracle.prefill("gdn", q, k, v, g, beta, None, np.array([0, 6, 4, 8]), 1.0)


def test_oracle_empty_input_returns_initial_state(oracle_mod):
    rng = np.random.default_rng(1)
    s0 = rng.standard_normal((2, 1, 3, 3))
    e = np.zeros((0, 1, 3))
    o, sf = oracle.prefill("gdn", e, e, e, np.zeros((0, 1)), np.zeros((0, 1)), s0,
                           np.array([0, 0, 0]), 1.0)
    assert o.shape == (0, 1, 3)
    assert np.array_equal(sf, s0)


# Plausible slips, each planted in a copy of oracle.c: (description, original, replacement).
MUTANTS = [
    ("drop the scalar decay", "for (size_t e = 0; e < (size_t)Dk * Dv; ++e) H[e] *= a;", ""),
    ("sign of the delta term", "p[j] = bt * (vt[j] - p[j]);", "p[j] = bt * (vt[j] + p[j]);"),
    ("drop beta", "p[j] = bt * (vt[j] - p[j]);", "p[j] = (vt[j] - p[j]);"),
    ("read output with k", "const double qi = qt[i];", "const double qi = kt[i];"),
    ("projection uses q", "p[j] += H[(size_t)i * Dv + j] * ki;", "p[j] += H[(size_t)i * Dv + j] * qt[i];"),
    ("write uses q", "H[(size_t)i * Dv + j] += ki * p[j];", "H[(size_t)i * Dv + j] += qt[i] * p[j];"),
    ("kda gate channel index", "const double a = exp(gt[i]);", "const double a = exp(gt[0]);"),
    ("grouped head index", "const int hk = h / group;", "const int hk = h % Hqk;"),
    ("drop the output scale", "for (int j = 0; j < Dv; ++j) ot[j] *= scale;", ""),
    ("ignore s0", "memcpy(H, s0_nh, sizeof(double) * (size_t)Dk * Dv);",
     "memset(H, 0, sizeof(double) * (size_t)Dk * Dv);"),
    ("gate sign", "const double a = exp(g[(size_t)t * Hv + h]);",
     "const double a = exp(-g[(size_t)t * Hv + h]);"),
    ("output from the pre-update state",
     "    /* u <- beta_t (v_t - p) (stored over p) */",
     "    { double *ot0 = o + ((size_t)t * Hv + h) * Dv;\n"
     "      for (int j = 0; j < Dv; ++j) { ot0[j] = 0.0; for (int i = 0; i < Dk; ++i)"
     " ot0[j] += H[(size_t)i * Dv + j] * qt[i] * scale; } }\n"
     "    /* u <- beta_t (v_t - p) (stored over p) */"),
]


def test_planted_mistakes_are_caught(oracle_mod):
    """Each planted slip in a copy of the oracle must make at least one pin fail."""
    src = open(oracle.SOURCE).read()
    tmp = tempfile.mkdtemp(prefix="oracle_mut_")
    try:
        for i, (desc, old, new) in enumerate(MUTANTS):
            assert src.count(old) == 1, f"mutant '{desc}': anchor not unique in oracle.c"
            msrc = src.replace(old, new)
            if desc == "output from the pre-update state":
                # disable the correct output computation after the update
                msrc = msrc.replace("for (int j = 0; j < Dv; ++j) ot[j] = 0.0;",
                                    "if (0) for (int j = 0; j < Dv; ++j) ot[j] = 0.0;")
                msrc = msrc.replace("for (int j = 0; j < Dv; ++j) ot[j] += H[(size_t)i * Dv + j] * qi;",
                                    "if (0) ot[0] += qi;")
                msrc = msrc.replace("for (int j = 0; j < Dv; ++j) ot[j] *= scale;", "")
            path = os.path.join(tmp, f"m{i}.c")
            with open(path, "w") as f:
                f.write(msrc)
            lib = oracle.load_library(oracle.compile_source(path, os.path.join(tmp, f"m{i}.so")))

            def run(kind, q, k, v, g, beta, s0, cu, scale, _lib=lib):
                return oracle.prefill(kind, q, k, v, g, beta, s0, cu, scale, nthreads=1, lib=_lib)

            failed = []
            for pin in PINS:
                try:
                    pin(run)
                except AssertionError:
                    failed.append(pin.__name__)
            assert failed, f"planted mistake '{desc}' passed every pin"
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
