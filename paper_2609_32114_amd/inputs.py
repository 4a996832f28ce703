"""Seeded synthetic inputs shaped like the paper's prefill workloads.

This module holds no arithmetic of the method itself: it only draws random
tensors (numpy PCG64, fixed draw order), applies the input conventions of the
workloads (per-token L2 normalisation of q and k, log-gate = -softplus(x),
beta = sigmoid(x)) and rounds to the storage dtype.  Both the GPU tests and
the fp64 oracle consume exactly the arrays returned here.

Workloads (chunk size 64 throughout; the paper's kernels use C = 64 with
FP32 gates/states, Sec. 7.1 "Baselines"; sequence lengths and head counts
follow the paper's sweeps, Table 1 and Sec. 7.2-7.4):

  0  GDN, 1 sequence T=256,  Hqk=Hv=1,  d=64,  fp32, zero initial state
  1  GDN, 1 sequence T=4096, Hqk=Hv=16, d=128, bf16, zero initial state
  2  GDN, 1 sequence T=32768, H=16, d=128, bf16, s0 = 0.02*N(0,1)
  3  KDA, 1 sequence T=8192, H=16, d=128, bf16 (per-channel log-gate)
  4  GDN varlen: 8 sequences, lengths uniform in [512, 8192], Hqk=16, Hv=32,
     d=128, bf16, per-sequence s0 = 0.02*N(0,1)

Draw order (seed = 1000 + workload index unless given): lengths (varlen
only), q, k, v, g_raw, beta_raw, s0.

Stress variants (parity only, never timed) cover what the base
distributions cannot: with g = -softplus(N(0,1)) the state decays by about
e^-52 per 64-token chunk, so inter-chunk propagation and s0 barely matter.
  "lm"   long memory: g = -0.01*softplus(N(0,1))
  "dn"   DeltaNet limit: g = 0
  "ks"   key stress: keys from a random 4-dim subspace per head, beta = 1
  "s0"   lm gates plus a nonzero 0.02*N(0,1) initial state
  "lg"   large gates: g = -softplus(3*N(0,1)) (exercises KDA exponent bounds)
  "fg"   forget runs: base gates, except that runs of 8-24 consecutive tokens
         (gaps of 8-56 tokens between them) have g = -30 (a gate of about
         1e-13) on a random quarter of the key channels of each head (KDA),
         or on the head's scalar gate (GDN)

raw=True keeps the same draws as raw projections (q, k unnormalised, g and
beta untransformed) for the kernels' in-kernel preprocessing.  Decode inputs
(make_decode_case) draw one token per sequence the same way plus a state
pool; the decode workload is a 256-sequence serving batch with workload 1's
head shape.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CHUNK = 64


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); return them as fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).reshape(x.shape)


def _l2norm(x: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(x.astype(np.float32) ** 2, axis=-1, keepdims=True, dtype=np.float32))
    return (x / np.maximum(n, np.float32(1e-6))).astype(np.float32)


def _softplus(x: np.ndarray) -> np.ndarray:
    return np.logaddexp(np.float32(0), x).astype(np.float32)


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return (1.0 / (1.0 + np.exp(-x.astype(np.float64)))).astype(np.float32)


@dataclass
class Workload:
    name: str
    kind: str            # "gdn" or "kda"
    lengths: tuple       # per-sequence lengths (None -> drawn, varlen)
    Hqk: int
    Hv: int
    Dk: int
    Dv: int
    dtype: str           # "bf16" or "f32"
    with_s0: bool
    varlen_draw: tuple = ()   # (n_seq, lo, hi) when lengths are drawn
    notes: str = ""


WORKLOADS = {
    0: Workload("gdn_T256_H1_d64_f32", "gdn", (256,), 1, 1, 64, 64, "f32", False),
    1: Workload("gdn_T4096_H16_d128_bf16", "gdn", (4096,), 16, 16, 128, 128, "bf16", False),
    2: Workload("gdn_T32768_H16_d128_bf16_s0", "gdn", (32768,), 16, 16, 128, 128, "bf16", True),
    3: Workload("kda_T8192_H16_d128_bf16", "kda", (8192,), 16, 16, 128, 128, "bf16", False),
    4: Workload("gdn_varlen8_U512-8192_Hv32_Hqk16_d128_bf16_s0", "gdn", None, 16, 32, 128, 128,
                "bf16", True, varlen_draw=(8, 512, 8192)),
}


@dataclass
class Inputs:
    kind: str
    dtype: str
    q: np.ndarray        # [T, Hqk, Dk] fp32 holding dtype-representable values
    k: np.ndarray
    v: np.ndarray        # [T, Hv, Dv]
    g: np.ndarray        # [T, Hv] or [T, Hv, Dk] fp32
    beta: np.ndarray     # [T, Hv] fp32
    s0: np.ndarray | None  # [N, Hv, Dk, Dv] fp32
    cu_seqlens: np.ndarray  # int32 [N+1]
    scale: float = 1.0
    meta: dict = field(default_factory=dict)

    @property
    def T(self):
        return int(self.q.shape[0])

    @property
    def N(self):
        return int(self.cu_seqlens.shape[0] - 1)


def make_case(kind="gdn", lengths=(256,), Hqk=1, Hv=1, Dk=64, Dv=64, dtype="f32",
              with_s0=False, variant="base", seed=0, scale=1.0, varlen_draw=None,
              raw=False) -> Inputs:
    """Draw one seeded input set.  ``lengths`` may be None with ``varlen_draw``.

    raw=True returns the raw projections instead (same draws): q and k not
    normalised, g and beta the untransformed N(0,1) draws, for the kernels'
    in-kernel preprocessing (base variant only)."""
    if raw and variant != "base":
        raise ValueError("raw projections exist for the base variant only")
    rng = np.random.Generator(np.random.PCG64(seed))
    if lengths is None:
        n, lo, hi = varlen_draw
        lengths = tuple(int(x) for x in rng.integers(lo, hi, endpoint=True, size=n))
    lengths = tuple(int(x) for x in lengths)
    T = int(sum(lengths))
    cu = np.zeros(len(lengths) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lengths)
    N = len(lengths)

    q = rng.standard_normal((T, Hqk, Dk), dtype=np.float32)
    k = rng.standard_normal((T, Hqk, Dk), dtype=np.float32)
    v = rng.standard_normal((T, Hv, Dv), dtype=np.float32)
    gshape = (T, Hv) if kind == "gdn" else (T, Hv, Dk)
    g_raw = rng.standard_normal(gshape, dtype=np.float32)
    b_raw = rng.standard_normal((T, Hv), dtype=np.float32)
    s0 = None
    if with_s0 or variant == "s0":
        s0 = (np.float32(0.02) * rng.standard_normal((N, Hv, Dk, Dv), dtype=np.float32))

    if variant == "ks":
        basis = rng.standard_normal((Hqk, 4, Dk), dtype=np.float32)
        coef = k[:, :, :4]
        k = np.einsum("thc,hcd->thd", coef, basis).astype(np.float32)
    if not raw:
        q = _l2norm(q)
        k = _l2norm(k)

    if raw:
        g = g_raw
    elif variant in ("lm", "s0"):
        g = (np.float32(-0.01) * _softplus(g_raw)).astype(np.float32)
    elif variant == "dn":
        g = np.zeros(gshape, dtype=np.float32)
    elif variant == "lg":
        g = -_softplus(np.float32(3.0) * g_raw)
    elif variant == "fg":
        g = -_softplus(g_raw)
        lanes = [(h, None) for h in range(Hv)] if kind == "gdn" else \
            [(h, int(c)) for h in range(Hv) for c in rng.permutation(Dk)[:Dk // 4]]
        for n in range(N):
            for h, c in lanes:
                t = int(cu[n]) + int(rng.integers(0, 32))
                while t < cu[n + 1]:
                    run = int(rng.integers(8, 24, endpoint=True))
                    sl = slice(t, min(t + run, int(cu[n + 1])))
                    if c is None:
                        g[sl, h] = -30.0
                    else:
                        g[sl, h, c] = -30.0
                    t += run + int(rng.integers(8, 56, endpoint=True))
    else:
        g = -_softplus(g_raw)
    beta = np.ones((T, Hv), dtype=np.float32) if variant == "ks" else _sigmoid(b_raw)
    if raw:
        beta = b_raw

    if dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    elif dtype != "f32":
        raise ValueError(dtype)
    return Inputs(kind=kind, dtype=dtype, q=q, k=k, v=v, g=g.astype(np.float32),
                  beta=beta, s0=s0, cu_seqlens=cu, scale=float(scale),
                  meta=dict(seed=seed, variant=variant, lengths=lengths, raw=raw))


def make_workload(idx: int, variant: str = "base", seed: int | None = None,
                  kind: str | None = None, raw: bool = False) -> Inputs:
    w = WORKLOADS[idx]
    return make_case(kind=kind or w.kind, lengths=w.lengths, Hqk=w.Hqk, Hv=w.Hv, Dk=w.Dk,
                     Dv=w.Dv, dtype=w.dtype, with_s0=w.with_s0, variant=variant,
                     seed=1000 + idx if seed is None else seed,
                     varlen_draw=w.varlen_draw or None, raw=raw)


@dataclass
class DecodeInputs:
    kind: str
    dtype: str
    q: np.ndarray        # [N, Hqk, Dk]
    k: np.ndarray
    v: np.ndarray        # [N, Hv, Dv]
    g: np.ndarray        # [N, Hv] or [N, Hv, Dk]
    beta: np.ndarray     # [N, Hv]
    state: np.ndarray    # [S, Hv, Dk, Dv] fp32 pool
    slots: np.ndarray | None  # int32 [N] or None
    scale: float = 1.0
    meta: dict = field(default_factory=dict)


# Decode workload: one token for each of 256 sequences of a serving batch,
# with the prefill workload's head shape (H = 16, d = 128, bf16).
DECODE_WORKLOAD = dict(kind="gdn", N=256, Hqk=16, Hv=16, Dk=128, Dv=128, dtype="bf16")


def make_decode_case(kind="gdn", N=4, Hqk=1, Hv=1, Dk=64, Dv=64, dtype="f32", pool=None,
                     pad=0, seed=0, scale=1.0, raw=False) -> DecodeInputs:
    """One decode step's inputs: a token per sequence drawn like the prefill
    inputs, a state pool of ``pool`` slots (default N) of 0.1*N(0,1) values (a
    state a prefill left), and, when pool is given, a random slot per
    sequence (distinct) with ``pad`` entries set to -1 (padding)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    q = rng.standard_normal((N, Hqk, Dk), dtype=np.float32)
    k = rng.standard_normal((N, Hqk, Dk), dtype=np.float32)
    v = rng.standard_normal((N, Hv, Dv), dtype=np.float32)
    gshape = (N, Hv) if kind == "gdn" else (N, Hv, Dk)
    g_raw = rng.standard_normal(gshape, dtype=np.float32)
    b_raw = rng.standard_normal((N, Hv), dtype=np.float32)
    S = N if pool is None else int(pool)
    state = np.float32(0.1) * rng.standard_normal((S, Hv, Dk, Dv), dtype=np.float32)
    slots = None
    if pool is not None:
        if S < N - pad:
            raise ValueError("pool too small for the live sequences")
        slots = rng.permutation(S)[:N].astype(np.int32)
        if pad:
            slots[rng.choice(N, size=pad, replace=False)] = -1
    if raw:
        g, beta = g_raw, b_raw
    else:
        q, k = _l2norm(q), _l2norm(k)
        g, beta = -_softplus(g_raw), _sigmoid(b_raw)
    if dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    elif dtype != "f32":
        raise ValueError(dtype)
    return DecodeInputs(kind=kind, dtype=dtype, q=q, k=k, v=v, g=g.astype(np.float32),
                        beta=beta.astype(np.float32), state=state, slots=slots,
                        scale=float(scale), meta=dict(seed=seed, N=N, pool=S, pad=pad, raw=raw))
