"""fp64 CPU oracle for delta-rule linear-attention prefill (GDN and KDA).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU product path never imports
this package.

The arithmetic lives in ``oracle.c`` (plain C, fp64, token by token; see its
header for the definition and the paper passages it follows).  This module
only builds that file with gcc and marshals numpy arrays into it.

Pins: every function here is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle.py`` (closed forms, invariants, special cases, brute
force, planted-mistake builds), ``tests/test_chunked_ref.py`` (an
independent chunkwise fp64 formulation) and ``tests/test_oracle_pre_decode.py``
(preprocessing against library routines and closed forms, with its own
planted-mistake builds; decode against the prefill handoff, the one-token
closed form and the slot mapping).  No function is "parity unpinned".
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_CFLAGS = ["-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
           "-fno-fast-math", "-ffp-contract=off"]


def compile_source(src: str, out: str) -> str:
    """Compile a C source with the oracle's flags into shared library ``out``."""
    tmp = out + ".tmp"
    subprocess.run(["gcc", *_CFLAGS, src, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc -O2 -fopenmp, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(SOURCE):
        compile_source(SOURCE, _LIB)
    return _LIB


def load_library(path: str):
    """Load a compiled oracle library (the default one, or a test's planted-mistake build)."""
    lib = ctypes.CDLL(path)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int)
    for name in ("oracle_gdn_prefill", "oracle_kda_prefill"):
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = [dp, dp, dp, dp, dp, dp, ip, ctypes.c_int, ctypes.c_int,
                       ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                       ctypes.c_double, dp, dp, ctypes.c_int]
    fn = lib.oracle_preprocess
    fn.restype = ctypes.c_int
    fn.argtypes = [dp, dp, dp, dp] + [ctypes.c_int] * 6
    return lib


def _default_lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = load_library(_LIB)
    return _lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


# Preprocessing flags (oracle_preprocess in oracle.c).
PRE_QK_L2NORM, PRE_GATE_SOFTPLUS, PRE_BETA_SIGMOID = 1, 2, 4


def preprocess(kind: str, q, k, g, beta, flags: int, lib=None):
    """Raw projections -> recurrence inputs (fp64 copies; see oracle_preprocess).

    flags: PRE_QK_L2NORM (q, k / max(||.||, 1e-6) per token and head),
    PRE_GATE_SOFTPLUS (g -> -softplus(g)), PRE_BETA_SIGMOID (beta -> sigmoid).
    Returns (q, k, g, beta) as new fp64 arrays.
    """
    if kind not in ("gdn", "kda"):
        raise ValueError(kind)
    q, k, g, beta = (np.array(x, dtype=np.float64, copy=True, order="C") for x in (q, k, g, beta))
    T, Hqk, Dk = q.shape
    Hv = beta.shape[1]
    lib = lib if lib is not None else _default_lib()
    rc = lib.oracle_preprocess(_ptr(q), _ptr(k), _ptr(g), _ptr(beta), T, Hqk, Hv, Dk,
                               int(kind == "kda"), int(flags))
    if rc != 0:
        raise ValueError("oracle_preprocess rejected its arguments")
    return q, k, g, beta


def prefill(kind: str, q, k, v, g, beta, s0=None, cu_seqlens=None, scale=1.0,
            nthreads: int = 0, lib=None, pre: int = 0):
    """Run the oracle.

    Arrays follow the library layouts (any float dtype; widened exactly to fp64):
      q, k [T, Hqk, Dk]; v [T, Hv, Dv]; g [T, Hv] (gdn) or [T, Hv, Dk] (kda);
      beta [T, Hv]; s0 [N, Hv, Dk, Dv] or None; cu_seqlens int [N+1] or None
      (None means a single sequence of length T).
    pre: preprocessing flags applied to q, k, g, beta first (``preprocess``).
    Returns (o [T, Hv, Dv] fp64, s_final [N, Hv, Dk, Dv] fp64).
    """
    if kind not in ("gdn", "kda"):
        raise ValueError(kind)
    if pre:
        q, k, g, beta = preprocess(kind, q, k, g, beta, pre, lib=lib)
    q, k, v, g, beta = (_f64(x) for x in (q, k, v, g, beta))
    T, Hqk, Dk = q.shape
    Hv, Dv = v.shape[1], v.shape[2]
    if cu_seqlens is None:
        cu = np.array([0, T], dtype=np.int32)
    else:
        cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    N = cu.shape[0] - 1
    s0c = None if s0 is None else _f64(s0)
    if s0c is not None and s0c.shape != (N, Hv, Dk, Dv):
        raise ValueError(f"s0 shape {s0c.shape} != {(N, Hv, Dk, Dv)}")
    o = np.zeros((T, Hv, Dv), dtype=np.float64)
    sf = np.zeros((N, Hv, Dk, Dv), dtype=np.float64)
    lib = lib if lib is not None else _default_lib()
    fn = lib.oracle_gdn_prefill if kind == "gdn" else lib.oracle_kda_prefill
    rc = fn(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(s0c),
            cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), N, T, Hqk, Hv, Dk, Dv,
            float(scale), _ptr(o), _ptr(sf), int(nthreads))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return o, sf


def gdn_prefill(q, k, v, g, beta, s0=None, cu_seqlens=None, scale=1.0, nthreads=0):
    return prefill("gdn", q, k, v, g, beta, s0, cu_seqlens, scale, nthreads)


def kda_prefill(q, k, v, g, beta, s0=None, cu_seqlens=None, scale=1.0, nthreads=0):
    return prefill("kda", q, k, v, g, beta, s0, cu_seqlens, scale, nthreads)


def decode(kind: str, q, k, v, g, beta, state, scale=1.0, slots=None, pre: int = 0,
           nthreads: int = 0, lib=None):
    """One decode step: one token for each of N sequences (paper Sec. 2.1: the
    token-by-token recurrence serves decoding).

    q, k [N, Hqk, Dk]; v [N, Hv, Dv]; g [N, Hv] (gdn) or [N, Hv, Dk] (kda);
    beta [N, Hv]; state [S, Hv, Dk, Dv], the pool the sequences' states live in;
    slots int [N] or None (None: sequence n uses slot n).  A slot outside
    [0, S) marks a padding entry: its output row is zero and no state changes.
    This is the oracle's prefill with every sequence one token long, started
    from the sequence's state.  Returns (o [N, Hv, Dv], new state pool), fp64.
    """
    state = np.array(state, dtype=np.float64, copy=True)
    N = np.shape(q)[0]
    S = state.shape[0]
    slots = np.arange(N) if slots is None else np.asarray(slots, dtype=np.int64)
    live = (slots >= 0) & (slots < S)
    idx = np.nonzero(live)[0]
    Hv, Dv = np.shape(v)[1], np.shape(v)[2]
    o = np.zeros((N, Hv, Dv), dtype=np.float64)
    if idx.size == 0:
        return o, state
    sel = lambda x: np.asarray(x)[idx]
    cu = np.arange(idx.size + 1, dtype=np.int32)
    ol, sf = prefill(kind, sel(q), sel(k), sel(v), sel(g), sel(beta), state[slots[idx]], cu,
                     scale, nthreads=nthreads, lib=lib, pre=pre)
    o[idx] = ol
    state[slots[idx]] = sf
    return o, state


def run_inputs(inp, nthreads: int = 0, pre: int = 0):
    """Run the oracle on an ``Inputs`` record from the seeded generator module."""
    return prefill(inp.kind, inp.q, inp.k, inp.v, inp.g, inp.beta, inp.s0,
                   inp.cu_seqlens, inp.scale, nthreads, pre=pre)
