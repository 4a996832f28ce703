"""Helpers for GPU parity tests: move seeded inputs to the device, run the HIP
path through the C ABI, run the oracle on the same values, compare."""

import os
import sys

import numpy as np

import oracle
from paper_2609_32114_amd.inputs import Inputs

# max|gpu - ref| / max|ref| per tensor: fp32 inputs 1e-4, bf16 inputs (fp32 state
# and accumulation) 2e-2, on outputs and final states alike.
TOL = {"f32": 1e-4, "bf16": 2e-2}

# every comparison made in this process: (label, dtype, kind, max-rel o, max-rel s, nmse o, nmse s)
RESULTS = []


def oracle_threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return 8


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(inp: Inputs):
    import torch
    dt = torch.bfloat16 if inp.dtype == "bf16" else torch.float32
    dev = "cuda"
    t = lambda x, d=torch.float32: torch.from_numpy(np.ascontiguousarray(x)).to(dev).to(d)
    return dict(q=t(inp.q, dt), k=t(inp.k, dt), v=t(inp.v, dt), g=t(inp.g), beta=t(inp.beta),
                s0=None if inp.s0 is None else t(inp.s0),
                cu=torch.from_numpy(inp.cu_seqlens.astype(np.int32)).to(dev))


def run_gpu(inp: Inputs, dev=None, **kw):
    import torch
    import paper_2609_32114_amd as P
    d = dev or to_device(inp)
    fn = P.gdn_prefill if inp.kind == "gdn" else P.kda_prefill
    o, sf = fn(d["q"], d["k"], d["v"], d["g"], d["beta"], initial_state=d["s0"],
               cu_seqlens=d["cu"], scale=inp.scale, **kw)
    torch.cuda.synchronize()
    o64 = o.float().cpu().numpy().astype(np.float64)
    sf64 = None if sf is None else sf.cpu().numpy().astype(np.float64)
    return o64, sf64


def relerr(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(a - ref))) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def nmse(a, ref):
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.sum(ref * ref))
    return float(np.sum((np.asarray(a) - ref) ** 2) / den) if den > 0 else 0.0


def sub_heads(inp: Inputs, heads):
    """The same problem restricted to value heads `heads` (each gets its own q/k head)."""
    Hqk, Hv = inp.q.shape[1], inp.v.shape[1]
    grp = Hv // Hqk
    hk = [h // grp for h in heads]
    return Inputs(kind=inp.kind, dtype=inp.dtype, q=inp.q[:, hk], k=inp.k[:, hk],
                  v=inp.v[:, heads], g=inp.g[:, heads], beta=inp.beta[:, heads],
                  s0=None if inp.s0 is None else inp.s0[:, heads], cu_seqlens=inp.cu_seqlens,
                  scale=inp.scale, meta=dict(inp.meta, heads=list(heads)))


def check_against_oracle(inp: Inputs, heads=None, tol=None, label=""):
    """Run both sides; compare all heads, or only `heads` (oracle on those heads alone)."""
    tol = tol if tol is not None else TOL[inp.dtype]
    say(f"[gpu] {label} kind={inp.kind} dtype={inp.dtype} T={inp.T} N={inp.N} "
        f"q={inp.q.shape} v={inp.v.shape} heads={heads} meta={inp.meta}")
    o, sf = run_gpu(inp)
    ref_inp = inp if heads is None else sub_heads(inp, heads)
    ro, rs = oracle.run_inputs(ref_inp, nthreads=oracle_threads())
    if heads is not None:
        o, sf = o[:, heads], sf[:, heads]
    eo, es = relerr(o, ro), relerr(sf, rs)
    no, ns = nmse(o, ro), nmse(sf, rs)
    say(f"       max-rel o={eo:.3e} s={es:.3e}  nmse o={no:.3e} s={ns:.3e}")
    RESULTS.append((label, inp.dtype, inp.kind, eo, es, no, ns))
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(sf))
    assert eo <= tol, f"{label}: output max-rel {eo:.3e} > {tol}"
    assert es <= tol, f"{label}: state max-rel {es:.3e} > {tol}"
    return eo, es
