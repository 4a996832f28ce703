"""GPU: the chunk-local factors the chunk-local kernel leaves in the workspace
(operators #1-#4 of paper Sec. 2.1 and the state-independent parts of #5 and
#6) against fp64 values of the independent chunked formulation
(tests/chunked_ref.py), read back through hagdn_workspace_region:

    NM = -Kt W,  B = Kt U~,  Q' = Q e^gamma - P W,  O_loc = P U~,  decay = e^gamma_last

with Kt = (K * e^(gamma_last - gamma))^T.  Each factor's max|gpu - ref| / max|ref|
over the call is printed (the per-kernel error budget) and bounded by the
end-to-end tolerance: 2e-2 for bf16 inputs, 1e-4 for fp32."""

import numpy as np
import pytest

from chunked_ref import chunk_step
from gpu_harness import TOL, relerr, say, to_device
from paper_2609_32114_amd.inputs import make_case

pytestmark = pytest.mark.gpu


def kmap(grp, j):
    return 4 * grp + j if j < 4 else 12 + 4 * grp + j


def dv_of(n, j):
    return 32 * (n >> 1) + 8 * (j >> 2) + 4 * (n & 1) + (j & 3)


def _frag_index(rows, kdim):
    """(position, row, k) of every element of a fragment-order matrix [rows, kdim]."""
    pos, r_, k_ = [], [], []
    kb_n = kdim // 32
    for t in range(rows // 16):
        for kb in range(kb_n):
            b = t * kb_n + kb
            for lane in range(64):
                col, grp = lane & 15, lane >> 4
                for j in range(8):
                    pos.append((b * 64 + lane) * 8 + j)
                    r_.append(16 * t + col)
                    k_.append(32 * kb + kmap(grp, j))
    return np.array(pos), np.array(r_), np.array(k_)


def _b_index(Dk, Dv):
    pos, r_, c_ = [], [], []
    for n in range(Dv // 16):
        for lane in range(64):
            col, grp = lane & 15, lane >> 4
            for m in range(Dk // 16):
                for e in range(4):
                    pos.append(((n * 64 + lane) * (Dk // 16) + m) * 4 + e)
                    r_.append(16 * m + 4 * grp + e)
                    c_.append(dv_of(n, col))
    return np.array(pos), np.array(r_), np.array(c_)


def _ol_index(Dv):
    pos, r_, c_ = [], [], []
    for m in range(Dv // 16):
        for lane in range(64):
            col, grp = lane & 15, lane >> 4
            for nt in range(4):
                for e in range(4):
                    pos.append(((m * 64 + lane) * 4 + nt) * 4 + e)
                    r_.append(16 * nt + col)
                    c_.append(dv_of(m, 4 * grp + e))
    return np.array(pos), np.array(r_), np.array(c_)


def _unpack(raw, idx, shape):
    pos, r, c = idx
    out = np.zeros(shape)
    out[r, c] = raw[pos]
    return out


CASES = [
    # kind, length, Hqk, Hv, Dk, Dv, dtype, variant
    ("gdn", 200, 1, 2, 128, 128, "bf16", "base"),
    ("kda", 200, 1, 2, 128, 128, "bf16", "base"),
    ("kda", 200, 1, 2, 128, 128, "bf16", "fg"),
    ("gdn", 130, 1, 1, 64, 128, "f32", "lm"),
    ("kda", 130, 2, 2, 128, 64, "f32", "base"),
    ("kda", 150, 1, 1, 64, 64, "f32", "fg"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-T{c[1]}-d{c[4]}x{c[5]}-{c[6]}-{c[7]}")
def test_chunk_local_factors(case):
    import torch
    import paper_2609_32114_amd as P
    kind, T, Hqk, Hv, Dk, Dv, dtype, variant = case
    inp = make_case(kind, (T,), Hqk, Hv, Dk, Dv, dtype, variant=variant, seed=17)
    d = to_device(inp)
    dt = P.HAGDN_BF16 if dtype == "bf16" else P.HAGDN_F32
    ws = torch.zeros(P.workspace_size(kind, 1, T, Hqk, Hv, Dk, Dv, dt), dtype=torch.uint8, device="cuda")
    fn = P.gdn_prefill if kind == "gdn" else P.kda_prefill
    fn(d["q"], d["k"], d["v"], d["g"], d["beta"], cu_seqlens=d["cu"], workspace=ws)
    torch.cuda.synchronize()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def region(r):
        off, n = P.workspace_region(kind, 1, T, Hqk, Hv, Dk, Dv, dt, r)
        t = ws[off:off + n].view(torch.float32 if r == P.WS_DECAY else tdt)
        return t.float().cpu().numpy().astype(np.float64)

    nm, bc, qp, ol, dec = (region(r) for r in (P.WS_NM, P.WS_B, P.WS_QP, P.WS_OLOC, P.WS_DECAY))
    i_nm, i_b, i_qp, i_ol = _frag_index(Dk, Dk), _b_index(Dk, Dv), _frag_index(64, Dk), _ol_index(Dv)
    got = {k: [] for k in ("NM", "B", "Qp", "Ol", "dec")}
    ref = {k: [] for k in got}
    grp = Hv // Hqk
    nch = (T + 63) // 64
    for c in range(nch):
        c0, c1 = 64 * c, min(64 * c + 64, T)
        n = c1 - c0
        for h in range(Hv):
            blk = c * Hv + h
            hk = h // grp
            r = chunk_step(kind, inp.q[c0:c1, hk].astype(np.float64), inp.k[c0:c1, hk].astype(np.float64),
                           inp.v[c0:c1, h].astype(np.float64), inp.g[c0:c1, h].astype(np.float64),
                           inp.beta[c0:c1, h].astype(np.float64), np.zeros((Dk, Dv)))
            gam = r["gamma"] if kind == "kda" else np.repeat(r["gamma"][:, None], Dk, axis=1)
            qe = inp.q[c0:c1, hk].astype(np.float64) * np.exp(gam)
            QP = np.zeros((64, Dk))
            QP[:n] = qe - r["P"] @ r["W"]
            OL = np.zeros((64, Dv))
            OL[:n] = r["P"] @ r["Ut"]
            ref["NM"].append(-r["Kt"].T @ r["W"])
            ref["B"].append(r["Kt"].T @ r["Ut"])
            ref["Qp"].append(QP)
            ref["Ol"].append(OL)
            ref["dec"].append(r["decay"] if kind == "kda" else r["decay"][:1])
            got["NM"].append(_unpack(nm[blk * Dk * Dk:(blk + 1) * Dk * Dk], i_nm, (Dk, Dk)))
            got["B"].append(_unpack(bc[blk * Dk * Dv:(blk + 1) * Dk * Dv], i_b, (Dk, Dv)))
            got["Qp"].append(_unpack(qp[blk * 64 * Dk:(blk + 1) * 64 * Dk], i_qp, (64, Dk)))
            got["Ol"].append(_unpack(ol[blk * 64 * Dv:(blk + 1) * 64 * Dv], i_ol, (64, Dv)))
            got["dec"].append(dec[blk * Dk:blk * Dk + (Dk if kind == "kda" else 1)])
    errs = {k: relerr(np.stack(got[k]), np.stack(ref[k])) for k in got}
    say(f"[gpu] chunk-local factors {case}: " + "  ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert np.all(np.isfinite(np.stack(got[k]))), k
        assert v <= TOL[dtype], f"{k}: max-rel {v:.3e}"
