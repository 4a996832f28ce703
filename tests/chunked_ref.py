"""Independent fp64 chunkwise formulation of delta-rule prefill (test helper).

This is the Map-Reduce-Map decomposition of the paper (Sec. 2.1, "Chunkwise
Map-Reduce-Map Execution": operators #1 Gate, #2 KKT, #3 Solve, #4 W/U in
the first Map; #5 H in the Reduce; #6 O in the final Map), derived here from
the token recurrence and written plainly in numpy.  It serves as a
brute-force cross-check of the token-by-token oracle (they must agree to
fp64 rounding for every chunk size) and as the fp64 reference for the GPU's
per-chunk intermediates.  It is not the oracle and shares no code with it.

For a chunk of n tokens with entering state H0 (d_k x d_v), gamma the
inclusive cumulative log-gate inside the chunk (op #1; a d_k-vector per token
for KDA):
  A[r,s] = b_r <k_r, exp(gamma_r - gamma_s) * k_s>   for s < r     (op #2)
  T      = (I + A)^-1                                              (op #3)
  W      = T Diag(b) (K * exp(gamma)),  U~ = T Diag(b) V           (op #4; W = A^-1 K, Sec. 5)
  U      = U~ - W H0                      (the "v_c" of op #5-read, Sec. 5)
  P[r,s] = <q_r, exp(gamma_r - gamma_s) * k_s>        for s <= r
  O      = scale ((Q * exp(gamma)) H0 + P U)                       (op #6)
  H1     = Diag(exp(gamma_n)) H0 + (K * exp(gamma_n - gamma))^T U  (op #5-update)
"""

import numpy as np
import scipy.linalg


def chunk_step(kind, q, k, v, g, beta, H0, scale=1.0):
    """One chunk for one head.  q,k [n,Dk]; v [n,Dv]; g [n] or [n,Dk]; beta [n]; H0 [Dk,Dv].
    Returns dict of every intermediate and (O, H1)."""
    n, Dk = k.shape
    gam = np.cumsum(g, axis=0)                                    # op #1
    if kind == "gdn":
        gam_k = np.repeat(gam[:, None], Dk, axis=1)
    else:
        gam_k = gam
    # pairwise decay exp(gamma_r - gamma_s) per channel, only for s <= r
    diff = gam_k[:, None, :] - gam_k[None, :, :]                  # [r, s, Dk]
    lower_incl = np.tril(np.ones((n, n), dtype=bool))
    dec = np.where(lower_incl[:, :, None], np.exp(np.where(lower_incl[:, :, None], diff, 0.0)), 0.0)
    KK = np.einsum("rd,rsd,sd->rs", k, dec, k)
    A = beta[:, None] * np.tril(KK, -1)                           # op #2
    T = scipy.linalg.solve_triangular(np.eye(n) + A, np.eye(n), lower=True, unit_diagonal=True)  # op #3
    Kg = k * np.exp(gam_k)
    W = T @ (beta[:, None] * Kg)                                  # op #4
    Ut = T @ (beta[:, None] * v)
    U = Ut - W @ H0                                               # op #5-read
    P = np.tril(np.einsum("rd,rsd,sd->rs", q, dec, k))
    O = scale * ((q * np.exp(gam_k)) @ H0 + P @ U)                # op #6
    last = gam_k[-1]
    Kt = k * np.exp(last[None, :] - gam_k)
    H1 = np.exp(last)[:, None] * H0 + Kt.T @ U                    # op #5-update
    return dict(gamma=gam, A=A, T=T, W=W, Ut=Ut, U=U, P=P, Kt=Kt, decay=np.exp(last), O=O, H1=H1)


def chunked_prefill(kind, q, k, v, g, beta, s0=None, cu_seqlens=None, scale=1.0, chunk=64):
    """Full prefill by chunks.  Same layouts as the oracle; returns (o, s_final) in fp64."""
    q, k, v, g, beta = (np.asarray(x, dtype=np.float64) for x in (q, k, v, g, beta))
    T_total, Hqk, Dk = q.shape
    Hv, Dv = v.shape[1:]
    cu = np.array([0, T_total]) if cu_seqlens is None else np.asarray(cu_seqlens)
    N = len(cu) - 1
    grp = Hv // Hqk
    o = np.zeros((T_total, Hv, Dv))
    sf = np.zeros((N, Hv, Dk, Dv))
    for n in range(N):
        for h in range(Hv):
            hk = h // grp
            H = np.zeros((Dk, Dv)) if s0 is None else np.array(s0[n, h], dtype=np.float64)
            for c0 in range(int(cu[n]), int(cu[n + 1]), chunk):
                c1 = min(c0 + chunk, int(cu[n + 1]))
                r = chunk_step(kind, q[c0:c1, hk], k[c0:c1, hk], v[c0:c1, h], g[c0:c1, h],
                               beta[c0:c1, h], H, scale)
                o[c0:c1, h] = r["O"]
                H = r["H1"]
            sf[n, h] = H
    return o, sf
