"""Algorithmic work and traffic of one chunkwise delta-rule prefill.

Counts per (token, value head) with chunk size C and head dims d_k, d_v; these
are the units the roofline fractions are quoted in.

MACs, chunkwise form (paper Sec. 2.1 operators #2-#6 and Sec. 5's GEMM set
KS, QS, KK^T, QK^T): KK^T, QK^T, T.(K*e^gamma), T.V and P.U each cost C*d per
token; W.H, K~^T.U and Q.H each cost d_k*d_v; the triangular solve costs about
C^2/2.  With C = 64 and d = 128 this is 92,160 MAC per token-head, which
reproduces the paper's Table 1 linear-attention MAC column exactly.

Bytes (algorithmic): what the method itself must move once -- read q, k, v,
gate, beta (and s0 when given), write o and the final state.
"""

from __future__ import annotations


def macs_per_token_head(C: int = 64, dk: int = 128, dv: int = 128) -> float:
    # the C*d terms: KK^T and QK^T contract over d_k; the T.K, T.V and P.U
    # terms produce d_k or d_v columns.
    cd = 2 * C * dk + C * dk + C * dv + C * dv
    dd = 3 * dk * dv
    return float(cd + dd + C * C / 2)


def flops(T_total: int, Hv: int, C: int = 64, dk: int = 128, dv: int = 128) -> float:
    return 2.0 * macs_per_token_head(C, dk, dv) * T_total * Hv


def algorithmic_bytes(T_total: int, N: int, Hqk: int, Hv: int, dk: int, dv: int,
                      elt_bytes: int, kda: bool, with_s0: bool) -> int:
    """q, k, v, o in the I/O dtype; g, beta fp32; s0 (if given) and s_final fp32."""
    per_token = (2 * Hqk * dk + 2 * Hv * dv) * elt_bytes          # q, k, v, o
    per_token += Hv * 4 * (dk if kda else 1) + Hv * 4              # gate, beta
    state = N * Hv * dk * dv * 4
    return per_token * T_total + state * (2 if with_s0 else 1)


def kernel_bytes(kernel: str, T_total: int, N: int, Hqk: int, Hv: int, dk: int, dv: int,
                 elt_bytes: int, kda: bool, with_s0: bool, chunk: int = 64, seg_chunks: int = 0) -> int:
    """Compulsory bytes of one kernel of the pipeline: every input it reads and
    every output it writes, each counted once.  Per-chunk blocks are counted per
    (chunk, value head); the timed workloads are single sequences with
    T % 64 == 0, so chunks = T / 64, cut into segments of seg_chunks chunks
    (0: one segment).

      chunk_index   cu_seqlens in; sequence, chunk and segment tables out
      chunk_local   q, k, v, gate, beta in; -M (dk x dk), B (dk x dv), Q' (64 x dk),
                    O_loc (64 x dv) and the chunk decay out
      seg_transfer  -M, B, decay of the chunks of every segment but the last in;
                    the segment maps A (dk x dk) and B_seg (dk x dv fp32) out
      state_prop    -M, B, decay, Q', O_loc, the segment maps and s0 in; o, s_final
                    out (operators #5 and #6)
      overlap_setup the overlapped launch's queues (2 KiB) and ready flags cleared
      overlapped    chunk_local and state_prop in one launch: q, k, v, gate, beta
                    and s0 in, o and s_final out; the factors pass between its
                    workgroups (through the L2 of their XCD) and are not counted
    """
    e = elt_bytes
    chunks = (T_total + chunk - 1) // chunk
    cb = chunks * Hv  # (chunk, value head) blocks
    gate = Hv * 4 * (dk if kda else 1)
    state = N * Hv * dk * dv * 4
    decb = (dk if kda else 1) * 4           # decay bytes per block
    L = seg_chunks if seg_chunks > 0 else max(chunks, 1)
    segs = max(1, -(-chunks // L))
    map_chunks = min(chunks, (segs - 1) * L)  # chunks of segments that have a map
    maps = (segs - 1) * Hv * (dk * dk * e + dk * dv * 4)
    if kernel == "chunk_index":
        return (N + 1) * 4 + N * 16 + (T_total // chunk + N) * 16 + 4 + N * 8 + (chunks // L + N) * 16
    if kernel == "chunk_local":
        rd = T_total * (2 * Hqk * dk * e + Hv * dv * e + gate + Hv * 4)
        wr = cb * ((dk * dk + dk * dv + chunk * dk + chunk * dv) * e + decb)
        return rd + wr
    if kernel == "seg_transfer":
        return map_chunks * Hv * ((dk * dk + dk * dv) * e + decb) + maps
    if kernel == "state_prop":
        rd = cb * ((dk * dk + dk * dv + chunk * dk + chunk * dv) * e + decb) + maps
        rd += state if with_s0 else 0
        wr = T_total * Hv * dv * e + state
        return rd + wr
    if kernel == "overlap_setup":
        return 2048 + cb * 4
    if kernel == "overlapped":
        rd = T_total * (2 * Hqk * dk * e + Hv * dv * e + gate + Hv * 4) + (state if with_s0 else 0)
        return rd + T_total * Hv * dv * e + state
    raise KeyError(kernel)


def decode_bytes(N: int, Hqk: int, Hv: int, dk: int, dv: int, elt_bytes: int, kda: bool,
                 slots: bool = False) -> int:
    """Compulsory bytes of one decode step over N live sequences: q, k, v, o of
    one token each (I/O dtype), gate and beta (fp32), and the fp32 state of
    every (sequence, value head) read once and written once (plus the slot
    indices when given)."""
    e = elt_bytes
    tok = N * (2 * Hqk * dk * e + 2 * Hv * dv * e + Hv * 4 * (dk if kda else 1) + Hv * 4)
    return tok + 2 * N * Hv * dk * dv * 4 + (4 * N if slots else 0)


def decode_flops(N: int, Hv: int, dk: int, dv: int) -> float:
    """Decay, H^T k, rank-1 update and H^T q: about 4 multiply-adds per state element."""
    return 8.0 * N * Hv * dk * dv
