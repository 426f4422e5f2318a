"""Block-decomposition form of the SSD forward, float64 numpy -- TEST INFRASTRUCTURE ONLY.

Written from Section 6 (hardware-efficient SSD algorithm): the semiseparable
matrix M is cut into Q x Q blocks.  Its diagonal blocks are small SSMs computed
in the quadratic dual form (Section 5, eq. ssm-quad: M = L o (C B^T)); its
off-diagonal blocks factor into right factors (chunk-final states assuming a
zero initial state), centre factors (a scalar SSM scan over chunk totals, the
1-SS multiplication of eq. 1ss / Appendix B) and left factors (state -> output).
The last block may be shorter than Q (Section 6 notes uneven partitions are
valid).  Variable-length rows (Section 8.3) keep every quantity inside its own
sequence; sequences that start inside a chunk restart from their own initial
state.

This module writes the decomposition out step by step (returning its
intermediates: chunk states, entering states) so that the CPU tests can show
the block form equals the sequential oracle (``oracle.forward``) at every
chunk length, including ragged last chunks and packed rows -- the identity
the chunked kernels rely on.  It shares no code with the HIP path.
"""
from __future__ import annotations

import numpy as np


def _chunks(T, Q):
    return [(s, min(T, s + Q)) for s in range(0, T, Q)]


def forward(x, dt, A_log, B, C, D=None, initial_states=None, seq_idx=None,
            chunk_size=64, nseq=None):
    """Returns (y, final_states, intermediates).

    intermediates: dict with
      ``cs``      (b,H,nC,Q) chunk-local inclusive cumsum of a = dt*A (pad 0),
      ``S``       (b,nC,H,P,N) right factors (chunk states from zero, own sequence),
      ``h_in``    (b,nC,H,P,N) state entering each chunk (centre factors applied).
    """
    x, dt, A_log, B, C = (np.asarray(v, dtype=np.float64) for v in (x, dt, A_log, B, C))
    b, T, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    hpg = H // G
    Q = int(chunk_size)
    ch = _chunks(T, Q)
    nC = len(ch)
    D = np.zeros(H) if D is None else np.asarray(D, dtype=np.float64)
    if seq_idx is not None:
        q = np.asarray(seq_idx).reshape(-1).astype(np.int64)
        nseq = int(q[-1]) + 1 if nseq is None else nseq
        first = np.r_[True, q[1:] != q[:-1]]
        start_of = {int(q[t]): t for t in range(T) if first[t]}
        units = nseq
    else:
        q = None
        units = b
    init = (np.zeros((units, H, P, N)) if initial_states is None
            else np.asarray(initial_states, dtype=np.float64))
    A = -np.exp(A_log)

    y = np.zeros((b, T, H, P))
    fin = np.zeros((units, H, P, N))
    cs_all = np.zeros((b, H, nC, Q))
    S_all = np.zeros((b, nC, H, P, N))
    hin_all = np.zeros((b, nC, H, P, N))
    for bb in range(b):
        for h in range(H):
            g = h // hpg
            a = dt[bb, :, h] * A[h]                       # log-decay per token
            Xt = dt[bb, :, h, None] * x[bb, :, h, :]      # discretised input (T,P)
            h_prev = init[bb if q is None else int(q[0]), h].copy()
            for c, (s0, s1) in enumerate(ch):
                L = s1 - s0
                cs = np.cumsum(a[s0:s1])                  # chunk-local cumsum
                cs_all[bb, h, c, :L] = cs
                Cc, Bc, Xc = C[bb, s0:s1, g], B[bb, s0:s1, g], Xt[s0:s1]
                qc = None if q is None else q[s0:s1]
                # diagonal block: (L o C B^T) X, L_ts = exp(cs_t - cs_s), s <= t
                seg = cs[:, None] - cs[None, :]
                mask = np.tril(np.ones((L, L), dtype=bool))
                if qc is not None:
                    mask &= qc[:, None] == qc[None, :]
                Lmat = np.where(mask, np.exp(np.where(mask, seg, 0.0)), 0.0)
                y_diag = (Lmat * (Cc @ Bc.T)) @ Xc
                # right factor: state at the chunk end from a zero start,
                # restricted to the chunk's last sequence
                w = np.exp(cs[-1] - cs)
                if qc is not None:
                    w = np.where(qc == qc[-1], w, 0.0)
                S = (Xc * w[:, None]).T @ Bc              # (P,N)
                S_all[bb, c, h] = S
                hin_all[bb, c, h] = h_prev
                # left factor: incoming state of each token's sequence
                y_off = np.zeros((L, P))
                if qc is None:
                    y_off = np.exp(cs)[:, None] * (Cc @ h_prev.T)
                else:
                    for t in range(L):
                        qt = int(qc[t])
                        st = start_of[qt]
                        if st < s0 or (s0 == 0 and st == 0):
                            inc, base = h_prev, 0.0
                        else:
                            inc, base = init[qt, h], (cs[st - s0 - 1] if st > s0 else 0.0)
                        y_off[t] = np.exp(cs[t] - base) * (inc @ Cc[t])
                y[bb, s0:s1, h] = y_diag + y_off + D[h] * x[bb, s0:s1, h]
                # centre factor: scan step over the chunk
                if qc is None:
                    h_new = np.exp(cs[-1]) * h_prev + S
                else:
                    ql = int(qc[-1])
                    st = start_of[ql]
                    if st < s0 or (s0 == 0 and st == 0):
                        h_new = np.exp(cs[-1]) * h_prev + S
                    else:
                        base = cs[st - s0 - 1] if st > s0 else 0.0
                        h_new = np.exp(cs[-1] - base) * init[ql, h] + S
                    # final states of sequences that end inside this chunk
                    for t in range(L - 1):
                        if qc[t + 1] != qc[t]:
                            qt = int(qc[t])
                            st = start_of[qt]
                            if st < s0 or (s0 == 0 and st == 0):
                                inc, base = h_prev, 0.0
                            else:
                                inc, base = init[qt, h], (cs[st - s0 - 1] if st > s0 else 0.0)
                            sel = np.arange(L) <= t
                            sel &= qc == qt
                            we = np.where(sel, np.exp(cs[t] - cs), 0.0)
                            fin[qt, h] = np.exp(cs[t] - base) * inc + (Xc * we[:, None]).T @ Bc
                    # a sequence ending on the chunk's last token
                    if s1 == T or q[s1] != ql:
                        fin[ql, h] = h_new
                h_prev = h_new
            fin[bb if q is None else int(q[-1]), h] = h_prev
    return y, fin, {"cs": cs_all, "S": S_all, "h_in": hin_all}
