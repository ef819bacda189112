"""Float64 oracle for packed variable-length exact self-attention.

TEST INFRASTRUCTURE ONLY. This module is imported by ``tests/``, by
``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of ``bench.py``;
nothing on the GPU path may import or call it.

What it computes
----------------
The paper trains with exact softmax attention (Flash Attention is enabled
for every run, Sec. 4.1 "Implementation details"); under Ulysses sequence
parallelism every device attends over the whole sequence with a subset of
the heads (Sec. 6.1, "Sequence parallelism").  A batch of variable-length
sequences packed back to back (the "packed parallel" layout of Sec. 1) is
described by prefix sums ``cu_seqlens``: sequence ``b`` owns token rows
``cu_seqlens[b] .. cu_seqlens[b+1]-1``.  Attention is block diagonal: a
query only ever sees keys of its own sequence.

For one sequence and one head, with ``s`` rows,
    S   = scale * Q K^T                       (s x s)
    causal: S_ij = -inf for j > i (the diagonal is kept)
    LSE_i = ln sum_j exp(S_ij)                (natural log)
    P   = exp(S - LSE)                        (rows sum to one)
    O   = P V
and, for the scalar loss l = <dO, O>, the analytic gradients
    dV  = P^T dO
    dP  = dO V^T
    Dlt_i = sum_j P_ij dP_ij
    dS  = P o (dP - Dlt)                      (softmax Jacobian)
    dQ  = scale * dS K
    dK  = scale * dS^T Q
This is the plain definition written out in float64; long sequences are
processed in blocks of query rows, each block still taking its softmax over
the full key row, so no step is an approximation.

Layout: q, k, v, o, do, dq, dk, dv are ``[T, H, D]``; lse is ``[H, T]``.
Rows beyond ``cu_seqlens[-1]`` are not outputs (left as zero / NaN).
"""

from __future__ import annotations

import numpy as np

_ROW_BLOCK = 1024


def _check(cu_seqlens, T):
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    if cu.ndim != 1 or cu.size < 1 or cu[0] != 0 or np.any(np.diff(cu) < 0) or cu[-1] > T:
        raise ValueError("cu_seqlens must start at 0, be non-decreasing and end within T")
    return cu


def _scores(Qb, K, scale, causal, row0):
    """Scores of query rows ``row0 .. row0+len(Qb)-1`` against every key."""
    S = scale * (Qb @ K.T)
    if causal:
        i = np.arange(row0, row0 + Qb.shape[0])[:, None]
        j = np.arange(K.shape[0])[None, :]
        S = np.where(j > i, -np.inf, S)
    return S


def _log_sum_exp_rows(S):
    mx = S.max(axis=1)
    return mx + np.log(np.exp(S - mx[:, None]).sum(axis=1))


def attention_forward(q, k, v, cu_seqlens, scale, causal=False, row_block=_ROW_BLOCK):
    """Return ``(o, lse)`` in float64 for packed sequences."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, H, D = q.shape
    cu = _check(cu_seqlens, T)
    o = np.zeros((T, H, D))
    lse = np.full((H, T), np.nan)
    for b in range(cu.size - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        for h in range(H):
            Q, K, V = q[s0:s1, h], k[s0:s1, h], v[s0:s1, h]
            for r0 in range(0, s1 - s0, row_block):
                r1 = min(s1 - s0, r0 + row_block)
                S = _scores(Q[r0:r1], K, scale, causal, r0)
                L = _log_sum_exp_rows(S)
                P = np.exp(S - L[:, None])
                o[s0 + r0:s0 + r1, h] = P @ V
                lse[h, s0 + r0:s0 + r1] = L
    return o, lse


def attention_backward(do, q, k, v, cu_seqlens, scale, causal=False, row_block=_ROW_BLOCK):
    """Return ``(dq, dk, dv)`` in float64 for the loss ``<dO, O>``."""
    do = np.asarray(do, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, H, D = q.shape
    cu = _check(cu_seqlens, T)
    dq = np.zeros((T, H, D))
    dk = np.zeros((T, H, D))
    dv = np.zeros((T, H, D))
    for b in range(cu.size - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        for h in range(H):
            Q, K, V, dO = q[s0:s1, h], k[s0:s1, h], v[s0:s1, h], do[s0:s1, h]
            dK = np.zeros_like(K)
            dV = np.zeros_like(V)
            for r0 in range(0, s1 - s0, row_block):
                r1 = min(s1 - s0, r0 + row_block)
                S = _scores(Q[r0:r1], K, scale, causal, r0)
                P = np.exp(S - _log_sum_exp_rows(S)[:, None])
                dOb = dO[r0:r1]
                dV += P.T @ dOb
                dP = dOb @ V.T
                Dlt = (P * dP).sum(axis=1)
                dS = P * (dP - Dlt[:, None])
                dq[s0 + r0:s0 + r1, h] = scale * (dS @ K)
                dK += scale * (dS.T @ Q[r0:r1])
            dk[s0:s1, h] = dK
            dv[s0:s1, h] = dV
    return dq, dk, dv


def _locate(cu, rows):
    """Sequence index of each packed token row."""
    b = np.searchsorted(cu, rows, side="right") - 1
    if np.any(rows < 0) or np.any(rows >= cu[-1]):
        raise ValueError("sampled rows must lie inside the packed sequences")
    return b


def _groups(cu, rows, heads):
    """Sampled (row, head) pairs grouped by (sequence, head): {(b, h): indices}."""
    seq = _locate(cu, rows)
    groups = {}
    for n, (h, b) in enumerate(zip(heads.tolist(), seq.tolist())):
        groups.setdefault((b, h), []).append(n)
    return groups


def _scores_at(Qr, K, scale, causal, pos):
    """Scores of query rows at sequence positions ``pos`` against every key
    of their sequence (key j masked for query i when j > pos_i, causal)."""
    S = scale * (Qr @ K.T)
    if causal:
        S = np.where(np.arange(K.shape[0])[None, :] > np.asarray(pos)[:, None], -np.inf, S)
    return S


def attention_rows(q, k, v, cu_seqlens, scale, causal, rows, heads, row_block=256):
    """O and LSE for the sampled (token row, head) pairs only.

    Each sampled output is the definition evaluated for that one query row
    over its full key row, so the cost is O(s*D) per sample however long its
    sequence is (rows of one (sequence, head) are evaluated together, in
    blocks of ``row_block``).  Returns ``(o_rows [n, D], lse_rows [n])``.
    """
    q = np.asarray(q)
    T = q.shape[0]
    cu = _check(cu_seqlens, T)
    rows = np.asarray(rows, dtype=np.int64)
    heads = np.asarray(heads, dtype=np.int64)
    o_rows = np.zeros((rows.size, q.shape[2]))
    lse_rows = np.zeros(rows.size)
    for (b, h), idx in _groups(cu, rows, heads).items():
        s0, s1 = int(cu[b]), int(cu[b + 1])
        K = np.asarray(k[s0:s1, h], dtype=np.float64)
        V = np.asarray(v[s0:s1, h], dtype=np.float64)
        idx = np.asarray(idx)
        for c0 in range(0, idx.size, row_block):
            sel = idx[c0:c0 + row_block]
            Qr = np.asarray(q[rows[sel], h], dtype=np.float64)
            S = _scores_at(Qr, K, scale, causal, rows[sel] - s0)
            L = _log_sum_exp_rows(S)
            o_rows[sel] = np.exp(S - L[:, None]) @ V
            lse_rows[sel] = L
    return o_rows, lse_rows


def attention_dq_rows(do, q, k, v, cu_seqlens, scale, causal, rows, heads, row_block=256):
    """dQ for the sampled (token row, head) pairs only (row-local: O(s*D)
    per row, over the row's full softmax)."""
    q = np.asarray(q)
    T = q.shape[0]
    cu = _check(cu_seqlens, T)
    rows = np.asarray(rows, dtype=np.int64)
    heads = np.asarray(heads, dtype=np.int64)
    out = np.zeros((rows.size, q.shape[2]))
    for (b, h), idx in _groups(cu, rows, heads).items():
        s0, s1 = int(cu[b]), int(cu[b + 1])
        K = np.asarray(k[s0:s1, h], dtype=np.float64)
        V = np.asarray(v[s0:s1, h], dtype=np.float64)
        idx = np.asarray(idx)
        for c0 in range(0, idx.size, row_block):
            sel = idx[c0:c0 + row_block]
            Qr = np.asarray(q[rows[sel], h], dtype=np.float64)
            dOr = np.asarray(do[rows[sel], h], dtype=np.float64)
            S = _scores_at(Qr, K, scale, causal, rows[sel] - s0)
            P = np.exp(S - _log_sum_exp_rows(S)[:, None])
            dP = dOr @ V.T
            dS = P * (dP - (P * dP).sum(axis=1)[:, None])
            out[sel] = scale * (dS @ K)
    return out


def attention_dkdv_rows(do, q, k, v, cu_seqlens, scale, causal, rows, heads, row_block=_ROW_BLOCK):
    """dK and dV for sampled (key row, head) pairs.

    A key's gradient depends on every query row of its sequence through that
    row's full softmax, so this evaluates the full rows (O(s^2*D) per distinct
    (sequence, head)) and keeps only the sampled key columns.
    Returns ``(dk_rows [n, D], dv_rows [n, D])``.
    """
    q = np.asarray(q)
    T = q.shape[0]
    cu = _check(cu_seqlens, T)
    rows = np.asarray(rows, dtype=np.int64)
    heads = np.asarray(heads, dtype=np.int64)
    seq = _locate(cu, rows)
    dk_rows = np.zeros((rows.size, q.shape[2]))
    dv_rows = np.zeros((rows.size, q.shape[2]))
    groups = {}
    for n, (h, b) in enumerate(zip(heads, seq)):
        groups.setdefault((int(b), int(h)), []).append(n)
    for (b, h), idx in groups.items():
        s0, s1 = int(cu[b]), int(cu[b + 1])
        cols = rows[idx] - s0
        Q = np.asarray(q[s0:s1, h], dtype=np.float64)
        K = np.asarray(k[s0:s1, h], dtype=np.float64)
        V = np.asarray(v[s0:s1, h], dtype=np.float64)
        dO = np.asarray(do[s0:s1, h], dtype=np.float64)
        dKc = np.zeros((cols.size, K.shape[1]))
        dVc = np.zeros((cols.size, K.shape[1]))
        for r0 in range(0, s1 - s0, row_block):
            r1 = min(s1 - s0, r0 + row_block)
            S = _scores(Q[r0:r1], K, scale, causal, r0)
            P = np.exp(S - _log_sum_exp_rows(S)[:, None])
            dP = dO[r0:r1] @ V.T
            dS = P * (dP - (P * dP).sum(axis=1)[:, None])
            dVc += P[:, cols].T @ dO[r0:r1]
            dKc += scale * (dS[:, cols].T @ Q[r0:r1])
        dk_rows[idx] = dKc
        dv_rows[idx] = dVc
    return dk_rows, dv_rows


def attention_dkdv_cols_given(do, q, k, v, cu_seqlens, scale, causal, rows, heads, lse, delta,
                              row_block=16384):
    """dK and dV for sampled (key row, head) pairs, given each query's LSE
    ([H, T]) and Delta_i = sum_j P_ij dP_ij ([H, T]) instead of recomputing
    them:
        P_ij  = exp(scale q_i . k_j - LSE_i)   (0 where j > i, causal)
        dV_j  = sum_i P_ij dO_i
        dK_j  = scale sum_i P_ij (dO_i . v_j - Delta_i) q_i
    the same definition with the row normalisers supplied.  The cost is
    O(s*D) per key, so key columns of sequences too long for the full-row
    evaluation of attention_dkdv_rows can be checked.  With the exact LSE
    and Delta it equals attention_dkdv_rows; given approximate ones the
    result moves by the same relative amount (|dP/P| = |dLSE|).
    Returns ``(dk_rows [n, D], dv_rows [n, D])``."""
    q = np.asarray(q)
    T = q.shape[0]
    cu = _check(cu_seqlens, T)
    rows = np.asarray(rows, dtype=np.int64)
    heads = np.asarray(heads, dtype=np.int64)
    dk_rows = np.zeros((rows.size, q.shape[2]))
    dv_rows = np.zeros((rows.size, q.shape[2]))
    for (b, h), idx in _groups(cu, rows, heads).items():
        s0, s1 = int(cu[b]), int(cu[b + 1])
        idx = np.asarray(idx)
        cols = rows[idx] - s0
        Kc = np.asarray(k[rows[idx], h], dtype=np.float64)
        Vc = np.asarray(v[rows[idx], h], dtype=np.float64)
        dKc = np.zeros((cols.size, Kc.shape[1]))
        dVc = np.zeros((cols.size, Kc.shape[1]))
        for r0 in range(0, s1 - s0, row_block):
            r1 = min(s1 - s0, r0 + row_block)
            Qb = np.asarray(q[s0 + r0:s0 + r1, h], dtype=np.float64)
            dOb = np.asarray(do[s0 + r0:s0 + r1, h], dtype=np.float64)
            Lb = np.asarray(lse[h, s0 + r0:s0 + r1], dtype=np.float64)
            Db = np.asarray(delta[h, s0 + r0:s0 + r1], dtype=np.float64)
            P = np.exp(scale * (Qb @ Kc.T) - Lb[:, None])
            if causal:
                P = np.where(cols[None, :] > np.arange(r0, r1)[:, None], 0.0, P)
            dS = P * (dOb @ Vc.T - Db[:, None])
            dVc += P.T @ dOb
            dKc += scale * (dS.T @ Qb)
        dk_rows[idx] = dKc
        dv_rows[idx] = dVc
    return dk_rows, dv_rows


def valid_pairs(cu_seqlens, causal=False):
    """Number of (query, key) pairs inside the diagonal blocks."""
    s = np.diff(np.asarray(cu_seqlens, dtype=np.int64))
    if causal:
        return int(np.sum(s * (s + 1) // 2))
    return int(np.sum(s * s))
