"""Oracle: causal softmax attention with grouped key/value heads, float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Definition followed (Section 2.1, "Multi-head Attention"): for head ``h`` and
query position ``i`` the output is softmax(Q_i . K_{<=i} / sqrt(d_h)) . V_{<=i},
where d_h is the per-head query width.  Grouped-query attention (same section)
lets G consecutive query heads share one key/value head, so query head ``h``
reads key/value head ``h // G`` (the grouping of the scheduling example in
Section 4.1: Q0..Q3 all use K0).

Layouts (the per-device layout after the Ulysses re-layout of Section 3.1):
    q   [S, Hq, d]      k, v [S, Hkv, d]      o [S, Hq, d]
    lse [Hq, S]  natural-log log-sum-exp of the scaled scores of each row

Softmax is evaluated the plain way: the full score row is materialised,
its maximum subtracted, exponentiated and normalised.  Rows are processed in
blocks only to bound memory; rows are independent, so the block size does not
change any row's arithmetic.  With ``causal`` true, key j is visible to query
i iff j <= i (the diagonal is included, "K_{<=i}").

The backward pass is the analytic gradient of that definition:
    P_ij  = exp(s_ij - lse_i),  s_ij = q_i.k_j / sqrt(d)
    D_i   = sum_j P_ij (dO_i . v_j) = dO_i . o_i
    dS_ij = P_ij (dO_i . v_j - D_i)
    dQ_i  = sum_j dS_ij k_j / sqrt(d)
    dK_j  = sum_{h in group} sum_i dS_ij q_i / sqrt(d)
    dV_j  = sum_{h in group} sum_i P_ij dO_i
"""

import numpy as np

ROW_BLOCK = 256


def _check(q, k, v):
    if q.ndim != 3 or k.ndim != 3 or v.ndim != 3:
        raise ValueError("q, k, v must be [S, H, d]")
    S, Hq, d = q.shape
    if k.shape != v.shape or k.shape[0] != S or k.shape[2] != d:
        raise ValueError("k, v must be [S, Hkv, d] matching q")
    Hkv = k.shape[1]
    if Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    return S, Hq, Hkv, d


def kv_head_of(h, Hq, Hkv):
    """Key/value head read by query head ``h``: consecutive groups of G."""
    return h // (Hq // Hkv)


def _scores(q_rows, rows, k_h, causal, d):
    """Scaled scores of the given query rows against the keys they may see.

    Returns (s, n) where s is [len(rows), n] and keys >= n are invisible to
    every row in the block (causal); masked entries inside are -inf.
    """
    n = int(rows.max()) + 1 if causal else k_h.shape[0]
    s = (q_rows @ k_h[:n].T) / np.sqrt(d)
    if causal:
        s = np.where(np.arange(n)[None, :] > rows[:, None], -np.inf, s)
    return s, n


def attn_fwd(q, k, v, causal=True, rows=None):
    """Forward of attention for all rows (or the listed query ``rows``).

    Returns ``o`` [len(rows), Hq, d] and ``lse`` [Hq, len(rows)], float64.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    S, Hq, Hkv, d = _check(q, k, v)
    rows = np.arange(S) if rows is None else np.asarray(rows, np.int64)
    o = np.zeros((len(rows), Hq, d))
    lse = np.zeros((Hq, len(rows)))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for b0 in range(0, len(rows), ROW_BLOCK):
            r = rows[b0:b0 + ROW_BLOCK]
            s, n = _scores(q[r, h, :], r, k[:, g, :], causal, d)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            l = e.sum(axis=1, keepdims=True)
            o[b0:b0 + len(r), h, :] = (e / l) @ v[:n, g, :]
            lse[h, b0:b0 + len(r)] = (m + np.log(l))[:, 0]
    return o, lse


def attn_bwd(q, k, v, do, causal=True):
    """Gradients (dq, dk, dv) of attention for the upstream gradient ``do``.

    The oracle recomputes its own o and lse from (q, k, v); it takes nothing
    from the code under test.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    do = np.asarray(do, np.float64)
    S, Hq, Hkv, d = _check(q, k, v)
    o, lse = attn_fwd(q, k, v, causal)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    scale = 1.0 / np.sqrt(d)
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        D = np.sum(do[:, h, :] * o[:, h, :], axis=1)
        for b0 in range(0, S, ROW_BLOCK):
            r = np.arange(b0, min(S, b0 + ROW_BLOCK))
            s, n = _scores(q[r, h, :], r, k[:, g, :], causal, d)
            p = np.exp(s - lse[h, r][:, None])
            dp = do[r, h, :] @ v[:n, g, :].T
            ds = p * (dp - D[r][:, None])
            dq[r, h, :] = (ds @ k[:n, g, :]) * scale
            dk[:n, g, :] += (ds.T @ q[r, h, :]) * scale
            dv[:n, g, :] += p.T @ do[r, h, :]
    return dq, dk, dv


def attn_bwd_rows(q, k, v, do, rows, causal=True):
    """dQ and D at the listed query rows only.

    dQ_i depends on row i alone (through o_i, lse_i and D_i), so a subset of
    rows is exact.  Returns (dq [len(rows), Hq, d], D [Hq, len(rows)]).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    do = np.asarray(do, np.float64)
    S, Hq, Hkv, d = _check(q, k, v)
    rows = np.asarray(rows, np.int64)
    o, lse = attn_fwd(q, k, v, causal, rows=rows)
    dq = np.zeros((len(rows), Hq, d))
    Dout = np.zeros((Hq, len(rows)))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for b0 in range(0, len(rows), ROW_BLOCK):
            r = rows[b0:b0 + ROW_BLOCK]
            sl = slice(b0, b0 + len(r))
            D = np.sum(do[r, h, :] * o[sl, h, :], axis=1)
            s, n = _scores(q[r, h, :], r, k[:, g, :], causal, d)
            p = np.exp(s - lse[h, sl][:, None])
            dp = do[r, h, :] @ v[:n, g, :].T
            ds = p * (dp - D[:, None])
            dq[sl, h, :] = (ds @ k[:n, g, :]) / np.sqrt(d)
            Dout[h, sl] = D
    return dq, Dout


def attn_bwd_key_tail(q, k, v, do, j0):
    """dK and dV for the key positions j >= j0 of causal attention, exactly.

    Under the causal mask only queries i >= j contribute to key j, so the
    tail [j0, S) needs the query rows [j0, S) (each with its full row
    softmax).  Returns (dk [S-j0, Hkv, d], dv [S-j0, Hkv, d]).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    do = np.asarray(do, np.float64)
    S, Hq, Hkv, d = _check(q, k, v)
    rows = np.arange(j0, S)
    o, lse = attn_fwd(q, k, v, True, rows=rows)
    dk = np.zeros((S - j0, Hkv, d))
    dv = np.zeros((S - j0, Hkv, d))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for b0 in range(0, len(rows), ROW_BLOCK):
            r = rows[b0:b0 + ROW_BLOCK]
            sl = slice(b0, b0 + len(r))
            D = np.sum(do[r, h, :] * o[sl, h, :], axis=1)
            s, n = _scores(q[r, h, :], r, k[:, g, :], True, d)
            p = np.exp(s - lse[h, sl][:, None])
            dp = do[r, h, :] @ v[:n, g, :].T
            ds = p * (dp - D[:, None])
            dk[:n - j0, g, :] += (ds[:, j0:].T @ q[r, h, :]) / np.sqrt(d)
            dv[:n - j0, g, :] += p[:, j0:].T @ do[r, h, :]
    return dk, dv


def attn_fwd_chunked(q, k, v, U, causal=True):
    """Forward evaluated head chunk by head chunk (Section 3.3).

    Chunk c holds the local query heads [c*U, (c+1)*U); its heads read the
    same key/value heads as in the unchunked call.  The result is assembled
    into one preallocated output, as the paper fills ``final_out`` slot by
    slot.  Heads are independent, so this equals ``attn_fwd`` exactly.
    """
    S, Hq, Hkv, d = _check(np.asarray(q), np.asarray(k), np.asarray(v))
    if Hq % U != 0:
        raise ValueError("U must divide Hq")
    G = Hq // Hkv
    o = np.zeros((S, Hq, d))
    lse = np.zeros((Hq, S))
    for c in range(Hq // U):
        heads = list(range(c * U, (c + 1) * U))
        kvs = sorted({h // G for h in heads})
        kv_index = {g: t for t, g in enumerate(kvs)}
        # The chunk's own GQA problem: its U query heads with their kv heads.
        qc = np.asarray(q, np.float64)[:, heads, :]
        kc = np.asarray(k, np.float64)[:, kvs, :]
        vc = np.asarray(v, np.float64)[:, kvs, :]
        for u, h in enumerate(heads):
            oc, lc = attn_fwd(qc[:, [u], :], kc[:, [kv_index[h // G]], :],
                              vc[:, [kv_index[h // G]], :], causal)
            o[:, h, :] = oc[:, 0, :]
            lse[h, :] = lc[0]
    return o, lse


def attn_bwd_chunked(q, k, v, do, U, causal=True):
    """Backward head chunk by head chunk; dK/dV accumulate across chunks.

    The key/value gradients of a group are summed over the chunks that hold
    its query heads (Appendix A: the per-group dK, dV accumulators persist
    across stages).  Equal to ``attn_bwd`` up to float64 summation order.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    do = np.asarray(do, np.float64)
    S, Hq, Hkv, d = _check(q, k, v)
    G = Hq // Hkv
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for c in range(Hq // U):
        for h in range(c * U, (c + 1) * U):
            g = h // G
            a, b, e = attn_bwd(q[:, [h], :], k[:, [g], :], v[:, [g], :],
                               do[:, [h], :], causal)
            dq[:, h, :] = a[:, 0, :]
            dk[:, g, :] += b[:, 0, :]
            dv[:, g, :] += e[:, 0, :]
    return dq, dk, dv


def attn_rows_at(q_rows, pos, k, v, do_rows=None, causal=True):
    """Forward (and dQ, D when ``do_rows`` is given) for query rows supplied
    directly with their sequence positions ``pos``.

    The same definition as ``attn_fwd`` / ``attn_bwd_rows``; only the listed
    rows of q (and dO) are ever needed, so callers with very long sequences
    pass just those rows.  Returns (o, lse) or (o, lse, dq, D) with the row
    axis first for o and dq, and [Hq, rows] for lse and D.
    """
    q_rows = np.asarray(q_rows, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    pos = np.asarray(pos, np.int64)
    R, Hq, d = q_rows.shape
    Hkv = k.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    o = np.zeros((R, Hq, d))
    lse = np.zeros((Hq, R))
    want_grad = do_rows is not None
    if want_grad:
        do_rows = np.asarray(do_rows, np.float64)
        dq = np.zeros((R, Hq, d))
        Dout = np.zeros((Hq, R))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for b0 in range(0, R, ROW_BLOCK):
            sl = slice(b0, min(R, b0 + ROW_BLOCK))
            s, n = _scores(q_rows[sl, h, :], pos[sl], k[:, g, :], causal, d)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            l = e.sum(axis=1, keepdims=True)
            o[sl, h, :] = (e / l) @ v[:n, g, :]
            lse[h, sl] = (m + np.log(l))[:, 0]
            if want_grad:
                D = np.sum(do_rows[sl, h, :] * o[sl, h, :], axis=1)
                p = np.exp(s - lse[h, sl][:, None])
                dp = do_rows[sl, h, :] @ v[:n, g, :].T
                ds = p * (dp - D[:, None])
                dq[sl, h, :] = (ds @ k[:n, g, :]) / np.sqrt(d)
                Dout[h, sl] = D
    if want_grad:
        return o, lse, dq, Dout
    return o, lse


def attn_key_tail_at(q_tail, do_tail, k, v, j0):
    """dK, dV of causal attention for keys [j0, S) from the query and
    upstream-gradient rows [j0, S) only (same definition as
    ``attn_bwd_key_tail``)."""
    q_tail = np.asarray(q_tail, np.float64)
    do_tail = np.asarray(do_tail, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    S, Hkv, d = k.shape
    Hq = q_tail.shape[1]
    pos = np.arange(j0, S)
    dk = np.zeros((S - j0, Hkv, d))
    dv = np.zeros((S - j0, Hkv, d))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for b0 in range(0, len(pos), ROW_BLOCK):
            sl = slice(b0, min(len(pos), b0 + ROW_BLOCK))
            s, n = _scores(q_tail[sl, h, :], pos[sl], k[:, g, :], True, d)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            l = e.sum(axis=1, keepdims=True)
            o = (e / l) @ v[:n, g, :]
            lse = m + np.log(l)
            D = np.sum(do_tail[sl, h, :] * o, axis=1)
            p = np.exp(s - lse)
            dp = do_tail[sl, h, :] @ v[:n, g, :].T
            ds = p * (dp - D[:, None])
            dk[:n - j0, g, :] += (ds[:, j0:].T @ q_tail[sl, h, :]) / np.sqrt(d)
            dv[:n - j0, g, :] += p[:, j0:].T @ do_tail[sl, h, :]
    return dk, dv


def attn_key_cols_given(q, do, k, v, o, lse, cols, causal=True, row_block=4096):
    """dK and dV at the listed key columns, given each query row's lse and o.

    The Section 2.1 gradient for key j of key/value head g:
        dV_j = sum_{h in group g} sum_{i sees j} P_ij dO_i
        dK_j = sum_{h in group g} sum_{i sees j} P_ij (dO_i.v_j - D_i) q_i / sqrt(d)
    with P_ij = exp(q_i.k_j / sqrt(d) - lse_i) and D_i = dO_i . o_i.  Unlike
    ``attn_bwd`` the row statistics lse [Hq, S] and the output o [S, Hq, d]
    are the caller's: with the oracle's own they give exactly the oracle's
    gradient; with another implementation's they give that implementation's
    gradient as it should be for its own statistics ("conditioned" on them),
    which isolates the error of its key-gradient accumulation.  Only the
    listed columns are formed, so one column costs O(S Hq d) work at any
    length.  q, do, o may be any float arrays; rows are taken to float64 in
    blocks of ``row_block``.  Returns (dk, dv), each [len(cols), Hkv, d].
    """
    cols = np.asarray(cols, np.int64)
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    kc = np.asarray(k[cols], np.float64)
    vc = np.asarray(v[cols], np.float64)
    lse = np.asarray(lse, np.float64)
    dk = np.zeros((len(cols), Hkv, d))
    dv = np.zeros((len(cols), Hkv, d))
    lo = int(cols.min()) if causal else 0
    for b0 in range(lo, S, row_block):
        b1 = min(S, b0 + row_block)
        r = np.arange(b0, b1)
        qb = np.asarray(q[b0:b1], np.float64)
        dob = np.asarray(do[b0:b1], np.float64)
        ob = np.asarray(o[b0:b1], np.float64)
        vis = cols[None, :] <= r[:, None] if causal else np.ones((len(r), len(cols)), bool)
        for h in range(Hq):
            g = kv_head_of(h, Hq, Hkv)
            s = (qb[:, h, :] @ kc[:, g, :].T) / np.sqrt(d)
            p = np.where(vis, np.exp(np.where(vis, s, 0.0) - lse[h, b0:b1][:, None]), 0.0)
            D = np.sum(dob[:, h, :] * ob[:, h, :], axis=1)
            dp = dob[:, h, :] @ vc[:, g, :].T
            ds = p * (dp - D[:, None])
            dv[:, g, :] += p.T @ dob[:, h, :]
            dk[:, g, :] += (ds.T @ qb[:, h, :]) / np.sqrt(d)
    return dk, dv
