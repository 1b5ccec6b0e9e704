"""Oracle: the attention block around the kernel -- projections in, out.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The block follows the paper's description of one device's attention stage
(Section 3.2 walk-through of DS-Ulysses, Section 3.3 and the Appendix A
paragraphs "Untied Ulysses (forward)" / "(backward)"): the hidden states X
are projected to Q, K, V, attention runs per head, the per-head outputs fill
``final_out`` and the output projection proj_o maps it back to d_model.

Weight layout used here (no bias, no normalisation):
    x    [S, dm]
    wqkv [dm, (Hq + 2 Hkv) d]  columns = [Q heads | K heads | V heads],
                               each head a block of d consecutive columns
    wo   [Hq d, dm]            rows = the heads of final_out, in order
    y    [S, dm] = final_out.reshape(S, Hq d) @ wo

Rotary embedding (optional, ``rope_base``): the projected Q and K heads are
rotated at positions pos0 + s before attention (``oracle.rope``; the paper's
Section 4 "Implementation" runs it fused and in place).  V is not rotated.

Backward (chain rule on the same definition):
    dO    = dY wo^T              dWo   = final_out^T dY
    dQ, dK, dV from the attention gradient (with RoPE: with respect to the
                  rotated Q, K, then turned back by the inverse rotation)
    dX    = [dQ|dK|dV] wqkv^T    dWqkv = X^T [dQ|dK|dV]
"""

import numpy as np

from . import attention
from .rope import rope


def split_qkv(qkv, Hq, Hkv, d):
    S = qkv.shape[0]
    q = qkv[:, :Hq * d].reshape(S, Hq, d)
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(S, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(S, Hkv, d)
    return q, k, v


def _rotate(t, S, rope_base, pos0, inverse=False):
    if rope_base is None:
        return t
    return rope(t, pos0 + np.arange(S), rope_base, inverse)


def layer_fwd(x, wqkv, wo, Hq, Hkv, d, causal=True, rope_base=None, pos0=0):
    """Returns (y [S, dm], final_out [S, Hq, d], lse [Hq, S])."""
    x = np.asarray(x, np.float64)
    wqkv = np.asarray(wqkv, np.float64)
    wo = np.asarray(wo, np.float64)
    S = x.shape[0]
    q, k, v = split_qkv(x @ wqkv, Hq, Hkv, d)
    q = _rotate(q, S, rope_base, pos0)
    k = _rotate(k, S, rope_base, pos0)
    o, lse = attention.attn_fwd(q, k, v, causal)
    y = o.reshape(S, Hq * d) @ wo
    return y, o, lse


def layer_bwd(x, wqkv, wo, dy, Hq, Hkv, d, causal=True, rope_base=None, pos0=0):
    """Returns (dx [S, dm], dwqkv [dm, (Hq+2Hkv)d], dwo [Hq d, dm])."""
    x = np.asarray(x, np.float64)
    wqkv = np.asarray(wqkv, np.float64)
    wo = np.asarray(wo, np.float64)
    dy = np.asarray(dy, np.float64)
    S = x.shape[0]
    q, k, v = split_qkv(x @ wqkv, Hq, Hkv, d)
    q = _rotate(q, S, rope_base, pos0)
    k = _rotate(k, S, rope_base, pos0)
    o, _ = attention.attn_fwd(q, k, v, causal)
    do = (dy @ wo.T).reshape(S, Hq, d)
    dwo = o.reshape(S, Hq * d).T @ dy
    dq, dk, dv = attention.attn_bwd(q, k, v, do, causal)
    dq = _rotate(dq, S, rope_base, pos0, inverse=True)
    dk = _rotate(dk, S, rope_base, pos0, inverse=True)
    dqkv = np.concatenate([dq.reshape(S, -1), dk.reshape(S, -1),
                           dv.reshape(S, -1)], axis=1)
    dx = dqkv @ wqkv.T
    dwqkv = x.T @ dqkv
    return dx, dwqkv, dwo


def layer_fwd_rows(x, wqkv, wo, Hq, Hkv, d, rows, rope_base=None, pos0=0):
    """y, final_out and lse at the listed rows only (causal).

    K and V are needed for every position (each row sees all earlier keys),
    Q and the output only at the listed rows.
    """
    x = np.asarray(x, np.float64)
    wqkv = np.asarray(wqkv, np.float64)
    wo = np.asarray(wo, np.float64)
    rows = np.asarray(rows, np.int64)
    S = x.shape[0]
    kv = x @ wqkv[:, Hq * d:]
    k = _rotate(kv[:, :Hkv * d].reshape(S, Hkv, d), S, rope_base, pos0)
    v = kv[:, Hkv * d:].reshape(S, Hkv, d)
    qr = (x[rows] @ wqkv[:, :Hq * d]).reshape(len(rows), Hq, d)
    if rope_base is not None:
        qr = rope(qr, pos0 + rows, rope_base)
    # Place the sampled query rows at their own positions; other rows are
    # never read because each listed row only sees keys <= itself.
    q = np.zeros((S, Hq, d))
    q[rows] = qr
    o, lse = attention.attn_fwd(q, k, v, True, rows=rows)
    y = o.reshape(len(rows), Hq * d) @ wo
    return y, o, lse


def layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, j0, rope_base=None, pos0=0):
    """dX at the rows [j0, S) of the causal block (same chain rule as
    ``layer_bwd``).

    Row s of dX = [dQ_s | dK_s | dV_s] wqkv^T.  dQ_s is row-local; under the
    causal mask dK_s and dV_s receive only from query rows >= s, so the rows
    [j0, S) need the attention gradient of those query rows alone (each with
    its full row softmax).  K and V are needed at every position.
    """
    x = np.asarray(x, np.float64)
    wqkv = np.asarray(wqkv, np.float64)
    wo = np.asarray(wo, np.float64)
    dy = np.asarray(dy, np.float64)
    S = x.shape[0]
    q, k, v = split_qkv(x @ wqkv, Hq, Hkv, d)
    q = _rotate(q, S, rope_base, pos0)
    k = _rotate(k, S, rope_base, pos0)
    do = (dy @ wo.T).reshape(S, Hq, d)
    tail = np.arange(j0, S)
    dq, _ = attention.attn_bwd_rows(q, k, v, do, tail)
    dk, dv = attention.attn_bwd_key_tail(q, k, v, do, j0)
    if rope_base is not None:
        dq = rope(dq, pos0 + tail, rope_base, inverse=True)
        dk = rope(dk, pos0 + tail, rope_base, inverse=True)
    n = len(tail)
    dqkv = np.concatenate([dq.reshape(n, -1), dk.reshape(n, -1), dv.reshape(n, -1)], axis=1)
    return dqkv @ wqkv.T


def dwo_given_output(o, dy, cols):
    """Columns ``cols`` of dWo = final_out^T dY for a given final_out o
    [S, Hq, d] (the chain rule of y = final_out wo): [Hq d, len(cols)].

    With the oracle's own final_out this is the oracle's dWo; with another
    implementation's saved output it is the weight gradient that output
    implies ("conditioned" on it), which checks the reduction over the whole
    sequence without re-running attention.
    """
    o = np.asarray(o, np.float64)
    S = o.shape[0]
    dyc = np.asarray(dy[:, cols], np.float64)
    return o.reshape(S, -1).T @ dyc


def attention_inputs(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=None, pos0=0):
    """The attention operands of the block's backward (the first steps of
    ``layer_bwd``): q, k (rotated when ``rope_base`` is given), v and the
    gradient of final_out dO = dY wo^T, each [S, H, d] in float64."""
    x = np.asarray(x, np.float64)
    S = x.shape[0]
    q, k, v = split_qkv(x @ np.asarray(wqkv, np.float64), Hq, Hkv, d)
    q = _rotate(q, S, rope_base, pos0)
    k = _rotate(k, S, rope_base, pos0)
    do = (np.asarray(dy, np.float64) @ np.asarray(wo, np.float64).T).reshape(S, Hq, d)
    return q, k, v, do


def dwqkv_given_grads(x, dq, dk, dv, cols, rope_base=None, pos0=0):
    """Columns ``cols`` of dWqkv = x^T [dQ | dK | dV] for given attention
    gradients with respect to the (rotated) q, k and to v, each [S, H, d]:
    the gradients of the rotated q, k are turned back first (the chain rule
    of the rotation).  With the oracle's own gradients this is the oracle's
    dWqkv; with another implementation's it is the weight gradient those
    imply ("conditioned" on them).  Returns [d_model, len(cols)]."""
    x = np.asarray(x, np.float64)
    S = x.shape[0]
    dq = _rotate(np.asarray(dq, np.float64), S, rope_base, pos0, inverse=True)
    dk = _rotate(np.asarray(dk, np.float64), S, rope_base, pos0, inverse=True)
    dqkv = np.concatenate([dq.reshape(S, -1), dk.reshape(S, -1),
                           np.asarray(dv, np.float64).reshape(S, -1)], axis=1)
    return x.T @ dqkv[:, cols]
