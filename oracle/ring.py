"""Oracle: one ring step of context-parallel attention, and the merge of
partial results, float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Ring Attention (paper Section 2.2, "Context Parallelism") shards the
sequence across devices and streams key/value blocks past each device's
queries; the hybrid the paper builds on (Section 4, "Implementation": USP,
Ulysses inside a node and a ring across nodes) therefore needs, per device
and per ring step, attention of a query block against one key/value block
that sits elsewhere in the sequence, and a way to combine the partial
results of successive steps (the online-softmax-compatible ring variant of
Section 2.2).

Ring step.  Queries q [Sq, Hq, d] sit at global positions q_offset + i, keys
and values k, v [Skv, Hkv, d] at kv_offset + j.  With ``causal`` true, key j
is visible to query i iff kv_offset + j <= q_offset + i, i.e. j <= i + delta
with delta = q_offset - kv_offset.  Output: the softmax-weighted values over
the visible keys of the block, o [Sq, Hq, d], and the natural-log
log-sum-exp of the visible scaled scores, lse [Hq, Sq].  A row that sees no
key of the block has o = 0 and lse = -inf (the empty sum), which is the
neutral element of the merge below.

Merge.  For two partial results over disjoint key sets A and B of the same
query row, the softmax over A u B is

    lse = log(exp(lse_A) + exp(lse_B))
    o   = exp(lse_A - lse) o_A + exp(lse_B - lse) o_B

because each partial output is its block's weighted mean with weights
exp(s_j - lse_block).  Written here exactly as that definition (with the
larger lse factored out only to avoid overflow).
"""

import numpy as np

from .attention import kv_head_of


def attn_fwd_offset(q, k, v, delta, causal=True):
    """Attention of q [Sq, Hq, d] against one key/value block [Skv, Hkv, d]
    whose key j is visible to query i iff j <= i + delta (all keys when not
    causal).  Returns o [Sq, Hq, d] and lse [Hq, Sq], float64."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    Sq, Hq, d = q.shape
    Skv, Hkv = k.shape[0], k.shape[1]
    if v.shape != k.shape or k.shape[2] != d or Hq % Hkv:
        raise ValueError("shapes: q [Sq,Hq,d], k = v [Skv,Hkv,d], Hkv | Hq")
    o = np.zeros((Sq, Hq, d))
    lse = np.full((Hq, Sq), -np.inf)
    i = np.arange(Sq)[:, None]
    j = np.arange(Skv)[None, :]
    visible = (j <= i + delta) if causal else np.ones((Sq, Skv), bool)
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        s = (q[:, h, :] @ k[:, g, :].T) / np.sqrt(d)
        s = np.where(visible, s, -np.inf)
        any_vis = visible.any(axis=1)
        m = np.where(any_vis, s.max(axis=1, initial=-np.inf), 0.0)
        e = np.exp(s - m[:, None])
        l = e.sum(axis=1)
        rows = np.nonzero(any_vis)[0]
        o[rows, h, :] = (e[rows] / l[rows, None]) @ v[:, g, :]
        lse[h, rows] = m[rows] + np.log(l[rows])
    return o, lse


def lse_merge(o_a, lse_a, o_b, lse_b):
    """Softmax result over the union of two disjoint key sets from the two
    partial results (o [S, H, d], lse [H, S]); -inf rows are empty sets."""
    o_a = np.asarray(o_a, np.float64)
    o_b = np.asarray(o_b, np.float64)
    lse_a = np.asarray(lse_a, np.float64)
    lse_b = np.asarray(lse_b, np.float64)
    m = np.maximum(lse_a, lse_b)                      # [H, S]
    empty = np.isneginf(m)
    ms = np.where(empty, 0.0, m)
    wa = np.where(np.isneginf(lse_a), 0.0, np.exp(lse_a - ms))
    wb = np.where(np.isneginf(lse_b), 0.0, np.exp(lse_b - ms))
    tot = wa + wb
    lse = np.where(empty, -np.inf, ms + np.log(np.where(empty, 1.0, tot)))
    ca = np.where(empty, 0.0, wa / np.where(empty, 1.0, tot)).T[:, :, None]   # [S, H, 1]
    cb = np.where(empty, 0.0, wb / np.where(empty, 1.0, tot)).T[:, :, None]
    return ca * o_a + cb * o_b, lse
