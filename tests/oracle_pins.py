"""Pins for the attention oracle: checks that do not trust the oracle itself.

Each ``pin_*`` takes the oracle attention module ``A`` (the real one, or a
deliberately broken copy in the mutation test) and raises AssertionError when
``A`` disagrees with something the paper or mathematics fixes:

* brute-force scalar loops (pure Python, math.exp) for tiny shapes,
* torch's float64 ``scaled_dot_product_attention`` and autograd,
* central finite differences of <dO, O>,
* closed forms and exact invariants.
"""

import math

import numpy as np
import torch


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# --------------------------------------------------------------- brute force

def brute_attention(q, k, v, causal):
    """Scalar triple loop over (head, query, key) with math.exp."""
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    o = [[[0.0] * d for _ in range(Hq)] for _ in range(S)]
    lse = [[0.0] * S for _ in range(Hq)]
    for h in range(Hq):
        g = h // G
        for i in range(S):
            keys = range(i + 1) if causal else range(S)
            sc = []
            for j in keys:
                acc = 0.0
                for t in range(d):
                    acc += float(q[i, h, t]) * float(k[j, g, t])
                sc.append(acc / math.sqrt(d))
            m = max(sc)
            w = [math.exp(x - m) for x in sc]
            tot = sum(w)
            lse[h][i] = m + math.log(tot)
            for t in range(d):
                o[i][h][t] = sum(w[n] * float(v[j, g, t])
                                 for n, j in enumerate(keys)) / tot
    return np.array(o), np.array(lse)


def pin_brute_force(A):
    for (S, Hq, Hkv, d, causal, seed) in [(1, 1, 1, 4, True, 1),
                                          (7, 2, 1, 8, True, 2),
                                          (9, 4, 2, 4, True, 3),
                                          (6, 3, 3, 5, False, 4),
                                          (11, 4, 1, 3, False, 5)]:
        q = _rand((S, Hq, d), seed)
        k = _rand((S, Hkv, d), seed + 10)
        v = _rand((S, Hkv, d), seed + 20)
        o, lse = A.attn_fwd(q, k, v, causal)
        ob, lb = brute_attention(q, k, v, causal)
        np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


# ------------------------------------------------------ torch library routine

def _torch_ref(q, k, v, do, causal):
    """torch SDPA (float64, CPU) forward and autograd backward."""
    tq = torch.tensor(q).permute(1, 0, 2)[None].requires_grad_(True)
    tk = torch.tensor(k).permute(1, 0, 2)[None].requires_grad_(True)
    tv = torch.tensor(v).permute(1, 0, 2)[None].requires_grad_(True)
    o = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=causal, enable_gqa=True)
    o.backward(torch.tensor(do).permute(1, 0, 2)[None])
    f = lambda t: t[0].permute(1, 0, 2).detach().numpy()  # noqa: E731
    return f(o), f(tq.grad), f(tk.grad), f(tv.grad)


def pin_torch_sdpa(A):
    for (S, Hq, Hkv, d, causal, seed) in [(37, 4, 1, 16, True, 7),
                                          (64, 4, 2, 32, True, 8),
                                          (29, 2, 2, 8, False, 9),
                                          (300, 2, 1, 16, True, 10)]:
        q = _rand((S, Hq, d), seed)
        k = _rand((S, Hkv, d), seed + 1)
        v = _rand((S, Hkv, d), seed + 2)
        do = _rand((S, Hq, d), seed + 3)
        o_t, dq_t, dk_t, dv_t = _torch_ref(q, k, v, do, causal)
        o, _ = A.attn_fwd(q, k, v, causal)
        dq, dk, dv = A.attn_bwd(q, k, v, do, causal)
        for got, ref in ((o, o_t), (dq, dq_t), (dk, dk_t), (dv, dv_t)):
            np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10)


# --------------------------------------------------------- finite differences

def pin_finite_differences(A):
    S, Hq, Hkv, d = 6, 2, 1, 4
    q = _rand((S, Hq, d), 21)
    k = _rand((S, Hkv, d), 22)
    v = _rand((S, Hkv, d), 23)
    do = _rand((S, Hq, d), 24)

    def loss(q_, k_, v_):
        o, _ = A.attn_fwd(q_, k_, v_, True)
        return float(np.sum(o * do))

    dq, dk, dv = A.attn_bwd(q, k, v, do, True)
    eps = 1e-6
    rng = np.random.default_rng(25)
    for which, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(8):
            idx = tuple(int(rng.integers(0, n)) for n in x.shape)
            xp = x.copy(); xp[idx] += eps
            xm = x.copy(); xm[idx] -= eps
            args_p = {"q": q, "k": k, "v": v}; args_p[which] = xp
            args_m = {"q": q, "k": k, "v": v}; args_m[which] = xm
            fd = (loss(**{a + "_": b for a, b in args_p.items()})
                  - loss(**{a + "_": b for a, b in args_m.items()})) / (2 * eps)
            assert abs(fd - g[idx]) < 1e-7, (which, idx, fd, g[idx])


# ------------------------------------------------------ closed forms, special

def pin_closed_forms(A):
    d = 8
    # S = 1: the only key is itself, so O = V and lse = q.k / sqrt(d).
    q = _rand((1, 3, d), 31); k = _rand((1, 1, d), 32); v = _rand((1, 1, d), 33)
    o, lse = A.attn_fwd(q, k, v, True)
    np.testing.assert_allclose(o[0], np.repeat(v[0], 3, axis=0), atol=1e-14)
    np.testing.assert_allclose(lse[:, 0], q[0] @ k[0, 0] / math.sqrt(d),
                               atol=1e-14)
    # Q = 0: uniform weights over the visible prefix.
    S = 13
    q = np.zeros((S, 2, d)); k = _rand((S, 1, d), 34); v = _rand((S, 1, d), 35)
    o, lse = A.attn_fwd(q, k, v, True)
    for i in range(S):
        np.testing.assert_allclose(o[i, 1], v[:i + 1, 0].mean(axis=0),
                                   atol=1e-13)
        assert abs(lse[0, i] - math.log(i + 1)) < 1e-13
    # Non-causal Q = 0: every row is the mean of all of V.
    o, lse = A.attn_fwd(q, k, v, False)
    np.testing.assert_allclose(o[3, 0], v[:, 0].mean(axis=0), atol=1e-13)
    assert abs(lse[1, 0] - math.log(S)) < 1e-13
    # Row 0 of causal attention is V_0; constant V gives constant O.
    q = _rand((S, 2, d), 36, 3.0)
    o, _ = A.attn_fwd(q, k, v, True)
    np.testing.assert_allclose(o[0, 0], v[0, 0], atol=1e-13)
    vc = np.broadcast_to(_rand((1, 1, d), 37), (S, 1, d)).copy()
    o, _ = A.attn_fwd(q, k, vc, True)
    np.testing.assert_allclose(o, np.broadcast_to(vc[:1], (S, 2, d)),
                               atol=1e-13)
    # Shift invariance: K + 1 c^T adds q_i.c/sqrt(d) to every score of row i,
    # which softmax cancels; lse moves by exactly that amount.
    c = _rand((d,), 38)
    o1, l1 = A.attn_fwd(q, k, v, True)
    o2, l2 = A.attn_fwd(q, k + c[None, None, :], v, True)
    np.testing.assert_allclose(o2, o1, atol=1e-12)
    np.testing.assert_allclose(l2 - l1, (q @ c).T / math.sqrt(d), atol=1e-12)
    # Softmax rows sum to one: with V = identity-like one-hot columns the
    # output of row i is its probability row, which must sum to 1.
    S2 = 8
    q = _rand((S2, 1, S2), 39); k = _rand((S2, 1, S2), 40)
    v = np.eye(S2)[:, None, :]
    o, _ = A.attn_fwd(q, k, v, True)
    np.testing.assert_allclose(o[:, 0].sum(axis=1), np.ones(S2), atol=1e-13)
    assert np.all(np.triu(o[:, 0], 1) == 0.0)


def pin_gradient_invariants(A):
    S, Hq, Hkv, d = 40, 4, 2, 8
    q = _rand((S, Hq, d), 41); k = _rand((S, Hkv, d), 42)
    v = _rand((S, Hkv, d), 43); do = _rand((S, Hq, d), 44)
    dq, dk, dv = A.attn_bwd(q, k, v, do, True)
    G = Hq // Hkv
    # sum_j dS_ij = sum_j P_ij dP_ij - D_i = 0, hence sum_j dK_j = 0.
    np.testing.assert_allclose(dk.sum(axis=0), 0.0, atol=1e-11)
    # sum_j P_ij = 1, hence sum_j dV_j = sum over the group's rows of dO.
    for g in range(Hkv):
        np.testing.assert_allclose(dv[:, g].sum(axis=0),
                                   do[:, g * G:(g + 1) * G].sum(axis=(0, 1)),
                                   atol=1e-11)
    # Row 0 sees only key 0 (P = 1), so dS = dP - D = 0 and dQ_0 = 0.
    np.testing.assert_allclose(dq[0], 0.0, atol=1e-13)


def pin_gqa_equals_repeated_mha(A):
    S, Hq, Hkv, d = 33, 6, 2, 8
    G = Hq // Hkv
    q = _rand((S, Hq, d), 51); k = _rand((S, Hkv, d), 52)
    v = _rand((S, Hkv, d), 53); do = _rand((S, Hq, d), 54)
    kr = np.repeat(k, G, axis=1); vr = np.repeat(v, G, axis=1)
    o1, l1 = A.attn_fwd(q, k, v, True)
    o2, l2 = A.attn_fwd(q, kr, vr, True)
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    np.testing.assert_allclose(l1, l2, atol=1e-14)
    dq1, dk1, dv1 = A.attn_bwd(q, k, v, do, True)
    dq2, dk2, dv2 = A.attn_bwd(q, kr, vr, do, True)
    np.testing.assert_allclose(dq1, dq2, atol=1e-13)
    np.testing.assert_allclose(dk1, dk2.reshape(S, Hkv, G, d).sum(2),
                               atol=1e-12)
    np.testing.assert_allclose(dv1, dv2.reshape(S, Hkv, G, d).sum(2),
                               atol=1e-12)


def pin_key_cols_given_statistics(A):
    """The conditioned key-column gradient, given the module's own row
    statistics, against torch float64 autograd (GQA, causal, with key 0 and
    the diagonal key of the last row among the columns)."""
    S, Hq, Hkv, d = 40, 4, 2, 8
    q = _rand((S, Hq, d), 61); k = _rand((S, Hkv, d), 62)
    v = _rand((S, Hkv, d), 63); do = _rand((S, Hq, d), 64)
    o, lse = A.attn_fwd(q, k, v, True)
    _, _, dk_t, dv_t = _torch_ref(q, k, v, do, True)
    cols = np.array([0, 1, 17, S - 1])
    dk, dv = A.attn_key_cols_given(q, do, k, v, o, lse, cols, True, row_block=16)
    np.testing.assert_allclose(dk, dk_t[cols], rtol=0, atol=1e-10)
    np.testing.assert_allclose(dv, dv_t[cols], rtol=0, atol=1e-10)


ALL_PINS = [pin_brute_force, pin_torch_sdpa, pin_finite_differences,
            pin_closed_forms, pin_gradient_invariants,
            pin_gqa_equals_repeated_mha, pin_key_cols_given_statistics]
