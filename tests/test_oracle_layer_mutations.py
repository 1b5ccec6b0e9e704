"""Plant plausible mistakes in a copy of the layer oracle; its checks against
torch float64 autograd must reject every one (see test_oracle_mutations for
the attention oracle).  Each mutant is the module's source with one textual
change, executed on the CPU as a throw-away module of the oracle package."""

import os
import types

import numpy as np
import pytest
import torch

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "layer.py")

MUTANTS = {
    "tail_dk_unrotated": ("        dk = rope(dk, pos0 + tail, rope_base, inverse=True)\n",
                          ""),
    "tail_wrong_weight": ("    return dqkv @ wqkv.T\n", "    return dqkv @ wqkv[:, ::-1].T\n"),
    "dwo_uses_dy_rows": ("    return o.reshape(S, -1).T @ dyc", "    return o.reshape(S, -1).T @ dyc[::-1]"),
    "grads_dq_unrotated": (
        "    dq = _rotate(np.asarray(dq, np.float64), S, rope_base, pos0, inverse=True)",
        "    dq = np.asarray(dq, np.float64)"),
    "grads_k_v_swapped": (
        "                           np.asarray(dv, np.float64).reshape(S, -1)], axis=1)\n    return x.T @ dqkv[:, cols]",
        "                           np.asarray(dk, np.float64).reshape(S, -1)], axis=1)\n    return x.T @ dqkv[:, cols]"),
    "inputs_do_not_transposed": (
        "    do = (np.asarray(dy, np.float64) @ np.asarray(wo, np.float64).T).reshape(S, Hq, d)",
        "    do = (np.asarray(dy, np.float64) @ np.asarray(wo, np.float64)[:, ::-1].T).reshape(S, Hq, d)"),
    "inputs_v_rotated": (
        "    q = _rotate(q, S, rope_base, pos0)\n    k = _rotate(k, S, rope_base, pos0)\n    do = (np.asarray(dy",
        "    q = _rotate(q, S, rope_base, pos0)\n    k = _rotate(k, S, rope_base, pos0)\n"
        "    v = _rotate(v, S, rope_base, pos0)\n    do = (np.asarray(dy"),
}


def _mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mod = types.ModuleType(f"oracle.layer_mutant_{name}")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def _inputs(seed, S, dm, Hq, Hkv, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((S, dm)), rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.3,
            rng.standard_normal((Hq * d, dm)) * 0.3, rng.standard_normal((S, dm)))


def _torch_grads(x, wqkv, wo, dy, Hq, Hkv, d, base):
    """torch float64 autograd of the block with rotate-half RoPE at position s
    (angle s * base^(-e/(d/2)) on the pairs (e, e + d/2))."""
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(wqkv, requires_grad=True)
    to = torch.tensor(wo, requires_grad=True)
    S = x.shape[0]
    qkv = tx @ tw
    h = d // 2
    ang = torch.arange(S, dtype=torch.float64)[:, None, None] * \
        base ** (-torch.arange(h, dtype=torch.float64) / h)[None, None, :]
    c, s = torch.cos(ang), torch.sin(ang)

    def rot(t):
        a, b = t[..., :h], t[..., h:]
        return torch.cat([a * c - b * s, b * c + a * s], dim=-1)

    q = rot(qkv[:, :Hq * d].reshape(S, Hq, d)).permute(1, 0, 2)[None]
    k = rot(qkv[:, Hq * d:(Hq + Hkv) * d].reshape(S, Hkv, d)).permute(1, 0, 2)[None]
    v = qkv[:, (Hq + Hkv) * d:].reshape(S, Hkv, d).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True, enable_gqa=True)
    y = o[0].permute(1, 0, 2).reshape(S, Hq * d) @ to
    y.backward(torch.tensor(dy))
    return tx.grad.numpy(), tw.grad.numpy(), to.grad.numpy()


def _checks(L):
    """Raises AssertionError if any of the new layer helpers disagrees with
    torch autograd."""
    from oracle import attention as A
    S, dm, Hq, Hkv, d, base = 36, 16, 4, 2, 8, 50.0
    x, wqkv, wo, dy = _inputs(21, S, dm, Hq, Hkv, d)
    dx_t, dw_t, dwo_t = _torch_grads(x, wqkv, wo, dy, Hq, Hkv, d, base)
    np.testing.assert_allclose(L.layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, 20, rope_base=base),
                               dx_t[20:], rtol=0, atol=1e-9)
    _, o, _ = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d, rope_base=base)
    cols = np.array([0, 7, dm - 1])
    np.testing.assert_allclose(L.dwo_given_output(o, dy, cols), dwo_t[:, cols], rtol=0, atol=1e-9)
    q, k, v, do = L.attention_inputs(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=base)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    wc = np.arange(dw_t.shape[1])
    np.testing.assert_allclose(L.dwqkv_given_grads(x, dq, dk, dv, wc, rope_base=base),
                               dw_t, rtol=0, atol=1e-9)


def test_checks_pass_on_the_oracle():
    from oracle import layer as L
    _checks(L)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_checks_reject_mutant(name):
    with pytest.raises(AssertionError):
        _checks(_mutant(name))
