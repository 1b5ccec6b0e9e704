"""The layer oracle against torch float64 autograd (a library routine)."""

import numpy as np
import torch

from oracle import layer as L


def _torch_layer(x, wqkv, wo, dy, Hq, Hkv, d):
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(wqkv, requires_grad=True)
    to = torch.tensor(wo, requires_grad=True)
    S = x.shape[0]
    qkv = tx @ tw
    q = qkv[:, :Hq * d].reshape(S, Hq, d).permute(1, 0, 2)[None]
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(S, Hkv, d).permute(1, 0, 2)[None]
    v = qkv[:, (Hq + Hkv) * d:].reshape(S, Hkv, d).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(
        q, k, v, is_causal=True, enable_gqa=True)
    y = o[0].permute(1, 0, 2).reshape(S, Hq * d) @ to
    y.backward(torch.tensor(dy))
    return (y.detach().numpy(), tx.grad.numpy(), tw.grad.numpy(),
            to.grad.numpy())


def test_layer_against_torch_autograd():
    rng = np.random.default_rng(5)
    S, dm, Hq, Hkv, d = 45, 24, 4, 2, 6
    x = rng.standard_normal((S, dm))
    wqkv = rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.3
    wo = rng.standard_normal((Hq * d, dm)) * 0.3
    dy = rng.standard_normal((S, dm))
    y_t, dx_t, dw_t, dwo_t = _torch_layer(x, wqkv, wo, dy, Hq, Hkv, d)
    y, o, lse = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d)
    dx, dw, dwo = L.layer_bwd(x, wqkv, wo, dy, Hq, Hkv, d)
    np.testing.assert_allclose(y, y_t, atol=1e-11)
    np.testing.assert_allclose(dx, dx_t, atol=1e-10)
    np.testing.assert_allclose(dw, dw_t, atol=1e-10)
    np.testing.assert_allclose(dwo, dwo_t, atol=1e-10)


def test_layer_rows_match_full():
    rng = np.random.default_rng(6)
    S, dm, Hq, Hkv, d = 70, 16, 2, 1, 8
    x = rng.standard_normal((S, dm))
    wqkv = rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.3
    wo = rng.standard_normal((Hq * d, dm)) * 0.3
    y, o, lse = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d)
    rows = np.array([0, 3, 31, 69])
    yr, orow, lr = L.layer_fwd_rows(x, wqkv, wo, Hq, Hkv, d, rows)
    np.testing.assert_allclose(yr, y[rows], atol=1e-12)
    np.testing.assert_allclose(orow, o[rows], atol=1e-12)
    np.testing.assert_allclose(lr, lse[:, rows], atol=1e-12)


def _layer_inputs(seed, S, dm, Hq, Hkv, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((S, dm)), rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.3,
            rng.standard_normal((Hq * d, dm)) * 0.3, rng.standard_normal((S, dm)))


def test_layer_bwd_tail_matches_torch_autograd():
    """dX on the last rows from the tail chain rule equals torch float64
    autograd's dX there (no rotary embedding)."""
    S, dm, Hq, Hkv, d = 60, 20, 4, 2, 6
    x, wqkv, wo, dy = _layer_inputs(11, S, dm, Hq, Hkv, d)
    _, dx_t, _, _ = _torch_layer(x, wqkv, wo, dy, Hq, Hkv, d)
    for j0 in (0, 1, 37, 59):
        got = L.layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, j0)
        np.testing.assert_allclose(got, dx_t[j0:], rtol=0, atol=1e-10)


def test_layer_bwd_tail_with_rope_matches_full_backward():
    S, dm, Hq, Hkv, d = 50, 16, 2, 1, 8
    x, wqkv, wo, dy = _layer_inputs(12, S, dm, Hq, Hkv, d)
    dx, _, _ = L.layer_bwd(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=100.0, pos0=7)
    got = L.layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, 30, rope_base=100.0, pos0=7)
    np.testing.assert_allclose(got, dx[30:], rtol=0, atol=1e-11)
    # a global position shift changes nothing (scores depend on i - j only),
    # a different base does
    same = L.layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, 30, rope_base=100.0, pos0=8)
    np.testing.assert_allclose(same, dx[30:], rtol=0, atol=1e-11)
    bad = L.layer_bwd_tail(x, wqkv, wo, dy, Hq, Hkv, d, 30, rope_base=50.0, pos0=7)
    assert np.abs(bad - dx[30:]).max() > 1e-3


def test_dwo_given_output_matches_torch_autograd():
    S, dm, Hq, Hkv, d = 45, 24, 4, 2, 6
    x, wqkv, wo, dy = _layer_inputs(13, S, dm, Hq, Hkv, d)
    _, _, _, dwo_t = _torch_layer(x, wqkv, wo, dy, Hq, Hkv, d)
    _, o, _ = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d)
    cols = np.array([0, 5, 23])
    np.testing.assert_allclose(L.dwo_given_output(o, dy, cols), dwo_t[:, cols], rtol=0,
                               atol=1e-10)


def test_dwqkv_given_grads_matches_torch_autograd():
    """The weight gradient of Wqkv from the attention gradients (the chain
    rule through the projection) equals torch float64 autograd's dWqkv."""
    S, dm, Hq, Hkv, d = 45, 24, 4, 2, 6
    x, wqkv, wo, dy = _layer_inputs(14, S, dm, Hq, Hkv, d)
    _, _, dw_t, _ = _torch_layer(x, wqkv, wo, dy, Hq, Hkv, d)
    from oracle import attention as A
    q, k, v, do = L.attention_inputs(x, wqkv, wo, dy, Hq, Hkv, d)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    cols = np.array([0, 3, Hq * d, (Hq + Hkv) * d + 1, (Hq + 2 * Hkv) * d - 1])
    np.testing.assert_allclose(L.dwqkv_given_grads(x, dq, dk, dv, cols), dw_t[:, cols],
                               rtol=0, atol=1e-10)


def test_dwqkv_given_grads_with_rope_matches_full_backward():
    S, dm, Hq, Hkv, d = 50, 16, 2, 1, 8
    x, wqkv, wo, dy = _layer_inputs(15, S, dm, Hq, Hkv, d)
    _, dw, _ = L.layer_bwd(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=100.0, pos0=3)
    from oracle import attention as A
    q, k, v, do = L.attention_inputs(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=100.0, pos0=3)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    cols = np.arange(dw.shape[1])
    got = L.dwqkv_given_grads(x, dq, dk, dv, cols, rope_base=100.0, pos0=3)
    np.testing.assert_allclose(got, dw, rtol=0, atol=1e-10)
    # the gradients of the rotated q, k must be turned back: without the
    # inverse rotation the Q and K columns are wrong
    bad = L.dwqkv_given_grads(x, dq, dk, dv, cols)
    assert np.abs(bad[:, :(Hq + Hkv) * d] - dw[:, :(Hq + Hkv) * d]).max() > 1e-3
