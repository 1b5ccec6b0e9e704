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
