"""Pins of the rotary-embedding oracle (oracle/rope.py) and of the layer
oracle with RoPE (oracle/layer.py), none of which trusts the oracle itself:

* RoFormer's block-diagonal rotation matrix, built entry by entry with
  math.cos / math.sin for its own (2i, 2i+1) pairing and conjugated by the
  permutation that maps that pairing onto pairs (e, e + d/2);
* the complex form (x_a + i x_b) exp(i p theta_e) with numpy complex numbers;
* hand-computed closed values (theta_0 = 1; base 10^4, d = 4 gives
  theta_1 = 1/100);
* exact properties: position 0 is the identity, norms are kept, scores depend
  on positions only through their difference, the inverse is the transpose;
* the layer with RoPE against torch float64 autograd through torch's own
  complex multiplication (view_as_complex / polar).

Planted mistakes in copies of both files must each be rejected by a pin."""

import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import layer as L
from oracle import rope as R


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def roformer_matrix(p, d, base):
    """RoFormer's R_{Theta,p}: 2x2 rotations on coordinate pairs (2i, 2i+1)
    with theta_i = base^(-2i/d), as nested Python lists."""
    m = [[0.0] * d for _ in range(d)]
    for i in range(d // 2):
        t = p * base ** (-2.0 * i / d)
        c, s = math.cos(t), math.sin(t)
        m[2 * i][2 * i], m[2 * i][2 * i + 1] = c, -s
        m[2 * i + 1][2 * i], m[2 * i + 1][2 * i + 1] = s, c
    return m


def pin_roformer_matrix(mod):
    """y = P R P^T x, P sending coordinate 2i -> i and 2i+1 -> i + d/2."""
    for d, base, seed in ((4, 10000.0, 1), (8, 500000.0, 2), (6, 10.0, 3)):
        S, H = 7, 2
        x = _rand((S, H, d), seed)
        pos = np.array([0, 1, 2, 5, 17, 1000, 123457])
        y = mod.rope(x, pos, base)
        src = [c for i in range(d // 2) for c in (i, i + d // 2)]   # RoFormer index -> ours
        for s in range(S):
            m = roformer_matrix(int(pos[s]), d, base)
            for h in range(H):
                xr = [x[s, h, src[j]] for j in range(d)]
                yr = [sum(m[r][j] * xr[j] for j in range(d)) for r in range(d)]
                for r in range(d):
                    assert abs(y[s, h, src[r]] - yr[r]) < 1e-12, (d, s, h, r)


def pin_complex_form(mod):
    d, base = 16, 1e6
    x = _rand((9, 3, d), 4)
    pos = np.arange(9) * 4099 + 11
    z = x[..., :d // 2] + 1j * x[..., d // 2:]
    th = base ** (-np.arange(d // 2) * 2.0 / d)
    w = z * np.exp(1j * pos[:, None, None] * th[None, None, :])
    y = mod.rope(x, pos, base)
    np.testing.assert_allclose(y[..., :d // 2], w.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(y[..., d // 2:], w.imag, rtol=0, atol=1e-12)
    wi = z * np.exp(-1j * pos[:, None, None] * th[None, None, :])
    yi = mod.rope(x, pos, base, inverse=True)
    np.testing.assert_allclose(yi[..., :d // 2], wi.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(yi[..., d // 2:], wi.imag, rtol=0, atol=1e-12)


def pin_closed_values(mod):
    e = np.eye(4)[:, None, :]                     # four unit vectors, d = 4
    y = mod.rope(e, np.array([3, 100, 2, 100]), 10000.0)
    # pair 0 (coordinates 0, 2) turns by p radians; pair 1 (1, 3) by p/100.
    np.testing.assert_allclose(y[0, 0], [math.cos(3), 0, math.sin(3), 0], atol=1e-15)
    np.testing.assert_allclose(y[1, 0], [0, math.cos(1), 0, math.sin(1)], atol=1e-15)
    np.testing.assert_allclose(y[2, 0], [-math.sin(2), 0, math.cos(2), 0], atol=1e-15)
    np.testing.assert_allclose(y[3, 0], [0, -math.sin(1), 0, math.cos(1)], atol=1e-15)
    np.testing.assert_allclose(mod.rope_theta(4, 10000.0), [1.0, 0.01], rtol=1e-15)


def pin_invariants(mod):
    d, base = 12, 5e5
    x = _rand((6, 2, d), 5)
    y0 = mod.rope(x, np.zeros(6, int), base)
    np.testing.assert_array_equal(y0, x)
    pos = np.array([1, 7, 4096, 65537, 1 << 20, (1 << 24) - 1])
    y = mod.rope(x, pos, base)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-14)
    half = d // 2
    np.testing.assert_allclose(y[..., :half] ** 2 + y[..., half:] ** 2,
                               x[..., :half] ** 2 + x[..., half:] ** 2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(mod.rope(y, pos, base, inverse=True), x, rtol=0, atol=1e-12)
    # The inverse is the transpose: <R x, g> = <x, R^-1 g>.
    g = _rand((6, 2, d), 6)
    lhs = np.sum(y * g, axis=-1)
    rhs = np.sum(x * mod.rope(g, pos, base, inverse=True), axis=-1)
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


def pin_relative_positions(mod):
    """<R_p q, R_p' k> depends only on p - p'."""
    d, base = 8, 10000.0
    q, k = _rand((1, 1, d), 7), _rand((1, 1, d), 8)

    def score(p, pk):
        return float(np.sum(mod.rope(q, [p], base) * mod.rope(k, [pk], base)))

    for delta in (0, 1, 5, 300):
        ref = score(delta, 0)
        for shift in (1, 17, 99991):
            assert abs(score(delta + shift, shift) - ref) < 1e-10, (delta, shift)
    assert abs(score(5, 0) - score(0, 5)) > 1e-3      # not symmetric in p - p'


PINS = [pin_roformer_matrix, pin_complex_form, pin_closed_values, pin_invariants,
        pin_relative_positions]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_rope_oracle_pins(pin):
    pin(R)


# ----------------------------------------------------------- layer with RoPE

def _torch_rope(t, pos, base):
    """t [S, H, d] rotated through torch complex multiplication."""
    S, H, d = t.shape
    th = base ** (-torch.arange(d // 2, dtype=torch.float64) * 2.0 / d)
    ang = torch.tensor(pos, dtype=torch.float64)[:, None] * th[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    z = torch.view_as_complex(torch.stack([t[..., :d // 2], t[..., d // 2:]], dim=-1).contiguous())
    w = torch.view_as_real(z * rot)
    return torch.cat([w[..., 0], w[..., 1]], dim=-1)


def _torch_layer_rope(x, wqkv, wo, dy, Hq, Hkv, d, base, pos0):
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(wqkv, requires_grad=True)
    to = torch.tensor(wo, requires_grad=True)
    S = x.shape[0]
    pos = pos0 + np.arange(S)
    qkv = tx @ tw
    q = _torch_rope(qkv[:, :Hq * d].reshape(S, Hq, d), pos, base)
    k = _torch_rope(qkv[:, Hq * d:(Hq + Hkv) * d].reshape(S, Hkv, d), pos, base)
    v = qkv[:, (Hq + Hkv) * d:].reshape(S, Hkv, d)
    o = torch.nn.functional.scaled_dot_product_attention(
        q.permute(1, 0, 2)[None], k.permute(1, 0, 2)[None], v.permute(1, 0, 2)[None],
        is_causal=True, enable_gqa=True)
    y = o[0].permute(1, 0, 2).reshape(S, Hq * d) @ to
    y.backward(torch.tensor(dy))
    return y.detach().numpy(), tx.grad.numpy(), tw.grad.numpy(), to.grad.numpy()


def pin_layer_rope_autograd(Lmod):
    rng = np.random.default_rng(9)
    S, dm, Hq, Hkv, d = 33, 16, 4, 2, 8
    x = rng.standard_normal((S, dm))
    wqkv = rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.4
    wo = rng.standard_normal((Hq * d, dm)) * 0.4
    dy = rng.standard_normal((S, dm))
    for base, pos0 in ((10000.0, 0), (500000.0, 1 << 20)):
        y_t, dx_t, dw_t, dwo_t = _torch_layer_rope(x, wqkv, wo, dy, Hq, Hkv, d, base, pos0)
        y, _, _ = Lmod.layer_fwd(x, wqkv, wo, Hq, Hkv, d, rope_base=base, pos0=pos0)
        dx, dw, dwo = Lmod.layer_bwd(x, wqkv, wo, dy, Hq, Hkv, d, rope_base=base, pos0=pos0)
        np.testing.assert_allclose(y, y_t, atol=1e-11)
        np.testing.assert_allclose(dx, dx_t, atol=1e-10)
        np.testing.assert_allclose(dw, dw_t, atol=1e-10)
        np.testing.assert_allclose(dwo, dwo_t, atol=1e-10)


def pin_layer_rope_rows(Lmod):
    rng = np.random.default_rng(10)
    S, dm, Hq, Hkv, d = 50, 16, 2, 1, 8
    x = rng.standard_normal((S, dm))
    wqkv = rng.standard_normal((dm, (Hq + 2 * Hkv) * d)) * 0.4
    wo = rng.standard_normal((Hq * d, dm)) * 0.4
    y, o, lse = Lmod.layer_fwd(x, wqkv, wo, Hq, Hkv, d, rope_base=1e4, pos0=77)
    rows = np.array([0, 9, 31, 49])
    yr, orow, lr = Lmod.layer_fwd_rows(x, wqkv, wo, Hq, Hkv, d, rows, rope_base=1e4, pos0=77)
    np.testing.assert_allclose(yr, y[rows], atol=1e-12)
    np.testing.assert_allclose(orow, o[rows], atol=1e-12)
    np.testing.assert_allclose(lr, lse[:, rows], atol=1e-12)


LAYER_PINS = [pin_layer_rope_autograd, pin_layer_rope_rows]


@pytest.mark.parametrize("pin", LAYER_PINS, ids=lambda p: p.__name__)
def test_layer_rope_pins(pin):
    pin(L)


def test_layer_without_rope_unchanged():
    rng = np.random.default_rng(11)
    S, dm, Hq, Hkv, d = 20, 8, 2, 1, 4
    x = rng.standard_normal((S, dm))
    wqkv = rng.standard_normal((dm, (Hq + 2 * Hkv) * d))
    wo = rng.standard_normal((Hq * d, dm))
    y0, _, _ = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d)
    y1, _, _ = L.layer_fwd(x, wqkv, wo, Hq, Hkv, d, rope_base=1e4)
    assert np.abs(y0 - y1).max() > 1e-3      # the rotation does change the result


# ------------------------------------------------------------------ mutants

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROPE_MUTANTS = {
    "sin_sign": ("xa * c - xb * s", "xa * c + xb * s"),
    "theta_exponent": ("(-2.0 * e / d)", "(-1.0 * e / d)"),
    "inverse_ignored": ("ang = -ang", "ang = ang"),
    "interleaved_pairs": ("xa, xb = x[..., :half], x[..., half:]",
                          "xa, xb = x[..., 0::2], x[..., 1::2]"),
    "position_plus_one": ("pos[:, None] * rope_theta", "(pos[:, None] + 1) * rope_theta"),
    "b_uses_sin_of_b": ("xb * c + xa * s", "xb * c + xb * s"),
}
LAYER_MUTANTS = {
    "dq_not_turned_back": ("dq = _rotate(dq, S, rope_base, pos0, inverse=True)",
                           "dq = _rotate(dq, S, rope_base, pos0, inverse=False)"),
    "dk_not_turned_back": ("dk = _rotate(dk, S, rope_base, pos0, inverse=True)", "pass"),
    "v_rotated": ("v = kv[:, Hkv * d:].reshape(S, Hkv, d)",
                  "v = _rotate(kv[:, Hkv * d:].reshape(S, Hkv, d), S, rope_base, pos0)"),
    "rows_ignore_pos0": ("qr = rope(qr, pos0 + rows, rope_base)", "qr = rope(qr, rows, rope_base)"),
}


def _load_mutant(relpath, old, new, name):
    src = open(os.path.join(ROOT, relpath)).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mod = types.ModuleType(f"mutant_{name}")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def _caught(mod, pins):
    caught = []
    for pin in pins:
        try:
            with np.errstate(all="ignore"):
                pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    return caught


@pytest.mark.parametrize("name", sorted(ROPE_MUTANTS))
def test_rope_pins_reject_mutant(name):
    mod = _load_mutant("oracle/rope.py", *ROPE_MUTANTS[name], name)
    assert _caught(mod, PINS), f"no pin rejects mutant {name}"


@pytest.mark.parametrize("name", sorted(LAYER_MUTANTS))
def test_layer_rope_pins_reject_mutant(name):
    mod = _load_mutant("oracle/layer.py", *LAYER_MUTANTS[name], name)
    assert _caught(mod, LAYER_PINS), f"no pin rejects mutant {name}"
