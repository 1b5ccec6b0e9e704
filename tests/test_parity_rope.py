"""GPU parity of the rotary embedding against the oracle (oracle/rope.py,
oracle/layer.py), through the C ABI:

* upipe_rope (in place, standalone) at small and very large positions, every
  frequency base the models use, forward and inverse; an element-wise bound
  tight enough to catch an angle error of 1e-4 rad;
* the layer with RoPE fused into the projection (forward outputs, input and
  weight gradients) for every chunk size U, bitwise identical across U;
* the Llama3-8B layer width at a short sequence, full oracle."""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import layer as L
from oracle import rope as R
from tol import as64, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _upipe():
    from paper_2602_21196_amd import upipe
    upipe.lib()
    return upipe


def _bits_equal(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def _half_ulp(a):
    """Half a bf16 unit in the last place at |a| (8 significant bits)."""
    a = np.abs(a)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, 2.0 ** (e - 8), 0.0)


def _pair_norm(x):
    half = x.shape[-1] // 2
    pair = np.sqrt(x[..., :half] ** 2 + x[..., half:] ** 2)
    return np.concatenate([pair, pair], axis=-1)


def _check_rotation(got, x, ref):
    """|got - ref| <= half a bf16 ulp (the one rounding of the result) plus
    2e-5 |pair| for fp32 rotation and angle error: an angle mistake of 1e-4
    rad moves an output by up to 1e-4 |pair| and fails."""
    got, x = as64(got), as64(x)
    pair = _pair_norm(x)
    err = np.abs(got - ref)
    arith = (err - _half_ulp(np.maximum(np.abs(ref), np.abs(got)))) / np.maximum(pair, 1e-30)
    worst = float(arith.max())
    print(f"  rotation: max err {err.max():.3e}, worst (err - half ulp) / |pair| {worst:.3e}")
    assert worst <= 2e-5, worst


CASES = [  # S, H, pos0, base, inverse
    (1000, 5, 0, 1e4, 0),
    (777, 8, (1 << 31) + 12345, 5e5, 0),
    (129, 1, (1 << 32) - 129, 1e6, 1),
    (1, 3, 7, 1e4, 1),
    (4096, 32, 1 << 20, 5e5, 0),
]


@pytest.mark.parametrize("S,H,pos0,base,inverse", CASES)
def test_rope_inplace_matches_oracle(S, H, pos0, base, inverse):
    up = _upipe()
    g = torch.Generator().manual_seed(S + H)
    x = (3 * torch.randn((S, H, 128), generator=g)).to(torch.bfloat16)
    ref = R.rope(as64(x), pos0 + np.arange(S), base, inverse=bool(inverse))
    xd = x.to(DEV)
    print(f"rope S={S} H={H} pos0={pos0} base={base} inverse={inverse}", flush=True)
    up.rope(xd, base, pos0=pos0, inverse=bool(inverse))
    torch.cuda.synchronize()
    _check_rotation(xd.cpu(), x, ref)
    # and back: the first rounding (at most half an ulp of each rotated
    # coordinate, 2^-9 |pair| in all) turned back, plus one more rounding
    up.rope(xd, base, pos0=pos0, inverse=not inverse)
    torch.cuda.synchronize()
    back, x64 = as64(xd.cpu()), as64(x)
    pair = _pair_norm(x64)
    err = np.abs(back - x64)
    bound = 2.0 ** -8 * pair + 1e-4 * pair + _half_ulp(np.maximum(np.abs(x64), np.abs(back)))
    print(f"  round trip: max err {err.max():.3e}")
    assert np.all(err <= bound), float((err - bound).max())


def _run_layer(x, wqkv, wo, dy, Hq, Hkv, U, base, pos0):
    up = _upipe()
    xd, wd, wod, dyd = (t.to(DEV) for t in (x, wqkv, wo, dy))
    y, o, lse = up.layer_fwd(xd, wd, wod, Hq, Hkv, U=U, rope_base=base, pos0=pos0)
    dx, dw, dwo = up.layer_bwd(xd, wd, wod, o, lse, dyd, Hq, Hkv, U=U, rope_base=base,
                               pos0=pos0)
    torch.cuda.synchronize()
    return [t.cpu() for t in (y, o, lse, dx, dw, dwo)]


NAMES = ("y", "o_saved", "lse", "dx", "dwqkv", "dwo")
RMS = (False, False, False, False, True, True)


def _blocks(Hq, Hkv):
    d = 128
    return (None, None, None, None,
            [slice(0, Hq * d), slice(Hq * d, (Hq + Hkv) * d),
             slice((Hq + Hkv) * d, (Hq + 2 * Hkv) * d)], None)


def _oracle_layer(x, wqkv, wo, dy, Hq, Hkv, base, pos0):
    x64, w64, wo64, dy64 = (as64(t) for t in (x, wqkv, wo, dy))
    y, o, lse = L.layer_fwd(x64, w64, wo64, Hq, Hkv, 128, rope_base=base, pos0=pos0)
    dx, dw, dwo = L.layer_bwd(x64, w64, wo64, dy64, Hq, Hkv, 128, rope_base=base, pos0=pos0)
    return (y, o, lse, dx, dw, dwo)


@pytest.mark.parametrize("S,dm,Hq,Hkv,base,pos0", [(300, 256, 4, 1, 1e4, 0),
                                                   (513, 384, 4, 2, 5e5, 1 << 30),
                                                   (129, 128, 2, 2, 1e6, 3)])
def test_layer_rope_all_chunk_sizes(S, dm, Hq, Hkv, base, pos0):
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 60 + S)
    ref = _oracle_layer(x, wqkv, wo, dy, Hq, Hkv, base, pos0)
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"layer+rope S={S} dm={dm} Hq={Hq} Hkv={Hkv} U={U}", flush=True)
        got = _run_layer(x, wqkv, wo, dy, Hq, Hkv, U, base, pos0)
        for name, g, r, rs, bl in zip(NAMES, got, ref, RMS, _blocks(Hq, Hkv)):
            assert_close(f"{name} U={U}", g, r, rms_scaled=rs, blocks=bl)
        if first is None:
            first = got
        else:
            for name, a, b in zip(NAMES, first, got):
                assert _bits_equal(a, b), f"{name}: U=1 vs U={U}"


def test_layer_rope_changes_result_and_zero_base_is_plain():
    """base 0 is the plain layer; a real base changes every output."""
    S, dm, Hq, Hkv = 256, 256, 2, 1
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 5)
    up = _upipe()
    xd, wd, wod = (t.to(DEV) for t in (x, wqkv, wo))
    y0, _, _ = up.layer_fwd(xd, wd, wod, Hq, Hkv)
    y1, _, _ = up.layer_fwd(xd, wd, wod, Hq, Hkv, rope_base=0.0, pos0=12345)
    y2, _, _ = up.layer_fwd(xd, wd, wod, Hq, Hkv, rope_base=1e4)
    torch.cuda.synchronize()
    assert _bits_equal(y0, y1)
    assert not torch.equal(y0[1:], y2[1:])
    # row 0 sits at position 0 (no rotation) and sees only key 0: unchanged
    assert torch.equal(y0[0], y2[0])


@pytest.mark.timeout(300)
def test_layer_rope_llama_width_short_sequence():
    """d_model = 4096 with Llama 3's base, every output against the oracle."""
    S, dm, Hq, Hkv, base = 2048, 4096, 4, 1, 500000.0
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 8)
    ref = _oracle_layer(x, wqkv, wo, dy, Hq, Hkv, base, 0)
    got = {U: _run_layer(x, wqkv, wo, dy, Hq, Hkv, U, base, 0) for U in (1, 4)}
    for name, g, r, rs, bl in zip(NAMES, got[1], ref, RMS, _blocks(Hq, Hkv)):
        assert_close(name, g, r, rms_scaled=rs, blocks=bl)
    for name, a, b in zip(NAMES, got[1], got[4]):
        assert _bits_equal(a, b), name
