"""GPU parity of batched calls (B > 1 sequences through one workspace):
every sequence of a batch gives bitwise what a call on that sequence alone
gives; the layer's weight gradients are the sum over the batch, checked
against the oracle's per-sequence gradients summed."""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as A
from oracle import layer as L
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


@pytest.mark.parametrize("B,S,Hq,Hkv,U", [(3, 300, 4, 1, 2), (2, 1000, 8, 2, 4), (4, 129, 2, 2, 1)])
def test_attention_batch_equals_single_sequences(B, S, Hq, Hkv, U):
    up = _upipe()
    seqs = [W.attention_inputs(S, Hq, Hkv, 128, 300 + b) for b in range(B)]
    q, k, v, do = (torch.stack([s[i] for s in seqs]).to(DEV) for i in range(4))
    print(f"batch B={B} S={S} Hq={Hq} Hkv={Hkv} U={U}", flush=True)
    o, lse = up.attn_fwd(q, k, v, causal=True, U=U)
    dq, dk, dv = up.attn_bwd(q, k, v, o, lse, do, causal=True, U=U)
    assert tuple(lse.shape) == (B, Hq, S)
    for b in range(B):
        o1, l1 = up.attn_fwd(q[b], k[b], v[b], causal=True, U=U)
        g1 = up.attn_bwd(q[b], k[b], v[b], o1, l1, do[b], causal=True, U=U)
        torch.cuda.synchronize()
        assert _bits_equal(o[b], o1) and _bits_equal(lse[b], l1), b
        for name, a, c in zip(("dq", "dk", "dv"), (dq[b], dk[b], dv[b]), g1):
            assert _bits_equal(a, c), (name, b)
    # the last sequence against the oracle (offsets into the batch are right)
    b = B - 1
    q64, k64, v64, do64 = (as64(t) for t in seqs[b])
    o_r, lse_r = A.attn_fwd(q64, k64, v64, True)
    dq_r, dk_r, dv_r = A.attn_bwd(q64, k64, v64, do64, True)
    assert_close("o", o[b].cpu(), o_r)
    assert_close("lse", lse[b].cpu(), lse_r)
    assert_close("dq", dq[b].cpu(), dq_r)
    assert_close("dk", dk[b].cpu(), dk_r)
    assert_close("dv", dv[b].cpu(), dv_r)


@pytest.mark.parametrize("B,S,dm,Hq,Hkv,base,full", [(2, 300, 256, 4, 1, 0.0, False),
                                                     (3, 256, 384, 4, 2, 5e5, False),
                                                     (2, 513, 256, 2, 1, 1e4, True)])
def test_layer_batch(B, S, dm, Hq, Hkv, base, full):
    """Per-sequence outputs bitwise equal to single calls; weight gradients
    equal the oracle's sum over the batch; bitwise equal across U."""
    up = _upipe()
    x0, wqkv, wo, dy0 = W.layer_inputs(S, dm, Hq, Hkv, 128, 500 + S)
    g = torch.Generator().manual_seed(S)
    xs = [x0] + [torch.randn((S, dm), generator=g).to(torch.bfloat16) for _ in range(B - 1)]
    dys = [dy0] + [torch.randn((S, dm), generator=g).to(torch.bfloat16) for _ in range(B - 1)]
    x = torch.stack(xs).to(DEV)
    dy = torch.stack(dys).to(DEV)
    wd, wod = wqkv.to(DEV), wo.to(DEV)
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"layer batch B={B} S={S} dm={dm} Hq={Hq} Hkv={Hkv} U={U} full={full}", flush=True)
        y, o, lse = up.layer_fwd(x, wd, wod, Hq, Hkv, U=U, rope_base=base)
        if full:
            dx, dw, dwo = up.layer_bwd(x, wd, wod, None, None, dy, Hq, Hkv, U=U, rope_base=base)
        else:
            dx, dw, dwo = up.layer_bwd(x, wd, wod, o, lse, dy, Hq, Hkv, U=U, rope_base=base)
        torch.cuda.synchronize()
        got = [t.cpu() for t in (y, o, lse, dx, dw, dwo)]
        if first is None:
            first = got
            for b in range(B):   # every sequence as if alone
                y1, o1, l1 = up.layer_fwd(x[b], wd, wod, Hq, Hkv, U=U, rope_base=base)
                dx1, _, _ = up.layer_bwd(x[b], wd, wod, o1, l1, dy[b], Hq, Hkv, U=U,
                                         rope_base=base)
                torch.cuda.synchronize()
                for name, a, c in zip(("y", "o", "lse", "dx"), (y[b], o[b], lse[b], dx[b]),
                                      (y1, o1, l1, dx1)):
                    assert _bits_equal(a, c), (name, b)
        else:
            for name, a, c in zip(("y", "o", "lse", "dx", "dwqkv", "dwo"), first, got):
                assert _bits_equal(a, c), f"{name}: U=1 vs U={U}"
    rb = base if base else None
    w64, wo64 = as64(wqkv), as64(wo)
    dw_sum = dwo_sum = 0.0
    for b in range(B):
        _, dw_r, dwo_r = L.layer_bwd(as64(xs[b]), w64, wo64, as64(dys[b]), Hq, Hkv, 128,
                                     rope_base=rb)
        dw_sum = dw_sum + dw_r
        dwo_sum = dwo_sum + dwo_r
    d = 128
    blocks = [slice(0, Hq * d), slice(Hq * d, (Hq + Hkv) * d),
              slice((Hq + Hkv) * d, (Hq + 2 * Hkv) * d)]
    assert_close("dwqkv (sum over batch)", first[4], dw_sum, rms_scaled=True, blocks=blocks)
    assert_close("dwo (sum over batch)", first[5], dwo_sum, rms_scaled=True)
