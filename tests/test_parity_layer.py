"""GPU parity of the attention block (QKV projection slice, attention,
output-projection accumulation, and the backward with recomputation)."""

import numpy as np
import pytest
import torch

import workloads as W
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


def _run(x, wqkv, wo, dy, Hq, Hkv, U, rope_base=0.0):
    up = _upipe()
    xd, wd, wod, dyd = (t.to(DEV) for t in (x, wqkv, wo, dy))
    y, o, lse = up.layer_fwd(xd, wd, wod, Hq, Hkv, U=U, rope_base=rope_base)
    dx, dw, dwo = up.layer_bwd(xd, wd, wod, o, lse, dyd, Hq, Hkv, U=U, rope_base=rope_base)
    torch.cuda.synchronize()
    return [t.cpu() for t in (y, o, lse, dx, dw, dwo)]


NAMES = ("y", "o_saved", "lse", "dx", "dwqkv", "dwo")
RMS = (False, False, False, False, True, True)


def _blocks(Hq, Hkv):
    """Per-output-block scales: the Q, K, V column groups of dWqkv."""
    d = 128
    return (None, None, None, None,
            [slice(0, Hq * d), slice(Hq * d, (Hq + Hkv) * d),
             slice((Hq + Hkv) * d, (Hq + 2 * Hkv) * d)], None)


@pytest.mark.parametrize("S,dm,Hq,Hkv", [(300, 256, 4, 1), (513, 384, 4, 2),
                                         (128, 128, 2, 2), (1, 256, 2, 1)])
def test_layer_small_all_chunk_sizes(S, dm, Hq, Hkv):
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 40 + S)
    x64, w64, wo64, dy64 = (as64(t) for t in (x, wqkv, wo, dy))
    y, o, lse = L.layer_fwd(x64, w64, wo64, Hq, Hkv, 128)
    dx, dw, dwo = L.layer_bwd(x64, w64, wo64, dy64, Hq, Hkv, 128)
    ref = (y, o, lse, dx, dw, dwo)
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"layer S={S} dm={dm} Hq={Hq} Hkv={Hkv} U={U}", flush=True)
        got = _run(x, wqkv, wo, dy, Hq, Hkv, U)
        for name, g, r, rs, bl in zip(NAMES, got, ref, RMS, _blocks(Hq, Hkv)):
            assert_close(f"{name} U={U}", g, r, rms_scaled=rs, blocks=bl)
        if first is None:
            first = got
        else:
            for name, a, b in zip(NAMES, first, got):
                assert _bits_equal(a, b), f"{name}: U=1 vs U={U}"


@pytest.mark.timeout(300)
def test_layer_llama_width_short_sequence():
    """d_model = 4096 as in the Llama3-8B layer share, S short enough for the
    full oracle: every output including the weight gradients."""
    S, dm, Hq, Hkv = 2048, 4096, 4, 1
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 7)
    x64, w64, wo64, dy64 = (as64(t) for t in (x, wqkv, wo, dy))
    y, o, lse = L.layer_fwd(x64, w64, wo64, Hq, Hkv, 128)
    dx, dw, dwo = L.layer_bwd(x64, w64, wo64, dy64, Hq, Hkv, 128)
    got = {}
    for U in (1, 4):
        got[U] = _run(x, wqkv, wo, dy, Hq, Hkv, U)
    for name, g, r, rs, bl in zip(NAMES, got[1], (y, o, lse, dx, dw, dwo), RMS,
                                  _blocks(Hq, Hkv)):
        assert_close(name, g, r, rms_scaled=rs, blocks=bl)
    for name, a, b in zip(NAMES, got[1], got[4]):
        assert _bits_equal(a, b), name


@pytest.mark.timeout(900)
def test_llama8b_layer_share_sampled():
    """The Llama3-8B layer share (S = 256K, d_model = 4096, RoPE with Llama 3's
    base): bitwise equal across U and between kept and recomputed attention
    output; sampled rows, the dX tail, and weight-gradient columns over the
    whole sequence against the oracle."""
    w = W.WORKLOADS["llama8b_layer"]
    S, dm, Hq, Hkv, d = w.S, w.d_model, w.Hq, w.Hkv, w.d
    base = w.extra.get("rope_base")
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, d, w.seed)
    outs = {}
    for U in w.U_sweep:
        print(f"llama8b_layer S={S} U={U} rope_base={base}", flush=True)
        outs[U] = _run(x, wqkv, wo, dy, Hq, Hkv, U, rope_base=base or 0.0)
    for U in w.U_sweep[1:]:
        for name, a, b in zip(NAMES, outs[1], outs[U]):
            assert _bits_equal(a, b), f"{name}: U=1 vs U={U}"
    # full checkpointing (attention output recomputed in the backward), as
    # bench.py --checkpointing full times it: bitwise the kept-output result
    print(f"llama8b_layer S={S} U=1 full checkpointing", flush=True)
    up = _upipe()
    xd, wd, wod, dyd = (t.to(DEV) for t in (x, wqkv, wo, dy))
    full = up.layer_bwd(xd, wd, wod, None, None, dyd, Hq, Hkv, U=1, rope_base=base or 0.0)
    torch.cuda.synchronize()
    for name, a, b in zip(("dx", "dwqkv", "dwo"), outs[1][3:], full):
        assert _bits_equal(a, b.cpu()), f"{name}: kept vs recomputed output"
    del xd, wd, wod, dyd, full
    y, o, lse, dx, dwqkv, dwo = outs[1]
    x64, w64, wo64, dy64 = (as64(t) for t in (x, wqkv, wo, dy))
    rows = W.sample_rows(S, 128, w.seed)
    print("oracle sampled rows", flush=True)
    y_r, o_r, lse_r = L.layer_fwd_rows(x64, w64, wo64, Hq, Hkv, d, rows, rope_base=base)
    assert_close("y rows", y[rows], y_r)
    assert_close("o rows", o[rows], o_r)
    assert_close("lse rows", lse[:, rows], lse_r)
    # dX on the last rows: dq rows are row-local, dk/dv of the key tail need
    # only the query rows at or after it.
    j0 = S - 256
    print("oracle dx tail", flush=True)
    assert_close("dx tail rows", dx[j0:],
                 L.layer_bwd_tail(x64, w64, wo64, dy64, Hq, Hkv, d, j0, rope_base=base))
    # dWo over the whole sequence (the fixed split-K path with all its pieces),
    # on sampled columns, conditioned on the GPU's saved attention output.
    cols = W.sample_key_cols(dm, 64, w.seed)
    print(f"oracle dwo: {len(cols)} columns conditioned on the GPU's o_saved", flush=True)
    assert_close("dwo cols (conditioned on GPU o_saved)", dwo[:, cols],
                 L.dwo_given_output(o.float().numpy(), dy64, cols), rms_scaled=True)
    # dWqkv over the whole sequence (the same split-K path) on sampled columns
    # of the Q, K and V groups, conditioned on attention gradients: the
    # attention entry points of this library run on bf16 q, k, v, dO that the
    # oracle forms in float64 from x, Wqkv, Wo and dY, and the oracle takes
    # x^T [dQ | dK | dV] of their output (rotated gradients turned back).
    print("oracle dwqkv: attention operands in float64", flush=True)
    qa, ka, va, doa = L.attention_inputs(x64, w64, wo64, dy64, Hq, Hkv, d, rope_base=base)
    up = _upipe()
    ops = [torch.from_numpy(t).to(torch.bfloat16).to(DEV) for t in (qa, ka, va, doa)]
    del qa, ka, va, doa
    o_a, lse_a = up.attn_fwd(ops[0], ops[1], ops[2], U=1)
    grads = up.attn_bwd(ops[0], ops[1], ops[2], o_a, lse_a, ops[3], U=1)
    torch.cuda.synchronize()
    dq_a, dk_a, dv_a = (as64(t) for t in grads)
    del ops, o_a, lse_a, grads
    qcols = W.sample_key_cols(Hq * d, 24, w.seed)
    kcols = [Hq * d + c for c in W.sample_key_cols(Hkv * d, 20, w.seed + 1)]
    vcols = [(Hq + Hkv) * d + c for c in W.sample_key_cols(Hkv * d, 20, w.seed + 2)]
    cols = qcols + kcols + vcols
    print(f"oracle dwqkv: {len(cols)} columns", flush=True)
    ref = L.dwqkv_given_grads(x64, dq_a, dk_a, dv_a, cols, rope_base=base)
    nq, nk = len(qcols), len(kcols)
    assert_close("dwqkv cols (conditioned on attention-entry-point dQ, dK, dV)", dwqkv[:, cols],
                 ref, rms_scaled=True,
                 blocks=[slice(0, nq), slice(nq, nq + nk), slice(nq + nk, len(cols))])


@pytest.mark.parametrize("S,dm,Hq,Hkv,base", [(300, 256, 4, 1, 0.0), (513, 384, 4, 2, 5e5),
                                              (2048, 1024, 8, 2, 1e6)])
def test_full_checkpointing_equals_kept_output(S, dm, Hq, Hkv, base):
    """Backward without the saved attention output (each chunk's forward
    recomputed) gives bitwise the results of the backward that reads it, for
    every U; and both match the oracle."""
    up = _upipe()
    x, wqkv, wo, dy = W.layer_inputs(S, dm, Hq, Hkv, 128, 80 + S)
    xd, wd, wod, dyd = (t.to(DEV) for t in (x, wqkv, wo, dy))
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"full checkpointing S={S} dm={dm} Hq={Hq} Hkv={Hkv} U={U}", flush=True)
        y, o, lse = up.layer_fwd(xd, wd, wod, Hq, Hkv, U=U, rope_base=base)
        kept = up.layer_bwd(xd, wd, wod, o, lse, dyd, Hq, Hkv, U=U, rope_base=base)
        full = up.layer_bwd(xd, wd, wod, None, None, dyd, Hq, Hkv, U=U, rope_base=base)
        torch.cuda.synchronize()
        for name, a, b in zip(("dx", "dwqkv", "dwo"), kept, full):
            assert _bits_equal(a, b), f"{name}: kept vs recomputed output, U={U}"
        if first is None:
            first = [t.cpu() for t in full]
        else:
            for name, a, b in zip(("dx", "dwqkv", "dwo"), first, full):
                assert _bits_equal(a, b.cpu()), f"{name}: U=1 vs U={U}"
    x64, w64, wo64, dy64 = (as64(t) for t in (x, wqkv, wo, dy))
    rb = base if base else None
    ref = L.layer_bwd(x64, w64, wo64, dy64, Hq, Hkv, 128, rope_base=rb)
    for name, g, r, bl in zip(("dx", "dwqkv", "dwo"), first, ref, (None, _blocks(Hq, Hkv)[4], None)):
        assert_close(name, g, r, rms_scaled=name != "dx", blocks=bl)
