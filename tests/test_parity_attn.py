"""GPU parity: the HIP attention path (through the C ABI) against the oracle.

Element-by-element on small and ragged shapes, sampled rows plus exact
invariants at the Llama3-8B per-GPU share (S = 131072, Hq = 4, Hkv = 1),
bitwise identity across chunk sizes U and across repeated calls.
"""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as A
from tol import as64, assert_close

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _upipe():
    from paper_2602_21196_amd import upipe
    upipe.lib()
    return upipe


def _run(q, k, v, do, causal, U):
    up = _upipe()
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o, lse = up.attn_fwd(qd, kd, vd, causal=causal, U=U)
    dq, dk, dv = up.attn_bwd(qd, kd, vd, o, lse, dod, causal=causal, U=U)
    torch.cuda.synchronize()
    return [t.cpu() for t in (o, lse, dq, dk, dv)]


def _bits_equal(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def _oracle(q, k, v, do, causal):
    q64, k64, v64, do64 = (as64(t) for t in (q, k, v, do))
    o, lse = A.attn_fwd(q64, k64, v64, causal)
    dq, dk, dv = A.attn_bwd(q64, k64, v64, do64, causal)
    return o, lse, dq, dk, dv


NAMES = ("o", "lse", "dq", "dk", "dv")


def test_tiny_workload_both_chunk_sizes():
    w = W.WORKLOADS["tiny"]
    q, k, v, do = W.attention_inputs(w.S, w.Hq, w.Hkv, w.d, w.seed)
    ref = _oracle(q, k, v, do, True)
    outs = {}
    for U in w.U_sweep:
        print(f"tiny S={w.S} Hq={w.Hq} Hkv={w.Hkv} U={U}", flush=True)
        outs[U] = _run(q, k, v, do, True, U)
        for name, got, r in zip(NAMES, outs[U], ref):
            assert_close(f"{name} U={U}", got, r)
    for a, b in zip(outs[1], outs[2]):
        assert _bits_equal(a, b)


SHAPES = [
    # S, Hq, Hkv, causal
    (1, 1, 1, True),
    (17, 2, 1, True),
    (129, 4, 1, True),
    (300, 6, 3, True),      # groups of 2 split by U = 3 (carried dK/dV)
    (1000, 8, 2, True),
    (200, 4, 4, True),
    (257, 2, 1, False),
    (96, 4, 2, False),
    (2500, 4, 2, False),    # many tiles, ragged tail; the forward splits its key range
    (4100, 8, 2, True),     # U = 2: carried per-head dK/dV; U = 4: one group per launch;
                            # U = 8: two groups per launch
]


@pytest.mark.parametrize("S,Hq,Hkv,causal", SHAPES)
def test_shapes_all_chunk_sizes(S, Hq, Hkv, causal):
    q, k, v, do = W.attention_inputs(S, Hq, Hkv, 128, 100 + S + Hq)
    ref = _oracle(q, k, v, do, causal)
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"shape S={S} Hq={Hq} Hkv={Hkv} causal={causal} U={U}", flush=True)
        got = _run(q, k, v, do, causal, U)
        for name, g, r in zip(NAMES, got, ref):
            assert_close(f"{name} S={S} U={U}", g, r)
        if first is None:
            first = got
        else:
            for name, a, b in zip(NAMES, first, got):
                assert _bits_equal(a, b), f"{name} differs between U=1 and U={U}"


def test_repeat_calls_are_bitwise_identical():
    q, k, v, do = W.attention_inputs(700, 4, 1, 128, 11)
    a = _run(q, k, v, do, True, 2)
    b = _run(q, k, v, do, True, 2)
    for name, x, y in zip(NAMES, a, b):
        assert _bits_equal(x, y), name


def test_workspace_contents_do_not_leak_between_calls():
    up = _upipe()
    q, k, v, do = (t.to(DEV) for t in W.attention_inputs(384, 2, 1, 128, 12))
    need = up.upipe_attn_bwd_workspace_size(384, 2, 1, 128, 1)
    ws = torch.full((need,), 0x7F, dtype=torch.uint8, device=DEV)
    o, lse = up.attn_fwd(q, k, v, U=1)
    g1 = up.attn_bwd(q, k, v, o, lse, do, U=1, ws=ws)
    ws.fill_(0xFF)  # NaN patterns everywhere
    g2 = up.attn_bwd(q, k, v, o, lse, do, U=1, ws=ws)
    torch.cuda.synchronize()
    for a, b in zip(g1, g2):
        assert _bits_equal(a.cpu(), b.cpu())


@pytest.mark.timeout(600)
def test_llama8b_share_sampled_rows_and_invariants():
    w = W.WORKLOADS["llama8b_share"]
    S, Hq, Hkv, d = w.S, w.Hq, w.Hkv, w.d
    q, k, v, do = W.attention_inputs(S, Hq, Hkv, d, w.seed)
    outs = {}
    for U in w.U_sweep:
        print(f"llama8b_share S={S} U={U}", flush=True)
        outs[U] = _run(q, k, v, do, True, U)
    for U in w.U_sweep[1:]:
        for name, a, b in zip(NAMES, outs[w.U_sweep[0]], outs[U]):
            assert _bits_equal(a, b), f"{name} differs between U=1 and U={U}"
    o, lse, dq, dk, dv = outs[1]
    q64, k64, v64, do64 = (as64(t) for t in (q, k, v, do))
    rows = W.sample_rows(S, 256, w.seed)
    print(f"oracle rows={len(rows)}", flush=True)
    o_r, lse_r = A.attn_fwd(q64, k64, v64, True, rows=rows)
    assert_close("o rows", o[rows], o_r)
    assert_close("lse rows", lse[:, rows], lse_r)
    dq_r, _ = A.attn_bwd_rows(q64, k64, v64, do64, rows)
    assert_close("dq rows", dq[rows], dq_r)
    j0 = S - 512
    print("oracle key tail", flush=True)
    dk_t, dv_t = A.attn_bwd_key_tail(q64, k64, v64, do64, j0)
    assert_close("dk tail", dk[j0:], dk_t)
    assert_close("dv tail", dv[j0:], dv_t)
    # Interior keys (the longest fp32 chains, key 0 gathers from every row):
    # dK_j, dV_j in float64 from the definition, conditioned on the GPU's lse
    # and on D = dO.O from the GPU's O.
    cols = W.sample_key_cols(S, 64, w.seed)
    print(f"oracle: {len(cols)} key columns conditioned on the GPU's lse and O", flush=True)
    dk_c, dv_c = A.attn_key_cols_given(q.float().numpy(), do.float().numpy(), k64, v64,
                                       o.float().numpy(), lse.numpy(), cols)
    assert_close("dk cols (conditioned on GPU lse, D)", dk[cols], dk_c)
    assert_close("dv cols (conditioned on GPU lse)", dv[cols], dv_c)
    # Whole-tensor invariants: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i.
    dk64, dv64 = as64(dk), as64(dv)
    col_scale = np.sqrt(S) * np.sqrt(np.mean(dk64 ** 2, axis=0))
    assert np.all(np.abs(dk64.sum(axis=0)) <= 0.05 * col_scale + 1e-6)
    ref_dv = do64.sum(axis=(0, 1))
    dv_sum = dv64.sum(axis=0)[0]
    scale = np.sqrt(S) * np.sqrt(np.mean(dv64 ** 2))
    assert np.all(np.abs(dv_sum - ref_dv) <= 0.05 * scale + 1e-6)
    print(f"dk col-sum max {np.abs(dk64.sum(axis=0)).max():.3e} "
          f"dv sum err max {np.abs(dv_sum - ref_dv).max():.3e}", flush=True)
