"""GPU parity of the ring step (upipe_attn_fwd_ring) and the LSE merge
(upipe_lse_merge) against the oracle (oracle/ring.py), through the C ABI.

Cases: query/key blocks of ragged lengths at negative, zero and positive
offsets (rows that see no key, the diagonal, fully visible blocks),
non-causal blocks, grouped heads and every chunk size U; the merge on random
partials including empty rows; full causal attention rebuilt on the GPU
from ring steps over key blocks plus merges; and the full-size ring step of
the Llama3-8B share (32K queries against 32K keys, the forward's key range
split in two), on sampled rows."""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as A
from oracle import ring as R
from tol import as64, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _upipe():
    from paper_2602_21196_amd import upipe
    upipe.lib()
    return upipe


def _inputs(Sq, Skv, Hq, Hkv, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((Sq, Hq, 128), generator=g).to(torch.bfloat16)
    k = torch.randn((Skv, Hkv, 128), generator=g).to(torch.bfloat16)
    v = torch.randn((Skv, Hkv, 128), generator=g).to(torch.bfloat16)
    return q, k, v


def _check_lse(name, got, ref):
    got = got.double().numpy()
    empty = np.isneginf(ref)
    assert np.array_equal(np.isneginf(got), empty), f"{name}: empty rows differ"
    assert_close(name, torch.from_numpy(np.where(empty, 0.0, got)), np.where(empty, 0.0, ref))


CASES = [  # Sq, Skv, q_offset, kv_offset, Hq, Hkv, causal
    (256, 256, 0, 0, 2, 1, True),          # plain causal
    (300, 129, 500, 200, 4, 2, True),      # keys entirely in the past, partly masked
    (200, 333, 0, 150, 2, 1, True),        # keys start after the first queries: empty rows
    (129, 500, 1000, 0, 2, 2, True),       # all keys visible
    (257, 100, 0, 5000, 2, 1, True),       # no key visible to any row
    (96, 300, 40, 40, 4, 1, False),        # non-causal block
    (1000, 777, 1777, 1000, 8, 2, True),   # several tiles and stages, ragged tails
]


@pytest.mark.parametrize("Sq,Skv,qo,ko,Hq,Hkv,causal", CASES)
def test_ring_step_matches_oracle(Sq, Skv, qo, ko, Hq, Hkv, causal):
    up = _upipe()
    q, k, v = _inputs(Sq, Skv, Hq, Hkv, seed=Sq + 7 * Skv)
    o_ref, lse_ref = R.attn_fwd_offset(as64(q), as64(k), as64(v), qo - ko, causal)
    ref = None
    for U in [u for u in (1, 2, 4, 8) if Hq % u == 0]:
        o, lse = up.attn_fwd_ring(q.to(DEV), k.to(DEV), v.to(DEV), qo, ko, causal=causal, U=U)
        torch.cuda.synchronize()
        o, lse = o.cpu(), lse.cpu()
        if ref is None:
            assert_close("o", o, o_ref)
            _check_lse("lse", lse, lse_ref)
            ref = (o, lse)
        else:   # chunk size changes nothing, bit for bit
            assert torch.equal(o.view(torch.int16), ref[0].view(torch.int16))
            assert torch.equal(lse.view(torch.int32), ref[1].view(torch.int32))


def test_ring_step_equal_lengths_is_the_plain_forward():
    up = _upipe()
    q, k, v = _inputs(777, 777, 4, 1, seed=3)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    o1, l1 = up.attn_fwd(qd, kd, vd, causal=True, U=2)
    o2, l2 = up.attn_fwd_ring(qd, kd, vd, 12345, 12345, causal=True, U=2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))


def test_lse_merge_matches_oracle():
    up = _upipe()
    S, H = 1000, 6
    g = torch.Generator().manual_seed(11)
    o_a = torch.randn((S, H, 128), generator=g).to(torch.bfloat16)
    o_b = torch.randn((S, H, 128), generator=g).to(torch.bfloat16)
    lse_a = (3 * torch.randn((H, S), generator=g)).float()
    lse_b = (3 * torch.randn((H, S), generator=g)).float()
    lse_a[0, :50] = -float("inf")                 # empty a
    lse_b[1, 20:80] = -float("inf")               # empty b
    lse_a[2, 100:120] = -float("inf")
    lse_b[2, 100:120] = -float("inf")             # both empty
    lse_b[3, :] = lse_a[3, :] + 40.0              # b dominates
    o_ref, lse_ref = R.lse_merge(as64(o_a), lse_a.double().numpy(), as64(o_b),
                                 lse_b.double().numpy())
    od, ld = o_a.to(DEV), lse_a.to(DEV)
    up.lse_merge(od, ld, o_b.to(DEV), lse_b.to(DEV))
    torch.cuda.synchronize()
    assert_close("o", od.cpu(), o_ref)
    _check_lse("lse", ld.cpu(), lse_ref)
    assert torch.all(od.cpu()[100:120, 2].float() == 0)


@pytest.mark.parametrize("S,cuts", [(1024, (0, 256, 512, 768, 1024)),
                                    (1000, (0, 333, 700, 1000))])
def test_ring_decomposition_rebuilds_causal_attention(S, cuts):
    """Queries [qa, qb) against key blocks [a, b) at their global offsets,
    merged on the GPU, give the causal attention of those rows."""
    up = _upipe()
    q, k, v = _inputs(S, S, 4, 1, seed=S)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    qa, qb = 128, S - 100
    o_acc = torch.zeros((qb - qa, 4, 128), dtype=torch.bfloat16, device=DEV)
    lse_acc = torch.full((4, qb - qa), -float("inf"), dtype=torch.float32, device=DEV)
    for a, b in zip(cuts[:-1], cuts[1:]):
        o_p, lse_p = up.attn_fwd_ring(qd[qa:qb].contiguous(), kd[a:b].contiguous(),
                                      vd[a:b].contiguous(), qa, a, causal=True, U=1)
        up.lse_merge(o_acc, lse_acc, o_p, lse_p)
    torch.cuda.synchronize()
    rows = np.arange(qa, qb)
    o_ref, lse_ref = A.attn_fwd(as64(q), as64(k), as64(v), causal=True, rows=rows)
    assert_close("o", o_acc.cpu(), o_ref)
    assert_close("lse", lse_acc.cpu(), lse_ref)
    o_full, lse_full = up.attn_fwd(qd, kd, vd, causal=True, U=1)
    torch.cuda.synchronize()
    # against the GPU's own one-block forward: only bf16 rounding of the partials
    diff = (o_acc.cpu().float() - o_full.cpu()[qa:qb].float()).abs().max().item()
    assert diff <= 2.0 ** -6, diff


@pytest.mark.timeout(300)
def test_llama8b_ring_step_sampled():
    """The ring step bench.py times (a 32K query block against the preceding
    32K key/value block, Llama3-8B share split four ways), in the launch
    configuration it times: bitwise equal across U; sampled rows of the
    step and of its merge into the block's own causal result against the
    oracle.  Every key of the block is visible to every row, so the oracle's
    offset attention over the sampled rows alone is exact."""
    up = _upipe()
    w = W.WORKLOADS["llama8b_ring"]
    Sq, Skv, Hq, Hkv = w.S, w.extra["kv_len"], w.Hq, w.Hkv
    qo, ko = w.extra["q_offset"], w.extra["kv_offset"]
    assert qo - ko >= Skv - 1
    q, k, v = W.inputs_for(w)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    outs = {}
    for U in w.U_sweep:
        print(f"llama8b_ring Sq={Sq} Skv={Skv} U={U}", flush=True)
        o, lse = up.attn_fwd_ring(qd, kd, vd, qo, ko, causal=True, U=U)
        torch.cuda.synchronize()
        outs[U] = (o, lse)
    o1, l1 = outs[w.U_sweep[0]]
    for U in w.U_sweep[1:]:
        assert torch.equal(outs[U][0].view(torch.int16), o1.view(torch.int16)), U
        assert torch.equal(outs[U][1].view(torch.int32), l1.view(torch.int32)), U
    rows = W.sample_rows(Sq, 128, w.seed)
    print("oracle sampled rows", flush=True)
    o_r, lse_r = R.attn_fwd_offset(as64(q[rows]), as64(k), as64(v), qo - ko)
    o_c, l_c = o1.cpu(), l1.cpu()
    assert_close("o rows", o_c[rows], o_r)
    _check_lse("lse rows", l_c[:, rows], lse_r)
    # merged into the block's own causal part (keys = the block's first
    # Hkv query heads, as in bench.py's running result)
    kself = q[:, :Hkv].contiguous()
    ksd = kself.to(DEV)
    o_acc, lse_acc = up.attn_fwd_ring(qd, ksd, ksd, qo, qo, causal=True, U=1)
    up.lse_merge(o_acc, lse_acc, o1, l1)
    torch.cuda.synchronize()
    o_own, lse_own = A.attn_rows_at(as64(q[rows]), np.asarray(rows), as64(kself), as64(kself),
                                    causal=True)
    o_m, lse_m = R.lse_merge(o_own, lse_own, o_r, lse_r)
    assert_close("merged o rows", o_acc.cpu()[rows], o_m)
    _check_lse("merged lse rows", lse_acc.cpu()[:, rows], lse_m)
