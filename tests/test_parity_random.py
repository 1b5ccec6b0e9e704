"""GPU parity on seeded random valid shapes: lengths from 1 to 3000 (tile
edges and ragged tails), 1-4 key/value heads, groups of 1-4 query heads,
causal or not.  For every valid chunk size U the outputs are bitwise equal,
and they match the oracle element by element; the allocation-free forward
matches the workspace forward bitwise."""

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as A
from tol import as64, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _shapes(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        S = int(rng.choice([int(rng.integers(1, 300)), int(rng.integers(300, 3000)),
                            128 * int(rng.integers(1, 24)) + int(rng.choice([-1, 0, 1]))]))
        Hkv = int(rng.choice([1, 2, 4]))
        G = int(rng.choice([1, 2, 4]))
        out.append((max(S, 1), Hkv * G, Hkv, bool(rng.integers(0, 2))))
    return out


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("S,Hq,Hkv,causal", _shapes(12, 2024))
def test_random_shape(S, Hq, Hkv, causal):
    from paper_2602_21196_amd import upipe
    q, k, v, do = W.attention_inputs(S, Hq, Hkv, 128, 7000 + S + Hq)
    q64, k64, v64, do64 = (as64(t) for t in (q, k, v, do))
    o_r, lse_r = A.attn_fwd(q64, k64, v64, causal)
    dq_r, dk_r, dv_r = A.attn_bwd(q64, k64, v64, do64, causal)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    first = None
    for U in [u for u in range(1, Hq + 1) if Hq % u == 0]:
        print(f"random shape S={S} Hq={Hq} Hkv={Hkv} causal={causal} U={U}", flush=True)
        o, lse = upipe.attn_fwd(qd, kd, vd, causal=causal, U=U)
        g = upipe.attn_bwd(qd, kd, vd, o, lse, dod, causal=causal, U=U)
        torch.cuda.synchronize()
        got = [t.cpu() for t in (o, lse) + tuple(g)]
        if first is None:
            first = got
            for name, a, r in zip(("o", "lse", "dq", "dk", "dv"), got,
                                  (o_r, lse_r, dq_r, dk_r, dv_r)):
                assert_close(name, a, r)
        else:
            for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), first, got):
                assert torch.equal(_bits(a), _bits(b)), f"{name}: U=1 vs U={U}"
        need = upipe.upipe_attn_fwd_workspace_size(S, Hq, Hkv, 128, U)
        if need <= upipe.upipe_attn_fwd_noalloc_scratch_bytes():
            o2 = torch.empty_like(qd)
            lse2 = torch.empty_like(lse)
            st = upipe.upipe_attn_fwd_noalloc(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(),
                                              o2.data_ptr(), lse2.data_ptr(), S, Hq, Hkv, 128,
                                              int(causal), U,
                                              torch.cuda.current_stream().cuda_stream)
            assert st == 0
            torch.cuda.synchronize()
            assert torch.equal(_bits(o2), _bits(o)) and torch.equal(_bits(lse2), _bits(lse))
