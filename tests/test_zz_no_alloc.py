"""The allocation-free forward (upipe_attn_fwd_noalloc, a static scratch array
instead of a workspace) through the C ABI against upipe_attn_fwd: bitwise
equal outputs on two calls in a row, the second with a smaller input (what
the first call left in the shared array must not leak into the second); the
size limit is rejected on the host."""

import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _upipe():
    from paper_2602_21196_amd import upipe
    upipe.lib()
    return upipe


def _bits(a):
    return a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32)


def _noalloc(up, q, k, v, causal, U):
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    o = torch.empty_like(q)
    lse = torch.empty((Hq, S), dtype=torch.float32, device=q.device)
    st = up.upipe_attn_fwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                   lse.data_ptr(), S, Hq, Hkv, d, int(causal), U,
                                   torch.cuda.current_stream().cuda_stream)
    assert st == 0, up.upipe_status_string(st)
    return o, lse


@pytest.mark.parametrize("first,second", [
    ((8192, 4, 1, True, 1), (1000, 2, 1, True, 2)),     # in place K/V, then packed, ragged
    ((4100, 8, 2, True, 4), (384, 4, 4, False, 1)),     # split key range, then non-causal
])
def test_noalloc_matches_workspace_call_twice(first, second):
    up = _upipe()
    for i, (S, Hq, Hkv, causal, U) in enumerate((first, second)):
        print(f"noalloc call {i}: S={S} Hq={Hq} Hkv={Hkv} causal={causal} U={U}", flush=True)
        q, k, v, _ = (t.to(DEV) for t in W.attention_inputs(S, Hq, Hkv, 128, 900 + S))
        o_ref, lse_ref = up.attn_fwd(q, k, v, causal=causal, U=U)
        o, lse = _noalloc(up, q, k, v, causal, U)
        torch.cuda.synchronize()
        assert torch.equal(_bits(o), _bits(o_ref)), "o differs from upipe_attn_fwd"
        assert torch.equal(_bits(lse), _bits(lse_ref)), "lse differs from upipe_attn_fwd"


def test_noalloc_rejects_shapes_beyond_its_scratch():
    up = _upipe()
    cap = up.upipe_attn_fwd_noalloc_scratch_bytes()
    assert cap == 64 << 20
    S = 1 << 20   # K, V in place but Q and O chunks alone need 512 MiB
    assert up.upipe_attn_fwd_workspace_size(S, 4, 1, 128, 1) > cap
    fake = 1 << 20
    assert up.upipe_attn_fwd_noalloc(fake, fake, fake, fake, fake, S, 4, 1, 128, 1, 1,
                                     None) == -3
    assert up.upipe_attn_fwd_noalloc(fake, fake, fake, fake, fake, 512, 4, 1, 64, 1, 1,
                                     None) == -2
    assert up.upipe_attn_fwd_noalloc(None, fake, fake, fake, fake, 512, 4, 1, 128, 1, 1,
                                     None) == -1
