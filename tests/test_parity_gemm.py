"""GPU parity of the projection product on its own (upipe_gemm_bf16, the
kernel behind the block's QKV and output projections) against the float64
product of the same bf16 inputs (a plain matrix product: numpy is the
library routine)."""

import numpy as np
import pytest
import torch

from tol import as64, assert_close

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("M,N,K,std_b", [(256, 384, 512, 1.0), (1024, 128, 4096, 0.02),
                                         (128, 1024, 128, 1.0), (2048, 4096, 512, 0.02)])
def test_gemm_against_float64_product(M, N, K, std_b):
    from paper_2602_21196_amd import upipe
    g = torch.Generator().manual_seed(M + N + K)
    a = torch.randn((M, K), generator=g).to(torch.bfloat16)
    b = (torch.randn((K, N), generator=g) * std_b).to(torch.bfloat16)
    print(f"gemm M={M} N={N} K={K}", flush=True)
    c = upipe.gemm(a.to(DEV), b.to(DEV))
    c2 = upipe.gemm(a.to(DEV), b.to(DEV))
    torch.cuda.synchronize()
    ref = as64(a) @ as64(b)
    # entries grow like sqrt(K) std_b: the max-abs bar on the rms-scaled error
    assert_close("c", c.cpu(), ref, rms_scaled=True)
    assert torch.equal(c.view(torch.int16), c2.view(torch.int16))
