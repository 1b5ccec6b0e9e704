"""MI355X (gfx950) head-chunked causal GQA attention: the per-GPU hot path of
UPipe (arXiv 2602.21196) as a C-ABI HIP library with a thin ctypes binding.

    from paper_2602_21196_amd import upipe
    o, lse = upipe.attn_fwd(q, k, v, causal=True, U=1)

The library is loaded on first use (``upipe.lib()``); nothing is imported or
built at package import time.
"""

__all__ = ["upipe"]
