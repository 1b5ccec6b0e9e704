"""CPU oracle for head-chunked causal GQA attention (UPipe, arXiv 2602.21196).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
path (``paper_2602_21196_amd``) and imports nothing from it.

Everything here is plain numpy in float64, written from the paper's
definitions so that each function can be checked against the paper by eye:

* ``attention``  -- causal softmax attention with grouped key/value heads
  (Section 2.1, "Multi-head Attention") and its analytic gradient.
* ``layer``      -- the attention block around it: QKV projection,
  attention, output projection (Section 3.2 walk-through, Appendix A
  paragraphs on the forward and backward of the block).
* ``ring``       -- one ring step of context-parallel attention (a query
  block against a key/value block at another offset) and the log-sum-exp
  merge of partial results (Section 2.2, Section 4 "Implementation").
* ``rope``       -- rotary position embedding of queries and keys and its
  inverse (Section 4 "Implementation", RoFormer's definition).
* ``schedule``   -- the head-chunk plan: nu = H/U stages and the GQA
  out-of-order head schedule with its communication count (Section 4.1,
  "Grouped-Query Attention Scheduling"; Section 3.3 "Untied Ulysses").
* ``memory``     -- the paper's activation-memory accounting (Section 3.4
  "Memory Savings", Tables ``tab:gqa_fwd_mem`` and ``tab:gqa_bwd_mem``).

Every function is pinned by ``tests/test_oracle_*.py`` against things other
than itself: closed forms, brute-force scalar loops, torch's fp64
``scaled_dot_product_attention`` and autograd, finite differences, exact
invariants and the values the paper prints.
"""

from . import attention, layer, memory, ring, rope, schedule  # noqa: F401
