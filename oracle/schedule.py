"""Oracle: the head-chunk plan and the GQA head schedule.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 3.3 ("Untied Ulysses"): with H heads and C context-parallel devices
the attention block runs in nu = H/U stages of U heads each; U must be a
multiple of C so every device gets U/C heads per stage.

Section 3.1 (DS-Ulysses walk-through): after the input all-to-all, device p
holds the full sequence for the contiguous block of heads
[p H/C, (p+1) H/C) -- and, with grouped-query attention, the key/value heads
[p Hkv/C, (p+1) Hkv/C) that those query heads read.

Section 4.1 ("Grouped-Query Attention Scheduling"): heads are processed out
of order so that key/value heads are sent once.  Stage s sends, for every
device, the next query heads of that device's groups; a key/value head is
communicated only at the first stage that needs it and reused afterwards.
In the paper's example (C = 4, G = 4, H = 16, U = C) stage 0 carries
Q0, Q4, Q8, Q12 together with K0..K3 and stage 1 carries Q1, Q5, Q9, Q13
with no key/value heads.  The communication count goes from 3 (H/C)(C-1)
head slices for the naive order to (3 + G - 1) H/(C G) (C-1).

On one device the schedule reduces to taking its local heads in ascending
order, U/C at a time: local chunk c holds local heads [c U_l, (c+1) U_l).
"""


def _validate(H, Hkv, C, U):
    if min(H, Hkv, C, U) < 1:
        raise ValueError("all counts must be positive")
    if H % Hkv:
        raise ValueError("H must be a multiple of Hkv")
    if U % C:
        raise ValueError("U must be a multiple of C")
    if H % U:
        raise ValueError("U must divide H")
    if H % C or Hkv % C:
        raise ValueError("C must divide H and Hkv")


def gqa_schedule(H, Hkv, C, U):
    """Global stage plan of the GQA-aware schedule.

    Returns (stages, kv_stage): ``stages[s]`` lists the global query heads of
    stage s, device by device (device p's U/C heads, then device p+1's ...),
    and ``kv_stage[g]`` is the stage at which key/value head g is sent.
    """
    _validate(H, Hkv, C, U)
    G = H // Hkv
    per_dev_q = H // C
    per_stage = U // C
    stages = []
    kv_stage = [None] * Hkv
    for s in range(H // U):
        heads = []
        for p in range(C):
            for j in range(per_stage):
                h = p * per_dev_q + s * per_stage + j
                heads.append(h)
                if kv_stage[h // G] is None:
                    kv_stage[h // G] = s
        stages.append(heads)
    return stages, kv_stage


def naive_schedule(H, Hkv, C, U):
    """Stage s processes the global heads [sU, (s+1)U) in order."""
    _validate(H, Hkv, C, U)
    return [list(range(s * U, (s + 1) * U)) for s in range(H // U)]


def comm_heads_naive(H, Hkv, C, U):
    """Head slices each device sends over all stages, naive order.

    Per stage a device sends (C-1)/C of its U sequence-shard heads for each
    of Q, K and V (with K and V repeated per query head, as in the paper's
    naive example K0, K0, K0, K0).
    """
    _validate(H, Hkv, C, U)
    return sum(3 * (U // C) * (C - 1) for _ in naive_schedule(H, Hkv, C, U))


def comm_heads_scheduled(H, Hkv, C, U):
    """Head slices each device sends over all stages, GQA schedule."""
    stages, kv_stage = gqa_schedule(H, Hkv, C, U)
    total = 0
    for s, heads in enumerate(stages):
        q_slices = (len(heads) // C) * (C - 1)
        kv_new = sum(1 for st in kv_stage if st == s)
        # every key/value head sent this stage is spread over C devices:
        # each device sends (C-1)/C of it, so C of them cost C-1 slices.
        kv_slices = 2 * kv_new * (C - 1) // C
        total += q_slices + kv_slices
    return total


def local_chunks(Hq, Hkv, U):
    """One device's chunk plan: local heads per chunk and new kv heads.

    Returns a list of (heads, kv_heads, kv_new) per chunk, where kv_new are
    the key/value heads first needed by that chunk.
    """
    if Hq % Hkv or Hq % U or U < 1:
        raise ValueError("need Hkv | Hq and U | Hq")
    G = Hq // Hkv
    seen = set()
    plan = []
    for c in range(Hq // U):
        heads = list(range(c * U, (c + 1) * U))
        kvs = sorted({h // G for h in heads})
        new = [g for g in kvs if g not in seen]
        seen.update(kvs)
        plan.append((heads, kvs, new))
    return plan
