"""Seeded synthetic workloads: shapes, seeds and input generators.

This module holds no attention arithmetic.  Both the HIP path's tests/bench
and the CPU oracle consume the tensors it produces, so that the two sides see
identical bf16 bytes.

Recipe: a CPU ``torch.Generator`` seeded with the workload's seed draws
float32 standard normals tensor by tensor in the listed order; each tensor is
drawn in row blocks of ``ROWS_PER_DRAW`` rows (so very long sequences never
need one huge float32 buffer), multiplied by its standard deviation and
rounded to bfloat16 (round to nearest even).  These stand in for the
activations of Llama3-8B and Qwen3-32B training on C4 in the paper
(Section 5.1); no dataset or trained weight is used.
"""

from dataclasses import dataclass, field

import torch

ROWS_PER_DRAW = 65536


@dataclass(frozen=True)
class Workload:
    name: str
    S: int
    Hq: int
    Hkv: int
    d: int
    seed: int
    U_sweep: tuple
    d_model: int = 0          # 0 = attention only, no projections
    note: str = ""
    extra: dict = field(default_factory=dict, compare=False)

    @property
    def is_layer(self):
        return self.d_model > 0


WORKLOADS = {
    "tiny": Workload("tiny", 512, 2, 1, 128, 0, (1, 2),
                     note="tiny oracle case, attention fwd+bwd"),
    "llama8b_share": Workload(
        "llama8b_share", 131072, 4, 1, 128, 1, (1, 2, 4),
        note="Llama3-8B per-GPU share at 8-way Ulysses: 32/8 query heads, "
             "8/8 kv heads, S=128K"),
    "llama8b_layer": Workload(
        "llama8b_layer", 262144, 4, 1, 128, 2, (1, 2, 4), d_model=4096,
        note="Llama3-8B per-GPU layer share: QKV slice with fused RoPE "
             "(base 500000, Llama 3's), attention, O-proj",
        extra={"rope_base": 500000.0}),
    "qwen32b_share": Workload(
        "qwen32b_share", 524288, 8, 1, 128, 3, (1, 2, 4, 8),
        note="Qwen3-32B-shaped per-GPU share: 64/8 query heads, 8/8 kv "
             "heads, S=512K"),
    "llama8b_4m": Workload(
        "llama8b_4m", 4194304, 4, 1, 128, 4, (1,),
        note="Llama3-8B share at 4M tokens"),
    "llama8b_ring": Workload(
        "llama8b_ring", 32768, 4, 1, 128, 5, (1, 2, 4),
        note="one ring step of the Llama3-8B share with the sequence split 4 "
             "ways across ring ranks (Ulysses + Ring hybrid): a 32K query "
             "block against the preceding 32K key/value block (all keys "
             "visible), merged into the running result",
        extra={"ring": True, "kv_len": 32768, "q_offset": 32768, "kv_offset": 0}),
}


def _draw(gen, shape, std=1.0):
    """float32 N(0, std^2) in row blocks, rounded to bf16 (RNE)."""
    out = torch.empty(shape, dtype=torch.bfloat16)
    rows = shape[0]
    flat = out.view(rows, -1)
    for r0 in range(0, rows, ROWS_PER_DRAW):
        r1 = min(rows, r0 + ROWS_PER_DRAW)
        blk = torch.randn((r1 - r0, flat.shape[1]), generator=gen,
                          dtype=torch.float32)
        if std != 1.0:
            blk.mul_(std)
        flat[r0:r1] = blk.to(torch.bfloat16)
    return out


def attention_inputs(S, Hq, Hkv, d, seed):
    """q [S,Hq,d], k [S,Hkv,d], v [S,Hkv,d], do [S,Hq,d] as bf16 CPU tensors."""
    gen = torch.Generator(device="cpu").manual_seed(seed)
    q = _draw(gen, (S, Hq, d))
    k = _draw(gen, (S, Hkv, d))
    v = _draw(gen, (S, Hkv, d))
    do = _draw(gen, (S, Hq, d))
    return q, k, v, do


def layer_inputs(S, d_model, Hq, Hkv, d, seed, w_std=0.02):
    """x [S,dm], wqkv [dm,(Hq+2Hkv)d], wo [Hq d, dm], dy [S,dm], bf16 CPU."""
    gen = torch.Generator(device="cpu").manual_seed(seed)
    x = _draw(gen, (S, d_model))
    wqkv = _draw(gen, (d_model, (Hq + 2 * Hkv) * d), w_std)
    wo = _draw(gen, (Hq * d, d_model), w_std)
    dy = _draw(gen, (S, d_model))
    return x, wqkv, wo, dy


def batch_attention_inputs(S, Hq, Hkv, d, seed, B):
    """q, k, v, do [B, S, H, d]: sequence b drawn as attention_inputs with seed
    + b (B = 1 gives attention_inputs itself, with a leading batch of 1)."""
    seqs = [attention_inputs(S, Hq, Hkv, d, seed + b) for b in range(B)]
    return tuple(torch.stack([t[i] for t in seqs]) for i in range(4))


def batch_layer_inputs(S, d_model, Hq, Hkv, d, seed, B, w_std=0.02):
    """x [B, S, dm], wqkv, wo (shared), dy [B, S, dm]: sequence b's x and dy are
    those of layer_inputs with seed + b."""
    xs, dys = [], []
    wqkv = wo = None
    for b in range(B):
        x, wq, wo_b, dy = layer_inputs(S, d_model, Hq, Hkv, d, seed + b, w_std)
        if b == 0:
            wqkv, wo = wq, wo_b
        xs.append(x)
        dys.append(dy)
    return torch.stack(xs), wqkv, wo, torch.stack(dys)


def ring_inputs(w: Workload):
    """q [S,Hq,d] (the query block), k, v [kv_len,Hkv,d] (the key block)."""
    gen = torch.Generator(device="cpu").manual_seed(w.seed)
    q = _draw(gen, (w.S, w.Hq, w.d))
    k = _draw(gen, (w.extra["kv_len"], w.Hkv, w.d))
    v = _draw(gen, (w.extra["kv_len"], w.Hkv, w.d))
    return q, k, v


def ring_pairs(Sq, Skv, delta, causal=True):
    """Visible (query, key) pairs of one head in a ring step: query i sees
    key j < Skv iff j <= i + delta (all keys when not causal)."""
    if not causal:
        return Sq * Skv
    total = 0
    lo = max(0, -delta)                      # first row seeing any key
    full = max(lo, min(Sq, Skv - 1 - delta))  # rows < full see i + delta + 1 keys
    n = full - lo
    if n > 0:
        total += n * (lo + delta + 1) + n * (n - 1) // 2
    total += max(0, Sq - max(full, lo)) * Skv if Skv - 1 - delta < Sq else 0
    return total


def inputs_for(w: Workload):
    if w.is_layer:
        return layer_inputs(w.S, w.d_model, w.Hq, w.Hkv, w.d, w.seed)
    if w.extra.get("ring"):
        return ring_inputs(w)
    return attention_inputs(w.S, w.Hq, w.Hkv, w.d, w.seed)


def sample_rows(S, n_random, seed):
    """Query rows for sampled checks: fixed edge rows plus seeded random rows."""
    fixed = {0, 1, 127, 128, S // 2, S - 1}
    fixed = {r for r in fixed if 0 <= r < S}
    gen = torch.Generator(device="cpu").manual_seed(seed + 1000)
    rnd = torch.randint(0, S, (n_random,), generator=gen).tolist()
    return sorted(fixed | set(rnd))


def sample_key_cols(S, n, seed):
    """Key columns for sampled key-gradient checks: the keys with the longest
    accumulation chains and the tile edges (0, 1, 127, 128), the middle and
    the last key, filled up to n with seeded random keys."""
    fixed = {0, 1, 127, 128, S // 2, S - 1}
    cols = {c for c in fixed if 0 <= c < S}
    gen = torch.Generator(device="cpu").manual_seed(seed + 2000)
    while len(cols) < min(n, S):
        cols.add(int(torch.randint(0, S, (1,), generator=gen)))
    return sorted(cols)


def causal_pairs(S):
    """Number of visible (query, key) pairs of one causal head."""
    return S * (S + 1) // 2


def attention_flops(S, Hq, d, causal=True):
    """Algorithmic fwd+bwd flops: 4d per visible pair forward, 2.5x backward."""
    pairs = causal_pairs(S) if causal else S * S
    fwd = 4 * d * Hq * pairs
    return fwd, int(2.5 * fwd)
