"""Schedule and memory-accounting oracles against what the paper prints."""

import json
import os
from fractions import Fraction as F

import pytest

from oracle import memory as M
from oracle import schedule as SCH

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------ schedule

def test_gqa_schedule_paper_example():
    g = _golden("gqa_schedule_example.json")
    stages, kv_stage = SCH.gqa_schedule(g["H"], g["Hkv"], g["C"], g["U"])
    for s, heads in enumerate(g["stages_prefix"]):
        assert stages[s] == heads
    for s, kvs in g["kv_sent_at_stage"].items():
        assert sorted(i for i, st in enumerate(kv_stage) if st == int(s)) == kvs


def test_stage_counts_of_the_paper_models():
    for case in _golden("stage_counts.json")["cases"]:
        stages, _ = SCH.gqa_schedule(case["H"], case["Hkv"], case["C"],
                                     case["U"])
        assert len(stages) == case["stages"], case["model"]


@pytest.mark.parametrize("H,Hkv,C", [(16, 4, 4), (32, 8, 8), (64, 8, 8),
                                     (64, 16, 4), (48, 8, 4), (8, 2, 2)])
def test_comm_volume_closed_forms(H, Hkv, C):
    g = _golden("gqa_schedule_example.json")
    G = H // Hkv
    U = C
    env = {"H": H, "C": C, "G": G}
    assert SCH.comm_heads_naive(H, Hkv, C, U) == eval(g["comm_naive"], env)
    assert SCH.comm_heads_scheduled(H, Hkv, C, U) == eval(
        g["comm_scheduled"], env)
    assert SCH.comm_heads_scheduled(H, Hkv, C, U) < SCH.comm_heads_naive(
        H, Hkv, C, U)


@pytest.mark.parametrize("H,Hkv,C,U", [(16, 4, 4, 4), (32, 8, 8, 16),
                                       (64, 16, 4, 8), (8, 8, 2, 4)])
def test_schedule_is_a_partition(H, Hkv, C, U):
    stages, kv_stage = SCH.gqa_schedule(H, Hkv, C, U)
    flat = [h for s in stages for h in s]
    assert sorted(flat) == list(range(H))
    assert all(len(s) == U for s in stages)
    G = H // Hkv
    # Each kv head is sent exactly at the first stage that reads it, and each
    # device only ever receives query heads whose kv head it owns.
    for s, heads in enumerate(stages):
        for p in range(C):
            mine = heads[p * U // C:(p + 1) * U // C]
            for h in mine:
                assert kv_stage[h // G] <= s
                assert (h // G) // (Hkv // C) == p


def test_schedule_rejects_bad_shapes():
    with pytest.raises(ValueError):
        SCH.gqa_schedule(16, 4, 4, 6)      # U not a multiple of C
    with pytest.raises(ValueError):
        SCH.gqa_schedule(16, 4, 3, 3)      # C does not divide H
    with pytest.raises(ValueError):
        SCH.local_chunks(4, 1, 3)


def test_local_chunks_cover_heads_once():
    plan = SCH.local_chunks(8, 2, 2)
    assert [h for heads, _, _ in plan for h in heads] == list(range(8))
    assert [new for _, _, new in plan] == [[0], [], [1], []]


# -------------------------------------------------------------------- memory

def test_memory_saving_claim():
    g = _golden("memory_claims.json")
    S, d = 1 << 20, 128
    uly = M.intermediate_bytes_ulysses(S, g["C"], g["H"], d)
    up = M.intermediate_bytes_upipe(S, g["C"], g["U"], d)
    assert uly == g["ulysses_bytes_per_S_dhead"] * S * d
    assert up == g["upipe_bytes_per_S_dhead"] * S * d
    assert (1 - up / uly) * 100 == F(str(g["reduction_percent"]))
    assert M.saving_fraction(g["H"], g["U"]) * 100 == F(
        str(g["reduction_percent"]))


@pytest.mark.parametrize("G", [1, 2, 4, 8])
@pytest.mark.parametrize("nu", [1, 2, 3, 4, 8])
def test_fwd_table_matches_live_sets(G, nu):
    table = M.fwd_table("upipe", G, nu)
    live = M.upipe_fwd_live_sets(G, nu)
    assert M.total(live["before"]) == table[0]
    assert M.total(live["inp_all_to_all"]) == table[1]
    assert M.total(live["attn_kernel"]) == table[2]
    assert M.total(live["out_all_to_all"]) == table[3]


@pytest.mark.parametrize("G", [1, 2, 4, 8])
@pytest.mark.parametrize("nu", [1, 2, 3, 4, 8])
def test_bwd_table_matches_live_sets(G, nu):
    table = M.bwd_table("upipe", G, nu)
    live = M.upipe_bwd_live_sets(G, nu)
    assert M.total(live["before"]) == table[0]
    assert M.total(live["out_all_to_all_stage0"]) == table[1]
    k0 = M.total(live["kernel_stage0"])
    k1 = M.total(live["kernel_stage1"])
    assert (max(k0, k1) if nu > 1 else k0) == table[2]
    assert M.total(live["inp_all_to_all_stage0_end"]) == table[3]


@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_table_special_cases(G):
    # nu = 1: UPipe collapses to Ulysses with offloading (Appendix A).
    up_f = M.fwd_table("upipe", G, 1)
    off_f = M.fwd_table("ulysses_offload", G)
    assert up_f == off_f
    up_b = M.bwd_table("upipe", G, 1)
    off_b = M.bwd_table("ulysses_offload", G)
    assert up_b[2] == off_b[2] and up_b[3] == off_b[3]
    # nu = 2: both arguments of the kernel max are equal; nu >= 3: stage 1.
    g = M.gamma(G)
    assert 3 + 2 * g / 2 == 2 + 2 * g / 2 + F(2 * 1, 2)
    for nu in (3, 4, 8):
        assert 2 + 2 * g / nu + F(2 * (nu - 1), nu) > 3 + 2 * g / nu
    # More stages never use more memory in any column.
    for nu in (1, 2, 4, 8):
        a = M.fwd_table("upipe", G, nu)
        b = M.fwd_table("upipe", G, 2 * nu)
        assert all(x >= y for x, y in zip(a, b))
