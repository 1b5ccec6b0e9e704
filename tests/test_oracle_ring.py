"""Pins of the ring-step oracle (oracle/ring.py): brute force on tiny shapes,
a closed form, the decomposition of full causal attention into merged ring
steps, and the merge's neutral element and symmetry.  A few planted mistakes
in a copy of the oracle must each be caught by some pin."""

import math
import os
import types

import numpy as np
import pytest

from oracle import attention as A
from oracle import ring as R


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def brute_ring(q, k, v, delta, causal):
    """Per-element loops: softmax over the visible keys of each row."""
    Sq, Hq, d = q.shape
    Skv, Hkv = k.shape[:2]
    G = Hq // Hkv
    o = np.zeros((Sq, Hq, d))
    lse = np.full((Hq, Sq), -math.inf)
    for h in range(Hq):
        g = h // G
        for i in range(Sq):
            vis = [j for j in range(Skv) if (not causal) or j <= i + delta]
            if not vis:
                continue
            s = [sum(q[i, h, e] * k[j, g, e] for e in range(d)) / math.sqrt(d) for j in vis]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            tot = sum(w)
            for e in range(d):
                o[i, h, e] = sum(w[n] * v[vis[n], g, e] for n in range(len(vis))) / tot
            lse[h, i] = m + math.log(tot)
    return o, lse


def pin_brute_force(mod):
    q, k, v = _rand((5, 2, 4), 1), _rand((7, 1, 4), 2), _rand((7, 1, 4), 3)
    for delta in (-6, -2, 0, 1, 3, 9):
        for causal in (True, False):
            o, lse = mod.attn_fwd_offset(q, k, v, delta, causal)
            ob, lb = brute_ring(q, k, v, delta, causal)
            np.testing.assert_allclose(o, ob, rtol=1e-12, atol=1e-12)
            np.testing.assert_array_equal(np.isneginf(lse), np.isneginf(lb))
            fin = np.isfinite(lb)
            np.testing.assert_allclose(lse[fin], lb[fin], rtol=1e-12, atol=1e-12)


def pin_zero_queries(mod):
    """q = 0: uniform weights, o_i = mean of the visible v, lse_i = log(count)."""
    Sq, Skv, delta = 6, 9, 2
    q = np.zeros((Sq, 2, 8))
    k, v = _rand((Skv, 1, 8), 4), _rand((Skv, 1, 8), 5)
    o, lse = mod.attn_fwd_offset(q, k, v, delta, True)
    for i in range(Sq):
        n = min(Skv, i + delta + 1)
        np.testing.assert_allclose(o[i, 0], v[:n, 0].mean(axis=0), rtol=1e-12, atol=1e-12)
        assert abs(lse[0, i] - math.log(n)) < 1e-12


def pin_ring_decomposition(mod):
    """Full causal attention = merge of the ring steps over key blocks."""
    S, Hq, Hkv, d = 24, 4, 2, 8
    q, k, v = _rand((S, Hq, d), 6), _rand((S, Hkv, d), 7), _rand((S, Hkv, d), 8)
    o_ref, lse_ref = A.attn_fwd(q, k, v, causal=True)
    for cuts in ((0, 8, 24), (0, 5, 13, 24), (0, 24)):
        qs = slice(4, 20)                      # a query block at global rows 4..19
        o_acc = np.zeros((16, Hq, d))
        lse_acc = np.full((Hq, 16), -np.inf)
        for a, b in zip(cuts[:-1], cuts[1:]):
            o_p, lse_p = mod.attn_fwd_offset(q[qs], k[a:b], v[a:b], 4 - a, True)
            o_acc, lse_acc = mod.lse_merge(o_acc, lse_acc, o_p, lse_p)
        np.testing.assert_allclose(o_acc, o_ref[qs], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse_acc, lse_ref[:, qs], rtol=1e-12, atol=1e-12)


def pin_merge_identity_and_symmetry(mod):
    o_a, lse_a = _rand((5, 3, 4), 9), _rand((3, 5), 10)
    o_b, lse_b = _rand((5, 3, 4), 11), _rand((3, 5), 12)
    empty = np.full((3, 5), -np.inf)
    o, lse = mod.lse_merge(o_a, lse_a, np.zeros_like(o_a), empty)
    np.testing.assert_allclose(o, o_a, rtol=1e-15, atol=0)
    np.testing.assert_allclose(lse, lse_a, rtol=1e-15, atol=0)
    o1, l1 = mod.lse_merge(o_a, lse_a, o_b, lse_b)
    o2, l2 = mod.lse_merge(o_b, lse_b, o_a, lse_a)
    np.testing.assert_allclose(o1, o2, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(np.exp(l1), np.exp(lse_a) + np.exp(lse_b), rtol=1e-13)
    o, lse = mod.lse_merge(np.zeros_like(o_a), empty, np.zeros_like(o_a), empty)
    assert np.all(np.isneginf(lse)) and np.all(o == 0)


PINS = [pin_brute_force, pin_zero_queries, pin_ring_decomposition,
        pin_merge_identity_and_symmetry]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_ring_oracle_pins(pin):
    pin(R)


SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "ring.py")
MUTANTS = {
    "mask_strict": ("visible = (j <= i + delta)", "visible = (j < i + delta)"),
    "mask_sign": ("visible = (j <= i + delta)", "visible = (j <= i - delta)"),
    "lse_drops_max": ("lse[h, rows] = m[rows] + np.log(l[rows])", "lse[h, rows] = np.log(l[rows])"),
    "merge_weight_swap": ("cb = np.where(empty, 0.0, wb / np.where(empty, 1.0, tot))",
                          "cb = np.where(empty, 0.0, wa / np.where(empty, 1.0, tot))"),
    "merge_lse_max_only": ("lse = np.where(empty, -np.inf, ms + np.log(np.where(empty, 1.0, tot)))",
                           "lse = np.where(empty, -np.inf, ms)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_ring_pins_reject_mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mod = types.ModuleType(f"ring_mutant_{name}")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mod)
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"no pin rejects mutant {name}"
