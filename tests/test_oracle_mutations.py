"""Plant plausible mistakes in a copy of the attention oracle; pins must fail.

Each mutant is the oracle's source with one textual change (a dropped term,
a wrong sign, a wrong index or operand), executed as a throw-away module on
the CPU.  The test passes only if at least one pin rejects every mutant,
which shows that the pins constrain each part of the oracle.
"""

import os
import types

import pytest

import oracle_pins as P

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "attention.py")

MUTANTS = {
    "scale_1_over_d": ("(q_rows @ k_h[:n].T) / np.sqrt(d)",
                       "(q_rows @ k_h[:n].T) / d"),
    "diagonal_masked": ("np.arange(n)[None, :] > rows[:, None]",
                        "np.arange(n)[None, :] >= rows[:, None]"),
    "no_causal_mask": ("np.arange(n)[None, :] > rows[:, None]",
                       "np.arange(n)[None, :] > n"),
    "gqa_modulo_map": ("return h // (Hq // Hkv)", "return h % Hkv"),
    "lse_drops_max": ("lse[h, b0:b0 + len(r)] = (m + np.log(l))[:, 0]",
                      "lse[h, b0:b0 + len(r)] = (np.log(l))[:, 0]"),
    "unnormalised_o": ("o[b0:b0 + len(r), h, :] = (e / l) @ v[:n, g, :]",
                       "o[b0:b0 + len(r), h, :] = e @ v[:n, g, :]"),
    "ds_sign": ("ds = p * (dp - D[r][:, None])",
                "ds = p * (dp + D[r][:, None])"),
    "dk_no_scale": ("dk[:n, g, :] += (ds.T @ q[r, h, :]) * scale",
                    "dk[:n, g, :] += (ds.T @ q[r, h, :])"),
    "dv_wrong_operand": ("dv[:n, g, :] += p.T @ do[r, h, :]",
                         "dv[:n, g, :] += ds.T @ do[r, h, :]"),
    "dp_uses_k": ("dp = do[r, h, :] @ v[:n, g, :].T\n            ds = p * (dp - D[r]",
                  "dp = do[r, h, :] @ k[:n, g, :].T\n            ds = p * (dp - D[r]"),
    "dq_uses_v": ("dq[r, h, :] = (ds @ k[:n, g, :]) * scale",
                  "dq[r, h, :] = (ds @ v[:n, g, :]) * scale"),
    "D_from_q": ("D = np.sum(do[:, h, :] * o[:, h, :], axis=1)",
                 "D = np.sum(do[:, h, :] * q[:, h, :], axis=1)"),
    # the conditioned key columns (attn_key_cols_given)
    "cols_drop_lse": ("np.exp(np.where(vis, s, 0.0) - lse[h, b0:b1][:, None])",
                      "np.exp(np.where(vis, s, 0.0))"),
    "cols_diagonal_masked": ("vis = cols[None, :] <= r[:, None] if causal",
                             "vis = cols[None, :] < r[:, None] if causal"),
    "cols_dv_wrong_operand": ("dv[:, g, :] += p.T @ dob[:, h, :]",
                              "dv[:, g, :] += ds.T @ dob[:, h, :]"),
    "cols_dk_no_scale": ("dk[:, g, :] += (ds.T @ qb[:, h, :]) / np.sqrt(d)",
                         "dk[:, g, :] += (ds.T @ qb[:, h, :])"),
    "cols_D_from_q": ("D = np.sum(dob[:, h, :] * ob[:, h, :], axis=1)",
                      "D = np.sum(dob[:, h, :] * qb[:, h, :], axis=1)"),
}


def _mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"),
         mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name):
    mod = _mutant(name)
    caught = []
    for pin in P.ALL_PINS:
        try:
            with __import__("numpy").errstate(all="ignore"):
                pin(mod)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin rejects mutant {name}"
