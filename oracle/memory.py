"""Oracle: the paper's activation-memory accounting for the attention block.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Two independent statements in the paper are encoded here so that tests can
hold one against the other:

1. The closed forms printed in Tables ``tab:gqa_fwd_mem`` (Section 3.2) and
   ``tab:gqa_bwd_mem`` (Appendix A), in units of one local hidden-state shard
   (S/C * d_model bf16 elements), with gamma = 1 + 2/G the combined size of
   Q, K, V and nu = H/U the number of stages.  Only the two rows the tests
   can hold against something else are kept: UPipe, and Ulysses with
   offloading, which is what UPipe reduces to at nu = 1.
2. The live-tensor inventories of the Appendix A paragraphs ("DeepSpeed-
   Ulysses (forward/backward)", "Untied Ulysses (forward/backward)"): which
   tensors are alive at each moment and how large each is.

Section 3.4 ("Memory Savings") gives the byte counts of the intermediate
tensors: 12 (S/C) H d_head bytes for DS-Ulysses (QKV plus the all-to-all
buffers, bf16) and 12 (S/C) U d_head bytes for UPipe.
"""

from fractions import Fraction as F


def gamma(G):
    """Combined size of Q, K, V relative to one hidden-state shard."""
    return 1 + F(2, G)


# ---- Section 3.4 ---------------------------------------------------------

def intermediate_bytes_ulysses(S, C, H, d_head):
    return 12 * F(S, C) * H * d_head


def intermediate_bytes_upipe(S, C, U, d_head):
    return 12 * F(S, C) * U * d_head


def saving_fraction(H, U):
    """1 - UPipe/Ulysses intermediate bytes; the S, C, d factors cancel."""
    return 1 - F(U, H)


# ---- Table tab:gqa_fwd_mem (closed forms) --------------------------------
# columns: before attn block, during inp_all_to_all, during attn kernel,
#          during out_all_to_all

def fwd_table(method, G, nu=1):
    g = gamma(G)
    if method == "ulysses_offload":
        return (F(1), g + 2, g + 2, F(3))
    if method == "upipe":
        return (F(1), 2 + g / nu, 2 + g / nu, 2 + F(1, nu))
    raise ValueError(method)


# ---- Table tab:gqa_bwd_mem (closed forms) --------------------------------
# columns: before bwd attn, during out_all_to_all, during bwd attn kernel,
#          during inp_all_to_all

def bwd_table(method, G, nu=1):
    g = gamma(G)
    if method == "ulysses_offload":
        return (F(3), F(4), 2 * g + 3, g + 2)
    if method == "upipe":
        kernel = max(3 + 2 * g / nu, 2 + 2 * g / nu + F(2 * (nu - 1), nu))
        return (F(3), 3 + F(1, nu), kernel, 2 + g / nu + F(2 * (nu - 1), nu))
    raise ValueError(method)


# ---- Appendix A live-set inventories -------------------------------------

def upipe_fwd_live_sets(G, nu):
    """Live tensors (name -> size in units) at each forward moment."""
    g = gamma(G)
    return {
        "before": {"X": F(1)},
        # final_out slot i doubles as the destination of Q'^i
        "inp_all_to_all": {"X": F(1), "final_out": F(1), "QKV^i": g / nu},
        "attn_kernel": {"X": F(1), "final_out(holds Q'^i)": F(1),
                        "K'^i,V'^i": F(2, G) / nu, "O'^i": F(1, nu)},
        "out_all_to_all": {"X": F(1), "final_out": F(1),
                           "in-flight chunk": F(1, nu)},
    }


def upipe_bwd_live_sets(G, nu):
    """Live tensors at the backward moments of the global peak."""
    g = gamma(G)
    rest = F(nu - 1, nu)
    return {
        "before": {"X": F(1), "final_out": F(1), "d_final_out": F(1)},
        "out_all_to_all_stage0": {"X": F(1), "final_out": F(1),
                                  "d_final_out": F(1),
                                  "in-flight chunk": F(1, nu)},
        "kernel_stage0": {"X": F(1), "final_out": F(1), "d_final_out": F(1),
                          "dQ',dK',dV'": g / nu, "Q',K',V'": g / nu},
        "kernel_stage1": {"X": F(1), "dX": F(1),
                          "final_out rest": rest, "d_final_out rest": rest,
                          "dQ',dK',dV'": g / nu, "Q',K',V'": g / nu},
        "inp_all_to_all_stage0_end": {"X": F(1), "dX": F(1),
                                      "final_out rest": rest,
                                      "d_final_out rest": rest,
                                      "dQ^0,dK^0,dV^0": g / nu},
    }


def total(live):
    return sum(live.values(), F(0))
