"""The attention oracle against its pins, plus its sampled/chunked variants."""

import numpy as np
import pytest

from oracle import attention as A
import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(A)


def _inputs(S, Hq, Hkv, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((S, Hq, d)), rng.standard_normal((S, Hkv, d)),
            rng.standard_normal((S, Hkv, d)), rng.standard_normal((S, Hq, d)))


def test_rows_variants_match_full():
    q, k, v, do = _inputs(600, 4, 2, 16, 3)
    o, lse = A.attn_fwd(q, k, v)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    rows = np.array([0, 1, 5, 255, 256, 257, 599])
    o_r, lse_r = A.attn_fwd(q, k, v, rows=rows)
    # Same rows, fewer keys per block: only BLAS summation order differs.
    np.testing.assert_allclose(o_r, o[rows], atol=1e-14)
    np.testing.assert_allclose(lse_r, lse[:, rows], atol=1e-14)
    dq_r, D_r = A.attn_bwd_rows(q, k, v, do, rows)
    np.testing.assert_allclose(dq_r, dq[rows], atol=1e-13)
    np.testing.assert_allclose(D_r, np.sum(do * o, axis=2).T[:, rows],
                               atol=1e-13)
    dk_t, dv_t = A.attn_bwd_key_tail(q, k, v, do, 450)
    np.testing.assert_allclose(dk_t, dk[450:], atol=1e-12)
    np.testing.assert_allclose(dv_t, dv[450:], atol=1e-12)


@pytest.mark.parametrize("U", [1, 2, 4])
def test_chunked_equals_unchunked(U):
    q, k, v, do = _inputs(70, 4, 2, 8, 4)
    o, lse = A.attn_fwd(q, k, v)
    oc, lc = A.attn_fwd_chunked(q, k, v, U)
    np.testing.assert_array_equal(oc, o)
    np.testing.assert_array_equal(lc, lse)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    dqc, dkc, dvc = A.attn_bwd_chunked(q, k, v, do, U)
    np.testing.assert_array_equal(dqc, dq)
    np.testing.assert_allclose(dkc, dk, atol=1e-13)
    np.testing.assert_allclose(dvc, dv, atol=1e-13)


def test_shape_errors():
    q, k, v, _ = _inputs(5, 3, 2, 4, 0)
    with pytest.raises(ValueError):
        A.attn_fwd(q, k, v)


def test_row_helpers_with_positions_match_full():
    q, k, v, do = _inputs(520, 4, 2, 16, 9)
    o, lse = A.attn_fwd(q, k, v)
    dq, dk, dv = A.attn_bwd(q, k, v, do)
    rows = np.array([0, 3, 257, 300, 519])
    o_r, lse_r, dq_r, D_r = A.attn_rows_at(q[rows], rows, k, v, do[rows])
    np.testing.assert_allclose(o_r, o[rows], atol=1e-14)
    np.testing.assert_allclose(lse_r, lse[:, rows], atol=1e-14)
    np.testing.assert_allclose(dq_r, dq[rows], atol=1e-13)
    np.testing.assert_allclose(D_r, np.sum(do * o, axis=2).T[:, rows], atol=1e-13)
    o2, lse2 = A.attn_rows_at(q[rows], rows, k, v)
    np.testing.assert_array_equal(o2, o_r)
    dk_t, dv_t = A.attn_key_tail_at(q[400:], do[400:], k, v, 400)
    np.testing.assert_allclose(dk_t, dk[400:], atol=1e-12)
    np.testing.assert_allclose(dv_t, dv[400:], atol=1e-12)


@pytest.mark.parametrize("S,Hq,Hkv,causal", [(300, 4, 1, True), (257, 4, 2, True),
                                             (90, 2, 2, False)])
def test_key_cols_given_statistics_match_torch_autograd(S, Hq, Hkv, causal):
    """With the exact row statistics (the oracle's o and lse), the conditioned
    key columns are the key gradient itself: checked against torch float64
    autograd of scaled_dot_product_attention (a library routine) and, at a
    row block that splits the sequence, against the oracle's full backward."""
    q, k, v, do = _inputs(S, Hq, Hkv, 16, 21 + S)
    o, lse = A.attn_fwd(q, k, v, causal)
    _, _, dk_t, dv_t = P._torch_ref(q, k, v, do, causal)
    cols = np.array([0, 1, 5, S // 2, S - 2, S - 1])
    dk_c, dv_c = A.attn_key_cols_given(q, do, k, v, o, lse, cols, causal, row_block=64)
    np.testing.assert_allclose(dk_c, dk_t[cols], rtol=0, atol=1e-10)
    np.testing.assert_allclose(dv_c, dv_t[cols], rtol=0, atol=1e-10)
    _, dk, dv = A.attn_bwd(q, k, v, do, causal)
    np.testing.assert_allclose(dk_c, dk[cols], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv_c, dv[cols], rtol=0, atol=1e-12)


def test_key_cols_given_statistics_are_conditioned():
    """The result depends on the supplied lse and o exactly as the definition
    says: raising every lse of head h by c scales that head's P by exp(-c)
    (dV_j and the P dP part of dK_j scale with it); shifting o changes only D,
    i.e. adds sum_i P_ij (dO_i.delta) q_i / sqrt(d) to dK_j and leaves dV_j."""
    q, k, v, do = _inputs(200, 2, 1, 8, 33)
    o, lse = A.attn_fwd(q, k, v)
    cols = np.array([0, 7, 100, 199])
    dk0, dv0 = A.attn_key_cols_given(q, do, k, v, o, lse, cols)
    c = 0.7
    dk1, dv1 = A.attn_key_cols_given(q, do, k, v, o, lse + c, cols)
    np.testing.assert_allclose(dv1, dv0 * np.exp(-c), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dk1, dk0 * np.exp(-c), rtol=1e-12, atol=1e-14)
    delta = np.zeros_like(o)
    delta[:, :, 0] = 0.25
    dk2, dv2 = A.attn_key_cols_given(q, do, k, v, o + delta, lse, cols)
    np.testing.assert_array_equal(dv2, dv0)
    s = np.einsum("ihd,jd->hij", q, k[:, 0, :]) / np.sqrt(8)
    p = np.exp(s - lse[:, :, None]) * (np.arange(200)[None, :, None] >= np.arange(200)[None, None, :])
    extra = -np.einsum("hij,ih,ihd->jd", p, 0.25 * do[:, :, 0], q) / np.sqrt(8)
    np.testing.assert_allclose(dk2[:, 0, :], dk0[:, 0, :] + extra[cols], rtol=0, atol=1e-12)
