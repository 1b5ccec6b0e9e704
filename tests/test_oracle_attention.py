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
