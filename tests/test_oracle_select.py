"""Pins of oracle O2 (fixed-size top-k active sets, ties to the lower id).

Reference: a brute-force Python sort by (-score, id) on tiny inputs with
heavily tied scores, plus the order properties any correct top-k has.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st


def brute_topk(s, k):
    order = sorted(range(len(s)), key=lambda n: (-float(s[n]), n))
    return sorted(order[:k])


def mask_of(ids, F):
    words = np.zeros((F + 31) // 32, dtype=np.uint32)
    for n in ids:
        words[n // 32] |= np.uint32(1 << (n % 32))
    return words


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 80).flatmap(
    lambda F: st.tuples(st.just(F), st.integers(1, F),
                        st.lists(st.sampled_from([-1.0, -0.0, 0.0, 0.5, 1.0, 2.0, -3.5]),
                                 min_size=F, max_size=F))))
def test_select_brute_force_ties(orc, case):
    F, k, vals = case
    s = np.array([vals], dtype=np.float32)
    mask, ids = orc.select(s, k)
    assert list(ids[0]) == brute_topk(vals, k)
    assert np.array_equal(mask[0], mask_of(ids[0], F))


@pytest.mark.parametrize("F,k", [(64, 7), (100, 100), (1000, 1), (1000, 333), (33, 32)])
def test_select_random_properties(orc, F, k):
    rng = np.random.default_rng(F * 7 + k)
    s = rng.normal(size=(3, F)).astype(np.float32)
    mask, ids = orc.select(s, k)
    for l in range(3):
        sel = set(ids[l].tolist())
        assert len(sel) == k and list(ids[l]) == sorted(sel)
        inside = s[l][ids[l]]
        outside = np.delete(s[l], ids[l])
        if outside.size:
            assert inside.min() >= outside.max()
        assert list(ids[l]) == brute_topk(s[l], k)
        # pad bits of the last word are zero
        if F % 32:
            assert int(mask[l][-1]) >> (F % 32) == 0


def test_select_k_equals_F_and_signed_zero(orc):
    s = np.array([[0.0, -0.0, 1.0, -0.0, 0.0]], dtype=np.float32)
    _, ids = orc.select(s, 5)
    assert list(ids[0]) == [0, 1, 2, 3, 4]
    _, ids = orc.select(s, 3)
    assert list(ids[0]) == [0, 1, 2]  # -0 == +0, ties to lower id


def test_select_nan_is_error(orc):
    s = np.array([[1.0, np.nan, 0.5]], dtype=np.float32)
    with pytest.raises(orc.OracleError):
        orc.select(s, 1)
