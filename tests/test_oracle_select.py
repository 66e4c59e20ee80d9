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


def test_select_and_delta_from_several_threads(orc):
    """O2 and O3 sort through comparators that read their keys from a
    pointer set by the call; calls from several host threads at once (as in
    the tests that run two decode pipelines side by side) must give exactly
    what one thread gives."""
    import threading

    rng = np.random.default_rng(3)
    L, F, k, C = 3, 5000, 700, 1500
    scores = [rng.standard_normal((L, F)).astype(np.float32) for _ in range(6)]
    ref_sel = [orc.select(s, k)[1] for s in scores]

    def delta_run(ids):
        st = orc.State(L, F, C)
        return [orc.delta(t, ids[t], st, C)["in_slots"] for t in range(len(ids))]

    seqs = [[np.sort(rng.choice(F, k, replace=False)).reshape(1, k).repeat(L, 0).astype(np.int32)
             for _ in range(4)] for _ in range(6)]
    ref_delta = [delta_run(s) for s in seqs]
    bad = []

    def work(i):
        for _ in range(10):
            if not np.array_equal(orc.select(scores[i], k)[1], ref_sel[i]):
                bad.append(("select", i))
            got = delta_run(seqs[i])
            if not all(np.array_equal(a, b) for a, b in zip(got, ref_delta[i])):
                bad.append(("delta", i))

    th = [threading.Thread(target=work, args=(i,)) for i in range(6)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not bad, bad[:5]
