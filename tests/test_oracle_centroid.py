"""Pins of the oracle's centroid-ID predictor (O7 heads, O8 choice and
intersection) and of the delta with per-layer active counts, each against
something other than the oracle itself: numpy dense products, numpy's argmax
(first maximum) and bit operations, exact dyadic arithmetic, and the
ordered-dict LRU simulator of the delta pins."""
import numpy as np
import pytest

import oracle as orc
from test_oracle_delta import LRUSim


def bits_of(mask_words: np.ndarray, F: int) -> np.ndarray:
    """[.., W] uint32 LSB-first words -> [.., F] bool."""
    b = np.unpackbits(mask_words.view(np.uint8).reshape(*mask_words.shape[:-1], -1),
                      axis=-1, bitorder="little")
    return b[..., :F].astype(bool)


def words_of(bits: np.ndarray) -> np.ndarray:
    """[.., F] bool -> [.., ceil(F/32)] uint32 LSB-first."""
    F = bits.shape[-1]
    W = (F + 31) // 32
    pad = np.zeros((*bits.shape[:-1], 32 * W), dtype=np.uint8)
    pad[..., :F] = bits
    return np.packbits(pad, axis=-1, bitorder="little").view(np.uint32)


# ---------------- O7: heads -------------------------------------------------

@pytest.mark.parametrize("wdtype", ["f32", "f16", "bf16"])
def test_logits_are_the_dense_product(wdtype):
    rng = np.random.default_rng(3)
    H, K, D = 6, 40, 72
    W = rng.normal(0, D ** -0.5, size=(H, K, D))
    f = rng.normal(size=D)
    Wb, fb = orc.encode(wdtype, W), orc.encode(wdtype, f)
    got = orc.centroid_logits(Wb, fb, H, K, D, wdtype, wdtype).astype(np.float64)
    Wd, fd = orc.decode(wdtype, Wb), orc.decode(wdtype, fb)
    ref = Wd.reshape(H * K, D) @ fd
    # exact sum rounded once to binary32: half an ulp of fp32 plus the numpy
    # product's own rounding (D terms in double)
    bound = np.abs(ref) * 2.0 ** -24 + D * 2.0 ** -52 * (np.abs(Wd.reshape(H * K, D)) @ np.abs(fd))
    assert np.all(np.abs(got.reshape(-1) - ref) <= bound)


def test_logits_exact_on_dyadic_inputs():
    rng = np.random.default_rng(4)
    H, K, D = 4, 17, 64
    W = rng.integers(-3, 4, size=(H, K, D)) * 2.0 ** -3
    f = rng.integers(-4, 5, size=D).astype(np.float64)
    got = orc.centroid_logits(orc.encode("f16", W), orc.encode("f16", f), H, K, D, "f16", "f16")
    assert np.array_equal(got.astype(np.float64), (W.reshape(H * K, D) @ f).reshape(H, K))


# ---------------- O8: choice and intersection -------------------------------

def random_bank(rng, L, K, F, density):
    bits = rng.random((2, L, K, F)) < density
    return bits, words_of(bits)


@pytest.mark.parametrize("F", [31, 32, 100, 257])
def test_argmax_and_intersection_match_numpy(F):
    rng = np.random.default_rng(F)
    L, K, k = 3, 24, F
    bits, bank = random_bank(rng, L, K, F, 0.5)
    for case in range(4):
        if case % 2:  # heavy ties: few distinct values
            logits = rng.integers(0, 3, size=(2 * L, K)).astype(np.float32)
        else:
            logits = rng.normal(size=(2 * L, K)).astype(np.float32)
        out = orc.centroid_active(logits, bank, L, F, K, k)
        cids = np.argmax(logits, axis=1).reshape(2, L)  # numpy: the first maximum
        assert np.array_equal(out["cids"], cids)
        for l in range(L):
            inter = bits[0, l, cids[0, l]] & bits[1, l, cids[1, l]]
            ids = np.flatnonzero(inter)
            assert out["counts"][l] == ids.size
            assert np.array_equal(out["active_ids"][l][:ids.size], ids)
            assert np.all(out["active_ids"][l][ids.size:] == -1)
            assert np.array_equal(bits_of(out["mask"][l], F), inter)
        assert not out["overflow"]


def test_one_hot_heads_pick_the_named_centroid():
    # head h has a single positive row c_h: its logits are one-hot
    L, K, D, F = 2, 8, 16, 64
    target = np.array([3, 0, 7, 5])
    W = np.zeros((2 * L, K, D))
    for h, c in enumerate(target):
        W[h, c, :] = 1.0
    f = np.ones(D)
    logits = orc.centroid_logits(orc.encode("f32", W), orc.encode("f32", f), 2 * L, K, D, "f32",
                                 "f32")
    bank = np.zeros((2, L, K, 2), dtype=np.uint32)
    bank[0, 0, 3] = [0xF0F0F0F0, 0x1]
    bank[1, 0, 7] = [0xFF00FF00, 0x3]
    bank[0, 1, 0] = [0xFFFFFFFF, 0xFFFFFFFF]
    bank[1, 1, 5] = [0x0, 0x80000000]
    out = orc.centroid_active(logits, bank, L, F, K, F)
    assert out["cids"].tolist() == [[3, 0], [7, 5]]
    assert out["mask"][0].tolist() == [0xF000F000, 0x1] and out["counts"][0] == 9
    assert out["active_ids"][1][:1].tolist() == [63] and out["counts"][1] == 1


def test_intersection_larger_than_capacity_keeps_smallest_ids():
    L, K, F, k = 1, 2, 40, 5
    bank = np.zeros((2, L, K, 2), dtype=np.uint32)
    bank[0, 0, 1] = [0xFFFFFFFF, 0xFF]
    bank[1, 0, 0] = [0x0F0F0F0F, 0x0F]
    logits = np.array([[0.0, 1.0], [2.0, 1.0]], dtype=np.float32)
    out = orc.centroid_active(logits, bank, L, F, K, k)
    assert out["overflow"]
    assert out["counts"].tolist() == [5]
    assert out["active_ids"][0].tolist() == [0, 1, 2, 3, 8]
    assert bits_of(out["mask"][0], F).sum() == 20  # the mask keeps every member


def test_nan_logit_is_an_error():
    logits = np.zeros((2, 4), dtype=np.float32)
    logits[1, 2] = np.nan
    with pytest.raises(orc.OracleError):
        orc.centroid_active(logits, np.zeros((2, 1, 4, 1), np.uint32), 1, 10, 4, 3)


# ---------------- O3 with per-layer counts ----------------------------------

def test_delta_n_with_full_counts_equals_delta():
    rng = np.random.default_rng(5)
    L, F, k, C = 2, 60, 10, 25
    s1, s2 = orc.State(L, F, C), orc.State(L, F, C)
    for t in range(6):
        A = np.sort(np.stack([rng.choice(F, k, replace=False) for _ in range(L)]), axis=1)
        a = orc.delta(t, A, s1, C)
        b = orc.delta_n(t, A, np.full(L, k), s2, C)
        for n in a:
            assert np.array_equal(a[n], b[n]), n
    assert np.array_equal(s1.slot_of, s2.slot_of) and np.array_equal(s1.last_used, s2.last_used)


@pytest.mark.parametrize("F,k,C", [(50, 12, 20), (90, 30, 40)])
def test_delta_n_variable_sets_follow_lru(F, k, C):
    rng = np.random.default_rng(F + k)
    st = orc.State(1, F, C)
    sim = LRUSim(C)
    for t in range(15):
        n = int(rng.integers(0, k + 1))
        A = np.sort(rng.choice(F, n, replace=False)).astype(np.int32)
        row = np.full((1, k), -1, np.int32)
        row[0, :n] = A
        out = orc.delta_n(t, row, np.array([n]), st, C)
        inc, vic = sim.access(list(A))
        c = out["counts"][0]
        assert c[0] == len(inc) and c[2] == len(vic) and c[1] == n - len(inc)
        assert out["in_ids"][0][:c[0]].tolist() == inc
        assert out["ev_ids"][0][:c[2]].tolist() == vic
        # every active neuron resident, at the slot the list reports
        assert np.array_equal(st.slot_of[0][A], out["active_slots"][0][:n])
        assert np.all(st.slot_of[0][A] >= 0)
        assert np.array_equal(st.last_used[0][A], np.full(n, t))
        assert np.all(out["active_slots"][0][n:] == -1)


def test_delta_n_rejects_counts_outside_the_list():
    st = orc.State(1, 20, 8)
    with pytest.raises(orc.OracleError):
        orc.delta_n(0, np.arange(4, dtype=np.int32).reshape(1, 4), np.array([5]), st, 8)
