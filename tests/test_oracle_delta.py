"""Pins of oracle O3 (delta against the resident set and slot-map update).

References: hand-worked examples of eqs. (2)-(3) and the slot-map rules
(tests/golden/delta_examples.json), the set equations themselves when the
buffer holds exactly the active set (C = k), an ordered-dict LRU cache
simulator when C > k, and the invariants any valid slot map satisfies.
"""
import json
import os
from collections import OrderedDict

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "delta_examples.json")


def lists(out, l):
    c = out["counts"][l]
    return {
        "in_ids": out["in_ids"][l][: c[0]].tolist(),
        "in_slots": out["in_slots"][l][: c[0]].tolist(),
        "hit_ids": out["hit_ids"][l][: c[1]].tolist(),
        "ev_ids": out["ev_ids"][l][: c[2]].tolist(),
        "ev_slots": out["ev_slots"][l][: c[2]].tolist(),
        "active_slots": out["active_slots"][l].tolist(),
    }


def test_golden_examples(orc):
    with open(GOLDEN) as f:
        data = json.load(f)
    for ex in data["examples"]:
        F, C, k = ex["F"], ex["C"], ex["k"]
        state = orc.State(1, F, C)
        for t, tok in enumerate(ex["tokens"]):
            out = orc.delta(t, np.array([tok["active"]], np.int32), state, C)
            got = lists(out, 0)
            for key in ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids", "active_slots"):
                assert got[key] == tok[key], (ex["name"], t, key, got[key], tok[key])
        assert state.slot_of[0].tolist() == ex["final_slot_of"], ex["name"]


def random_active_sequence(rng, F, k, T, stay=0.8):
    """Active sets with some token-to-token persistence."""
    cur = set(rng.choice(F, k, replace=False).tolist())
    seq = [sorted(cur)]
    for _ in range(T - 1):
        keep = [n for n in cur if rng.random() < stay]
        pool = [n for n in range(F) if n not in keep]
        extra = rng.choice(pool, k - len(keep), replace=False).tolist()
        cur = set(keep) | set(extra)
        seq.append(sorted(cur))
    return seq


def check_invariants(state, out, A, l, C, t, prev_resident):
    P, Q, U = state.slot_of[l], state.neuron_of[l], state.last_used[l]
    g = lists(out, l)
    I, H, V = set(g["in_ids"]), set(g["hit_ids"]), set(g["ev_ids"])
    Aset = set(A)
    assert I | H == Aset and not (I & H)                      # delta + hits = active set
    assert H == Aset & prev_resident and I == Aset - prev_resident
    assert not (V & Aset) and V <= prev_resident               # only non-active rows leave
    nfree = C - len(prev_resident)
    assert len(V) == max(0, len(I) - nfree)                    # evict only when full
    resident = {n for n in range(len(P)) if P[n] >= 0}
    assert resident == (prev_resident - V) | I
    assert len(resident) <= C and Aset <= resident
    for n in resident:                                         # P and Q are inverses
        assert Q[P[n]] == n
    assert sum(1 for s in range(C) if Q[s] >= 0) == len(resident)
    assert g["in_ids"] == sorted(g["in_ids"]) and g["in_slots"] == sorted(g["in_slots"])
    assert g["active_slots"] == [int(P[n]) for n in A]
    assert all(U[n] == t for n in A)
    return resident


@pytest.mark.parametrize("F,k,C", [(40, 8, 8), (60, 10, 25), (200, 30, 45), (50, 50, 50)])
def test_invariants_random(orc, F, k, C):
    rng = np.random.default_rng(F + k + C)
    L = 2
    seqs = [random_active_sequence(rng, F, k, 30) for _ in range(L)]
    state = orc.State(L, F, C)
    resident = [set() for _ in range(L)]
    for t in range(30):
        A = np.array([seqs[l][t] for l in range(L)], np.int32)
        out = orc.delta(t, A, state, C)
        for l in range(L):
            resident[l] = check_invariants(state, out, A[l].tolist(), l, C, t, resident[l])
        if t == 0:  # cold start: every active row incoming, slots 0..k-1
            for l in range(L):
                assert lists(out, l)["in_slots"] == list(range(k))


@pytest.mark.parametrize("F,k", [(30, 6), (100, 17)])
def test_buffer_equal_to_active_set_gives_eqs_2_3(orc, F, k):
    rng = np.random.default_rng(F)
    seq = random_active_sequence(rng, F, k, 25, stay=0.7)
    state = orc.State(1, F, k)
    for t, A in enumerate(seq):
        out = orc.delta(t, np.array([A], np.int32), state, k)
        g = lists(out, 0)
        if t > 0:
            prev = set(seq[t - 1])
            assert set(g["in_ids"]) == set(A) - prev              # D_in
            assert set(g["ev_ids"]) == prev - set(A)              # D_out
            assert sorted(g["in_slots"]) == sorted(g["ev_slots"])  # freed slots reused


class LRUSim:
    """Textbook LRU cache of `cap` rows with batched per-token access: rows of
    one token count as used at the same time and are recorded in ascending id
    order, so the eviction order is (last token, id)."""

    def __init__(self, cap):
        self.cap = cap
        self.od = OrderedDict()

    def access(self, A):
        Aset = set(A)
        incoming = [n for n in A if n not in self.od]
        room = self.cap - len(self.od)
        victims = []
        if len(incoming) > room:
            need = len(incoming) - room
            for n in list(self.od.keys()):
                if need == 0:
                    break
                if n not in Aset:
                    victims.append(n)
                    need -= 1
            for n in victims:
                del self.od[n]
        for n in sorted(A):
            self.od.pop(n, None)
            self.od[n] = True
        return sorted(incoming), sorted(victims)


@pytest.mark.parametrize("F,k,C,stay", [(40, 5, 12, 0.6), (120, 20, 50, 0.8), (64, 16, 17, 0.5)])
def test_matches_lru_simulator(orc, F, k, C, stay):
    rng = np.random.default_rng(C)
    seq = random_active_sequence(rng, F, k, 60, stay=stay)
    sim = LRUSim(C)
    state = orc.State(1, F, C)
    for t, A in enumerate(seq):
        out = orc.delta(t, np.array([A], np.int32), state, C)
        g = lists(out, 0)
        inc, vic = sim.access(A)
        assert g["in_ids"] == inc and g["ev_ids"] == vic, t
        assert {n for n in range(F) if state.slot_of[0][n] >= 0} == set(sim.od.keys())


def test_precondition_errors(orc):
    state = orc.State(1, 10, 3)
    with pytest.raises(orc.OracleError):
        orc.delta(0, np.array([[3, 3]], np.int32), state, 3)      # not strictly ascending
    with pytest.raises(orc.OracleError):
        orc.delta(0, np.array([[1, 2, 3, 4]], np.int32), state, 3)  # k > C
