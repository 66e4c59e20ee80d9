"""The parity verdict of bench.py's oracle leg, on the CPU: references built
by the oracle itself (standing in for the GPU's first tokens) pass, and a
wrong active id, a wrong delta entry, a wrong slot map or an MLP output
outside the tolerance each turn the verdict false."""
import copy

import numpy as np
import pytest
import torch

import bench
import oracle as orc
from paper_2608_22643_amd import workload as W


@pytest.fixture(scope="module")
def tiny():
    cfg = W.get("tiny")
    store = W.storage(cfg)
    host = torch.from_numpy(store.view(np.uint8).reshape(-1).copy())
    A, Bm = W.predictor(cfg)
    h = W.hidden(cfg, 64)
    st = orc.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    refs = []
    for t in range(3):  # what the GPU leg keeps: its first tokens from cold start
        s = orc.predict(cfg, h[t], A, Bm).astype(np.float32)
        _, ids = orc.select(s, cfg.k)
        lists = orc.delta(t, ids, st, cfg.capacity)
        y = np.stack([orc.sparse_mlp(cfg, l, h[t], store, ids[l]) for l in range(cfg.layers)])
        refs.append({"scores": s, "ids": ids.copy(), "lists": copy.deepcopy(lists),
                     "state": (st.slot_of.copy(), st.neuron_of.copy(), st.last_used.copy()),
                     "y": y})
    return cfg, host, refs


def verdict(cfg, host, refs):
    return bench.cpu_baseline(cfg, host, 0.0, refs)["parity"]


def test_parity_passes_on_oracle_references(tiny):
    cfg, host, refs = tiny
    v = verdict(cfg, host, refs)
    assert v["tokens"] == 3 and v["ok"], v
    assert v["mlp_max_abs_err"] <= 1e-5 * 4 and v["scores_max_rel_diff"] < 1e-6


@pytest.mark.parametrize("plant", ["id", "delta", "slot_map", "mlp"])
def test_parity_catches_planted_mistakes(tiny, plant):
    cfg, host, refs = tiny
    bad = copy.deepcopy(refs)
    r = bad[1]
    if plant == "id":
        r["ids"][0, 0] = (r["ids"][0, 0] + 1) % cfg.d_ffn
        key = "select_exact"
    elif plant == "delta":
        r["lists"]["active_slots"][1, 2] += 1
        key = "delta_exact"
    elif plant == "slot_map":
        P = r["state"][0].copy()
        P[2, int(r["ids"][2, 0])] = -1
        r["state"] = (P, r["state"][1], r["state"][2])
        key = "slot_maps_exact"
    else:
        y = r["y"].copy()
        y[1, 7] = np.float32(y[1, 7] + 1.0)
        r["y"] = y
        key = "mlp_within_tol"
    v = verdict(cfg, host, bad)
    assert not v[key] and not v["ok"], (plant, v)
