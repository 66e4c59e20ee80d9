"""The parity verdict of bench.py's oracle leg, on the CPU: references built
by the oracle itself (standing in for the GPU's first tokens, and for the
sampled layers of a full-size run) pass, and a wrong active id, a wrong delta
entry, a wrong slot map or an MLP output outside the tolerance each turn the
verdict false."""
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


def verdict(cfg, host, refs, samples=()):
    return bench.cpu_baseline(cfg, host, 0.0, refs, samples)["parity"]


def sample_of(cfg, refs, t=2, layers=(0, 2)):
    """What the full-size leg keeps: a few layers of one token."""
    r = refs[t]
    L = list(layers)
    return {"cfg": cfg, "tokens": 64, "token": t, "layers": L, "scores": r["scores"][L].copy(),
            "ids": r["ids"][L].copy(), "y": r["y"][L].copy()}


def test_sampled_layers_checked(tiny):
    cfg, host, refs = tiny
    good = verdict(cfg, host, refs, [sample_of(cfg, refs)])
    assert good["ok"] and good["sampled"]["tiny"]["ok"], good
    bad = sample_of(cfg, refs)
    bad["y"][1, 3] = np.float32(bad["y"][1, 3] + 1.0)
    v = verdict(cfg, host, refs, [bad])
    assert not v["sampled"]["tiny"]["mlp_within_tol"] and not v["ok"], v
    bad = sample_of(cfg, refs)
    bad["ids"][0, 1] = (bad["ids"][0, 1] + 1) % cfg.d_ffn
    v = verdict(cfg, host, refs, [bad])
    assert not v["sampled"]["tiny"]["select_exact"] and not v["ok"], v


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
