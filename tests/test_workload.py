"""Generator checks and the paper's printed arithmetic.

* the counter-based generator gives the same element regardless of which
  sub-range is generated;
* record layout arithmetic reproduces the per-layer buffer sizes the paper
  prints (tests/golden/paper_numbers.json);
* the low-rank predictor's parameter share is close to the paper's 2.86%;
* consecutive top-k sets of the synthetic workload overlap as the closed form
  P(X > q, Y > q) / p predicts (persistence target of the paper).
"""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")


def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_generator_is_counter_based(wl):
    cfg = wl.Config("g", 4, 64, 40, 8, 0.1, 0.5, "f16", "f16", 4, rho_given=0.5)
    full = wl.storage(cfg)
    part = wl.storage(cfg, layer0=2, layers=1)
    assert np.array_equal(full[2], part[0])
    again = wl.storage(cfg)
    assert np.array_equal(full, again)
    other = wl.storage(cfg.with_(seed=1))
    assert not np.array_equal(full, other)


def test_generator_distribution(wl, orc):
    cfg = wl.Config("g", 2, 256, 512, 32, 0.1, 0.5, "f32", "f32", 4, rho_given=0.5)
    v = wl.storage(cfg).astype(np.float64).ravel()
    assert abs(v.mean()) < 2e-4 and abs(v.std() - 0.02) < 2e-4
    A, B = wl.predictor(cfg)
    assert abs(A.std() - 1 / np.sqrt(256)) < 2e-3 and abs(B.std() - 1 / np.sqrt(32)) < 5e-3


def test_hidden_ar1_correlation(wl):
    cfg = wl.Config("g", 1, 4096, 64, 8, 0.1, 0.5, "f32", "f32", 64, rho_given=0.9)
    _, h = wl.hidden(cfg, want_f64=True)
    c = np.mean([np.corrcoef(h[t], h[t + 1])[0, 1] for t in range(63)])
    assert abs(c - 0.9) < 0.01
    assert abs(h.std() - 1.0) < 0.02


def test_record_layout_matches_printed_buffer_sizes():
    g = golden()["record_layout"]
    rec = 3 * g["d_model"] * g["bytes_per_element"]
    assert rec == 24 * 1024
    for rows, mib in g["buffer_rows_and_MiB"]:
        assert round(rows * rec / 2 ** 20) == mib


def test_kmax_percentages():
    g = golden()["kmax_budgets"]
    for kmax, pct in g["kmax_and_percent_active"]:
        assert round(100 * kmax / g["d_ffn"], 1) == pct


def test_predictor_share_close_to_paper(wl):
    g = golden()["predictor"]
    comps = g["components_M"]
    assert abs(sum(comps.values()) - g["total_params_M"]) < 0.11
    # residual trunk: 4 blocks of (8T x 4T + 4T x 8T) weights, T = 512
    T = g["T"]
    assert abs(g["trunk_blocks"] * 2 * (8 * T) * (4 * T) / 1e6 - comps["residual_trunk"]) < 0.1
    cfg = wl.get("7b")
    lowrank = cfg.layers * cfg.rank * (cfg.d_model + cfg.d_ffn)
    # Llama-2-7B-shaped model: 32 layers x (4 d^2 attention + 3 d F MLP) + 2 x 32000 x d
    model = 32 * (4 * 4096 ** 2 + 3 * 4096 * 11008) + 2 * 32000 * 4096
    share = 100 * lowrank / model
    assert abs(share - g["percent_of_base_model"]) < 0.1, share


@pytest.mark.parametrize("p,target", [(0.15, 0.835), (0.10, 0.85), (0.15, 0.70)])
def test_rho_solves_closed_form(wl, p, target):
    rho = wl.rho_for_persistence(p, target)
    assert abs(wl.persistence_closed_form(rho, p) - target) < 1e-6


def test_measured_persistence_matches_closed_form(wl, orc):
    # 7B-like activity (15%) and persistence target (83.5%) at a reduced width
    base = wl.get("7b")
    cfg = wl.Config("p", 2, 256, 11008, 64, 0.15, 0.5, "f32", "f32", 24,
                    persistence=0.835)
    assert abs(cfg.rho - base.rho) < 1e-9
    A, B = wl.predictor(cfg)
    h = wl.hidden(cfg)
    prev = None
    overlaps = []
    for t in range(cfg.tokens):
        s = orc.predict(cfg, h[t], A, B)
        _, ids = orc.select(s, cfg.k)
        if prev is not None:
            for l in range(cfg.layers):
                overlaps.append(len(set(ids[l]) & set(prev[l])) / cfg.k)
        prev = ids
    m = float(np.mean(overlaps))
    lo, hi = golden()["persistence"]["low"], golden()["persistence"]["high"]
    assert lo <= m <= hi, m
    assert abs(m - 0.835) < 0.01, m
