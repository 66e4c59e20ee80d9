"""The dense-prefix solver against brute force over every prefix length."""
import itertools

import pytest

from paper_2608_22643_amd import split
from paper_2608_22643_amd import workload as W


def brute(budget, n, lb, bb, fixed, min_dense):
    fits = [d for d in range(min_dense, n + 1)
            if split.resident_bytes(d, n, lb, bb, fixed) <= budget]
    return max(fits) if fits else None


@pytest.mark.parametrize("n,lb,bb,fixed", [(32, 352, 129, 5000), (32, 352, 231, 5000),
                                           (8, 10, 10, 3), (5, 7, 0, 0), (40, 100, 40, 17)])
def test_closed_form_matches_brute_force(n, lb, bb, fixed):
    for budget, min_dense in itertools.product(range(0, n * lb + fixed + 50, 7), (0, 1, 2)):
        want = brute(budget, n, lb, bb, fixed, min_dense)
        if want is None:
            with pytest.raises(ValueError):
                split.dense_prefix(budget, n, lb, bb, fixed, min_dense)
        else:
            assert split.dense_prefix(budget, n, lb, bb, fixed, min_dense) == want


def test_larger_buffers_move_the_peak_earlier():
    # the paper's observation: bigger K_max buffers leave less room for dense layers
    mib = 1 << 20
    d = [split.dense_prefix(12186 * mib, 32, 336 * mib, b * mib, 4000 * mib) for b in (129, 168, 231)]
    assert d[0] > d[1] > d[2]


def test_config_wrapper_counts_layer_zero_and_predictor():
    cfg = W.get("7b")
    rec = cfg.record_bytes
    pred = cfg.layers * cfg.rank * (cfg.d_model + cfg.d_ffn) * 2
    need = pred + 5 * cfg.d_ffn * rec + (cfg.layers + 1 - 5) * cfg.capacity * rec
    assert split.for_config(cfg, need) == 5
    assert split.for_config(cfg, need - 1) == 4
    assert split.for_config(cfg, 1 << 50) == cfg.layers + 1


def test_rejects_bad_arguments():
    with pytest.raises(ValueError):
        split.dense_prefix(100, 4, 5, 6)  # buffer larger than a layer
    with pytest.raises(ValueError):
        split.resident_bytes(5, 4, 1, 1, 0)
