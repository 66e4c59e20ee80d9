"""Failure handling of host staging, forced from the host (a test hook makes
np_stage_rows fail before its first chunk, so every kernel still exits
normally): the failed staging marks the resident buffer, the next sparse-MLP
and staging calls on it return NP_ERR_STATE, and np_state_reset lifts the
mark; the decode then restarts from a cold start in lockstep with the
oracle."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import compare_delta, mlp_tolerance, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("overlap", [True, False])
def test_failed_staging_marks_resident(overlap, monkeypatch):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny")
    L, d, F, k = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k
    say(f"[stage failure] tiny memcpy overlap={overlap}")
    pipe = DecodePipeline(cfg, tier="host", staging="memcpy", overlap=overlap, tokens=6)
    pipe.step(0)
    pipe.step(1)
    torch.cuda.synchronize()
    monkeypatch.setenv("NP_TEST_FAIL_STAGE_AFTER", "0")
    with pytest.raises(B.NPError) as e:
        pipe.step(2)
    assert e.value.status == B.NP_ERR_HIP and "injected" in str(e.value)
    monkeypatch.delenv("NP_TEST_FAIL_STAGE_AFTER")
    torch.cuda.synchronize()
    s = pipe.shape
    with pytest.raises(B.NPError) as e:
        B.np_sparse_mlp(s, 0, pipe.x_ptr(2), pipe.resident, pipe.lists["active_slots"].data_ptr(), k,
                        pipe.y.data_ptr(), pipe.ws, pipe.main)
    assert e.value.status == B.NP_ERR_STATE
    with pytest.raises(B.NPError) as e:
        pipe.step(3)  # predict, select and delta run; its staging is refused
    assert e.value.status == B.NP_ERR_STATE
    torch.cuda.synchronize()
    # a cold start lifts the mark: three tokens in lockstep with the oracle
    pipe.reset()
    h = W.hidden(cfg, 6)
    store = W.storage(cfg)
    st = orc.State(L, F, cfg.capacity)
    for t in range(3):
        pipe.step(t)
        torch.cuda.synchronize()
        _, ids = orc.select(pipe.scores.cpu().numpy().reshape(L, F), k)
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, -1), ids), t
        compare_delta(pipe.host_lists(), orc.delta(t, ids, st, cfg.capacity), L)
        y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64)), (t, l)
    assert pipe.device_error() == 0
