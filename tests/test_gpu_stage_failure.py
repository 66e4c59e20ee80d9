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


def test_reset_lifts_only_its_own_mark(monkeypatch):
    """Two decode pipelines, each with its own resident buffer: a failed
    staging into the first marks only that buffer; the second keeps staging
    and computing; a reset that names the second buffer leaves the first's
    mark; the first pipeline's own cold start lifts it."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny")
    k = cfg.k
    a = DecodePipeline(cfg, tier="host", staging="memcpy", overlap=False, tokens=4)
    b = DecodePipeline(cfg, tier="host", staging="memcpy", overlap=False, tokens=4)
    a.step(0)
    b.step(0)
    torch.cuda.synchronize()
    monkeypatch.setenv("NP_TEST_FAIL_STAGE_AFTER", "0")
    with pytest.raises(B.NPError):
        a.step(1)
    monkeypatch.delenv("NP_TEST_FAIL_STAGE_AFTER")
    torch.cuda.synchronize()

    def mlp(p):
        B.np_sparse_mlp(p.shape, 0, p.x_ptr(1), p.resident, p.lists["active_slots"].data_ptr(), k,
                        p.y.data_ptr(), p.ws, p.main)

    with pytest.raises(B.NPError) as e:
        mlp(a)
    assert e.value.status == B.NP_ERR_STATE
    b.step(1)  # the other pipeline is not affected
    mlp(b)
    b.reset()  # names b's resident buffer only
    with pytest.raises(B.NPError) as e:
        mlp(a)
    assert e.value.status == B.NP_ERR_STATE
    a.reset()
    mlp(a)
    torch.cuda.synchronize()
    assert a.device_error() == 0 and b.device_error() == 0
