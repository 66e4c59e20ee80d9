"""Two decode pipelines staging through the host at the same time, from two
host threads (each with its own staging buffer, landing area, streams and
state): np_stage_rows keeps its between-call state per staging buffer, so
the two runs are independent, and each must follow the oracle in lockstep
(delta lists bit for bit, every occupied resident slot byte-equal to its
storage record, MLP outputs within the fp32 bound)."""
import threading

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import workload as W
from gpu_util import compare_delta, mlp_tolerance, say

pytestmark = pytest.mark.gpu


def run_one(cfg, overlap, T, errors, idx):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    try:
        torch.cuda.set_device(0)
        L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
        pipe = DecodePipeline(cfg, tier="host", staging="memcpy", overlap=overlap, tokens=T,
                              staging_mib=0.25, landing_mib=0.05)
        h = W.hidden(cfg, T)
        store = W.storage(cfg)
        st = orc.State(L, F, C)
        for t in range(T):
            pipe.step(t)
            pipe.main.synchronize()
            pipe.side.synchronize()
            _, ids = orc.select(pipe.scores.cpu().numpy().reshape(L, F), k)
            assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, -1), ids), t
            compare_delta(pipe.host_lists(), orc.delta(t, ids, st, C), L)
            res = pipe.resident.cpu().numpy().view(np.float32).reshape(L, C, -1)
            for l, s in np.argwhere(st.neuron_of >= 0):
                assert np.array_equal(res[l, s], store[l, st.neuron_of[l, s]]), (t, l, s)
            y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
            for l in range(L):
                _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
                assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64)), (t, l)
        assert pipe.device_error() == 0
    except BaseException as e:  # noqa: BLE001  (reported by the main thread)
        errors[idx] = e


def test_two_pipelines_stage_at_once():
    T = 10
    # two workloads of the tiny shape with different seeds; landing areas of
    # a few records, so each token's staging runs several rounds
    cfgs = [W.get("tiny"), W.get("tiny").with_(seed=3)]
    say("[concurrent staging] two pipelines, two host threads")
    errors = [None, None]
    th = [threading.Thread(target=run_one, args=(c, ov, T, errors, i))
          for i, (c, ov) in enumerate(zip(cfgs, (True, False)))]
    for t in th:
        t.start()
    for t in th:
        t.join(timeout=300)
    assert not any(t.is_alive() for t in th), "a staging thread did not finish"
    for e in errors:
        if e is not None:
            raise e
