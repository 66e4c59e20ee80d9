"""Parity at the full 7B shape (31 downstream layers, d=4096, F=11008,
r=416, k=1651, C=5504, fp16) in the launch configuration bench.py times:
storage tier in HBM, gather staging on a side stream in layer chunks, the
decode step replayed from a HIP graph with the token index from the device
step counter.

Per token, against the oracle: every score within the predictor's fp32
bound; every mask, active-id list, delta list and slot map bit for bit (the
oracle's select runs on the GPU's scores, so both take the same decisions);
the oracle's own scores through its own top-k against the GPU's sets, every
difference a near-tie within the score bound;
resident records byte-equal to the storage rows on a sample of slots; MLP
outputs within the fp16 tolerance on every layer of one steady token and on
sampled layers of the others.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import workload as W
from gpu_util import check_native_mask, compare_delta, decode_y, mlp_tolerance, say

pytestmark = pytest.mark.gpu


def test_fullsize_7b_graph_step():
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("7b")
    L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
    T = 4
    say(f"[fullsize] 7b: generating the {cfg.storage_bytes / 1e9:.2f} GB storage tier")
    host = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, host.data_ptr())
    store = host.numpy().view(np.uint16).reshape(L, F, 3 * d)
    pipe = DecodePipeline(cfg, tier="device", staging="gather", overlap=True, tokens=T,
                          host_storage=host)
    pipe.capture_graph()
    A, Bm = W.predictor(cfg)
    h = W.hidden(cfg, T)
    absA = np.abs(orc.decode(cfg.wdtype, A)).reshape(L, cfg.rank, d)
    absB = np.abs(orc.decode(cfg.wdtype, Bm)).reshape(L, F, cfg.rank)

    def bound(ht):  # fp32 accumulation bound of s = B (A h): (d + r + 2) u sum |B||A||h|
        hd = np.abs(orc.decode(cfg.adtype, ht))
        mag = np.stack([absB[l] @ (absA[l] @ hd) for l in range(L)])
        return (d + cfg.rank + 2) * 2.0 ** -24 * mag

    st = orc.State(L, F, C)
    rng = np.random.default_rng(7)
    esz = 2
    for t in range(T):
        say(f"[fullsize] token {t}")
        pipe.step_graph(t)
        torch.cuda.synchronize()
        scores = pipe.scores.cpu().numpy().reshape(L, F)
        ref_s = orc.predict(cfg, h[t], A, Bm).astype(np.float64)
        tol = bound(h[t]) + np.abs(ref_s) * 2.0 ** -23
        assert np.all(np.abs(scores.astype(np.float64) - ref_s) <= tol), t
        mask, ids = orc.select(scores, k)
        n_tie = check_native_mask(pipe.active_ids.cpu().numpy().reshape(L, k), ref_s, tol, k)
        say(f"[fullsize] token {t}: native-mask near-ties {n_tie}")
        assert np.array_equal(pipe.mask.cpu().numpy().view(np.uint32).reshape(L, -1), mask), t
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, k), ids), t
        ref = orc.delta(t, ids, st, C)
        compare_delta(pipe.host_lists(), ref, L)
        P, Q, U = pipe.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of), t
        assert np.array_equal(U, st.last_used), t
        # resident records: 256 occupied slots drawn at random
        res = pipe.resident.view(L, C, 3 * d * esz)
        occ = np.argwhere(st.neuron_of >= 0)
        for l, s in occ[rng.choice(len(occ), 256, replace=False)]:
            got = res[l, s].cpu().numpy().view(np.uint16)
            assert np.array_equal(got, store[l, st.neuron_of[l, s]]), (t, l, s)
        y = pipe.y.cpu().numpy().view(np.uint16).reshape(L, d)
        layers = range(L) if t == 2 else sorted(rng.choice(L, 4, replace=False))
        for l in layers:
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
            got = decode_y(orc, cfg.adtype, y[l])
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (t, l)
    assert pipe.device_error() == 0


def test_fullsize_7b_long_sequence():
    """64 tokens of the 7B decode replayed from a HIP graph, in lockstep with
    the oracle's selection and delta on every token (masks, ids, every delta
    list and the slot maps bit for bit: the resident set fills, then LRU
    victims appear), resident records on sampled slots every 8th token, and
    the MLP output of two layers every 16th token."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("7b")
    L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
    T = 64
    say(f"[fullsize] 7b long sequence, {T} tokens")
    host = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, host.data_ptr())
    store = host.numpy().view(np.uint16).reshape(L, F, 3 * d)
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T, host_storage=host)
    pipe.capture_graph()
    h = W.hidden(cfg, T)
    st = orc.State(L, F, C)
    rng = np.random.default_rng(9)
    evictions = 0
    for t in range(T):
        pipe.step_graph(t)
        torch.cuda.synchronize()
        scores = pipe.scores.cpu().numpy().reshape(L, F)
        mask, ids = orc.select(scores, k)
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, k), ids), t
        assert np.array_equal(pipe.mask.cpu().numpy().view(np.uint32).reshape(L, -1), mask), t
        ref = orc.delta(t, ids, st, C)
        compare_delta(pipe.host_lists(), ref, L)
        evictions += int(ref["counts"][:, 2].sum())
        P, Q, U = pipe.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of), t
        assert np.array_equal(U, st.last_used), t
        if t % 8 == 7:
            res = pipe.resident.view(L, C, 3 * d * 2)
            occ = np.argwhere(st.neuron_of >= 0)
            for l, s in occ[rng.choice(len(occ), 64, replace=False)]:
                got = res[l, s].cpu().numpy().view(np.uint16)
                assert np.array_equal(got, store[l, st.neuron_of[l, s]]), (t, l, s)
        if t % 16 == 15:
            y = pipe.y.cpu().numpy().view(np.uint16).reshape(L, d)
            for l in sorted(rng.choice(L, 2, replace=False)):
                _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
                got = decode_y(orc, cfg.adtype, y[l])
                assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (t, l)
    assert evictions > 0, "the sequence never filled the resident set"
    assert pipe.device_error() == 0
