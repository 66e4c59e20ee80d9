"""Parity of the dense-prefix MLP (np_dense_mlp) with the oracle's dense
matrix-form MLP (O6), and of a decode path with a dense prefix in front of
the sparse layers (the prefix running while the sparse rows are staged)."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import DEV, Bufs, compare_delta, decode_y, mlp_tolerance, say, to_dev
from test_gpu_parity import SHAPES

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "ragged_f16", "ragged_bf16", "wide_f16", "wide_bf16",
                                  "k_eq_f"])
def test_dense_mlp(name):
    cfg = SHAPES[name]
    L, d, F = cfg.layers, cfg.d_model, cfg.d_ffn
    say(f"[dense] {name} d={d} F={F}")
    bufs = Bufs(cfg)
    bufs.reset()
    store = W.storage(cfg)
    h = W.hidden(cfg, 2)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    for l in range(L):
        w = to_dev(store[l])
        for t in range(2):
            B.np_dense_mlp(bufs.shape, w, to_dev(h[t]), y, bufs.ws)
            torch.cuda.synchronize()
            _, ref64 = orc.dense_mlp(cfg, l, h[t], store, want_f64=True)
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (l, t)
    assert B.np_device_error(bufs.ws) == 0


def test_dense_mlp_dyadic_7b_width():
    """A whole 7B-sized dense layer (d 4096, F 11008: the rows kernel in
    several rounds) on dyadic records (m 2^-6, |m| <= 1) and x in {-1, 0, 1}:
    every sum exact while max|a| < 2^12 and every column's sum of |a_n D_nj|
    stays below 2^6 (checked), so y equals O6's value for value."""
    cfg = W.Config("dense_dyadic", 1, 4096, 11008, 16, 0.15, 0.5, "f16", "f16", 2,
                   rho_given=0.5, dyadic=True, dyadic_w_range=1, dyadic_h_range=1)
    d = cfg.d_model
    say("[dense dyadic] d=4096 F=11008")
    bufs = Bufs(cfg)
    store = W.storage(cfg)
    h = W.hidden(cfg, 2)
    rec = orc.decode(cfg.wdtype, store[0])
    w = to_dev(store[0])
    y = torch.zeros(d * 2, dtype=torch.uint8, device=DEV)
    for t in range(2):
        xv = orc.decode(cfg.adtype, h[t])
        a = np.maximum(rec[:, :d] @ xv, 0) * (rec[:, d:2 * d] @ xv)
        assert np.max(np.abs(a)) < 2.0 ** 12 and np.max(np.abs(a) @ np.abs(rec[:, 2 * d:])) < 2.0 ** 6
        B.np_dense_mlp(bufs.shape, w, to_dev(h[t]), y, bufs.ws)
        torch.cuda.synchronize()
        ref = orc.dense_mlp(cfg, 0, h[t], store)
        assert np.array_equal(decode_y(orc, cfg.adtype, y.cpu().numpy()),
                              decode_y(orc, cfg.adtype, ref)), t
    assert B.np_device_error(bufs.ws) == 0


@pytest.mark.parametrize("tier,staging,overlap", [("device", "gather", False),
                                                  ("host", "memcpy", True),
                                                  ("file", "file", True)])
def test_dense_prefix_pipeline(tier, staging, overlap):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny")
    dl = 2
    say(f"[dense prefix] tier={tier} staging={staging} overlap={overlap}")
    T = 6
    pipe = DecodePipeline(cfg, tier=tier, staging=staging, overlap=overlap, tokens=T,
                          dense_layers=dl)
    dcfg = W.dense_config(cfg, dl)
    dstore = W.storage(dcfg)
    store = W.storage(cfg)
    h = W.hidden(cfg, T)
    A, Bm = W.predictor(cfg)
    st = orc.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    L, d = cfg.layers, cfg.d_model
    for t in range(T):
        pipe.step(t)
        torch.cuda.synchronize()
        yd = pipe.y_dense.cpu().numpy().reshape(dl, d).astype(np.float64)
        for l in range(dl):
            _, ref64 = orc.dense_mlp(dcfg, l, h[t], dstore, want_f64=True)
            assert np.all(np.abs(yd[l] - ref64) <= mlp_tolerance("f32", ref64)), (t, l)
        scores = pipe.scores.cpu().numpy().reshape(L, -1)
        _, ids = orc.select(scores, cfg.k)
        ref = orc.delta(t, ids, st, cfg.capacity)
        compare_delta(pipe.host_lists(), ref, L)
        y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64)), (t, l)
    assert pipe.device_error() == 0
