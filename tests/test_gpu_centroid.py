"""Parity of the centroid-ID predictor and of the variable-count calls with
the oracle, through the C ABI.

Bars: logits within the fp32 accumulation bound of the heads; centroid ids,
intersection masks, active lists and counts bit-exact in lockstep (the
oracle's choice runs on the GPU's fp32 logits); delta lists and slot maps
bit-exact; MLP outputs within the tolerance of the activation type.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import DEV, Bufs, compare_delta, decode_y, from_dev, mlp_tolerance, say, to_dev
from test_gpu_parity import cfg_small, stage_and_check

pytestmark = pytest.mark.gpu


def ccfg(name, L, d, F, r, k, C, dt, K, D):
    return cfg_small(name, L, d, F, r, k, C, dt, centroid_k=K, feat_dim=D)


SHAPES = {
    "tiny_f32": ccfg("c_tiny", 3, 64, 1024, 8, 102, 300, "f32", 64, 128),
    "ragged_f16": ccfg("c_ragged_f16", 2, 64, 1000, 8, 150, 400, "f16", 100, 264),
    "ragged_bf16": ccfg("c_ragged_bf16", 3, 64, 777, 8, 120, 200, "bf16", 37, 520),
    "f_11001": ccfg("c_f11001", 2, 64, 11001, 8, 1650, 5000, "f16", 512, 4096),
    "f_20000": ccfg("c_f20000", 1, 64, 20000, 8, 3000, 6000, "bf16", 16, 64),
    "f_max": ccfg("c_fmax", 1, 64, 65535, 8, 8192, 8192, "f32", 8, 32),
}


class CBufs:
    """Device buffers of the centroid predictor for one shape."""

    def __init__(self, cfg, bank=None, heads=None):
        L, K, F, k = cfg.layers, cfg.centroid_k, cfg.d_ffn, cfg.k
        self.cfg, self.words = cfg, (F + 31) // 32
        self.heads_np = W.centroid_heads(cfg) if heads is None else heads
        self.bank_np = W.centroid_bank(cfg) if bank is None else bank
        self.heads, self.bank = to_dev(self.heads_np), to_dev(self.bank_np)
        self.model = B.np_centroid_model(K, cfg.feat_dim, self.heads.data_ptr(),
                                         self.bank.data_ptr())
        i32 = lambda n: torch.full((max(n, 4),), -7, dtype=torch.int32, device=DEV)
        self.logits = torch.zeros(2 * L * K, dtype=torch.float32, device=DEV)
        self.cids, self.counts = i32(2 * L), i32(L)
        self.mask = i32(L * self.words)
        self.ids = i32(L * k)

    def run(self, bufs, feat):
        B.np_centroid_select(bufs.shape, self.model, feat, self.logits, self.cids, self.mask,
                             self.ids, self.counts, bufs.ws)
        torch.cuda.synchronize()
        cfg = self.cfg
        L, K = cfg.layers, cfg.centroid_k
        return dict(logits=from_dev(self.logits, np.float32, (2 * L, K)),
                    cids=from_dev(self.cids, np.int32, (-1,))[:2 * L].reshape(2, L),
                    mask=from_dev(self.mask, np.uint32, (L, self.words)),
                    ids=from_dev(self.ids, np.int32, (L, cfg.k)),
                    counts=from_dev(self.counts, np.int32, (-1,))[:L])


@pytest.mark.parametrize("name", list(SHAPES))
def test_centroid_select(name):
    cfg = SHAPES[name]
    L, K, D, F, k = cfg.layers, cfg.centroid_k, cfg.feat_dim, cfg.d_ffn, cfg.k
    say(f"[centroid] {name} L'={L} F={F} k={k} K={K} D={D}")
    bufs = Bufs(cfg)
    bufs.reset()
    cb = CBufs(cfg)
    feats = W.features(cfg, 3)
    Hd = np.abs(orc.decode(cfg.wdtype, cb.heads_np)).reshape(2 * L * K, D)
    for t in range(3):
        got = cb.run(bufs, to_dev(feats[t]))
        ref = orc.centroid_logits(cb.heads_np, feats[t], 2 * L, K, D, cfg.wdtype, cfg.adtype)
        fd = np.abs(orc.decode(cfg.adtype, feats[t]))
        bound = (D + 2) * 2.0 ** -24 * (Hd @ fd).reshape(2 * L, K) + np.abs(ref) * 2.0 ** -23
        assert np.all(np.abs(got["logits"].astype(np.float64) - ref) <= bound)
        o = orc.centroid_active(got["logits"], cb.bank_np, L, F, K, k)
        assert np.array_equal(got["cids"], o["cids"])
        assert np.array_equal(got["mask"], o["mask"])
        assert np.array_equal(got["counts"], o["counts"])
        for l in range(L):
            n = o["counts"][l]
            assert np.array_equal(got["ids"][l][:n], o["active_ids"][l][:n]), (t, l)
        assert o["overflow"] == bool(B.np_device_error(bufs.ws) & B.NP_DEVERR_OVERFLOW)
    assert B.np_device_error(bufs.ws) == 0


def test_centroid_ties_nan_and_overflow():
    """Dyadic heads and integer features make exact logits with many ties;
    a NaN row never wins and raises its bit; a full bank overflows the list."""
    cfg = ccfg("c_ties", 2, 64, 300, 8, 40, 100, "f16", 48, 64)
    L, K, D, F, k = cfg.layers, cfg.centroid_k, cfg.feat_dim, cfg.d_ffn, cfg.k
    rng = np.random.default_rng(9)
    heads = orc.encode("f16", rng.integers(-1, 2, size=(2, L, K, D)) * 2.0 ** -3)
    feat = orc.encode("f16", rng.integers(-1, 2, size=D).astype(np.float64))
    bufs = Bufs(cfg)
    bufs.reset()
    cb = CBufs(cfg, heads=heads)
    got = cb.run(bufs, to_dev(feat))
    exact = orc.centroid_logits(heads, feat, 2 * L, K, D, "f16", "f16")
    assert np.array_equal(got["logits"], exact)
    assert len(np.unique(exact)) < exact.size  # ties exist
    o = orc.centroid_active(got["logits"], cb.bank_np, L, F, K, k)
    assert np.array_equal(got["cids"], o["cids"]) and np.array_equal(got["mask"], o["mask"])
    assert B.np_device_error(bufs.ws) == 0
    # NaN in the row of the best gate centroid of layer 0
    best = int(o["cids"][0, 0])
    h2 = heads.copy()
    h2[0, 0, best, 0] = 0x7E00  # fp16 quiet NaN
    cb2 = CBufs(cfg, heads=h2)
    got2 = cb2.run(bufs, to_dev(feat))
    assert np.isnan(got2["logits"][0, best])
    assert got2["cids"][0, 0] != best
    assert B.np_device_error(bufs.ws) & B.NP_DEVERR_NAN_SCORE
    # every mask full: the intersection is all F neurons, the list the first k
    bufs.reset()
    full = np.full_like(cb.bank_np, 0xFFFFFFFF)
    cb3 = CBufs(cfg, heads=heads, bank=full)
    got3 = cb3.run(bufs, to_dev(feat))
    assert got3["counts"].tolist() == [k] * L
    assert np.array_equal(got3["ids"], np.tile(np.arange(k, dtype=np.int32), (L, 1)))
    assert B.np_device_error(bufs.ws) & B.NP_DEVERR_OVERFLOW


@pytest.mark.parametrize("name", ["tiny_f32", "ragged_bf16", "f_11001", "f_max"])
def test_delta_n_variable_sets(name):
    cfg = SHAPES[name]
    L, F, k, C = cfg.layers, cfg.d_ffn, cfg.k, cfg.capacity
    say(f"[delta_n] {name}")
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(F)
    st = orc.State(L, F, C)
    counts_dev = torch.zeros(max(L, 4), dtype=torch.int32, device=DEV)
    cur = [np.sort(rng.choice(F, k, replace=False)) for _ in range(L)]
    for t in range(10):
        A = np.full((L, k), -1, np.int32)
        n = np.empty(L, np.int32)
        for l in range(L):
            nl = int(rng.choice([0, k, rng.integers(0, k + 1)])) if t else k
            keep = cur[l][rng.random(cur[l].size) < 0.8][:nl]
            rest = np.setdiff1d(np.arange(F), keep)
            cur[l] = np.sort(np.concatenate([keep, rng.choice(rest, nl - keep.size, replace=False)]))
            A[l, :nl] = cur[l]
            n[l] = nl
        bufs.ids.copy_(torch.from_numpy(A.reshape(-1)))
        counts_dev[:L].copy_(torch.from_numpy(n))
        B.np_delta_n(bufs.shape, t, bufs.ids, counts_dev, bufs.state, bufs.out, bufs.ws)
        torch.cuda.synchronize()
        ref = orc.delta_n(t, A, n, st, C)
        got = bufs.host_lists()
        for l in range(L):  # active_slots are defined for the first n[l] entries only
            got["active_slots"][l][n[l]:] = -1
        compare_delta(got, ref, L)
        P, Q, U = bufs.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of)
        assert np.array_equal(U, st.last_used)
    assert B.np_device_error(bufs.ws) == 0


def test_sparse_mlp_n_device_counts():
    cfg = cfg_small("mlp_n", 3, 5120, 2000, 64, 300, 700, "f16")
    say(f"[mlp_n] d={cfg.d_model}")
    bufs, resident, store, st = stage_and_check(cfg, "gather_device")
    L, k, d, esz = cfg.layers, cfg.k, cfg.d_model, 2
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    slots = bufs.lists["active_slots"].cpu().numpy().reshape(L, k)
    y = torch.zeros(L * d * esz, dtype=torch.uint8, device=DEV)
    for n in ([0, 1, 300], [63, 64, 65], [257, 299, 300]):
        counts = torch.tensor(n + [0], dtype=torch.int32, device=DEV)
        for l in range(L):
            B.np_sparse_mlp_n(bufs.shape, l, x, resident, bufs.lists["active_slots"].data_ptr()
                              + 4 * l * k, counts, y.data_ptr() + l * d * esz, bufs.ws)
        torch.cuda.synchronize()
        yb = y.cpu().numpy()
        for l in range(L):
            ids = np.sort(st.neuron_of[l][slots[l][:n[l]]]).astype(np.int32)
            _, ref64 = orc.sparse_mlp(cfg, l, h, store, ids, want_f64=True)
            got = decode_y(orc, cfg.adtype, yb[l * d * esz:(l + 1) * d * esz])
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (n, l)
    assert B.np_device_error(bufs.ws) == 0


@pytest.mark.parametrize("graph", [False, True])
def test_centroid_pipeline_lockstep(graph):
    """The whole decode path with the centroid predictor against the oracle,
    token by token: choice and sets, delta, resident bytes and MLP outputs."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny").with_(centroid_k=64, feat_dim=128)
    L, d, F, K, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.centroid_k, cfg.k, cfg.capacity
    T = 8
    say(f"[centroid lockstep] graph={graph}")
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T, predictor="centroid")
    if graph:
        pipe.capture_graph()
    h = W.hidden(cfg, T)
    store = W.storage(cfg)
    bank = W.centroid_bank(cfg)
    st = orc.State(L, F, C)
    res_ref = np.zeros((L, C, 3 * d), np.float32)
    for t in range(T):
        pipe.step_graph(t) if graph else pipe.step(t)
        torch.cuda.synchronize()
        logits = pipe.logits.cpu().numpy().reshape(2 * L, K)
        o = orc.centroid_active(logits, bank, L, F, K, k)
        n = pipe.active_counts.cpu().numpy()[:L]
        assert np.array_equal(n, o["counts"])
        ids = pipe.active_ids.cpu().numpy().reshape(L, k)
        for l in range(L):
            assert np.array_equal(ids[l][:n[l]], o["active_ids"][l][:n[l]])
        ref = orc.delta_n(t, o["active_ids"], o["counts"], st, C)
        got = pipe.host_lists()
        for l in range(L):
            got["active_slots"][l][n[l]:] = -1
        compare_delta(got, ref, L)
        orc.stage(cfg, ref["counts"], ref["in_ids"], ref["in_slots"], store, res_ref)
        got_res = pipe.resident.cpu().numpy().view(np.float32).reshape(res_ref.shape)
        occupied = st.neuron_of >= 0
        assert np.array_equal(got_res[occupied], res_ref[occupied])
        y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, o["active_ids"][l][:n[l]],
                                      want_f64=True)
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64))
    assert pipe.device_error() == 0


def test_centroid_pipeline_7b_fullsize():
    """The decode path with the centroid predictor at the full 7B shape
    (K = 512 centroids, D = 4096 features, 2 x 31 heads), 16 eager tokens in
    lockstep with the oracle: logits within the fp32 bound on the first
    token; centroid ids, intersection masks, lists, counts, delta lists and
    slot maps bit for bit on every token; MLP outputs sampled."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("7b")
    L, d, F, K, D, k, C = (cfg.layers, cfg.d_model, cfg.d_ffn, cfg.centroid_k, cfg.feat_dim,
                           cfg.k, cfg.capacity)
    T = 16
    say(f"[centroid fullsize] 7b K={K} D={D}, {T} tokens")
    host = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, host.data_ptr())
    store = host.numpy().view(np.uint16).reshape(L, F, 3 * d)
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T, host_storage=host,
                          predictor="centroid")
    heads = W.centroid_heads(cfg)
    feats = W.features(cfg, T)
    bank = W.centroid_bank(cfg)
    h = W.hidden(cfg, T)
    st = orc.State(L, F, C)
    rng = np.random.default_rng(4)
    for t in range(T):
        pipe.step(t)
        torch.cuda.synchronize()
        logits = pipe.logits.cpu().numpy().reshape(2 * L, K)
        if t == 0:
            ref = orc.centroid_logits(heads, feats[0], 2 * L, K, D, cfg.wdtype, cfg.adtype)
            Hd = np.abs(orc.decode(cfg.wdtype, heads).reshape(2 * L * K, D))
            fd = np.abs(orc.decode(cfg.adtype, feats[0]))
            bound = (D + 2) * 2.0 ** -24 * (Hd @ fd).reshape(2 * L, K) + np.abs(ref) * 2.0 ** -23
            assert np.all(np.abs(logits.astype(np.float64) - ref) <= bound)
        o = orc.centroid_active(logits, bank, L, F, K, k)
        n = pipe.active_counts.cpu().numpy()[:L]
        assert np.array_equal(n, o["counts"]), t
        assert np.array_equal(pipe.cids.cpu().numpy()[:2 * L].reshape(2, L), o["cids"]), t
        assert np.array_equal(pipe.mask.cpu().numpy().view(np.uint32).reshape(L, -1), o["mask"])
        ids = pipe.active_ids.cpu().numpy().reshape(L, k)
        for l in range(L):
            assert np.array_equal(ids[l][:n[l]], o["active_ids"][l][:n[l]]), (t, l)
        ref_d = orc.delta_n(t, o["active_ids"], o["counts"], st, C)
        got = pipe.host_lists()
        for l in range(L):
            got["active_slots"][l][n[l]:] = -1
        compare_delta(got, ref_d, L)
        P, Q, U = pipe.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of), t
        if t % 5 == 4:
            y = pipe.y.cpu().numpy().view(np.uint16).reshape(L, d)
            for l in sorted(rng.choice(L, 2, replace=False)):
                _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, o["active_ids"][l][:n[l]],
                                          want_f64=True)
                got_y = decode_y(orc, cfg.adtype, y[l])
                assert np.all(np.abs(got_y - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (t, l)
    assert pipe.device_error() == 0
