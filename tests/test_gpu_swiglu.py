"""Parity of the SwiGLU MLP and the magnitude-threshold sparsity of eq. 1 with
the oracle: the gated MLP calls with act = SwiGLU (O5/O6), np_sparse_mlp_t
with per-layer thresholds (O5 with threshold), the batch activations on the
matrix cores (O9), the percentile (O10, bit for bit on the GPU's values) and
the thresholded active set (O11, bit for bit on the GPU's activations), and
the whole calibration chain at the full SwiGLU 7B shape.

Where floating point decides a row's fate (|a| against T), the GPU and the
oracle compute a in different precisions; rows within the activation error
bound of T may go either way, and the test widens the output tolerance by
exactly their possible contribution."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import DEV, Bufs, compare_delta, decode_y, mlp_tolerance, say, to_dev
from test_gpu_parity import SHAPES

pytestmark = pytest.mark.gpu

SW = {
    "tiny": W.get("tiny_swiglu"),
    "ragged_f16": SHAPES["ragged_f16"].with_(act="swiglu"),
    "ragged_bf16": SHAPES["ragged_bf16"].with_(act="swiglu"),
    "wide_bf16": SHAPES["wide_bf16"].with_(act="swiglu"),
    "f_11001": SHAPES["f_11001"].with_(act="swiglu"),
}


def resident_of(cfg, store, rng):
    """A resident buffer [L'][C][3d] holding a random C-subset of each
    layer's records; returns it and the neuron of every slot [L'][C]."""
    L, F, C = cfg.layers, cfg.d_ffn, cfg.capacity
    neuron = np.stack([rng.permutation(F)[:C] for _ in range(L)]).astype(np.int32)
    res = np.stack([store[l][neuron[l]] for l in range(L)])
    return to_dev(res), neuron


def parts(cfg, rec, X):
    """g, u (double) and the magnitude sums |G||x|, |U||x| for the records
    rec [n][3d] (storage bits) and tokens X [t][d] (storage bits)."""
    d = cfg.d_model
    R = orc.decode(cfg.wdtype, rec)
    G, U = R[:, :d], R[:, d:2 * d]
    Xd = orc.decode(cfg.adtype, X).reshape(-1, d)
    return (Xd @ G.T, Xd @ U.T, np.abs(Xd) @ np.abs(G).T, np.abs(Xd) @ np.abs(U).T)


def act_bound(cfg, g, u, sg, su):
    """Bound on |a_gpu - a| for a = act(g, u): fp32 accumulation of each sum,
    (d + 2) u_32 sum|w x|; the activation's slope (|SiLU'| < 1.1, ReLU 1);
    and a few float32 roundings of a (exp, 1 + e, the divide, the product)."""
    eg = (cfg.d_model + 2) * 2.0 ** -24 * sg
    eu = (cfg.d_model + 2) * 2.0 ** -24 * su
    a = g / (1.0 + np.exp(-g)) * u if cfg.act == "swiglu" else np.maximum(g, 0.0) * u
    return 1.1 * eg * (np.abs(u) + eu) + (np.abs(g) + eg) * eu + 2.0 ** -20 * np.abs(a) + 1e-30, a


# ---------------- gated MLP with SwiGLU ---------------------------------------

@pytest.mark.parametrize("name", sorted(SW))
def test_swiglu_sparse_dense_and_variable_mlp(name):
    cfg = SW[name]
    L, d, k, C = cfg.layers, cfg.d_model, cfg.k, cfg.capacity
    say(f"[swiglu mlp] {name} d={d} F={cfg.d_ffn} k={k}")
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(11)
    store = W.storage(cfg)
    res, neuron = resident_of(cfg, store, rng)
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    counts = torch.tensor(rng.integers(0, k + 1, size=L), dtype=torch.int32, device=DEV)
    for l in range(L):
        slots = np.sort(rng.choice(C, k, replace=False)).astype(np.int32)
        sl = to_dev(slots)
        for mode in ("fixed", "variable", "dense"):
            if mode == "fixed":
                B.np_sparse_mlp(bufs.shape, l, x, res, sl, k, y, bufs.ws)
                ids = neuron[l][slots]
            elif mode == "variable":
                B.np_sparse_mlp_n(bufs.shape, l, x, res, sl, counts, y, bufs.ws)
                ids = neuron[l][slots[:int(counts[l])]]
            else:
                B.np_dense_mlp(bufs.shape, to_dev(store[l]), x, y, bufs.ws)
            torch.cuda.synchronize()
            if mode == "dense":
                _, ref64 = orc.dense_mlp(cfg, l, h, store, want_f64=True)
            else:
                _, ref64 = orc.sparse_mlp(cfg, l, h, store, ids.astype(np.int32), want_f64=True)
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (l, mode)
    assert B.np_device_error(bufs.ws) == 0


# ---------------- eq. 1 in the sparse MLP --------------------------------------

def gap_threshold(a, lo=0.3, hi=0.6):
    """A float32 threshold in the widest gap of the sorted magnitudes between
    the lo and hi quantiles (a threshold no row sits close to)."""
    s = np.sort(np.abs(a))
    i0, i1 = max(int(lo * s.size), 0), max(int(hi * s.size), 2)
    j = i0 + int(np.argmax(np.diff(s[i0:i1])))
    return np.float32((s[j] + s[j + 1]) / 2), s[j + 1] - s[j]


@pytest.mark.parametrize("name", ["tiny", "ragged_f16", "ragged_bf16", "f_11001"])
def test_threshold_mlp(name):
    cfg = SW[name]
    L, d, k, C = cfg.layers, cfg.d_model, cfg.k, cfg.capacity
    say(f"[eq1 mlp] {name}")
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(12)
    store = W.storage(cfg)
    res, neuron = resident_of(cfg, store, rng)
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    y0 = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    all_slots = [np.sort(rng.choice(C, k, replace=False)).astype(np.int32) for _ in range(L)]
    T = np.zeros(L, np.float32)
    for l in range(L):
        g, u, sg, su = parts(cfg, store[l][neuron[l][all_slots[l]]], h)
        bound, a = act_bound(cfg, g[0], u[0], sg[0], su[0])
        T[l], gap = gap_threshold(a)
        assert np.all(np.abs(np.abs(a) - T[l]) > bound), "threshold within the error bound"
    thr = to_dev(T)
    counts = torch.tensor(rng.integers(1, k + 1, size=L), dtype=torch.int32, device=DEV)
    for l in range(L):
        sl = to_dev(all_slots[l])
        for use_counts in (False, True):
            n = int(counts[l]) if use_counts else k
            B.np_sparse_mlp_t(bufs.shape, l, x, res, sl, k, counts if use_counts else None, thr,
                              y, bufs.ws)
            torch.cuda.synchronize()
            ids = neuron[l][all_slots[l][:n]].astype(np.int32)
            _, ref64 = orc.sparse_mlp(cfg, l, h, store, ids, want_f64=True, threshold=float(T[l]))
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (l, n)
        # no thresholds: the same bits as np_sparse_mlp
        B.np_sparse_mlp_t(bufs.shape, l, x, res, sl, k, None, None, y, bufs.ws)
        B.np_sparse_mlp(bufs.shape, l, x, res, sl, k, y0, bufs.ws)
        torch.cuda.synchronize()
        assert torch.equal(y, y0), l
    assert B.np_device_error(bufs.ws) == 0


# ---------------- O9: batch activations on the matrix cores --------------------

@pytest.mark.parametrize("name,n", [("tiny", 1), ("tiny", 37), ("ragged_f16", 128),
                                    ("ragged_bf16", 200), ("wide_bf16", 33), ("f_11001", 64)])
@pytest.mark.parametrize("act", ["relu", "swiglu"])
def test_act_batch(name, n, act):
    cfg = SW[name].with_(act=act)
    F, d = cfg.d_ffn, cfg.d_model
    say(f"[act batch] {name} act={act} n={n} d={d} F={F}")
    shape = B.make_shape(cfg.layers, d, F, cfg.rank, cfg.k, cfg.capacity, cfg.wdtype,
                         cfg.adtype, act)
    store = W.storage(cfg, 0, 1)
    X = W.hidden(cfg, n)
    acts = torch.full((n * F,), float("nan"), dtype=torch.float32, device=DEV)
    B.np_act_batch(shape, to_dev(store[0]), to_dev(X), n, acts)
    torch.cuda.synchronize()
    got = acts.cpu().numpy().reshape(n, F).astype(np.float64)
    rows = sorted(set([0, n - 1, n // 2]))
    ref = orc.act_batch(cfg, store[0], X[rows], len(rows))
    g, u, sg, su = parts(cfg, store[0], X[rows])
    bound, a = act_bound(cfg, g, u, sg, su)
    assert np.all(np.abs(ref - a) <= 1e-9 * (np.abs(a) + bound))  # numpy agrees with O9
    assert np.all(np.abs(got[rows] - ref) <= bound), np.max(np.abs(got[rows] - ref) / bound)
    assert not np.isnan(got).any()  # every output written


@pytest.mark.parametrize("d,F,wdt,n", [(4096, 2000, "f16", 1), (4096, 2000, "f16", 128),
                                       (4096, 2000, "f16", 129), (5120, 1000, "f16", 77),
                                       (8192, 1000, "bf16", 64)])
def test_act_batch_dyadic_bit_exact(d, F, wdt, n):
    """The matrix-core batch activations on dyadic records (m 2^-6, |m| <= 1)
    and tokens in {-1, 0, 1}, ReLU-gated: g and u are multiples of 2^-6 below
    d 2^-6 and a = max(g, 0) u a multiple of 2^-12 below 2^12, all exact in
    fp32, so every activation equals O9's: the 7B, 13B and 70B widths, a
    ragged tile of neurons (F not a multiple of 64), one token, a full
    launch of 128 and one token past it."""
    cfg = W.Config("act_dyadic", 1, d, F, 16, 0.1, 0.5, wdt, wdt, n, rho_given=0.5,
                   dyadic=True, dyadic_w_range=1, dyadic_h_range=1)
    say(f"[act batch dyadic] d={d} F={F} {wdt} n={n}")
    shape = B.make_shape(1, d, F, cfg.rank, cfg.k, cfg.capacity, wdt, wdt, "relu")
    store = W.storage(cfg, 0, 1)
    X = W.hidden(cfg, n)
    assert set(np.unique(orc.decode(wdt, X))) <= {-1.0, 0.0, 1.0}
    acts = torch.full((n * F,), float("nan"), dtype=torch.float32, device=DEV)
    B.np_act_batch(shape, to_dev(store[0]), to_dev(X), n, acts)
    torch.cuda.synchronize()
    got = acts.cpu().numpy().reshape(n, F).astype(np.float64)
    ref = orc.act_batch(cfg, store[0], X, n)
    assert np.max(np.abs(ref)) < 2.0 ** 12
    assert np.array_equal(got, ref), int(np.sum(got != ref))


# ---------------- O10: percentile -------------------------------------------------

@pytest.mark.parametrize("n", [1, 5, 1000, 1001, 32768, 32769, 65536 + 3, 200000, (1 << 20) + 2])
@pytest.mark.parametrize("spread", [False, True])
def test_percentile_bit_exact(n, spread):
    """One workgroup per row (a workspace with only the error word), and rows
    spread over several workgroups (a workspace with room for the per-row
    histograms: taken for n > 32768)."""
    say(f"[percentile] n={n} spread={spread}")
    rng = np.random.default_rng(n)
    rows = 3
    v = rng.normal(size=(rows, n)).astype(np.float32)
    v[1] = np.round(v[1] * 4) / 4            # many ties
    v[2, : n // 2] = -v[2, : n // 2]         # signs
    if n > 4:
        v[2, 1] = -0.0
        v[2, 2] = np.float32(1e-40)          # a subnormal
    dv = to_dev(v)
    out = torch.zeros(rows, dtype=torch.float32, device=DEV)
    wsb = B.percentile_ws_bytes(rows) if spread else 4096
    ws = torch.zeros(wsb, dtype=torch.uint8, device=DEV)
    for alpha in (0.0, 12.5, 50.0, 61.6, 99.0, 100.0):
        B.np_percentile(dv, rows, n, alpha, out, ws, wsb)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), orc.percentile(v, alpha)), alpha
    assert int(ws[:4].view(torch.int32)[0]) == 0
    v[0, n // 2] = np.nan
    B.np_percentile(to_dev(v), rows, n, 50.0, out, ws, wsb)
    assert B.np_device_error(ws) & B.NP_DEVERR_NAN_SCORE


# ---------------- O11: thresholded active set ------------------------------------

@pytest.mark.parametrize("F,k", [(31, 31), (100, 40), (257, 100), (1001, 500), (14336, 5500),
                                 (65535, 8192)])
def test_threshold_active_bit_exact(F, k):
    say(f"[threshold active] F={F} k={k}")
    rows = 5
    rng = np.random.default_rng(F)
    acts = rng.normal(size=(rows, F)).astype(np.float32)
    T = np.array([0.0, 0.25, 0.8, 1.5, 4.0], np.float32)
    acts[1, ::7] = T[1]                      # magnitudes equal to T are kept
    acts[1, 3::7] = -T[1]
    cfg_shape = B.make_shape(1, 64, F, 8, k, k, "f32")
    W_ = (F + 31) // 32
    mask = torch.full((rows * W_,), -7, dtype=torch.int32, device=DEV)
    ids = torch.full((rows * k,), -7, dtype=torch.int32, device=DEV)
    counts = torch.full((rows,), -7, dtype=torch.int32, device=DEV)
    ws = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    B.np_threshold_active(cfg_shape, to_dev(acts), rows, to_dev(T), mask, ids, counts, ws)
    torch.cuda.synchronize()
    ref = orc.threshold_active(acts, T, k)
    gm = mask.cpu().numpy().view(np.uint32).reshape(rows, W_)
    gi = ids.cpu().numpy().reshape(rows, k)
    gc = counts.cpu().numpy()
    assert np.array_equal(gm, ref["mask"]) and np.array_equal(gc, ref["counts"])
    for r in range(rows):
        assert np.array_equal(gi[r][:gc[r]], ref["active_ids"][r][:gc[r]]), r
    err = B.np_device_error(ws)
    assert bool(err & B.NP_DEVERR_OVERFLOW) == ref["overflow"] and not err & B.NP_DEVERR_NAN_SCORE
    acts[2, F // 2] = np.nan
    ws.zero_()
    B.np_threshold_active(cfg_shape, to_dev(acts), rows, to_dev(T), mask, ids, counts, ws)
    assert B.np_device_error(ws) & B.NP_DEVERR_NAN_SCORE


# ---------------- the calibration chain at the full SwiGLU 7B shape --------------

def test_calibration_chain_7b_swiglu():
    """One layer of the SwiGLU 7B shape (d 4096, F 14336, fp16): activations of
    128 calibration tokens on the matrix cores, the percentile T at
    alpha = 61.6 (38.4% of the neurons kept), eq. 1 on a decode token's
    activations, and the thresholded MLP over the resulting set."""
    cfg = W.get("7b_swiglu")
    F, d, n = cfg.d_ffn, cfg.d_model, 128
    say(f"[calibration] 7b_swiglu layer 0: F={F} d={d} n={n}")
    kcap = 8192  # list capacity above the expected 38.4% of F: no overflow
    shape = B.make_shape(1, d, F, cfg.rank, kcap, F, cfg.wdtype, cfg.adtype, "swiglu")
    store = W.storage(cfg, 0, 1)
    X = W.hidden(cfg, n + 1)
    w = to_dev(store[0])
    acts = torch.empty(n * F, dtype=torch.float32, device=DEV)
    B.np_act_batch(shape, w, to_dev(X[:n]), n, acts)
    torch.cuda.synchronize()
    got = acts.cpu().numpy().reshape(n, F)
    rows = [0, 77, n - 1]
    ref = orc.act_batch(cfg, store[0], X[rows], len(rows))
    g, u, sg, su = parts(cfg, store[0], X[rows])
    bound, _ = act_bound(cfg, g, u, sg, su)
    assert np.all(np.abs(got[rows].astype(np.float64) - ref) <= bound)
    # T(alpha) over the whole batch, bit for bit on the GPU's activations
    ws = torch.zeros(B.np_workspace_size(shape), dtype=torch.uint8, device=DEV)
    T = torch.zeros(1, dtype=torch.float32, device=DEV)
    B.np_percentile(acts, 1, n * F, 61.6, T, ws, ws.numel())
    torch.cuda.synchronize()
    assert T.cpu().numpy()[0] == orc.percentile(got.reshape(1, -1), 61.6)[0]
    # eq. 1 on the next token's activations (bit for bit on the GPU's values)
    a1 = torch.empty(F, dtype=torch.float32, device=DEV)
    B.np_act_batch(shape, w, to_dev(X[n]), 1, a1)
    mask = torch.zeros((F + 31) // 32, dtype=torch.int32, device=DEV)
    ids = torch.full((kcap,), -1, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int32, device=DEV)
    B.np_threshold_active(shape, a1, 1, T, mask, ids, cnt, ws)
    torch.cuda.synchronize()
    a1h = a1.cpu().numpy()
    ref = orc.threshold_active(a1h[None], T.cpu().numpy(), kcap)
    c = int(cnt.cpu()[0])
    assert c == ref["counts"][0] and c > 0.25 * F
    assert np.array_equal(ids.cpu().numpy()[:c], ref["active_ids"][0][:c])
    # the thresholded MLP over that set (the layer fully resident: slot = id)
    y = torch.zeros(d, dtype=torch.float16, device=DEV)
    B.np_sparse_mlp_t(shape, 0, to_dev(X[n]), w, ids, c, cnt, T, y, ws)
    torch.cuda.synchronize()
    sel = ids.cpu().numpy()[:c].astype(np.int32)
    Tf = float(T.cpu()[0])
    _, ref64 = orc.sparse_mlp(cfg.with_(layers=1), 0, X[n], store, sel, want_f64=True,
                              threshold=Tf)
    # rows whose |a| lies within the activation bound of T may go either way
    g, u, sg, su = parts(cfg, store[0][sel], X[n])
    bound, a = act_bound(cfg, g[0], u[0], sg[0], su[0])
    near = np.abs(np.abs(a) - Tf) <= bound
    D = np.abs(orc.decode(cfg.wdtype, store[0][sel][near][:, 2 * d:]))
    extra = np.abs(a[near]) @ D if near.any() else 0.0
    got_y = decode_y(orc, cfg.adtype, y.cpu().numpy().view(np.uint16))
    assert np.all(np.abs(got_y - ref64) <= mlp_tolerance(cfg.adtype, ref64) + extra)
    assert B.np_device_error(ws) == 0


# ---------------- calibration + the decode path with thresholds ------------------

@pytest.mark.parametrize("graph", [False, True])
def test_swiglu_centroid_threshold_pipeline(graph):
    """Thresholds from calibrate.thresholds (bit for bit the oracle's
    percentile of the GPU's activations, those within the O9 bound), then the
    decode path with the centroid predictor and the thresholded SwiGLU MLP,
    token by token against the oracle."""
    from paper_2608_22643_amd import calibrate
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny_swiglu").with_(centroid_k=64, feat_dim=128)
    L, d, F, K, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.centroid_k, cfg.k, cfg.capacity
    n = 48
    say(f"[swiglu pipeline] graph={graph}")
    store = W.storage(cfg)
    xc = W.hidden(cfg.with_(seed=cfg.seed + 101), n)
    bufs = Bufs(cfg)
    bufs.reset()
    acts = torch.empty(L * n * F, dtype=torch.float32, device=DEV)
    thr = calibrate.thresholds(cfg, to_dev(store), to_dev(xc), n, 55.0, bufs.ws, acts=acts)
    torch.cuda.synchronize()
    ah = acts.cpu().numpy().reshape(L, n * F)
    Th = thr.cpu().numpy()
    assert np.array_equal(Th, orc.percentile(ah, 55.0))
    for l in range(L):
        rows = [0, n - 1]
        ref = orc.act_batch(cfg, store[l], xc[rows], 2)
        g, u, sg, su = parts(cfg, store[l], xc[rows])
        bound, _ = act_bound(cfg, g, u, sg, su)
        assert np.all(np.abs(ah[l].reshape(n, F)[rows] - ref) <= bound), l
    T = 6
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T, predictor="centroid",
                          thresholds=thr)
    if graph:
        pipe.capture_graph()
    h = W.hidden(cfg, T)
    bank = W.centroid_bank(cfg)
    st = orc.State(L, F, C)
    for t in range(T):
        pipe.step_graph(t) if graph else pipe.step(t)
        torch.cuda.synchronize()
        logits = pipe.logits.cpu().numpy().reshape(2 * L, K)
        o = orc.centroid_active(logits, bank, L, F, K, k)
        cnt = pipe.active_counts.cpu().numpy()[:L]
        assert np.array_equal(cnt, o["counts"])
        ref = orc.delta_n(t, o["active_ids"], o["counts"], st, C)
        got = pipe.host_lists()
        for l in range(L):
            got["active_slots"][l][cnt[l]:] = -1
        compare_delta(got, ref, L)
        y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            ids = o["active_ids"][l][:cnt[l]].astype(np.int32)
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids, want_f64=True,
                                      threshold=float(Th[l]))
            g, u, sg, su = parts(cfg, store[l][ids], h[t])
            bound, a = act_bound(cfg, g[0], u[0], sg[0], su[0])
            near = np.abs(np.abs(a) - Th[l]) <= bound
            extra = 0.0
            if near.any():
                D = np.abs(orc.decode(cfg.wdtype, store[l][ids][near][:, 2 * d:]))
                extra = np.abs(a[near]) @ D
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64) + extra), (t, l)
    assert pipe.device_error() == 0
