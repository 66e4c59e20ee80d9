"""Pins of oracle O4 (staging) and O5/O6 (sparse and dense MLP).

References: numpy dense products on the decoded records (the all-active
sparse MLP must equal the dense MLP), the closed form for a single active
row, order invariance, a dyadic input that makes every sum exact, and
byte equality of staged records.
"""
import numpy as np
import pytest


def small_cfg(wl, wdtype, L=3, d=64, F=48, dyadic=False, k=12, C=24):
    return wl.Config("t", L, d, F, 8, k / F, C / F, wdtype, wdtype, 4, rho_given=0.9,
                     dyadic=dyadic, dyadic_w_range=3, dyadic_h_range=4)


def dense_numpy(orc, cfg, store, layer, x):
    rec = orc.decode(cfg.wdtype, store[layer])            # [F][3d]
    d = cfg.d_model
    G, U, D = rec[:, :d], rec[:, d:2 * d], rec[:, 2 * d:]
    xv = orc.decode(cfg.adtype, x)
    act = np.maximum(G @ xv, 0.0) * (U @ xv)
    return D.T @ act, G, U, D, xv


@pytest.mark.parametrize("wdtype", ["f32", "f16", "bf16"])
def test_all_active_sparse_equals_dense(orc, wl, wdtype):
    cfg = small_cfg(wl, wdtype)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    for layer in range(cfg.layers):
        ids = np.arange(cfg.d_ffn, dtype=np.int32)
        y, y64 = orc.sparse_mlp(cfg, layer, x, store, ids, want_f64=True)
        yd, yd64 = orc.dense_mlp(cfg, layer, x, store, want_f64=True)
        ref, G, U, D, xv = dense_numpy(orc, cfg, store, layer, x)
        scale = np.abs(D.T) @ (np.abs(G @ xv) * np.abs(U @ xv)) + 1e-300
        assert np.all(np.abs(y64 - ref) <= 1e-12 * scale)
        assert np.all(np.abs(yd64 - ref) <= 1e-12 * scale)
        assert np.array_equal(y, yd) or np.max(np.abs(
            orc.decode(cfg.adtype, y) - orc.decode(cfg.adtype, yd))) <= np.max(np.abs(ref)) * 2 ** -7


@pytest.mark.parametrize("wdtype", ["f32", "bf16"])
def test_single_row_closed_form(orc, wl, wdtype):
    cfg = small_cfg(wl, wdtype)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    _, G, U, D, xv = dense_numpy(orc, cfg, store, 1, x)
    for n in (0, 7, cfg.d_ffn - 1):
        _, y64 = orc.sparse_mlp(cfg, 1, x, store, np.array([n], np.int32), want_f64=True)
        g, u = G[n] @ xv, U[n] @ xv
        ref = max(g, 0.0) * u * D[n]
        assert np.allclose(y64, ref, rtol=1e-13, atol=1e-300)


def test_row_order_irrelevant(orc, wl):
    cfg = small_cfg(wl, "f16")
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    rng = np.random.default_rng(0)
    ids = np.sort(rng.choice(cfg.d_ffn, 20, replace=False)).astype(np.int32)
    _, a = orc.sparse_mlp(cfg, 2, x, store, ids, want_f64=True)
    _, b = orc.sparse_mlp(cfg, 2, x, store, rng.permutation(ids).astype(np.int32), want_f64=True)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-14)


def test_dyadic_exact(orc, wl):
    cfg = small_cfg(wl, "f32", d=128, F=64, dyadic=True)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    ids = np.array([1, 5, 9, 33, 63], np.int32)
    y, y64 = orc.sparse_mlp(cfg, 0, x, store, ids, want_f64=True)
    rec = orc.decode("f32", store[0])
    d = cfg.d_model
    xv = orc.decode("f32", x)
    # exact integer arithmetic in units of 2^-18
    Gi = np.rint(rec[:, :d] * 64).astype(np.int64)
    Ui = np.rint(rec[:, d:2 * d] * 64).astype(np.int64)
    Di = np.rint(rec[:, 2 * d:] * 64).astype(np.int64)
    xi = np.rint(xv).astype(np.int64)
    acc = np.zeros(d, np.int64)
    for n in ids:
        g, u = int(Gi[n] @ xi), int(Ui[n] @ xi)
        acc += max(g, 0) * u * Di[n]
    assert np.array_equal(y64, acc.astype(np.float64) * 2.0 ** -18)
    assert np.array_equal(y.astype(np.float64), acc.astype(np.float64) * 2.0 ** -18)


def test_stage_byte_copy(orc, wl):
    cfg = small_cfg(wl, "bf16")
    store = wl.storage(cfg)
    resident = np.zeros((cfg.layers, cfg.capacity, 3 * cfg.d_model), np.uint16)
    L, k = cfg.layers, cfg.k
    counts = np.zeros((L, 4), np.int32)
    in_ids = np.full((L, k), -1, np.int32)
    in_slots = np.full((L, k), -1, np.int32)
    rng = np.random.default_rng(4)
    for l in range(L):
        n = int(rng.integers(0, k + 1))
        counts[l, 0] = n
        in_ids[l, :n] = np.sort(rng.choice(cfg.d_ffn, n, replace=False))
        in_slots[l, :n] = np.sort(rng.choice(cfg.capacity, n, replace=False))
    orc.stage(cfg, counts, in_ids, in_slots, store, resident)
    for l in range(L):
        filled = set()
        for j in range(counts[l, 0]):
            assert np.array_equal(resident[l, in_slots[l, j]], store[l, in_ids[l, j]])
            filled.add(int(in_slots[l, j]))
        for s in range(cfg.capacity):
            if s not in filled:
                assert not resident[l, s].any()
