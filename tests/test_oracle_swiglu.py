"""Pins of the oracle's SwiGLU activation, the eq. 1 threshold in O5/O6, the
batch activations (O9), the percentile (O10) and the thresholded active set
(O11), each against something other than the oracle itself: numpy dense
products with scipy's logistic function, the closed form sigma(1) = e/(1+e)
and the limits of SiLU, exact dyadic arithmetic (a threshold equal to an
activation), numpy's inverted-CDF percentile and the defining property of
the m-th smallest value, and numpy's flatnonzero."""
import numpy as np
import pytest
from scipy.special import expit


def small_cfg(wl, wdtype, act="swiglu", L=3, d=64, F=48, dyadic=False, k=12, C=24):
    return wl.Config("t", L, d, F, 8, k / F, C / F, wdtype, wdtype, 4, rho_given=0.9,
                     dyadic=dyadic, dyadic_w_range=3, dyadic_h_range=4, act=act)


def parts(orc, cfg, store, layer, x):
    rec = orc.decode(cfg.wdtype, store[layer])  # [F][3d]
    d = cfg.d_model
    G, U, D = rec[:, :d], rec[:, d:2 * d], rec[:, 2 * d:]
    xv = orc.decode(cfg.adtype, x)
    return G @ xv, U @ xv, D, G, U, xv


def act_numpy(act, g, u):
    return g * expit(g) * u if act == "swiglu" else np.maximum(g, 0.0) * u


# ---------------- SwiGLU in O5 / O6 -----------------------------------------

@pytest.mark.parametrize("wdtype", ["f32", "f16", "bf16"])
def test_swiglu_all_active_equals_numpy(orc, wl, wdtype):
    cfg = small_cfg(wl, wdtype)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    for layer in range(cfg.layers):
        g, u, D, G, U, xv = parts(orc, cfg, store, layer, x)
        ref = D.T @ act_numpy("swiglu", g, u)
        scale = np.abs(D.T) @ ((np.abs(G) @ np.abs(xv)) * (np.abs(U) @ np.abs(xv))) + 1e-300
        ids = np.arange(cfg.d_ffn, dtype=np.int32)
        _, y64 = orc.sparse_mlp(cfg, layer, x, store, ids, want_f64=True)
        _, yd64 = orc.dense_mlp(cfg, layer, x, store, want_f64=True)
        assert np.all(np.abs(y64 - ref) <= 1e-12 * scale)
        assert np.all(np.abs(yd64 - ref) <= 1e-12 * scale)


def test_swiglu_single_row_closed_form(orc, wl):
    cfg = small_cfg(wl, "f32")
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    g, u, D, *_ = parts(orc, cfg, store, 2, x)
    for n in (0, 11, cfg.d_ffn - 1):
        _, y64 = orc.sparse_mlp(cfg, 2, x, store, np.array([n], np.int32), want_f64=True)
        assert np.allclose(y64, g[n] / (1.0 + np.exp(-g[n])) * u[n] * D[n], rtol=1e-13,
                           atol=1e-300)


def hand_layer(orc, gvals, d=8):
    """One layer of f32 records whose gate sums over x = e_0 are gvals and
    whose up sums are 1; down rows are zero."""
    F = len(gvals)
    rec = np.zeros((F, 3 * d))
    rec[:, 0] = gvals
    rec[:, d] = 1.0
    x = np.zeros(d)
    x[0] = 1.0
    return orc.encode("f32", rec), orc.encode("f32", x)


def test_silu_closed_forms_and_limits(orc, wl):
    gvals = [0.0, 1.0, -1.0, 40.0, -40.0, 2.0]
    w, x = hand_layer(orc, gvals)
    cfg = small_cfg(wl, "f32", d=8, F=len(gvals))
    a = orc.act_batch(cfg, w, x, 1)[0]
    e = np.e
    assert a[0] == 0.0                                   # SiLU(0) = 0
    assert a[1] == pytest.approx(e / (1.0 + e), rel=1e-15)  # sigma(1) = e / (1 + e)
    assert a[2] == pytest.approx(-1.0 / (1.0 + e), rel=1e-15)
    assert a[3] == pytest.approx(40.0, rel=1e-15)        # SiLU(g) -> g
    assert abs(a[4]) < 1e-15 and a[4] < 0.0              # SiLU(g) -> 0 from below
    assert a[5] - (-2.0 * expit(-2.0)) == pytest.approx(2.0, rel=1e-15)  # SiLU(g)-SiLU(-g)=g
    relu = orc.act_batch(small_cfg(wl, "f32", act="relu", d=8, F=len(gvals)), w, x, 1)[0]
    assert relu.tolist() == [0.0, 1.0, 0.0, 40.0, 0.0, 2.0]


# ---------------- O9 ----------------------------------------------------------

@pytest.mark.parametrize("act", ["relu", "swiglu"])
@pytest.mark.parametrize("wdtype", ["f32", "bf16"])
def test_act_batch_matches_numpy(orc, wl, act, wdtype):
    cfg = small_cfg(wl, wdtype, act=act, F=40)
    store = wl.storage(cfg)
    X = wl.hidden(cfg, 5)
    A = orc.act_batch(cfg, store[1], X, 5)
    for i in range(5):
        g, u, _, G, U, xv = parts(orc, cfg, store, 1, X[i])
        scale = (np.abs(G) @ np.abs(xv)) * (np.abs(U) @ np.abs(xv)) + 1e-300
        assert np.all(np.abs(A[i] - act_numpy(act, g, u)) <= 1e-12 * scale)


# ---------------- eq. 1 in O5 / O6 --------------------------------------------

def dyadic_cfg(wl, act="relu"):
    return small_cfg(wl, "f32", act=act, d=128, F=64, dyadic=True)


def test_threshold_equal_to_an_activation_is_kept(orc, wl):
    # dyadic ReLU layer: every g, u, a and y is exact in double, so the
    # threshold can equal an activation exactly; eq. 1 keeps |a| = T
    cfg = dyadic_cfg(wl)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    g, u, D, *_ = parts(orc, cfg, store, 0, x)
    a = np.maximum(g, 0.0) * u
    mags = np.unique(np.abs(a[a != 0]))
    assert mags.size >= 4
    ids = np.arange(cfg.d_ffn, dtype=np.int32)
    for T in (mags[0], mags[mags.size // 2], mags[-1]):
        keep = np.abs(a) >= T
        ref = D.T @ np.where(keep, a, 0.0)
        _, y64 = orc.sparse_mlp(cfg, 0, x, store, ids, want_f64=True, threshold=float(T))
        _, yd64 = orc.dense_mlp(cfg, 0, x, store, want_f64=True, threshold=float(T))
        assert np.array_equal(y64, ref) and np.array_equal(yd64, ref)
        # O11 on the same (exact) activations keeps the same neurons
        out = orc.threshold_active(a.astype(np.float32)[None], [T], cfg.d_ffn)
        assert np.array_equal(out["active_ids"][0][:out["counts"][0]], np.flatnonzero(keep))


def test_zero_threshold_is_the_identity(orc, wl):
    cfg = small_cfg(wl, "f16")
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    ids = np.array([0, 3, 17, 40], np.int32)
    a = orc.sparse_mlp(cfg, 1, x, store, ids, want_f64=True)[1]
    b = orc.sparse_mlp(cfg, 1, x, store, ids, want_f64=True, threshold=0.0)[1]
    assert np.array_equal(a, b)


def test_threshold_over_all_rows_equals_the_thresholded_set(orc, wl):
    # rows removed by eq. 1 contribute nothing: the thresholded MLP over every
    # row equals the plain MLP over the O11 set (threshold in a wide gap of
    # the magnitudes, so float32 and double decisions agree)
    cfg = small_cfg(wl, "f32", F=96)
    store = wl.storage(cfg)
    x = wl.hidden(cfg, 1)[0]
    g, u, *_ = parts(orc, cfg, store, 2, x)
    a = act_numpy("swiglu", g, u)
    s = np.sort(np.abs(a))
    j = int(np.argmax(np.diff(s[30:70]))) + 30
    T = float(np.float32((s[j] + s[j + 1]) / 2))
    out = orc.threshold_active(a.astype(np.float32)[None], [T], cfg.d_ffn)
    sel = out["active_ids"][0][:out["counts"][0]]
    assert np.array_equal(sel, np.flatnonzero(np.abs(a) >= T))
    ids = np.arange(cfg.d_ffn, dtype=np.int32)
    _, y_thr = orc.sparse_mlp(cfg, 2, x, store, ids, want_f64=True, threshold=T)
    _, y_set = orc.sparse_mlp(cfg, 2, x, store, sel, want_f64=True)
    assert np.allclose(y_thr, y_set, rtol=1e-12, atol=1e-15)


# ---------------- O10 ----------------------------------------------------------

@pytest.mark.parametrize("n", [1, 7, 100, 1001])
def test_percentile_matches_numpy_inverted_cdf(orc, n):
    rng = np.random.default_rng(n)
    v = rng.normal(size=(3, n)).astype(np.float32)
    for alpha in (0.0, 10.0, 33.3, 50.0, 85.0, 99.9, 100.0):
        got = orc.percentile(v, alpha)
        for r in range(3):
            mag = np.abs(v[r]).astype(np.float64)
            ref = np.percentile(mag, alpha, method="inverted_cdf")
            m = orc.percentile_rank(n, alpha)
            # numpy's inverted CDF is the m-th smallest unless alpha*n/100 is
            # within rounding of an integer; the defining property holds always
            assert np.sum(mag < got[r]) < m <= np.sum(mag <= got[r])
            if abs(alpha * n / 100 - round(alpha * n / 100)) > 1e-9:
                assert got[r] == np.float32(ref)


def test_percentile_ties_and_errors(orc):
    v = np.array([[3.0, -1.0, 1.0, 1.0, -1.0, 2.0]], np.float32)
    assert orc.percentile(v, 50.0)[0] == 1.0   # m = 3 of |v| = 1 1 1 1 2 3
    assert orc.percentile(v, 70.0)[0] == 2.0   # m = ceil(4.2) = 5
    assert orc.percentile_rank(6, 0.0) == 1 and orc.percentile_rank(6, 100.0) == 6
    with pytest.raises(orc.OracleError):
        orc.percentile(np.array([[1.0, np.nan]], np.float32), 50.0)
    with pytest.raises(orc.OracleError):
        orc.percentile(v, 100.5)


# ---------------- O11 ----------------------------------------------------------

@pytest.mark.parametrize("F", [31, 32, 100, 257])
def test_threshold_active_matches_numpy(orc, F):
    rng = np.random.default_rng(F)
    acts = rng.normal(size=(4, F)).astype(np.float32)
    T = np.array([0.0, 0.5, 1.0, 3.0], np.float32)
    out = orc.threshold_active(acts, T, F)
    for r in range(4):
        ids = np.flatnonzero(np.abs(acts[r]) >= T[r])
        assert out["counts"][r] == ids.size
        assert np.array_equal(out["active_ids"][r][:ids.size], ids)
        assert np.all(out["active_ids"][r][ids.size:] == -1)
        bits = np.unpackbits(out["mask"][r].view(np.uint8), bitorder="little")[:F].astype(bool)
        assert np.array_equal(bits, np.abs(acts[r]) >= T[r])
        assert not np.unpackbits(out["mask"][r].view(np.uint8), bitorder="little")[F:].any()
    assert not out["overflow"]


def test_threshold_active_capacity_and_nan(orc):
    acts = np.array([[5.0, -4.0, 0.1, 3.0, -2.0, 0.0]], np.float32)
    out = orc.threshold_active(acts, [1.0], 3)
    assert out["overflow"] and out["counts"].tolist() == [3]
    assert out["active_ids"][0].tolist() == [0, 1, 3]
    assert int(out["mask"][0][0]) == 0b011011   # the mask keeps every member
    with pytest.raises(orc.OracleError):
        orc.threshold_active(np.array([[1.0, np.nan]], np.float32), [0.5], 2)
