"""Pins of oracle O1 (low-rank predictor, z_l = A_l h, s_l = fp32(B_l z_l)).

Independent references: the associativity identity s = (B_l A_l) h evaluated
as one dense product in numpy, the special case r = d with A = I (a plain
GEMV), and a dyadic input for which every sum is exact.
"""
import numpy as np
import pytest


def small_cfg(wl, wdtype="f32", adtype="f32", L=3, d=64, F=96, r=16, dyadic=False):
    return wl.Config("t", L, d, F, r, 0.25, 0.5, wdtype, adtype, 4, rho_given=0.9,
                     dyadic=dyadic, dyadic_h_range=4)


@pytest.mark.parametrize("wdtype", ["f32", "f16", "bf16"])
def test_predict_equals_dense_product(orc, wl, wdtype):
    cfg = small_cfg(wl, wdtype=wdtype, adtype=wdtype)
    A, B = wl.predictor(cfg)
    h = wl.hidden(cfg, 3)
    for t in range(3):
        s = orc.predict(cfg, h[t], A, B)
        Ad, Bd = orc.decode(cfg.wdtype, A), orc.decode(cfg.wdtype, B)
        hd = orc.decode(cfg.adtype, h[t])
        for l in range(cfg.layers):
            W = Bd[l] @ Ad[l]                    # F x d, associativity
            ref = W @ hd
            bound = np.abs(Bd[l]) @ (np.abs(Ad[l]) @ np.abs(hd))
            err = np.abs(s[l].astype(np.float64) - ref)
            # one fp32 rounding of the oracle plus fp64 rounding of both sides
            assert np.all(err <= np.abs(ref) * 2.0 ** -24 + bound * 1e-13), (l, err.max())


def test_predict_identity_factor_is_gemv(orc, wl):
    cfg = small_cfg(wl, L=2, d=32, F=80, r=32)
    A = np.zeros((2, 32, 32), np.float32)
    A[:] = np.eye(32, dtype=np.float32)
    _, B = wl.predictor(cfg)
    h = wl.hidden(cfg, 1)[0]
    s = orc.predict(cfg, h, A, B)
    for l in range(2):
        ref = (B[l].astype(np.float64) @ h.astype(np.float64)).astype(np.float32)
        assert np.array_equal(s[l], ref)


def test_predict_dyadic_exact(orc, wl):
    cfg = small_cfg(wl, wdtype="f16", adtype="f16", d=128, F=200, r=24, dyadic=True)
    A, B = wl.predictor(cfg)
    h = wl.hidden(cfg, 2)
    for t in range(2):
        s = orc.predict(cfg, h[t], A, B)
        Ad, Bd = orc.decode("f16", A), orc.decode("f16", B)
        hd = orc.decode("f16", h[t])
        # all values are small multiples of powers of two: fp64 is exact
        ref = np.einsum("lfr,lrd,d->lf", Bd, Ad, hd)
        assert np.array_equal(s.astype(np.float64), ref)


def test_predict_layers_are_independent(orc, wl):
    cfg = small_cfg(wl)
    A, B = wl.predictor(cfg)
    h = wl.hidden(cfg, 1)[0]
    s0 = orc.predict(cfg, h, A, B)
    A2 = A.copy()
    A2[1] *= 2.0
    s1 = orc.predict(cfg, h, A2, B)
    assert np.array_equal(s0[0], s1[0]) and np.array_equal(s0[2], s1[2])
    assert np.allclose(s1[1], 2 * s0[1], rtol=1e-6)
