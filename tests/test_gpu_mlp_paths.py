"""The sparse MLP's three reduction paths against the oracle, on shapes that
each path accepts: the two-kernel path (the default), the single kernel
with a partial-sum reduction after a grid barrier (NP_MLP_FUSED=1) and the
single kernel without partial sums (column bands; 16-bit records with whole
wave slices, at most four rows per thread, the grid resident;
NP_MLP_COLSPLIT=1).  Row counts from 0 to the path's
maximum (fewer rows than workgroups, one row per workgroup, ragged), device
counts, SwiGLU with eq. 1 thresholds, a slot outside the buffer, and bit-for-
bit repeatability of each path; workgroups of 4 to 10 waves of one-vector
slices (d 512 to 5120) and of 8 waves of two-vector slices (d 8192); and
dyadic records on every shape and path, where y must equal the oracle's
exactly."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import DEV, Bufs, decode_y, mlp_tolerance, say, to_dev

pytestmark = pytest.mark.gpu


def cfg_small(name, L, d, F, r, k, C, dt, **kw):
    return W.Config(name, L, d, F, r, k / F, C / F, dt, dt, 4, rho_given=0.9, k_override=k,
                    c_override=C, **kw)


# (d, F, k, C): threads = d / 8 per workgroup, bands = d / 16 workgroups,
# at most 4 * threads rows for the column-band kernel
SHAPES = {
    "d512_f16": cfg_small("d512_f16", 2, 512, 3000, 8, 256, 600, "f16"),
    "d1024_bf16": cfg_small("d1024_bf16", 3, 1024, 5000, 16, 512, 1200, "bf16"),
    "d2048_f16": cfg_small("d2048_f16", 2, 2048, 7000, 16, 1000, 2000, "f16"),
    "d4096_bf16": cfg_small("d4096_bf16", 2, 4096, 11008, 16, 1651, 5504, "bf16"),
    # 9 and 10 waves per workgroup: 8-row rounds in four stages
    "d4608_bf16": cfg_small("d4608_bf16", 2, 4608, 5000, 16, 1200, 2000, "bf16"),
    "d5120_f16": cfg_small("d5120_f16", 2, 5120, 6000, 16, 1658, 2600, "f16"),
    # 128-vector slices: 8 waves of two vectors per lane, 4-row rounds
    "d8192_bf16": cfg_small("d8192_bf16", 2, 8192, 6000, 16, 2867, 3200, "bf16"),
}
PATHS = {"colsplit": {"NP_MLP_COLSPLIT": "1"}, "two_kernel": {},
         "fused": {"NP_MLP_FUSED": "1"}}
# further launch rules at the 7B width, checked with dyadic records: two
# rounds of 8 rows (k above 8 x 256), and a small set in 4-row rounds on
# twice the workgroups (fewer than 128 workgroups of 8 rows)
DYADIC_SHAPES = {**SHAPES,
                 "d4096_f16_k3302": cfg_small("d4096_f16_k3302", 1, 4096, 6000, 16, 3302, 4000,
                                              "f16"),
                 "d4096_f16_k550": cfg_small("d4096_f16_k550", 1, 4096, 6000, 16, 550, 4000,
                                             "f16")}


def resident_of(cfg, store, rng):
    L, F, C = cfg.layers, cfg.d_ffn, cfg.capacity
    neuron = np.stack([rng.permutation(F)[:C] for _ in range(L)]).astype(np.int32)
    return to_dev(np.stack([store[l][neuron[l]] for l in range(L)])), neuron


def setup(cfg, seed):
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(seed)
    store = W.storage(cfg)
    res, neuron = resident_of(cfg, store, rng)
    h = W.hidden(cfg, 1)[0]
    return bufs, rng, store, res, neuron, h


@pytest.mark.parametrize("path", list(PATHS))
@pytest.mark.parametrize("name", list(SHAPES))
def test_mlp_paths_row_counts(name, path, monkeypatch):
    for k_, v_ in PATHS[path].items():
        monkeypatch.setenv(k_, v_)
    cfg = SHAPES[name]
    d, k, C = cfg.d_model, cfg.k, cfg.capacity
    bands = d // 16
    say(f"[mlp path] {name} {path}")
    bufs, rng, store, res, neuron, h = setup(cfg, 21)
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    y2 = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    slots = np.sort(rng.choice(C, k, replace=False)).astype(np.int32)
    sl = to_dev(slots)
    for n in sorted({0, 1, 7, bands - 1, bands, bands + 1, k // 2 + 3, k}):
        for l in range(cfg.layers):
            B.np_sparse_mlp(bufs.shape, l, x, res, sl, n, y, bufs.ws)
            B.np_sparse_mlp(bufs.shape, l, x, res, sl, n, y2, bufs.ws)
            torch.cuda.synchronize()
            assert torch.equal(y, y2), (n, l)  # repeatable bit for bit
            _, ref64 = orc.sparse_mlp(cfg, l, h, store, neuron[l][slots[:n]].astype(np.int32),
                                      want_f64=True)
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (n, l)
    assert B.np_device_error(bufs.ws) == 0


@pytest.mark.parametrize("path", list(PATHS))
@pytest.mark.parametrize("name", list(DYADIC_SHAPES))
def test_mlp_paths_dyadic_bit_exact(name, path, monkeypatch):
    """Dyadic records (m 2^-6, |m| <= 1) and x in {-1, 0, 1}: g and u are
    multiples of 2^-6, a of 2^-12 below 2^12 and every partial sum of y a
    multiple of 2^-18 below 2^6, so every sum is exact in fp32 in any order
    and y is the exact value rounded once to nearest even -- on every launch
    shape of the rows kernel (4 to 10 waves of one-vector slices, 8 waves of
    two-vector slices in 4-row rounds, two rounds of 8 rows, a small set in
    4-row rounds), every reduction path and every row
    count, the GPU's y equals the oracle's value for value (the sign of a
    zero aside)."""
    for k_, v_ in PATHS[path].items():
        monkeypatch.setenv(k_, v_)
    cfg = DYADIC_SHAPES[name].with_(dyadic=True, dyadic_w_range=1, dyadic_h_range=1)
    d, k, C = cfg.d_model, cfg.k, cfg.capacity
    bands = d // 16
    say(f"[mlp path dyadic] {name} {path}")
    bufs, rng, store, res, neuron, h = setup(cfg, 24)
    x = to_dev(h)
    xv = orc.decode(cfg.adtype, h)
    assert set(np.unique(xv)) <= {-1.0, 0.0, 1.0}
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    slots = rng.permutation(C)[:k].astype(np.int32)  # any order of slots
    sl = to_dev(slots)
    for l in range(cfg.layers):
        rec = orc.decode(cfg.wdtype, store[l][neuron[l][slots]])
        assert np.all(np.abs(rec) * 64 <= 1) and np.all(rec * 64 == np.round(rec * 64))
        g, u = rec[:, :d] @ xv, rec[:, d:2 * d] @ xv
        a = np.maximum(g, 0) * u
        assert np.max(np.abs(a)) < 2.0 ** 12
        assert np.max(np.abs(a) @ np.abs(rec[:, 2 * d:])) < 2.0 ** 6
    for n in sorted({0, 1, 7, bands - 1, bands, bands + 1, k // 2 + 3, k}):
        for l in range(cfg.layers):
            B.np_sparse_mlp(bufs.shape, l, x, res, sl, n, y, bufs.ws)
            torch.cuda.synchronize()
            ref = orc.sparse_mlp(cfg, l, h, store, neuron[l][slots[:n]].astype(np.int32))
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.array_equal(got, decode_y(orc, cfg.adtype, ref)), (n, l)
    if path == "two_kernel":
        # the device-count form and the allocation-free entry point run the
        # same kernels: the same exact values
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        for n in sorted({1, k // 3, k}):
            cnt = torch.full((cfg.layers,), n, dtype=torch.int32, device=DEV)
            for l in range(cfg.layers):
                ref = decode_y(orc, cfg.adtype,
                               orc.sparse_mlp(cfg, l, h, store, neuron[l][slots[:n]].astype(np.int32)))
                B.np_sparse_mlp_n(bufs.shape, l, x, res, sl, cnt, y, bufs.ws)
                torch.cuda.synchronize()
                assert np.array_equal(decode_y(orc, cfg.adtype, y.cpu().numpy()), ref), ("n", n, l)
                B.np_sparse_mlp_noalloc(bufs.shape, l, x, res, sl, n, y, err)
                torch.cuda.synchronize()
                assert np.array_equal(decode_y(orc, cfg.adtype, y.cpu().numpy()), ref), ("na", n, l)
        assert int(err.item()) == 0
    # eq. 1 on exact activations: a threshold equal to one row's |a| keeps
    # that row (only a magnitude below the threshold is zeroed), one just
    # above it drops the row
    for l in range(cfg.layers):
        rec = orc.decode(cfg.wdtype, store[l][neuron[l][slots]])
        a = np.maximum(rec[:, :d] @ xv, 0) * (rec[:, d:2 * d] @ xv)
        mags = np.unique(np.abs(a[a != 0]))
        t0 = np.float32(mags[len(mags) // 2])
        assert float(t0) == mags[len(mags) // 2]  # exact in fp32
        for thr in (t0, np.nextafter(t0, np.float32(np.inf))):
            T = to_dev(np.full(cfg.layers, thr, np.float32))
            B.np_sparse_mlp_t(bufs.shape, l, x, res, sl, k, None, T, y, bufs.ws)
            torch.cuda.synchronize()
            ref = orc.sparse_mlp(cfg, l, h, store, neuron[l][slots].astype(np.int32),
                                 threshold=float(thr))
            got = decode_y(orc, cfg.adtype, y.cpu().numpy())
            assert np.array_equal(got, decode_y(orc, cfg.adtype, ref)), (l, float(thr))
    assert B.np_device_error(bufs.ws) == 0


@pytest.mark.parametrize("path", list(PATHS))
@pytest.mark.parametrize("name", ["d1024_bf16", "d4096_bf16", "d5120_f16"])
def test_mlp_paths_counts_swiglu_thresholds(name, path, monkeypatch):
    for k_, v_ in PATHS[path].items():
        monkeypatch.setenv(k_, v_)
    cfg = SHAPES[name].with_(act="swiglu")
    L, d, k, C = cfg.layers, cfg.d_model, cfg.k, cfg.capacity
    say(f"[mlp path swiglu] {name} {path}")
    bufs, rng, store, res, neuron, h = setup(cfg, 22)
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    all_slots = [np.sort(rng.choice(C, k, replace=False)).astype(np.int32) for _ in range(L)]
    # thresholds in the widest gap of each layer's activation magnitudes
    T = np.zeros(L, np.float32)
    for l in range(L):
        rec = orc.decode(cfg.wdtype, store[l][neuron[l][all_slots[l]]])
        xv = orc.decode(cfg.adtype, h)
        g, u = rec[:, :d] @ xv, rec[:, d:2 * d] @ xv
        a = np.abs(g / (1 + np.exp(-g)) * u)
        s = np.sort(a)
        j = int(np.argmax(np.diff(s[k // 4:k // 2]))) + k // 4
        T[l] = np.float32((s[j] + s[j + 1]) / 2)
    counts = torch.tensor(rng.integers(0, k + 1, size=L), dtype=torch.int32, device=DEV)
    thr = to_dev(T)
    for l in range(L):
        B.np_sparse_mlp_t(bufs.shape, l, x, res, to_dev(all_slots[l]), k, counts, thr, y, bufs.ws)
        torch.cuda.synchronize()
        n = int(counts[l])
        ids = neuron[l][all_slots[l][:n]].astype(np.int32)
        _, ref64 = orc.sparse_mlp(cfg, l, h, store, ids, want_f64=True, threshold=float(T[l]))
        got = decode_y(orc, cfg.adtype, y.cpu().numpy())
        assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (l, n)
    assert B.np_device_error(bufs.ws) == 0


@pytest.mark.parametrize("path", list(PATHS))
def test_mlp_paths_bad_slot(path, monkeypatch):
    for k_, v_ in PATHS[path].items():
        monkeypatch.setenv(k_, v_)
    cfg = SHAPES["d2048_f16"]
    say(f"[mlp path bad slot] {path}")
    bufs, rng, store, res, neuron, h = setup(cfg, 23)
    y = torch.zeros(cfg.d_model, dtype=torch.float16, device=DEV)
    bad = torch.tensor([0, cfg.capacity + 5, -1, 2] + list(range(3, 200)), dtype=torch.int32,
                       device=DEV)
    B.np_sparse_mlp(bufs.shape, 1, to_dev(h), res, bad, bad.numel(), y, bufs.ws)
    assert B.np_device_error(bufs.ws) & B.NP_DEVERR_NOT_RESIDENT


def test_mlp_multi_round():
    """More active rows than one 8-row round per workgroup (2 to 3 rounds,
    workgroups with different round counts in one launch), and SwiGLU with a
    threshold on a second layer."""
    cfg = cfg_small("d4096_many", 2, 4096, 6000, 16, 4200, 4500, "f16")
    say("[mlp multi-round]")
    bufs, rng, store, res, neuron, h = setup(cfg, 24)
    x = to_dev(h)
    y = torch.zeros(cfg.d_model, dtype=torch.float16, device=DEV)
    y2 = torch.zeros_like(y)
    slots = rng.permutation(cfg.capacity)[:cfg.k].astype(np.int32)
    sl = to_dev(slots)
    for n in (2048, 2049, 2304, 2560, 3000, 4100, 4200):
        B.np_sparse_mlp(bufs.shape, 0, x, res, sl, n, y, bufs.ws)
        B.np_sparse_mlp(bufs.shape, 0, x, res, sl, n, y2, bufs.ws)
        torch.cuda.synchronize()
        assert torch.equal(y, y2), n
        _, ref64 = orc.sparse_mlp(cfg, 0, h, store, neuron[0][slots[:n]].astype(np.int32),
                                  want_f64=True)
        got = decode_y(orc, cfg.adtype, y.cpu().view(torch.uint8).numpy())
        assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), n
    # SwiGLU with a threshold that drops about a third of the rows
    sw = cfg.with_(act="swiglu")
    bufs2 = Bufs(sw)
    bufs2.reset()
    n = 3000
    ids = neuron[1][slots[:n]].astype(np.int32)
    rec = orc.decode(sw.wdtype, store[1][ids])
    xv = orc.decode(sw.adtype, h)
    g, u = rec[:, :4096] @ xv, rec[:, 4096:8192] @ xv
    a = np.sort(np.abs(g / (1 + np.exp(-g)) * u))
    j = int(np.argmax(np.diff(a[n // 4:n // 2]))) + n // 4
    T = np.float32((a[j] + a[j + 1]) / 2)
    thr = to_dev(np.array([0.0, T], np.float32))
    counts = to_dev(np.array([0, n], np.int32))
    B.np_sparse_mlp_t(bufs2.shape, 1, x, res, sl, cfg.k, counts, thr, y, bufs2.ws)
    torch.cuda.synchronize()
    _, ref64 = orc.sparse_mlp(sw, 1, h, store, ids, want_f64=True, threshold=float(T))
    got = decode_y(orc, sw.adtype, y.cpu().view(torch.uint8).numpy())
    assert np.all(np.abs(got - ref64) <= mlp_tolerance(sw.adtype, ref64))
    assert B.np_device_error(bufs.ws) == 0 and B.np_device_error(bufs2.ws) == 0


@pytest.mark.parametrize("name", ["d512_f16", "d4096_bf16", "d5120_f16", "d8192_bf16"])
def test_mlp_ids_form_matches_slots_form(name):
    """np_sparse_mlp_ids (active ids and the layer's slot map, the lookup done
    in the kernel) against np_sparse_mlp on the slots that lookup gives: the
    same rows in the same order, so the same bits; and the oracle.  An id
    outside [0, F) or an id whose slot is -1 is reported as not resident."""
    cfg = SHAPES[name]
    L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
    say(f"[mlp ids form] {name}")
    bufs, rng, store, res, neuron, h = setup(cfg, 25)
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    y2 = torch.full((d * esz,), 0x5A, dtype=torch.uint8, device=DEV)
    for l in range(L):
        slot_of = np.full(F, -1, np.int32)
        slot_of[neuron[l]] = np.arange(C, dtype=np.int32)
        ids = np.sort(rng.choice(neuron[l], k, replace=False)).astype(np.int32)
        for n in sorted({0, 1, 9, k // 3, k}):
            B.np_sparse_mlp(bufs.shape, l, x, res, to_dev(slot_of[ids]), n, y, bufs.ws)
            B.np_sparse_mlp_ids(bufs.shape, l, x, res, to_dev(ids), to_dev(slot_of), n, y2,
                                bufs.ws)
            torch.cuda.synchronize()
            assert torch.equal(y, y2), (l, n)
            _, ref64 = orc.sparse_mlp(cfg, l, h, store, ids[:n], want_f64=True)
            got = decode_y(orc, cfg.adtype, y2.cpu().numpy())
            assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), (l, n)
    assert B.np_device_error(bufs.ws) == 0
    slot_of = np.full(F, -1, np.int32)
    slot_of[neuron[0]] = np.arange(C, dtype=np.int32)
    absent = np.setdiff1d(np.arange(F), neuron[0])[:1]
    for bad in (np.array([0, F + 3], np.int32), absent.astype(np.int32)):
        bufs.reset()
        B.np_sparse_mlp_ids(bufs.shape, 0, x, res, to_dev(bad), to_dev(slot_of), bad.size, y2,
                            bufs.ws)
        assert B.np_device_error(bufs.ws) & B.NP_DEVERR_NOT_RESIDENT
