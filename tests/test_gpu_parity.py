"""Parity of each HIP step with the CPU oracle, called through the C ABI.

Bars: masks, delta lists, slot maps and resident bytes bit-exact; scores
within the fp32 accumulation bound of the predictor; MLP outputs within the
tolerance of the activation type (fp16 2e-2 absolute, fp32 1e-5 relative,
bf16 max(2e-2, 1 ulp)).  Selection and delta are compared in lockstep: the
oracle's select runs on the GPU's scores, so both take the same integer
decisions from the same fp32 values.
"""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import (DEV, Bufs, compare_delta, decode_y, from_dev, mlp_tolerance, say,
                      score_bound, to_dev)

pytestmark = pytest.mark.gpu


def cfg_small(name, L, d, F, r, k, C, dt, **kw):
    return W.Config(name, L, d, F, r, k / F, C / F, dt, dt, 4, rho_given=0.9, k_override=k,
                    c_override=C, **kw)


SHAPES = {
    "tiny": W.get("tiny"),
    "ragged_f16": cfg_small("ragged_f16", 2, 264, 1000, 24, 100, 300, "f16"),
    "ragged_bf16": cfg_small("ragged_bf16", 3, 520, 777, 40, 50, 60, "bf16"),
    "wide_f16": cfg_small("wide_f16", 2, 5120, 2000, 64, 300, 700, "f16"),
    "wide_bf16": cfg_small("wide_bf16", 2, 8192, 1500, 96, 200, 450, "bf16"),
    "k_eq_c": cfg_small("k_eq_c", 2, 128, 640, 16, 64, 64, "f32"),
    "k_eq_f": cfg_small("k_eq_f", 2, 64, 96, 8, 96, 96, "f32"),
    "k_one": cfg_small("k_one", 2, 64, 333, 8, 1, 5, "f32"),
    # wide layers: the per-layer kernels size their workgroups by F
    "f_11001": cfg_small("f_11001", 2, 64, 11001, 8, 1650, 5000, "f16"),
    "f_20000": cfg_small("f_20000", 2, 64, 20000, 16, 2500, 6000, "bf16"),
    "f_max": cfg_small("f_max", 1, 64, 65535, 8, 8192, 8192, "f32"),
    # the largest d and r the shape check accepts: 16-bit d 16384 with r 1024
    # (the sparse MLP on 16 waves of two-vector slices, 2-row rounds), fp32
    # d 8192 with r 512
    "d_max_f16": cfg_small("d_max_f16", 2, 16384, 1000, 1024, 100, 200, "f16"),
    "d_max_f32": cfg_small("d_max_f32", 2, 8192, 700, 512, 64, 150, "f32"),
}


@pytest.mark.parametrize("mfma", ["0", "1"])
@pytest.mark.parametrize("name", list(SHAPES))
def test_predict(name, mfma, monkeypatch):
    """Both predictor paths: the per-lane dot products (default) and the
    matrix-core kernels (NP_PREDICT_MFMA=1), against O1 within the fp32
    accumulation bound; ragged d and r (tails of the 32-element steps)."""
    monkeypatch.setenv("NP_PREDICT_MFMA", mfma)
    cfg = SHAPES[name]
    say(f"[predict] {name} mfma={mfma} L'={cfg.layers} d={cfg.d_model} F={cfg.d_ffn} "
        f"r={cfg.rank}")
    bufs = Bufs(cfg)
    A, Bm = W.predictor(cfg)
    h = W.hidden(cfg, 2)
    dA, dB = to_dev(A), to_dev(Bm)
    for t in range(2):
        dh = to_dev(h[t])
        B.np_predict(bufs.shape, dh, dA, dB, bufs.scores, bufs.ws)
        torch.cuda.synchronize()
        got = from_dev(bufs.scores, np.float32, (cfg.layers, cfg.d_ffn)).astype(np.float64)
        ref = orc.predict(cfg, h[t], A, Bm).astype(np.float64)
        tol = score_bound(cfg, A, Bm, h[t]) + np.abs(ref) * 2.0 ** -23
        assert np.all(np.abs(got - ref) <= tol), np.max(np.abs(got - ref) / tol)


# the widths and ranks of the 7B, 13B and 70B predictors (fewer rows of B),
# and the largest 16-bit shape the check accepts
PREDICT_DYADIC = {
    "w7b": cfg_small("w7b", 2, 4096, 3000, 416, 300, 600, "f16"),
    "w13b": cfg_small("w13b", 2, 5120, 3000, 512, 300, 600, "f16"),
    "w70b": cfg_small("w70b", 2, 8192, 3000, 768, 300, 600, "bf16"),
    "d_max_f16": SHAPES["d_max_f16"],
}


@pytest.mark.parametrize("mfma", ["0", "1"])
@pytest.mark.parametrize("name", list(PREDICT_DYADIC))
def test_predict_dyadic_bit_exact(name, mfma, monkeypatch):
    """Dyadic factors (entries m 2^-3, |m| <= 1) and h in {-1, 0, 1}: z is a
    multiple of 2^-3 below d 2^-3 and every partial sum of a score a
    multiple of 2^-6 below r d 2^-6 <= 2^18, so both predictor paths (the
    matrix-core one splitting z into 16-bit parts) compute every score
    exactly, and the GPU's scores equal O1's bit for bit."""
    monkeypatch.setenv("NP_PREDICT_MFMA", mfma)
    cfg = PREDICT_DYADIC[name].with_(dyadic=True, dyadic_h_range=1)
    assert cfg.rank * cfg.d_model <= 2 ** 24
    say(f"[predict dyadic] {name} mfma={mfma} d={cfg.d_model} r={cfg.rank}")
    bufs = Bufs(cfg)
    A, Bm = W.predictor(cfg)
    h = W.hidden(cfg, 2)
    assert set(np.unique(orc.decode(cfg.adtype, h))) <= {-1.0, 0.0, 1.0}
    dA, dB = to_dev(A), to_dev(Bm)
    for t in range(2):
        B.np_predict(bufs.shape, to_dev(h[t]), dA, dB, bufs.scores, bufs.ws)
        torch.cuda.synchronize()
        got = from_dev(bufs.scores, np.float32, (cfg.layers, cfg.d_ffn))
        ref = orc.predict(cfg, h[t], A, Bm).reshape(cfg.layers, cfg.d_ffn)
        assert np.array_equal(got, ref), (t, int(np.sum(got != ref)))


@pytest.mark.parametrize("scale", [3e2, 1e-4])
@pytest.mark.parametrize("name", ["ragged_f16", "ragged_bf16", "wide_f16"])
def test_predict_mfma_z_range(name, scale, monkeypatch):
    """The matrix-core scores kernel splits the fp32 z into three 16-bit parts
    after scaling each layer by a power of two (binary16): inputs scaled so
    that z is far above and far below 1 keep the scores within the bound."""
    monkeypatch.setenv("NP_PREDICT_MFMA", "1")
    cfg = SHAPES[name]
    say(f"[predict z range] {name} scale={scale}")
    bufs = Bufs(cfg)
    A, Bm = W.predictor(cfg)
    h = orc.encode(cfg.adtype, orc.decode(cfg.adtype, W.hidden(cfg, 1)[0]) * scale)
    B.np_predict(bufs.shape, to_dev(h), to_dev(A), to_dev(Bm), bufs.scores, bufs.ws)
    torch.cuda.synchronize()
    got = from_dev(bufs.scores, np.float32, (cfg.layers, cfg.d_ffn)).astype(np.float64)
    ref = orc.predict(cfg, h, A, Bm).astype(np.float64)
    tol = score_bound(cfg, A, Bm, h) + np.abs(ref) * 2.0 ** -23
    assert np.all(np.abs(got - ref) <= tol), np.max(np.abs(got - ref) / tol)


def run_select(bufs, scores_np):
    bufs.scores.copy_(torch.from_numpy(scores_np.reshape(-1)))
    B.np_select(bufs.shape, bufs.scores, bufs.mask, bufs.ids, bufs.ws)
    torch.cuda.synchronize()
    L = bufs.cfg.layers
    return (from_dev(bufs.mask, np.uint32, (L, bufs.words)),
            from_dev(bufs.ids, np.int32, (L, bufs.cfg.k)))


@pytest.mark.parametrize("name", list(SHAPES))
def test_select_lockstep(name):
    cfg = SHAPES[name]
    say(f"[select] {name} F={cfg.d_ffn} k={cfg.k}")
    bufs = Bufs(cfg)
    rng = np.random.default_rng(11)
    L, F = cfg.layers, cfg.d_ffn
    cases = [rng.normal(size=(L, F)).astype(np.float32),
             # heavy ties, signed zeros, infinities
             rng.choice(np.array([-np.inf, -1.0, -0.0, 0.0, 0.5, 1.0, np.inf], np.float32),
                        size=(L, F)),
             np.zeros((L, F), np.float32),
             rng.integers(-3, 4, size=(L, F)).astype(np.float32)]
    for sc in cases:
        mask, ids = run_select(bufs, sc)
        rmask, rids = orc.select(sc, cfg.k)
        assert np.array_equal(ids, rids)
        assert np.array_equal(mask, rmask)
    assert B.np_device_error(bufs.ws) == 0


def test_select_nan_sets_error_bit():
    cfg = SHAPES["k_one"]
    bufs = Bufs(cfg)
    bufs.reset()
    sc = np.ones((cfg.layers, cfg.d_ffn), np.float32)
    sc[1, 7] = np.nan
    run_select(bufs, sc)
    assert B.np_device_error(bufs.ws) & B.NP_DEVERR_NAN_SCORE


def active_sequence(rng, F, k, T, stay):
    cur = rng.choice(F, k, replace=False)
    seq = [np.sort(cur)]
    for _ in range(T - 1):
        keep = cur[rng.random(k) < stay]
        rest = np.setdiff1d(np.arange(F), keep)
        cur = np.concatenate([keep, rng.choice(rest, k - keep.size, replace=False)])
        seq.append(np.sort(cur))
    return seq


@pytest.mark.parametrize("name", list(SHAPES))
@pytest.mark.parametrize("stay", [0.0, 0.5, 0.9])
def test_delta_sequence(name, stay):
    cfg = SHAPES[name]
    say(f"[delta] {name} k={cfg.k} C={cfg.capacity} stay={stay}")
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(int(stay * 10) + cfg.k)
    L, k = cfg.layers, cfg.k
    seqs = [active_sequence(rng, cfg.d_ffn, k, 12, stay) for _ in range(L)]
    st = orc.State(L, cfg.d_ffn, cfg.capacity)
    for t in range(12):
        A = np.stack([seqs[l][t] for l in range(L)]).astype(np.int32)
        bufs.ids.copy_(torch.from_numpy(A.reshape(-1)))
        B.np_delta(bufs.shape, t, bufs.ids, bufs.state, bufs.out, bufs.ws)
        torch.cuda.synchronize()
        ref = orc.delta(t, A, st, cfg.capacity)
        compare_delta(bufs.host_lists(), ref, L)
        P, Q, U = bufs.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of)
        assert np.array_equal(U, st.last_used)
    assert B.np_device_error(bufs.ws) == 0


def stage_and_check(cfg, mode, staging_records=None):
    """Runs deltas on a random active sequence and stages each token with
    `mode`; compares the whole resident buffer with the oracle's copy."""
    bufs = Bufs(cfg)
    bufs.reset()
    L, k, C, F = cfg.layers, cfg.k, cfg.capacity, cfg.d_ffn
    store = W.storage(cfg)
    rec = cfg.record_bytes
    if mode == "gather_device":
        dstore = to_dev(store)
    else:
        dstore = torch.empty(store.nbytes, dtype=torch.uint8, pin_memory=True)
        dstore.numpy()[:] = store.view(np.uint8).reshape(-1)
    resident = torch.zeros(cfg.resident_bytes, dtype=torch.uint8, device=DEV)
    ref_res = np.zeros(cfg.resident_bytes, np.uint8)
    fd = -1
    if mode == "file":  # the storage tier as a file, read with O_DIRECT when records allow
        import os
        import tempfile

        path = os.path.join(tempfile.mkdtemp(), "storage.bin")
        store.tofile(path)
        direct = rec % 512 == 0
        fd = os.open(path, os.O_RDONLY | (os.O_DIRECT if direct else 0))
        say(f"[stage] file tier {path} direct={direct}")
    if mode in ("memcpy", "file"):
        cap = staging_records or 64
        staging = torch.empty(2 * cap * (rec + 4) + 8192, dtype=torch.uint8, pin_memory=True)
        landing = torch.empty(cap * (rec + 4), dtype=torch.uint8, device=DEV)
        io = B.HostBuffer(cap * (rec + 4))  # direct reads land in ordinary host memory
        pc = torch.empty(L * 4, dtype=torch.int32, pin_memory=True)
        pi = torch.empty(L * k, dtype=torch.int32, pin_memory=True)
        ps = torch.empty(L * k, dtype=torch.int32, pin_memory=True)
        plan = B.np_stage_plan(pc.data_ptr(), pi.data_ptr(), ps.data_ptr())
    rng = np.random.default_rng(5)
    seqs = [active_sequence(rng, F, k, 6, 0.7) for _ in range(L)]
    st = orc.State(L, F, C)
    for t in range(6):
        A = np.stack([seqs[l][t] for l in range(L)]).astype(np.int32)
        bufs.ids.copy_(torch.from_numpy(A.reshape(-1)))
        B.np_delta(bufs.shape, t, bufs.ids, bufs.state, bufs.out, bufs.ws)
        if mode in ("memcpy", "file"):
            torch.cuda.synchronize()
            pc.copy_(bufs.counts)
            pi.copy_(bufs.lists["in_ids"])
            ps.copy_(bufs.lists["in_slots"])
            if mode == "memcpy":
                B.np_stage_rows(bufs.shape, plan, 0, L, dstore, resident, staging,
                                staging.numel(), landing, landing.numel(),
                                torch.cuda.current_stream())
            else:
                B.np_stage_file(bufs.shape, plan, 0, L, fd, 0, resident, staging,
                                staging.numel(), io, io.nbytes, landing, landing.numel(),
                                torch.cuda.current_stream())
        else:
            B.np_stage_gather(bufs.shape, bufs.out, 0, L, dstore, resident, bufs.ws)
        torch.cuda.synchronize()
        ref = orc.delta(t, A, st, C)
        orc.stage(cfg, ref["counts"], ref["in_ids"], ref["in_slots"], store,
                  ref_res.view(store.dtype).reshape(L, C, -1))
        got = resident.cpu().numpy()
        assert np.array_equal(got, ref_res), f"resident bytes differ at token {t}"
    assert B.np_device_error(bufs.ws) == 0
    if fd >= 0:
        import os

        os.close(fd)
        os.remove(path)
    return bufs, resident, store, st


@pytest.mark.parametrize("name", ["tiny", "ragged_f16", "ragged_bf16", "k_eq_c"])
@pytest.mark.parametrize("mode", ["gather_device", "gather_host", "memcpy", "file"])
def test_stage(name, mode):
    cfg = SHAPES[name]
    say(f"[stage] {name} {mode}")
    stage_and_check(cfg, mode)


@pytest.mark.parametrize("records", [1, 3, 1000])
@pytest.mark.parametrize("mode", ["memcpy", "file"])
def test_stage_chunk_invariance(records, mode):
    cfg = SHAPES["ragged_f16"] if mode == "memcpy" else SHAPES["wide_f16"]
    say(f"[stage chunks] {mode} records per chunk {records}")
    stage_and_check(cfg, mode, staging_records=records)


@pytest.mark.parametrize("first_kib,growth", [(1, 100), (1, 150), (64, 100), (8192, 300)])
def test_stage_piece_schedule_invariance(first_kib, growth, monkeypatch):
    """The placed bytes do not depend on how the staging pieces are sized:
    one-record pieces throughout, pieces growing from one record, a fixed
    small size, and a first piece larger than the piece capacity."""
    monkeypatch.setenv("NP_STAGE_FIRST_KIB", str(first_kib))
    monkeypatch.setenv("NP_STAGE_GROWTH_PCT", str(growth))
    say(f"[stage pieces] first {first_kib} KiB, growth {growth}%")
    stage_and_check(SHAPES["ragged_f16"], "memcpy", staging_records=1000)


def test_stage_rows_rejects_small_staging():
    cfg = SHAPES["tiny"]
    bufs = Bufs(cfg)
    pc = np.zeros(cfg.layers * 4, np.int32)
    pi = np.zeros(cfg.layers * cfg.k, np.int32)
    plan = B.np_stage_plan(pc.ctypes.data, pi.ctypes.data, pi.ctypes.data)
    stg = torch.empty(1024, dtype=torch.uint8, pin_memory=True)
    land = torch.empty(1024, dtype=torch.uint8, device=DEV)
    res = torch.empty(cfg.resident_bytes, dtype=torch.uint8, device=DEV)
    with pytest.raises(B.NPError) as e:
        B.np_stage_rows(bufs.shape, plan, 0, cfg.layers, stg, res, stg, stg.numel(), land,
                        land.numel(), torch.cuda.current_stream())
    assert e.value.status == B.NP_ERR_CAPACITY


@pytest.mark.parametrize("name", list(SHAPES))
def test_sparse_mlp(name):
    check_sparse_mlp(SHAPES[name])


# the single-kernel reduction (grid barrier) applies to whole wave slices and
# at least 64 rows; the two-kernel one to every shape: both against the oracle
@pytest.mark.parametrize("name", ["wide_f16", "wide_bf16"])
@pytest.mark.parametrize("fused", ["0", "1"])
def test_sparse_mlp_both_reductions(name, fused, monkeypatch):
    monkeypatch.setenv("NP_MLP_FUSED", fused)
    check_sparse_mlp(SHAPES[name])


def test_sparse_mlp_row_counts():
    """Prefixes of the active list: fewer rows than workgroups, exactly one
    wave of partial rows, and the full list (both reductions' boundaries)."""
    cfg = SHAPES["wide_f16"]
    say(f"[mlp rows] {cfg.name}")
    bufs, resident, store, st = stage_and_check(cfg, "gather_device")
    d, k, esz = cfg.d_model, cfg.k, W.ITEMSIZE[cfg.adtype]
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    slots = bufs.lists["active_slots"].cpu().numpy().reshape(cfg.layers, k)
    neuron_of = st.neuron_of
    y = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    for n in (1, 63, 64, 65, 255, 256, 257, k):
        B.np_sparse_mlp(bufs.shape, 1, x, resident, bufs.lists["active_slots"].data_ptr() + 4 * k,
                        n, y, bufs.ws)
        torch.cuda.synchronize()
        ids = np.sort(neuron_of[1][slots[1][:n]]).astype(np.int32)
        _, ref64 = orc.sparse_mlp(cfg, 1, h, store, ids, want_f64=True)
        got = decode_y(orc, cfg.adtype, y.cpu().numpy())
        assert np.all(np.abs(got - ref64) <= mlp_tolerance(cfg.adtype, ref64)), n
    assert B.np_device_error(bufs.ws) == 0


def check_sparse_mlp(cfg):
    say(f"[mlp] {cfg.name} d={cfg.d_model} k={cfg.k}")
    bufs, resident, store, st = stage_and_check(cfg, "gather_device")
    L, k, d = cfg.layers, cfg.k, cfg.d_model
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    y = torch.zeros(L * d * esz, dtype=torch.uint8, device=DEV)
    slots = bufs.lists["active_slots"]
    for l in range(L):
        B.np_sparse_mlp(bufs.shape, l, x, resident, slots.data_ptr() + 4 * l * k, k,
                        y.data_ptr() + l * d * esz, bufs.ws)
    torch.cuda.synchronize()
    lists = bufs.host_lists()
    ybits = y.cpu().numpy()
    for l in range(L):
        active = np.sort(np.concatenate([lists["hit_ids"][l][:lists["counts"][l][1]],
                                         lists["in_ids"][l][:lists["counts"][l][0]]]))
        _, ref64 = orc.sparse_mlp(cfg, l, h, store, active.astype(np.int32), want_f64=True)
        got = decode_y(orc, cfg.adtype, ybits[l * d * esz:(l + 1) * d * esz])
        tol = mlp_tolerance(cfg.adtype, ref64)
        assert np.all(np.abs(got - ref64) <= tol), (l, np.max(np.abs(got - ref64)))
    assert B.np_device_error(bufs.ws) == 0


def test_sparse_mlp_empty_and_bad_slot():
    cfg = SHAPES["ragged_f16"]
    bufs = Bufs(cfg)
    bufs.reset()
    resident = torch.zeros(cfg.resident_bytes, dtype=torch.uint8, device=DEV)
    x = to_dev(W.hidden(cfg, 1)[0])
    y = torch.full((cfg.d_model,), 7.0, dtype=torch.float16, device=DEV)
    B.np_sparse_mlp(bufs.shape, 0, x, resident, None, 0, y, bufs.ws)
    torch.cuda.synchronize()
    assert torch.all(y == 0)
    assert B.np_device_error(bufs.ws) == 0
    bad = torch.tensor([0, cfg.capacity + 5, -1, 2], dtype=torch.int32, device=DEV)
    B.np_sparse_mlp(bufs.shape, 1, x, resident, bad, 4, y, bufs.ws)
    assert B.np_device_error(bufs.ws) & B.NP_DEVERR_NOT_RESIDENT


def test_dyadic_end_to_end_bit_exact():
    """Dyadic inputs: every sum is exact, so the whole token -- scores, masks,
    delta, resident bytes and MLP output bits -- must match the oracle run
    on its own (no lockstep)."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("dyadic_tiny")
    say(f"[dyadic] {cfg.name}")
    T = 6
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T)
    h = W.hidden(cfg, T)
    A, Bm = W.predictor(cfg)
    store = W.storage(cfg)
    st = orc.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    L, d, F = cfg.layers, cfg.d_model, cfg.d_ffn
    for t in range(T):
        pipe.step(t)
        torch.cuda.synchronize()
        s_ref = orc.predict(cfg, h[t], A, Bm)
        assert np.array_equal(pipe.scores.cpu().numpy().reshape(L, F), s_ref)
        mask, ids = orc.select(s_ref, cfg.k)
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, -1), ids)
        ref = orc.delta(t, ids, st, cfg.capacity)
        compare_delta(pipe.host_lists(), ref, L)
        y = pipe.y.cpu().numpy().reshape(L, d)
        for l in range(L):
            yb = orc.sparse_mlp(cfg, l, h[t], store, ids[l])
            assert np.array_equal(y[l].view(np.uint32), yb.view(np.uint32)), (t, l)
    assert pipe.device_error() == 0


@pytest.mark.parametrize("tier,staging,overlap", [("device", "gather", False),
                                                  ("device", "gather", True),
                                                  ("host", "gather", True),
                                                  ("host", "memcpy", True),
                                                  ("host", "memcpy", False),
                                                  ("file", "file", True),
                                                  ("file", "file", False)])
def test_lockstep_tiny(tier, staging, overlap):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny")
    say(f"[lockstep] tiny tier={tier} staging={staging} overlap={overlap}")
    T = cfg.tokens
    pipe = DecodePipeline(cfg, tier=tier, staging=staging, overlap=overlap, tokens=T)
    h = W.hidden(cfg, T)
    A, Bm = W.predictor(cfg)
    store = W.storage(cfg)
    st = orc.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    L, d, F = cfg.layers, cfg.d_model, cfg.d_ffn
    res_ref = np.zeros((L, cfg.capacity, 3 * d), np.float32)
    for t in range(T):
        pipe.step(t)
        torch.cuda.synchronize()
        scores = pipe.scores.cpu().numpy().reshape(L, F)
        mask, ids = orc.select(scores, cfg.k)
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, -1), ids)
        assert np.array_equal(pipe.mask.cpu().numpy().view(np.uint32).reshape(L, -1), mask)
        ref = orc.delta(t, ids, st, cfg.capacity)
        compare_delta(pipe.host_lists(), ref, L)
        orc.stage(cfg, ref["counts"], ref["in_ids"], ref["in_slots"], store, res_ref)
        got_res = pipe.resident.cpu().numpy().view(np.float32).reshape(res_ref.shape)
        occupied = st.neuron_of >= 0  # slots never written hold no defined bytes
        assert np.array_equal(got_res[occupied], res_ref[occupied])
        y = pipe.y.cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64))
    # a token past the pipeline's hidden states is refused before anything
    # is enqueued (its row of h does not exist)
    for bad in (T, -1):
        with pytest.raises(IndexError):
            pipe.step(bad)
    assert pipe.device_error() == 0


@pytest.mark.parametrize("name,overlap", [("tiny", True), ("tiny", False),
                                          ("dyadic_tiny", True)])
def test_graph_replay_matches_eager(name, overlap):
    """A captured decode step replayed per token (token index from the device
    step counter, x from a fixed buffer) gives bit for bit what the eager step
    gives, on every replay, with eager work and synchronisation between the
    replays; both follow the oracle's delta in lockstep."""
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get(name)
    T = min(cfg.tokens, 8)
    say(f"[graph] {name} overlap={overlap} tokens={T}")
    eager = DecodePipeline(cfg, tier="device", staging="gather", overlap=overlap, tokens=T)
    graph = DecodePipeline(cfg, tier="device", staging="gather", overlap=overlap, tokens=T)
    graph.capture_graph()
    st = orc.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    L = cfg.layers
    for t in range(T):
        eager.step(t)
        graph.step_graph(t)
        torch.cuda.synchronize()
        _ = (torch.arange(4096, device="cuda", dtype=torch.float32) * t).sum().item()
        for a in ("scores", "mask", "active_ids", "y", "counts"):
            ga, ea = getattr(graph, a), getattr(eager, a)
            assert torch.equal(ga.view(torch.uint8), ea.view(torch.uint8)), (t, a)
        for (gs, es) in zip(graph.host_state(), eager.host_state()):
            assert np.array_equal(gs, es), t
        gl, el = graph.host_lists(), eager.host_lists()
        ids = graph.active_ids.cpu().numpy().reshape(L, -1)
        ref = orc.delta(t, ids, st, cfg.capacity)
        compare_delta(gl, ref, L)
        compare_delta(el, ref, L)
        occupied = torch.from_numpy(np.repeat(st.neuron_of.reshape(-1) >= 0, cfg.record_bytes))
        assert torch.equal(graph.resident.cpu()[occupied], eager.resident.cpu()[occupied]), t
    with pytest.raises(IndexError):  # the pipeline holds T rows of h: one more would read past them
        graph.step_graph(T)
    assert graph.device_error() == 0 and eager.device_error() == 0
