"""The dyadic variant of the 7B shape end to end, bit for bit, with no
lockstep: 31 downstream layers, d 4096, F 11008, r 416, k 1651, C 5504,
fp16, 8 tokens, in the configuration bench.py times (storage tier in HBM,
gather staging, eager launches on one stream), with the storage tier in
pinned host memory (np_stage_rows in side-stream layer groups) and in a file
(np_stage_file).  MLP weights are m 2^-6
(|m| <= 3), predictor entries m 2^-3 (|m| <= 1) and h in {-1, 0, 1}, so every
sum on the path is exact in fp32 in any order provided |a| < 2^12 for every
active row and sum_n |a_n D_nj| < 2^6 for every column j (then every partial
sum of y is a multiple of 2^-18 below 2^6).  The seed is checked against
those bounds on the oracle's own active sets before the run and moved on when
a bound fails.  The oracle then runs alone (O1 -> O2 -> O3 -> O4 -> O5 on its
own outputs) and every score, mask, id list, delta list, slot map, last_used
entry, the resident bytes (the slots written each token, and every occupied
slot at the end) and every layer's MLP output bits must equal the GPU's."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import workload as W
from gpu_util import compare_delta, say

pytestmark = pytest.mark.gpu

T = 8


POOL = ThreadPoolExecutor(max_workers=16)  # the oracle's C calls run without the GIL


def exact_bounds(cfg, store, h, ids):
    """max |a| and max_j sum_n |a_n D_nj| over the layers of one token.  In
    fp32 (torch, CPU): g and u are multiples of 2^-6 below 2^8 and so exact;
    while the bounds hold, a and the column sums are exact too, and a bound
    that fails still shows as a value at or above it."""
    d = cfg.d_model
    x = torch.from_numpy(h.copy()).view(torch.float16).float()
    amax = ymax = 0.0
    for l in range(cfg.layers):
        rec = torch.from_numpy(store[l, ids[l]]).view(torch.float16).float()
        g, u = rec[:, :d] @ x, rec[:, d:2 * d] @ x
        a = torch.clamp(g, min=0.0) * u
        amax = max(amax, float(a.abs().max()))
        ymax = max(ymax, float((a.abs() @ rec[:, 2 * d:].abs()).max()))
    return amax, ymax


def oracle_ids(cfg, h, A, Bm, t):
    """O1 layer by layer on the thread pool, then O2."""
    one = cfg.with_(layers=1)
    parts = POOL.map(lambda l: orc.predict(one, h[t], A[l], Bm[l]), range(cfg.layers))
    s = np.concatenate(list(parts))
    return s, orc.select(s, cfg.k)


def oracle_mlp(cfg, h, store, ids):
    """O5 of every layer on the thread pool (storage bits of y)."""
    return np.stack(list(POOL.map(lambda l: orc.sparse_mlp(cfg, l, h, store, ids[l]),
                                  range(cfg.layers))))


@pytest.fixture(scope="module")
def dyadic_7b():
    """The first seed whose tokens meet the exactness bounds: its config, the
    pinned storage tier and a uint16 view of it."""
    base = W.get("dyadic_7b")
    L, d, F, k, C = base.layers, base.d_model, base.d_ffn, base.k, base.capacity
    cfg = host = store = None
    for seed in range(4):  # re-seed when an exactness bound fails
        c = base.with_(seed=seed)
        say(f"[dyadic7b] seed {seed}: generating {c.storage_bytes / 1e9:.2f} GB of records")
        hb = torch.empty(c.storage_bytes, dtype=torch.uint8, pin_memory=True)
        W.fill_storage(c, hb.data_ptr())
        st_np = hb.numpy().view(np.uint16).reshape(L, F, 3 * d)
        h = W.hidden(c, T)
        A, Bm = W.predictor(c)
        ok = True
        for t in range(T):
            s, (_, ids) = oracle_ids(c, h, A, Bm, t)
            amax, ymax = exact_bounds(c, st_np, h[t], ids)
            smax = float(np.max(np.abs(s)))
            say(f"[dyadic7b] seed {seed} token {t}: max|s| {smax} max|a| {amax} "
                f"max sum|aD| {ymax:.3f}")
            if not (amax < 2.0 ** 12 and ymax < 2.0 ** 6 and smax * 64 < 2.0 ** 24):
                ok = False
                break
        if ok:
            cfg, host, store = c, hb, st_np
            break
        del hb
    assert cfg is not None, "no seed in 0..3 meets the exactness bounds"
    return cfg, host, store


# the step bench.py times (storage tier in HBM, gather staging, one stream)
# and the step with the storage tier in pinned host memory (np_stage_rows in
# side-stream layer groups, every fourth group gathered by the GPU, MLPs
# enqueued by the helper thread), and in a file read with io_uring
@pytest.mark.parametrize("tier,staging,overlap", [("device", "gather", False),
                                                  ("host", "memcpy", True),
                                                  ("file", "file", True)])
def test_dyadic_7b_end_to_end_bit_exact(dyadic_7b, tier, staging, overlap):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg, host, store = dyadic_7b
    say(f"[dyadic7b] tier={tier} staging={staging} overlap={overlap}")
    pipe = DecodePipeline(cfg, tier=tier, staging=staging, overlap=overlap, tokens=T,
                          host_storage=host)
    try:
        run_and_check(pipe, cfg, store)
    finally:
        pipe.close()  # the file tier's storage file is removed


def run_and_check(pipe, cfg, store):
    L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
    h = W.hidden(cfg, T)
    A, Bm = W.predictor(cfg)
    st = orc.State(L, F, C)
    res_ref = np.zeros((L, C, 3 * d), dtype=np.uint16)
    rec_bytes = cfg.record_bytes
    gpu_res = pipe.resident.view(L, C, rec_bytes)
    for t in range(T):
        say(f"[dyadic7b] token {t}")
        pipe.step(t)
        torch.cuda.synchronize()
        s_ref, (mask, ids) = oracle_ids(cfg, h, A, Bm, t)
        assert np.array_equal(pipe.scores.cpu().numpy().reshape(L, F), s_ref), t
        assert np.array_equal(pipe.mask.cpu().numpy().view(np.uint32).reshape(L, -1), mask), t
        assert np.array_equal(pipe.active_ids.cpu().numpy().reshape(L, k), ids), t
        ref = orc.delta(t, ids, st, C)
        compare_delta(pipe.host_lists(), ref, L)
        P, Q, U = pipe.host_state()
        assert np.array_equal(P, st.slot_of) and np.array_equal(Q, st.neuron_of), t
        assert np.array_equal(U, st.last_used), t
        orc.stage(cfg, ref["counts"], ref["in_ids"], ref["in_slots"], store, res_ref)
        for l in range(L):  # every slot written this token
            n = int(ref["counts"][l][0])
            if n == 0:
                continue
            sl = ref["in_slots"][l][:n]
            got = gpu_res[l][torch.from_numpy(sl.astype(np.int64)).to(gpu_res.device)]
            assert np.array_equal(got.cpu().numpy().view(np.uint16), res_ref[l, sl]), (t, l)
        y = pipe.y.cpu().numpy().view(np.uint16).reshape(L, d)
        yb = oracle_mlp(cfg, h[t], store, ids)
        for l in range(L):
            assert np.array_equal(y[l], yb[l]), (t, l)
    say("[dyadic7b] every occupied slot at the end")
    all_res = pipe.resident.cpu().numpy().view(np.uint16).reshape(L, C, 3 * d)
    occ = st.neuron_of >= 0
    assert np.array_equal(all_res[occ], res_ref[occ])
    assert pipe.device_error() == 0
