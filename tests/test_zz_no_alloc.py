"""np_sparse_mlp_noalloc (partial sums in the library's own device array, no
workspace) against np_sparse_mlp (workspace) on the same inputs: the same
kernels in the same order, so y must match bit for bit; both are also checked
against the oracle's O5 within the output tolerance.  Two calls in a row, the
second with a smaller input (fewer rows, a smaller d), so a second call that
read what the first left in the shared array would show; a slot outside the
buffer must set NP_DEVERR_NOT_RESIDENT in the caller's error word."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W
from gpu_util import DEV, Bufs, decode_y, mlp_tolerance, say, to_dev

pytestmark = pytest.mark.gpu


def cfg_small(name, L, d, F, r, k, C, dt):
    return W.Config(name, L, d, F, r, k / F, C / F, dt, dt, 4, rho_given=0.9, k_override=k,
                    c_override=C)


# first call: a 7B-shaped layer (d 4096, k 1651, 207 workgroups of partials);
# second call: a smaller shape and fewer rows
BIG = cfg_small("na_big", 2, 4096, 11008, 16, 1651, 5504, "f16")
SMALL = cfg_small("na_small", 2, 1024, 3000, 16, 300, 700, "f16")
WIDE = cfg_small("na_wide", 1, 8192, 4000, 16, 900, 1200, "bf16")


def one_call(cfg, n, seed, err):
    """np_sparse_mlp and np_sparse_mlp_noalloc on the same seeded inputs;
    returns (y_ws bits, y_noalloc bits, oracle f64, adtype)."""
    bufs = Bufs(cfg)
    bufs.reset()
    rng = np.random.default_rng(seed)
    L, F, C, d = cfg.layers, cfg.d_ffn, cfg.capacity, cfg.d_model
    store = W.storage(cfg)
    neuron = np.stack([rng.permutation(F)[:C] for _ in range(L)]).astype(np.int32)
    res = to_dev(np.stack([store[l][neuron[l]] for l in range(L)]))
    h = W.hidden(cfg, 1)[0]
    x = to_dev(h)
    esz = W.ITEMSIZE[cfg.adtype]
    layer = L - 1
    slots = np.sort(rng.choice(C, n, replace=False)).astype(np.int32)
    sl = to_dev(slots)
    y_ws = torch.zeros(d * esz, dtype=torch.uint8, device=DEV)
    y_na = torch.full((d * esz,), 0x5A, dtype=torch.uint8, device=DEV)
    B.np_sparse_mlp(bufs.shape, layer, x, res, sl, n, y_ws, bufs.ws)
    B.np_sparse_mlp_noalloc(bufs.shape, layer, x, res, sl, n, y_na, err)
    torch.cuda.synchronize()
    assert B.np_device_error(bufs.ws) == 0
    ids = neuron[layer][slots]
    _, ref64 = orc.sparse_mlp(cfg, layer, h, store, np.sort(ids), want_f64=True)
    dt = np.float32 if cfg.adtype == "f32" else np.uint16
    return (y_ws.cpu().numpy().view(dt), y_na.cpu().numpy().view(dt), ref64, cfg.adtype)


def check(y_ws, y_na, ref64, adtype):
    assert np.array_equal(y_ws, y_na), "noalloc y differs from np_sparse_mlp's"
    y = decode_y(orc, adtype, y_na)
    assert np.all(np.abs(y - ref64) <= mlp_tolerance(adtype, ref64))


def test_noalloc_matches_workspace_path_twice():
    err = torch.zeros(4, dtype=torch.int32, device=DEV)
    say("[noalloc] big then small")
    check(*one_call(BIG, BIG.k, 5, err))
    check(*one_call(SMALL, 137, 6, err))
    say("[noalloc] d 8192 bf16, then the big shape again with few rows")
    check(*one_call(WIDE, WIDE.k, 7, err))
    check(*one_call(BIG, 3, 8, err))
    torch.cuda.synchronize()
    assert int(err[0].item()) == 0


def test_noalloc_zero_rows_and_bad_slot():
    cfg = SMALL
    bufs = Bufs(cfg)
    bufs.reset()
    d = cfg.d_model
    err = torch.zeros(4, dtype=torch.int32, device=DEV)
    x = torch.zeros(d * 2, dtype=torch.uint8, device=DEV)
    res = torch.zeros(cfg.resident_bytes, dtype=torch.uint8, device=DEV)
    y = torch.full((d * 2,), 0x5A, dtype=torch.uint8, device=DEV)
    sl = to_dev(np.array([0, 1, 2, cfg.capacity + 5], dtype=np.int32))
    B.np_sparse_mlp_noalloc(bufs.shape, 0, x, res, sl, 0, y, err)
    torch.cuda.synchronize()
    assert not y.any(), "zero rows give y = 0"
    B.np_sparse_mlp_noalloc(bufs.shape, 0, x, res, sl, 4, y, err)
    torch.cuda.synchronize()
    assert int(err[0].item()) & B.NP_DEVERR_NOT_RESIDENT
