"""Helpers for the GPU tests: device buffers for one shape and direct calls
through the C ABI binding (no pipeline logic), plus tolerance rules."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W

DEV = "cuda:0"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.uint8).reshape(-1).copy()).to(DEV)


def from_dev(t: torch.Tensor, dtype, shape) -> np.ndarray:
    return t.cpu().numpy().view(dtype).reshape(shape)


class Bufs:
    """Device buffers of one shape (state, lists, scores, ids, ws)."""

    def __init__(self, cfg: W.Config):
        self.cfg = cfg
        L, F, C, k, d = cfg.layers, cfg.d_ffn, cfg.capacity, cfg.k, cfg.d_model
        self.shape = B.make_shape(L, d, F, cfg.rank, k, C, cfg.wdtype, cfg.adtype, cfg.act)
        i32 = lambda n: torch.full((n,), -7, dtype=torch.int32, device=DEV)
        self.slot_of, self.neuron_of, self.last_used = i32(L * F), i32(L * C), i32(L * F)
        self.state = B.np_state(self.slot_of.data_ptr(), self.neuron_of.data_ptr(),
                                self.last_used.data_ptr())
        self.names = ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids", "active_slots")
        self.lists = {n: i32(L * k) for n in self.names}
        self.counts = i32(L * 4)
        self.out = B.np_delta_out(*[self.lists[n].data_ptr() for n in self.names],
                                  self.counts.data_ptr())
        self.scores = torch.zeros(L * F, dtype=torch.float32, device=DEV)
        self.words = (F + 31) // 32
        self.mask = i32(L * self.words)
        self.ids = i32(L * k)
        self.ws = torch.zeros(B.np_workspace_size(self.shape), dtype=torch.uint8, device=DEV)
        self.stream = torch.cuda.current_stream()

    def reset(self, resident=None):
        B.np_state_reset(self.shape, self.state, self.ws, self.stream, resident)

    def host_lists(self):
        L, k = self.cfg.layers, self.cfg.k
        d = {n: from_dev(self.lists[n], np.int32, (L, k)) for n in self.names}
        d["counts"] = from_dev(self.counts, np.int32, (L, 4))
        return d

    def host_state(self):
        L, F, C = self.cfg.layers, self.cfg.d_ffn, self.cfg.capacity
        return (from_dev(self.slot_of, np.int32, (L, F)), from_dev(self.neuron_of, np.int32, (L, C)),
                from_dev(self.last_used, np.int32, (L, F)))


def compare_delta(gpu: dict, ref: dict, L: int):
    """Bit-exact comparison of the defined part of every delta list."""
    assert np.array_equal(gpu["counts"], ref["counts"]), (gpu["counts"], ref["counts"])
    for l in range(L):
        c = ref["counts"][l]
        for name, n in (("in_ids", c[0]), ("in_slots", c[0]), ("hit_ids", c[1]),
                        ("ev_ids", c[2]), ("ev_slots", c[2])):
            assert np.array_equal(gpu[name][l][:n], ref[name][l][:n]), (l, name)
    assert np.array_equal(gpu["active_slots"], ref["active_slots"])


def mlp_tolerance(adtype: str, ref64: np.ndarray) -> np.ndarray:
    """Per-element tolerance on the sparse-MLP output.
    fp16: 2e-2 absolute; fp32: 1e-5 relative to max|y|; bf16: max(2e-2, one
    bf16 ulp of |y|)."""
    if adtype == "f16":
        return np.full(ref64.shape, 2e-2)
    if adtype == "f32":
        return np.full(ref64.shape, 1e-5 * max(np.max(np.abs(ref64)), 1e-30))
    a = np.abs(ref64)
    ulp = np.where(a > 0, 2.0 ** (np.floor(np.log2(np.maximum(a, 1e-300))) - 7), 2.0 ** -133)
    return np.maximum(2e-2, ulp)


def decode_y(orc, adtype: str, y_bits: np.ndarray) -> np.ndarray:
    if adtype == "f32":
        return y_bits.view(np.float32).astype(np.float64)
    return orc.decode(adtype, y_bits.view(np.uint16))


def score_bound(cfg, A, Bm, h):
    """fp32 accumulation bound of s = B (A h): (d + r + 2) u sum |B||A||h|."""
    import oracle as orc

    Ad, Bd = orc.decode(cfg.wdtype, A), orc.decode(cfg.wdtype, Bm)
    hd = np.abs(orc.decode(cfg.adtype, h))
    L = cfg.layers
    Ad = np.abs(Ad).reshape(L, cfg.rank, cfg.d_model)
    Bd = np.abs(Bd).reshape(L, cfg.d_ffn, cfg.rank)
    mag = np.stack([Bd[l] @ (Ad[l] @ hd) for l in range(L)])
    return (cfg.d_model + cfg.rank + 2) * 2.0 ** -24 * mag


def check_native_mask(gpu_ids: np.ndarray, ref_scores: np.ndarray, tol: np.ndarray, k: int) -> int:
    """The oracle's own scores (O1, independent of the GPU's) through its own
    top-k (O2) against the GPU's active sets: every id in one set and not
    the other must be a near-tie, its oracle score within twice the layer's
    largest score error bound of the oracle's k-th largest score (a GPU
    score error can move it across the threshold only then).  Returns the
    number of such ids over all layers."""
    import oracle as orc

    _, native = orc.select(ref_scores.astype(np.float32), k)
    n_diff = 0
    for l in range(gpu_ids.shape[0]):
        diff = np.setxor1d(gpu_ids[l], native[l])
        if diff.size == 0:
            continue
        s = ref_scores[l].astype(np.float64)
        kth = np.sort(s)[-k]
        width = 2.0 * float(np.max(tol[l]))
        assert np.all(np.abs(s[diff] - kth) <= width), (l, diff, s[diff], kth, width)
        n_diff += diff.size
    return n_diff
