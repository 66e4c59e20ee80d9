"""CPU oracle of the NeuroPrefetcher decode hot path -- TEST INFRASTRUCTURE.

Plain, slow, fp64 statement of each step (arXiv 2608.22643, Sec. 3.3-3.5),
implemented in ``np_oracle.c`` and wrapped here with ctypes over numpy
arrays.  Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py`` use it; the product path never imports it.  It shares no code
with the HIP library.

Functions (each cites the passage it follows in ``np_oracle.c``):
  predict       O1  z_l = A_l h, scores_l = fp32(B_l z_l)            Sec. 3.1/3.3
  select        O2  top-k by (score desc, id asc), mask + ids         Sec. 3.4
  delta         O3  hits / incoming / LRU victims / slot map update   Sec. 3.4 eqs. 2-3
  stage         O4  record copy storage[l][id] -> resident[l][slot]   Sec. 3.5
  sparse_mlp    O5  sum over active n of eq1(act(g_n, u_n)) downT_n   Sec. 3.3/3.4, eq. 1
  dense_mlp     O6  matrix form over all F neurons (pins O5)
  centroid_logits / centroid_active  O7/O8  heads, argmax, mask AND    Sec. 3.3/3.4
  act_batch     O9  activations of a batch of tokens                  Sec. 3.2
  percentile    O10 nearest-rank alpha-th percentile of |A|           Sec. 3.2
  threshold_active O11 eq. 1 as a mask + ascending ids                eq. 1
  decode/encode     IEEE binary16 / bfloat16 / binary32 <-> float64
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "np_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

DTYPES = {"f32": 0, "f16": 1, "bf16": 2}
ACTS = {"relu": 0, "swiglu": 1}
_ITEMSIZE = {"f32": 4, "f16": 2, "bf16": 2}
_NP_STORAGE = {"f32": np.float32, "f16": np.uint16, "bf16": np.uint16}

_lib = None


def build(force: bool = False) -> str:
    """Compile np_oracle.c into liboracle.so with gcc (plain C, -O2)."""
    if force or not os.path.exists(_LIB_PATH) or (
        os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)
    ):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("NP_ORACLE_LIB_OVERRIDE")  # mutation tests only
        if not path:
            if not os.path.exists(_LIB_PATH):
                build()
            path = _LIB_PATH
        L = ctypes.CDLL(path)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        L.orc_decode.argtypes = [i32, vp, i64, vp]
        L.orc_encode.argtypes = [i32, vp, i64, vp]
        L.orc_predict.argtypes = [i32] * 6 + [vp] * 4
        L.orc_select.argtypes = [i32, i32, i32, vp, vp, vp]
        L.orc_delta.argtypes = [i32, i32, i32, i32, ctypes.c_int32] + [vp] * 11
        L.orc_stage.argtypes = [i32] * 6 + [vp] * 5
        f64 = ctypes.c_double
        L.orc_sparse_mlp.argtypes = [i32] * 5 + [f64, i32] + [vp, vp, vp, i32, vp, vp]
        L.orc_dense_mlp.argtypes = [i32] * 5 + [f64, i32] + [vp, vp, vp, vp]
        L.orc_act_batch.argtypes = [i32] * 5 + [vp, vp, i32, vp]
        L.orc_percentile_rank.argtypes = [i64, f64]
        L.orc_percentile_rank.restype = i64
        L.orc_percentile.argtypes = [vp, i32, i64, f64, vp]
        L.orc_threshold_active.argtypes = [i32] * 3 + [vp] * 5
        L.orc_delta_n.argtypes = [i32, i32, i32, i32, ctypes.c_int32] + [vp] * 12
        L.orc_centroid_logits.argtypes = [i32] * 5 + [vp, vp, vp]
        L.orc_centroid_active.argtypes = [i32] * 4 + [vp] * 6
        for f in ("orc_predict", "orc_select", "orc_delta", "orc_sparse_mlp", "orc_dense_mlp",
                  "orc_delta_n", "orc_centroid_logits", "orc_centroid_active", "orc_act_batch",
                  "orc_percentile", "orc_threshold_active"):
            getattr(L, f).restype = i32
        L.orc_stage.restype = None
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


class OracleError(RuntimeError):
    pass


def decode(dtype: str, bits: np.ndarray) -> np.ndarray:
    """Storage bits (uint16 / uint32 / float32 arrays) -> float64."""
    bits = np.ascontiguousarray(bits)
    out = np.empty(bits.size, dtype=np.float64)
    lib().orc_decode(DTYPES[dtype], _ptr(bits), bits.size, _ptr(out))
    return out.reshape(bits.shape)


def encode(dtype: str, values) -> np.ndarray:
    """float64 -> storage bits with one round-to-nearest-even."""
    v = np.ascontiguousarray(np.asarray(values, dtype=np.float64))
    out = np.empty(v.size, dtype=_NP_STORAGE[dtype])
    lib().orc_encode(DTYPES[dtype], _ptr(v), v.size, _ptr(out))
    return out.reshape(v.shape)


def predict(shape, h, A, B) -> np.ndarray:
    """O1.  shape: object with layers, d_model, d_ffn, rank, wdtype, adtype
    (dtype names).  h [d], A [L'][r][d], B [L'][F][r] as storage bits."""
    L, d, F, r = shape.layers, shape.d_model, shape.d_ffn, shape.rank
    h, A, B = (np.ascontiguousarray(a) for a in (h, A, B))
    assert A.size == L * r * d and B.size == L * F * r and h.size == d
    scores = np.empty((L, F), dtype=np.float32)
    rc = lib().orc_predict(L, d, F, r, DTYPES[shape.wdtype], DTYPES[shape.adtype],
                           _ptr(h), _ptr(A), _ptr(B), _ptr(scores))
    if rc:
        raise OracleError(f"orc_predict failed ({rc})")
    return scores


def select(scores: np.ndarray, k: int):
    """O2.  scores [L'][F] float32 -> (mask [L'][ceil(F/32)] uint32,
    active_ids [L'][k] int32 ascending).  Raises on a NaN score."""
    scores = np.ascontiguousarray(scores, dtype=np.float32)
    L, F = scores.shape
    words = (F + 31) // 32
    mask = np.empty((L, words), dtype=np.uint32)
    ids = np.empty((L, k), dtype=np.int32)
    rc = lib().orc_select(L, F, k, _ptr(scores), _ptr(mask), _ptr(ids))
    if rc == 1:
        raise OracleError("NaN score")
    if rc:
        raise OracleError(f"orc_select failed ({rc})")
    return mask, ids


class State:
    """Residency state of O3: slot_of [L'][F], neuron_of [L'][C],
    last_used [L'][F], all int32, -1 at cold start."""

    def __init__(self, L: int, F: int, C: int):
        self.slot_of = np.full((L, F), -1, dtype=np.int32)
        self.neuron_of = np.full((L, C), -1, dtype=np.int32)
        self.last_used = np.full((L, F), -1, dtype=np.int32)

    def copy(self) -> "State":
        s = State.__new__(State)
        s.slot_of = self.slot_of.copy()
        s.neuron_of = self.neuron_of.copy()
        s.last_used = self.last_used.copy()
        return s


def delta(token: int, active_ids: np.ndarray, state: State, C: int) -> dict:
    """O3 for every layer; updates `state` in place.  Returns dict of
    in_ids, in_slots, ev_ids, ev_slots, hit_ids, active_slots ([L'][k] int32,
    entries beyond the counts are -1) and counts [L'][4]."""
    active_ids = np.ascontiguousarray(active_ids, dtype=np.int32)
    L, k = active_ids.shape
    F = state.slot_of.shape[1]
    out = {n: np.full((L, k), -1, dtype=np.int32)
           for n in ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids", "active_slots")}
    out["counts"] = np.zeros((L, 4), dtype=np.int32)
    rc = lib().orc_delta(L, F, C, k, int(token), _ptr(active_ids),
                         _ptr(state.slot_of), _ptr(state.neuron_of), _ptr(state.last_used),
                         _ptr(out["in_ids"]), _ptr(out["in_slots"]), _ptr(out["ev_ids"]),
                         _ptr(out["ev_slots"]), _ptr(out["hit_ids"]), _ptr(out["active_slots"]),
                         _ptr(out["counts"]))
    if rc:
        raise OracleError(f"orc_delta precondition failed ({rc})")
    return out


def delta_n(token: int, active_ids: np.ndarray, active_counts, state: State, C: int) -> dict:
    """O3 with per-layer active counts (the first active_counts[l] entries of
    row l of active_ids); otherwise as delta()."""
    active_ids = np.ascontiguousarray(active_ids, dtype=np.int32)
    active_counts = np.ascontiguousarray(active_counts, dtype=np.int32)
    L, k = active_ids.shape
    assert active_counts.shape == (L,)
    F = state.slot_of.shape[1]
    out = {n: np.full((L, k), -1, dtype=np.int32)
           for n in ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids", "active_slots")}
    out["counts"] = np.zeros((L, 4), dtype=np.int32)
    rc = lib().orc_delta_n(L, F, C, k, int(token), _ptr(active_ids), _ptr(active_counts),
                           _ptr(state.slot_of), _ptr(state.neuron_of), _ptr(state.last_used),
                           _ptr(out["in_ids"]), _ptr(out["in_slots"]), _ptr(out["ev_ids"]),
                           _ptr(out["ev_slots"]), _ptr(out["hit_ids"]), _ptr(out["active_slots"]),
                           _ptr(out["counts"]))
    if rc:
        raise OracleError(f"orc_delta_n precondition failed ({rc})")
    return out


def centroid_logits(heads, feat, H: int, K: int, D: int, wdtype: str, adtype: str) -> np.ndarray:
    """O7: logits [H][K] float32 of the centroid heads ([H][K][D] storage bits)
    on the feature vector ([D] storage bits)."""
    heads, feat = np.ascontiguousarray(heads), np.ascontiguousarray(feat)
    assert heads.size == H * K * D and feat.size == D
    out = np.empty((H, K), dtype=np.float32)
    rc = lib().orc_centroid_logits(H, K, D, DTYPES[wdtype], DTYPES[adtype], _ptr(heads),
                                   _ptr(feat), _ptr(out))
    if rc:
        raise OracleError(f"orc_centroid_logits failed ({rc})")
    return out


def centroid_active(logits: np.ndarray, bank: np.ndarray, L: int, F: int, K: int, k: int) -> dict:
    """O8: centroid ids [2][L'], intersection mask [L'][W], active_ids [L'][k]
    (-1 beyond the count), counts [L'], overflow (a layer had more than k)."""
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    bank = np.ascontiguousarray(bank, dtype=np.uint32)
    W = (F + 31) // 32
    assert logits.shape == (2 * L, K) and bank.size == 2 * L * K * W
    out = {"cids": np.empty((2, L), dtype=np.int32), "mask": np.empty((L, W), dtype=np.uint32),
           "active_ids": np.full((L, k), -1, dtype=np.int32), "counts": np.empty(L, dtype=np.int32)}
    rc = lib().orc_centroid_active(L, F, K, k, _ptr(logits), _ptr(bank), _ptr(out["cids"]),
                                   _ptr(out["mask"]), _ptr(out["active_ids"]), _ptr(out["counts"]))
    if rc == 1:
        raise OracleError("orc_centroid_active: NaN logit")
    if rc not in (0, 3):
        raise OracleError(f"orc_centroid_active failed ({rc})")
    out["overflow"] = rc == 3
    return out


def stage(shape, counts, in_ids, in_slots, storage: np.ndarray, resident: np.ndarray) -> None:
    """O4: resident[l][in_slots] <- storage[l][in_ids] (byte copy, in place)."""
    L, F, C, k, d = shape.layers, shape.d_ffn, shape.capacity, shape.k, shape.d_model
    counts, in_ids, in_slots = (np.ascontiguousarray(a, dtype=np.int32)
                                for a in (counts, in_ids, in_slots))
    assert storage.nbytes == L * F * 3 * d * _ITEMSIZE[shape.wdtype]
    assert resident.nbytes == L * C * 3 * d * _ITEMSIZE[shape.wdtype]
    lib().orc_stage(L, F, C, k, d, DTYPES[shape.wdtype], _ptr(counts), _ptr(in_ids),
                    _ptr(in_slots), _ptr(storage), _ptr(resident))


def _act(shape) -> int:
    return ACTS[getattr(shape, "act", "relu")]


def sparse_mlp(shape, layer: int, x, storage, ids, want_f64: bool = False,
               threshold: float = 0.0):
    """O5 from the storage tier, with the activation ``shape.act`` ("relu"
    when absent) and the eq. 1 threshold.  Returns y (storage bits of
    adtype), and the unrounded float64 sums when want_f64."""
    F, d = shape.d_ffn, shape.d_model
    x = np.ascontiguousarray(x)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    y = np.empty(d, dtype=_NP_STORAGE[shape.adtype])
    y64 = np.empty(d, dtype=np.float64)
    rc = lib().orc_sparse_mlp(F, d, DTYPES[shape.wdtype], DTYPES[shape.adtype], _act(shape),
                              float(threshold), int(layer), _ptr(x), _ptr(storage), _ptr(ids),
                              ids.size, _ptr(y), _ptr(y64))
    if rc:
        raise OracleError(f"orc_sparse_mlp failed ({rc})")
    return (y, y64) if want_f64 else y


def dense_mlp(shape, layer: int, x, storage, want_f64: bool = False, threshold: float = 0.0):
    """O6: the dense matrix-form MLP over all F neurons (activation and
    threshold as in sparse_mlp)."""
    F, d = shape.d_ffn, shape.d_model
    x = np.ascontiguousarray(x)
    y = np.empty(d, dtype=_NP_STORAGE[shape.adtype])
    y64 = np.empty(d, dtype=np.float64)
    rc = lib().orc_dense_mlp(F, d, DTYPES[shape.wdtype], DTYPES[shape.adtype], _act(shape),
                             float(threshold), int(layer), _ptr(x), _ptr(storage), _ptr(y),
                             _ptr(y64))
    if rc:
        raise OracleError(f"orc_dense_mlp failed ({rc})")
    return (y, y64) if want_f64 else y


def act_batch(shape, weights, x, n: int) -> np.ndarray:
    """O9: activations [n][F] (float64, unrounded) of one layer's records
    ``weights`` ([F][3d] storage bits) over the tokens ``x`` ([n][d])."""
    F, d = shape.d_ffn, shape.d_model
    weights, x = np.ascontiguousarray(weights), np.ascontiguousarray(x)
    assert weights.size == F * 3 * d and x.size == n * d
    out = np.empty((n, F), dtype=np.float64)
    rc = lib().orc_act_batch(F, d, DTYPES[shape.wdtype], DTYPES[shape.adtype], _act(shape),
                             _ptr(weights), _ptr(x), int(n), _ptr(out))
    if rc:
        raise OracleError(f"orc_act_batch failed ({rc})")
    return out


def percentile_rank(n: int, alpha: float) -> int:
    """m = ceil(alpha * n / 100) in double, clamped to [1, n] (O10)."""
    return int(lib().orc_percentile_rank(int(n), float(alpha)))


def percentile(values: np.ndarray, alpha: float) -> np.ndarray:
    """O10: per row of ``values`` ([rows][n] float32), the nearest-rank
    alpha-th percentile of the magnitudes, as float32 [rows]."""
    v = np.ascontiguousarray(values, dtype=np.float32)
    v2 = v.reshape(-1, v.shape[-1]) if v.ndim > 1 else v.reshape(1, -1)
    out = np.empty(v2.shape[0], dtype=np.float32)
    rc = lib().orc_percentile(_ptr(v2), v2.shape[0], v2.shape[1], float(alpha), _ptr(out))
    if rc:
        raise OracleError(f"orc_percentile failed ({rc})")
    return out


def threshold_active(acts: np.ndarray, thresholds, k: int) -> dict:
    """O11: eq. 1 as a mask.  acts [rows][F] float32, thresholds [rows]
    float32 -> mask [rows][W] uint32, active_ids [rows][k] (-1 past the
    count), counts [rows], overflow (some row had more than k)."""
    a = np.ascontiguousarray(acts, dtype=np.float32)
    rows, F = a.shape
    t = np.ascontiguousarray(np.broadcast_to(np.asarray(thresholds, dtype=np.float32), (rows,)))
    W = (F + 31) // 32
    mask = np.empty((rows, W), dtype=np.uint32)
    ids = np.full((rows, k), -1, dtype=np.int32)
    counts = np.empty(rows, dtype=np.int32)
    rc = lib().orc_threshold_active(rows, F, int(k), _ptr(a), _ptr(t), _ptr(mask), _ptr(ids),
                                    _ptr(counts))
    if rc not in (0, 3):
        raise OracleError(f"orc_threshold_active failed ({rc})")
    return {"mask": mask, "active_ids": ids, "counts": counts, "overflow": rc == 3}
