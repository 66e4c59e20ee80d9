"""Thin ctypes binding of libneuroprefetch (include/neuroprefetch.h).

Argument marshalling only: every function forwards to the C ABI function of
the same name.  Pointers may be passed as ints or as torch tensors (their
data_ptr); streams as ints (hipStream_t) or torch streams.  A non-OK status
raises NPError with the library's detail text.  There is no fallback: if the
HIP library is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libneuroprefetch.so")

(NP_OK, NP_ERR_INVALID_ARG, NP_ERR_CAPACITY, NP_ERR_HIP, NP_ERR_UNSUPPORTED, NP_ERR_STATE,
 NP_ERR_IO) = range(7)
NP_F32, NP_F16, NP_BF16 = 0, 1, 2
DTYPE_CODE = {"f32": NP_F32, "f16": NP_F16, "bf16": NP_BF16}
NP_ACT_RELU, NP_ACT_SWIGLU = 0, 1
ACT_CODE = {"relu": NP_ACT_RELU, "swiglu": NP_ACT_SWIGLU}
NP_DEVERR_NAN_SCORE = 0x1
NP_DEVERR_NOT_RESIDENT = 0x2
NP_DEVERR_STATE = 0x4
NP_DEVERR_SPIN_LIMIT = 0x8
NP_DEVERR_OVERFLOW = 0x10
NP_TOKEN_AUTO = -1  # np_delta: token index from the workspace step counter

# every symbol the header declares
EXPORTS = ("np_status_str", "np_last_error", "np_shape_check", "np_workspace_size",
           "np_state_reset", "np_predict", "np_select", "np_delta", "np_stage_rows",
           "np_stage_gather", "np_sparse_mlp", "np_centroid_select", "np_delta_n",
           "np_sparse_mlp_n", "np_dense_mlp", "np_sparse_mlp_t", "np_act_batch",
           "np_percentile", "np_threshold_active", "np_stage_file", "np_read_records",
           "np_device_error", "np_sparse_mlp_noalloc", "np_sparse_mlp_ids", "np_select_delta")


class NPError(RuntimeError):
    def __init__(self, status: int, fn: str, detail: str):
        super().__init__(f"{fn}: {status_name(status)}: {detail}")
        self.status = status


class np_shape(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("d_ffn", ctypes.c_int32), ("rank", ctypes.c_int32), ("k", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("wdtype", ctypes.c_int32),
                ("adtype", ctypes.c_int32), ("act", ctypes.c_int32)]


class np_state(ctypes.Structure):
    _fields_ = [("slot_of", ctypes.c_void_p), ("neuron_of", ctypes.c_void_p),
                ("last_used", ctypes.c_void_p)]


class np_delta_out(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids", "active_slots", "counts")]


class np_centroid_model(ctypes.Structure):
    _fields_ = [("n_centroids", ctypes.c_int32), ("feat_dim", ctypes.c_int32),
                ("heads", ctypes.c_void_p), ("bank", ctypes.c_void_p)]


class np_stage_plan(ctypes.Structure):
    _fields_ = [("counts", ctypes.c_void_p), ("in_ids", ctypes.c_void_p),
                ("in_slots", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        S = ctypes.POINTER(np_shape)
        L.np_status_str.argtypes = [i32]
        L.np_status_str.restype = ctypes.c_char_p
        L.np_last_error.argtypes = []
        L.np_last_error.restype = ctypes.c_char_p
        L.np_shape_check.argtypes = [S]
        L.np_workspace_size.argtypes = [S, ctypes.POINTER(sz), ctypes.POINTER(sz)]
        L.np_state_reset.argtypes = [S, ctypes.POINTER(np_state), vp, vp, vp]
        L.np_predict.argtypes = [S, vp, vp, vp, vp, vp, vp]
        L.np_select.argtypes = [S, vp, vp, vp, vp, vp]
        L.np_delta.argtypes = [S, i32, vp, ctypes.POINTER(np_state), ctypes.POINTER(np_delta_out),
                               vp, vp]
        L.np_stage_rows.argtypes = [S, ctypes.POINTER(np_stage_plan), i32, i32, vp, vp, vp, sz, vp,
                                    sz, vp, vp, vp]
        L.np_stage_gather.argtypes = [S, ctypes.POINTER(np_delta_out), i32, i32, vp, vp, vp, vp]
        L.np_sparse_mlp.argtypes = [S, i32, vp, vp, vp, i32, vp, vp, vp]
        L.np_device_error.argtypes = [vp, vp, ctypes.POINTER(i32)]
        L.np_sparse_mlp_noalloc.argtypes = [S, i32, vp, vp, vp, i32, vp, vp, vp]
        L.np_sparse_mlp_ids.argtypes = [S, i32, vp, vp, vp, vp, i32, vp, vp, vp]
        L.np_select_delta.argtypes = [S, i32, vp, vp, vp, ctypes.POINTER(np_state),
                                      ctypes.POINTER(np_delta_out), vp, vp]
        L.np_centroid_select.argtypes = [S, ctypes.POINTER(np_centroid_model), vp, vp, vp, vp,
                                         vp, vp, vp, vp]
        L.np_delta_n.argtypes = [S, i32, vp, vp, ctypes.POINTER(np_state),
                                 ctypes.POINTER(np_delta_out), vp, vp]
        L.np_sparse_mlp_n.argtypes = [S, i32, vp, vp, vp, vp, vp, vp, vp]
        L.np_dense_mlp.argtypes = [S, vp, vp, vp, vp, vp]
        L.np_sparse_mlp_t.argtypes = [S, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp]
        L.np_act_batch.argtypes = [S, vp, vp, i32, vp, vp, vp]
        L.np_percentile.argtypes = [vp, i32, ctypes.c_int64, ctypes.c_double, vp, vp,
                                    ctypes.c_size_t, vp]
        L.np_threshold_active.argtypes = [S, vp, i32, vp, vp, vp, vp, vp, vp]
        i64 = ctypes.c_int64
        L.np_stage_file.argtypes = [S, ctypes.POINTER(np_stage_plan), i32, i32, i32, i64, vp, vp,
                                    sz, vp, sz, vp, sz, vp, vp, vp]
        L.np_read_records.argtypes = [i32, i64, i64, vp, i32, vp]
        for f in EXPORTS[2:]:
            getattr(L, f).restype = i32
        _lib = L
    return _lib


def status_name(st: int) -> str:
    try:
        return lib().np_status_str(st).decode()
    except Exception:  # library missing: still produce a message
        return str(st)


def _p(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    raise TypeError(f"cannot pass {type(x)} as a pointer")


def _s(stream) -> int | None:
    if stream is None or isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st: int, fn: str) -> None:
    if st != NP_OK:
        raise NPError(st, fn, lib().np_last_error().decode())


def make_shape(layers, d_model, d_ffn, rank, k, capacity, wdtype, adtype=None,
               act="relu") -> np_shape:
    wd = DTYPE_CODE.get(wdtype, wdtype)
    ad = wd if adtype is None else DTYPE_CODE.get(adtype, adtype)
    return np_shape(layers, d_model, d_ffn, rank, k, capacity, wd, ad, ACT_CODE.get(act, act))


def np_shape_check(shape: np_shape) -> None:
    _check(lib().np_shape_check(ctypes.byref(shape)), "np_shape_check")


def np_workspace_size(shape: np_shape) -> int:
    """Device workspace bytes (np_workspace_sizes gives the pinned host size too)."""
    return np_workspace_sizes(shape)[0]


def np_workspace_sizes(shape: np_shape) -> tuple[int, int]:
    """(device workspace bytes, pinned host bytes for host staging)."""
    n, h = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib().np_workspace_size(ctypes.byref(shape), ctypes.byref(n), ctypes.byref(h)),
           "np_workspace_size")
    return n.value, h.value


def np_state_reset(shape, state: np_state, ws, stream=None, dev_resident=None) -> None:
    _check(lib().np_state_reset(ctypes.byref(shape), ctypes.byref(state), _p(dev_resident),
                                _p(ws), _s(stream)), "np_state_reset")


def np_predict(shape, h, A, B, scores, ws, stream=None) -> None:
    _check(lib().np_predict(ctypes.byref(shape), _p(h), _p(A), _p(B), _p(scores), _p(ws),
                            _s(stream)), "np_predict")


def np_select(shape, scores, mask, active_ids, ws, stream=None) -> None:
    _check(lib().np_select(ctypes.byref(shape), _p(scores), _p(mask), _p(active_ids), _p(ws),
                           _s(stream)), "np_select")


def np_delta(shape, token: int, active_ids, state: np_state, out: np_delta_out, ws,
             stream=None) -> None:
    _check(lib().np_delta(ctypes.byref(shape), int(token), _p(active_ids), ctypes.byref(state),
                          ctypes.byref(out), _p(ws), _s(stream)), "np_delta")


def np_select_delta(shape, token: int, scores, mask, active_ids, state: np_state,
                    out: np_delta_out, ws, stream=None) -> None:
    _check(lib().np_select_delta(ctypes.byref(shape), int(token), _p(scores), _p(mask),
                                 _p(active_ids), ctypes.byref(state), ctypes.byref(out), _p(ws),
                                 _s(stream)), "np_select_delta")


def np_stage_rows(shape, plan: np_stage_plan, layer_begin: int, layer_end: int, host_storage,
                  dev_resident, host_staging, staging_bytes: int, dev_landing, landing_bytes: int,
                  side=None, wait_before=None, layer_ready=None) -> None:
    ev_arr = None
    if layer_ready is not None:
        ev_arr = (ctypes.c_void_p * len(layer_ready))(*[_ev(e) for e in layer_ready])
    _check(lib().np_stage_rows(ctypes.byref(shape), ctypes.byref(plan), int(layer_begin),
                               int(layer_end), _p(host_storage), _p(dev_resident),
                               _p(host_staging), int(staging_bytes), _p(dev_landing),
                               int(landing_bytes), _s(side), _ev(wait_before), ev_arr),
           "np_stage_rows")


def np_stage_file(shape, plan: np_stage_plan, layer_begin: int, layer_end: int, fd: int,
                  file_offset: int, dev_resident, host_staging, staging_bytes: int, io_buffer,
                  io_buffer_bytes: int, dev_landing, landing_bytes: int, side=None,
                  wait_before=None, layer_ready=None) -> None:
    ev_arr = None
    if layer_ready is not None:
        ev_arr = (ctypes.c_void_p * len(layer_ready))(*[_ev(e) for e in layer_ready])
    _check(lib().np_stage_file(ctypes.byref(shape), ctypes.byref(plan), int(layer_begin),
                               int(layer_end), int(fd), int(file_offset), _p(dev_resident),
                               _p(host_staging), int(staging_bytes), _p(io_buffer),
                               int(io_buffer_bytes), _p(dev_landing), int(landing_bytes),
                               _s(side), _ev(wait_before), ev_arr), "np_stage_file")


class HostBuffer:
    """Ordinary page-aligned host memory (an anonymous mapping): the read
    target of direct file I/O.  `ptr` is its address; it lives as long as
    this object."""

    def __init__(self, nbytes: int):
        import mmap

        self.nbytes = int(nbytes)
        self._map = mmap.mmap(-1, max(self.nbytes, 1))
        self.ptr = ctypes.addressof(ctypes.c_char.from_buffer(self._map))

    def data_ptr(self) -> int:
        return self.ptr


def np_read_records(fd: int, file_offset: int, record_bytes: int, ids, n: int, dst) -> None:
    _check(lib().np_read_records(int(fd), int(file_offset), int(record_bytes), _p(ids), int(n),
                                 _p(dst)), "np_read_records")


def np_stage_gather(shape, out: np_delta_out, layer_begin: int, layer_end: int, storage,
                    dev_resident, ws, stream=None) -> None:
    _check(lib().np_stage_gather(ctypes.byref(shape), ctypes.byref(out), int(layer_begin),
                                 int(layer_end), _p(storage), _p(dev_resident), _p(ws),
                                 _s(stream)), "np_stage_gather")


def np_sparse_mlp(shape, layer: int, x, dev_resident, active_slots, n_active: int, y, ws,
                  stream=None) -> None:
    _check(lib().np_sparse_mlp(ctypes.byref(shape), int(layer), _p(x), _p(dev_resident),
                               _p(active_slots), int(n_active), _p(y), _p(ws), _s(stream)),
           "np_sparse_mlp")


def np_sparse_mlp_noalloc(shape, layer: int, x, dev_resident, active_slots, n_active: int, y,
                          dev_error, stream=None) -> None:
    _check(lib().np_sparse_mlp_noalloc(ctypes.byref(shape), int(layer), _p(x), _p(dev_resident),
                                       _p(active_slots), int(n_active), _p(y), _p(dev_error),
                                       _s(stream)), "np_sparse_mlp_noalloc")


def np_sparse_mlp_ids(shape, layer: int, x, dev_resident, active_ids, slot_of, n_active: int, y,
                      ws, stream=None) -> None:
    _check(lib().np_sparse_mlp_ids(ctypes.byref(shape), int(layer), _p(x), _p(dev_resident),
                                   _p(active_ids), _p(slot_of), int(n_active), _p(y), _p(ws),
                                   _s(stream)), "np_sparse_mlp_ids")


def np_centroid_select(shape, model: np_centroid_model, feat, logits, centroid_ids, mask,
                       active_ids, active_counts, ws, stream=None) -> None:
    _check(lib().np_centroid_select(ctypes.byref(shape), ctypes.byref(model), _p(feat),
                                    _p(logits), _p(centroid_ids), _p(mask), _p(active_ids),
                                    _p(active_counts), _p(ws), _s(stream)), "np_centroid_select")


def np_delta_n(shape, token: int, active_ids, active_counts, state: np_state, out: np_delta_out,
               ws, stream=None) -> None:
    _check(lib().np_delta_n(ctypes.byref(shape), int(token), _p(active_ids), _p(active_counts),
                            ctypes.byref(state), ctypes.byref(out), _p(ws), _s(stream)),
           "np_delta_n")


def np_sparse_mlp_n(shape, layer: int, x, dev_resident, active_slots, active_counts, y, ws,
                    stream=None) -> None:
    _check(lib().np_sparse_mlp_n(ctypes.byref(shape), int(layer), _p(x), _p(dev_resident),
                                 _p(active_slots), _p(active_counts), _p(y), _p(ws), _s(stream)),
           "np_sparse_mlp_n")


def np_dense_mlp(shape, weights, x, y, ws, stream=None) -> None:
    _check(lib().np_dense_mlp(ctypes.byref(shape), _p(weights), _p(x), _p(y), _p(ws),
                              _s(stream)), "np_dense_mlp")


def np_sparse_mlp_t(shape, layer: int, x, dev_resident, active_slots, n_active: int,
                    active_counts, thresholds, y, ws, stream=None) -> None:
    _check(lib().np_sparse_mlp_t(ctypes.byref(shape), int(layer), _p(x), _p(dev_resident),
                                 _p(active_slots), int(n_active), _p(active_counts),
                                 _p(thresholds), _p(y), _p(ws), _s(stream)), "np_sparse_mlp_t")


def np_act_batch(shape, weights, x, n: int, acts, ws=None, stream=None) -> None:
    _check(lib().np_act_batch(ctypes.byref(shape), _p(weights), _p(x), int(n), _p(acts), _p(ws),
                              _s(stream)), "np_act_batch")


def percentile_ws_bytes(rows: int) -> int:
    """NP_PERCENTILE_WS_BYTES(rows) of the header."""
    return 4352 + 8208 * int(rows)


def np_percentile(values, rows: int, n: int, alpha: float, out, ws, ws_bytes: int,
                  stream=None) -> None:
    _check(lib().np_percentile(_p(values), int(rows), int(n), float(alpha), _p(out), _p(ws),
                               int(ws_bytes), _s(stream)), "np_percentile")


def np_threshold_active(shape, acts, rows: int, thresholds, mask, active_ids, active_counts, ws,
                        stream=None) -> None:
    _check(lib().np_threshold_active(ctypes.byref(shape), _p(acts), int(rows), _p(thresholds),
                                     _p(mask), _p(active_ids), _p(active_counts), _p(ws),
                                     _s(stream)), "np_threshold_active")


def np_device_error(ws, stream=None) -> int:
    code = ctypes.c_int32(0)
    _check(lib().np_device_error(_p(ws), _s(stream), ctypes.byref(code)), "np_device_error")
    return code.value


def _ev(e) -> int | None:
    """hipEvent_t of a torch.cuda.Event (recorded once so that it exists) or an int."""
    if e is None or isinstance(e, int):
        return e
    return e.cuda_event
