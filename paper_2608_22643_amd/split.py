"""Dense/sparse split of the layers (Sec. 3.1; Sec. 4, dense/sparse
partitioning): the first d layers keep their MLP weights resident and run
dense, the remaining ones keep a row buffer of K_max = C neurons each.  The
operating point d* is the largest dense prefix that still fits the device
memory budget together with the sparse suffix's row buffers and the weights
that stay resident regardless of the split (predictor, attention, embeddings,
...), passed in as `fixed_bytes`.  Host arithmetic only.
"""
from __future__ import annotations


def resident_bytes(d: int, n_layers: int, layer_bytes: int, buffer_bytes: int,
                   fixed_bytes: int) -> int:
    """Device bytes with a dense prefix of d of the n_layers MLP layers."""
    if not 0 <= d <= n_layers:
        raise ValueError(f"dense prefix {d} outside [0, {n_layers}]")
    return fixed_bytes + d * layer_bytes + (n_layers - d) * buffer_bytes


def dense_prefix(budget_bytes: int, n_layers: int, layer_bytes: int, buffer_bytes: int,
                 fixed_bytes: int = 0, min_dense: int = 1) -> int:
    """d*: the largest d in [min_dense, n_layers] whose resident bytes fit
    budget_bytes.  A dense layer holds all F records and a buffer C of them
    (C <= F), so the footprint grows with d and d* is found in closed form.
    Raises ValueError when even min_dense does not fit (the paper's
    whole-layer fallback is not implemented here)."""
    if buffer_bytes > layer_bytes or min(n_layers, layer_bytes, buffer_bytes) < 0:
        raise ValueError("need 0 <= buffer_bytes <= layer_bytes and n_layers >= 0")
    if resident_bytes(min_dense, n_layers, layer_bytes, buffer_bytes, fixed_bytes) > budget_bytes:
        raise ValueError("the budget does not hold the minimum dense prefix and the buffers")
    if layer_bytes == buffer_bytes:
        return n_layers
    room = budget_bytes - fixed_bytes - n_layers * buffer_bytes
    return min(n_layers, room // (layer_bytes - buffer_bytes))


def for_config(cfg, budget_bytes: int, fixed_bytes: int | None = None, min_dense: int = 1) -> int:
    """d* for a workload configuration: N = L' + 1 layers (layer 0 and the L'
    predicted ones), dense layers of F records, buffers of C records;
    fixed_bytes defaults to the low-rank predictor's factors."""
    rec = cfg.record_bytes
    if fixed_bytes is None:
        w = 4 if cfg.wdtype == "f32" else 2
        fixed_bytes = cfg.layers * cfg.rank * (cfg.d_model + cfg.d_ffn) * w
    return dense_prefix(budget_bytes, cfg.layers + 1, cfg.d_ffn * rec, cfg.capacity * rec,
                        fixed_bytes, min_dense)
