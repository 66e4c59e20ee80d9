"""Per-layer magnitude thresholds for eq. 1 (Sec. 3.2), calibrated on the GPU.

For each downstream layer l the activations A(i, l) = act(G_l x_i, U_l x_i)
of a batch of calibration tokens are computed on the matrix cores
(np_act_batch), and T(l, alpha) is the nearest-rank alpha-th percentile of
their magnitudes (np_percentile, all layers in one call).  Eq. 1 then
zeroes activations with |a| < T(l, alpha): a fraction just under alpha/100
of the calibration activations.  Every step runs in the HIP library; this
module only sizes buffers and sequences the calls.
"""
from __future__ import annotations

import torch

from . import binding as B
from . import workload as W


def thresholds(cfg: W.Config, storage: torch.Tensor, x: torch.Tensor, n_tokens: int,
               alpha: float, ws: torch.Tensor, stream=None,
               acts: torch.Tensor | None = None) -> torch.Tensor:
    """T(l, alpha) of every layer of `storage` ([L'][F][3d] records of
    cfg.wdtype, device) over the tokens `x` ([n_tokens][d] of cfg.adtype,
    device).  Returns a device float32 tensor [L'].  `acts` ([L'][n][F]
    float32, device) may be passed to keep the activations."""
    L, F, d = cfg.layers, cfg.d_ffn, cfg.d_model
    shape = B.make_shape(L, d, F, cfg.rank, cfg.k, cfg.capacity, cfg.wdtype, cfg.adtype,
                         cfg.act)
    dev = storage.device
    if acts is None:
        acts = torch.empty(L * n_tokens * F, dtype=torch.float32, device=dev)
    assert acts.numel() >= L * n_tokens * F and storage.numel() >= cfg.storage_bytes
    layer_bytes = F * cfg.record_bytes
    for l in range(L):
        B.np_act_batch(shape, storage.data_ptr() + l * layer_bytes, x, n_tokens,
                       acts.data_ptr() + l * n_tokens * F * 4, ws, stream)
    out = torch.empty(L, dtype=torch.float32, device=dev)
    B.np_percentile(acts, L, n_tokens * F, alpha, out, ws, ws.numel() * ws.element_size(), stream)
    return out
