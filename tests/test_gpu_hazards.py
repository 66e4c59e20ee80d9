"""Cross-stream ordering of the overlapped decode step (Sec. 3.5: staging
runs beside compute on a stream of its own).  Two orders must hold whatever
the timing: the MLP of layer l reads its rows only after they are staged
(read after write), and staging for token t + 1 overwrites a victim slot only
after token t's MLPs have read it (write after read).  A fixed-length delay
kernel (a bounded clock spin that always exits) is put on the side stream
before each token's staging, or on the main stream before each token's MLPs,
and tokens are enqueued back to back with no host synchronisation between
them (the memcpy path still reads each plan on the host); every token's MLP
outputs, saved by a device copy on the main stream, must match the oracle.
Gather (storage tier in mapped host memory) and memcpy staging, tiny shape in
fp32 (a record read too early or overwritten too soon moves y far beyond the
1e-5 relative bound)."""
import numpy as np
import pytest
import torch

import oracle as orc
from paper_2608_22643_amd import workload as W
from gpu_util import compare_delta, mlp_tolerance, say

pytestmark = pytest.mark.gpu

DELAY_CYCLES = 2_000_000  # about a millisecond of spinning per delay


def delay(stream):
    with torch.cuda.stream(stream):
        torch.cuda._sleep(DELAY_CYCLES)


@pytest.mark.parametrize("where", ["side", "main"])
@pytest.mark.parametrize("staging", ["gather", "memcpy"])
def test_delayed_stream_keeps_results(staging, where):
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("tiny")
    L, d, F, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.k, cfg.capacity
    T = 8
    say(f"[hazard] {staging} delay on {where}")
    pipe = DecodePipeline(cfg, tier="host", staging=staging, overlap=True, tokens=T)
    if where == "side":
        pipe.delay_side = delay
    else:
        pipe.delay_main = delay
    ys = torch.empty((T, L * d), dtype=torch.float32, device="cuda")
    sc = torch.empty((T, L * F), dtype=torch.float32, device="cuda")
    lists = []
    for t in range(T):
        pipe.step(t)
        with torch.cuda.stream(pipe.main):
            ys[t].copy_(pipe.y)
            sc[t].copy_(pipe.scores)
            lists.append({n: v.clone() for n, v in pipe.lists.items()} | {"counts": pipe.counts.clone()})
    torch.cuda.synchronize()
    h = W.hidden(cfg, T)
    store = W.storage(cfg)
    st = orc.State(L, F, C)
    for t in range(T):
        _, ids = orc.select(sc[t].cpu().numpy().reshape(L, F), k)
        ref = orc.delta(t, ids, st, C)
        got = {n: v.cpu().numpy().reshape(L, -1) for n, v in lists[t].items()}
        compare_delta(got, ref, L)
        y = ys[t].cpu().numpy().reshape(L, d).astype(np.float64)
        for l in range(L):
            _, ref64 = orc.sparse_mlp(cfg, l, h[t], store, ids[l], want_f64=True)
            assert np.all(np.abs(y[l] - ref64) <= mlp_tolerance("f32", ref64)), (t, l)
    assert pipe.device_error() == 0
