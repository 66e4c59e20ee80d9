"""Decode-step benchmark of the NeuroPrefetcher hot path on one MI355X.

One step = one decode token through the whole path: np_predict, np_select,
np_delta, staging of the incoming rows and np_sparse_mlp for every downstream
layer.  Inputs are synthetic and already resident in HBM when the timed
region starts (predictor factors, hidden states, and the storage tier the
incoming rows are staged from); the step's own work is timed, nothing is
skipped.  Prints one JSON line.  By default each call is launched from
Python on one stream (--graph 1: the step captured once as a HIP graph and
replayed per token).

Extra measurements in the same run:
  * the same steps replayed from a captured HIP graph ("graph_tok_s", or
    "eager_tok_s" for the eager launches when --graph 1);
  * the sparse-MLP call's average time, from HIP events bracketing each
    token's block of back-to-back calls on their stream, against the HBM
    roofline;
  * a per-step breakdown (predict / select / delta / stage / mlp);
  * the same step with the storage tier in pinned host memory (np_stage_rows
    staging over the host link, the stated tier of the 13B and 70B
    configurations) for 7B, 13B and 70B -- "end_to_end_pinned_host" and
    "host_tier", PCIe-inclusive, never `value`;
  * np_predict on both of its paths (per-lane dot products and matrix cores);
  * the CPU oracle on a bounded sample, on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0

# Hardware byte counters of the two np_sparse_mlp kernels at the 7B shape,
# from two rocprofv3 --pmc passes over this benchmark (FETCH_SIZE, then
# WRITE_SIZE; mean KiB per dispatch), and the same counters for the
# calibration copy (--calib-mib 256: 262144 KiB read and written once).  The
# figures hold only for the kernel sources they were taken on (hash below);
# after any change to those sources "traffic" is reported as null.
MLP_COUNTERS = {
    "config": "7b",
    "sources": ("paper_2608_22643_amd/csrc/np_mlp.hip", "paper_2608_22643_amd/csrc/np_device.hpp"),
    "sha256": "f4501ceab414e882c8e7347a81de167eef7b38ae8efc2dfd73e1f7495d4605cf"
              "9e0e1f0b7a61ef93b9be1fc993a31341e591454ab40b4db720567ea646fc39f8",
    "fetch_kib": {"rows": 19930.0, "reduce": 1681.5},
    "write_kib": {"rows": 3373.6, "reduce": 8.0},
    "copy_fetch_kib": 131088.2, "copy_write_kib": 262144.0, "copy_kib": 262144.0,
}


def mlp_traffic(cfg):
    """HBM bytes per np_sparse_mlp call from the counters above (each counter
    scaled by true bytes / counter for the plain copy), or None when they do
    not apply to this configuration or these kernel sources."""
    import hashlib

    c = MLP_COUNTERS
    if cfg.name != c["config"]:
        return None, None
    h = "".join(hashlib.sha256(open(os.path.join(ROOT, f), "rb").read()).hexdigest()
                for f in c["sources"])
    if h != c["sha256"]:
        return None, None
    rf = c["copy_kib"] / c["copy_fetch_kib"]
    wf = c["copy_kib"] / c["copy_write_kib"]
    detail = {k: {"read_MB": round(c["fetch_kib"][k] * rf * 1024 / 1e6, 2),
                  "write_MB": round(c["write_kib"][k] * wf * 1024 / 1e6, 2)}
              for k in ("rows", "reduce")}
    total = sum((c["fetch_kib"][k] * rf + c["write_kib"][k] * wf) * 1024 for k in ("rows", "reduce"))
    detail["scale"] = {"fetch": round(rf, 4), "write": round(wf, 4)}
    return int(total), detail


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def mlp_bytes_per_launch(cfg) -> int:
    """Algorithmic bytes of one np_sparse_mlp launch: k records of 3d weights,
    k int32 slots, x and y."""
    esz = 4 if cfg.wdtype == "f32" else 2
    return cfg.k * 3 * cfg.d_model * esz + cfg.k * 4 + 2 * cfg.d_model * esz


def predict_bytes(cfg) -> int:
    """Algorithmic bytes of one np_predict (all L' layers): A [L'][r][d] and
    B [L'][F][r] in the weight type, h, and the fp32 scores written."""
    esz = 4 if cfg.wdtype == "f32" else 2
    L, d, F, r = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.rank
    return L * r * d * esz + L * F * r * esz + d * esz + L * F * 4


def trace_marker():
    """A one-element float fill kernel.  In a kernel trace of this script the
    only float fills are these markers; in run order they bracket the steps
    the sparse-MLP roofline is taken on, the empty np_sparse_mlp calls, and
    each np_stage_rows staging window of the host-tier legs (7B, then 70B,
    then 13B; the overlapped mode first)."""
    import torch

    torch.cuda.synchronize()
    torch.empty(1, dtype=torch.float32, device="cuda").fill_(1.0)
    torch.cuda.synchronize()


def timed_graph_steps(pipe, t0, steps):
    """Times `steps` decode tokens replayed from the captured step graph."""
    import torch

    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(steps):
        pipe.step_graph(t0 + i)
    torch.cuda.synchronize()
    return time.perf_counter() - t_start


def timed_steps(pipe, t0, steps, with_mlp_events=True, step_us=None):
    """Times `steps` decode tokens.  With with_mlp_events, one pair of HIP
    events on the main stream brackets each token's block of L' back-to-back
    np_sparse_mlp calls; the mean per call over the timed region is returned
    (gaps between the calls included).  A list passed as step_us receives
    each token's device time, from an event before its np_predict to the end
    of its last np_sparse_mlp (on the same stream)."""
    import torch

    L = pipe.cfg.layers
    evs = starts = None
    if with_mlp_events:
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(steps)]
        if step_us is not None:
            starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(steps):
        if starts:
            starts[i].record(pipe.main)
        pipe.step(t0 + i, mlp_block_events=evs[i] if evs else None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    mlp_us = None
    if evs:
        mlp_us = sum(a.elapsed_time(b) * 1e3 for a, b in evs) / (steps * L)
    if starts:
        step_us.extend(a.elapsed_time(e[1]) * 1e3 for a, e in zip(starts, evs))
    return wall, mlp_us


def mlp_dispatch_floor(pipe, blocks: int = 10) -> dict:
    """np_sparse_mlp with no active rows, L' calls back to back: each call is
    the rows kernel on one workgroup (it writes a zero partial) and the reduce
    kernel, so the span per call is the fixed cost of a call -- two dispatches
    and the boundaries between them.  Each block of calls is queued behind a
    sleep kernel on the calls' stream so that the host's enqueue rate does not
    set the pace; events on that stream bracket the block.  In a kernel trace
    of this script the blocks sit between the third and fourth one-element
    float fills, so the durations the profiler records for the same empty
    dispatches can be set beside this span."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B
    from paper_2608_22643_amd import workload as W

    cfg, m = pipe.cfg, pipe.main
    L, k = cfg.layers, cfg.k
    ybytes = cfg.d_model * W.ITEMSIZE[cfg.adtype]
    slots = pipe.lists["active_slots"].data_ptr()
    spans = []
    trace_marker()
    for _ in range(blocks):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(m):
            torch.cuda._sleep(2_000_000)  # about 1 ms: the block is queued before it ends
        e0.record(m)
        for l in range(L):
            B.np_sparse_mlp(pipe.shape, l, pipe.x_ptr(0), pipe.resident, slots + l * k * 4, 0,
                            pipe.y.data_ptr() + l * ybytes, pipe.ws, m)
        e1.record(m)
        e1.synchronize()
        spans.append(e0.elapsed_time(e1) * 1e3 / L)
    trace_marker()
    if pipe.device_error():
        raise RuntimeError(f"empty np_sparse_mlp calls: device error word {pipe.device_error():#x}")
    return {"us_per_call": round(float(np.median(spans)), 3),
            "min_us_per_call": round(float(np.min(spans)), 3), "calls": L * blocks,
            "note": "np_sparse_mlp with 0 active rows (one rows workgroup + the reduce kernel), "
                    "L' calls back to back behind a sleep kernel: the fixed cost of a call"}


def mlp_same_layer(pipe, blocks: int = 5) -> dict:
    """L' back-to-back np_sparse_mlp calls on one layer's k rows, behind a
    sleep kernel: after the first call every record has been read once, so
    this is the call with its records as cache-resident as the hardware
    keeps them -- the most that fetching layer l+1's records ahead of its
    call could save."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B

    cfg, m = pipe.cfg, pipe.main
    L, k = cfg.layers, cfg.k
    slots = pipe.lists["active_slots"].data_ptr()
    spans = []
    for _ in range(blocks):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(m):
            torch.cuda._sleep(2_000_000)
        e0.record(m)
        for _l in range(L):
            B.np_sparse_mlp(pipe.shape, 0, pipe.x_ptr(0), pipe.resident, slots, k,
                            pipe.y.data_ptr(), pipe.ws, m)
        e1.record(m)
        e1.synchronize()
        spans.append(e0.elapsed_time(e1) * 1e3 / L)
    return {"us_per_call": round(float(np.median(spans)), 3), "calls": L * blocks,
            "note": "layer 0's k rows, L' calls back to back behind a sleep kernel"}


def read_ref_per_call(nbytes: int, calls: int, blocks: int = 5) -> dict:
    """The library GEMV (torch.mv) at one sparse-MLP call's byte count: calls
    back to back, each on its own [nbytes / 8192][4096] fp16 matrix (distinct
    bytes, as the layers' records are), behind a sleep kernel; the span per
    call is a library kernel's rate for one launch of this size."""
    import numpy as np
    import torch

    rows = (nbytes + 8191) // 8192
    ws = [torch.ones(rows, 4096, dtype=torch.float16, device="cuda") for _ in range(calls)]
    x = torch.ones(4096, dtype=torch.float16, device="cuda")
    for w in ws:
        torch.mv(w, x)
    spans = []
    for _ in range(blocks):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(2_000_000)
        e0.record()
        for w in ws:
            torch.mv(w, x)
        e1.record()
        e1.synchronize()
        spans.append(e0.elapsed_time(e1) * 1e3 / calls)
    us = float(np.median(spans))
    del ws, x
    return {"us_per_call": round(us, 3), "bytes_per_call": rows * 8192,
            "GBps": round(rows * 8192 / (us * 1e-6) / 1e9, 1), "calls": calls * blocks,
            "kernel": f"torch.mv over {calls} distinct [{rows}][4096] fp16 matrices"}


def read_ref_gbps(nbytes: int = 2 << 30, reps: int = 5) -> float:
    """A read-bound library kernel of the same run for reference: torch.mv
    (the library GEMV) of a [nbytes / 8192][4096] fp16 matrix by a vector,
    timed with events (GB/s of matrix bytes read)."""
    import torch

    w = torch.ones(nbytes // 8192, 4096, dtype=torch.float16, device="cuda")
    x = torch.ones(4096, dtype=torch.float16, device="cuda")
    torch.mv(w, x)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        torch.mv(w, x)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    del w, x
    return nbytes / (us * 1e-6) / 1e9


def persistence_of(ids_seq):
    """Mean over consecutive tokens and layers of |A_t & A_t-1| / k, from the
    active-id lists of consecutive tokens ([L'][k] arrays)."""
    import numpy as np

    vals = []
    for a, b in zip(ids_seq, ids_seq[1:]):
        for l in range(a.shape[0]):
            vals.append(np.intersect1d(a[l], b[l], assume_unique=True).size / a.shape[1])
    return float(np.mean(vals)) if vals else None


def breakdown(pipe, t0, steps):
    """Per-phase device time (µs, median over its tokens) from events on the
    main stream, one phase at a time (no overlap).  Even tokens run the
    active-set selection and the delta as the step runs them, in one call
    (np_select_delta: "select_delta"); odd tokens run them as the two calls
    np_select and np_delta ("select", "delta"), for comparison.  Both give the
    same results bit for bit, so the state evolves the same either way."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B

    s, cfg = pipe.shape, pipe.cfg
    L, k = cfg.layers, cfg.k
    acc = {}
    counts, ids = [], []
    ybytes = cfg.d_model * (4 if cfg.adtype == "f32" else 2)

    def add(name, a, b):
        acc.setdefault(name, []).append(a.elapsed_time(b) * 1e3)

    for i in range(steps):
        t = t0 + i
        fused = i % 2 == 0
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        m = pipe.main
        ev[0].record(m)
        B.np_predict(s, pipe.x_ptr(t), pipe.A, pipe.B, pipe.scores, pipe.ws, m)
        ev[1].record(m)
        if fused:
            B.np_select_delta(s, t, pipe.scores, pipe.mask, pipe.active_ids, pipe.state,
                              pipe.out, pipe.ws, m)
            ev[2].record(m)
        else:
            B.np_select(s, pipe.scores, pipe.mask, pipe.active_ids, pipe.ws, m)
            ev[2].record(m)
            B.np_delta(s, t, pipe.active_ids, pipe.state, pipe.out, pipe.ws, m)
        ev[3].record(m)
        B.np_stage_gather(s, pipe.out, 0, L, pipe.storage, pipe.resident, pipe.ws, m)
        ev[4].record(m)
        slots = pipe.lists["active_slots"].data_ptr()
        for l in range(L):
            B.np_sparse_mlp(s, l, pipe.x_ptr(t), pipe.resident, slots + 4 * l * k, k,
                            pipe.y.data_ptr() + l * ybytes, pipe.ws, m)
        ev[5].record(m)
        torch.cuda.synchronize()
        add("predict", ev[0], ev[1])
        if fused:
            add("select_delta", ev[1], ev[3])
        else:
            add("select", ev[1], ev[2])
            add("delta", ev[2], ev[3])
        add("stage", ev[3], ev[4])
        add("mlp", ev[4], ev[5])
        counts.append(delta_stats(pipe))
        ids.append(pipe.active_ids.cpu().numpy().reshape(L, k))
    out = {n: round(float(np.median(v)), 2) for n, v in acc.items()}
    return out, counts, ids


def select_delta_calls(pipe, t0: int, n: int = 8) -> dict:
    """The active-set selection and the delta per call, without the event
    overhead of timing one call: np_predict first writes the scores of n
    consecutive tokens into n buffers, then the n tokens' np_select_delta
    calls run back to back between two events (and, for n further tokens,
    np_select + np_delta), queued behind a sleep kernel so that the host's
    enqueue rate does not set the pace.  Each call advances the residency
    state as in the decode step.  Used last on a pipeline: the tokens' rows
    are not staged and their MLPs are not run."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B

    s, cfg, m = pipe.shape, pipe.cfg, pipe.main
    sc = torch.empty((2 * n, pipe.scores.numel()), dtype=torch.float32, device=pipe.scores.device)
    for i in range(2 * n):
        B.np_predict(s, pipe.x_ptr(t0 + i), pipe.A, pipe.B, sc[i], pipe.ws, m)
    out = {}
    for name, base in (("fused", 0), ("two_calls", n)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(m):
            torch.cuda._sleep(2_000_000)
        e0.record(m)
        for i in range(n):
            t = t0 + base + i
            if name == "fused":
                B.np_select_delta(s, t, sc[base + i], pipe.mask, pipe.active_ids, pipe.state,
                                  pipe.out, pipe.ws, m)
            else:
                B.np_select(s, sc[base + i], pipe.mask, pipe.active_ids, pipe.ws, m)
                B.np_delta(s, t, pipe.active_ids, pipe.state, pipe.out, pipe.ws, m)
        e1.record(m)
        e1.synchronize()
        out[name + "_us"] = round(e0.elapsed_time(e1) * 1e3 / n, 2)
    if pipe.device_error():
        raise RuntimeError(f"select/delta calls: device error word {pipe.device_error():#x}")
    out["tokens"] = n
    out["note"] = ("per token, the calls of consecutive tokens back to back between two events "
                   "(np_select_delta; np_select + np_delta)")
    return out


def predictor_paths(pipe, t: int, pbytes: int, reps: int = 20) -> dict:
    """np_predict alone, back to back on its stream, on both of its paths:
    per-lane dot products ("vgpr", the default unless NP_PREDICT_MFMA=1) and
    the matrix cores ("mfma").  Bytes: A, B, h and the fp32 scores."""
    import torch

    from paper_2608_22643_amd import binding as B

    saved = os.environ.get("NP_PREDICT_MFMA")
    out = {"bytes": pbytes}
    try:
        for name, flag in (("vgpr", "0"), ("mfma", "1")):
            os.environ["NP_PREDICT_MFMA"] = flag
            m = pipe.main
            for _ in range(3):
                B.np_predict(pipe.shape, pipe.x_ptr(t), pipe.A, pipe.B, pipe.scores, pipe.ws, m)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(m)
            for _ in range(reps):
                B.np_predict(pipe.shape, pipe.x_ptr(t), pipe.A, pipe.B, pipe.scores, pipe.ws, m)
            e1.record(m)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            gbps = pbytes / (us * 1e-6) / 1e9
            out[name] = {"avg_us": round(us, 2), "achieved_GBps": round(gbps, 1),
                         "frac": round(gbps / HBM_PEAK_GBPS, 4)}
    finally:
        if saved is None:
            os.environ.pop("NP_PREDICT_MFMA", None)
        else:
            os.environ["NP_PREDICT_MFMA"] = saved
    out["default"] = "mfma" if saved == "1" else "vgpr"
    out.update(out[out["default"]])
    return out


def h2d_peak_gbps(nbytes: int = 1 << 30) -> float:
    """One pinned host -> device hipMemcpyAsync of `nbytes`, timed with events."""
    import torch

    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst.copy_(src, non_blocking=True)  # first touch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    dst.copy_(src, non_blocking=True)
    e1.record()
    torch.cuda.synchronize()
    return nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9


def staging_rates(pipe, t0: int, steps: int) -> dict:
    """np_stage_rows alone (memcpy tier): staged bytes over the time from the
    plan's arrival on the host (host packing included) to the end of its
    copies and scatters as the host sees it, next to a 1 GiB pinned
    hipMemcpyAsync measured in the same run; the same span on the device (the
    event after the plan's copy to the event after the last scatter, both
    timing-enabled for this window), which leaves out how long the host takes
    to wake from its waits; and the host side alone: the time until the
    calls return, when every record has been packed into pinned staging and
    every piece's copy enqueued."""
    import torch

    L = pipe.cfg.layers
    plan_ev, last_ev = pipe.ev_plan, pipe.layer_ready[L - 1] if pipe.layer_ready else None
    timed = last_ev is not None
    if timed:  # the pipeline's own events, swapped for timing-enabled ones
        pipe.ev_plan = torch.cuda.Event(enable_timing=True)
        pipe.layer_ready[L - 1] = torch.cuda.Event(enable_timing=True)
        pipe.layer_ready[L - 1].record(pipe.side)
    dev_s = 0.0
    pipe.stage_log = []
    trace_marker()  # a kernel trace shows this window's copies between two markers
    try:
        for i in range(steps):
            pipe.step(t0 + i)  # waits for the token's staging before it returns
            if timed:
                dev_s += pipe.ev_plan.elapsed_time(pipe.layer_ready[L - 1]) * 1e-3
        torch.cuda.synchronize()
    finally:
        if timed:
            torch.cuda.synchronize()
            pipe.ev_plan, pipe.layer_ready[L - 1] = plan_ev, last_ev
    trace_marker()
    nb = sum(e[0] for e in pipe.stage_log)
    sec = sum(e[1] for e in pipe.stage_log)
    call = sum(e[2] for e in pipe.stage_log)
    pipe.stage_log = None
    out = {"staging_h2d_GBps": round(nb / sec / 1e9, 2),
           "staged_MB_per_token": round(nb / steps / 1e6, 2), "tokens": steps,
           "staged_bytes": int(nb),
           "staging_ms_per_token": round(sec * 1e3 / steps, 3),
           "host_call_ms_per_token": round(call * 1e3 / steps, 3)}
    if timed:
        out["device_staging_GBps"] = round(nb / dev_s / 1e9, 2)
        out["device_staging_ms_per_token"] = round(dev_s * 1e3 / steps, 3)
    out["h2d_peak_GBps"] = round(h2d_peak_gbps(), 2)
    return out


def pinned_host_run(cfg, host_storage, steps: int, tokens: int, t0: int = 0,
                    fill: int = 0) -> dict:
    """The spec step with the storage tier in pinned host memory:
    np_predict, np_select, np_delta, np_stage_rows (the plan read on the host,
    records packed into pinned staging and sent with hipMemcpyAsync, then
    scattered) and the sparse MLPs, per token, for the step with staging on a
    side stream in layer groups (each group's MLPs run while the next group
    is staged; every fourth group is gathered by the GPU from the pinned tier
    instead of packed) and on the main stream; then the mapped-memory gather
    of the same tier (np_stage_gather, the GPU reading pinned memory over the
    host link) for every group.  Reports tokens/s of each, the staging rate of np_stage_rows alone
    against a 1 GiB pinned hipMemcpyAsync of the same run, and the host's
    share (packing and enqueueing).  Each pipeline starts cold and runs 4 +
    `fill` untimed tokens first (with fill, the resident buffer is full and
    every timed token evicts)."""
    import torch

    from paper_2608_22643_amd.pipeline import DecodePipeline

    out = {}
    best = None
    for staging, overlap in (("memcpy", True), ("memcpy", False), ("gather", True)):
        key = f"{'np_stage_rows' if staging == 'memcpy' else 'np_stage_gather'}" + \
              ("_overlap" if overlap else "")
        p = DecodePipeline(cfg, tier="host", staging=staging, overlap=overlap, tokens=tokens,
                           host_storage=host_storage)
        for i in range(4 + fill):
            p.step(t0 + i)
        torch.cuda.synchronize()
        wall, _ = timed_steps(p, t0 + 4 + fill, steps, with_mlp_events=False)
        rec = {"tok_s": round(steps / wall, 2), "ms_per_token": round(wall * 1e3 / steps, 3)}
        if p.gather_every:
            rec["gpu_gathered_groups"] = (f"every {p.gather_every}th layer group from the "
                                          f"second on, {p.gather_every - 1} in {p.gather_every} "
                                          f"packed by the host (staging alone: every group packed)")
        if staging == "memcpy":
            rec.update(staging_rates(p, t0 + 4 + fill + steps, max(3, steps // 2)))
            if best is None or rec["tok_s"] > out[best]["tok_s"]:
                best = key
        if p.device_error():
            raise RuntimeError(f"{cfg.name} host tier: device error word {p.device_error():#x}")
        out[key] = rec
        del p
        torch.cuda.empty_cache()
    out["tok_s"] = out[best]["tok_s"]
    # the staging rate of the faster mode: between device events where the
    # mode records them (plan copy done to last scatter done), else as the
    # host sees it; on a freshly started box the host's wake from its final
    # wait alone has added about 0.5 ms per token to the second
    out["staging_GBps"] = out[best].get("device_staging_GBps", out[best]["staging_h2d_GBps"])
    out["staging_timed_by"] = "device events" if "device_staging_GBps" in out[best] else "host"
    out["host_observed_staging_GBps"] = out[best]["staging_h2d_GBps"]
    out["h2d_peak_GBps"] = out[best]["h2d_peak_GBps"]
    out["mode"] = best
    return out


def file_tier_run(cfg, host_storage, steps: int) -> dict:
    """The storage tier as a file on the local disk (Sec. 3.5: neuron-centric
    layer-major file, O_DIRECT, io_uring at queue depth 256): the decode step
    with file staging, the staging rate (reads + copies + scatter), and the
    record-read rate of np_read_records on a token-like read list (about 70
    sorted random records per layer) at queue depths 1, 32 and 256."""
    import os

    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B
    from paper_2608_22643_amd.pipeline import DecodePipeline

    T = 1 + 3 + 2 * steps + 4
    t = time.perf_counter()
    # staging pieces of 64 MiB and a read buffer of 128 MiB: each layer
    # group's records are read as one batch of requests (the paper's
    # token-level submission, per group)
    pipe = DecodePipeline(cfg, tier="file", staging="file", overlap=True, tokens=T,
                          host_storage=host_storage, staging_mib=256, landing_mib=128)
    write_s = time.perf_counter() - t
    for i in range(4):
        pipe.step(i)
    torch.cuda.synchronize()
    wall, _ = timed_steps(pipe, 4, steps, with_mlp_events=False)
    rates = staging_rates(pipe, 4 + steps, max(3, steps // 2))
    rec = cfg.record_bytes
    rng = np.random.default_rng(1)
    ids = np.concatenate([l * cfg.d_ffn + np.sort(rng.choice(cfg.d_ffn, 70, replace=False))
                          for l in range(cfg.layers)]).astype(np.int32)
    dst = B.HostBuffer(ids.size * rec)  # ordinary memory: the target of direct reads
    reads = {}
    for qd in (1, 32, 256):
        os.environ["NP_IO_QD"] = str(qd)
        t = time.perf_counter()
        B.np_read_records(pipe.storage_fd, 0, rec, ids.ctypes.data, ids.size, dst)
        reads[f"qd{qd}_GBps"] = round(ids.size * rec / (time.perf_counter() - t) / 1e9, 2)
    os.environ.pop("NP_IO_QD", None)
    if pipe.device_error():
        raise RuntimeError(f"file tier: device error word {pipe.device_error():#x}")
    out = {"tok_s": round(steps / wall, 2), "ms_per_step": round(wall * 1e3 / steps, 3),
           "direct_io": pipe.storage_direct, "file_GB": round(cfg.storage_bytes / 1e9, 2),
           "file_write_s": round(write_s, 1),
           "stage_GBps": rates["staging_h2d_GBps"],
           "staged_MB_per_token": rates["staged_MB_per_token"],
           "record_reads": dict(reads, records=int(ids.size), MB=round(ids.size * rec / 1e6, 1)),
           "note": "local virtio block device of the GPU host (no NVMe present); O_DIRECT "
                   "reads bypass the page cache"}
    pipe.close()
    del pipe, dst
    torch.cuda.empty_cache()
    return out


def delta_stats(pipe):
    import numpy as np

    c = pipe.counts.cpu().numpy().reshape(-1, 4)
    return c


def hbm_config_run(name: str, steps: int, fill: int = 0) -> tuple[dict, dict]:
    """A configuration whose storage tier, resident set and predictor all fit
    in one GPU's HBM at full size (the 70B shape: 111 GB + 39 GB + 4.5 GB):
    steps launched as the main measurement, the sparse-MLP call against the
    HBM roofline, and the delta figures.  Returns the figures and a sample of
    the last token (two layers' scores, selection and MLP outputs) for the
    oracle leg to check."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import workload as W
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get(name)
    T = 4 + fill + 2 * steps + 4 + 4 + fill + 3 * steps + 16
    t = time.perf_counter()
    # the storage tier generated once into pinned host memory: copied to HBM
    # for the HBM leg, read over the host link in the stated tier's leg
    host_storage = None
    try:
        host_storage = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
        W.fill_storage(cfg, host_storage.data_ptr())
    except RuntimeError as e:  # not enough pinnable host memory: generate per layer
        log(f"[bench] {name}: no pinned copy of the storage tier ({str(e).splitlines()[0]})")
        host_storage = None
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T,
                          host_storage=host_storage)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t
    log(f"[bench] {name}: every tier in HBM ({torch.cuda.memory_allocated() / 1e9:.1f} GB), "
        f"generated in {setup_s:.1f} s")
    for i in range(4 + fill):
        pipe.step(i)
    wall, _ = timed_steps(pipe, 4 + fill, steps, with_mlp_events=False)
    _, mlp_us = timed_steps(pipe, 4 + fill + steps, steps)
    torch.cuda.synchronize()
    counts = delta_stats(pipe)
    if pipe.device_error():
        raise RuntimeError(f"{name}: device error word {pipe.device_error():#x}")
    L, F, k, d = cfg.layers, cfg.d_ffn, cfg.k, cfg.d_model
    last = 4 + fill + 2 * steps - 1
    layers = [0, L - 1]
    scores = pipe.scores.cpu().numpy().reshape(L, F)
    ids = pipe.active_ids.cpu().numpy().reshape(L, k)
    yb = pipe.y.cpu().view(torch.uint8).numpy()
    y = yb.view(np.float32 if cfg.adtype == "f32" else np.uint16).reshape(L, d)
    sample = {"cfg": cfg, "tokens": T, "token": last, "layers": layers,
              "scores": scores[layers].copy(), "ids": ids[layers].copy(), "y": y[layers].copy()}
    bytes_launch = mlp_bytes_per_launch(cfg)
    achieved = bytes_launch / (mlp_us * 1e-6) / 1e9
    out = {"workload": f"{cfg.name}-shaped decode, every tier in HBM: {L} downstream layers, "
                       f"d={d}, F={F}, rank {cfg.rank}, k={k}, C={cfg.capacity}, {cfg.wdtype}",
           "hbm_GB": round(torch.cuda.memory_allocated() / 1e9, 1),
           "tok_s": round(steps / wall, 2), "ms_per_step": round(wall * 1e3 / steps, 4),
           "sparse_mlp": {"avg_launch_us": round(mlp_us, 3), "bytes_per_launch": bytes_launch,
                          "achieved_GBps": round(achieved, 1),
                          "frac": round(achieved / HBM_PEAK_GBPS, 4)},
           "incoming_rows_per_token": int(counts[:, 0].sum())}
    del pipe
    torch.cuda.empty_cache()
    # the stated tier: resident set in HBM, the rest in pinned host memory.
    # When the host cannot pin the whole storage tier, the leg runs on the
    # first layers only (the same per-layer shapes; halved until it fits) and
    # says so.
    host_cfg = cfg
    n = cfg.layers
    while host_storage is None and n > 8:
        n //= 2
        host_cfg = cfg.with_(name=f"{cfg.name}-first{n}", layers=n)
        try:
            host_storage = torch.empty(host_cfg.storage_bytes, dtype=torch.uint8,
                                       pin_memory=True)
            W.fill_storage(host_cfg, host_storage.data_ptr())
            log(f"[bench] {name}: host tier on the first {n} of {cfg.layers} layers "
                f"({host_cfg.storage_bytes / 1e9:.1f} GB pinned)")
        except RuntimeError as e:
            log(f"[bench] {name}: {n} layers not pinnable ({str(e).splitlines()[0]})")
            host_storage = None
    if host_storage is not None:
        ht = pinned_host_run(host_cfg, host_storage, steps, T, 4 + fill + 2 * steps + 4, fill)
        ht["layers"] = host_cfg.layers
        ht["pinned_GB"] = round(host_cfg.storage_bytes / 1e9, 1)
        ht["ms_per_layer"] = round(1e3 / ht["tok_s"] / host_cfg.layers, 4)
        if host_cfg.layers != cfg.layers:
            ht["note"] = (f"first {host_cfg.layers} of {cfg.layers} downstream layers: the host "
                          f"could not pin the whole {cfg.storage_bytes / 1e9:.0f} GB storage tier")
        out["host_tier"] = ht
        del host_storage
    return out, sample


def extra_config(name: str, steps: int, graph: bool, overlap: bool, fill: int = 0) -> dict:
    """The same measurements, shorter, on another configuration (13B shape):
    steps with the storage tier in HBM (launched as the main measurement),
    the sparse-MLP call against the HBM roofline, and the step with the
    storage tier in pinned host memory (memcpy staging) with its staging
    rate."""
    import torch

    from paper_2608_22643_amd import workload as W
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get(name)
    T = 4 + fill + 2 * steps + 4 + fill + 3 * steps + 16
    t = time.perf_counter()
    host_storage = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, host_storage.data_ptr())
    log(f"[bench] {name}: storage tier generated: {cfg.storage_bytes / 1e9:.2f} GB in "
        f"{time.perf_counter() - t:.1f} s")
    pipe = DecodePipeline(cfg, tier="device", staging="gather", overlap=overlap, tokens=T,
                          host_storage=host_storage)
    if graph:
        pipe.capture_graph()
        for i in range(4 + fill):
            pipe.step_graph(i)
        wall = timed_graph_steps(pipe, 4 + fill, steps)
    else:
        for i in range(4 + fill):
            pipe.step(i)
        wall, _ = timed_steps(pipe, 4 + fill, steps, with_mlp_events=False)
    _, mlp_us = timed_steps(pipe, 4 + fill + steps, steps)
    counts = delta_stats(pipe)
    if pipe.device_error():
        raise RuntimeError(f"{name}: device error word {pipe.device_error():#x}")
    bytes_launch = mlp_bytes_per_launch(cfg)
    achieved = bytes_launch / (mlp_us * 1e-6) / 1e9
    out = {"workload": f"{cfg.name}-shaped decode: {cfg.layers} downstream layers, d={cfg.d_model}, "
                       f"F={cfg.d_ffn}, rank {cfg.rank}, k={cfg.k}, C={cfg.capacity}, {cfg.wdtype}",
           "tok_s": round(steps / wall, 2), "ms_per_step": round(wall * 1e3 / steps, 4),
           "sparse_mlp": {"avg_launch_us": round(mlp_us, 3), "bytes_per_launch": bytes_launch,
                          "achieved_GBps": round(achieved, 1),
                          "frac": round(achieved / HBM_PEAK_GBPS, 4)},
           "incoming_rows_per_token": int(counts[:, 0].sum())}
    del pipe
    torch.cuda.empty_cache()
    out["host_tier"] = pinned_host_run(cfg, host_storage, steps, T, 0, fill)
    del host_storage
    torch.cuda.empty_cache()
    return out


def centroid_run(cfg, host_storage, steps: int) -> dict:
    """The decode step with the paper's own predictor (centroid-ID heads and
    gate/up mask intersection; variable-size active sets) on the same
    workload: step rate, the predictor's time, set sizes, persistence."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B
    from paper_2608_22643_amd.pipeline import DecodePipeline

    T = 1 + 3 + steps + 8
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T,
                          host_storage=host_storage, predictor="centroid")
    for i in range(4):
        pipe.step(i)
    wall, _ = timed_steps(pipe, 4, steps, with_mlp_events=False)
    # the predictor alone, and the set statistics of a few tokens
    L, k = cfg.layers, cfg.k
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sizes, overlap, prev = [], [], None
    pred_us = 0.0
    for i in range(4):
        t = 4 + steps + i
        torch.cuda.synchronize()
        e0.record(pipe.main)
        B.np_centroid_select(pipe.shape, pipe.model, pipe.f_ptr(t), pipe.logits, pipe.cids,
                             pipe.mask, pipe.active_ids, pipe.active_counts, pipe.ws, pipe.main)
        e1.record(pipe.main)
        torch.cuda.synchronize()
        pred_us += e0.elapsed_time(e1) * 1e3
        n = pipe.active_counts.cpu().numpy()[:L]
        ids = pipe.active_ids.cpu().numpy().reshape(L, k)
        sets = [set(ids[l][:n[l]].tolist()) for l in range(L)]
        sizes.append(float(n.mean()))
        if prev is not None:
            overlap.append(np.mean([len(a & b) / max(1, len(b)) for a, b in zip(prev, sets)]))
        prev = sets
    if pipe.device_error():
        raise RuntimeError(f"centroid run: device error word {pipe.device_error():#x}")
    K, D = cfg.centroid_k, cfg.feat_dim
    out = {"tok_s": round(steps / wall, 2), "ms_per_step": round(wall * 1e3 / steps, 4),
           "predictor_us": round(pred_us / 4, 2),
           "predictor_heads_MB": round(2 * L * K * D * (4 if cfg.wdtype == "f32" else 2) / 1e6, 1),
           "mean_active_per_layer": round(float(np.mean(sizes)), 1),
           "persistence": round(float(np.mean(overlap)), 4),
           "centroids": K, "feat_dim": D}
    del pipe
    torch.cuda.empty_cache()
    return out


def swiglu_run(steps: int, calib_tokens: int = 128, alpha: float = 61.6) -> dict:
    """The SwiGLU model shape (Sec. 4: d 4096, intermediate 14336, fp16, the
    K_max = 5500 budget) with magnitude-threshold sparsity (eq. 1, Sec. 3.2):
    per-layer thresholds calibrated on the GPU from calib_tokens synthetic
    tokens at alpha = 61.6 (38.4% of the activations kept), then the decode
    step with the centroid predictor and the thresholded SwiGLU MLP.  Reports
    the calibration kernels against their rooflines and the step rate."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import binding as B
    from paper_2608_22643_amd import calibrate
    from paper_2608_22643_amd import workload as W
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get("7b_swiglu")
    L, F, d = cfg.layers, cfg.d_ffn, cfg.d_model
    esz = W.ITEMSIZE[cfg.wdtype]
    T = 1 + 4 + 2 * steps + 8
    hs = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, hs.data_ptr())
    pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T, host_storage=hs,
                          predictor="centroid")
    del hs
    xc = W.hidden(cfg.with_(seed=cfg.seed + 101), calib_tokens)
    xc = torch.from_numpy(np.ascontiguousarray(xc).view(np.uint8).reshape(-1).copy()).cuda()
    acts = torch.empty(L * calib_tokens * F, dtype=torch.float32, device="cuda")
    thr = calibrate.thresholds(cfg, pipe.storage, xc, calib_tokens, alpha, pipe.ws, acts=acts)
    torch.cuda.synchronize()
    # the calibration kernels, timed on their stream
    shape = pipe.shape
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    layer_bytes = F * cfg.record_bytes
    stream = torch.cuda.current_stream()
    ev[0].record(stream)
    for l in range(L):
        B.np_act_batch(shape, pipe.storage.data_ptr() + l * layer_bytes, xc, calib_tokens,
                       acts.data_ptr() + l * calib_tokens * F * 4, pipe.ws, stream)
    ev[1].record(stream)
    out = torch.empty(L, dtype=torch.float32, device="cuda")
    B.np_percentile(acts, L, calib_tokens * F, alpha, out, pipe.ws, pipe.ws.numel(), stream)
    ev[2].record(stream)
    torch.cuda.synchronize()
    ab_us = ev[0].elapsed_time(ev[1]) * 1e3 / L
    pct_us = ev[1].elapsed_time(ev[2]) * 1e3
    if not torch.equal(out, thr):
        raise RuntimeError("calibration: thresholds differ between two identical runs")
    # eq. 1 as active sets (np_threshold_active) over one token's activations
    # of every layer, with room for 8192 ids per layer (its own workspace, so
    # that an overflow would be reported here, not as the pipeline's error)
    a0 = acts.view(L, calib_tokens, F)[:, 0, :].contiguous()
    tshape = B.make_shape(L, d, F, cfg.rank, min(F, 8192), F, cfg.wdtype, act="swiglu")
    tws = torch.zeros(B.np_workspace_size(tshape), dtype=torch.uint8, device="cuda")
    tmask = torch.empty(L * ((F + 31) // 32), dtype=torch.int32, device="cuda")
    tids = torch.empty(L * min(F, 8192), dtype=torch.int32, device="cuda")
    tcnt = torch.empty(L, dtype=torch.int32, device="cuda")
    B.np_threshold_active(tshape, a0, L, thr, tmask, tids, tcnt, tws, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        B.np_threshold_active(tshape, a0, L, thr, tmask, tids, tcnt, tws, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ta_us = e0.elapsed_time(e1) * 1e3 / 10
    ta_err = B.np_device_error(tws)
    ta_kept = float(tcnt.float().mean())
    del a0, tmask, tids, tcnt, tws
    ab_bytes = F * 2 * d * esz + calib_tokens * d * esz + calib_tokens * F * 4
    ab_flops = 4.0 * F * d * calib_tokens
    ab_gbps = ab_bytes / (ab_us * 1e-6) / 1e9
    kept = float((acts.view(L, -1).abs() >= thr.view(L, 1)).float().mean())
    pipe.set_thresholds(thr)
    for i in range(5):
        pipe.step(i)
    wall, _ = timed_steps(pipe, 5, steps, with_mlp_events=False)
    _, mlp_us = timed_steps(pipe, 5 + steps, steps)
    counts = []  # rows per np_sparse_mlp_t call, over a few more tokens
    for i in range(6):
        pipe.step(5 + 2 * steps + i)
        counts.append(pipe.active_counts.cpu().numpy()[:L].mean())
    if pipe.device_error():
        raise RuntimeError(f"swiglu run: device error word {pipe.device_error():#x}")
    rows = float(np.mean(counts))
    mlp_bytes = rows * 3 * d * esz
    mlp_gbps = mlp_bytes / (mlp_us * 1e-6) / 1e9
    res = {"config": f"{L} downstream layers, d={d}, F={F}, K_max={cfg.k}, C={cfg.capacity}, "
                     f"{cfg.wdtype}, SwiGLU, centroid predictor, eq. 1 thresholds",
           "tok_s": round(steps / wall, 2), "ms_per_step": round(wall * 1e3 / steps, 4),
           "mean_active_per_layer": round(rows, 1),
           "mlp_us_per_call": round(mlp_us, 3), "mlp_GBps": round(mlp_gbps, 1),
           "mlp_frac": round(mlp_gbps / HBM_PEAK_GBPS, 4),
           "calibration": {
               "tokens": calib_tokens, "alpha": alpha,
               "kept_fraction": round(kept, 4),
               "threshold_mean": round(float(thr.mean()), 5),
               "act_batch_us_per_layer": round(ab_us, 2),
               "act_batch_roofline": {"bound": "hbm", "achieved": round(ab_gbps, 1),
                                      "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                      "frac": round(ab_gbps / HBM_PEAK_GBPS, 4),
                                      "bytes_per_launch": ab_bytes,
                                      "mfma_TFLOPs": round(ab_flops / (ab_us * 1e-6) / 1e12, 1),
                                      "mfma_peak_TFLOPs": 2500.0},
               "percentile_us": round(pct_us, 1),
               "percentile_values": L * calib_tokens * F,
               "threshold_active_us": round(ta_us, 2),
               "threshold_active_mean_ids": round(ta_kept, 1),
               "threshold_active_error_word": ta_err}}
    del pipe, acts
    torch.cuda.empty_cache()
    return res


def sweep_run(host_storage, steps: int) -> dict:
    """The 7B sweep (activity 5/15/30%, persistence 70/82/85/95%, residency
    25/50/75%, one factor at a time around 15% / 83.5% / 50%): per point the
    step rate, incoming rows and staged bytes per token, the hit share, and
    the sparse MLP's per-call time and HBM rate.  The records are the same at
    every point (same shapes and seed), so the 7B storage tier is reused."""
    import numpy as np
    import torch

    from paper_2608_22643_amd import workload as W
    from paper_2608_22643_amd.pipeline import DecodePipeline

    out = {}
    warm = 120  # the resident set fills for ~C / (incoming per layer) tokens
    for cfg in W.sweep_configs():
        T = warm + 2 * steps + 8
        pipe = DecodePipeline(cfg, tier="device", staging="gather", tokens=T,
                              host_storage=host_storage)
        for i in range(warm):
            pipe.step(i)
        wall, mlp_us = timed_steps(pipe, warm, steps)
        _, per_tok, ids = breakdown(pipe, warm + steps, max(3, steps // 2))
        if pipe.device_error():
            raise RuntimeError(f"sweep {cfg.name}: device error word {pipe.device_error():#x}")
        n_in = float(np.mean([c[:, 0].sum() for c in per_tok]))
        n_hit = float(np.mean([c[:, 1].sum() for c in per_tok]))
        b = mlp_bytes_per_launch(cfg)
        out[cfg.name] = {"k": cfg.k, "C": cfg.capacity, "persistence": cfg.persistence,
                         "persistence_measured": round(persistence_of(ids), 4),
                         "tok_s": round(steps / wall, 1),
                         "incoming_rows_per_token": round(n_in, 1),
                         "staged_MB_per_token": round(n_in * cfg.record_bytes / 1e6, 2),
                         "reuse_pct": round(100.0 * n_hit / (cfg.k * cfg.layers), 2),
                         "mlp_us_per_call": round(mlp_us, 2),
                         "mlp_GBps": round(b / (mlp_us * 1e-6) / 1e9, 1)}
        del pipe
        torch.cuda.empty_cache()
    return out


def dense_mlp_roofline(cfg, host_storage, reps: int = 3) -> dict:
    """np_dense_mlp over every layer of the storage tier (all F records of a
    layer: the dense prefix's MLP), back to back, against the HBM roofline."""
    import torch

    from paper_2608_22643_amd import binding as B

    L, d = cfg.layers, cfg.d_model
    esz = 4 if cfg.wdtype == "f32" else 2
    layer_bytes = cfg.d_ffn * cfg.record_bytes
    dev = torch.device("cuda")
    w = torch.empty(cfg.storage_bytes, dtype=torch.uint8, device=dev)
    w.copy_(host_storage)
    x = torch.zeros(d, dtype=torch.float16 if esz == 2 else torch.float32, device=dev)
    y = torch.empty(L * d, dtype=x.dtype, device=dev)
    shape = B.make_shape(L, d, cfg.d_ffn, cfg.rank, cfg.k, cfg.capacity, cfg.wdtype, cfg.adtype,
                         cfg.act)
    ws = torch.zeros(B.np_workspace_size(shape), dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream()

    def block():
        for l in range(L):
            B.np_dense_mlp(shape, w.data_ptr() + l * layer_bytes, x, y.data_ptr() + l * d * esz,
                           ws, st)
    block()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(reps):
        block()
    e1.record(st)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * L)
    byts = layer_bytes + 2 * d * esz
    if B.np_device_error(ws):
        raise RuntimeError("dense MLP: device error")
    del w
    torch.cuda.empty_cache()
    return {"avg_launch_us": round(us, 3), "bytes_per_launch": byts,
            "achieved_GBps": round(byts / (us * 1e-6) / 1e9, 1),
            "frac": round(byts / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)}


def dense_prefix_sweep(cfg, host_storage, prefixes, steps: int) -> dict:
    """Decode steps with d of the downstream layers run dense (weights
    resident) and the other L' - d sparse, for each d: storage tier in HBM
    (gather staging) and in pinned host memory (memcpy staging on a side
    stream, overlapping the dense prefix).  The synthetic analogue of the
    paper's dense-prefix sweep, without its memory cap (see split.py for d*)."""
    import torch

    from paper_2608_22643_amd.pipeline import DecodePipeline

    out = {}
    layer_bytes = cfg.d_ffn * cfg.record_bytes
    for dl in prefixes:
        sc = cfg.with_(layers=cfg.layers - dl)
        hs = host_storage[:sc.storage_bytes]  # the first L' - d layers' records
        row = {}
        for tier, staging, overlap in (("device", "gather", False), ("host", "memcpy", True)):
            T = 4 + steps + 2
            p = DecodePipeline(sc, tier=tier, staging=staging, overlap=overlap, tokens=T,
                               host_storage=hs, dense_layers=dl)
            for i in range(4):
                p.step(i)
            wall, _ = timed_steps(p, 4, steps, with_mlp_events=False)
            if p.device_error():
                raise RuntimeError(f"dense sweep d={dl}: device error {p.device_error():#x}")
            row[f"{tier}_tok_s"] = round(steps / wall, 2)
            del p
            torch.cuda.empty_cache()
        row["resident_GB"] = round((dl * layer_bytes + sc.resident_bytes) / 1e9, 2)
        out[str(dl)] = row
        log(f"[bench] dense prefix {dl}: {row}")
    return out


def capture_outputs(pipe) -> dict:
    """One token's results on the host: scores, selection, delta lists, slot
    maps and the sparse-MLP outputs of every layer (after a synchronize)."""
    cfg = pipe.cfg
    L, F, k, d = cfg.layers, cfg.d_ffn, cfg.k, cfg.d_model
    out = {"scores": pipe.scores.cpu().numpy().reshape(L, F).copy(),
           "ids": pipe.active_ids.cpu().numpy().reshape(L, k).copy(),
           "lists": pipe.host_lists(), "state": pipe.host_state()}
    yb = pipe.y.cpu().view(torch_uint8()).numpy()
    out["y"] = yb.view("float32" if cfg.adtype == "f32" else "uint16").reshape(L, d).copy()
    return out


def torch_uint8():
    import torch

    return torch.uint8


def mlp_tol(adtype: str, ref64):
    """The sparse-MLP output tolerance of the GPU tests: fp16 2e-2 absolute;
    fp32 1e-5 relative to max |y|; bf16 max(2e-2, one bf16 ulp of |y|)."""
    import numpy as np

    if adtype == "f16":
        return np.full(ref64.shape, 2e-2)
    if adtype == "f32":
        return np.full(ref64.shape, 1e-5 * max(float(np.max(np.abs(ref64))), 1e-30))
    a = np.abs(ref64)
    ulp = np.where(a > 0, 2.0 ** (np.floor(np.log2(np.maximum(a, 1e-300))) - 7), 2.0 ** -133)
    return np.maximum(2e-2, ulp)


def cpu_baseline(cfg, host_storage, seconds: float, gpu_ref=(), big_samples=()):
    """The oracle (plain C, fp64, one thread) on whole tokens of the same
    workload until `seconds` of CPU work have run (at least one token, and
    every token of gpu_ref).  For the tokens in gpu_ref (the GPU's first
    tokens from cold start) it runs in lockstep with the GPU as the tests do:
    its select takes the GPU's scores (fp32 rounding may move ties at the
    k-th score), and the selection, every delta list, the slot maps and the
    MLP outputs are compared; the verdict is returned under "parity".  Each
    of big_samples (a few layers of the last token of a full-size
    configuration run with every tier in HBM) is checked the same way: the
    selection on the GPU's scores, and the MLP outputs against the oracle
    over those layers' regenerated records."""
    import numpy as np

    import oracle
    from paper_2608_22643_amd import workload as W

    oracle.build()
    A, Bm = W.predictor(cfg)
    h = W.hidden(cfg, 64)
    store = host_storage.numpy().view(np.float32 if cfg.wdtype == "f32" else np.uint16)
    store = store.reshape(cfg.layers, cfg.d_ffn, 3 * cfg.d_model)
    st = oracle.State(cfg.layers, cfg.d_ffn, cfg.capacity)
    L = cfg.layers
    checks = {"tokens": 0, "scores_max_rel_diff": 0.0, "select_exact": True, "delta_exact": True,
              "slot_maps_exact": True, "mlp_max_abs_err": 0.0, "mlp_within_tol": True}
    n, t0 = 0, time.perf_counter()
    step_s = {"predict": 0.0, "select": 0.0, "delta": 0.0, "sparse_mlp": 0.0}
    while True:
        ta = time.perf_counter()
        s = oracle.predict(cfg, h[n], A, Bm)
        step_s["predict"] += time.perf_counter() - ta
        ref = gpu_ref[n] if n < len(gpu_ref) else None
        if ref is not None:
            gs = ref["scores"]
            scale = max(float(np.max(np.abs(s))), 1e-30)
            checks["scores_max_rel_diff"] = max(checks["scores_max_rel_diff"],
                                                float(np.max(np.abs(gs.astype(np.float64) - s))) / scale)
            s = gs
        ta = time.perf_counter()
        _, ids = oracle.select(s, cfg.k)
        tb = time.perf_counter()
        dl = oracle.delta(n, ids, st, cfg.capacity)
        tc = time.perf_counter()
        ys = [oracle.sparse_mlp(cfg, l, h[n], store, ids[l], want_f64=ref is not None)
              for l in range(L)]
        step_s["select"] += tb - ta
        step_s["delta"] += tc - tb
        step_s["sparse_mlp"] += time.perf_counter() - tc
        if ref is not None:
            checks["tokens"] += 1
            checks["select_exact"] &= bool(np.array_equal(ids, ref["ids"]))
            gl = ref["lists"]
            ok = np.array_equal(gl["counts"], dl["counts"]) and np.array_equal(
                gl["active_slots"], dl["active_slots"])
            for l in range(L):
                c = dl["counts"][l]
                for name, m in (("in_ids", c[0]), ("in_slots", c[0]), ("hit_ids", c[1]),
                                ("ev_ids", c[2]), ("ev_slots", c[2])):
                    ok = ok and np.array_equal(gl[name][l][:m], dl[name][l][:m])
            checks["delta_exact"] &= bool(ok)
            P, Q, U = ref["state"]
            checks["slot_maps_exact"] &= bool(np.array_equal(P, st.slot_of) and
                                              np.array_equal(Q, st.neuron_of) and
                                              np.array_equal(U, st.last_used))
            for l in range(L):
                ref64 = ys[l][1]
                got = (ref["y"][l].astype(np.float64) if cfg.adtype == "f32"
                       else oracle.decode(cfg.adtype, ref["y"][l]))
                err = np.abs(got - ref64)
                checks["mlp_max_abs_err"] = max(checks["mlp_max_abs_err"], float(np.max(err)))
                checks["mlp_within_tol"] &= bool(np.all(err <= mlp_tol(cfg.adtype, ref64)))
        n += 1
        el = time.perf_counter() - t0
        if (el >= seconds and n >= len(gpu_ref)) or n >= 64:
            break
    out = {"value": round(n / el, 4), "unit": "tokens/s", "cores": 1, "kind": "oracle",
           "sample": f"{n} whole decode tokens (cold start first) of the {cfg.name} workload: "
                     f"predict, select, delta, sparse MLP of all {cfg.layers} layers; "
                     f"staging omitted (a byte copy); {el:.1f} s on 1 host thread",
           "cpu_model": cpu_model(), "cpu_detail": cpu_detail(), "host_cpus": os.cpu_count(),
           "per_step_ms_per_token": {k: round(v * 1e3 / n, 2) for k, v in step_s.items()}}
    # the same tokens again with the work of each step spread over the host
    # threads layer by layer (the oracle's C calls release the interpreter
    # lock): O1 and O2 on one layer per call, the sparse MLPs one layer per
    # call; O3 stays one call over all layers (its state is the whole buffer)
    threads = min(len(os.sched_getaffinity(0)), L) if hasattr(os, "sched_getaffinity") else 1
    if threads > 1:
        from concurrent.futures import ThreadPoolExecutor
        from types import SimpleNamespace

        one = SimpleNamespace(layers=1, d_model=cfg.d_model, d_ffn=cfg.d_ffn, rank=cfg.rank,
                              wdtype=cfg.wdtype, adtype=cfg.adtype)
        st2 = oracle.State(cfg.layers, cfg.d_ffn, cfg.capacity)
        step2 = {"predict": 0.0, "select": 0.0, "delta": 0.0, "sparse_mlp": 0.0}
        t1 = time.perf_counter()
        with ThreadPoolExecutor(threads) as ex:
            for i in range(n):
                ta = time.perf_counter()
                s2 = np.concatenate(list(ex.map(
                    lambda l: oracle.predict(one, h[i], A[l], Bm[l]), range(L))))
                tb = time.perf_counter()
                ids2 = np.concatenate(list(ex.map(
                    lambda l: oracle.select(s2[l:l + 1], cfg.k)[1], range(L))))
                tc = time.perf_counter()
                oracle.delta(i, ids2, st2, cfg.capacity)
                td = time.perf_counter()
                list(ex.map(lambda l: oracle.sparse_mlp(cfg, l, h[i], store, ids2[l]), range(L)))
                te = time.perf_counter()
                for k2, v2 in (("predict", tb - ta), ("select", tc - tb), ("delta", td - tc),
                               ("sparse_mlp", te - td)):
                    step2[k2] += v2
        el2 = time.perf_counter() - t1
        out["all_cores"] = {"value": round(n / el2, 4), "cores": threads,
                            "per_step_ms_per_token": {k2: round(v2 * 1e3 / n, 2)
                                                      for k2, v2 in step2.items()},
                            "note": "the same tokens, O1, O2 and the sparse MLPs one layer per "
                                    "call on a thread pool, O3 one call"}
    for smp in big_samples:  # sampled layers of the full-size HBM configurations
        bc = smp["cfg"]
        hb = W.hidden(bc, smp["tokens"])[smp["token"]]
        res = {"token": smp["token"], "layers": smp["layers"], "select_exact": True,
               "mlp_max_abs_err": 0.0, "mlp_within_tol": True}
        for i, l in enumerate(smp["layers"]):
            _, ids1 = oracle.select(smp["scores"][i:i + 1], bc.k)
            res["select_exact"] &= bool(np.array_equal(ids1[0], smp["ids"][i]))
            rec = W.storage(bc, l, 1)  # the layer's records, regenerated
            _, ref64 = oracle.sparse_mlp(bc, 0, hb, rec, smp["ids"][i], want_f64=True)
            got = (smp["y"][i].astype(np.float64) if bc.adtype == "f32"
                   else oracle.decode(bc.adtype, smp["y"][i]))
            err = np.abs(got - ref64)
            res["mlp_max_abs_err"] = max(res["mlp_max_abs_err"], float(np.max(err)))
            res["mlp_within_tol"] &= bool(np.all(err <= mlp_tol(bc.adtype, ref64)))
        res["mlp_max_abs_err"] = float(f"{res['mlp_max_abs_err']:.3g}")
        res["ok"] = bool(res["select_exact"] and res["mlp_within_tol"])
        checks.setdefault("sampled", {})[bc.name] = res
    if gpu_ref:
        checks["scores_max_rel_diff"] = float(f"{checks['scores_max_rel_diff']:.3g}")
        checks["mlp_max_abs_err"] = float(f"{checks['mlp_max_abs_err']:.3g}")
        checks["ok"] = bool(checks["select_exact"] and checks["delta_exact"] and
                            checks["slot_maps_exact"] and checks["mlp_within_tol"] and
                            all(v["ok"] for v in checks.get("sampled", {}).values()))
        out["parity"] = checks
    return out


def pinned_host_summary(main_name, host, big, extra) -> dict | None:
    """The end-to-end rate of the decode step with the storage tier in pinned
    host memory and np_stage_rows staging (the step's stated tier for 13B and
    70B, where only part of the rows fits the resident buffer), per
    configuration: tokens/s of the faster np_stage_rows mode, its staging
    rate (between device events, and as the host sees it) and the same run's
    pinned-copy peak.  PCIe-inclusive; the headline
    `value` keeps the storage tier in HBM."""
    rows = {}
    for name, h in [(main_name, host)] + [(n, (v or {}).get("host_tier"))
                                          for n, v in {**big, **extra}.items()]:
        if h:
            rows[name] = {"tok_s": h["tok_s"], "staging_GBps": h["staging_GBps"],
                          "h2d_peak_GBps": h["h2d_peak_GBps"], "mode": h["mode"]}
            for key in ("staging_timed_by", "host_observed_staging_GBps", "layers",
                        "ms_per_layer", "note"):
                if key in h:
                    rows[name][key] = h[key]
    return rows or None


def cpu_detail() -> dict:
    """Family, model, stepping, clock and cache of the first host CPU (from
    /proc/cpuinfo), and the CPUs this process may run on."""
    keys = {"cpu family": "family", "model": "model", "stepping": "stepping",
            "cpu MHz": "mhz", "cache size": "cache"}
    out = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break
                k, _, v = line.partition(":")
                if k.strip() in keys:
                    out[keys[k.strip()]] = v.strip()
    except OSError:
        pass
    if hasattr(os, "sched_getaffinity"):
        out["usable_cpus"] = len(os.sched_getaffinity(0))
    return out


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="7b")
    ap.add_argument("--overlap", type=int, default=0,
                    help="stage on a side stream in layer chunks (measured slower: each "
                         "cross-stream event costs about 10 us on the GPU)")
    ap.add_argument("--host-tier-steps", type=int, default=20)
    ap.add_argument("--fill-tokens", type=int, default=64,
                    help="untimed tokens after the warmup that fill the resident buffer, so "
                         "that every timed token of the decode step evicts (steady state)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--breakdown-steps", type=int, default=10)
    ap.add_argument("--mlp-steps", type=int, default=50)
    ap.add_argument("--parity-tokens", type=int, default=3,
                    help="first tokens checked against the oracle in its leg")
    ap.add_argument("--hbm-configs", default="70b",
                    help="configurations run at full size with every tier in HBM")
    ap.add_argument("--hbm-steps", type=int, default=20)
    ap.add_argument("--extra-configs", default="13b",
                    help="comma-separated further configurations measured after the main one")
    ap.add_argument("--extra-steps", type=int, default=30)
    ap.add_argument("--dense-prefixes", default="0,8,16",
                    help="comma-separated dense-prefix lengths for the split sweep ('' to skip)")
    ap.add_argument("--dense-steps", type=int, default=10)
    ap.add_argument("--dense-reps", type=int, default=3,
                    help="timed passes of the dense-MLP roofline over all layers (0: skip)")
    ap.add_argument("--centroid-steps", type=int, default=30,
                    help="steps with the centroid-ID predictor (0: skip)")
    ap.add_argument("--sweep-steps", type=int, default=10,
                    help="steps per point of the 7B sweep (0: skip; 7B configuration only)")
    ap.add_argument("--file-tier-steps", type=int, default=10,
                    help="steps with the storage tier in a local file (0: skip)")
    ap.add_argument("--swiglu-steps", type=int, default=30,
                    help="steps of the SwiGLU 7B shape with calibrated eq. 1 thresholds (0: skip)")
    ap.add_argument("--calib-mib", type=int, default=256,
                    help="size of one plain device-to-device copy run after the timing, "
                         "the reference for hardware byte counters")
    ap.add_argument("--graph", type=int, default=0,
                    help="time the step replayed from a captured HIP graph (default: eager "
                         "launches, which need no per-token input copy; the graph's rate is "
                         "reported as graph_tok_s)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the hot path here is measured on one GPU)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_22643_amd import workload as W
    from paper_2608_22643_amd.pipeline import DecodePipeline

    cfg = W.get(args.config)
    K, Wm = args.steps, args.warmup
    Fl = args.fill_tokens
    T = (1 + Wm + Fl + 2 * K + args.mlp_steps + args.breakdown_steps + 16 +
         4 + Fl + 2 * args.host_tier_steps + 8)
    log(f"[bench] config {cfg.name}: L'={cfg.layers} d={cfg.d_model} F={cfg.d_ffn} r={cfg.rank} "
        f"k={cfg.k} C={cfg.capacity} {cfg.wdtype}; tokens {T}")
    t = time.perf_counter()
    host_storage = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
    W.fill_storage(cfg, host_storage.data_ptr())
    log(f"[bench] storage tier generated: {cfg.storage_bytes / 1e9:.2f} GB in "
        f"{time.perf_counter() - t:.1f} s")
    pipe = DecodePipeline(cfg, tier="device", staging="gather", overlap=bool(args.overlap),
                          tokens=T, host_storage=host_storage)
    log("[bench] pipeline ready (storage tier in HBM)")
    graph = bool(args.graph)
    if graph:
        pipe.capture_graph()
        log("[bench] decode step captured as a HIP graph")
    step = pipe.step_graph if graph else pipe.step
    # cold start, then warmup; the first tokens' outputs are kept for the
    # parity check of the oracle leg
    gpu_ref = []
    keep = args.parity_tokens if args.cpu_seconds > 0 else 0
    torch.cuda.synchronize()
    c0 = time.perf_counter()
    step(0)
    torch.cuda.synchronize()
    cold_ms = (time.perf_counter() - c0) * 1e3
    if keep > 0:
        gpu_ref.append(capture_outputs(pipe))
    for i in range(Wm):
        step(1 + i)
        if len(gpu_ref) < keep:
            torch.cuda.synchronize()
            gpu_ref.append(capture_outputs(pipe))
    # the resident buffer filled to steady state before the timed steps (with
    # the default fill every timed token evicts, as in a long decode)
    for i in range(Fl):
        step(1 + Wm + i)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({Wm} warmup + {Fl} fill tokens)")
    t0 = 1 + Wm + Fl
    if graph:
        wall = timed_graph_steps(pipe, t0, K)
    else:
        wall, _ = timed_steps(pipe, t0, K, with_mlp_events=False)
    log(f"[bench] timed {K} steps ({'graph' if graph else 'eager'}): {wall * 1e3 / K:.3f} ms/step")
    t1 = t0 + K
    other_ms = None
    if graph:  # the same steps launched one call at a time, for comparison
        ew, _ = timed_steps(pipe, t1, K, with_mlp_events=False)
        other_ms = ew * 1e3 / K
        log(f"[bench] eager launches: {other_ms:.3f} ms/step")
        t1 += K
    else:  # the same steps replayed from a graph (a second pipeline from token 0)
        gp = DecodePipeline(cfg, tier="device", staging="gather", overlap=bool(args.overlap),
                            tokens=T, host_storage=host_storage)
        gp.capture_graph()
        for i in range(t0):
            gp.step_graph(i)
        other_ms = timed_graph_steps(gp, t0, K) * 1e3 / K
        log(f"[bench] graph replay: {other_ms:.3f} ms/step")
        del gp
        torch.cuda.empty_cache()
    # sparse-MLP roofline: further steps, each token's block of calls
    # bracketed by events (staging of the token finished before the block)
    trace_marker()
    step_list = []
    _, mlp_us = timed_steps(pipe, t1, args.mlp_steps, step_us=step_list)
    trace_marker()
    step_pct = {"p50": round(float(np.percentile(step_list, 50)), 2),
                "p99": round(float(np.percentile(step_list, 99)), 2), "tokens": len(step_list),
                "note": "device time per token, np_predict start to last np_sparse_mlp end"}
    log(f"[bench] np_sparse_mlp: {mlp_us:.2f} us per call")
    floor = mlp_dispatch_floor(pipe)
    log(f"[bench] np_sparse_mlp with no rows: {floor}")
    same_layer = mlp_same_layer(pipe)
    log(f"[bench] np_sparse_mlp on one layer repeated: {same_layer}")
    err = pipe.device_error()
    if err:
        log(f"[bench] device error word {err:#x}")
        sys.exit(1)
    ms_per_step = wall * 1e3 / K
    bytes_launch = mlp_bytes_per_launch(cfg)
    traffic, traffic_detail = mlp_traffic(cfg)
    achieved = bytes_launch / (mlp_us * 1e-6) / 1e9
    # per-phase breakdown (no overlap) and delta statistics over its tokens
    t1 += args.mlp_steps
    bd, per_tok, ids = breakdown(pipe, t1, max(2, args.breakdown_steps))
    log(f"[bench] breakdown us: {bd}")
    pbytes = predict_bytes(cfg)
    predictor = predictor_paths(pipe, t1, pbytes)
    log(f"[bench] predictor: {predictor}")
    sd_calls = select_delta_calls(pipe, t1 + max(2, args.breakdown_steps))
    log(f"[bench] select/delta per call: {sd_calls}")
    n_in = np.mean([c[:, 0].sum() for c in per_tok])
    n_hit = np.mean([c[:, 1].sum() for c in per_tok])
    rec = cfg.record_bytes
    stats = {"incoming_rows_per_token": round(float(n_in), 1),
             "staged_MB_per_token": round(float(n_in) * rec / 1e6, 2),
             "reuse_pct": round(100.0 * float(n_hit) / (cfg.k * cfg.layers), 2),
             "persistence_pct": round(100.0 * persistence_of(ids), 2),
             "tokens": len(per_tok)}
    del pipe
    torch.cuda.empty_cache()
    # storage tier in pinned host memory: the PCIe-inclusive rate
    host = None
    if args.host_tier_steps > 0:
        host = pinned_host_run(cfg, host_storage, args.host_tier_steps, T, 0, Fl)
        host["note"] = "storage tier in pinned host memory; staging crosses the host link"
        log(f"[bench] host tier: {host}")
    sweep7b = None
    if args.sweep_steps > 0 and cfg.name == "7b":
        sweep7b = sweep_run(host_storage, args.sweep_steps)
        log(f"[bench] 7B sweep: {sweep7b}")
    file_tier = None
    if args.file_tier_steps > 0:
        file_tier = file_tier_run(cfg, host_storage, args.file_tier_steps)
        log(f"[bench] file tier: {file_tier}")
    dense = dense_mlp_roofline(cfg, host_storage, args.dense_reps) if args.dense_reps > 0 else None
    if dense:
        log(f"[bench] dense MLP: {dense}")
    sweep = None
    prefixes = [int(v) for v in args.dense_prefixes.split(",") if v]
    if prefixes:
        sweep = dense_prefix_sweep(cfg, host_storage, prefixes, args.dense_steps)
    centroid = None
    if args.centroid_steps > 0:
        centroid = centroid_run(cfg, host_storage, args.centroid_steps)
        log(f"[bench] centroid predictor: {centroid}")
    swiglu = None
    if args.swiglu_steps > 0:
        swiglu = swiglu_run(args.swiglu_steps)
        log(f"[bench] swiglu: {swiglu}")
    if args.calib_mib > 0:  # a copy of known size: reads and writes calib_mib MiB once
        src = torch.ones(args.calib_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    read_ref = round(read_ref_gbps(), 1)
    log(f"[bench] read reference: {read_ref} GB/s")
    read_call = read_ref_per_call(mlp_bytes_per_launch(cfg), cfg.layers)
    log(f"[bench] read reference per call: {read_call}")
    big, big_samples = {}, []
    for name in [n for n in args.hbm_configs.split(",") if n]:
        big[name], smp = hbm_config_run(name, args.hbm_steps, Fl)
        big_samples.append(smp)
        log(f"[bench] {name}: {big[name]}")
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(cfg, host_storage, args.cpu_seconds, gpu_ref, big_samples)
        log(f"[bench] cpu baseline: {cpu}")
    extra = {}
    for name in [n for n in args.extra_configs.split(",") if n]:
        del host_storage
        host_storage = None
        extra[name] = extra_config(name, args.extra_steps, graph, bool(args.overlap), Fl)
        log(f"[bench] {name}: {extra[name]}")
    line = {
        "metric": "sparse-MLP decode tokens/sec + achieved HBM GB/s (% peak), 7B-shaped, batch 1",
        "value": round(1e3 / ms_per_step, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.wdtype,
        "data": "synthetic (seeded generator; no model weights or datasets)",
        "config": {"workload": f"{cfg.name}-shaped decode: {cfg.layers} downstream layers, "
                               f"d={cfg.d_model}, F={cfg.d_ffn}, rank {cfg.rank}, k={cfg.k} "
                               f"({cfg.active_frac:.0%}), C={cfg.capacity} "
                               f"({cfg.resident_frac:.0%}), {cfg.wdtype}, batch 1",
                   "storage_tier": "HBM", "staging": "np_stage_gather",
                   "resident_buffer": f"full: {Fl} untimed fill tokens after the warmup, so "
                                      f"every timed token evicts" if Fl >= 64 else
                                      f"{Fl} untimed fill tokens after the warmup",
                   "overlap": bool(args.overlap),
                   "launch": "hip_graph" if graph else "eager"},
        "roofline": {"bound": "hbm", "kernel": "np_sparse_mlp",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "traffic_detail": traffic_detail,
                     "bytes_per_launch": bytes_launch, "avg_launch_us": round(mlp_us, 3),
                     "frac_of_read_ref": round(achieved / read_ref, 4),
                     "empty_call": floor, "same_layer": same_layer,
                     "read_ref_per_call": read_call,
                     "speedup_vs_read_ref_per_call": round(read_call["us_per_call"] / mlp_us, 3)},
        "step_us": step_pct,
        "predictor": predictor,
        "read_ref": {"GBps": read_ref, "kernel": "torch.mv (library GEMV) over a 2 GiB [262144][4096] fp16 matrix"},
        ("eager_tok_s" if graph else "graph_tok_s"): round(1e3 / other_ms, 2),
        "sparse_mlp_tok_s": round(1e6 / (mlp_us * cfg.layers), 1),
        "cold_start_ms": round(cold_ms, 2),
        "breakdown_us": bd,
        "select_delta_per_call": sd_calls,
        "delta": stats,
        "end_to_end_pinned_host": pinned_host_summary(cfg.name, host, big, extra),
        "host_tier": host,
        "file_tier": file_tier,
        "sweep_7b": sweep7b,
        "cpu_baseline": cpu,
        "parity": (cpu or {}).get("parity"),
        "dense_mlp": dense,
        "dense_prefix_sweep": sweep,
        "centroid_predictor": centroid,
        "swiglu_7b": swiglu,
        "other_configs": {**big, **extra} or None,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
