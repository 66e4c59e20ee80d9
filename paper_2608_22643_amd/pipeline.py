"""Per-token decode loop over the C ABI (the runtime around the kernels).

DecodePipeline owns the device buffers of one configuration (torch
allocations: PyTorch supplies memory and streams only) and runs one decode
token per step():

    np_predict -> np_select -> np_delta -> staging -> np_sparse_mlp x L'

Staging modes:
  "gather"  np_stage_gather straight from np_delta's device lists; the storage
            tier is device memory ("device" tier) or mapped pinned host memory
            ("host" tier, read over the host link by the kernel).  No host
            synchronisation anywhere in the step.
  "memcpy"  np_stage_rows: the delta's plan (counts, incoming ids and slots)
            is copied to pinned host memory, the host packs coalesced records
            into pinned staging pieces and each piece (records and their
            destination rows) goes over with one hipMemcpyAsync on a side
            stream, then a scatter kernel places its records.  Needs the
            "host" tier.
  "file"    np_stage_file: as "memcpy", but the coalesced records are read
            from the storage tier in a file (tier "file"; O_DIRECT when the
            record size allows) through io_uring, up to 256 reads in flight
            (Sec. 3.5).  The file is written once at set-up (storage_path, or
            a temporary file removed by close()).

The MLP's gated form follows cfg.act (ReLU-gated or SwiGLU).  With
thresholds (one per downstream layer, e.g. from calibrate.thresholds) every
sparse layer applies eq. 1 to its active rows (np_sparse_mlp_t).

With dense_layers = d > 0, d dense-prefix layers (all F records of each kept
resident, Sec. 3.1) run with np_dense_mlp, enqueued right after the delta and
before staging starts, so the GPU computes them while the host reads and
stages the sparse layers' rows.

With overlap=True staging runs in layer groups (layer 0, layers 1-2, then
four layers at a time) on a side stream, each group followed by events, and
layer l's MLP waits only for the group holding layer l: staging later layers
overlaps the MLPs of earlier ones.  Gather staging puts the first group on the
main stream; host staging (memcpy, file) calls np_stage_rows / np_stage_file
once per group and hands that group's MLPs to a helper thread right after
the call, so they run while the host packs the next group; with memcpy
staging every gather_every-th group (the second, the sixth, ...) is instead
copied by np_stage_gather from the pinned tier on a second side stream, the
GPU reading it over the host link while the host packs.  The side stream waits for np_delta
of the same token, which itself follows the previous token's MLP on the main
stream, so a victim slot is never overwritten while the previous token still
reads it.

Graph mode (capture_graph / step_graph): one decode step is captured once as
a HIP graph and replayed per token.  The step then has no per-token argument:
the graph's first nodes copy h_t into a fixed input buffer, t taken from a
device-side row index that its last node advances, and np_delta takes the
token index from the workspace step counter (NP_TOKEN_AUTO), which
np_state_reset sets to 0, so graph tokens must start at a cold start (t = 0)
and run in order.  Only "gather" staging can be captured (np_stage_rows waits
on the host for the plan).
"""
from __future__ import annotations

import time

import numpy as np
import torch

from . import binding as B
from . import workload as W

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _i32(n, device):
    return torch.empty(n, dtype=torch.int32, device=device)


_MLP_POOL = None


def _mlp_pool():
    """One helper thread per process that enqueues MLP groups in order."""
    global _MLP_POOL
    if _MLP_POOL is None:
        from concurrent.futures import ThreadPoolExecutor

        _MLP_POOL = ThreadPoolExecutor(max_workers=1, thread_name_prefix="np-mlp-enqueue")
    return _MLP_POOL


class DecodePipeline:
    def __init__(self, cfg: W.Config, device: str = "cuda:0", tier: str = "device",
                 staging: str = "gather", overlap: bool = False, tokens: int | None = None,
                 staging_mib: float = 64, landing_mib: float = 128,
                 host_storage: torch.Tensor | None = None, predictor: str = "lowrank",
                 dense_layers: int = 0, thresholds=None, storage_path: str | None = None):
        if predictor not in ("lowrank", "centroid"):
            raise ValueError(f"unknown predictor {predictor!r}")
        if dense_layers < 0:
            raise ValueError("dense_layers must be >= 0")
        self.predictor = predictor
        self.dense_layers = dense_layers
        if staging == "memcpy" and tier != "host":
            raise ValueError("memcpy staging reads a pinned host storage tier")
        if (staging == "file") != (tier == "file"):
            raise ValueError("the file tier is staged with staging='file' and only so")
        self.storage_fd, self.storage_path, self._own_file = -1, None, False
        self.cfg, self.device, self.tier, self.staging, self.overlap = cfg, device, tier, staging, overlap
        torch.cuda.set_device(device)
        L, d, F, r, k, C = cfg.layers, cfg.d_model, cfg.d_ffn, cfg.rank, cfg.k, cfg.capacity
        self.shape = B.make_shape(L, d, F, r, k, C, cfg.wdtype, cfg.adtype, cfg.act)
        B.np_shape_check(self.shape)
        self.thr = None  # eq. 1 thresholds, device float32 [L']
        if thresholds is not None:
            self.set_thresholds(thresholds)
        self.T = cfg.tokens if tokens is None else tokens
        dev = torch.device(device)
        # inputs resident in HBM: predictor factors and hidden states
        self.A = self.B = None
        if predictor == "lowrank":
            A, Bm = W.predictor(cfg)
            self.A = torch.from_numpy(A.view(np.uint8)).to(dev)
            self.B = torch.from_numpy(Bm.view(np.uint8)).to(dev)
        h = W.hidden(cfg, self.T)
        self.h = torch.from_numpy(h.view(np.uint8).reshape(self.T, -1)).to(dev)
        self.row_bytes = d * W.ITEMSIZE[cfg.adtype]
        # storage tier (host_storage: an already generated pinned copy to reuse)
        if host_storage is not None:
            assert host_storage.numel() == cfg.storage_bytes and host_storage.is_pinned()
        if tier == "host":
            if host_storage is not None:
                self.storage = host_storage
            else:
                self.storage = torch.empty(cfg.storage_bytes, dtype=torch.uint8, pin_memory=True)
                W.fill_storage(cfg, self.storage.data_ptr())
        elif tier == "file":
            self.storage = None
            self._open_storage_file(storage_path, host_storage)
        else:
            self.storage = torch.empty(cfg.storage_bytes, dtype=torch.uint8, device=dev)
            if host_storage is not None:
                self.storage.copy_(host_storage)
            else:
                layer_bytes = F * cfg.record_bytes
                buf = torch.empty(layer_bytes, dtype=torch.uint8, pin_memory=True)
                for l in range(L):
                    W.fill_storage(cfg, buf.data_ptr(), l, 1)
                    self.storage[l * layer_bytes:(l + 1) * layer_bytes].copy_(buf)
                torch.cuda.synchronize()
                del buf
            torch.cuda.synchronize()
        self.resident = torch.empty(cfg.resident_bytes, dtype=torch.uint8, device=dev)
        # dense prefix (Sec. 3.1): dense_layers layers with all F records resident
        if dense_layers:
            dcfg = W.dense_config(cfg, dense_layers)
            self.dense_layer_bytes = F * cfg.record_bytes
            self.dense_w = torch.empty(dense_layers * self.dense_layer_bytes, dtype=torch.uint8,
                                       device=dev)
            buf = torch.empty(self.dense_layer_bytes, dtype=torch.uint8, pin_memory=True)
            for l in range(dense_layers):
                W.fill_storage(dcfg, buf.data_ptr(), l, 1)
                self.dense_w[l * self.dense_layer_bytes:(l + 1) * self.dense_layer_bytes].copy_(buf)
            torch.cuda.synchronize()
            del buf
            self.y_dense = torch.empty(dense_layers * d, dtype=TORCH_DT[cfg.adtype], device=dev)
        # residency state and step outputs
        self.slot_of, self.neuron_of, self.last_used = _i32(L * F, dev), _i32(L * C, dev), _i32(L * F, dev)
        self.state = B.np_state(self.slot_of.data_ptr(), self.neuron_of.data_ptr(),
                                self.last_used.data_ptr())
        # the staging plan (counts, in_ids, in_slots) in one block, each part
        # at a 16-byte boundary, so the host reads it with one copy
        kp = (L * k + 3) // 4 * 4
        self.plan_dev = _i32(L * 4 + 2 * kp, dev)
        self.counts = self.plan_dev[:L * 4]
        self.lists = {"in_ids": self.plan_dev[L * 4:L * 4 + L * k],
                      "in_slots": self.plan_dev[L * 4 + kp:L * 4 + kp + L * k]}
        self.lists.update({n: _i32(L * k, dev) for n in
                           ("ev_ids", "ev_slots", "hit_ids", "active_slots")})
        self.out = B.np_delta_out(*[self.lists[n].data_ptr() for n in
                                    ("in_ids", "in_slots", "ev_ids", "ev_slots", "hit_ids",
                                     "active_slots")], self.counts.data_ptr())
        self.scores = torch.empty(L * F, dtype=torch.float32, device=dev)
        self.words = (F + 31) // 32
        self.mask = _i32(L * self.words, dev)
        self.active_ids = _i32(L * k, dev)
        self.y = torch.empty(L * d, dtype=TORCH_DT[cfg.adtype], device=dev)
        if predictor == "centroid":  # Sec. 3.3-3.4: centroid heads and mask bank
            K, D = cfg.centroid_k, cfg.feat_dim
            self.heads = torch.from_numpy(W.centroid_heads(cfg).view(np.uint8).reshape(-1)).to(dev)
            self.bank = torch.from_numpy(W.centroid_bank(cfg).view(np.uint8).reshape(-1)).to(dev)
            f = W.features(cfg, self.T)
            self.feat = torch.from_numpy(f.view(np.uint8).reshape(self.T, -1)).to(dev)
            self.feat_bytes = D * W.ITEMSIZE[cfg.adtype]
            self.model = B.np_centroid_model(K, D, self.heads.data_ptr(), self.bank.data_ptr())
            self.logits = torch.empty(2 * L * K, dtype=torch.float32, device=dev)
            self.cids = _i32(max(2 * L, 4), dev)
            self.active_counts = _i32(max(L, 4), dev)
        self.ws = torch.zeros(B.np_workspace_size(self.shape), dtype=torch.uint8, device=dev)
        self.main = torch.cuda.Stream(device=dev)
        self.side = torch.cuda.Stream(device=dev) if overlap else self.main
        # host staging with overlap: every gather_every-th layer group
        # (starting with the second) is gathered by the GPU from the pinned
        # storage tier on a second side stream, the others packed by the host
        self.gather_every = 4 if (overlap and tier == "host" and staging == "memcpy") else 0
        self.side2 = torch.cuda.Stream(device=dev) if self.gather_every else None
        self.ev_delta = torch.cuda.Event()
        self.layer_ready = [torch.cuda.Event() for _ in range(L)] if overlap else None
        # staging groups of the overlapped paths: layer 0, layers 1-2, then
        # four layers at a time, so the first MLPs start early and each later
        # group's MLPs run while the next group is staged
        cuts = sorted({0, min(1, L), min(3, L), L} | set(range(3, L, 4)))
        self.chunks = list(zip(cuts[:-1], cuts[1:]))
        self.gather_ready = [torch.cuda.Event() for _ in self.chunks] if self.gather_every else None
        if staging in ("memcpy", "file"):
            self.plan_host = torch.empty(self.plan_dev.numel(), dtype=torch.int32,
                                         pin_memory=True)
            self.plan_counts = self.plan_host[:L * 4]
            self.plan_ids = self.plan_host[L * 4:L * 4 + L * k]
            self.plan_slots = self.plan_host[L * 4 + kp:L * 4 + kp + L * k]
            self.plan = B.np_stage_plan(self.plan_counts.data_ptr(), self.plan_ids.data_ptr(),
                                        self.plan_slots.data_ptr())
            self.staging_buf = torch.empty(int(staging_mib * (1 << 20)), dtype=torch.uint8,
                                           pin_memory=True)
            # file reads land in ordinary host memory (a direct read cannot
            # target pinned memory), one staging piece at a time
            self.io_buf = (B.HostBuffer(int(staging_mib * (1 << 20)) // 2) if staging == "file"
                           else None)
            self.landing = torch.empty(int(landing_mib * (1 << 20)), dtype=torch.uint8, device=dev)
            self.ev_plan = torch.cuda.Event()
            # events handed to the library must exist: record them once
            for e in (self.layer_ready or []):
                e.record(self.side)
            self.ev_delta.record(self.main)
            torch.cuda.synchronize()
        # test hooks: callables run with a stream, to enqueue a fixed-length
        # delay on the side stream just before a token's staging
        # (delay_side) or on the main stream just before its MLPs (delay_main)
        self.delay_side = self.delay_main = None
        # host staging with overlap: MLP groups enqueued by a helper thread
        self.mlp_thread = True
        # memcpy staging: when a list, each step appends (bytes staged, seconds
        # from the plan's arrival on the host to the end of the copies and
        # scatters, seconds spent in the staging calls) and waits for the
        # staging before it enqueues the MLPs
        self.stage_log = None
        self.reset()

    # ------------------------------------------------------------------
    def reset(self) -> None:
        """Cold start: every slot map entry -1 (the next token loads its
        whole active set)."""
        B.np_state_reset(self.shape, self.state, self.ws, self.main, self.resident)
        self.main.synchronize()

    def _check_token(self, t: int) -> None:
        if not 0 <= t < self.T:
            raise IndexError(f"token {t} outside the {self.T} tokens this pipeline holds")

    def x_ptr(self, t: int) -> int:
        self._check_token(t)
        return self.h.data_ptr() + t * self.row_bytes

    def f_ptr(self, t: int) -> int:
        self._check_token(t)
        return self.feat.data_ptr() + t * self.feat_bytes

    def step(self, t: int, mlp_block_events=None) -> None:
        """Enqueue one decode token (index t of the hidden-state sequence).
        mlp_block_events: optional (start, end) torch events recorded on the
        main stream before the first and after the last np_sparse_mlp."""
        f = self.f_ptr(t) if self.predictor == "centroid" else None
        self._enqueue(t, self.x_ptr(t), mlp_block_events, f)

    def capture_graph(self) -> None:
        """Capture one decode step (token index from the device counter, x
        from a fixed buffer) as a HIP graph.  Nothing runs until replay."""
        if self.staging != "gather":
            raise ValueError("only gather staging can be captured in a graph")
        self.x_static = torch.empty((1, self.row_bytes), dtype=torch.uint8, device=self.device)
        self.x_row = torch.zeros(1, dtype=torch.int64, device=self.device)  # next token's row of h
        self.graph_t = 0
        self.graph = torch.cuda.CUDAGraph()
        f_ptr = None
        if self.predictor == "centroid":
            self.f_static = torch.empty((1, self.feat_bytes), dtype=torch.uint8,
                                        device=self.device)
            f_ptr = self.f_static.data_ptr()
        with torch.cuda.graph(self.graph, stream=self.main, capture_error_mode="thread_local"):
            torch.index_select(self.h, 0, self.x_row, out=self.x_static)
            if f_ptr is not None:
                torch.index_select(self.feat, 0, self.x_row, out=self.f_static)
            self._enqueue(B.NP_TOKEN_AUTO, self.x_static.data_ptr(), None, f_ptr)
            self.x_row.add_(1)

    def step_graph(self, t: int) -> None:
        """Replay the captured step for token t (tokens 0, 1, 2, ... in order
        after a cold start)."""
        if t != self.graph_t:
            raise ValueError(f"graph tokens run in order from 0: expected {self.graph_t}, got {t}")
        self._check_token(t)  # the graph reads row t of the hidden states
        with torch.cuda.stream(self.main):
            self.graph.replay()
        self.graph_t += 1

    def _enqueue(self, token: int, x_ptr: int, mlp_block_events, f_ptr=None) -> None:
        s, cfg = self.shape, self.cfg
        L, k = cfg.layers, cfg.k
        main = self.main
        centroid = self.predictor == "centroid"
        if centroid:
            B.np_centroid_select(s, self.model, f_ptr, self.logits, self.cids, self.mask,
                                 self.active_ids, self.active_counts, self.ws, main)
            B.np_delta_n(s, token, self.active_ids, self.active_counts, self.state, self.out,
                         self.ws, main)
        else:
            B.np_predict(s, x_ptr, self.A, self.B, self.scores, self.ws, main)
            B.np_select_delta(s, token, self.scores, self.mask, self.active_ids, self.state,
                              self.out, self.ws, main)
        ready = None  # ready[l]: the event layer l's MLP waits for
        slots = self.lists["active_slots"]
        ybytes = cfg.d_model * W.ITEMSIZE[cfg.adtype]
        # the dense prefix: on the GPU while the host stages the sparse rows
        for l in range(self.dense_layers):
            B.np_dense_mlp(s, self.dense_w.data_ptr() + l * self.dense_layer_bytes, x_ptr,
                           self.y_dense.data_ptr() + l * ybytes, self.ws, main)
        def mlp(l):
            if self.thr is not None:
                B.np_sparse_mlp_t(s, l, x_ptr, self.resident, slots.data_ptr() + l * k * 4, k,
                                  self.active_counts if centroid else None, self.thr,
                                  self.y.data_ptr() + l * ybytes, self.ws, main)
            elif centroid:
                B.np_sparse_mlp_n(s, l, x_ptr, self.resident, slots.data_ptr() + l * k * 4,
                                  self.active_counts, self.y.data_ptr() + l * ybytes, self.ws,
                                  main)
            else:
                B.np_sparse_mlp(s, l, x_ptr, self.resident, slots.data_ptr() + l * k * 4, k,
                                self.y.data_ptr() + l * ybytes, self.ws, main)

        if self.staging == "gather":
            if self.overlap:
                # the first chunk on the main stream (the first MLP follows it
                # in stream order), the others on the side stream
                lb0, le0 = self.chunks[0]
                B.np_stage_gather(s, self.out, lb0, le0, self.storage, self.resident, self.ws, main)
                self.ev_delta.record(main)
                self.side.wait_event(self.ev_delta)
                if self.delay_side is not None:
                    self.delay_side(self.side)
                ready = [None] * L
                for lb, le in self.chunks[1:]:
                    B.np_stage_gather(s, self.out, lb, le, self.storage, self.resident,
                                      self.ws, self.side)
                    self.layer_ready[lb].record(self.side)
                    ready[lb] = self.layer_ready[lb]
            else:
                B.np_stage_gather(s, self.out, 0, L, self.storage, self.resident, self.ws, main)
            if mlp_block_events is not None:
                for e in (ready or []):  # time the MLP block, not the wait for staging
                    if e is not None:
                        main.wait_event(e)
                mlp_block_events[0].record(main)
            if self.delay_main is not None:
                self.delay_main(main)
            for l in range(L):
                if ready is not None and ready[l] is not None:
                    main.wait_event(ready[l])
                mlp(l)
            if mlp_block_events is not None:
                mlp_block_events[1].record(main)
            return
        # staging through the host: the plan is read on the host first
        with torch.cuda.stream(main):
            self.plan_host.copy_(self.plan_dev, non_blocking=True)
        self.ev_plan.record(main)
        self.ev_plan.synchronize()  # the host reads the plan
        t0 = time.perf_counter()
        t_call = 0.0
        # with overlap, staging runs on the side stream one layer group at a
        # time and each group's MLPs are enqueued once its staging call has
        # returned, so they run while the host packs the next groups
        groups = self.chunks if self.overlap else [(0, L)]
        if self.delay_side is not None:
            self.delay_side(self.side)
        if self.delay_main is not None:
            self.delay_main(main)
        # with overlap, a helper thread enqueues each group's MLPs while this
        # thread packs the next groups (the library calls release the
        # interpreter lock): packing is the host's critical path
        helper = self.overlap and self.stage_log is None and self.mlp_thread
        futs = []

        def enqueue_group(lb, le, ev=None):
            for l in range(lb, le):
                # one wait per group, on its last layer's event: a group's
                # layers land with one or two staging pieces, and each wait
                # costs the main stream several microseconds (7B: 460 against
                # 405 tokens/s with a wait per layer)
                if self.overlap and l == lb:
                    main.wait_event(ev if ev is not None else self.layer_ready[le - 1])
                if l == 0 and mlp_block_events is not None:
                    mlp_block_events[0].record(main)
                mlp(l)

        # the GPU-gathered groups go first, on their own stream: the GPU reads
        # their records over the link while the host packs the other groups
        # (7B: 773-777 against 711-715 tokens/s with every group packed; 13B:
        # 472 against 445-448; every second group gathered is slower)
        gathered = set()
        if self.gather_every and self.stage_log is None:
            gathered = {gi for gi in range(len(groups)) if gi % self.gather_every == 1}
            if gathered:
                self.side2.wait_event(self.ev_plan)  # after the delta and the previous MLPs
                if self.delay_side is not None:
                    self.delay_side(self.side2)
                for gi in sorted(gathered):
                    lb, le = groups[gi]
                    B.np_stage_gather(s, self.out, lb, le, self.storage, self.resident, self.ws,
                                      self.side2)
                    self.gather_ready[gi].record(self.side2)
        try:
            for gi, (lb, le) in enumerate(groups):
                if gi in gathered:
                    if helper:
                        futs.append(_mlp_pool().submit(enqueue_group, lb, le,
                                                       self.gather_ready[gi]))
                    else:
                        enqueue_group(lb, le, self.gather_ready[gi])
                    continue
                wait = self.ev_plan if (self.overlap and gi == 0) else None
                tc = time.perf_counter()
                if self.staging == "file":
                    B.np_stage_file(s, self.plan, lb, le, self.storage_fd, 0, self.resident,
                                    self.staging_buf, self.staging_buf.numel(), self.io_buf,
                                    self.io_buf.nbytes, self.landing, self.landing.numel(),
                                    self.side, wait, self.layer_ready)
                else:
                    B.np_stage_rows(s, self.plan, lb, le, self.storage, self.resident,
                                    self.staging_buf, self.staging_buf.numel(), self.landing,
                                    self.landing.numel(), self.side, wait, self.layer_ready)
                t_call += time.perf_counter() - tc
                if self.stage_log is not None:
                    continue  # staging alone: the MLPs follow the whole staging
                if helper:  # the group's layer_ready events are recorded: hand it over
                    futs.append(_mlp_pool().submit(enqueue_group, lb, le))
                else:
                    enqueue_group(lb, le)
        finally:  # the helper has finished with this token's groups
            for fu in futs:
                fu.exception()
        for fu in futs:  # every MLP of this token is enqueued (errors re-raised)
            fu.result()
        if self.stage_log is not None:  # staging alone: host packing + copies + scatter
            if self.overlap:  # the scatters run on the library's scatter stream
                self.layer_ready[L - 1].synchronize()
            else:
                self.side.synchronize()
            n_rec = int(self.plan_counts.view(L, 4)[:, 0].sum())
            self.stage_log.append((n_rec * cfg.record_bytes, time.perf_counter() - t0, t_call))
            if self.overlap:  # every layer is staged: one wait
                main.wait_event(self.layer_ready[L - 1])
            for l in range(L):
                if l == 0 and mlp_block_events is not None:
                    mlp_block_events[0].record(main)
                mlp(l)
        if mlp_block_events is not None:
            mlp_block_events[1].record(main)

    def _open_storage_file(self, path, host_storage) -> None:
        """Writes the storage tier ([L'][F][3d] records, layer-major: the
        neuron-centric file layout of Sec. 3.5) to `path` (a temporary file
        when None) and opens it for np_stage_file, with O_DIRECT when the
        record size is a multiple of 512 bytes."""
        import os
        import tempfile

        cfg = self.cfg
        if path is None:
            d = os.environ.get("NP_STORAGE_DIR") or tempfile.gettempdir()
            fd, path = tempfile.mkstemp(prefix="np_storage_", suffix=".bin", dir=d)
            os.close(fd)
            self._own_file = True
        self.storage_path = path
        if not (os.path.exists(path) and os.path.getsize(path) == cfg.storage_bytes):
            layer_bytes = cfg.d_ffn * cfg.record_bytes
            with open(path, "wb") as f:
                if host_storage is not None:
                    f.write(memoryview(host_storage.numpy()))
                else:
                    buf = np.empty(layer_bytes, dtype=np.uint8)
                    for l in range(cfg.layers):
                        W.fill_storage(cfg, buf.ctypes.data, l, 1)
                        f.write(memoryview(buf))
                f.flush()
                os.fsync(f.fileno())  # on the device before any timed read
        direct = cfg.record_bytes % 512 == 0
        self.storage_fd = os.open(path, os.O_RDONLY | (os.O_DIRECT if direct else 0))
        self.storage_direct = direct

    def close(self) -> None:
        """Closes the storage file (and removes it if the pipeline made it)."""
        import os

        if self.storage_fd >= 0:
            os.close(self.storage_fd)
            self.storage_fd = -1
            if self._own_file and self.storage_path:
                os.remove(self.storage_path)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_thresholds(self, thresholds) -> None:
        """Eq. 1 thresholds of the downstream layers (float32 [L'], host or
        device); every later step applies them.  Not for a captured graph:
        set them before capture_graph."""
        t = torch.as_tensor(thresholds, dtype=torch.float32).reshape(-1)
        if t.numel() != self.cfg.layers:
            raise ValueError(f"need {self.cfg.layers} thresholds, got {t.numel()}")
        self.thr = t.to(self.device).contiguous()

    def device_error(self) -> int:
        return B.np_device_error(self.ws, self.main)

    # host copies for checks -------------------------------------------
    def host_state(self):
        L, F, C = self.cfg.layers, self.cfg.d_ffn, self.cfg.capacity
        return (self.slot_of.cpu().numpy().reshape(L, F), self.neuron_of.cpu().numpy().reshape(L, C),
                self.last_used.cpu().numpy().reshape(L, F))

    def host_lists(self):
        L, k = self.cfg.layers, self.cfg.k
        d = {n: v.cpu().numpy().reshape(L, k) for n, v in self.lists.items()}
        d["counts"] = self.counts.cpu().numpy().reshape(L, 4)
        return d
