"""Device buffers and round drivers over the C ABI (used by tests, bench, smoke).

Torch provides device memory, pinned host memory and streams only; every step
of the round runs in libspecstream's kernels through the binding.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import torch

from . import specstream as ss
from .workloads import Workload

BF16_BYTES = 2


class RoundBuffers:
    """Queries, candidate K/V, workspace and outputs of one layer's round."""

    def __init__(self, w: Workload, layer: int = 0, device="cuda", split_tokens: int = 0,
                 mfma_min_rows: int = 0, max_chunk_tokens: Optional[int] = None,
                 kv_layout: int = ss.SS_KV_TOKEN_MAJOR, balance_permille: int = 0, counters_zeroed: int = 0):
        self.w = w
        self.layer = layer
        self.device = device
        self.q = w.q_all(layer, device)
        self.kc = w.k_cand_all(layer, device)
        self.vc = w.v_cand_all(layer, device)
        mct = max_chunk_tokens or max(1, max(sum(w.chunk_lens(j)) for j in range(max(1, w.num_chunks))))
        self.kv_layout = kv_layout
        self.desc = ss.make_desc(w.num_cand, w.num_q_heads, w.num_kv_heads, w.head_dim, w.softmax_scale,
                                 mct, split_tokens, mfma_min_rows, kv_layout, balance_permille, counters_zeroed)
        self.ws_bytes = ss.ss_round_workspace_bytes(self.desc)
        if self.ws_bytes == 0:
            raise ss.SpecStreamError(ss.SS_ERR_INVALID_ARGUMENT, "ss_round_workspace_bytes", ss.ss_last_error())
        # with counters_zeroed the rounds rely on the workspace's counter block being zero: zero-fill it once
        alloc = torch.zeros if counters_zeroed else torch.empty
        self.ws = alloc(self.ws_bytes, dtype=torch.uint8, device=device)
        rows = w.total_rows
        self.out = torch.empty(rows, w.num_q_heads, w.head_dim, dtype=torch.float32, device=device)
        self.lse = torch.empty(rows, w.num_q_heads, dtype=torch.float32, device=device)

    def set_layer(self, layer: int) -> None:
        """New per-layer queries (candidates and history are shared by layers)."""
        self.layer = layer
        self.q.copy_(self.w.q_all(layer, self.device))


def hbm_history(w: Workload, layer: int = 0, device="cuda", kv_layout: int = ss.SS_KV_TOKEN_MAJOR
                ) -> List[Tuple[torch.Tensor, torch.Tensor]]:
    """Every history chunk resident in device memory: [(k_j, v_j)] in the
    given chunk layout."""
    return [w.chunk_kv(j, layer, device, head_major=kv_layout == ss.SS_KV_HEAD_MAJOR,
                       kv_interleaved=kv_layout == ss.SS_KV_HEAD_MAJOR_KV) for j in range(w.num_chunks)]


def run_round(b: RoundBuffers, chunks: Sequence[Tuple[torch.Tensor, torch.Tensor]], stream: int,
              order: Optional[Sequence[int]] = None, cand_position: Optional[int] = None,
              lens: Optional[Sequence[Sequence[int]]] = None, batch: int = 1, scratch: bool = False) -> None:
    """Enqueue one whole round (init, history chunks, candidates, finalize)
    on `stream`; results land in b.out / b.lse.  ``batch`` > 1 groups that
    many consecutive chunks into one ss_attend_history_chunks call.  With
    ``scratch`` the round starts with ss_round_init_scratch (the
    library's own workspace) instead of b.ws."""
    w = b.w
    order = list(range(len(chunks))) if order is None else list(order)
    pos = len(order) if cand_position is None else cand_position
    step = max(1, batch)
    groups = [order[i0:i0 + step] for i0 in range(0, len(order), step)]
    if scratch:
        r = ss.ss_round_init_scratch(b.desc, b.q.data_ptr(), stream)
    else:
        r = ss.ss_round_init(b.desc, b.q.data_ptr(), b.ws.data_ptr(), b.ws_bytes, stream)

    def args(grp):
        ks = [chunks[j][0].data_ptr() if chunks[j][0].numel() else 0 for j in grp]
        vs = [chunks[j][1].data_ptr() if chunks[j][1].numel() else 0 for j in grp]
        ls = [w.chunk_lens(j) if lens is None else lens[j] for j in grp]
        return ks, vs, ls

    try:
        done = 0
        for gi, grp in enumerate(groups):
            if done <= pos < done + len(grp) or (pos == done and gi == 0):
                ss.ss_attend_local_candidates(r, b.kc.data_ptr(), b.vc.data_ptr(), stream)
            ks, vs, ls = args(grp)
            if batch > 1:
                ss.ss_attend_history_chunks(r, ks, vs, ls, None, None, stream)
            else:
                ss.ss_attend_history_chunk(r, ks[0], vs[0], ls[0], None, None, stream)
            done += len(grp)
        if pos >= len(order):
            ss.ss_attend_local_candidates(r, b.kc.data_ptr(), b.vc.data_ptr(), stream)
        ss.ss_round_finalize(r, b.out.data_ptr(), b.lse.data_ptr(), stream)
    finally:
        ss.ss_round_destroy(r)


def capture_round(b: RoundBuffers, chunks: Sequence[Tuple[torch.Tensor, torch.Tensor]], batch: int = 1,
                  pool=None) -> "torch.cuda.CUDAGraph":
    """Capture one whole round (the same calls as run_round) into a HIP graph.

    Every step the library enqueues is a kernel launch with its arguments by
    value (no memsets, no host waits), so a replay redoes the round on the
    buffers it was captured with: b.q, b.kc, b.vc, the chunks, b.ws and
    b.out / b.lse.  Replays serve loops that re-run a round of the same
    shape with new contents in those buffers, without the host's per-call
    work."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, pool=pool):
        run_round(b, chunks, torch.cuda.current_stream().cuda_stream, batch=batch)
    return g


class HostHistory:
    """One layer's history in pinned host memory, chunk j as its K then its V
    (each in the round's chunk layout; with the interleaved layout the chunk's
    one K-and-V buffer), for streaming through the two-slot pipeline."""

    def __init__(self, w: Workload, layer: int = 0, gen_device="cuda", kv_layout: int = ss.SS_KV_TOKEN_MAJOR):
        self.w = w
        hm = kv_layout == ss.SS_KV_HEAD_MAJOR
        il = kv_layout == ss.SS_KV_HEAD_MAJOR_KV
        tb = w.num_kv_heads * w.head_dim * BF16_BYTES
        self.sizes = [2 * sum(w.chunk_lens(j)) * tb for j in range(w.num_chunks)]
        self.offsets = []
        acc = 0
        for s in self.sizes:
            self.offsets.append(acc)
            acc += s
        self.total_bytes = acc
        self.buf = torch.empty(max(1, acc), dtype=torch.uint8, pin_memory=True)
        for j in range(w.num_chunks):
            if self.sizes[j] == 0:
                continue
            k, v = w.chunk_kv(j, layer, gen_device, head_major=hm, kv_interleaved=il)
            half = self.sizes[j] // 2
            o = self.offsets[j]
            if il:      # one buffer: the views' base holds K and V rows
                kv = torch.as_strided(k, (self.sizes[j] // BF16_BYTES,), (1,))
                self.buf[o:o + 2 * half].copy_(kv.view(torch.uint8).cpu())
            else:
                self.buf[o:o + half].copy_(k.view(-1).view(torch.uint8).cpu())
                self.buf[o + half:o + 2 * half].copy_(v.view(-1).view(torch.uint8).cpu())
            del k, v

    def chunk_ptr(self, j: int) -> int:
        return self.buf.data_ptr() + self.offsets[j]

    def max_chunk_bytes(self) -> int:
        return max(self.sizes) if self.sizes else 0


class Pipeline:
    """The library's two-slot pipeline with its staging buffers and copy stream."""

    def __init__(self, slot_bytes: int, device="cuda"):
        self.slot_bytes = max(256, slot_bytes)
        self.staging = [torch.empty(self.slot_bytes, dtype=torch.uint8, device=device) for _ in range(2)]
        self.copy_stream = torch.cuda.Stream(device=device)          # default priority
        self.handle = ss.ss_pipeline_create(self.staging[0].data_ptr(), self.staging[1].data_ptr(),
                                            self.slot_bytes, self.copy_stream.cuda_stream)

    def close(self) -> None:
        if self.handle:
            torch.cuda.synchronize()
            ss.ss_pipeline_destroy(self.handle)
            self.handle = None


def batch_bytes(host: HostHistory, batch: int) -> int:
    """Largest staging slot a transfer batch of `batch` adjacent chunks needs."""
    n = len(host.sizes)
    return max([sum(host.sizes[j:j + batch]) for j in range(0, n, batch)] or [0])


def run_round_streamed(b: RoundBuffers, host: HostHistory, pipe: Pipeline, stream: int,
                       order: Optional[Sequence[int]] = None, batch: int = 1) -> None:
    """Enqueue one round whose history streams from pinned host memory; with
    ``batch`` > 1, groups of that many adjacent chunks travel as one transfer
    batch (one copy, one attention launch)."""
    w = b.w
    if batch > 1 and order is not None:
        raise ValueError("transfer batches take the chunks in their host order")
    order = list(range(w.num_chunks)) if order is None else list(order)
    r = ss.ss_round_init(b.desc, b.q.data_ptr(), b.ws.data_ptr(), b.ws_bytes, stream)
    try:
        if batch > 1:
            for j0 in range(0, w.num_chunks, batch):
                grp = range(j0, min(w.num_chunks, j0 + batch))
                ss.ss_pipeline_attend_chunks(pipe.handle, r, host.chunk_ptr(j0), [w.chunk_lens(j) for j in grp],
                                             stream)
        for j in (order if batch <= 1 else []):
            ss.ss_pipeline_attend_chunk(pipe.handle, r, host.chunk_ptr(j), w.chunk_lens(j), stream)
        ss.ss_attend_local_candidates(r, b.kc.data_ptr(), b.vc.data_ptr(), stream)
        ss.ss_round_finalize(r, b.out.data_ptr(), b.lse.data_ptr(), stream)
    finally:
        ss.ss_round_destroy(r)


def _chunk_vofs(w: Workload, host: HostHistory, j: int, kv_layout: int) -> int:
    """Bytes from a chunk's K to its V in a staging buffer holding the chunk."""
    return 2 * w.head_dim if kv_layout == ss.SS_KV_HEAD_MAJOR_KV else host.sizes[j] // 2


def run_round_restored(b: RoundBuffers, host: HostHistory, dev: Sequence[torch.Tensor], copy: "torch.cuda.Stream",
                       stream: int) -> None:
    """Restore, then attend: every chunk of the history goes to its own
    device buffer (``dev[j]``, at least host.sizes[j] bytes) on the copy
    stream, and one batched call attends all of them once the last upload is
    done."""
    w = b.w
    n = w.num_chunks
    done = ss.ss_event_create()
    try:
        last = max([j for j in range(n) if host.sizes[j]], default=-1)
        for j in range(n):
            if host.sizes[j]:
                ss.ss_upload_chunk(dev[j].data_ptr(), host.chunk_ptr(j), host.sizes[j], copy.cuda_stream, None,
                                   done if j == last else None)
        r = ss.ss_round_init(b.desc, b.q.data_ptr(), b.ws.data_ptr(), b.ws_bytes, stream)
        try:
            ks = [dev[j].data_ptr() for j in range(n)]
            vs = [dev[j].data_ptr() + _chunk_vofs(w, host, j, b.kv_layout) for j in range(n)]
            ss.ss_attend_history_chunks(r, ks, vs, [w.chunk_lens(j) for j in range(n)],
                                        done if last >= 0 else None, None, stream)
            ss.ss_attend_local_candidates(r, b.kc.data_ptr(), b.vc.data_ptr(), stream)
            ss.ss_round_finalize(r, b.out.data_ptr(), b.lse.data_ptr(), stream)
        finally:
            ss.ss_round_destroy(r)
    finally:
        torch.cuda.synchronize()      # the events are destroyed only after the work that uses them
        ss.ss_event_destroy(done)


def run_round_single_slot(b: RoundBuffers, host: HostHistory, slot: torch.Tensor, copy: "torch.cuda.Stream",
                          stream: int) -> None:
    """Chunk by chunk through one staging buffer: chunk j is uploaded into
    ``slot`` once chunk j-1's attention has read it (its free event), and
    attended once its upload is done (its ready event), so uploads and
    attention alternate without overlapping."""
    w = b.w
    ready, free = ss.ss_event_create(), ss.ss_event_create()
    try:
        r = ss.ss_round_init(b.desc, b.q.data_ptr(), b.ws.data_ptr(), b.ws_bytes, stream)
        try:
            used = False
            for j in range(w.num_chunks):
                if not host.sizes[j]:
                    continue
                ss.ss_upload_chunk(slot.data_ptr(), host.chunk_ptr(j), host.sizes[j], copy.cuda_stream,
                                   free if used else None, ready)
                ss.ss_attend_history_chunk(r, slot.data_ptr(), slot.data_ptr() + _chunk_vofs(w, host, j, b.kv_layout),
                                           w.chunk_lens(j), ready, free, stream)
                used = True
            ss.ss_attend_local_candidates(r, b.kc.data_ptr(), b.vc.data_ptr(), stream)
            ss.ss_round_finalize(r, b.out.data_ptr(), b.lse.data_ptr(), stream)
        finally:
            ss.ss_round_destroy(r)
    finally:
        torch.cuda.synchronize()
        ss.ss_event_destroy(ready)
        ss.ss_event_destroy(free)
