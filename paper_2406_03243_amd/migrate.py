"""Multi-stage live migration of one request (Llumnix §4.2), driven over the
llmig C ABI.

Stage 0 copies every block the request has filled so far while decoding goes
on; each later stage copies the blocks filled during the previous stage; once
little enough is left, the request is drained from its batch and a final
stage copies the rest, partial last block included.  Only that final stage is
downtime.  Non-final stages copy whole blocks only: a block still being
appended to is left for a later stage, which is also what makes the copy
race-free against decoding's writes (blocks already copied are never written
again, because the KV cache is append-only).

The copies run on a migration stream of their own; decoding's KV writes run on
a decode stream; an event recorded after each batch of writes orders the next
stage after them.  All streams keep the default priority.
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass

import numpy as np
import torch

from .llmig import LlmigError, MigrationHandle, Pool, llmig_pack, llmig_plan, llmig_unpack, llmig_write_tokens


# Timing event pairs whose times have been read, kept for the next stages:
# creating and first recording a pair costs more host time than the stage's
# launch itself.
_spare_timers: list = []


def _timer_pair():
    if _spare_timers:
        return _spare_timers.pop()
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


# Ordering events (no timing) of the drivers below, likewise kept: creating
# and first recording one costs ~15 us of host time, which at the start of a
# migration sits in front of its first launch.  An event may be recorded
# again once every wait on its previous recording has been enqueued (a
# stream's wait takes the recording current at the time of the call).
_spare_events: list = []


def _order_event():
    return _spare_events.pop() if _spare_events else torch.cuda.Event()


def _after_decode(ev, mig_stream, dec_stream) -> None:
    """Orders the migration stream's next work after everything the decode
    stream has enqueued so far.  When the decode stream has nothing left to
    run, its writes are already visible and no wait is enqueued (a wait
    costs ~19 us in front of the first stage's launch)."""
    if not dec_stream.query():
        ev.record(dec_stream)
        mig_stream.wait_event(ev)


@dataclass
class StageRecord:
    length: int        # tokens resident when the stage was planned
    from_tok: int
    to_tok: int
    blocks: int
    final: bool
    gpu_us: float = 0.0


class Migration:
    """One request's migration, driven through the library's coordinator
    (which plans, reserves destination blocks and launches each stage in one
    call).  Keeps the host-side records: the stages so far, their GPU times,
    and which destination blocks were consumed from the free list.  A
    stage's token range is the coordinator's: it starts where the previous
    stage ended and ends at the coordinator's count of copied tokens after
    the call, so the records cannot drift from what the library reserved."""

    def __init__(self, src: Pool, dst: Pool, src_table, dst_free_list, stream: torch.cuda.Stream,
                 max_workgroups: int = 0, block_size: int | None = None):
        self.src, self.dst, self.stream = src, dst, stream
        self.bs = src.block_size if block_size is None else int(block_size)
        self.src_table = np.ascontiguousarray(np.asarray(src_table, dtype=np.int32))
        self._free0 = np.ascontiguousarray(np.asarray(dst_free_list, dtype=np.int32))
        self._consumed = 0
        self.copied_tok = 0
        self.finished_at = None
        self.stages: list[StageRecord] = []
        self._events = []
        self.coord = MigrationHandle(self.bs)
        if max_workgroups:
            self.coord.set_max_workgroups(max_workgroups)
        # addresses for the stage calls, taken once (the arrays live as long
        # as the migration): the final stage's call is on the downtime path
        self._table_ptr = self.src_table.ctypes.data
        self._free_ptr = self._free0.ctypes.data
        if src is not None:
            self._handles = (src.handle, dst.handle)
            self._stream_ptr = stream.cuda_stream

    @property
    def free(self) -> np.ndarray:
        """What is left of the destination free list."""
        return self._free0[self._consumed:]

    @property
    def dst_table(self) -> np.ndarray:
        """Destination block of every logical block copied so far (the
        consumed head of the free list, in logical order)."""
        return self._free0[:self._consumed]

    def remaining_blocks(self, length: int) -> int:
        """Blocks of a request now holding ``length`` tokens that no stage
        has copied yet (the input of the driver's decision to end)."""
        return math.ceil(length / self.bs) - self.copied_tok // self.bs

    def _record(self, length: int, n: int, final: bool, ev) -> StageRecord:
        to_tok = self.coord.copied_tokens()
        rec = StageRecord(length, self.copied_tok, to_tok, n, final)
        self.stages.append(rec)
        self._events.append(ev)
        self._consumed += n
        self.copied_tok = to_tok
        return rec

    def stage(self, length: int, final: bool, time_it: bool = True) -> StageRecord:
        """Plan, reserve and launch the next stage for a request that now
        holds ``length`` tokens (a non-final stage stops at the last whole
        block: the coordinator's rule)."""
        ev = None
        if time_it:
            # recorded by the library right around its launches: kernel time
            # without the host work that plans and checks the stage
            ev = _timer_pair()
            self.coord.set_stage_events(*ev)
        try:
            n = self.coord.stage_ptrs(*self._handles, self._table_ptr, self.src_table.size, length, final,
                                      self._free_ptr + 4 * self._consumed, self._free0.size - self._consumed,
                                      self._stream_ptr)
        except LlmigError as e:
            self._consumed += getattr(e, "consumed", 0)   # reserved before a HIP failure: abort returns them
            raise
        if time_it and n == 0:
            _spare_timers.append(ev)    # not recorded by the library: free again
            ev = None
        return self._record(length, n, final, ev)

    def finish(self, length: int, time_it: bool = False) -> StageRecord:
        """The final stage for a drained request now holding ``length``
        tokens, returning once its copy is complete (one library call that
        launches and waits, so no host work sits between the two).
        ``finished_at`` is the perf_counter time at which the call returned;
        the bookkeeping after it is not downtime."""
        ev = None
        if time_it:
            ev = _timer_pair()
            self.coord.set_stage_events(*ev)
        try:
            n = self.coord.finish_ptrs(*self._handles, self._table_ptr, self.src_table.size, length,
                                       self._free_ptr + 4 * self._consumed, self._free0.size - self._consumed,
                                       self._stream_ptr)
            self.finished_at = time.perf_counter()   # the host has seen the copy complete
        except LlmigError as e:
            self._consumed += getattr(e, "consumed", 0)
            raise
        if time_it and n == 0:
            _spare_timers.append(ev)
            ev = None
        return self._record(length, n, True, ev)

    def plan(self, length: int, final: bool):
        """The same step without the copy (host only): reserve and plan the
        next stage.  Returns (record, map_src, map_dst)."""
        ms, md = self.coord.next(self.src_table, length, final, self.free)
        return self._record(length, len(md), final, None), ms, md

    def abort(self) -> np.ndarray:
        """Abort: the destination blocks reserved so far, to be released."""
        return self.coord.abort()

    def commit(self) -> np.ndarray:
        """Commit after the final stage: the request's destination table."""
        return self.coord.commit()

    def collect_times(self) -> None:
        """Fill in each timed stage's GPU time (after the stream is
        synchronised); the events go back to the spares."""
        for k, (rec, ev) in enumerate(zip(self.stages, self._events)):
            if ev is not None:
                rec.gpu_us = ev[0].elapsed_time(ev[1]) * 1e3
                _spare_timers.append(ev)
                self._events[k] = None


def run_scheduled(src: Pool, dst: Pool, src_table, dst_free_list, initial_len: int, appends,
                  mig_stream, dec_stream, time_all: bool = False, time_final: bool = False):
    """A migration whose decoding appends a known batch of tokens before each
    incremental stage (``appends`` is a list of device tensors laid out
    [L][K,V][n_tok][slot_bytes]); the stage after the last batch is final.
    Each stage is planned after the host has seen the batch before it
    written.
    Stage 0 is timed with events on the migration stream; the incremental
    stages too when ``time_all``, the final one when ``time_final`` (its
    events then add their own host work to the downtime).  Returns
    (migration, downtime_us): downtime is host wall time from the start of
    the final stage's planning until the host sees it complete."""
    m = Migration(src, dst, src_table, dst_free_list, mig_stream)
    length = initial_len
    ev = _order_event()             # orders each stage after the decode writes before it
    _after_decode(ev, mig_stream, dec_stream)
    m.stage(length, final=not appends)
    downtime_us = None
    for k, data in enumerate(appends):
        n_tok = data.numel() // (src.num_layers * 2 * src.slot_bytes)
        llmig_write_tokens(src, src_table, length, data, stream=dec_stream)
        length += n_tok
        ev.record(dec_stream)
        final = k == len(appends) - 1
        if final:
            # The final stage starts once the previous stage's copy is done
            # and the request is drained (its last token written).
            mig_stream.synchronize()
            ev.synchronize()
            t0 = time.perf_counter()
            m.finish(length, time_it=time_final)
            downtime_us = (m.finished_at - t0) * 1e6
        else:
            # The next stage is planned once the host has seen this batch
            # written, as an engine plans it after the decode step that
            # produced its tokens; the batch is then complete and the stage
            # needs no wait on the decode stream.  (The host waits while
            # stage 0 still copies, so the wait costs the GPU nothing.)
            ev.synchronize()
            m.stage(length, final=False, time_it=time_all)
    if downtime_us is None:
        t0 = time.perf_counter()
        mig_stream.synchronize()
        downtime_us = (time.perf_counter() - t0) * 1e6
    _spare_events.append(ev)
    m.collect_times()
    return m, downtime_us


def run_timed(src: Pool, dst: Pool, src_table, initial_len: int, dst_free_list, append_pool,
              mig_stream, dec_stream, step_ms: float = 20.0, last_stage_max_blocks: int = 1,
              max_stages: int = 8, max_workgroups: int = 0, time_final: bool = False):
    """A migration whose decoding speed is simulated: while a stage copies,
    decoding produces max(1, ceil(stage_time / step_ms)) tokens, which are
    written once the stage is over.  The next stage is final when at most
    ``last_stage_max_blocks`` blocks remain, or at ``max_stages``.
    ``append_pool`` is a device tensor [L][K,V][max_tokens][slot_bytes] the
    appended tokens are drawn from.  ``max_workgroups`` caps the copy grid
    (0: uncapped).  ``time_final`` times the final stage with events as
    well.  Returns (migration, downtime_us)."""
    m = Migration(src, dst, src_table, dst_free_list, mig_stream, max_workgroups)
    length = initial_len
    max_tok = append_pool.shape[2]
    used = 0
    ev = _order_event()             # orders each stage after the decode writes before it
    _after_decode(ev, mig_stream, dec_stream)
    rec = m.stage(length, final=False)
    while True:
        mig_stream.synchronize()
        m.collect_times()
        n_tok = max(1, math.ceil(rec.gpu_us / (step_ms * 1e3)))
        if used + n_tok > max_tok:
            raise RuntimeError("append pool exhausted")
        with torch.cuda.stream(dec_stream):
            data = append_pool[:, :, used:used + n_tok].contiguous()
        llmig_write_tokens(src, src_table, length, data, stream=dec_stream)
        used += n_tok
        length += n_tok
        ev.record(dec_stream)
        if m.remaining_blocks(length) <= last_stage_max_blocks or len(m.stages) + 1 >= max_stages:
            ev.synchronize()
            t0 = time.perf_counter()
            m.finish(length, time_it=time_final)
            downtime_us = (m.finished_at - t0) * 1e6
            break
        mig_stream.wait_event(ev)
        rec = m.stage(length, final=False)
    _spare_events.append(ev)
    m.collect_times()
    return m, downtime_us


def run_carried(src: Pool, dst: Pool, src_table, initial_len: int, dst_free_list, decode_step, append_data,
                attn_stream, mig_stream, dec_stream, split: int = 1, carry_final: bool = False):
    """A migration whose first stage rides on decode steps (Llumnix §4.2's
    stage 0, copied while the request keeps decoding): the coordinator
    reserves and plans the stage (every whole block), and ``split`` decode
    steps carry it, each writing its share of the blocks into ``dst`` as its
    attention reads them (llmig_decode_attention_migrate).
    ``decode_step(carry)`` enqueues one decode step on ``attn_stream``;
    ``carry`` is (dst pool, device ids, first logical block) for the blocks
    that step writes.  Each step produces one token of the request, which
    decode writes on ``dec_stream`` from ``append_data`` ([L][K,V][n][slot
    bytes], n >= split); it lands past the stage's blocks.
    Then the final stage.  By default the host waits for the steps and
    their writes, the request is drained and a stage on ``mig_stream``
    copies the rest (downtime: host wall time from its planning until the
    host sees it complete).  With ``carry_final`` the request's last decode
    step on the source carries the final stage itself (the rest, its partly
    filled last block included, ordered after the last token's write), so
    no copy is left once the request leaves the batch: downtime 0, and the
    cost is that step's.  Returns (migration, downtime_us, (start, end)
    events around the carrying steps on ``attn_stream``)."""
    m = Migration(src, dst, src_table, dst_free_list, mig_stream)
    length = initial_len
    rec, _, md = m.plan(length, final=False)
    first = rec.from_tok // m.bs
    with torch.cuda.stream(attn_stream):
        ids = torch.from_numpy(md).to(attn_stream.device)
    bounds = [len(md) * k // split for k in range(split + 1)]
    t = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    t[0].record(attn_stream)
    for k in range(split):
        decode_step((dst, ids[bounds[k]:bounds[k + 1]], first + bounds[k]))
        with torch.cuda.stream(dec_stream):
            data = append_data[:, :, k:k + 1].contiguous()
        llmig_write_tokens(src, src_table, length, data, stream=dec_stream)
        length += 1
    ev = _order_event()
    ev.record(dec_stream)
    if carry_final:
        rec_f, _, md_f = m.plan(length, final=True)
        with torch.cuda.stream(attn_stream):
            ids_f = torch.from_numpy(md_f).to(attn_stream.device)
        attn_stream.wait_event(ev)              # the last token is written before the step reads it
        t_f = torch.cuda.Event(enable_timing=True)
        t_f.record(attn_stream)
        decode_step((dst, ids_f, rec_f.from_tok // m.bs))
        t[1].record(attn_stream)
        t[1].synchronize()
        _spare_events.append(ev)
        rec.gpu_us = t[0].elapsed_time(t_f) * 1e3
        rec_f.gpu_us = t_f.elapsed_time(t[1]) * 1e3
        m.finished_at = time.perf_counter()
        return m, 0.0, t
    t[1].record(attn_stream)
    t[1].synchronize()
    ev.synchronize()
    _spare_events.append(ev)
    t0 = time.perf_counter()
    m.finish(length)
    downtime_us = (m.finished_at - t0) * 1e6
    rec.gpu_us = t[0].elapsed_time(t[1]) * 1e3
    return m, downtime_us, t


def plan_batch(tables, lengths, dst_free_list, block_size: int):
    """Plan a batched migration of several requests as one stage each
    (request order, destination blocks taken from the head of the free list
    in turn).  Returns (map_src, map_dst, per-request destination tables)."""
    free = np.ascontiguousarray(np.asarray(dst_free_list, dtype=np.int32))
    srcs, dsts = [], []
    for table, length in zip(tables, lengths):
        ms, md = llmig_plan(table, free, int(length), 0, int(length), block_size)
        srcs.append(ms)
        dsts.append(md)
        free = free[len(md):]
    return np.concatenate(srcs), np.concatenate(dsts), dsts


def run_host_staged(src: Pool, dst: Pool, map_src, map_dst, host_bufs, pack_stream, unpack_stream,
                    chunk_pairs: int, dev_bufs=None):
    """Block fusion through pinned host memory (Llumnix §5): chunks of
    ``chunk_pairs`` block pairs go from the source pool to one of two pinned
    host buffers and from there into the destination pool, the two buffers
    alternating so that one chunk's way out overlaps the previous chunk's way
    in.  Events order each unpack after its pack and each reuse of a buffer
    after the work that read it.

    Without ``dev_bufs`` the pack kernel stores straight into the pinned
    buffer and the unpack kernel loads straight from it, over PCIe.  With
    ``dev_bufs`` (two pairs of device buffers of the same size) the kernels
    pack into and unpack from device memory and the copy engines move the
    buffers across PCIe (hipMemcpyAsync).  Returns once all work is enqueued."""
    n = len(map_src)
    freed = [None, None]                 # event after which host buffer k may be rewritten
    for c, lo in enumerate(range(0, n, chunk_pairs)):
        hi = min(n, lo + chunk_pairs)
        k = c % 2
        host = host_bufs[k]
        if freed[k] is not None:
            pack_stream.wait_event(freed[k])
        if dev_bufs is None:
            llmig_pack(src, map_src[lo:hi], host, stream=pack_stream)
        else:
            out_dev, in_dev = dev_bufs[k]
            llmig_pack(src, map_src[lo:hi], out_dev, stream=pack_stream)
            nbytes = (hi - lo) * src.num_layers * 2 * src.tile_bytes
            with torch.cuda.stream(pack_stream):
                host[:nbytes].copy_(out_dev[:nbytes], non_blocking=True)
        packed = torch.cuda.Event()
        packed.record(pack_stream)
        unpack_stream.wait_event(packed)
        if dev_bufs is None:
            llmig_unpack(dst, map_dst[lo:hi], host, stream=unpack_stream)
        else:
            with torch.cuda.stream(unpack_stream):
                in_dev[:nbytes].copy_(host[:nbytes], non_blocking=True)
            llmig_unpack(dst, map_dst[lo:hi], in_dev, stream=unpack_stream)
        ev = torch.cuda.Event()
        ev.record(unpack_stream)
        freed[k] = ev
