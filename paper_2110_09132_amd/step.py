"""Training steps of the sparse-embedding path, scheduled on streams.

A step of one table is the four C ABI calls in data order:
    gather (forward lookup, Sec. 4.1.1)
    grad_coalesce -> pack_by_owner (the exchange payload, Sec. 4.2.2 / 4.1.2)
    sparse_adam_apply (the update of the owned rows)
The library's step executor (emb_train_step) enqueues all four with one host
call.  With overlap=True the latency-bound work runs on side streams while
the lookup and the update stay on the main stream:
  by_owner=False: grad_coalesce on one side stream, pack_by_owner on another;
  by_owner=True:  grad_coalesce_by_owner (coalesce and pack in one), its sort
                  on one side stream and its reduction on another;
  split=True:     as by_owner, with the prior / delayed split of Vertical
                  Sparse Scheduling (grad_coalesce_split, given the next
                  batch's ids): the prior rows are updated right after the
                  lookup, the delayed rows on a third side stream beside the
                  next lookup.
The executor adds the cross-stream waits that keep every data dependency (see
emb_train_step in include/emb.h), through events or step signals.  This module only allocates the buffers,
rotates the buffer sets and fills in the arguments.
"""
from __future__ import annotations

import ctypes

import torch

from . import (EMB_ADAM_COEFFS_WORDS, EMB_BF16, EMB_F32, EmbError, Event, StepArgs, StepQueue, StepSchedule,
               StepSignals,
               _check, _grad, _need, _owners, adam_coeffs, grad_coalesce_split_workspace_bytes, lib, new_workspace,
               pack_by_owner_workspace_bytes)

# timing pairs of emb_step_schedule.timing; with the split, "pack" times the
# prior update and "adam" the delayed one
STAGES = ("gather", "coalesce", "pack", "adam")


class EmbeddingTable:
    """Device state of one table (W, Adam moments, row owners) and the buffers of its steps."""

    def __init__(self, W: torch.Tensor, row_owner: torch.Tensor, P: int, T_cap: int,
                 grad_dtype: torch.dtype = torch.float32, sets: int = 2):
        _need(W, torch.float32, "W")
        if W.dim() != 2:
            raise EmbError("W must be 2-D [V, D]")
        _owners(row_owner, W.shape[0], P)
        dev = W.device
        self.V, self.D = W.shape
        self.P, self.T_cap = P, T_cap
        self.W = W
        self.M = torch.zeros_like(W)
        self.S = torch.zeros_like(W)
        self.row_owner = row_owner
        i32, f32 = torch.int32, torch.float32
        self.lookup = torch.empty((T_cap, self.D), dtype=f32, device=dev)
        # `sets` buffer sets, rotated between consecutive steps
        self.sets = sets
        self.coals = [(torch.empty(T_cap, dtype=i32, device=dev), torch.empty(T_cap + 1, dtype=i32, device=dev),
                       torch.empty((T_cap, self.D), dtype=f32, device=dev), torch.empty(1, dtype=i32, device=dev))
                      for _ in range(sets)]
        # send counts / offsets sized for the 2P groups of the split
        self.send = [(torch.empty(T_cap, dtype=i32, device=dev), torch.empty((T_cap, self.D), dtype=f32, device=dev),
                      torch.empty(2 * P, dtype=i32, device=dev), torch.empty(2 * P + 1, dtype=i32, device=dev))
                     for _ in range(sets)]
        self.coal = self.coals[0]
        self.grad_code = EMB_BF16 if grad_dtype == torch.bfloat16 else EMB_F32
        nb = grad_coalesce_split_workspace_bytes(T_cap, T_cap, self.V, self.D, self.grad_code)  # serves every variant
        self.ws_coalesces = [new_workspace(nb, dev) for _ in range(sets)]
        self.ws_coalesce = self.ws_coalesces[0]
        self.ws_packs = [new_workspace(pack_by_owner_workspace_bytes(T_cap, P), dev) for _ in range(sets)]
        self.ws_pack = self.ws_packs[0]


def _stream_handle(s: torch.cuda.Stream) -> int:
    return s.cuda_stream


_SIDE_STREAMS: dict = {}


def side_streams(device=None):
    """The three side streams of a device, created once per process.  HIP maps
    streams onto a few hardware queues in creation order; creating streams
    once keeps the side streams on queues other than the main stream's."""
    dev = torch.cuda.current_device() if device is None else torch.device(device).index
    if dev not in _SIDE_STREAMS:
        _SIDE_STREAMS[dev] = tuple(torch.cuda.Stream(device=dev) for _ in range(3))
    return _SIDE_STREAMS[dev]


class StepPipeline:
    """Enqueues training steps of the hot path for a list of tables."""

    def __init__(self, tables, lr, beta1, beta2, eps, overlap: bool = True, dev_status: torch.Tensor | None = None,
                 streams: int = 3, by_owner: bool = True, split: bool = False, signals: bool = False,
                 sort_streams: int = 1, sets: int = 2, paired: bool = False, queued: bool = False):
        """streams (with overlap=True and by_owner=False): 2 puts coalesce and pack on one side
        stream, 3 gives each its own (more concurrency, one more cross-stream wait per step).
        by_owner: coalesce straight into the send layout (emb_grad_coalesce_by_owner).
        split: the prior / delayed split (implies by_owner); step() then needs the next ids.
        sort_streams (by_owner without the split, overlap=True): 2 runs the sorts of odd and even
        buffer sets on two side streams, so that a step's sort can run beside the previous step's
        (they share nothing; each waits only for the reduction of its own set's previous step);
        3 (with paired) runs sort and reduction of set i on side stream i mod 3, all three side
        streams (sets a multiple of 3).
        sets: buffer sets rotated between steps (every table needs at least this many; the split
        with events needs 2).  More sets let a step's sort start before the reduction of the step
        two back has finished.
        paired (with sort_streams >= 2): each sort stream also runs the reductions of its steps,
        right after their sorts (no cross-stream wait between the two halves).
        signals (with overlap=True): keep the cross-stream order with step signals (stream memory
        operations: about half the host time per step, for host-bound pipelines of small
        batches; with large batches events keep the GPU a few percent busier) instead of events.
        queued (overlap=True, events, by_owner without the split): enqueue each step from two host
        threads (StepQueue): the sort and the reduction from this one, the lookup and the update
        from the library's worker, so that a step costs the host about the larger half of its
        enqueue instead of both."""
        self.tables = list(tables)
        self.overlap = overlap
        self.main = torch.cuda.current_stream()
        s1, s2, s3 = side_streams()
        self.split = split
        self.by_owner = by_owner or split
        self.side = s1 if overlap else self.main  # coalesce (by_owner: its sort)
        self.side2 = s2 if (overlap and streams >= 3) else self.side  # pack (by_owner: the reduction)
        self.side3 = s3 if (overlap and split) else self.main  # the delayed update
        # the sorts of buffer set 1 (by_owner without the split): the third side stream
        self.side3_sort = s3 if (overlap and self.by_owner and not split and sort_streams >= 2) else None
        self.paired = paired and self.side3_sort is not None
        self.sort_streams = sort_streams if self.side3_sort is not None else 1
        if self.sort_streams >= 3 and not self.paired:
            raise ValueError("three sort streams run paired")
        if self.sort_streams >= 2 and sets % self.sort_streams:
            raise ValueError("the buffer sets must be a multiple of the sort streams")
        if any(tb.sets < sets for tb in self.tables):
            raise ValueError("a table has fewer buffer sets than the pipeline rotates")
        self.sets = sets
        self.count = 0
        self.events = []  # keeps the library events alive
        self.signals = [StepSignals() for _ in self.tables] if (overlap and signals) else []
        if queued and (not overlap or signals or split or not self.by_owner):
            raise ValueError("the two-thread enqueue takes overlapped owner-major steps with events, no split")
        self.queue = StepQueue() if queued else None
        self.args, self.sched = [], []
        st = 0 if dev_status is None else dev_status.data_ptr()
        for tb in self.tables:
            args, scheds = [], []
            for i in range(sets):
                uid, seg, ug, nu = tb.coals[i]
                sid, srows, cnt, offs = tb.send[i]
                a = StepArgs(table=tb.W.data_ptr(), exp_avg=tb.M.data_ptr(), exp_avg_sq=tb.S.data_ptr(), V=tb.V,
                             D=tb.D, row_owner=tb.row_owner.data_ptr(), P=tb.P, cap_rows=tb.T_cap,
                             lookup=tb.lookup.data_ptr(), uniq_ids=uid.data_ptr(), seg_offsets=seg.data_ptr(),
                             num_unique=nu.data_ptr(), uniq_grad=ug.data_ptr(), send_ids=sid.data_ptr(),
                             send_counts=cnt.data_ptr(), send_offsets=offs.data_ptr(), send_rows=srows.data_ptr(),
                             ws_coalesce=tb.ws_coalesces[i].data_ptr(),
                             ws_coalesce_bytes=tb.ws_coalesces[i].numel(),
                             ws_pack=tb.ws_packs[i].data_ptr(), ws_pack_bytes=tb.ws_packs[i].numel(), lr=lr,
                             beta1=beta1,
                             beta2=beta2, eps=eps, dev_status=st)
                evs = [Event() for _ in range(6)]
                self.events += evs
                if self.sort_streams >= 3:
                    sort_side = (self.side, self.side2, self.side3_sort)[i % 3]
                else:
                    sort_side = self.side3_sort if (i % 2 == 1 and self.side3_sort is not None) else self.side
                red_side = sort_side if self.paired else self.side2
                s = StepSchedule(lookup_update=_stream_handle(self.main), coalesce=_stream_handle(sort_side),
                                 pack=_stream_handle(red_side), delayed=_stream_handle(self.side3),
                                 sorted=evs[0].handle, coalesced=evs[1].handle, packed=evs[2].handle,
                                 updated=evs[3].handle, gathered=evs[4].handle, delayed_done=evs[5].handle,
                                 by_owner=1 if self.by_owner else 0, split=1 if split else 0,
                                 signals=self.signals[len(self.args)].handle if self.signals else None,
                                 sets=sets)
                args.append(a)
                scheds.append(s)
            self.args.append(args)
            self.sched.append(scheds)

    def step(self, batches, t: int, timing=None, next_ids=None, adam_coeffs_ptr=None):
        """Enqueue one step.  batches: [(ids int32 [T], grad [T, D]) per table]; t: Adam step (>= 1).
        timing: optional dict stage -> (begin Event, end Event) of library timing events, recorded
        around the calls of the first table on the streams they run on.
        next_ids (split): [ids int32 per table] of the next step's batches (an empty tensor after
        the last step).  adam_coeffs_ptr: optional device address of this step's update coefficients
        (emb_step_args.adam_coeffs; StepGraph sets it).  Inputs must be ready on the main stream
        when the first step is enqueued."""
        i = self.count % self.sets
        if self.count == 0 and self.overlap:
            for side in self._sides():
                side.wait_stream(self.main)
        if self.split and (next_ids is None or len(next_ids) != len(batches)):
            raise ValueError("the split schedule needs the next step's ids of every table")
        if len(batches) != len(self.tables):
            raise EmbError(f"{len(batches)} batches for {len(self.tables)} tables")
        for k, (ids, grad) in enumerate(batches):  # the kernels trust these sizes: check them first
            tb = self.tables[k]
            _need(ids, torch.int32, "ids")
            if ids.numel() > tb.T_cap:
                raise EmbError(f"{ids.numel()} tokens exceed the table's capacity of {tb.T_cap}")
            _, D = _grad(grad, ids.numel())
            if D != tb.D:
                raise EmbError(f"grad rows of {D} elements for a table of D = {tb.D}")
            if self.split:
                _need(next_ids[k], torch.int32, "next_ids")
                if next_ids[k].numel() > tb.T_cap:
                    raise EmbError(f"{next_ids[k].numel()} next ids exceed the table's capacity of {tb.T_cap}")
        for k, (ids, grad) in enumerate(batches):
            a, s = self.args[k][i], self.sched[k][i]
            a.ids = ids.data_ptr()
            a.T = ids.numel()
            if self.split:
                a.next_ids = next_ids[k].data_ptr()
                a.T_next = next_ids[k].numel()
            a.grad = grad.data_ptr()
            a.grad_dtype = EMB_BF16 if grad.dtype == torch.bfloat16 else EMB_F32
            a.step = t
            a.adam_coeffs = adam_coeffs_ptr
            s.reuse = 1 if self.count >= self.sets else 0
            for n in range(8):
                s.timing[n] = None
            if timing is not None and k == 0:
                for j, name in enumerate(STAGES):
                    if name in timing:
                        s.timing[2 * j] = timing[name][0].handle
                        s.timing[2 * j + 1] = timing[name][1].handle
            if self.queue is not None:
                _check(lib.emb_train_step_queued(self.queue.handle, ctypes.byref(a), ctypes.byref(s)),
                       "emb_train_step_queued")
            else:
                _check(lib.emb_train_step(ctypes.byref(a), ctypes.byref(s)), "emb_train_step")
        self.count += 1

    def _sides(self):
        return {x for x in (self.side, self.side2, self.side3, self.side3_sort) if x is not None} - {self.main}

    def finish(self):
        """Make the main stream wait for everything enqueued on the side streams (with the
        two-thread enqueue, once the worker has enqueued every step handed to it)."""
        if self.queue is not None:
            self.queue.flush()
        for side in self._sides():
            self.main.wait_stream(side)


class StepGraph:
    """`len(batches)` training steps of `tables` captured once into a HIP graph (stream capture of the
    step executor's calls, the cross-stream order by events) and replayed with one launch: for
    pipelines whose host enqueue time bounds them (small batches).  The steps' batches are fixed
    at capture (a loop feeding new batches would copy them into the captured buffers); the Adam
    step numbers are not: every step's update reads its coefficients from a device buffer that
    replay() fills for the step numbers it runs (emb_adam_coeffs; Sec. 5.7: one step count per
    iteration).  A replay runs after the work before it on its stream and before the work after
    it, whole, so the pipeline fills and drains once per replay: a graph should hold many steps.
    Events only (no step signals), no split.  Capture a graph after some eager steps have run in
    the process (the kernels' code is then loaded).  A graph holds at most one step per buffer
    set (no set is used twice inside one capture): the only configuration tested on the GPU; a
    graph of many steps over four sets ended its process with a segmentation fault whose cause
    is not known."""

    def __init__(self, tables, lr, beta1, beta2, eps, batches, sets: int = 4, sort_streams: int = 2,
                 paired: bool = True, dev_status: torch.Tensor | None = None):
        if len(batches) > sets:
            raise ValueError(f"a graph holds at most one step per buffer set ({len(batches)} steps, {sets} sets)")
        self.n = len(batches)
        self.hp = (lr, beta1, beta2, eps)
        dev = tables[0].W.device
        self.coeffs_dev = torch.zeros((self.n, EMB_ADAM_COEFFS_WORDS), dtype=torch.float32, device=dev)
        # two pinned staging buffers in turn: one can be refilled while the other's copy is pending
        self.coeffs_host = [torch.zeros((self.n, EMB_ADAM_COEFFS_WORDS), dtype=torch.float32, pin_memory=True)
                            for _ in range(2)]
        self.copied = [None, None]  # the event after each staging buffer's last copy
        self.turn = 0
        self.stream = torch.cuda.Stream(device=dev)  # the capture stream (not the default stream)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(self.stream):
            # a fresh pipeline: the first use of each buffer set in the capture waits for nothing before it
            self.pipe = StepPipeline(tables, lr, beta1, beta2, eps, overlap=True, dev_status=dev_status,
                                     signals=False, sets=sets, sort_streams=sort_streams, paired=paired)
            self.graph.capture_begin()
            try:
                for i, b in enumerate(batches):
                    self.pipe.step(b, 1, adam_coeffs_ptr=self.coeffs_dev[i].data_ptr())
                self.pipe.finish()
            finally:
                self.graph.capture_end()

    def replay(self, step0: int):
        """Run the captured steps on the current stream as Adam steps step0 .. step0 + n - 1."""
        buf = self.coeffs_host[self.turn]
        if self.copied[self.turn] is not None:
            self.copied[self.turn].synchronize()  # its previous copy has been read
        lr, b1, b2, eps = self.hp
        for i in range(self.n):
            adam_coeffs(lr, b1, b2, eps, step0 + i, buf[i])
        self.coeffs_dev.copy_(buf, non_blocking=True)
        ev = torch.cuda.Event()
        ev.record()
        self.copied[self.turn] = ev
        self.turn ^= 1
        self.graph.replay()
