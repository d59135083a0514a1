"""Asynchronous state reconciliation (Algorithm 1) on one MI355X.

The paper runs its primary and secondary resources as two model replicas on
separate GPUs.  On one MI355X they are two disjoint partitions of the device's
256 compute units: each is a HIP stream created with a CU mask, the primary
with most CUs and the secondary with a few per XCD.  The masks give every XCD
CUs in both partitions, so every workgroup of either stream has a CU to run on
however the runtime numbers CUs across XCDs.  Each role owns a KV cache (page
pool and block table); the swap at the end of a reconciliation exchanges
which cache the primary stream serves from, and no bytes move.

What runs where (Algorithm 1):
* every task (Increment + inference) is one ``csr_extend_attention`` with
  CSR_APPEND on the primary stream over X_static (+) X_dyn; only the state
  chunk (and any remainder left by a swap) is committed, X_dyn is recomputed
  by every task (Sec. III-D);
* at |X_static| >= tau_mem, X_E = Evict(X_static) is warmed up on the
  secondary stream: one ``csr_prefill`` writing the secondary cache (with RoPE
  the evicted tokens get their new, compacted positions);
* while a reconciliation runs, chunks are buffered; after the warm-up every
  catch-up round is one ``csr_extend_attention`` with CSR_APPEND of the whole
  buffer on the secondary stream, until at most N_catchup tokens wait; then the
  roles swap and the new primary's next task computes the remainder.

Completion of secondary work is observed by polling its events at each task,
so the serving loop never blocks on it.  This module only orchestrates: every
step of the computation is a call into the HIP library.  Token projections
(q, k, v per token id) come from a caller-supplied table of synthetic rows.
"""
from __future__ import annotations

import ctypes
import time
from dataclasses import dataclass
from typing import Callable, List, Optional, Tuple

import torch

from . import csr

Range = Tuple[int, int]  # token ids [start, end)


def rlen(ranges: List[Range]) -> int:
    return sum(b - a for a, b in ranges)


def xcd_spread_cus(per_xcd: int, num_cus: int = 256, num_xcds: int = 8) -> List[int]:
    """CU ids for a partition with ``per_xcd`` CUs on every XCD whether the
    runtime numbers CUs in blocks per XCD (id // 32) or round robin (id % 8).

    Block x (ids 32x .. 32x + 31) contributes ids 32x + 8j + ((x + k) mod 8)
    for j < c and k < t, per_xcd = c * t with c <= 4: c * t ids in every
    block, and residue r modulo 8 appears in exactly t blocks, c times each.
    """
    per_block = num_cus // num_xcds
    t = max(1, -(-per_xcd // 4))
    c = per_xcd // t if per_xcd > 0 else 0
    if per_block != 32 or num_xcds != 8 or per_xcd < 1 or c * t != per_xcd or c > 4 or t > 8:
        raise ValueError(f"cannot spread {per_xcd} CUs per XCD evenly (use 1-4, 6, 8, 9, 12, 15, 16, ...)")
    return sorted(per_block * x + num_xcds * j + (x + k) % num_xcds
                  for x in range(num_xcds) for j in range(c) for k in range(t))


_hip = None
_owned = set()  # raw handles of the CU-masked streams this module created and has not destroyed


def _hip_lib():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    return _hip


def cu_masked_stream(cu_ids: List[int], num_cus: int = 256) -> torch.cuda.ExternalStream:
    """A HIP stream (default priority) whose kernels run only on ``cu_ids``.

    The stream belongs to the caller, who ends it with ``destroy_streams``
    once its work is done (torch's ExternalStream never destroys the handle)."""
    _hip_lib()
    if not cu_ids:
        raise ValueError("empty CU set")
    words = [0] * ((num_cus + 31) // 32)
    for c in cu_ids:
        words[c // 32] |= 1 << (c % 32)
    arr = (ctypes.c_uint32 * len(words))(*words)
    s = ctypes.c_void_p()
    rc = _hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), len(words), arr)
    if rc != 0:
        raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
    _owned.add(s.value)
    return torch.cuda.ExternalStream(s.value)


def destroy_streams(*streams) -> None:
    """Wait for and destroy the given streams that ``cu_masked_stream`` created
    (others, e.g. torch's own streams, are left alone).  A process should end
    none of them alive: a stream left to the runtime's exit-time teardown is
    destroyed after tools hooked into the runtime (profilers) have shut down."""
    for st in streams:
        h = getattr(st, "cuda_stream", None)
        if h is None or h not in _owned:
            continue
        st.synchronize()
        rc = _hip_lib().hipStreamDestroy(ctypes.c_void_p(h))
        _owned.discard(h)
        if rc != 0:
            raise RuntimeError(f"hipStreamDestroy failed ({rc})")


class TokenTable:
    """Per-token projections q [N, Hq, d], k and v [N, Hkv, d] on the device."""

    def __init__(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor):
        self.q, self.k, self.v = q, k, v

    @staticmethod
    def synthetic(n: int, hq: int, hkv: int, d: int, seed: int = 0, scale: float = 0.5,
                  dtype=torch.bfloat16) -> "TokenTable":
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        mk = lambda h: (torch.randn((n, h, d), device="cuda", generator=g) * scale).to(dtype)  # noqa: E731
        return TokenTable(mk(hq), mk(hkv), mk(hkv))

    def gather(self, ranges: List[Range]):
        """Rows for the ids in ``ranges`` (in order), as contiguous q, k, v."""
        merged: List[Range] = []
        for a, b in ranges:
            if merged and merged[-1][1] == a:
                merged[-1] = (merged[-1][0], b)
            elif b > a:
                merged.append((a, b))
        ranges = merged
        if len(ranges) == 1:
            a, b = ranges[0]
            return self.q[a:b], self.k[a:b], self.v[a:b]
        return (torch.cat([self.q[a:b] for a, b in ranges]), torch.cat([self.k[a:b] for a, b in ranges]),
                torch.cat([self.v[a:b] for a, b in ranges]))


class Cache:
    """One resource's KV cache: a page pool, its block table, the committed length."""

    def __init__(self, name: str, pages: int, page_size: int, hkv: int, d: int, dtype, seed: int):
        self.name = name
        self.k_pool = torch.zeros((pages, page_size, hkv, d), dtype=dtype, device="cuda")
        self.v_pool = torch.zeros_like(self.k_pool)
        g = torch.Generator()
        g.manual_seed(seed)
        self.block_table = torch.randperm(pages, generator=g).to(torch.int32).reshape(1, pages).cuda()
        self.capacity = pages * page_size
        self.length = 0
        self.ids: List[Range] = []   # token ids held at positions 0 .. length-1

    def hold(self, ranges: List[Range]) -> None:
        for a, b in ranges:
            if self.ids and self.ids[-1][1] == a:
                self.ids[-1] = (self.ids[-1][0], b)
            else:
                self.ids.append((a, b))
        self.length += rlen(ranges)
        if self.length > self.capacity:
            raise RuntimeError(f"cache {self.name} overflow: {self.length} > {self.capacity} tokens")


@dataclass
class Task:
    index: int
    computed: List[Range]        # ids the task computed (cached prefix excluded), dyn last
    cache: str                   # which cache served it
    arrival: float               # host seconds since the run's reference point
    end_event: torch.cuda.Event
    out: Optional[torch.Tensor] = None


@dataclass
class Event:
    kind: str                    # warmup | catchup | swap
    task: int                    # index of the task before which it was observed or launched
    tokens: int
    host_time: float


class Reconciler:
    """Algorithm 1 over two caches and two streams (see the module comment).

    ``step(chunk, dyn)`` performs one task: advance the reconciliation (poll
    the secondary's work; catch up or swap), Increment with the state chunk,
    and serve the task on the primary.  ``gate(kind)`` may hold back the
    observation of a finished warm-up or catch-up (tests use it to fix the
    interleaving); ``sync_secondary`` waits for the secondary instead of
    polling once the gate opens.
    """

    def __init__(self, table: TokenTable, desc, x_pre: Range, tau_mem: int, n_catchup: int, cache_tokens: int,
                 primary_stream, secondary_stream, page_size: int = 16, seed: int = 0,
                 gate: Optional[Callable[[str], bool]] = None, sync_secondary: bool = False,
                 keep_outputs: bool = False, blocking: bool = False):
        hkv, d = desc.num_kv_heads, desc.head_dim
        pages = (cache_tokens + page_size - 1) // page_size
        dt = table.k.dtype
        self.table, self.desc = table, desc
        self.caches = [Cache("A", pages, page_size, hkv, d, dt, seed), Cache("B", pages, page_size, hkv, d, dt, seed + 1)]
        self.primary = 0
        self.x_pre = [x_pre]
        self.chunks: List[List[Range]] = []  # X_chunks of the primary's logical state
        self.tau_mem, self.n_catchup = tau_mem, n_catchup
        self.ps, self.ss = primary_stream, secondary_stream
        self.gate = gate or (lambda kind: True)
        self.sync_secondary = sync_secondary
        self.keep_outputs = keep_outputs
        self.blocking = blocking           # stop-the-world eviction on the primary stream (baseline)
        self.reconciling = False
        self.buffer: List[List[Range]] = []
        self.x_e_chunks: List[List[Range]] = []
        self.pending: List[Range] = []     # ids the primary's next task must compute first
        self.phase = "idle"
        self.sec_event: Optional[torch.cuda.Event] = None
        self.sec_started = 0.0
        self.inflight: list = []           # tensors kept alive until the secondary's event
        self.tasks: List[Task] = []
        self.events: List[Event] = []
        self.t0 = time.perf_counter()
        self.ref_event: Optional[torch.cuda.Event] = None
        self.warm_ms: List[float] = []     # host-observed warm-up and catch-up spans
        self.catchup_ms: List[float] = []

    # -- bookkeeping ------------------------------------------------------------
    def now(self) -> float:
        return time.perf_counter() - self.t0

    def static_len(self) -> int:
        return rlen(self.x_pre) + sum(rlen(c) for c in self.chunks)

    def logical_ids(self) -> List[Range]:
        return self.x_pre + [r for c in self.chunks for r in c]

    def primary_cache(self) -> Cache:
        return self.caches[self.primary]

    def secondary_cache(self) -> Cache:
        return self.caches[1 - self.primary]

    # -- the library calls --------------------------------------------------------
    def _one(self, v: int) -> torch.Tensor:
        return torch.full((1,), v, dtype=torch.int32, device="cuda")

    def _fits(self, cache: Cache, base: int, n: int) -> None:
        # The block table covers `capacity` positions; the library checks the
        # cached length and the chunk against it separately, so their sum is
        # checked here, before any launch.
        if base + n > cache.capacity:
            raise RuntimeError(f"cache {cache.name}: positions up to {base + n} exceed its {cache.capacity} slots")

    def _extend(self, cache: Cache, ranges: List[Range], stream):
        n = rlen(ranges)
        self._fits(cache, cache.length, n)
        q, k, v = self.table.gather(ranges)
        cu = torch.tensor([0, n], dtype=torch.int32, device="cuda")
        out, _ = csr.extend_attention(self.desc, q, k, v, cache.k_pool, cache.v_pool, cache.block_table,
                                      cache.block_table.shape[1], cu, self._one(cache.length), n, cache.length,
                                      append=True, want_lse=False, stream=stream)
        return out, (q, k, v, cu)

    def _warmup(self, cache: Cache, ranges: List[Range], stream):
        n = rlen(ranges)
        self._fits(cache, 0, n)
        q, k, v = self.table.gather(ranges)
        cu = torch.tensor([0, n], dtype=torch.int32, device="cuda")
        out, _ = csr.prefill(self.desc, q, k, v, cu, n, k_pool=cache.k_pool, v_pool=cache.v_pool,
                             block_table=cache.block_table, bt_stride=cache.block_table.shape[1], want_lse=False,
                             stream=stream)
        return (q, k, v, cu, out)

    def prime(self, initial_chunks: List[Range] = ()) -> None:
        """Fill the primary cache with X_pre (+) ``initial_chunks`` in one
        prefill (the state the serving loop starts from)."""
        cache = self.primary_cache()
        ranges = self.x_pre + list(initial_chunks)
        cache.length, cache.ids = 0, []
        with torch.cuda.stream(self.ps):
            keep = self._warmup(cache, ranges, self.ps)
        cache.hold(ranges)
        self.chunks = [[c] for c in initial_chunks]
        self.ps.synchronize()
        del keep

    # -- Algorithm 1 --------------------------------------------------------------
    def _launch_warmup(self, task_index: int) -> None:
        self.x_e_chunks = [list(c) for c in self.chunks[len(self.chunks) // 2:]]   # Evict: oldest half out
        x_e = self.x_pre + [r for c in self.x_e_chunks for r in c]
        sec = self.secondary_cache()
        stream = self.ps if self.blocking else self.ss
        # the secondary cache may still be read by tasks queued on the primary stream
        last = torch.cuda.Event()
        last.record(self.ps)
        stream.wait_event(last)
        sec.length, sec.ids = 0, []
        with torch.cuda.stream(stream):
            keep = self._warmup(sec, x_e, stream)
            ev = torch.cuda.Event()
            ev.record(stream)
        sec.hold(x_e)
        self.inflight = [keep]
        self.sec_event = ev
        self.sec_started = self.now()
        self.phase = "warmup"
        self.reconciling = True
        self.events.append(Event("warmup", task_index, rlen(x_e), self.sec_started))

    def _secondary_finished(self) -> bool:
        if self.sec_event is None or not self.gate(self.phase):
            return False
        if self.sync_secondary or self.blocking:
            self.sec_event.synchronize()
            return True
        return self.sec_event.query()

    def _advance(self, task_index: int) -> None:
        """Reconcile: act on finished secondary work (catch up or swap)."""
        while self.reconciling and self._secondary_finished():
            span = (self.now() - self.sec_started) * 1e3
            (self.warm_ms if self.phase == "warmup" else self.catchup_ms).append(span)
            self.inflight = []
            waiting = sum(rlen(c) for c in self.buffer)
            if waiting > self.n_catchup:
                ranges = [r for c in self.buffer for r in c]
                sec = self.secondary_cache()
                with torch.cuda.stream(self.ss):
                    _, keep = self._extend(sec, ranges, self.ss)
                    ev = torch.cuda.Event()
                    ev.record(self.ss)
                sec.hold(ranges)
                self.x_e_chunks += self.buffer
                self.buffer = []
                self.inflight = [keep]
                self.sec_event = ev
                self.sec_started = self.now()
                self.phase = "catchup"
                self.events.append(Event("catchup", task_index, waiting, self.sec_started))
                if not (self.sync_secondary or self.blocking):
                    return
                continue
            # swap the roles: the secondary's cache becomes the primary's
            remainder = self.buffer
            self.buffer = []
            self.chunks = [list(c) for c in self.x_e_chunks] + [list(c) for c in remainder]
            self.pending = [r for c in remainder for r in c]
            self.ps.wait_event(self.sec_event)
            self.primary = 1 - self.primary
            self.reconciling = False
            self.phase = "idle"
            self.sec_event = None
            self.events.append(Event("swap", task_index, rlen(self.pending), self.now()))
            return

    def start_clock(self) -> None:
        """Reference point for arrival times: an event on the primary stream,
        waited for, and the host clock read right after it."""
        self.ref_event = torch.cuda.Event(enable_timing=True)
        self.ref_event.record(self.ps)
        self.ref_event.synchronize()
        self.t0 = time.perf_counter()

    def step(self, chunk: Range, dyn: Optional[Range] = None, arrival: Optional[float] = None) -> Task:
        """One task: reconcile progress, Increment(chunk), inference on the primary.
        ``arrival`` (seconds after ``start_clock``) defaults to now."""
        index = len(self.tasks)
        self._advance(index)
        self.chunks.append([chunk])
        if self.reconciling:
            self.buffer.append([chunk])
        # the primary computes what its cache lacks (a swap's remainder), the chunk and X_dyn
        cache = self.primary_cache()
        computed = self.pending + [chunk] + ([dyn] if dyn else [])
        if self.ref_event is None:
            self.start_clock()
        arrival = self.now() if arrival is None else arrival
        with torch.cuda.stream(self.ps):
            out, _ = self._extend(cache, computed, self.ps)
            end = torch.cuda.Event(enable_timing=True)
            end.record(self.ps)
        cache.hold(self.pending + [chunk])
        self.pending = []
        task = Task(index, computed, cache.name, arrival, end, out if self.keep_outputs else None)
        self.tasks.append(task)
        if self.static_len() >= self.tau_mem and not self.reconciling:
            self._launch_warmup(index)
            if self.blocking:
                self._advance(index)
        return task

    def latencies_ms(self) -> List[float]:
        """Completion minus arrival for every task (GPU completion times mapped
        onto the host clock through the reference event)."""
        torch.cuda.synchronize()
        return [self.ref_event.elapsed_time(t.end_event) - t.arrival * 1e3 for t in self.tasks]
