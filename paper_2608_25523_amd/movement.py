"""Prefix movement between the KV pool and a pinned host page store.

An agent leaving the resident set has its prefix pages evicted to host
memory; one entering it has them loaded back (Sec. 4, Eq. (8)).  Both
directions are ``pfx_page_copy`` launches (the kernel reads or writes the
pinned store over the host link), on whatever stream the caller passes, so a
load can run beside attention on another stream.  The cost model of Eq. (8)
charges a transition mu / B_swap times the prefix tokens moved out and in
(transfers serialized); ``calibrate_swap`` measures B_swap per direction.

Product side: the binding and torch only.
"""

from __future__ import annotations

import numpy as np
import torch

from . import binding as B


class HostStore:
    """Pinned host pages in the pool's format ([pages][Hkv][16][d] bf16, K and
    V), with an allocator for their slots."""

    def __init__(self, num_pages: int, num_kv_heads: int, head_dim: int):
        shape = (num_pages, num_kv_heads, 16, head_dim)
        self.k = torch.empty(shape, dtype=torch.bfloat16, pin_memory=True)
        self.v = torch.empty(shape, dtype=torch.bfloat16, pin_memory=True)
        self.pool = B.make_pool(num_pages, num_kv_heads, head_dim, self.k, self.v)
        self.alloc = B.Allocator(num_pages)


class Mover:
    """Evicts and loads page lists between one device pool and one host
    store.  Each instance owns a device workspace for the page-id lists of
    one transfer at a time (stream-ordered reuse: a transfer must not start
    on a different stream before the previous one on this mover finished),
    and, for the copy-engine paths, a device staging area of max_pages
    pages."""

    def __init__(self, pool: B.pfx_pool, store: HostStore, max_pages: int, device="cuda", staging: bool = False):
        self.pool, self.store = pool, store
        self.ws = torch.empty(B.pfx_page_copy_workspace_bytes(max_pages) + 256, dtype=torch.uint8, device=device)
        self.max_pages = max_pages
        self.stage = None
        if staging:
            shape = (max_pages,) + tuple(store.k.shape[1:])
            self.stage_k = torch.empty(shape, dtype=torch.bfloat16, device=device)
            self.stage_v = torch.empty(shape, dtype=torch.bfloat16, device=device)
            self.stage = B.make_pool(max_pages, shape[1], shape[3], self.stage_k, self.stage_v)

    def _check(self, pool_pages, slots):
        if len(pool_pages) != len(slots) or len(pool_pages) > self.max_pages:
            raise ValueError("page lists differ in length or exceed the mover's workspace")
        pool_pages, slots = np.asarray(pool_pages), np.asarray(slots)
        if len(pool_pages) and (pool_pages.min() < 0 or pool_pages.max() >= self.pool.num_pages):
            raise ValueError("a pool page id is out of range")
        if len(slots) and (slots.min() < 0 or slots.max() >= self.store.pool.num_pages):
            raise ValueError("a store slot is out of range")

    def evict(self, pool_pages, slots, stream=None):
        """Pool pages -> store slots (device to host)."""
        self._check(pool_pages, slots)
        B.pfx_page_copy(self.store.pool, self.pool, slots, pool_pages, self.ws, stream=stream)

    def load(self, pool_pages, slots, stream=None):
        """Store slots -> pool pages (host to device)."""
        self._check(pool_pages, slots)
        B.pfx_page_copy(self.pool, self.store.pool, pool_pages, slots, self.ws, stream=stream)

    @staticmethod
    def _runs(slots):
        """Maximal runs of consecutive store slots: (list index, first slot, length)."""
        slots = np.asarray(slots, np.int64)
        cut = np.nonzero(np.diff(slots) != 1)[0] + 1
        starts = np.concatenate([[0], cut])
        ends = np.concatenate([cut, [len(slots)]])
        return [(int(a), int(slots[a]), int(b - a)) for a, b in zip(starts, ends)]

    def _on(self, stream):
        return torch.cuda.ExternalStream(stream) if stream is not None else torch.cuda.current_stream()

    # Runs of at least this many pages that are consecutive both in the
    # store and in the pool cross the host link straight into the pool.
    DIRECT_RUN = 8

    def load_dma(self, pool_pages, slots, stream=None, pool_tensors=None, after=None):
        """Store slots -> pool pages through the copy engines (no compute
        units wait on the host link).  Runs of pages consecutive in the store
        and in the pool (``pool_tensors``: the pool's K and V tensors) are
        copied straight into the pool, one asynchronous memory copy per run
        and tensor.  The other pages cross, run by run of consecutive store
        slots, into the device staging area, and one device-to-device page
        copy then places them.

        after: events recorded on another stream (say one after each decode
        step).  The transfer is then cut into len(after) parts of about equal
        size, and part i starts once after[i] has completed: its writes into
        HBM are spread over those steps.  (Attention beside a host-to-device
        stream at the link's full rate runs about 15% slower; the same bytes
        spread thinner cost it less, at the price of a longer transfer.)"""
        self._check(pool_pages, slots)
        pool_pages = np.asarray(pool_pages, np.int64)
        slots = np.asarray(slots, np.int64)
        staged = np.ones(len(slots), bool)
        ops = []  # (dst K, dst V, first dst page, first store slot, pages)
        if pool_tensors is not None:
            pk, pv = pool_tensors
            for i0, s0, ln in self._runs(slots):
                # split the slot run where the pool pages stop being consecutive
                pp = pool_pages[i0:i0 + ln]
                for j0, p0, m in self._runs(pp):
                    if m < self.DIRECT_RUN:
                        continue
                    ops.append((pk, pv, p0, s0 + j0, m))
                    staged[i0 + j0:i0 + j0 + m] = False
        idx = np.nonzero(staged)[0]
        if len(idx):
            if self.stage is None:
                raise RuntimeError("this mover has no staging area (staging=True)")
            for i0, s0, ln in self._runs(slots[idx]):
                ops.append((self.stage_k, self.stage_v, i0, s0, ln))
        parts = self._split(ops, len(after)) if after else [ops]
        cur = self._on(stream)
        with torch.cuda.stream(cur):
            for i, part in enumerate(parts):
                if after:
                    cur.wait_event(after[i])
                for dk, dv, d0, s0, n in part:
                    dk[d0:d0 + n].copy_(self.store.k[s0:s0 + n], non_blocking=True)
                    dv[d0:d0 + n].copy_(self.store.v[s0:s0 + n], non_blocking=True)
        if len(idx):
            B.pfx_page_copy(self.pool, self.stage, pool_pages[idx].astype(np.int32),
                            np.arange(len(idx), dtype=np.int32), self.ws, stream=stream)

    @staticmethod
    def _split(ops, nparts):
        """The copies cut into nparts lists of about equal page counts (a
        copy that straddles a boundary is split)."""
        total = sum(op[4] for op in ops)
        per = max(1, -(-total // max(1, nparts)))
        parts, cur, room = [], [], per
        for dk, dv, d0, s0, n in ops:
            while n > 0:
                take = min(n, room)
                cur.append((dk, dv, d0, s0, take))
                d0, s0, n, room = d0 + take, s0 + take, n - take, room - take
                if room == 0:
                    parts.append(cur)
                    cur, room = [], per
        if cur:
            parts.append(cur)
        while len(parts) < nparts:
            parts.append([])
        return parts[:nparts] if len(parts) > nparts else parts

    def evict_dma(self, pool_pages, slots, stream=None):
        """Pool pages -> store slots through the copy engines: one device
        page copy gathers the pages into the staging area, then every run of
        consecutive store slots crosses the host link by one asynchronous
        memory copy."""
        self._check(pool_pages, slots)
        if self.stage is None:
            raise RuntimeError("this mover has no staging area (staging=True)")
        n = len(pool_pages)
        B.pfx_page_copy(self.stage, self.pool, np.arange(n, dtype=np.int32), pool_pages, self.ws, stream=stream)
        with torch.cuda.stream(self._on(stream)):
            for i0, s0, ln in self._runs(slots):
                self.store.k[s0:s0 + ln].copy_(self.stage_k[i0:i0 + ln], non_blocking=True)
                self.store.v[s0:s0 + ln].copy_(self.stage_v[i0:i0 + ln], non_blocking=True)


def t_move(mu: float, b_swap: float, tokens_out, tokens_in) -> float:
    """Eq. (8): seconds to move the prefixes of a transition, transfers
    serialized: mu / B_swap times the prefix tokens evicted plus loaded."""
    return mu / b_swap * (float(np.sum(tokens_out)) + float(np.sum(tokens_in)))


def calibrate_swap(mover: Mover, pages_list, tau: int, reps: int = 3):
    """B_swap per direction from timed transfers of several sizes: a least
    squares fit of time = overhead + bytes / B over the sizes.  mu is tau
    bytes per token (K and V of every KV head), given by the pool shape.
    Returns dict(mu, b_out, b_in, overhead_out_s, overhead_in_s, samples)."""
    samples = []
    for pages in pages_list:
        pages = np.asarray(pages, np.int32)
        slots = np.arange(len(pages), dtype=np.int32)
        nbytes = len(pages) * 16 * tau
        row = {"pages": int(len(pages)), "bytes": int(nbytes)}
        for name, fn in (("out", mover.evict), ("in", mover.load)):
            fn(pages, slots)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn(pages, slots)
            e1.record()
            torch.cuda.synchronize()
            row[f"s_{name}"] = e0.elapsed_time(e1) * 1e-3 / reps
        samples.append(row)
    x = np.array([r["bytes"] for r in samples], float)
    out = {"mu": tau, "samples": samples}
    for name in ("out", "in"):
        y = np.array([r[f"s_{name}"] for r in samples])
        slope, icpt = np.polyfit(x, y, 1) if len(x) > 1 else (y[0] / x[0], 0.0)
        out[f"b_{name}"] = 1.0 / slope
        out[f"overhead_{name}_s"] = float(icpt)
    return out
