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
    on a different stream before the previous one on this mover finished)."""

    def __init__(self, pool: B.pfx_pool, store: HostStore, max_pages: int, device="cuda"):
        self.pool, self.store = pool, store
        self.ws = torch.empty(B.pfx_page_copy_workspace_bytes(max_pages) + 256, dtype=torch.uint8, device=device)
        self.max_pages = max_pages

    def _check(self, pool_pages, slots):
        if len(pool_pages) != len(slots) or len(pool_pages) > self.max_pages:
            raise ValueError("page lists differ in length or exceed the mover's workspace")

    def evict(self, pool_pages, slots, stream=None):
        """Pool pages -> store slots (device to host)."""
        self._check(pool_pages, slots)
        B.pfx_page_copy(self.store.pool, self.pool, slots, pool_pages, self.ws, stream=stream)

    def load(self, pool_pages, slots, stream=None):
        """Store slots -> pool pages (host to device)."""
        self._check(pool_pages, slots)
        B.pfx_page_copy(self.pool, self.store.pool, pool_pages, slots, self.ws, stream=stream)


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
