"""Executes prefix-state scheduling decisions (Sec. 3-4) on one GPU's KV
pool through the library's calls.

A decision S' = (R', Q') (``scheduler.Decision``) turns into:
  * movement (Eq. (8)): prefixes leaving the resident set are written to a
    pinned host page store and their pool pages freed; prefixes entering it
    get free pool pages and are loaded back (``pfx_page_copy`` both ways,
    serialized on the stream);
  * preemption: a preempted request's KV pages are freed; its tokens must be
    rebuilt when it is admitted again (Eq. (9));
  * admission: an admitted request gets pages for its prompt, whose K/V are
    appended and attended (one extend call over the prompt rows against its
    agent's resident prefix);
and each decode step appends one token per running request and attends
(one decode call: every running request of an agent reads that agent's
prefix pages once, Sec. 3, Eq. (2)).

Product side: the binding, the movement helpers and torch only.
"""

from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from .movement import HostStore, Mover

PAGE = 16


def _pages(tokens: int) -> int:
    return (tokens + PAGE - 1) // PAGE


class Engine:
    """One layer's KV pool plus the host store holding every agent's prefix.

    prefixes: per agent, (k_bits, v_bits) uint16 arrays [l_a][Hkv][d] of its
    static prefix KV (post-RoPE; the host store keeps the master copy)."""

    def __init__(self, num_pages: int, num_q_heads: int, num_kv_heads: int, head_dim: int, prefixes,
                 device="cuda"):
        self.hq, self.hkv, self.d = num_q_heads, num_kv_heads, head_dim
        self.num_pages = num_pages
        self.device = device
        shape = (num_pages, num_kv_heads, PAGE, head_dim)
        self.k_pool = torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self.v_pool = torch.zeros(shape, dtype=torch.bfloat16, device=device)
        self.pool = B.make_pool(num_pages, num_kv_heads, head_dim, self.k_pool, self.v_pool)
        self.alloc = B.Allocator(num_pages)
        self.prefix_len = [int(k.shape[0]) for k, _ in prefixes]
        store_pages = sum(_pages(l) for l in self.prefix_len)
        self.store = HostStore(store_pages, num_kv_heads, head_dim)
        self.mover = Mover(self.pool, self.store, max(1, max(_pages(l) for l in self.prefix_len)), device=device)
        self.store_slots = {}
        # The store's pages of each prefix, written once from the host arrays.
        for a, (k, v) in enumerate(prefixes):
            n = _pages(self.prefix_len[a])
            slots = self.store.alloc.alloc(n)
            self.store_slots[a] = slots
            for kind, src in (("k", k), ("v", v)):
                dst = getattr(self.store, kind)
                pad = np.zeros((n * PAGE, num_kv_heads, head_dim), np.uint16)
                pad[:len(src)] = src
                pages = torch.from_numpy(pad.reshape(n, PAGE, num_kv_heads, head_dim).transpose(0, 2, 1, 3)
                                         .copy().view(np.int16))
                dst.view(torch.int16)[torch.from_numpy(slots.astype(np.int64))] = pages
        self.resident = {}          # agent -> pool page ids of its prefix
        self.req_pages = {}         # request -> pool page ids of its own tokens
        self.req_len = {}           # request -> tokens in its pages
        self.req_agent = {}
        self.moved_tokens = 0       # prefix tokens moved in or out so far

    # ---- movement ----
    def evict(self, agent: int, stream=None):
        pages = self.resident.pop(agent)
        self.mover.evict(pages, self.store_slots[agent], stream=stream)
        self.alloc.free(pages)
        self.moved_tokens += self.prefix_len[agent]

    def load(self, agent: int, stream=None):
        pages = self.alloc.alloc(_pages(self.prefix_len[agent]))
        self.mover.load(pages, self.store_slots[agent], stream=stream)
        self.resident[agent] = pages
        self.moved_tokens += self.prefix_len[agent]

    def release(self, rid: int):
        """A finished or preempted request's pages go back to the pool."""
        self.alloc.free(self.req_pages.pop(rid))
        self.req_len.pop(rid)
        self.req_agent.pop(rid)

    # ---- batches ----
    def _grow(self, rid: int, tokens: int):
        have = self.req_pages.get(rid, np.zeros(0, np.int32))
        need = _pages(self.req_len.get(rid, 0) + tokens) - len(have)
        if need > 0:
            have = np.concatenate([have, self.alloc.alloc(need)]).astype(np.int32)
        self.req_pages[rid] = have
        self.req_len[rid] = self.req_len.get(rid, 0) + tokens

    def _plan(self, rids, n_rows, mode):
        agents = sorted(self.resident)
        index = {a: i for i, a in enumerate(agents)}
        pind = np.zeros(len(agents) + 1, np.int32)
        for i, a in enumerate(agents):
            pind[i + 1] = pind[i] + len(self.resident[a])
        pids = np.concatenate([self.resident[a] for a in agents]).astype(np.int32) if agents else np.zeros(0, np.int32)
        plen = np.array([self.prefix_len[a] for a in agents], np.int32)
        agent = np.array([index[self.req_agent[r]] if self.req_agent[r] >= 0 else -1 for r in rids], np.int32)
        sind = np.zeros(len(rids) + 1, np.int32)
        for i, r in enumerate(rids):
            sind[i + 1] = sind[i] + len(self.req_pages[r])
        sids = np.concatenate([self.req_pages[r] for r in rids]).astype(np.int32)
        slen = np.array([self.req_len[r] for r in rids], np.int32)
        qind = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
        return B.pfx_plan_create(self.pool, pind, pids, plen, agent, sind, sids, slen, qind, self.hq, mode).upload(
            device=self.device)

    def run(self, rids, n_rows, q, k_new, v_new, mode):
        """Append each request's n_rows new tokens (rows in request order) and
        attend; returns (o, lse) device tensors."""
        for r, n in zip(rids, n_rows):
            self._grow(r, int(n))
        plan = self._plan(rids, n_rows, mode)
        o = torch.empty_like(q)
        lse = torch.empty(q.shape[:2], dtype=torch.float32, device=self.device)
        B.pfx_append_kv(self.pool, plan, k_new, v_new)
        B.pfx_attention(self.pool, plan, q, o, lse)
        self._last_plan = plan
        return o, lse

    def prefill(self, rid: int, agent: int, q, k_new, v_new):
        """An admitted request's prompt: its tokens appended and attended
        (causal) against its agent's resident prefix."""
        if agent >= 0 and agent not in self.resident:
            raise RuntimeError(f"request {rid}: agent {agent}'s prefix is not resident")
        self.req_agent[rid] = agent
        return self.run([rid], [q.shape[0]], q, k_new, v_new, B.PFX_MODE_EXTEND)

    def decode(self, rids, q, k_new, v_new):
        """One decode step: one new token per request."""
        for r in rids:
            a = self.req_agent[r]
            if a >= 0 and a not in self.resident:
                raise RuntimeError(f"request {r}: agent {a}'s prefix is not resident")
        return self.run(list(rids), [1] * len(rids), q, k_new, v_new, B.PFX_MODE_DECODE)

    def apply(self, decision, stream=None):
        """Movement and preemption of a decision: prefixes of R_t - R' out,
        preempted requests released, prefixes of R' - R_t in (transfers
        serialized on the stream).  Admitted requests are prefilled by the
        caller with their prompts (``prefill``)."""
        r_new = set(decision.resident)
        for r in decision.preempted:
            self.release(r)
        for a in sorted(set(self.resident) - r_new):
            self.evict(a, stream=stream)
        for a in sorted(r_new - set(self.resident)):
            self.load(a, stream=stream)

    def read_pages(self, pages):
        idx = torch.from_numpy(np.asarray(pages, np.int64)).to(self.device)
        k = self.k_pool.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        v = self.v_pool.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        return k, v
