"""Seeded synthetic workloads shaped like the paper's agent workflows.

This module only draws sizes, lengths, page placements and random bf16
values.  It holds none of the attention arithmetic, so both the HIP path and
the fp64 oracle may consume what it produces.

The paper evaluates on MetaGPT traces and synthetic DAGs with an unspecified
prompt mix (Sec. 5.1); none of those prompts, traces or weights are used.
The five workloads below are synthetic stand-ins with the shapes of the
layer the paper's setting runs (prefix-sharing agents, grouped decode,
suffix extend, prefix movement) at Llama-3-8B and -70B attention shapes:

  1. tiny: Hq 8, Hkv 2, d 64; one 128-token prefix in a 64-page pool at
     shuffled page ids; 4 requests extend a 32-token suffix, then 16 decode
     steps each appending one token.
  2. decode-8B: Hq 32, Hkv 8, d 128; 4 prefixes x 2048 tokens; 64 decode
     requests, 16 per agent, suffix lengths U[64, 512]; 65,536-page pool.
  3. extend-8B: same shape; 3 prefixes x 4096; 32 extend requests with
     suffix lengths U[256, 2048] (every suffix token is a query row),
     request r belongs to agent r mod 3; 65,536-page pool.
  4. hetero-8B: same shape; 16 prefixes of log-uniform length in
     [512, 8192]; 256 decode requests assigned by a finite Zipf(1.1) over
     16 ranks (a seeded permutation maps rank -> agent); suffix lengths
     U[32, 1024]; 786,432-page (48 GiB) pool; 4 seeded agents start evicted
     in a host page store and are gathered back before decode.
  5. mixed-70B: Hq 64, Hkv 8, d 128; 8 prefixes x 8192; per layer 32 extend
     requests (suffix U[512, 4096]) and 448 decode requests (suffix
     U[64, 2048]) spread evenly over the agents; 80 layers, each with its own
     pool holding identical page tables.

Integer "uniform in [a, b]" is inclusive.  Values are float32 N(0, 1) rounded
to bf16 with round-to-nearest-even.  A suffix always starts on a fresh page;
the new tokens of a step are the last n_r of the suffix.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
# A quiet-NaN bf16 pattern used to poison pool slots that no step may read.
POISON_BF16 = 0x7FC1


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round-to-nearest-even (input generation)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def _pages(length: int) -> int:
    return (length + PAGE_SIZE - 1) // PAGE_SIZE


@dataclass
class Batch:
    """Host description of one step: pool shape, prefix table and requests."""
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_pages: int
    prefix_len: np.ndarray            # int32 [A]
    prefix_pages: list                # list of int32 arrays, one per agent
    agent: np.ndarray                 # int32 [R], -1 = no prefix
    suffix_len: np.ndarray            # int32 [R], includes this step's new tokens
    n_rows: np.ndarray                # int32 [R], query rows (new tokens) this step
    suffix_pages: list                # list of int32 arrays, one per request
    meta: dict = field(default_factory=dict)

    # ---- CSR views, as the C interface takes them ----
    def prefix_csr(self):
        indptr = np.zeros(len(self.prefix_pages) + 1, dtype=np.int32)
        for a, p in enumerate(self.prefix_pages):
            indptr[a + 1] = indptr[a] + len(p)
        ids = (np.concatenate(self.prefix_pages).astype(np.int32)
               if len(self.prefix_pages) else np.zeros(0, np.int32))
        return indptr, ids, np.asarray(self.prefix_len, dtype=np.int32)

    def suffix_csr(self):
        indptr = np.zeros(len(self.suffix_pages) + 1, dtype=np.int32)
        for r, p in enumerate(self.suffix_pages):
            indptr[r + 1] = indptr[r] + len(p)
        ids = (np.concatenate(self.suffix_pages).astype(np.int32)
               if len(self.suffix_pages) else np.zeros(0, np.int32))
        return indptr, ids

    def q_indptr(self):
        out = np.zeros(len(self.n_rows) + 1, dtype=np.int32)
        out[1:] = np.cumsum(self.n_rows)
        return out

    @property
    def num_tokens(self) -> int:
        return int(np.sum(self.n_rows))

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def used_pages(self) -> np.ndarray:
        parts = [np.asarray(p) for p in self.prefix_pages] + [np.asarray(p) for p in self.suffix_pages]
        return np.concatenate(parts).astype(np.int64) if parts else np.zeros(0, np.int64)

    # ---- algorithmic work (counts of tokens, not of padded pages) ----
    def unique_kv_bytes(self) -> int:
        """Bytes of K and V that a step must read at least once: every
        referenced agent prefix once, plus every request's own suffix."""
        tau = self.num_kv_heads * self.head_dim * 2 * 2
        agents = {int(a) for a, n in zip(self.agent, self.n_rows) if a >= 0 and n > 0}
        toks = sum(int(self.prefix_len[a]) for a in agents)
        toks += sum(int(l) for l, n in zip(self.suffix_len, self.n_rows) if n > 0)
        return toks * tau

    def attention_flops(self) -> int:
        """Causal-exact flops: 4*d per (query head, visible key) pair
        (one multiply-add for QK^T and one for PV)."""
        total = 0
        for r in range(len(self.agent)):
            n = int(self.n_rows[r])
            if n == 0:
                continue
            a = int(self.agent[r])
            p = int(self.prefix_len[a]) if a >= 0 else 0
            l = int(self.suffix_len[r])
            visible = n * p + sum(l - n + i + 1 for i in range(n))
            total += visible
        return 4 * self.head_dim * self.num_q_heads * total


def place_pages(rng: np.random.Generator, num_pages: int, prefix_len, suffix_len):
    """Scatter prefix and suffix pages over a seeded permutation of the pool."""
    need = sum(_pages(int(p)) for p in prefix_len) + sum(_pages(int(s)) for s in suffix_len)
    if need > num_pages:
        raise ValueError(f"workload needs {need} pages, pool has {num_pages}")
    if num_pages <= 4_000_000:
        order = rng.permutation(num_pages)[:need]
    else:  # pragma: no cover - not used by the configs
        order = rng.choice(num_pages, size=need, replace=False)
    order = order.astype(np.int32)
    at = 0
    prefix_pages, suffix_pages = [], []
    for p in prefix_len:
        k = _pages(int(p))
        prefix_pages.append(order[at:at + k].copy())
        at += k
    for s in suffix_len:
        k = _pages(int(s))
        suffix_pages.append(order[at:at + k].copy())
        at += k
    return prefix_pages, suffix_pages, order[at:]


def make_batch(seed: int, *, num_q_heads: int, num_kv_heads: int, head_dim: int,
               num_pages: int, prefix_len, agent, suffix_len, n_rows, meta=None) -> Batch:
    rng = np.random.Generator(np.random.PCG64(seed))
    prefix_len = np.asarray(prefix_len, dtype=np.int32)
    suffix_len = np.asarray(suffix_len, dtype=np.int32)
    pp, sp, _ = place_pages(rng, num_pages, prefix_len, suffix_len)
    return Batch(num_q_heads, num_kv_heads, head_dim, num_pages, prefix_len, pp,
                 np.asarray(agent, dtype=np.int32), suffix_len,
                 np.asarray(n_rows, dtype=np.int32), sp, dict(meta or {}))


def zipf_agents(rng: np.random.Generator, num_agents: int, num_requests: int, s: float):
    """Finite Zipf: P(rank k) proportional to k^-s for k = 1..num_agents; a seeded
    permutation maps ranks to agent ids."""
    w = np.arange(1, num_agents + 1, dtype=np.float64) ** (-s)
    w /= w.sum()
    ranks = rng.choice(num_agents, size=num_requests, p=w)
    perm = rng.permutation(num_agents)
    return perm[ranks].astype(np.int32)


def config_batch(cfg: int, seed: int | None = None) -> Batch:
    """The batch description (no values) of one of the five workloads.

    Config 1 returns its extend step; ``tiny_decode_step`` gives the decode
    steps that follow it.  Config 5 returns one layer's batch (all 80 layers
    share it).
    """
    seed = 1000 + cfg if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    sub = int(rng.integers(0, 2**31 - 1))
    if cfg == 1:
        return make_batch(sub, num_q_heads=8, num_kv_heads=2, head_dim=64, num_pages=64,
                          prefix_len=[128], agent=[0, 0, 0, 0], suffix_len=[32] * 4,
                          n_rows=[32] * 4, meta=dict(config=1, name="tiny"))
    if cfg == 2:
        agents = np.repeat(np.arange(4), 16).astype(np.int32)
        agents = agents[rng.permutation(64)]
        slen = rng.integers(64, 512, size=64, endpoint=True)
        return make_batch(sub, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536,
                          prefix_len=[2048] * 4, agent=agents, suffix_len=slen,
                          n_rows=np.ones(64, np.int32), meta=dict(config=2, name="decode-8B"))
    if cfg == 3:
        slen = rng.integers(256, 2048, size=32, endpoint=True)
        agents = (np.arange(32) % 3).astype(np.int32)
        return make_batch(sub, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536,
                          prefix_len=[4096] * 3, agent=agents, suffix_len=slen, n_rows=slen,
                          meta=dict(config=3, name="extend-8B"))
    if cfg == 4:
        plen = np.floor(np.exp(rng.uniform(math.log(512), math.log(8192), size=16))).astype(np.int32)
        agents = zipf_agents(rng, 16, 256, 1.1)
        slen = rng.integers(32, 1024, size=256, endpoint=True)
        evicted = np.sort(rng.choice(16, size=4, replace=False)).astype(np.int32)
        b = make_batch(sub, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=786432,
                       prefix_len=plen, agent=agents, suffix_len=slen,
                       n_rows=np.ones(256, np.int32),
                       meta=dict(config=4, name="hetero-8B", evicted=evicted))
        return b
    if cfg == 5:
        ext = rng.integers(512, 4096, size=32, endpoint=True)
        dec = rng.integers(64, 2048, size=448, endpoint=True)
        agents = np.concatenate([np.arange(32) % 8, np.arange(448) % 8]).astype(np.int32)
        slen = np.concatenate([ext, dec])
        nrows = np.concatenate([ext, np.ones(448, np.int64)])
        need = 8 * _pages(8192) + sum(_pages(int(s)) for s in slen)
        pool = int(math.ceil(need * 1.02))
        return make_batch(sub, num_q_heads=64, num_kv_heads=8, head_dim=128, num_pages=pool,
                          prefix_len=[8192] * 8, agent=agents, suffix_len=slen, n_rows=nrows,
                          meta=dict(config=5, name="mixed-70B", layers=80))
    raise ValueError(f"unknown config {cfg}")


def with_lengths(batch: Batch, suffix_len, n_rows) -> Batch:
    """The same pool, prefixes and request pages with other suffix lengths
    and query rows: each request keeps the first pages its length needs
    (its page list may have been sized for a longer suffix)."""
    suffix_len = np.asarray(suffix_len, dtype=np.int32)
    pages = [np.asarray(p[:_pages(int(l))], dtype=np.int32) for p, l in zip(batch.suffix_pages, suffix_len)]
    return Batch(batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.num_pages, batch.prefix_len,
                 batch.prefix_pages, batch.agent, suffix_len, np.asarray(n_rows, dtype=np.int32), pages,
                 dict(batch.meta))


def tiny_decode_step(extend: Batch, step: int, extra_pages: list) -> Batch:
    """Config 1, decode step ``step`` (0..15) after the extend step: every
    request has one new token at suffix position 32 + step.  ``extra_pages``
    holds, per request, the page added when the suffix outgrows two pages."""
    slen = extend.suffix_len + 1 + step
    pages = [np.concatenate([p, [e]]).astype(np.int32) for p, e in zip(extend.suffix_pages, extra_pages)]
    return Batch(extend.num_q_heads, extend.num_kv_heads, extend.head_dim, extend.num_pages,
                 extend.prefix_len, extend.prefix_pages, extend.agent, slen.astype(np.int32),
                 np.ones_like(extend.n_rows), pages, dict(extend.meta, step=step))


# --------------------------------------------------------------------------
# Values
# --------------------------------------------------------------------------

@dataclass
class HostValues:
    """bf16 bit patterns for one step, held compactly on the host.

    pages: sorted ids of the pool pages that hold data; k_pages / v_pages:
    [len(pages)][Hkv][16][d] contents of those pages *before* the append
    (poison in every slot that the step's append fills or nothing owns);
    q: [T][Hq][d]; k_new / v_new: [T][Hkv][d].
    """
    pages: np.ndarray
    k_pages: np.ndarray
    v_pages: np.ndarray
    q: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray

    def page_map(self, which: str):
        arr = self.k_pages if which == "k" else self.v_pages
        return {int(p): arr[i] for i, p in enumerate(self.pages)}


def _normal_bf16(rng, shape):
    return bf16_round(rng.standard_normal(size=shape, dtype=np.float32))


def host_values(batch: Batch, seed: int) -> HostValues:
    """Draw every value of a step on the host (configs 1-4 and small cases)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    hkv, d = batch.num_kv_heads, batch.head_dim
    pages = np.unique(batch.used_pages())
    index = {int(p): i for i, p in enumerate(pages)}
    kp = np.full((len(pages), hkv, PAGE_SIZE, d), POISON_BF16, dtype=np.uint16)
    vp = np.full_like(kp, POISON_BF16)

    def fill(page_list, length):
        for j in range(length):
            i = index[int(page_list[j // PAGE_SIZE])]
            kp[i, :, j % PAGE_SIZE, :] = _normal_bf16(rng, (hkv, d))
            vp[i, :, j % PAGE_SIZE, :] = _normal_bf16(rng, (hkv, d))

    for a, pl in enumerate(batch.prefix_pages):
        fill(pl, int(batch.prefix_len[a]))
    for r, pl in enumerate(batch.suffix_pages):
        fill(pl, int(batch.suffix_len[r]) - int(batch.n_rows[r]))
    t = batch.num_tokens
    q = _normal_bf16(rng, (t, batch.num_q_heads, d))
    kn = _normal_bf16(rng, (t, hkv, d))
    vn = _normal_bf16(rng, (t, hkv, d))
    return HostValues(pages, kp, vp, q, kn, vn)


def host_values_fast(batch: Batch, seed: int) -> HostValues:
    """Like ``host_values`` but draws whole pages at once (large configs).
    Slots a step's append fills, and slots past a run's end, are poisoned."""
    rng = np.random.Generator(np.random.PCG64(seed))
    hkv, d = batch.num_kv_heads, batch.head_dim
    pages = np.unique(batch.used_pages())
    index = {int(p): i for i, p in enumerate(pages)}
    kp = _normal_bf16(rng, (len(pages), hkv, PAGE_SIZE, d))
    vp = _normal_bf16(rng, (len(pages), hkv, PAGE_SIZE, d))

    def poison(page_list, start, end_exclusive_pages_tokens):
        for j in range(start, end_exclusive_pages_tokens):
            i = index[int(page_list[j // PAGE_SIZE])]
            kp[i, :, j % PAGE_SIZE, :] = POISON_BF16
            vp[i, :, j % PAGE_SIZE, :] = POISON_BF16

    for a, pl in enumerate(batch.prefix_pages):
        poison(pl, int(batch.prefix_len[a]), len(pl) * PAGE_SIZE)
    for r, pl in enumerate(batch.suffix_pages):
        poison(pl, int(batch.suffix_len[r]) - int(batch.n_rows[r]), len(pl) * PAGE_SIZE)
    t = batch.num_tokens
    q = _normal_bf16(rng, (t, batch.num_q_heads, d))
    kn = _normal_bf16(rng, (t, hkv, d))
    vn = _normal_bf16(rng, (t, hkv, d))
    return HostValues(pages, kp, vp, q, kn, vn)


def replicas(batch: Batch, count: int, seed: int) -> list:
    """``count`` copies of a batch's lengths and agents whose pages are
    pairwise disjoint within the same pool (replica 0 is ``batch`` itself).
    Used to rotate the benchmark over a working set larger than the GPU's
    last-level cache."""
    rng = np.random.Generator(np.random.PCG64(seed))
    used = set(int(p) for p in batch.used_pages())
    free = np.array([p for p in range(batch.num_pages) if p not in used], np.int32)
    free = free[rng.permutation(len(free))]
    out = [batch]
    at = 0
    per = len(batch.used_pages())
    for _ in range(count - 1):
        if at + per > len(free):
            break
        take = free[at:at + per]
        at += per
        k = 0
        pp, sp = [], []
        for pl in batch.prefix_pages:
            pp.append(take[k:k + len(pl)].copy())
            k += len(pl)
        for pl in batch.suffix_pages:
            sp.append(take[k:k + len(pl)].copy())
            k += len(pl)
        out.append(Batch(batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.num_pages, batch.prefix_len,
                         pp, batch.agent, batch.suffix_len, batch.n_rows, sp, dict(batch.meta, replica=len(out))))
    return out


def host_values_shaped(batch: Batch, seed: int, key_gain=None, q_gain: float = 1.0,
                       v_gain: float = 1.0) -> HostValues:
    """Like ``host_values``, with every value drawn N(0, 1) and multiplied
    before rounding to bf16: a key at absolute position p (prefix token j of
    an agent sits at p = j, suffix token j of request r at p = l_a(r) + j)
    by ``key_gain(p)``, queries by ``q_gain`` and values by ``v_gain``.
    A key gain that grows with p makes the largest scores rise along the
    sequence, so a running maximum keeps being raised."""
    rng = np.random.Generator(np.random.PCG64(seed))
    hkv, d = batch.num_kv_heads, batch.head_dim
    gain = key_gain or (lambda p: 1.0)
    pages = np.unique(batch.used_pages())
    index = {int(p): i for i, p in enumerate(pages)}
    kp = np.full((len(pages), hkv, PAGE_SIZE, d), POISON_BF16, dtype=np.uint16)
    vp = np.full_like(kp, POISON_BF16)

    def draw(shape, g):
        return bf16_round(rng.standard_normal(size=shape, dtype=np.float32) * np.float32(g))

    def fill(page_list, length, base):
        for j in range(length):
            i = index[int(page_list[j // PAGE_SIZE])]
            kp[i, :, j % PAGE_SIZE, :] = draw((hkv, d), gain(base + j))
            vp[i, :, j % PAGE_SIZE, :] = draw((hkv, d), v_gain)

    for a, pl in enumerate(batch.prefix_pages):
        fill(pl, int(batch.prefix_len[a]), 0)
    t = batch.num_tokens
    kn = np.zeros((t, hkv, d), np.uint16)
    vn = np.zeros_like(kn)
    row = 0
    for r, pl in enumerate(batch.suffix_pages):
        a = int(batch.agent[r])
        base = int(batch.prefix_len[a]) if a >= 0 else 0
        n, L = int(batch.n_rows[r]), int(batch.suffix_len[r])
        fill(pl, L - n, base)
        for i in range(n):
            kn[row] = draw((hkv, d), gain(base + L - n + i))
            vn[row] = draw((hkv, d), v_gain)
            row += 1
    q = draw((t, batch.num_q_heads, d), q_gain)
    return HostValues(pages, kp, vp, q, kn, vn)


def plant_one_hot(batch: Batch, hv: HostValues, seed: int, alpha_log2: int = 4) -> HostValues:
    """Queries aimed at one key each: for every query row and head, a seeded
    visible key j* (its agent's prefix, or its own suffix up to and including
    the row's own token) and q = 2^alpha_log2 * k[j*] (exact in bf16), so
    that one score stands far above all others."""
    rng = np.random.Generator(np.random.PCG64(seed))
    index = {int(p): i for i, p in enumerate(hv.pages)}
    g = batch.group
    q = hv.q.copy()
    shift = np.uint16(alpha_log2 << 7)   # add alpha_log2 to the bf16 exponent field
    row = 0
    for r in range(len(batch.agent)):
        a = int(batch.agent[r])
        P = int(batch.prefix_len[a]) if a >= 0 else 0
        n, L = int(batch.n_rows[r]), int(batch.suffix_len[r])
        for i in range(n):
            visible = P + L - n + i + 1
            for h in range(batch.num_q_heads):
                j = int(rng.integers(0, visible))
                if j < P:
                    pg, slot = batch.prefix_pages[a][j // PAGE_SIZE], j % PAGE_SIZE
                    k = hv.k_pages[index[int(pg)], h // g, slot]
                elif j - P < L - n:
                    s = j - P
                    pg, slot = batch.suffix_pages[r][s // PAGE_SIZE], s % PAGE_SIZE
                    k = hv.k_pages[index[int(pg)], h // g, slot]
                else:
                    k = hv.k_new[row - i + (j - P - (L - n)), h // g]
                nz = (k & np.uint16(0x7F80)) != 0   # zeros stay zero; normal values scale exactly
                q[row, h] = np.where(nz, k + shift, k)
            row += 1
    return HostValues(hv.pages, hv.k_pages, hv.v_pages, q, hv.k_new, hv.v_new)
