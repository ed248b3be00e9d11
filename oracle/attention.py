"""fp64 reference for attention over a paged KV pool with shared agent prefixes.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline leg of the benchmark, never by the product path.

What is computed, and where it comes from
-----------------------------------------
The paper (TOPAS, "Workflow-Aware Prefix-State Scheduling for Multi-Agent LLM
Serving") serves requests whose prompt is an agent's static prefix followed by
the request's own dynamic content (Sec. 1, the radix-tree prefix cache; Sec. 3,
"Workflow and objective": requests of agent a share a static prefix of length
l_a).  A resident prefix is paid for once and reused by every request of that
agent (Sec. 3, Eq. (2) and the sentence after it; Sec. 2, Diagnostic 1).  The
computation those requests run on the GPU is ordinary causal softmax attention
over the concatenation [agent prefix ; request suffix].  Prefix sharing,
paging and splitting the key range into pieces whose results are recombined
are exact rewrites of that textbook definition, so this oracle computes the
definition itself:

  * a request r of agent a(r) has P = l_{a(r)} prefix tokens (P = 0 without an
    agent), L_r suffix tokens already in its pages (the newest n_r of them are
    the ones being computed this step) and n_r query rows;
  * query row i sits at absolute position t_i = P + (L_r - n_r) + i and sees
    keys 0..t_i: the whole prefix, and the suffix causally, itself included;
  * with G = Hq / Hkv consecutive query heads per KV head (h_kv = h // G):
        x_j = s * <q_{i,h}, k_{j,h_kv}>,  s = 1/sqrt(d) unless given,
        O = sum_j exp(x_j - m) v_j / sum_j exp(x_j - m),  m = max_j x_j,
        LSE = m + ln sum_j exp(x_j - m).

Readings where the paper is silent (softmax scale, GQA head mapping, mask,
page layout, rounding) are the ones listed in the design notes of the
repository; the paper specifies no attention numerics at all.

Pins (tests/test_oracle.py): brute force over the concatenated sequence with a
dense mask; rows of the softmax sum to one; split/merge equals monolithic
under random chunkings and merge orders; Q = 0 gives the mean of the visible
values and LSE = ln(t+1); constant V is reproduced exactly; a one-hot query
selects one value row; with no prefix the result equals torch's causal
scaled-dot-product attention run in float64; a decode row equals the
matching extend row; results do not depend on physical page placement; a
hand-derived two-key example stored under tests/golden/.

Every array here is float64 except bf16 inputs, which arrive as their uint16
bit patterns and are widened exactly.
"""

from __future__ import annotations

import math
from typing import Iterable, Mapping, Sequence

import numpy as np

# Tokens per KV page.  The paper names a paged KV pool (Sec. 1 and Sec. 6,
# PagedAttention-style allocation) but no page size; 16 is the value used
# throughout this repository.
PAGE_SIZE = 16


# --------------------------------------------------------------------------
# bf16 widening
# --------------------------------------------------------------------------

def bf16_bits_to_f64(bits) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float64 exactly.

    A bf16 value is the upper 16 bits of an IEEE-754 binary32 value, so
    shifting the pattern left by 16 gives the binary32 with the same value,
    and binary32 -> binary64 is exact.
    """
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Paged storage
# --------------------------------------------------------------------------

def gather_tokens(pool, page_ids: Sequence[int], length: int) -> np.ndarray:
    """Read ``length`` consecutive logical tokens out of a paged pool.

    ``pool[p]`` must return the bf16 bits of page p, shaped [Hkv][PAGE][d]
    (a numpy array [num_pages][Hkv][PAGE][d] works, so does a dict of pages).
    Token j lives in page ``page_ids[j // PAGE]`` at slot ``j % PAGE``; the
    loop walks the pages in order and takes the slots each one holds.
    Returns float64 [length][Hkv][d].
    """
    first = np.asarray(pool[page_ids[0]])
    out = np.empty((length, first.shape[0], first.shape[2]), dtype=np.float64)
    for i in range(pages_needed(length)):
        page = np.asarray(pool[page_ids[i]])                # [Hkv][PAGE][d]
        lo = i * PAGE_SIZE
        hi = min(lo + PAGE_SIZE, length)
        out[lo:hi] = bf16_bits_to_f64(page[:, :hi - lo, :]).transpose(1, 0, 2)
    return out


def pages_needed(length: int) -> int:
    """Pages a run of ``length`` tokens occupies (a partial last page counts)."""
    return (length + PAGE_SIZE - 1) // PAGE_SIZE


# --------------------------------------------------------------------------
# Attention, one request at a time
# --------------------------------------------------------------------------

def attend_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                positions: Sequence[int], num_q_heads: int, scale: float,
                heads: Iterable[int] | None = None):
    """Causal softmax attention of a few query rows against one key sequence.

    q: float64 [n][Hq][d]; k, v: float64 [N][Hkv][d]; positions[i] is the
    absolute position of query row i, which sees keys 0..positions[i].
    Returns O [n][Hq][d] and LSE [n][Hq] (natural log); heads not listed in
    ``heads`` are left as NaN.
    """
    n = q.shape[0]
    hkv = k.shape[1]
    d = k.shape[2]
    group = num_q_heads // hkv
    o = np.full((n, num_q_heads, d), np.nan)
    lse = np.full((n, num_q_heads), np.nan)
    heads = range(num_q_heads) if heads is None else heads
    pos = np.asarray(positions, dtype=np.int64)
    if n == 0:
        return o, lse
    key_index = np.arange(k.shape[0])
    visible = key_index[None, :] <= pos[:, None]            # [n][N]
    for h in heads:
        hk = h // group                                     # GQA: consecutive q heads share a KV head
        x = scale * (q[:, h, :] @ k[:, hk, :].T)            # [n][N] scores
        x = np.where(visible, x, -np.inf)
        m = x.max(axis=1, keepdims=True)
        w = np.exp(x - m)                                   # masked keys give exp(-inf) = 0
        z = w.sum(axis=1, keepdims=True)
        o[:, h, :] = (w @ v[:, hk, :]) / z
        lse[:, h] = m[:, 0] + np.log(z[:, 0])
    return o, lse


def _request_sequence(pool_k, pool_v, prefix_pages, prefix_len, agent,
                      suffix_pages, suffix_len, r):
    """Logical K and V of request r: its agent's prefix then its own suffix."""
    a = int(agent[r])
    plen = int(prefix_len[a]) if a >= 0 else 0
    slen = int(suffix_len[r])
    parts_k, parts_v = [], []
    if plen:
        parts_k.append(gather_tokens(pool_k, prefix_pages[a], plen))
        parts_v.append(gather_tokens(pool_v, prefix_pages[a], plen))
    if slen:
        parts_k.append(gather_tokens(pool_k, suffix_pages[r], slen))
        parts_v.append(gather_tokens(pool_v, suffix_pages[r], slen))
    return np.concatenate(parts_k), np.concatenate(parts_v), plen


def prefix_shared_attention(pool_k, pool_v, prefix_pages, prefix_len, agent,
                            suffix_pages, suffix_len, n_rows, q_bits,
                            num_q_heads: int, scale: float | None = None,
                            rows: Mapping[int, Sequence[int]] | None = None,
                            heads: Iterable[int] | None = None):
    """Outputs of every query row of a batch (the plain definition).

    prefix_pages[a] / suffix_pages[r]: page-id lists; prefix_len[a];
    agent[r] (-1 = no prefix); suffix_len[r] = L_r (includes this step's
    n_r new tokens); n_rows[r] = n_r; q_bits: bf16 bits [sum n_r][Hq][d],
    request r's rows contiguous and in request order.
    ``rows``, if given, maps request -> row indices to evaluate (the others
    stay NaN); by default every row of every request is computed.
    Returns O float64 [sum n_r][Hq][d] and LSE float64 [sum n_r][Hq].
    """
    q_all = np.asarray(q_bits)
    total = q_all.shape[0]
    d = q_all.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    o = np.full((total, num_q_heads, d), np.nan)
    lse = np.full((total, num_q_heads), np.nan)
    offset = 0
    for r in range(len(agent)):
        n = int(n_rows[r])
        want = range(n) if rows is None else rows.get(r, ())
        want = [int(i) for i in want]
        if n and want:
            k, v, plen = _request_sequence(pool_k, pool_v, prefix_pages,
                                           prefix_len, agent, suffix_pages,
                                           suffix_len, r)
            base = plen + int(suffix_len[r]) - n
            qr = bf16_bits_to_f64(q_all[offset + np.asarray(want)])
            orr, lr = attend_rows(qr, k, v, [base + i for i in want],
                                  num_q_heads, scale, heads)
            o[offset + np.asarray(want)] = orr
            lse[offset + np.asarray(want)] = lr
        offset += n
    return o, lse


# --------------------------------------------------------------------------
# The method's structure: partial results over key ranges, then an LSE merge
# --------------------------------------------------------------------------

def merge_partials(o_parts: Sequence[np.ndarray], lse_parts: Sequence[np.ndarray]):
    """Combine attention results computed over disjoint key ranges.

    With partial outputs O_k (each already normalised over its own keys) and
    their log-sum-exps l_k, the result over the union of the ranges is
        l = ln sum_k exp(l_k),   O = sum_k exp(l_k - l) O_k.
    Shapes: O_k [..., d], l_k [...].
    """
    lse = np.log(sum(np.exp(l) for l in lse_parts))
    o = sum(np.exp(l - lse)[..., None] * ok for ok, l in zip(o_parts, lse_parts))
    return o, lse


def split_attention(pool_k, pool_v, prefix_pages, prefix_len, agent,
                    suffix_pages, suffix_len, n_rows, q_bits,
                    num_q_heads: int, scale: float | None = None,
                    prefix_chunk: int | None = None, suffix_chunk: int | None = None,
                    rng: np.random.Generator | None = None):
    """Same outputs as ``prefix_shared_attention``, computed the method's way.

    Each request's keys are cut into a prefix part (optionally into chunks of
    ``prefix_chunk`` tokens) and a suffix part (optionally chunks of
    ``suffix_chunk``); each piece is attended on its own, and the pieces are
    combined by ``merge_partials`` (in a random order when ``rng`` is given).
    Query rows that see none of a piece's keys take no part in that piece.
    """
    q_all = np.asarray(q_bits)
    d = q_all.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    total = q_all.shape[0]
    o = np.full((total, num_q_heads, d), np.nan)
    lse = np.full((total, num_q_heads), np.nan)
    offset = 0
    for r in range(len(agent)):
        n = int(n_rows[r])
        if n == 0:
            continue
        k, v, plen = _request_sequence(pool_k, pool_v, prefix_pages, prefix_len,
                                       agent, suffix_pages, suffix_len, r)
        slen = int(suffix_len[r])
        qr = bf16_bits_to_f64(q_all[offset:offset + n])
        pos = np.arange(n) + plen + slen - n
        pieces = []
        step = prefix_chunk or max(plen, 1)
        for lo in range(0, plen, step):
            pieces.append((lo, min(lo + step, plen)))
        step = suffix_chunk or max(slen, 1)
        for lo in range(plen, plen + slen, step):
            pieces.append((lo, min(lo + step, plen + slen)))
        if rng is not None:
            rng.shuffle(pieces)
        for i in range(n):
            o_parts, l_parts = [], []
            for lo, hi in pieces:
                if lo > pos[i]:
                    continue                     # the row sees none of these keys
                hi_i = min(hi, pos[i] + 1)
                # Positions are relative to the piece, so every key is visible.
                po, pl = attend_rows(qr[i:i + 1], k[lo:hi_i], v[lo:hi_i],
                                     [hi_i - lo - 1], num_q_heads, scale)
                o_parts.append(po[0])
                l_parts.append(pl[0])
            oi, li = merge_partials(o_parts, l_parts)
            o[offset + i] = oi
            lse[offset + i] = li
        offset += n
    return o, lse


# --------------------------------------------------------------------------
# Byte movement: KV append and page copy
# --------------------------------------------------------------------------

def append_kv(pool_k, pool_v, suffix_pages, suffix_len, n_rows, k_new, v_new):
    """Expected pools after writing each request's new tokens.

    Request r's n_r new tokens (rows of k_new / v_new, [sum n_r][Hkv][d] bf16
    bits, request order) go to suffix positions L_r - n_r .. L_r - 1, i.e.
    page suffix_pages[r][pos // PAGE], slot pos % PAGE.  Pure byte copy:
    returns modified copies of the input pools (numpy uint16 arrays).
    """
    out_k = np.array(pool_k, copy=True)
    out_v = np.array(pool_v, copy=True)
    row = 0
    for r in range(len(suffix_len)):
        n = int(n_rows[r])
        for i in range(n):
            pos = int(suffix_len[r]) - n + i
            page = suffix_pages[r][pos // PAGE_SIZE]
            out_k[page, :, pos % PAGE_SIZE, :] = k_new[row]
            out_v[page, :, pos % PAGE_SIZE, :] = v_new[row]
            row += 1
    return out_k, out_v


def page_copy(dst, src, dst_pages: Sequence[int], src_pages: Sequence[int]):
    """Expected destination store after copying whole pages.

    Prefix movement between host and GPU memory (Sec. 4.2, Eq. (8) and the
    paragraph before it: prefix KV moves as agents enter and leave the
    resident set) is a byte copy: dst[dst_pages[i]] = src[src_pages[i]].
    Pages not named in dst_pages are unchanged.
    """
    out = np.array(dst, copy=True)
    for di, si in zip(dst_pages, src_pages):
        out[di] = src[si]
    return out
