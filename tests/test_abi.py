"""Host-side tests of the C interface: no GPU needed (no kernel is launched).

The library is loaded, every function the header declares is exported, the
allocator and the plan builder are exercised, every validation error code is
reached, and the work list is checked to cover each visible (query row,
head, key) triple exactly once.
"""

import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2608_25523_amd import binding as B
from paper_2608_25523_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "pfx_attn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pfx_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 19
    lib = C.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.EXPORTED)


def test_version_and_error_text():
    assert B.pfx_version() == 20200
    with pytest.raises(B.PfxError):
        B.Allocator(-1)
    assert "num_pages" in B.pfx_last_error()


def test_allocator_is_lifo_and_checks():
    a = B.Allocator(5)
    assert list(a.alloc(3)) == [0, 1, 2]
    assert a.num_free() == 2
    a.free([1, 0])
    assert list(a.alloc(2)) == [0, 1]          # last freed comes back first
    with pytest.raises(B.PfxError) as e:
        a.alloc(4)
    assert e.value.code == B.PFX_ENOMEM
    assert a.num_free() == 2                    # nothing handed out on failure
    for bad in ([7], [3], [0, 0]):
        with pytest.raises(B.PfxError) as e:
            a.free(bad)
        assert e.value.code == B.PFX_EINVAL
    assert a.num_free() == 2


def small_batch(**over):
    kw = dict(num_q_heads=8, num_kv_heads=2, head_dim=64, num_pages=64, prefix_len=[40, 17],
              agent=[0, 1, 0, -1, 1], suffix_len=[5, 20, 33, 3, 16], n_rows=[1, 1, 33, 3, 2])
    kw.update(over)
    return W.make_batch(11, **kw)


def plan_for(batch, pool=None, mode=B.PFX_MODE_MIXED, **kw):
    pool = pool or B.make_pool(batch.num_pages, batch.num_kv_heads, batch.head_dim)
    return B.plan_from_batch(pool, batch, mode, **kw)


def expect_error(code, fn):
    with pytest.raises(B.PfxError) as e:
        fn()
    assert e.value.code == code, str(e.value)
    return str(e.value)


def raw_create(batch, pind=None, pids=None, plen=None, agent=None, sind=None, sids=None, slen=None, qind=None,
               hq=None, mode=B.PFX_MODE_MIXED, pool=None, **kw):
    a_pind, a_pids, a_plen = batch.prefix_csr()
    a_sind, a_sids = batch.suffix_csr()
    pool = pool or B.make_pool(batch.num_pages, batch.num_kv_heads, batch.head_dim)
    return B.pfx_plan_create(pool,
                             a_pind if pind is None else pind, a_pids if pids is None else pids,
                             a_plen if plen is None else plen, batch.agent if agent is None else agent,
                             a_sind if sind is None else sind, a_sids if sids is None else sids,
                             batch.suffix_len if slen is None else slen,
                             batch.q_indptr() if qind is None else qind,
                             batch.num_q_heads if hq is None else hq, mode, **kw)


def test_plan_validation_error_codes():
    b = small_batch()
    raw_create(b)  # valid
    pool = lambda **o: B.pfx_pool(o.get("n", 64), o.get("ps", 16), o.get("hkv", 2), o.get("d", 64), None, None)
    expect_error(B.PFX_EUNSUPPORTED, lambda: raw_create(b, pool=pool(ps=32)))
    expect_error(B.PFX_EUNSUPPORTED, lambda: raw_create(b, pool=pool(d=96)))
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, hq=7))                    # Hq % Hkv != 0
    expect_error(B.PFX_EUNSUPPORTED, lambda: raw_create(b, hq=6))              # G = 3
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, mode=7))
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, mode=B.PFX_MODE_DECODE))  # request with 33 rows
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, decode_workers=-1))
    # Eq. (2): pool of 10 pages cannot hold 3 + 2 prefix pages and 1+2+3+1+1 suffix pages
    msg = expect_error(B.PFX_ENOMEM, lambda: raw_create(b, pool=pool(n=12)))
    assert "13 pages" in msg
    sids = b.suffix_csr()[1].copy()
    sids[0] = 64
    expect_error(B.PFX_ERANGE, lambda: raw_create(b, sids=sids))               # page id out of range
    sids = b.suffix_csr()[1].copy()
    sids[1] = b.prefix_pages[0][0]
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, sids=sids))               # prefix page reused as suffix
    sids = b.suffix_csr()[1].copy()
    sids[2] = sids[1]
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, sids=sids))               # page owned twice
    expect_error(B.PFX_ERANGE, lambda: raw_create(b, agent=[0, 2, 0, -1, 1]))  # no agent 2
    expect_error(B.PFX_ERANGE, lambda: raw_create(b, agent=[0, 1, 0, -2, 1]))
    slen = b.suffix_len.copy(); slen[3] = 2
    expect_error(B.PFX_ERANGE, lambda: raw_create(b, slen=slen))               # 3 rows but L = 2
    slen = b.suffix_len.copy(); slen[0] = 40
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, slen=slen))               # page count != ceil(L/16)
    plen = np.array([40, 33], np.int32)
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, plen=plen))
    qind = b.q_indptr().copy(); qind[0] = 1
    expect_error(B.PFX_EINVAL, lambda: raw_create(b, qind=qind))
    plen = np.array([40, -1], np.int32)
    expect_error(B.PFX_ERANGE, lambda: raw_create(b, plen=plen))


def test_unreferenced_agent_pages_are_ignored():
    # Agent 1 has no request: its (possibly stale) pages are not validated or counted.
    b = small_batch(agent=[0, 0, 0, -1, 0])
    _, pids, _ = b.prefix_csr()
    pids = pids.copy()
    pids[-1] = 10_000
    p = raw_create(b, pids=pids)
    assert p.stats().pages_needed == 3 + (1 + 2 + 3 + 1 + 1)


def test_empty_batch_and_zero_row_requests():
    b = small_batch(agent=[], suffix_len=[], n_rows=[])
    p = plan_for(b)
    s = p.stats()
    assert (s.num_items, s.num_tokens, s.num_requests) == (0, 0, 0)
    b = small_batch(n_rows=[0, 0, 0, 0, 0])
    s = plan_for(b).stats()
    assert s.num_items == 0 and s.num_requests == 5


def enumerate_coverage(plan, batch):
    """Count, from the exported work lists, how often each (token, q head,
    logical key) triple is attended, and which output row each piece of a
    row writes: ('final', row) or ('part', slot, row)."""
    G, hkv, hq = batch.group, batch.num_kv_heads, batch.num_q_heads
    q_indptr = batch.q_indptr()
    tok_req = np.repeat(np.arange(len(batch.agent)), batch.n_rows)
    counts, outs = {}, {}

    def req_info(tok):
        r = int(tok_req[tok])
        a = int(batch.agent[r])
        plen = int(batch.prefix_len[a]) if a >= 0 else 0
        n, L = int(batch.n_rows[r]), int(batch.suffix_len[r])
        return r, a, plen, L - n + (tok - int(q_indptr[r]))

    def hit(tok, qh, k):
        counts[(tok, qh, k)] = counts.get((tok, qh, k), 0) + 1

    # Extend blocks: prefix then causal suffix, final rows.  Then the wide
    # prefix blocks: one piece of an agent's prefix against up to 128 of
    # its decode columns, partial rows.
    items, row_tok, page_list = plan.export(0), plan.export(1), plan.export(2)
    row_out = plan.export(8)
    mtok0, mhead0 = plan.export(6), plan.export(7).reshape(-1, hkv, 2)
    midx0 = {int(t): i for i, t in enumerate(mtok0)}
    n_ext = plan.stats().num_extend_items
    assert len(items) == n_ext + plan.stats().num_wide_blocks
    for it in items[n_ext:]:
        (h, rb, rc, nblk, s0p, s0b, s0e, s1p, s1b, s1e, cbase, slot, kind, req, tok0, _) = (int(x) for x in it[:16])
        assert kind == 0 and slot >= 0 and tok0 == -1 and s1e == s1b and s0b % 32 == 0
        assert 1 <= rc and rc * G <= 128 and nblk == (rc * G + 15) // 16
        first = [int(x) for x in it[16:32]]
        lead = [int(page_list[s0p + k]) for k in range(s0b // 16, (s0e + 15) // 16)]
        assert first[:min(16, len(lead))] == lead[:16]
        for j in range(rc):
            tok = int(row_tok[rb + j])
            r, a, plen, pos = req_info(tok)
            assert s0e <= plen
            for g in range(G):
                qh = h * G + g
                for k in range(s0b, s0e):
                    assert int(page_list[s0p + k // 16]) == int(batch.prefix_pages[a][k // 16])
                    hit(tok, qh, k)
                base, np_ = mhead0[midx0[tok], h]
                row = int(row_out[rb + j]) + g
                assert 0 <= slot < np_ and row == (base + slot) * G + g
                outs.setdefault((tok, qh), []).append(("part", slot, row))
    for it in items[:n_ext]:
        (h, rb, rc, nblk, s0p, s0b, s0e, s1p, s1b, s1e, cbase, slot, kind, req, tok0, _) = it[:16]
        assert kind == 2 and slot == -1 and int(row_out[rb]) == -1
        first = [int(x) for x in it[16:32]]
        lead = [int(page_list[s0p + k]) for k in range(s0b // 16, (s0e + 15) // 16)] if s0e > s0b else []
        lead += [int(page_list[s1p + k]) for k in range(s1b // 16, (s1e + 15) // 16)] if s1e > s1b else []
        assert first[:min(16, len(lead))] == lead[:16]
        assert tok0 == int(row_tok[rb])
        assert 1 <= nblk <= 8 and rc * G <= nblk * 16 and (rc * G > (nblk - 1) * 16)
        for j in range(rc):
            tok = int(row_tok[rb + j])
            assert tok == tok0 + j
            r, a, plen, pos = req_info(tok)
            for g in range(G):
                qh = h * G + g
                for k in range(s0b, s0e):
                    assert int(page_list[s0p + k // 16]) == int(batch.prefix_pages[a][k // 16])
                    hit(tok, qh, k)
                for k in range(s1b, s1e):
                    assert int(page_list[s1p + k // 16]) == int(batch.suffix_pages[r][k // 16])
                    if k <= tok + cbase:
                        assert tok + cbase == pos
                        hit(tok, qh, plen + k)
                outs.setdefault((tok, qh), []).append(("final", tok * hq + qh))

    # Decode: items cut into pieces of at most 64 steps, longest first.
    segs = plan.export(3)
    mtok, mhead = plan.export(6), plan.export(7).reshape(-1, hkv, 2)
    midx = {int(t): i for i, t in enumerate(mtok)}
    pieces = {}
    costs = []
    for sg in segs:
        kind, h, ncols, nst, k0, kend, cbase, slot, item, piece, causal = (int(x) for x in sg[:11])
        assert kind in (0, 1) and 1 <= ncols <= 64 and ncols % G == 0 and k0 % 32 == 0 and 1 <= nst <= 64
        costs.append((11 if kind == 0 else 10) * nst + 10)
        pieces.setdefault(item, []).append((piece, k0, nst, kend))
        tok0 = int(sg[16])
        r0 = int(tok_req[tok0])
        assert causal == (kind == 1 and int(batch.n_rows[r0]) > 1)
        for j in range(ncols // G):
            tok = int(sg[16 + j])
            r, a, plen, pos = req_info(tok)
            src = batch.prefix_pages[a] if kind == 0 else batch.suffix_pages[r]
            for i in range(nst):
                kk = k0 + 32 * i
                assert kk < kend
                blk0, blk1 = int(sg[144 + 2 * i]), int(sg[145 + 2 * i])
                assert blk0 == int(src[kk // 16]) * hkv + h
                assert blk1 == (int(src[kk // 16 + 1]) if kk + 16 < kend else int(src[kk // 16])) * hkv + h
                for g in range(G):
                    for k in range(kk, min(kk + 32, kend)):
                        if kind == 0:
                            hit(tok, h * G + g, k)
                        elif k <= tok + cbase:
                            assert tok + cbase == pos
                            hit(tok, h * G + g, plen + k)
            for g in range(G):
                row = int(sg[80 + j]) + g
                if slot < 0:
                    assert row == tok * hq + h * G + g
                    outs.setdefault((tok, h * G + g), []).append(("final", row))
                else:
                    base, np_ = mhead[midx[tok], h]
                    assert 0 <= slot < np_ and row == (base + slot) * G + g
                    outs.setdefault((tok, h * G + g), []).append(("part", slot, row))
    assert costs == sorted(costs, reverse=True)  # longest first
    # Each item's pieces tile its key range in order, as evenly as possible.
    for item, ps in pieces.items():
        ps.sort()
        assert [q[0] for q in ps] == list(range(len(ps)))
        ends = [(k0, k0 + 32 * n) for (_, k0, n, _) in ps]
        assert ends[0][0] == 0 and all(ends[i][1] == ends[i + 1][0] for i in range(len(ends) - 1))
        assert ends[-1][1] >= ps[0][3] > ends[-1][1] - 32
        sizes = [n for (_, _, n, _) in ps]
        assert max(sizes) - min(sizes) <= 1
    return counts, outs


@pytest.mark.parametrize("case", ["small", "split", "g1", "g2", "g16", "decode_only", "wide", "wide-valu"])
def test_plan_covers_every_visible_key_once(case):
    if case in ("wide", "wide-valu"):
        # agents with 70, 200 and 24 decode columns per KV head (G = 2): wide blocks for the first two
        reqs = [(0, 5 + i, 1) for i in range(35)] + [(1, 3 + i % 50, 1) for i in range(96)] + \
               [(1, 20, 2), (2, 9, 3)] + [(2, 4 + i, 1) for i in range(9)] + [(0, 300, 300), (-1, 30, 1)]
        b = W.make_batch(9, num_q_heads=16, num_kv_heads=8, head_dim=64, num_pages=4096, prefix_len=[400, 1000, 90],
                         agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
        kw = dict(piece_steps=5)
        if case == "wide-valu":
            kw["decode_engine"] = B.PFX_DECODE_VALU  # the same agents in 64-column pieces, no wide blocks
    elif case == "g2":
        reqs = [(0, 140, 140), (0, 19, 3), (0, 5, 1), (0, 44, 8), (-1, 9, 9)] + [(1, 3 + i, 1) for i in range(40)]
        b = W.make_batch(8, num_q_heads=16, num_kv_heads=8, head_dim=64, num_pages=256, prefix_len=[70, 33],
                         agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
        kw = dict(piece_steps=1)
    elif case == "small":
        b, kw = small_batch(), {}
    elif case == "split":
        b, kw = small_batch(prefix_len=[100, 17], suffix_len=[70, 20, 33, 3, 40]), dict(decode_workers=7)
    elif case == "g1":
        b, kw = small_batch(num_q_heads=2), {}
    elif case == "g16":
        b, kw = small_batch(num_q_heads=32, n_rows=[1, 1, 33, 1, 1]), dict(decode_workers=5)
    else:
        agents = np.arange(70) % 3 - 1
        b = W.make_batch(5, num_q_heads=8, num_kv_heads=2, head_dim=128, num_pages=512, prefix_len=[64, 300],
                         agent=agents, suffix_len=(np.arange(70) % 40) + 1, n_rows=np.ones(70, np.int32))
        kw = dict(decode_workers=64)
    p = plan_for(b, **kw)
    if case.startswith("wide"):
        assert (p.stats().num_wide_blocks > 0) == (case == "wide")
    counts, outs = enumerate_coverage(p, b)
    q_indptr = b.q_indptr()
    expected = 0
    for r in range(len(b.agent)):
        a = int(b.agent[r])
        plen = int(b.prefix_len[a]) if a >= 0 else 0
        n, L = int(b.n_rows[r]), int(b.suffix_len[r])
        for i in range(n):
            tok = int(q_indptr[r]) + i
            vis = plen + L - n + i + 1
            for qh in range(b.num_q_heads):
                for k in range(vis):
                    assert counts.get((tok, qh, k), 0) == 1, (tok, qh, k)
                expected += vis
    assert sum(counts.values()) == expected            # nothing invisible is attended
    # A row is written either once, final (extend), or as partial slots
    # 0 .. k-1 (decode, k >= 1), each once, merged afterwards; no two rows
    # share a partial row.
    part_rows = []
    mtok = set(int(t) for t in p.export(6))
    for (tok, qh), ws in outs.items():
        if ws[0][0] == "final":
            assert len(ws) == 1, (tok, qh, ws)
        else:
            slots = sorted(w[1] for w in ws)
            assert all(w[0] == "part" for w in ws) and slots == list(range(len(ws)))
            assert tok in mtok
            part_rows += [w[2] for w in ws]
    assert len(part_rows) == len(set(part_rows)) == p.stats().num_partial_rows
    s = p.stats()
    segs = p.export(3)
    wide = p.export(0)[s.num_extend_items:]
    wide_steps = int(sum((int(w[6]) - int(w[5]) + 31) // 32 for w in wide))
    assert s.num_decode_pieces == len(segs) and s.num_decode_steps == int(segs[:, 3].sum()) + wide_steps


def test_plan_is_deterministic_and_placement_independent():
    b = W.config_batch(2)
    p1, p2 = plan_for(b), plan_for(b)
    np.testing.assert_array_equal(p1.export(0), p2.export(0))
    # Same lengths, different page placement: same work list apart from page ids.
    b2 = W.make_batch(777, num_q_heads=b.num_q_heads, num_kv_heads=b.num_kv_heads, head_dim=b.head_dim,
                      num_pages=b.num_pages, prefix_len=b.prefix_len, agent=b.agent, suffix_len=b.suffix_len,
                      n_rows=b.n_rows)
    p3 = plan_for(b2)
    # Pieces and merge lists do not depend on placement, apart from the
    # page blocks of the steps.
    np.testing.assert_array_equal(p1.export(3)[:, :144], p3.export(3)[:, :144])
    for which in (6, 7):
        np.testing.assert_array_equal(p1.export(which), p3.export(which))
    assert not np.array_equal(p1.export(3)[:, 144:], p3.export(3)[:, 144:])
    np.testing.assert_array_equal(p1.export(1), p3.export(1))
    assert not np.array_equal(p1.export(2), p3.export(2))


def test_config_plans_build_and_group_prefixes():
    for cfg in (1, 2, 3, 4, 5):
        b = W.config_batch(cfg)
        s = plan_for(b).stats()
        assert s.num_tokens == b.num_tokens
        assert s.pages_needed <= b.num_pages
        if cfg == 2:
            # 4 agents x 8 KV heads, one 64-column row block each; 64 requests x 8 KV heads
            assert s.num_prefix_items == 4 * 8
            assert s.num_suffix_items == 64 * 8
            assert s.num_extend_items == 0
            steps = 4 * 8 * 2048 // 32 + 8 * sum((int(L) + 31) // 32 for L in b.suffix_len)
            assert s.num_decode_steps == steps
            # prefix items: 64 steps in 4 pieces; suffix items: one piece each (<= 16 steps)
            assert s.num_decode_pieces == 4 * 8 * 4 + 64 * 8
        if cfg == 3:
            assert s.num_prefix_items == 0 and s.num_suffix_items == 0
            assert s.num_extend_items == sum((int(n) + 31) // 32 for n in b.n_rows) * 8


def test_prefix_chunk_blocks_are_dealt_to_one_xcd():
    """The column blocks of one prefix chunk (same KV head and steps, other
    decode rows) sit a multiple of eight apart: decode pieces within one
    dealing round of 512 persistent workgroups (run on workgroups of one XCD
    residue, b mod 8), wide prefix blocks in their list (block i runs on
    workgroup i of the launch).  Configs 4 and 5 go wide for every agent
    with more than one 64-column block."""
    S = 512
    b = W.make_batch(5, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536, prefix_len=[3000, 2500],
                     agent=np.arange(140) % 2, suffix_len=30 + np.arange(140), n_rows=np.ones(140, np.int32))
    for batch in (W.config_batch(4), W.config_batch(5), b):
        p = plan_for(batch)
        segs = p.export(3)
        pos = {}
        for q, sg in enumerate(segs):
            if sg[0] == 0:                    # prefix piece; sg[144]: page block of its first step
                pos.setdefault(int(sg[144]), []).append(q)
        multi = [ps for ps in pos.values() if len(ps) > 1]

        def wg(q):
            n, x = divmod(q, S)
            return x if n % 2 == 0 else S - 1 - x

        assert all(len({q // S for q in ps}) == 1 and len({wg(q) % 8 for q in ps}) == 1 for ps in multi)
        wide = p.export(0)[p.stats().num_extend_items:]
        wpos = {}
        for q, w in enumerate(wide):
            wpos.setdefault((int(w[0]), int(w[16])), []).append(q)   # (KV head, first page of the piece)
        wmulti = [ps for ps in wpos.values() if len(ps) > 1]
        assert all(len({q % 8 for q in ps}) == 1 for ps in wmulti)
        assert multi or wmulti
        if batch is not b:
            assert not multi and wmulti           # every multi-block agent went wide


def test_upload_rejects_small_workspace_without_gpu_work():
    b = small_batch()
    p = plan_for(b)
    need = p.workspace_bytes()
    rc = B.LIB.pfx_plan_upload(p.h, C.c_void_p(256), need - 1, None)
    assert rc == B.PFX_ENOMEM
    rc = B.LIB.pfx_plan_upload(p.h, C.c_void_p(100), need, None)
    assert rc == B.PFX_EINVAL


def test_device_calls_validate_before_launch():
    b = small_batch()
    pool = B.make_pool(b.num_pages, b.num_kv_heads, b.head_dim)
    p = plan_for(b, pool=pool)
    # not uploaded yet -> EINVAL, nothing launched
    rc = B.LIB.pfx_attention(C.byref(pool), p.h, None, None, None, C.c_float(0), None)
    assert rc == B.PFX_EINVAL
    other = B.pfx_pool(b.num_pages, 16, b.num_kv_heads, 128, 1, 1)
    assert B.LIB.pfx_append_kv(C.byref(other), p.h, None, None, None) == B.PFX_EINVAL
    assert "shape" in B.pfx_last_error()
    assert B.LIB.pfx_merge_states(None, None, 1, 1, 128, None, None, None) == B.PFX_EINVAL
    assert B.LIB.pfx_merge_states(C.c_void_p(8), C.c_void_p(8), 0, 1, 128, C.c_void_p(8), None, None) == B.PFX_ERANGE
    src = B.pfx_pool(4, 16, 2, 64, 8, 8)
    dst = B.pfx_pool(6, 16, 2, 64, 8, 8)
    ids = (C.c_int32 * 2)(0, 6)
    srcs = (C.c_int32 * 2)(0, 1)
    ws = C.c_void_p(256)
    assert B.LIB.pfx_page_copy(C.byref(dst), C.byref(src), ids, srcs, 2, ws, 4096, None) == B.PFX_ERANGE
    ids = (C.c_int32 * 2)(3, 3)
    assert B.LIB.pfx_page_copy(C.byref(dst), C.byref(src), ids, srcs, 2, ws, 4096, None) == B.PFX_EINVAL
    ids = (C.c_int32 * 2)(3, 4)
    assert B.LIB.pfx_page_copy(C.byref(dst), C.byref(src), ids, srcs, 2, ws, 16, None) == B.PFX_ENOMEM
    bad = B.pfx_pool(6, 16, 2, 128, 8, 8)
    assert B.LIB.pfx_page_copy(C.byref(bad), C.byref(src), ids, srcs, 2, ws, 4096, None) == B.PFX_EINVAL
    # valid ids and workspace, page pointers HIP does not know: refused before any launch
    assert B.LIB.pfx_page_copy(C.byref(dst), C.byref(src), ids, srcs, 2, ws, 4096, None) == B.PFX_EINVAL
    assert "neither device nor pinned host" in B.pfx_last_error()


def plan_tables(p):
    return [p.export(w).copy() for w in (0, 1, 2, 3, 6, 7)] + [p.workspace_bytes()]


def same_tables(x, y):
    return all(np.array_equal(a, b) for a, b in zip(x, y))


def test_plan_host_image_reuse_never_touches_a_live_plan():
    # A destroyed plan's host image is handed to the next plan built on the
    # thread.  A live plan keeps its own: its tables stay as built while
    # other plans of other sizes come and go, and a plan rebuilt from the
    # same inputs is identical.
    import gc
    big, small = W.config_batch(2), small_batch()
    pool_big = B.make_pool(big.num_pages, big.num_kv_heads, big.head_dim)
    a = B.plan_from_batch(pool_big, big, B.PFX_MODE_MIXED)
    want = plan_tables(a)
    for k in range(4):
        b = plan_for(small) if k % 2 else B.plan_from_batch(pool_big, big, B.PFX_MODE_DECODE, piece_steps=5 + k)
        del b
        gc.collect()
        c = plan_for(small, mode=B.PFX_MODE_EXTEND)
        assert same_tables(plan_tables(a), want)
        del c
        gc.collect()
    again = B.plan_from_batch(pool_big, big, B.PFX_MODE_MIXED)
    assert same_tables(plan_tables(again), want)
    del a
    gc.collect()
    assert same_tables(plan_tables(again), want)


def test_default_piece_length_follows_the_launch_size():
    # 16 steps below 32768 decode steps, 64 from there; an explicit
    # piece_steps wins.
    for cfg, want in ((2, 16), (4, 64), (5, 64)):
        b = W.config_batch(cfg)
        p = plan_for(b)
        segs = p.export(3)
        steps = p.stats().num_decode_steps
        assert want // 2 < int(segs[:, 3].max()) <= want, (cfg, steps)   # items are cut evenly
        assert (steps >= 32768) == (want == 64)
    p = plan_for(W.config_batch(5), piece_steps=16)
    assert int(p.export(3)[:, 3].max()) == 16
    with pytest.raises(B.PfxError):
        plan_for(W.config_batch(2), piece_steps=65)


def test_decode_engine_option():
    b = W.config_batch(4)       # agents with more than 64 decode columns per KV head
    assert plan_for(b).stats().num_wide_blocks > 0
    pv = plan_for(b, decode_engine=B.PFX_DECODE_VALU)
    assert pv.stats().num_wide_blocks == 0
    for bad in (2, -1):
        msg = expect_error(B.PFX_EINVAL, lambda: plan_for(b, decode_engine=bad))
        assert "decode_engine" in msg



def test_extend_blocks_take_any_key_count():
    """An extend request over a 24,576-token prefix and a 17,000-token suffix
    (2,600 pages, far more than a block could hold in a fixed table) plans:
    only head_dim, page size and the query group are unsupported."""
    b = W.make_batch(24, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=4096, prefix_len=[24576],
                     agent=[0, -1], suffix_len=[300, 17000], n_rows=[300, 64])
    s = plan_for(b, mode=B.PFX_MODE_EXTEND).stats()
    assert s.num_extend_items == 8 * (10 + 2) and s.num_tokens == 364   # 32 rows x 4 heads per block
    blocks = plan_for(b, mode=B.PFX_MODE_EXTEND).export(0)
    assert blocks[:, 6].max() == 24576                   # s0_kend: the whole prefix in one block's first segment


class _FakeBuffer:
    """Stands in for a device tensor: a nonzero address that no call here
    ever dereferences (every case below fails validation first)."""

    def __init__(self, addr):
        self.addr = addr

    def data_ptr(self):
        return self.addr


def test_noalloc_validates_before_touching_the_device():
    b = small_batch()
    fake = [_FakeBuffer(0x10000 * (i + 1)) for i in range(6)]
    pool = B.make_pool(b.num_pages, b.num_kv_heads, b.head_dim, fake[0], fake[1])
    plan = plan_for(b, pool)
    # only one of k_new / v_new
    expect_error(B.PFX_EINVAL, lambda: B.pfx_attention_noalloc(pool, plan, fake[2], fake[3], k_new=fake[4], stream=0))
    # no q / o
    expect_error(B.PFX_EINVAL, lambda: B.pfx_attention_noalloc(pool, plan, None, fake[3], stream=0))
    # a pool of another shape
    other = B.make_pool(b.num_pages + 1, b.num_kv_heads, b.head_dim, fake[0], fake[1])
    expect_error(B.PFX_EINVAL, lambda: B.pfx_attention_noalloc(other, plan, fake[2], fake[3], stream=0))
    # a plan whose workspace exceeds the static array (checked before any HIP call)
    big = W.make_batch(14, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536, prefix_len=[30000],
                       agent=[0] * 120, suffix_len=[40] * 120, n_rows=[1] * 120)
    bpool = B.make_pool(big.num_pages, 8, 128, fake[0], fake[1])
    bplan = plan_for(big, bpool, B.PFX_MODE_DECODE, piece_steps=1)
    assert bplan.workspace_bytes() > B.PFX_NOALLOC_MAX_WORKSPACE
    expect_error(B.PFX_ENOMEM, lambda: B.pfx_attention_noalloc(bpool, bplan, fake[2], fake[3], fake[5],
                                                                 k_new=fake[4], v_new=fake[4], stream=0))
    assert "static scratch" in B.pfx_last_error()


def test_prefix_chunk_blocks_share_an_xcd():
    """Column blocks of one prefix chunk (same KV head and first page block)
    sit a multiple of eight positions apart in the launch order (decode
    pieces, and wide prefix blocks within their list), so they run on one
    XCD and read the chunk through its L2; only blocks beyond the shortest
    chunk of their group of eight may break the pattern."""
    n = [150, 70, 300]        # 4 KV heads, 3 pieces per prefix: groups of eight mix agents
    mixed = W.make_batch(3, num_q_heads=32, num_kv_heads=4, head_dim=128, num_pages=20000, prefix_len=[1536] * 3,
                         agent=np.concatenate([np.full(k, a) for a, k in enumerate(n)]),
                         suffix_len=np.full(sum(n), 40), n_rows=np.ones(sum(n), np.int32))
    for b, allowed in ((W.config_batch(5), 0.0), (W.config_batch(4), 0.0), (mixed, 0.11)):
        p = plan_for(b)
        off = total = 0
        for rows, kind_col, key_cols in ((p.export(3), 0, (1, 144, 3)),
                                         (p.export(0)[p.stats().num_extend_items:], 12, (0, 16, 5))):
            first = {}
            for pos, row in enumerate(rows):
                if row[kind_col] != 0:           # prefix pieces / wide prefix blocks only
                    continue
                key = tuple(int(row[c]) for c in key_cols)
                if key in first:
                    total += 1
                    off += (pos - first[key]) % 8 != 0
                else:
                    first[key] = pos
        assert total > 0 and off <= allowed * total, (off, total)
