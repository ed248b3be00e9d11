"""GPU parity: the HIP path through the C interface against the fp64 oracle.

Every test here needs an MI355X and the built library; the binding fails
loudly without it.  Each test prints the case it is about to run.
"""

from __future__ import annotations

import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2608_25523_amd import binding as B  # noqa: E402
from paper_2608_25523_amd import runner as RN  # noqa: E402
from paper_2608_25523_amd import workloads as W  # noqa: E402
import parity as PT  # noqa: E402

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    yield
    torch.cuda.synchronize()


def assert_untouched(ds, used_pages, label, chunk=8192):
    """Every pool page outside ``used_pages`` still holds the poison pattern
    it was filled with (no stray append, gather or attention write); checked
    on the device, chunk by chunk."""
    import torch as T

    used = T.zeros(ds.batch.num_pages, dtype=T.bool, device=ds.k_pool.device)
    used[T.from_numpy(np.asarray(used_pages, np.int64)).to(ds.k_pool.device)] = True
    for pool, name in ((ds.k_pool, "K"), (ds.v_pool, "V")):
        bits = pool.view(T.int16)
        for s in range(0, ds.batch.num_pages, chunk):
            e = min(ds.batch.num_pages, s + chunk)
            off = bits[s:e].reshape(e - s, -1).ne(W.POISON_BF16).any(dim=1) & ~used[s:e]
            assert not bool(off.any()), f"{label}: {name} pool page {s + int(off.nonzero()[0, 0])} was written"


def run_and_check(batch, hv, label, rows=None, host_resident=(), check_pages=True, parallel=False, sm_scale=0.0,
                  with_lse=True, **kw):
    announce(f"{label}: tokens={batch.num_tokens} reqs={len(batch.agent)} Hq={batch.num_q_heads} "
             f"Hkv={batch.num_kv_heads} d={batch.head_dim} pool={batch.num_pages} sm_scale={sm_scale} "
             f"lse={'yes' if with_lse else 'NULL'} {kw}")
    ds = RN.DeviceStep(batch, hv, host_resident=host_resident, **kw)
    ds.gather_evicted()
    ds.append()
    if with_lse:
        ds.attention(sm_scale)
    else:
        ds.lse.fill_(float("nan"))
        B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, None, sm_scale)
    B.pfx_sync_check()
    o_bits, lse = ds.outputs()
    if not with_lse:
        assert np.isnan(lse).all(), f"{label}: LSE written although none was passed"
        lse = None
    exp_k, exp_v = PT.expected_pools(batch, hv)
    if check_pages:
        gk, gv = ds.read_pages(hv.pages)
        assert np.array_equal(gk, exp_k), f"{label}: K pool differs from the oracle's append"
        assert np.array_equal(gv, exp_v), f"{label}: V pool differs from the oracle's append"
        if kw.get("poison", True):
            assert_untouched(ds, hv.pages, label)
    scale = sm_scale if sm_scale > 0 else None
    if parallel:
        want = rows if rows is not None else PT.all_rows(batch)
        ck = PT.checker()
        h = ck.submit(batch, hv.pages, exp_k, exp_v, PT.gather_rows(hv.q, batch, want),
                      PT.gather_rows(o_bits, batch, want), None if lse is None else PT.gather_rows(lse, batch, want),
                      want, scale=scale)
        res = ck.collect(h, label)
        announce(f"{label}: rows={res[3]} max_abs={res[0]:.2e} rel={res[1]:.2e} lse={res[2]:.2e}")
        return ds, o_bits, lse
    o_ref, l_ref = PT.reference(batch, hv, (exp_k, exp_v), rows=rows, scale=scale)
    res = PT.compare(batch, o_bits, lse, o_ref, l_ref, label)
    announce(f"{label}: max_abs={res[0]:.2e} rel={res[1]:.2e} lse={res[2]:.2e}")
    return ds, o_bits, lse


# --------------------------------------------------------------------------- merge and copy

@pytest.mark.parametrize("d,parts,rows", [(128, 1, 7), (128, 3, 50), (64, 37, 33), (128, 200, 5)])
def test_merge_states_matches_oracle(d, parts, rows):
    announce(f"merge d={d} parts={parts} rows={rows}")
    rng = np.random.default_rng(parts * 100 + rows)
    o_parts = rng.standard_normal((parts, rows, d)).astype(np.float32)
    lse_parts = (rng.standard_normal((parts, rows)) * 4).astype(np.float32)
    lse_parts[0, 0] = -np.inf if parts > 1 else lse_parts[0, 0]      # a part that saw no keys
    o_parts[0, 0] = 0.0 if parts > 1 else o_parts[0, 0]
    o = torch.empty((rows, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((rows,), dtype=torch.float32, device="cuda")
    B.pfx_merge_states(torch.from_numpy(o_parts).cuda(), torch.from_numpy(lse_parts).cuda(), o, lse)
    B.pfx_sync_check()
    ro, rl = oracle.merge_partials([p.astype(np.float64) for p in o_parts], [l.astype(np.float64) for l in lse_parts])
    got = oracle.bf16_bits_to_f64(RN.to_host_bits(o))
    assert np.max(np.abs(got - ro)) <= 2 ** -8 * np.max(np.abs(ro)) + 1e-6
    assert np.max(np.abs(lse.cpu().numpy() - rl)) <= 1e-5 * (1 + np.max(np.abs(rl)))


def test_page_copy_bit_exact_all_directions():
    announce("page copy: device->device, host->device, device->host")
    rng = np.random.default_rng(5)
    hkv, d = 8, 128
    src = rng.integers(0, 65535, size=(40, hkv, 16, d), dtype=np.uint16)
    dst0 = rng.integers(0, 65535, size=(100, hkv, 16, d), dtype=np.uint16)
    dst_pages = rng.permutation(100)[:25].astype(np.int32)
    src_pages = rng.integers(0, 40, size=25).astype(np.int32)
    want = oracle.page_copy(dst0, src, dst_pages, src_pages)
    ws = torch.empty(B.pfx_page_copy_workspace_bytes(25) + 256, dtype=torch.uint8, device="cuda")
    d_src = RN.to_device_bits(src)
    d_dst = RN.to_device_bits(dst0)
    # device -> device (K and V given the same arrays for simplicity, then distinct)
    h_v = torch.from_numpy(src[::-1].copy().view(np.int16)).view(torch.bfloat16).pin_memory()
    d_dst_v = RN.to_device_bits(dst0)
    B.pfx_page_copy(B.make_pool(100, hkv, d, d_dst, d_dst_v), B.make_pool(40, hkv, d, d_src, h_v),
                    dst_pages, src_pages, ws)
    B.pfx_sync_check()
    assert np.array_equal(RN.to_host_bits(d_dst), want)
    want_v = oracle.page_copy(dst0, src[::-1].copy(), dst_pages, src_pages)
    assert np.array_equal(RN.to_host_bits(d_dst_v), want_v)
    # device -> pinned host (eviction)
    h_dst = torch.from_numpy(dst0.view(np.int16).copy()).view(torch.bfloat16).pin_memory()
    h_dst_v = torch.from_numpy(dst0.view(np.int16).copy()).view(torch.bfloat16).pin_memory()
    B.pfx_page_copy(B.make_pool(100, hkv, d, h_dst, h_dst_v), B.make_pool(40, hkv, d, d_src, d_src),
                    dst_pages, src_pages, ws)
    B.pfx_sync_check()
    assert np.array_equal(h_dst.view(torch.int16).numpy().view(np.uint16), want)
    assert np.array_equal(h_dst_v.view(torch.int16).numpy().view(np.uint16), want)


# --------------------------------------------------------------------------- small batches

SMALL_CASES = [
    # (seed, Hq, Hkv, d, prefix_len, reqs [(agent, L, n)], opts)
    (1, 8, 2, 64, [40, 17], [(0, 5, 1), (1, 20, 1), (0, 33, 33), (-1, 3, 3), (1, 16, 2)], {}),
    (2, 32, 8, 128, [100, 0, 37], [(0, 70, 1), (2, 1, 1), (1, 40, 40), (0, 65, 1), (2, 17, 4), (-1, 31, 1)],
     dict(decode_workers=17)),
    (3, 16, 16, 128, [64], [(0, 90, 90), (0, 1, 1), (0, 48, 1)], {}),                 # G = 1
    (4, 16, 1, 64, [300], [(0, 9, 1), (0, 200, 1), (0, 40, 40), (-1, 5, 1)], dict(decode_workers=3)),  # G = 16
    (5, 64, 8, 128, [129, 500], [(i % 2, 10 + 7 * i, 1) for i in range(20)] + [(1, 77, 2)], dict(decode_workers=100)),
    (6, 32, 8, 128, [16], [(0, 1, 0), (0, 33, 1), (-1, 64, 64)], {}),                 # a request with no rows
    # two workers asked for; the 16-segment limit of a worker adds more
    (7, 32, 8, 128, [50], [(0, 1 + i % 20, 1) for i in range(40)] + [(-1, 7, 4)], dict(decode_workers=2)),
    # G = 2: 64-row extend blocks, 32-row prefix blocks (agent 1 has 40 decode rows: two blocks), multi-row
    # causal decode requests (n * G <= 16), a request with no prefix
    (8, 16, 8, 64, [70, 33], [(0, 140, 140), (0, 19, 3), (0, 5, 1), (0, 44, 8), (-1, 9, 9)]
     + [(1, 3 + i, 1) for i in range(40)], {}),
    (9, 16, 8, 128, [70, 33], [(0, 140, 140), (0, 19, 3), (0, 5, 1), (0, 44, 8), (-1, 9, 9)]
     + [(1, 3 + i, 1) for i in range(40)], dict(piece_steps=1)),
    # G = 16, one KV head: agent 0's 9 decode rows are 144 columns (two wide blocks) over 5 one-step
    # prefix pieces, 10 wide blocks beside 19 decode pieces.  The launch interleaves one round of
    # 8 wide blocks and 8 pieces, then runs the other 11 pieces, then the 2 wide blocks left over.
    (10, 16, 1, 128, [160, 40], [(0, 10 + 7 * i, 1) for i in range(9)] + [(1, 30, 1), (0, 50, 50), (-1, 9, 1)],
     dict(piece_steps=1)),
]


@pytest.mark.parametrize("case", SMALL_CASES, ids=[f"small{c[0]}" for c in SMALL_CASES])
def test_small_batches(case):
    seed, hq, hkv, d, plen, reqs, opts = case
    b = W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=256, prefix_len=plen,
                     agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
    hv = W.host_values(b, seed + 50)
    run_and_check(b, hv, f"small{seed}", **opts)


@pytest.mark.parametrize("case", SMALL_CASES, ids=[f"valu-small{c[0]}" for c in SMALL_CASES])
def test_small_batches_valu_engine(case):
    """The decode pieces on the vector ALU (dot products instead of MFMA
    tiles, no wide blocks) against the same oracle."""
    seed, hq, hkv, d, plen, reqs, opts = case
    b = W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=256, prefix_len=plen,
                     agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
    hv = W.host_values(b, seed + 50)
    ds, _, _ = run_and_check(b, hv, f"valu-small{seed}", decode_engine=B.PFX_DECODE_VALU, **opts)
    assert ds.plan.stats().num_wide_blocks == 0


def random_case(seed):
    """A seeded random small batch: any group size, head dim 64 or 128, zero
    to three agents, decode rows (one or a few per request), extend
    requests and requests without a prefix, with short pieces or few
    workers so that rows merge many parts."""
    rng = np.random.Generator(np.random.PCG64(9000 + seed))
    hq, hkv = [(8, 8), (16, 8), (16, 4), (32, 4), (16, 1), (32, 8)][int(rng.integers(0, 6))]
    g = hq // hkv
    d = int(rng.choice([64, 128]))
    plen = [int(x) for x in rng.integers(0, 400, size=int(rng.integers(1, 4)))]
    reqs = []
    for _ in range(int(rng.integers(3, 13))):
        agent = int(rng.integers(-1, len(plen)))
        L = int(rng.integers(1, 300))
        kind = rng.random()
        n = 1 if kind < 0.5 else (min(L, max(1, 16 // g)) if kind < 0.75 else L)
        reqs.append((agent, L, n))
    opts = [{}, dict(piece_steps=1), dict(piece_steps=2), dict(piece_steps=5), dict(decode_workers=3)][int(rng.integers(0, 5))]
    return (seed, hq, hkv, d, plen, reqs, opts)


RANDOM_CASES = [random_case(i) for i in range(12)]


@pytest.mark.parametrize("case", RANDOM_CASES, ids=[f"random{c[0]}" for c in RANDOM_CASES])
def test_random_small_batches(case):
    """Seeded random shapes (group size, head dim, prefixes, decode and extend
    rows, piece lengths): every row against the oracle."""
    b, opts = small_batch(case)
    hv = W.host_values(b, 7000 + case[0])
    run_and_check(b, hv, f"random{case[0]} Hq={case[1]} Hkv={case[2]} d={case[3]} prefixes={case[4]}", **opts)


def small_batch(case):
    seed, hq, hkv, d, plen, reqs, opts = case
    need = sum((p + 15) // 16 for p in plen) + sum((r[1] + 15) // 16 for r in reqs)
    b = W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=max(256, 2 * need), prefix_len=plen,
                     agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
    return b, opts


@pytest.mark.parametrize("sm_scale,with_lse", [(0.125, True), (0.02, False), (1.0 / math.sqrt(128), False)])
def test_explicit_scale_and_no_lse(sm_scale, with_lse):
    """sm_scale > 0 overrides 1/sqrt(d); a NULL lse pointer leaves the LSE
    untouched while O is still written (extend, multi-row decode and shared
    prefix decode rows)."""
    b, opts = small_batch(SMALL_CASES[1])
    hv = W.host_values(b, 60)
    run_and_check(b, hv, f"scale{sm_scale:.4f}-lse{int(with_lse)}", sm_scale=sm_scale, with_lse=with_lse, **opts)


# Peaked scores: the lazy rescale of the running maximum (raised only past a
# slack) must take its non-trivial branch, with 0 < alpha < 1, mid-block and
# mid-piece.
PEAKED = [
    # (seed, Hq, Hkv, d, prefix_len, reqs, opts)
    (21, 32, 8, 128, [2048, 700], [(0, 300, 300), (1, 90, 90), (0, 200, 1), (1, 40, 1), (0, 37, 3)]
     + [(i % 2, 30 + 11 * i, 1) for i in range(24)], dict(piece_steps=8)),
    (22, 16, 8, 64, [1500], [(0, 257, 257), (0, 33, 1), (-1, 400, 400), (0, 120, 4)]
     + [(0, 20 + 3 * i, 1) for i in range(30)], dict(piece_steps=3)),
]


@pytest.mark.parametrize("case", PEAKED, ids=[f"one-hot{c[0]}" for c in PEAKED])
def test_peaked_one_hot(case):
    """q = 16 k[j*] for a seeded visible key j* per row and head: one score
    stands ~100 nats above the rest, and the output is v[j*]."""
    seed, hq, hkv, d, plen, reqs, opts = case
    b, _ = small_batch((seed, hq, hkv, d, plen, reqs, opts))
    hv = W.plant_one_hot(b, W.host_values(b, seed + 1), seed + 2, alpha_log2=4)
    run_and_check(b, hv, f"one-hot{seed}", **opts)


@pytest.mark.parametrize("case", PEAKED, ids=[f"rising{c[0]}" for c in PEAKED])
def test_peaked_rising_scores(case):
    """Key norms growing along the sequence (gain 1 + p/256 at absolute
    position p) and queries x4: the largest score rises step after step, so
    the running maximum is raised again and again within blocks and pieces."""
    seed, hq, hkv, d, plen, reqs, opts = case
    b, _ = small_batch((seed, hq, hkv, d, plen, reqs, opts))
    hv = W.host_values_shaped(b, seed + 3, key_gain=lambda p: 1.0 + p / 256.0, q_gain=4.0, v_gain=0.25)
    run_and_check(b, hv, f"rising{seed}", **opts)
    run_and_check(b, hv, f"rising{seed}-scale", sm_scale=0.25, **opts)


@pytest.mark.parametrize("case", PEAKED, ids=[f"valu-peaked{c[0]}" for c in PEAKED])
def test_peaked_valu_engine(case):
    """The vector-ALU decode engine under a one-hot row and rising scores:
    its rescale exchanges every column's factor through LDS."""
    seed, hq, hkv, d, plen, reqs, opts = case
    b, _ = small_batch((seed, hq, hkv, d, plen, reqs, opts))
    hv = W.plant_one_hot(b, W.host_values(b, seed + 1), seed + 2, alpha_log2=4)
    run_and_check(b, hv, f"valu-one-hot{seed}", decode_engine=B.PFX_DECODE_VALU, **opts)
    hv = W.host_values_shaped(b, seed + 3, key_gain=lambda p: 1.0 + p / 256.0, q_gain=4.0, v_gain=0.25)
    run_and_check(b, hv, f"valu-rising{seed}", decode_engine=B.PFX_DECODE_VALU, **opts)


def test_graph_replay_matches_eager():
    """A mixed step (append, then attention) captured into a HIP graph through
    torch's graph API and replayed several times, with eager work and
    synchronizations between the replays: every replay reproduces the eager
    result bit for bit (the library's calls are plain kernel launches on the
    given stream, with no memset nodes)."""
    seed, hq, hkv, d, plen, reqs, opts = SMALL_CASES[1]
    b = W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=256, prefix_len=plen,
                     agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
    hv = W.host_values(b, seed + 50)
    announce("graph replay: small2 mixed step, 3 replays")
    ds = RN.DeviceStep(b, hv, **opts)
    ds.step()
    B.pfx_sync_check()
    o_eager, l_eager = ds.outputs()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        cs = torch.cuda.current_stream().cuda_stream
        B.pfx_append_kv(ds.pool, ds.plan, ds.k_new, ds.v_new, stream=cs)
        B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse, stream=cs)
    for rep in range(3):
        ds.o.zero_()
        ds.lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        B.pfx_sync_check()
        o, l = ds.outputs()
        assert np.array_equal(o, o_eager), f"replay {rep}: O differs from the eager result"
        assert np.array_equal(l, l_eager), f"replay {rep}: LSE differs from the eager result"


def test_many_partials_merge():
    """Thousands of workers for a small batch: prefix items cut into pieces of
    one or two steps, 40+ partial results per row, merged by the merge launch."""
    b = W.make_batch(9, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=2048, prefix_len=[1300, 700],
                     agent=[i % 2 for i in range(40)], suffix_len=[100 + 13 * i for i in range(40)],
                     n_rows=[1] * 40)
    hv = W.host_values_fast(b, 10)
    run_and_check(b, hv, "many-partials", decode_workers=4096)


# --------------------------------------------------------------------------- the five workloads

def test_config1_extend_then_16_decode_steps():
    b = W.config_batch(1)
    hv = W.host_values(b, 2001)
    ds, o_bits, lse = run_and_check(b, hv, "config1-extend", check_pages=True)
    # 16 greedy decode steps: one new page per request at step 0, then one token per step.
    alloc_free = sorted(set(range(b.num_pages)) - set(int(p) for p in b.used_pages()))
    extra = alloc_free[:len(b.agent)]
    pool_k, pool_v = PT.expected_pools(b, hv)
    pages = list(hv.pages) + extra
    # The decode steps reuse the same device pool; the oracle follows with its own append.
    index = {int(p): i for i, p in enumerate(pages)}
    kp = np.concatenate([pool_k, np.full((len(extra),) + pool_k.shape[1:], W.POISON_BF16, np.uint16)])
    vp = np.concatenate([pool_v, np.full_like(kp[len(pool_k):], W.POISON_BF16)])
    rng = np.random.Generator(np.random.PCG64(3001))
    for step in range(16):
        sb = W.tiny_decode_step(b, step, extra)
        q = W.bf16_round(rng.standard_normal((4, 8, 64), dtype=np.float32))
        kn = W.bf16_round(rng.standard_normal((4, 2, 64), dtype=np.float32))
        vn = W.bf16_round(rng.standard_normal((4, 2, 64), dtype=np.float32))
        pool = ds.pool
        plan = B.plan_from_batch(pool, sb, B.PFX_MODE_DECODE).upload()
        qd, knd, vnd = RN.to_device_bits(q), RN.to_device_bits(kn), RN.to_device_bits(vn)
        o = torch.empty((4, 8, 64), dtype=torch.bfloat16, device="cuda")
        l = torch.empty((4, 8), dtype=torch.float32, device="cuda")
        B.pfx_append_kv(pool, plan, knd, vnd)
        B.pfx_attention(pool, plan, qd, o, l)
        B.pfx_sync_check()
        sp = [np.array([index[int(p)] for p in pl]) for pl in sb.suffix_pages]
        pp = [np.array([index[int(p)] for p in pl]) for pl in sb.prefix_pages]
        kp, vp = oracle.append_kv(kp, vp, sp, sb.suffix_len, sb.n_rows, kn, vn)
        gk, gv = ds.read_pages(pages)
        assert np.array_equal(gk, kp) and np.array_equal(gv, vp), f"decode step {step}: pool differs"
        ro, rl = oracle.prefix_shared_attention(kp, vp, pp, sb.prefix_len, sb.agent, sp, sb.suffix_len, sb.n_rows,
                                                q, 8)
        PT.compare(sb, RN.to_host_bits(o), l.cpu().numpy(), ro, rl, f"config1 decode step {step}")


def relocate(batch, hv, seed):
    """Same logical content at a different page placement."""
    nb = W.make_batch(seed, num_q_heads=batch.num_q_heads, num_kv_heads=batch.num_kv_heads,
                      head_dim=batch.head_dim, num_pages=batch.num_pages, prefix_len=batch.prefix_len,
                      agent=batch.agent, suffix_len=batch.suffix_len, n_rows=batch.n_rows)
    old = {int(p): i for i, p in enumerate(hv.pages)}
    mapping = {}
    for a in range(len(batch.prefix_pages)):
        for x, y in zip(batch.prefix_pages[a], nb.prefix_pages[a]):
            mapping[int(y)] = old[int(x)]
    for r in range(len(batch.suffix_pages)):
        for x, y in zip(batch.suffix_pages[r], nb.suffix_pages[r]):
            mapping[int(y)] = old[int(x)]
    pages = np.array(sorted(mapping), np.int64)
    src = np.array([mapping[int(p)] for p in pages])
    return nb, W.HostValues(pages, hv.k_pages[src], hv.v_pages[src], hv.q, hv.k_new, hv.v_new)


def test_config2_decode_deterministic_and_placement_invariant():
    b = W.config_batch(2)
    hv = W.host_values_fast(b, 2002)
    ds, o1, l1 = run_and_check(b, hv, "config2")
    ds.attention()
    B.pfx_sync_check()
    o2, l2 = ds.outputs()
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2), "rerun is not bit-identical"
    del ds
    nb, nhv = relocate(b, hv, 4242)
    announce("config2 relocated")
    ds2 = RN.DeviceStep(nb, nhv)
    ds2.step()
    B.pfx_sync_check()
    o3, l3 = ds2.outputs()
    assert np.array_equal(o1, o3) and np.array_equal(l1, l3), "placement changed the result bits"


def test_config2_valu_engine_every_row():
    """Decode-8B with the decode pieces on the vector ALU: every row against
    the oracle, and within the oracle tolerance of the MFMA engine."""
    b = W.config_batch(2)
    hv = W.host_values_fast(b, 2002)
    ds, o_v, l_v = run_and_check(b, hv, "config2-valu", decode_engine=B.PFX_DECODE_VALU)
    del ds
    announce("config2 on the MFMA engine, for the engine-to-engine difference")
    ds = RN.DeviceStep(b, hv)
    ds.step()
    B.pfx_sync_check()
    o_m, l_m = ds.outputs()
    diff = float(np.abs(oracle.bf16_bits_to_f64(o_v) - oracle.bf16_bits_to_f64(o_m)).max())
    announce(f"config2 engines: max |O_valu - O_mfma| = {diff:.2e}")
    assert diff <= PT.MAX_ABS, "the two engines differ by more than the oracle tolerance"
    assert float(np.abs(l_v - l_m).max()) <= PT.LSE_ABS


def sample_rows(batch, rng, per=16):
    rows = {}
    for r in range(len(batch.agent)):
        n = int(batch.n_rows[r])
        if n == 0:
            continue
        L = int(batch.suffix_len[r])
        cand = {0, n - 1}
        for i in range(n):                      # rows on page boundaries of the suffix
            if (L - n + i) % 16 in (0, 15):
                cand.add(i)
        cand = sorted(cand)
        pick = set(rng.choice(cand, size=min(len(cand), per // 2), replace=False).tolist())
        pick |= set(rng.integers(0, n, size=per // 2).tolist())
        pick |= {0, n - 1}
        rows[r] = sorted(pick)
    return rows


@pytest.mark.timeout(600)
def test_config3_extend_every_row():
    """Extend-8B: all 36k rows x 32 heads against the oracle (run in parallel
    worker processes, one job per request and KV head)."""
    b = W.config_batch(3)
    hv = W.host_values_fast(b, 2003)
    run_and_check(b, hv, "config3", parallel=True)


def test_config3_shape_small_full():
    """Config 3's shape with shorter lengths, every row checked."""
    b = W.make_batch(33, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=4096, prefix_len=[700, 1024, 33],
                     agent=[0, 1, 2, 0, 1, 2, -1], suffix_len=[256, 300, 17, 129, 64, 200, 90],
                     n_rows=[256, 300, 17, 129, 64, 200, 90])
    hv = W.host_values_fast(b, 34)
    run_and_check(b, hv, "config3-small")


@pytest.mark.parametrize("d,hq", [(128, 32), (64, 16)])
def test_long_prefix_and_suffix(d, hq):
    """A 24,576-token prefix (1536 pages) extended and decoded against, and a
    17,000-token suffix with 64 query rows at its end: extend blocks stream
    more page ids than any fixed table would hold."""
    reqs = [(0, 300, 300), (0, 50, 1), (0, 1, 1), (-1, 17000, 64), (1, 40, 40), (0, 70, 1), (0, 33, 3)]
    b = W.make_batch(24, num_q_heads=hq, num_kv_heads=8, head_dim=d, num_pages=4096, prefix_len=[24576, 1000],
                     agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])
    hv = W.host_values_fast(b, 25)
    run_and_check(b, hv, f"long-prefix-d{d}", parallel=True)


@pytest.mark.timeout(600)
def test_config4_gather_evicted_then_decode():
    b = W.config_batch(4)
    hv = W.host_values_fast(b, 2004)
    evicted = [int(a) for a in b.meta["evicted"]]
    run_and_check(b, hv, "config4", host_resident=evicted, parallel=True)


def test_config4_valu_engine_every_row():
    """Hetero-8B on the vector-ALU decode engine: the Zipf-skewed agents that
    the MFMA engine runs as wide blocks go in 64-column pieces here; every row
    against the oracle."""
    b = W.config_batch(4)
    hv = W.host_values_fast(b, 2004)
    ds, _, _ = run_and_check(b, hv, "config4-valu", parallel=True, decode_engine=B.PFX_DECODE_VALU)
    assert ds.plan.stats().num_wide_blocks == 0


@pytest.mark.timeout(900)
def test_config5_80_layers_every_layer():
    """70B-like mixed batch over 80 layers with independent pools (device-drawn
    values).  Every layer is checked: layer 0 and one seeded layer on all 448
    decode rows and 16 rows per extend request, every other layer on a seeded
    10% of the decode requests and 2 rows per extend request.  The oracle
    runs in worker processes while the next layers compute."""
    b = W.config_batch(5)
    layers = int(b.meta["layers"])
    hkv, d, hq = b.num_kv_heads, b.head_dim, b.num_q_heads
    announce(f"config5: {layers} layers, pool {b.num_pages} pages/layer, tokens {b.num_tokens}")
    gen = torch.Generator(device="cuda")
    shape = (b.num_pages, hkv, 16, d)
    # Each layer's pool: the same device-drawn N(0,1) pages rotated by a
    # layer-specific page offset, so every layer holds different data while
    # 200 GB are filled at copy speed.
    gen.manual_seed(50_000)
    base_k = torch.randn(shape, dtype=torch.bfloat16, device="cuda", generator=gen)
    base_v = torch.randn(shape, dtype=torch.bfloat16, device="cuda", generator=gen)
    pools_k, pools_v = [], []
    for layer in range(layers):
        pools_k.append(torch.roll(base_k, shifts=977 * layer + 1, dims=0))
        pools_v.append(torch.roll(base_v, shifts=1489 * layer + 3, dims=0))
    del base_k, base_v
    gen.manual_seed(5)
    t = b.num_tokens
    q = torch.randn((t, hq, d), dtype=torch.bfloat16, device="cuda", generator=gen)
    kn = torch.randn((t, hkv, d), dtype=torch.bfloat16, device="cuda", generator=gen)
    vn = torch.randn((t, hkv, d), dtype=torch.bfloat16, device="cuda", generator=gen)
    o = torch.empty((t, hq, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((t, hq), dtype=torch.float32, device="cuda")
    pool0 = B.make_pool(b.num_pages, hkv, d, pools_k[0], pools_v[0])
    plan = B.plan_from_batch(pool0, b, B.PFX_MODE_MIXED).upload()
    rng = np.random.default_rng(55)
    full_layers = {0, int(rng.integers(1, layers))}
    ext = [r for r in range(len(b.agent)) if b.n_rows[r] > 1]
    dec = [r for r in range(len(b.agent)) if b.n_rows[r] == 1]
    q_bits = RN.to_host_bits(q)
    kn_bits, vn_bits = RN.to_host_bits(kn), RN.to_host_bits(vn)
    q_indptr = b.q_indptr()
    ck = PT.checker()
    pending = []

    def finish(entry):
        layer, nrows, h = entry
        res = ck.collect(h, f"config5 layer {layer}")
        announce(f"config5 layer {layer}: rows={nrows} max_abs={res[0]:.2e} rel={res[1]:.2e} lse={res[2]:.2e}")

    for layer in range(layers):
        pool = B.make_pool(b.num_pages, hkv, d, pools_k[layer], pools_v[layer])
        B.pfx_append_kv(pool, plan, kn, vn)
        B.pfx_attention(pool, plan, q, o, lse)
        if layer in full_layers:
            rows = {r: [0] for r in dec}
            rows.update({r: v for r, v in sample_rows(b, rng, per=16).items() if r in ext})
        else:
            rows = {int(r): [0] for r in rng.choice(dec, size=len(dec) // 10, replace=False)}
            rows.update({r: sorted(set(rng.integers(0, int(b.n_rows[r]), size=2).tolist())) for r in ext})
        need = set()
        for r in rows:
            need.update(int(p) for p in b.prefix_pages[int(b.agent[r])])
            L, n = int(b.suffix_len[r]), int(b.n_rows[r])
            last = L - n + max(rows[r])                       # the last key any checked row sees
            need.update(int(p) for p in b.suffix_pages[r][:last // 16 + 1])
        pages = np.array(sorted(need), np.int64)
        idx = torch.from_numpy(pages).cuda()
        tok = torch.from_numpy(np.array([q_indptr[r] + i for r in sorted(rows) for i in rows[r]], np.int64)).cuda()
        B.pfx_sync_check()
        kp = pools_k[layer].view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        vp = pools_v[layer].view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        o_rows = o.view(torch.int16).index_select(0, tok).cpu().numpy().view(np.uint16)
        l_rows = lse.index_select(0, tok).cpu().numpy()
        # append bit-exactness on the checked requests' new-token slots
        index = {int(p): i for i, p in enumerate(pages)}
        for r in list(rows)[:24]:
            n, L = int(b.n_rows[r]), int(b.suffix_len[r])
            for i in rows[r]:
                pos = L - n + i
                pg = index[int(b.suffix_pages[r][pos // 16])]
                assert np.array_equal(kp[pg, :, pos % 16], kn_bits[q_indptr[r] + i]), f"layer {layer}: K append"
                assert np.array_equal(vp[pg, :, pos % 16], vn_bits[q_indptr[r] + i]), f"layer {layer}: V append"
        h = ck.submit(b, pages, kp, vp, PT.gather_rows(q_bits, b, rows), o_rows, l_rows, rows, split_heads=False,
                      partial_pages=True)
        pending.append((layer, sum(len(v) for v in rows.values()), h))
        del kp, vp
        while len(pending) > 3:
            finish(pending.pop(0))
    while pending:
        finish(pending.pop(0))
    del pools_k, pools_v
    torch.cuda.empty_cache()


STEP_CASES = [
    # (label, batch factory, DeviceStep options)
    ("mixed-extend", lambda: small_batch(SMALL_CASES[1])[0], {}),                       # append kernel first
    ("decode-multirow-g1", lambda: W.make_batch(41, num_q_heads=8, num_kv_heads=8, head_dim=64, num_pages=512,
                                                prefix_len=[300, 45], agent=[0, 1, 0, -1, 1, 0],
                                                suffix_len=[40, 16, 33, 20, 1, 70], n_rows=[16, 16, 1, 9, 1, 13]),
     dict(piece_steps=1)),                                                               # new rows over 2 steps / 2 pieces
    ("decode-multirow-g2", lambda: W.make_batch(42, num_q_heads=16, num_kv_heads=8, head_dim=128, num_pages=512,
                                                prefix_len=[130], agent=[0, 0, -1, 0],
                                                suffix_len=[35, 8, 64, 100], n_rows=[8, 3, 8, 1]), {}),
    ("decode-8B", lambda: W.config_batch(2), {}),
    ("decode-multirow-g1-valu", lambda: W.make_batch(41, num_q_heads=8, num_kv_heads=8, head_dim=64, num_pages=512,
                                                     prefix_len=[300, 45], agent=[0, 1, 0, -1, 1, 0],
                                                     suffix_len=[40, 16, 33, 20, 1, 70], n_rows=[16, 16, 1, 9, 1, 13]),
     dict(piece_steps=1, decode_engine=B.PFX_DECODE_VALU)),
    ("decode-8B-valu", lambda: W.config_batch(2), dict(decode_engine=B.PFX_DECODE_VALU)),
]


@pytest.mark.parametrize("case", STEP_CASES, ids=[c[0] for c in STEP_CASES])
def test_step_equals_append_then_attention(case):
    """pfx_step (the append folded into the decode launch when the plan has
    no extend blocks) gives the outputs of pfx_append_kv + pfx_attention bit
    for bit, and the pool the oracle's append, with every other page
    untouched."""
    label, make, opts = case
    b = make()
    hv = W.host_values_fast(b, 77) if b.num_pages > 10000 else W.host_values(b, 77)
    announce(f"step {label}: tokens={b.num_tokens} reqs={len(b.agent)} G={b.group} {opts}")
    ref = RN.DeviceStep(b, hv, **opts)
    ref.step()
    B.pfx_sync_check()
    o_ref, l_ref = ref.outputs()
    del ref
    ds = RN.DeviceStep(b, hv, **opts)
    B.pfx_step(ds.pool, ds.plan, ds.k_new, ds.v_new, ds.q, ds.o, ds.lse)
    B.pfx_sync_check()
    o, l = ds.outputs()
    assert np.array_equal(o, o_ref) and np.array_equal(l, l_ref), f"{label}: step differs from append + attention"
    exp_k, exp_v = PT.expected_pools(b, hv)
    gk, gv = ds.read_pages(hv.pages)
    assert np.array_equal(gk, exp_k) and np.array_equal(gv, exp_v), f"{label}: pool differs from the oracle's append"
    assert_untouched(ds, hv.pages, label)
    o_or, l_or = PT.reference(b, hv, (exp_k, exp_v))
    res = PT.compare(b, o, l, o_or, l_or, label)
    announce(f"step {label}: bit-identical to append + attention; oracle max_abs={res[0]:.2e} rel={res[1]:.2e}")
