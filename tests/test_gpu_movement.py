"""Prefix movement on the GPU (Sec. 4.2, Eq. (8) and the paragraph before
it): an agent's prefix pages evicted to a pinned host store and loaded back,
the load on a second stream while attention for the other agents runs on
the first.  Pinned by bit-exact round trips (store bytes equal the pool's,
reloaded pool pages equal the originals, as the page-copy oracle states) and
by the decode outputs: bit-identical before eviction and after the reload,
and the overlapped attention bit-identical to the same call run alone."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2608_25523_amd import binding as B
from paper_2608_25523_amd import movement as MV
from paper_2608_25523_amd import runner as RN
from paper_2608_25523_amd import workloads as W

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu-test] {msg}", flush=True)


def host_bits(t):
    return t.view(torch.int16).numpy().view(np.uint16)


@pytest.mark.timeout(300)
def test_prefix_evict_and_reload_beside_attention():
    b = W.config_batch(2)
    hkv, d, hq = b.num_kv_heads, b.head_dim, b.num_q_heads
    announce(f"movement: config-2 batch, agent 0's {len(b.prefix_pages[0])} prefix pages out and back")
    ds = RN.DeviceStep(b, W.host_values_fast(b, 7), poison=False)
    ds.step()
    B.pfx_sync_check()
    o_before, lse_before = ds.outputs()

    agent = 0
    pages = np.asarray(b.prefix_pages[agent], np.int32)
    k0, v0 = ds.read_pages(pages)
    store = MV.HostStore(len(pages) + 8, hkv, d)
    slots = store.alloc.alloc(len(pages))
    mover = MV.Mover(ds.pool, store, len(pages))

    # Eviction: the store's slots take the pool's bytes, its other pages stay.
    store_k0, store_v0 = host_bits(store.k).copy(), host_bits(store.v).copy()
    mover.evict(pages, slots)
    B.pfx_sync_check()
    src = np.arange(len(pages))
    assert np.array_equal(host_bits(store.k), oracle.page_copy(store_k0, k0, slots, src))
    assert np.array_equal(host_bits(store.v), oracle.page_copy(store_v0, v0, slots, src))

    # The freed pool pages are reused: overwrite them.
    idx = torch.from_numpy(pages.astype(np.int64)).cuda()
    ds.k_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)
    ds.v_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)

    # Attention for the other agents' requests, alone first (reference) ...
    others = dataclasses.replace(b, n_rows=np.where(b.agent == agent, 0, b.n_rows).astype(np.int32))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(31)
    q2 = torch.randn((others.num_tokens, hq, d), dtype=torch.bfloat16, device="cuda", generator=gen)
    o2 = torch.empty_like(q2)
    lse2 = torch.empty((others.num_tokens, hq), dtype=torch.float32, device="cuda")
    plan2 = B.plan_from_batch(ds.pool, others, B.PFX_MODE_MIXED).upload()
    B.pfx_attention(ds.pool, plan2, q2, o2, lse2)
    B.pfx_sync_check()
    o2_alone, lse2_alone = RN.to_host_bits(o2), lse2.cpu().numpy()

    # ... then with agent 0's reload running on a second stream.
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(main)                       # the overwrite above comes first
    mover.load(pages, slots, stream=side.cuda_stream)
    for _ in range(10):
        B.pfx_attention(ds.pool, plan2, q2, o2, lse2)
    main.wait_stream(side)                       # the full step needs the reloaded prefix
    B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse)
    torch.cuda.synchronize()
    B.pfx_sync_check()

    k1, v1 = ds.read_pages(pages)
    assert np.array_equal(k1, k0) and np.array_equal(v1, v0), "reloaded prefix pages differ"
    assert np.array_equal(RN.to_host_bits(o2), o2_alone), "attention beside the reload differs from alone"
    assert np.array_equal(lse2.cpu().numpy(), lse2_alone)
    o_after, lse_after = ds.outputs()
    assert np.array_equal(o_after, o_before), "decode output changed across eviction and reload"
    assert np.array_equal(lse_after, lse_before)
    announce("movement: round trip bit-exact, outputs bit-identical")


@pytest.mark.timeout(300)
def test_prefix_round_trip_by_copy_engines():
    """The same round trip through the copy engines (evict: a device page
    copy into a staging area, then asynchronous memory copies to the store;
    load: the reverse), the load beside attention on a second stream: store
    bytes, reloaded pages and outputs as with the kernel copy."""
    b = W.config_batch(2)
    hkv, d, hq = b.num_kv_heads, b.head_dim, b.num_q_heads
    announce(f"movement (copy engines): agent 1's {len(b.prefix_pages[1])} prefix pages out and back")
    ds = RN.DeviceStep(b, W.host_values_fast(b, 8), poison=False)
    ds.step()
    B.pfx_sync_check()
    o_before, lse_before = ds.outputs()
    agent = 1
    pages = np.asarray(b.prefix_pages[agent], np.int32)
    k0, v0 = ds.read_pages(pages)
    store = MV.HostStore(2 * len(pages) + 8, hkv, d)
    store.alloc.alloc(5)                               # the prefix's slots do not start at 0
    slots = store.alloc.alloc(len(pages))
    slots = np.concatenate([slots[: len(pages) // 2], slots[len(pages) // 2:] + 3])  # two runs
    mover = MV.Mover(ds.pool, store, len(pages), staging=True)
    store_k0, store_v0 = host_bits(store.k).copy(), host_bits(store.v).copy()
    mover.evict_dma(pages, slots)
    torch.cuda.synchronize()
    B.pfx_sync_check()
    src = np.arange(len(pages))
    assert np.array_equal(host_bits(store.k), oracle.page_copy(store_k0, k0, slots, src))
    assert np.array_equal(host_bits(store.v), oracle.page_copy(store_v0, v0, slots, src))
    idx = torch.from_numpy(pages.astype(np.int64)).cuda()
    ds.k_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)
    ds.v_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)
    others = dataclasses.replace(b, n_rows=np.where(b.agent == agent, 0, b.n_rows).astype(np.int32))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(32)
    q2 = torch.randn((others.num_tokens, hq, d), dtype=torch.bfloat16, device="cuda", generator=gen)
    o2 = torch.empty_like(q2)
    lse2 = torch.empty((others.num_tokens, hq), dtype=torch.float32, device="cuda")
    plan2 = B.plan_from_batch(ds.pool, others, B.PFX_MODE_MIXED).upload()
    B.pfx_attention(ds.pool, plan2, q2, o2, lse2)
    B.pfx_sync_check()
    o2_alone, lse2_alone = RN.to_host_bits(o2), lse2.cpu().numpy()
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(main)
    mover.load_dma(pages, slots, stream=side.cuda_stream)
    for _ in range(10):
        B.pfx_attention(ds.pool, plan2, q2, o2, lse2)
    main.wait_stream(side)
    B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse)
    torch.cuda.synchronize()
    B.pfx_sync_check()
    k1, v1 = ds.read_pages(pages)
    assert np.array_equal(k1, k0) and np.array_equal(v1, v0), "reloaded prefix pages differ"
    assert np.array_equal(RN.to_host_bits(o2), o2_alone) and np.array_equal(lse2.cpu().numpy(), lse2_alone)
    o_after, lse_after = ds.outputs()
    assert np.array_equal(o_after, o_before) and np.array_equal(lse_after, lse_before)
    # Into consecutive free pool pages: the runs go straight into the pool.
    used = set(int(p) for p in b.used_pages())
    run_at = next(p for p in range(0, b.num_pages - len(pages)) if not any(q in used for q in range(p, p + len(pages))))
    run = np.arange(run_at, run_at + len(pages), dtype=np.int32)
    mover.load_dma(run, slots, pool_tensors=(ds.k_pool, ds.v_pool))
    torch.cuda.synchronize()
    k2, v2 = ds.read_pages(run)
    assert np.array_equal(k2, k0) and np.array_equal(v2, v0), "direct copies into consecutive pages differ"
    with pytest.raises(ValueError):
        mover.load_dma(run - run_at - 1, slots, pool_tensors=(ds.k_pool, ds.v_pool))
    # Paced: the staged reload cut into parts, part i waiting for the i-th of
    # the attention calls beside it.
    ds.k_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)
    ds.v_pool.view(torch.int16).index_fill_(0, idx, W.POISON_BF16)
    side.wait_stream(main)
    events = []
    for _ in range(12):
        B.pfx_attention(ds.pool, plan2, q2, o2, lse2)
        ev = torch.cuda.Event()
        ev.record(main)
        events.append(ev)
    mover.load_dma(pages, slots, stream=side.cuda_stream, after=events)
    main.wait_stream(side)
    torch.cuda.synchronize()
    B.pfx_sync_check()
    k3, v3 = ds.read_pages(pages)
    assert np.array_equal(k3, k0) and np.array_equal(v3, v0), "paced reload differs"
    assert np.array_equal(RN.to_host_bits(o2), o2_alone) and np.array_equal(lse2.cpu().numpy(), lse2_alone)
    announce("movement (copy engines): round trip bit-exact, outputs bit-identical, paced reload bit-exact")
