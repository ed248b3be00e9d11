"""Benchmark: shared-prefix decode attention (HBM GB/s) and extend attention
(TFLOP/s) at the Llama-3-8B attention-layer shape, on one MI355X.

A step is one pass of the hot path over one batch: the KV append of the
step's new tokens and attention for every query row, one pfx_step call (the
decode launch -- agent prefixes shared by their decode rows and each
request's own suffix, cut into pieces -- writes the new tokens into the
pool as it reads them; then the log-sum-exp merge of the pieces).  Inputs are
resident in HBM before timing starts.

Primary line (``value``): decode-8B -- Hq 32 / Hkv 8 / d 128, 4 agent
prefixes x 2048 tokens, 64 decode requests (16 per agent, suffix U[64, 512]),
1M-token (65,536-page) pool, pages scattered.  value = unique KV bytes per
step (each prefix once + every suffix) / step time.  The step rotates over
replicas of the batch on disjoint pages of the same pool so that the timed
working set exceeds the 256 MB last-level cache.

``extend``: extend-8B -- 3 prefixes x 4096, 32 requests with suffix
U[256, 2048] prefilled against their agent's prefix; TFLOP/s over the
causal-exact flop count.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--no-extend] [--no-configs] [--no-engines]
                       [--no-extras] [--engines-only] [--calib-copy]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2516.6      # MI355X dense bf16 MFMA, published
METRIC = "shared-prefix decode attn HBM GB/s; extend attn TFLOP/s (8B layer shape)"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def timed_steps(fn_step, fn_attn, steps, warmup, torch, group=10):
    """Run warmup + timed steps; returns (ms per step, mean ms of the
    attention call measured with events on the launch stream).

    Two passes: the steps with nothing between them (events only around the
    whole pass) give the step time; the same number of attention calls back
    to back, bracketed by one event pair, give the attention duration.
    (Event records inside a ~35 us step add several us to what they
    bracket.)"""
    for i in range(warmup):
        fn_step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(steps):
        fn_step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    step_ms = max(wall, e0.elapsed_time(e1) / steps)
    # The attention pass in groups of (up to) 10 back-to-back calls, one event
    # pair per group: the mean over all calls, and the spread over groups.
    attn, spread = attention_ms(fn_attn, max(steps, MIN_ATTN_CALLS), torch, group=group)
    return step_ms, attn, spread


# Attention is timed over at least this many calls, whatever --steps is.
MIN_ATTN_CALLS = 100


def attention_ms(fn_attn, calls, torch, group=10):
    """Mean ms of ``calls`` attention calls (rounded up to whole groups),
    launched back to back on the current stream in groups of ``group`` under
    one event pair each; p10 / p50 / p90 over the groups."""
    stream = torch.cuda.current_stream()
    for i in range(3):
        fn_attn(i)
    torch.cuda.synchronize()
    calls = (calls + group - 1) // group * group
    evs = []
    for g0 in range(0, calls, group):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for i in range(g0, g0 + group):
            fn_attn(i)
        b.record(stream)
        evs.append((a, b))
    torch.cuda.synchronize()
    per = sorted(a.elapsed_time(b) / group for a, b in evs)
    mean = sum(a.elapsed_time(b) for a, b in evs) / calls
    pct = lambda q: per[min(len(per) - 1, int(round(q * (len(per) - 1))))]
    return mean, {"p10": pct(0.1), "p50": pct(0.5), "p90": pct(0.9), "calls": calls}


def bench_decode(args, torch, B, RN, W):
    b = W.config_batch(2)
    hv = W.host_values_fast(b, 2002)
    ds = RN.DeviceStep(b, hv)
    reps = W.replicas(b, args.replicas, 77)
    # Replicas hold the same page contents at other pages (device copies).
    src = torch.from_numpy(b.used_pages()).cuda()
    plans = [ds.plan]
    for rb in reps[1:]:
        dst = torch.from_numpy(rb.used_pages()).cuda()
        ds.k_pool.view(torch.int16).index_copy_(0, dst, ds.k_pool.view(torch.int16).index_select(0, src))
        ds.v_pool.view(torch.int16).index_copy_(0, dst, ds.v_pool.view(torch.int16).index_select(0, src))
        plans.append(B.plan_from_batch(ds.pool, rb, B.PFX_MODE_DECODE).upload())
    torch.cuda.synchronize()

    def step(i):
        # append + attention in one call: the decode launch appends as it goes
        B.pfx_step(ds.pool, plans[i % len(plans)], ds.k_new, ds.v_new, ds.q, ds.o, ds.lse)

    def attn(i):
        B.pfx_attention(ds.pool, plans[i % len(plans)], ds.q, ds.o, ds.lse)

    def unfused(i):
        plan = plans[i % len(plans)]
        B.pfx_append_kv(ds.pool, plan, ds.k_new, ds.v_new)
        B.pfx_attention(ds.pool, plan, ds.q, ds.o, ds.lse)

    ms, attn_ms, spread = timed_steps(step, attn, args.steps, args.warmup, torch)
    unfused_ms, _ = attention_ms(unfused, max(args.steps, MIN_ATTN_CALLS), torch)
    # The same attention with the decode pieces on the vector ALU (dot
    # products instead of MFMA tiles), for the engine comparison.
    vplans = [B.plan_from_batch(ds.pool, rb, B.PFX_MODE_DECODE, decode_engine=B.PFX_DECODE_VALU).upload()
              for rb in reps]

    def attn_valu(i):
        B.pfx_attention(ds.pool, vplans[i % len(vplans)], ds.q, ds.o, ds.lse)

    for i in range(args.warmup):
        attn_valu(i)
    valu_ms, valu_spread = attention_ms(attn_valu, max(args.steps, MIN_ATTN_CALLS), torch)
    del vplans
    B.pfx_sync_check()
    graph_ms = graph_replay_ms(plans, ds, args.steps, torch, B)
    side = side_costs(b, ds, plans, args.steps, torch, B)
    u = b.unique_kv_bytes()
    st = ds.plan.stats()
    side["unfused_step_us"] = round(unfused_ms * 1e3, 3)
    return dict(batch=b, hv=hv, ms=ms, attn_ms=attn_ms, spread=spread, graph_ms=graph_ms, unique_bytes=u,
                replicas=len(plans), stats=st, side=side, valu_ms=valu_ms, valu_spread=valu_spread)


def bench_prefix_engines(args, torch, B, RN, W):
    """The grouped-decode prefix phase alone on each decode engine: decode-8B's
    agents and prefixes with a one-token suffix per request, so nearly all of
    the work is prefix steps shared by 64 columns.  Each engine at piece
    lengths 4, 8 and 16 steps (one workgroup per piece: 1024, 768 and 640
    workgroups), rotating over replicas as the decode-8B bench does."""
    rng = np.random.Generator(np.random.PCG64(2608))
    agents = np.repeat(np.arange(4), 16).astype(np.int32)[rng.permutation(64)]
    b = W.make_batch(2608, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536, prefix_len=[2048] * 4,
                     agent=agents, suffix_len=np.ones(64, np.int32), n_rows=np.ones(64, np.int32))
    ds = RN.DeviceStep(b, W.host_values_fast(b, 2609), poison=False)
    reps = W.replicas(b, args.replicas, 79)
    src = torch.from_numpy(b.used_pages()).cuda()
    for rb in reps[1:]:
        dst = torch.from_numpy(rb.used_pages()).cuda()
        ds.k_pool.view(torch.int16).index_copy_(0, dst, ds.k_pool.view(torch.int16).index_select(0, src))
        ds.v_pool.view(torch.int16).index_copy_(0, dst, ds.v_pool.view(torch.int16).index_select(0, src))
    torch.cuda.synchronize()
    out = {"workload": "decode-8B prefix phase: Hq32/Hkv8/d128, 4 prefixes x 2048, 64 decode reqs (16/agent) "
                       "with a 1-token suffix each", "unique_kv_bytes": b.unique_kv_bytes(), "replicas": len(reps)}
    for name, eng in (("mfma", B.PFX_DECODE_MFMA), ("valu", B.PFX_DECODE_VALU)):
        by = {}
        for ps in (4, 8, 16):
            plans = [B.plan_from_batch(ds.pool, rb, B.PFX_MODE_DECODE, piece_steps=ps, decode_engine=eng).upload()
                     for rb in reps]

            def attn(i, plans=plans):
                B.pfx_attention(ds.pool, plans[i % len(plans)], ds.q, ds.o, ds.lse)

            for i in range(args.warmup):
                attn(i)
            ms, _ = attention_ms(attn, max(args.steps, MIN_ATTN_CALLS), torch)
            by[ps] = round(ms * 1e3, 3)
            del plans
        best = min(by, key=by.get)
        out[name] = {"attn_us": by[best], "piece_steps": best, "attn_us_by_piece_steps": by}
    B.pfx_sync_check()
    out["valu_over_mfma"] = round(out["valu"]["attn_us"] / out["mfma"]["attn_us"], 3)
    return out


def side_costs(b, ds, plans, steps, torch, B):
    """The step's other parts, timed apart from attention: the KV append
    (events around back-to-back calls), and the plan -- built on the host
    from the batch's page tables (CPU wall time of the call, binding included) and copied
    into an already allocated workspace (events)."""
    n = max(steps, 20)
    append_ms = events_ms(lambda: B.pfx_append_kv(ds.pool, plans[0], ds.k_new, ds.v_new), n, torch)
    pind, pids, plen = b.prefix_csr()
    sind, sids = b.suffix_csr()
    qind = b.q_indptr()
    build = lambda: B.pfx_plan_create(ds.pool, pind, pids, plen, b.agent, sind, sids, b.suffix_len, qind,
                                      b.num_q_heads, B.PFX_MODE_DECODE)
    build()
    t0 = time.perf_counter()
    for _ in range(n):
        p = build()
    build_ms = (time.perf_counter() - t0) * 1e3 / n
    ws = torch.empty(p.workspace_bytes() + 256, dtype=torch.uint8, device="cuda")
    upload_ms = events_ms(lambda: p.upload(workspace=ws), n, torch)
    B.pfx_sync_check()
    return {"append_us": round(append_ms * 1e3, 3), "plan_build_host_us": round(build_ms * 1e3, 2),
            "plan_upload_us": round(upload_ms * 1e3, 3), "plan_workspace_bytes": int(p.workspace_bytes())}


def graph_replay_ms(plans, ds, steps, torch, B):
    """One decode step per replica plan captured into a HIP graph (through
    torch's graph API; the library's calls are plain kernel launches on the
    given stream), replayed: ms per step.  The last replayed step's output
    must equal the eager result of the same plan, else None."""
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        cs = torch.cuda.current_stream().cuda_stream
        for p in plans:
            B.pfx_step(ds.pool, p, ds.k_new, ds.v_new, ds.q, ds.o, ds.lse, stream=cs)
    torch.cuda.synchronize()
    reps = max(2, steps // len(plans))
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / (reps * len(plans))
    out_graph = ds.o.clone()
    B.pfx_attention(ds.pool, plans[-1], ds.q, ds.o, ds.lse)
    torch.cuda.synchronize()
    same = bool(torch.equal(out_graph.view(torch.int16), ds.o.view(torch.int16)))
    return ms if same else None


def bench_extend(args, torch, B, RN, W):
    """Extend-8B (config 3): steps of append + attention, then attention and
    append each timed back to back on their own."""
    b = W.config_batch(3)
    hv = W.host_values_fast(b, 2003)
    ds = RN.DeviceStep(b, hv, poison=False)
    torch.cuda.synchronize()

    def step(i):
        B.pfx_append_kv(ds.pool, ds.plan, ds.k_new, ds.v_new)
        B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse)

    def attn(i):
        B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse)

    steps = max(20, args.steps)
    ms, attn_ms, spread = timed_steps(step, attn, steps, max(2, args.warmup), torch, group=5)
    append_ms = events_ms(lambda: B.pfx_append_kv(ds.pool, ds.plan, ds.k_new, ds.v_new), 20, torch)
    B.pfx_sync_check()
    return dict(batch=b, hv=hv, ms=ms, attn_ms=attn_ms, spread=spread, append_ms=append_ms,
                flops=b.attention_flops(), steps=steps)


def cpu_baseline(res, W, seconds=12.0):
    """The fp64 oracle, as it stands, on a bounded sample of the decode step:
    whole requests (all heads) in request order, repeated until ``seconds``
    of CPU work; throughput in unique KV bytes per second."""
    import numpy as np

    import oracle

    b, hv = res["batch"], res["hv"]
    cores = len(os.sched_getaffinity(0))
    index = {int(p): i for i, p in enumerate(hv.pages)}
    pp = [np.array([index[int(p)] for p in pl]) for pl in b.prefix_pages]
    sp = [np.array([index[int(p)] for p in pl]) for pl in b.suffix_pages]
    kp, vp = oracle.append_kv(hv.k_pages, hv.v_pages, sp, b.suffix_len, b.n_rows, hv.k_new, hv.v_new)
    tau = b.num_kv_heads * b.head_dim * 4
    per_agent = {int(a): int(np.sum(b.agent == a)) for a in set(b.agent.tolist())}
    t0 = time.perf_counter()
    done = 0
    nbytes = 0.0
    while time.perf_counter() - t0 < seconds:
        r = done % len(b.agent)
        oracle.prefix_shared_attention(kp, vp, pp, b.prefix_len, b.agent, sp, b.suffix_len, b.n_rows, hv.q,
                                       b.num_q_heads, rows={r: [0]})
        # the request's unique share: its own suffix plus its agent's prefix
        # divided among the agent's requests (summing to U over the batch)
        a = int(b.agent[r])
        nbytes += (int(b.suffix_len[r]) + int(b.prefix_len[a]) / per_agent[a]) * tau
        done += 1
    dt = time.perf_counter() - t0
    threads = os.environ.get("OMP_NUM_THREADS", "unset")
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} decode requests (all 32 heads each; the 64-request decode-8B step cycled) in "
                      f"{dt:.1f} s, fp64 numpy oracle, BLAS threads {threads}"}


def cpu_baseline_extend(res, W, seconds=12.0, rows_per_call=64):
    """The fp64 oracle on a bounded sample of the extend-8B step: blocks of
    ``rows_per_call`` consecutive query rows (all 32 heads) of one request at
    a time, requests in turn, each block at a seeded random offset, until
    ``seconds`` of CPU work; throughput in causal-exact TFLOP/s of the rows
    computed."""
    import numpy as np

    import oracle

    b, hv = res["batch"], res["hv"]
    cores = len(os.sched_getaffinity(0))
    index = {int(p): i for i, p in enumerate(hv.pages)}
    pp = [np.array([index[int(p)] for p in pl]) for pl in b.prefix_pages]
    sp = [np.array([index[int(p)] for p in pl]) for pl in b.suffix_pages]
    kp, vp = oracle.append_kv(hv.k_pages, hv.v_pages, sp, b.suffix_len, b.n_rows, hv.k_new, hv.v_new)
    rng = np.random.default_rng(3003)
    t0 = time.perf_counter()
    done, flops, nrows = 0, 0, 0
    while time.perf_counter() - t0 < seconds:
        r = done % len(b.agent)
        n, L, P = int(b.n_rows[r]), int(b.suffix_len[r]), int(b.prefix_len[int(b.agent[r])])
        i0 = int(rng.integers(0, max(1, n - rows_per_call + 1)))
        rows = list(range(i0, min(n, i0 + rows_per_call)))
        oracle.prefix_shared_attention(kp, vp, pp, b.prefix_len, b.agent, sp, b.suffix_len, b.n_rows, hv.q,
                                       b.num_q_heads, rows={r: rows})
        flops += sum(4 * b.head_dim * b.num_q_heads * (P + L - n + i + 1) for i in rows)
        nrows += len(rows)
        done += 1
    dt = time.perf_counter() - t0
    threads = os.environ.get("OMP_NUM_THREADS", "unset")
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{nrows} extend rows (all 32 heads each) in {done} blocks of up to {rows_per_call} "
                      f"consecutive rows of one request, requests of the extend-8B step in turn, in {dt:.1f} s; "
                      f"fp64 numpy oracle, BLAS threads {threads}"}


def cpu_baseline_config5(torch, b, pool_k, pool_v, q, kind, u_layer, f_layer, layers, seconds=8.0, block=16):
    """The fp64 oracle on a bounded sample of one mixed-70B layer (layer 0's
    pool), the rest extrapolated: decode requests whole (all 64 heads), or
    extend blocks of ``block`` consecutive rows of one request (all heads),
    requests in turn.  Each sample is handed to the oracle as a one-request
    batch holding only its own pages (read back from the device beforehand,
    outside the timing; an extend block is its request truncated after the
    block's last row, which leaves every row's visible keys unchanged).
    Decode is scored in unique KV bytes per second (each request's suffix
    plus its share of its agent's prefix) and extrapolated to the 80 layers'
    unique bytes; extend in causal-exact flop per second, extrapolated to the
    80 layers' flops."""
    import numpy as np

    import oracle

    hq, hkv, d = b.num_q_heads, b.num_kv_heads, b.head_dim
    q_indptr = b.q_indptr()
    reqs = [r for r in range(len(b.agent)) if int(b.n_rows[r]) > 0]
    per_agent = {int(a): sum(1 for r in reqs if int(b.agent[r]) == a) for a in set(int(b.agent[r]) for r in reqs)}
    rng = np.random.default_rng(5005)

    def host_pages(pages):
        idx = torch.from_numpy(np.asarray(pages, np.int64)).to(pool_k.device)
        k = pool_k.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        v = pool_v.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        return k, v

    # Samples prepared up front: enough for the time budget, cycled if it runs out.
    prefix_cache, samples = {}, []
    for r in reqs[:: max(1, len(reqs) // 24)][:24]:
        a, n, L = int(b.agent[r]), int(b.n_rows[r]), int(b.suffix_len[r])
        P = int(b.prefix_len[a]) if a >= 0 else 0
        if a >= 0 and a not in prefix_cache:
            prefix_cache[a] = host_pages(b.prefix_pages[a])
        i0 = 0 if kind == "decode" else int(rng.integers(0, max(1, n - block + 1)))
        m = n if kind == "decode" else min(block, n - i0)
        keep_len = L - n + i0 + m                      # the suffix up to the sample's last row
        sk, sv = host_pages(b.suffix_pages[r][: (keep_len + 15) // 16])
        pk, pv = prefix_cache[a] if a >= 0 else (sk[:0], sv[:0])
        qs = q[int(q_indptr[r]) + i0: int(q_indptr[r]) + i0 + m].view(torch.int16).cpu().numpy().view(np.uint16)
        work = ((L + P / per_agent[a] if a >= 0 else L) * hkv * d * 4 if kind == "decode"
                else sum(4 * d * hq * (P + L - n + i0 + j + 1) for j in range(m)))
        samples.append((np.concatenate([pk, sk]), np.concatenate([pv, sv]), len(pk), P, a >= 0, keep_len, m, qs,
                        work))
    t0 = time.perf_counter()
    done, work, rows = 0, 0.0, 0
    while time.perf_counter() - t0 < seconds:
        kp, vp, npp, P, has, keep_len, m, qs, w = samples[done % len(samples)]
        oracle.prefix_shared_attention(kp, vp, [np.arange(npp)], [P], [0 if has else -1],
                                       [np.arange(npp, len(kp))], [keep_len], [m], qs, hq)
        work += w
        rows += m
        done += 1
    dt = time.perf_counter() - t0
    threads = os.environ.get("OMP_NUM_THREADS", "unset")
    rate = work / dt
    rec = {"cores": len(os.sched_getaffinity(0)), "kind": "oracle"}
    if kind == "decode":
        rec.update(value=round(rate / 1e9, 4), unit="GB/s",
                   extrapolated_s_80_layers=round(u_layer * layers / rate, 1),
                   sample=f"{done} decode requests of layer 0 (all {hq} heads each) in {dt:.1f} s, fp64 numpy "
                          f"oracle, BLAS threads {threads}; extrapolated by unique KV bytes")
    else:
        rec.update(value=round(rate / 1e12, 6), unit="TFLOP/s",
                   extrapolated_s_80_layers=round(f_layer * layers / rate, 1),
                   sample=f"{rows} extend rows of layer 0 (all {hq} heads each) in {done} blocks of up to {block} "
                          f"consecutive rows, in {dt:.1f} s, fp64 numpy oracle, BLAS threads {threads}; "
                          f"extrapolated by causal-exact flops")
    return rec


def copy_calibration(torch, B):
    """A plain device-to-device copy of known size through pfx_page_copy
    (used to scale the HBM byte counters read by rocprofv3)."""
    import numpy as np

    pages = 16384                      # 16384 pages x 32 KiB x (K + V) = 1 GiB read, 1 GiB written
    shape = (pages, 8, 16, 128)
    src_k = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    src_v = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    dst_k = torch.empty_like(src_k)
    dst_v = torch.empty_like(src_v)
    ids = np.arange(pages, dtype=np.int32)
    ws = torch.empty(B.pfx_page_copy_workspace_bytes(pages) + 256, dtype=torch.uint8, device="cuda")
    src = B.make_pool(pages, 8, 128, src_k, src_v)
    dst = B.make_pool(pages, 8, 128, dst_k, dst_v)
    for _ in range(3):
        B.pfx_page_copy(dst, src, ids, ids, ws)
    torch.cuda.synchronize()
    return 2 * pages * 8 * 16 * 128 * 2


def measured_copy_peak(torch, B, reps=10):
    """A measured HBM ceiling beside the nominal one: pfx_page_copy of 16384
    pages (32 KiB of K and 32 KiB of V each) device to device, in a seeded
    random order on both sides, timed with events (each call also uploads
    its two page-id lists); bytes read plus bytes written per second."""
    import numpy as np

    pages = 16384
    shape = (pages, 8, 16, 128)
    bufs = [torch.empty(shape, dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    rng = np.random.default_rng(4242)
    src_ids = rng.permutation(pages).astype(np.int32)
    dst_ids = rng.permutation(pages).astype(np.int32)
    ws = torch.empty(B.pfx_page_copy_workspace_bytes(pages) + 256, dtype=torch.uint8, device="cuda")
    src = B.make_pool(pages, 8, 128, bufs[0], bufs[1])
    dst = B.make_pool(pages, 8, 128, bufs[2], bufs[3])
    for _ in range(2):
        B.pfx_page_copy(dst, src, dst_ids, src_ids, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        B.pfx_page_copy(dst, src, dst_ids, src_ids, ws)
    e1.record()
    torch.cuda.synchronize()
    moved = 2 * (2 * pages * 8 * 16 * 128 * 2)  # K and V, read and written
    gbs = moved * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del bufs, ws
    return gbs


def events_ms(fn, n, torch, warm=3):
    """Mean ms of n back-to-back calls of fn under one event pair."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def bench_configs(torch, B, RN, W, cpu=True):
    """The other three workloads, in the default run: the tiny config-1
    extend and decode (launch-bound, reported only), config 4 (the
    pinned-host gather of 4 evicted prefixes, then decode over all 16 agents
    in the 48 GiB pool) and config 5 (80 layers' pools; its decode requests,
    its extend requests and the mixed batch, each planned once and called
    per layer)."""
    import dataclasses

    import numpy as np

    res = {}
    b = W.config_batch(1)
    ds = RN.DeviceStep(b, W.host_values_fast(b, 1001), poison=False)
    ext_ms, ext_sp = attention_ms(lambda i: B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse), 200, torch)
    sb = W.tiny_decode_step(b, 0, sorted(set(range(b.num_pages)) - set(int(p) for p in b.used_pages()))[:4])
    plan1 = B.plan_from_batch(ds.pool, sb, B.PFX_MODE_DECODE).upload()
    q1 = torch.zeros((4, 8, 64), dtype=torch.bfloat16, device="cuda")
    o1 = torch.empty_like(q1)
    l1 = torch.empty((4, 8), dtype=torch.float32, device="cuda")
    dec_ms, dec_sp = attention_ms(lambda i: B.pfx_attention(ds.pool, plan1, q1, o1, l1), 200, torch)
    res["config1"] = {"workload": "tiny: Hq8/Hkv2/d64, one 128-token prefix, 4 reqs x 32-token suffix",
                      "extend_attn_us": round(ext_ms * 1e3, 2), "decode_step_attn_us": round(dec_ms * 1e3, 2),
                      "note": "launch-bound; reported, not targeted"}
    del ds, plan1

    b = W.config_batch(4)
    evicted = [int(a) for a in b.meta["evicted"]]
    ds = RN.DeviceStep(b, W.host_values_fast(b, 2004), host_resident=evicted, poison=False)
    moved = 2 * len(ds.host_dst) * b.num_kv_heads * 16 * b.head_dim * 2
    g_ms = events_ms(ds.gather_evicted, 5, torch, warm=1)
    a_ms, a_sp = attention_ms(lambda i: B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse), MIN_ATTN_CALLS, torch)
    u = b.unique_kv_bytes()
    gbs = u / (a_ms * 1e-3) / 1e9
    res["config4"] = {"workload": "hetero-8B: 16 prefixes log-U[512,8192], 256 decode reqs Zipf(1.1), suffix "
                                  "U[32,1024], 48 GiB pool; 4 evicted prefixes gathered from pinned host first",
                      "decode_attn_us": round(a_ms * 1e3, 2),
                      "attn_us_p10_p50_p90": [round(a_sp[k] * 1e3, 2) for k in ("p10", "p50", "p90")],
                      "unique_kv_bytes": u, "decode_GBs": round(gbs, 1), "decode_frac": round(gbs / HBM_PEAK_GBS, 4),
                      "gather_bytes": moved, "gather_ms": round(g_ms, 4),
                      "gather_GBs_pcie_inclusive": round(moved / (g_ms * 1e-3) / 1e9, 1)}
    del ds
    torch.cuda.empty_cache()

    b = W.config_batch(5)
    layers = int(b.meta["layers"])
    hkv, d, hq = b.num_kv_heads, b.head_dim, b.num_q_heads
    gen = torch.Generator(device="cuda")
    gen.manual_seed(50_000)
    shape = (b.num_pages, hkv, 16, d)
    base_k = torch.randn(shape, dtype=torch.bfloat16, device="cuda", generator=gen)
    base_v = torch.randn(shape, dtype=torch.bfloat16, device="cuda", generator=gen)
    # Each layer's pool tensors stay referenced for as long as the
    # descriptors (which hold raw pointers) are used.
    keep = [(torch.roll(base_k, 977 * l + 1, 0), torch.roll(base_v, 1489 * l + 3, 0)) for l in range(layers)]
    pools = [B.make_pool(b.num_pages, hkv, d, kt, vt) for kt, vt in keep]
    del base_k, base_v
    dec_only = dataclasses.replace(b, n_rows=np.where(b.n_rows == 1, b.n_rows, 0).astype(np.int32))
    ext_only = dataclasses.replace(b, n_rows=np.where(b.n_rows > 1, b.n_rows, 0).astype(np.int32))
    u5 = dec_only.unique_kv_bytes()
    f5 = ext_only.attention_flops()
    out5 = {"workload": "mixed-70B: Hq64/Hkv8/d128, 8 prefixes x 8192; per layer 32 extend reqs (suffix "
                        "U[512,4096]) + 448 decode reqs (suffix U[64,2048]); 80 layers' pools, 2.6 GB each",
            "layers": layers, "decode_unique_kv_bytes_per_layer": u5, "extend_flops_per_layer": f5}
    for name, bb in (("decode", dec_only), ("extend", ext_only), ("mixed", b)):
        t = bb.num_tokens
        q = torch.randn((t, hq, d), dtype=torch.bfloat16, device="cuda", generator=gen)
        o = torch.empty_like(q)
        lse = torch.empty((t, hq), dtype=torch.float32, device="cuda")
        plan = B.plan_from_batch(pools[0], bb, B.PFX_MODE_MIXED).upload()
        B.pfx_attention(pools[0], plan, q, o, lse)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for l in range(layers):
            B.pfx_attention(pools[l], plan, q, o, lse)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        rec = {"ms_80_layers": round(ms, 3)}
        if name == "decode":
            g = u5 * layers / (ms * 1e-3) / 1e9
            rec.update(GBs=round(g, 1), frac=round(g / HBM_PEAK_GBS, 4))
        elif name == "extend":
            tf = f5 * layers / (ms * 1e-3) / 1e12
            rec.update(TFLOPs=round(tf, 1), frac=round(tf / BF16_PEAK_TFLOPS, 4))
        if cpu and name in ("decode", "extend"):
            rec["cpu_baseline"] = cpu_baseline_config5(torch, bb, keep[0][0], keep[0][1], q, name, u5, f5, layers)
        else:
            bound = max(u5 / (HBM_PEAK_GBS * 1e9),
                        (f5 + dec_only.attention_flops()) / (BF16_PEAK_TFLOPS * 1e12)) * layers * 1e3
            rec.update(peak_bound_ms_80_layers=round(bound, 3), frac_of_bound=round(bound / ms, 4))
        out5[name] = rec
        del q, o, lse, plan
    res["config5"] = out5
    del pools, keep
    torch.cuda.empty_cache()
    return res


def bench_extras(torch, B, RN, W):
    """Timed in the default run (skipped with --no-extras): prefix movement, the rebuild of a
    preempted request and the service-time tables."""
    res = {}
    res["movement"] = bench_movement(torch, B, RN, W)
    res["rebuild"] = bench_rebuild(torch, B, RN, W)
    from paper_2608_25523_amd import service as SV
    pre = SV.profile_prefill([256, 512, 1024, 2048, 4096, 8192], prefix_len=4096)
    dec = SV.profile_decode([1, 4, 16, 64], prefix_len=2048, suffix_len=288)
    res["service_tables"] = {
        "shape": "one layer, Hq32/Hkv8/d128; prefill over a 4096-token prefix; decode: B requests of one "
                 "agent, 2048-token prefix, 288-token suffixes",
        "t_prefill_us": {str(k): round(v * 1e6, 1) for k, v in pre.items()},
        "t_decode_step_us": {str(k): round(v * 1e6, 2) for k, v in dec.items()}}
    return res


def bench_rebuild(torch, B, RN, W, y=256, prompt=200, prefix=2048):
    """Rebuilding a preempted request's y generated tokens (Eq. (9)): by
    replaying y decode steps (append + attention each, plans built
    beforehand), and by one extend call over the y tokens (append +
    attention)."""
    import numpy as np

    full = W.make_batch(4050, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=512, prefix_len=[prefix],
                        agent=[0], suffix_len=[prompt + y], n_rows=[prompt + y])
    hv = W.host_values_fast(full, 4051)
    ds = RN.DeviceStep(full, hv, poison=False)
    kn, vn = RN.to_device_bits(hv.k_new), RN.to_device_bits(hv.v_new)
    q1 = torch.randn((1, 32, 128), dtype=torch.bfloat16, device="cuda")
    qy = torch.randn((y, 32, 128), dtype=torch.bfloat16, device="cuda")
    o1, l1 = torch.empty_like(q1), torch.empty((1, 32), dtype=torch.float32, device="cuda")
    oy, ly = torch.empty_like(qy), torch.empty((y, 32), dtype=torch.float32, device="cuda")
    plans = [B.plan_from_batch(ds.pool, W.with_lengths(full, [prompt + k + 1], [1]), B.PFX_MODE_DECODE).upload()
             for k in range(y)]
    plan_y = B.plan_from_batch(ds.pool, W.with_lengths(full, [prompt + y], [y]), B.PFX_MODE_EXTEND).upload()

    def by_decode():
        for k in range(y):
            B.pfx_append_kv(ds.pool, plans[k], kn[prompt + k:prompt + k + 1], vn[prompt + k:prompt + k + 1])
            B.pfx_attention(ds.pool, plans[k], q1, o1, l1)

    def by_extend():
        B.pfx_append_kv(ds.pool, plan_y, kn[prompt:], vn[prompt:])
        B.pfx_attention(ds.pool, plan_y, qy, oy, ly)

    dec_ms = events_ms(by_decode, 3, torch, warm=1)
    ext_ms = events_ms(by_extend, 10, torch)
    del ds, plans, plan_y
    return {"tokens": y, "prompt": prompt, "prefix": prefix, "by_decode_ms": round(dec_ms, 3),
            "t_decode_step_us": round(dec_ms / y * 1e3, 2), "by_extend_ms": round(ext_ms, 3),
            "decode_over_extend": round(dec_ms / ext_ms, 1)}


def bench_movement(torch, B, RN, W):
    """Prefix movement (Eq. (8)): B_swap per direction fitted from timed
    evictions and loads of 512, 2048 and 8192-token prefixes (mu = tau bytes
    per token); a serialized transition (two prefixes out, one in) against
    the model; and a 134 MB load on a second stream beside the decode-8B
    attention calls on the first, by the copy kernel and by the copy
    engines."""
    import numpy as np

    from paper_2608_25523_amd import movement as MV

    b = W.config_batch(2)
    ds = RN.DeviceStep(b, W.host_values_fast(b, 7), poison=False)
    hkv, d = b.num_kv_heads, b.head_dim
    tau = hkv * d * 2 * 2
    # Four replicas of the batch on disjoint pages (416 MB, more than the
    # 256 MB last-level cache), attention rotating over them, so the
    # attention figures alone and beside a load are both taken cold.
    reps = W.replicas(b, 4, 78)
    src = torch.from_numpy(b.used_pages()).cuda()
    plans = [ds.plan]
    for rb in reps[1:]:
        dst = torch.from_numpy(rb.used_pages()).cuda()
        ds.k_pool.view(torch.int16).index_copy_(0, dst, ds.k_pool.view(torch.int16).index_select(0, src))
        ds.v_pool.view(torch.int16).index_copy_(0, dst, ds.v_pool.view(torch.int16).index_select(0, src))
        plans.append(B.plan_from_batch(ds.pool, rb, B.PFX_MODE_DECODE).upload())
    used = set(int(p) for rb in reps for p in rb.used_pages())
    spare = np.array([p for p in range(b.num_pages) if p not in used], np.int32)
    rng = np.random.default_rng(77)
    spare = rng.permutation(spare)
    store = MV.HostStore(4096, hkv, d)
    mover = MV.Mover(ds.pool, store, 4096, staging=True)
    cal = MV.calibrate_swap(mover, [spare[:n] for n in (32, 128, 512)], tau)
    out = {"mu_bytes_per_token": tau, "b_swap_out_GBs": round(cal["b_out"] / 1e9, 2),
           "b_swap_in_GBs": round(cal["b_in"] / 1e9, 2),
           "overhead_out_us": round(cal["overhead_out_s"] * 1e6, 1), "overhead_in_us": round(cal["overhead_in_s"] * 1e6, 1)}
    # A transition: prefixes of 2048 and 512 tokens out, one of 8192 in, serialized.
    outs = [spare[512:640], spare[640:672]]
    ins = spare[1024:1536]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    at = 0
    for pg in outs:
        mover.evict(pg, np.arange(at, at + len(pg), dtype=np.int32))
        at += len(pg)
    mover.load(ins, np.arange(len(ins), dtype=np.int32))
    e1.record()
    torch.cuda.synchronize()
    t_meas = e0.elapsed_time(e1) * 1e-3
    tok_out, tok_in = 16 * sum(len(p) for p in outs), 16 * len(ins)
    t_model = tau * tok_out / cal["b_out"] + tau * tok_in / cal["b_in"]
    out["transition"] = {"tokens_out": tok_out, "tokens_in": tok_in, "measured_ms": round(t_meas * 1e3, 3),
                         "eq8_ms": round(t_model * 1e3, 3)}
    # Overlap: a 2048-page load on a second stream beside 30 attention calls.
    turn = [0]

    def attn():
        turn[0] += 1
        B.pfx_attention(ds.pool, plans[turn[0] % len(plans)], ds.q, ds.o, ds.lse)

    load_pages, load_slots = spare[2048:4096], np.arange(2048, dtype=np.int32)
    a_alone = events_ms(attn, 30, torch)
    l_alone = events_ms(lambda: mover.load(load_pages, load_slots), 3, torch, warm=1)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    m0, m1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    side.wait_stream(main)
    s0.record(side)
    mover.load(load_pages, load_slots, stream=side.cuda_stream)
    s1.record(side)
    m0.record(main)
    for _ in range(30):
        attn()
    m1.record(main)
    torch.cuda.synchronize()
    out["overlap"] = {"load_MB": round(len(load_pages) * 16 * tau / 1e6, 1), "load_alone_ms": round(l_alone, 3),
                      "load_beside_attention_ms": round(s0.elapsed_time(s1), 3),
                      "attention_alone_us": round(a_alone * 1e3, 2),
                      "attention_beside_load_us": round(m0.elapsed_time(m1) / 30 * 1e3, 2)}
    # The same load through the copy engines (store slots 0..2047 are one run).
    d_alone = events_ms(lambda: mover.load_dma(load_pages, load_slots), 3, torch, warm=1)
    torch.cuda.synchronize()
    side.wait_stream(main)
    s0.record(side)
    mover.load_dma(load_pages, load_slots, stream=side.cuda_stream)
    s1.record(side)
    m0.record(main)
    for _ in range(30):
        attn()
    m1.record(main)
    torch.cuda.synchronize()
    out["overlap_copy_engines"] = {"load_alone_ms": round(d_alone, 3),
                                   "load_beside_attention_ms": round(s0.elapsed_time(s1), 3),
                                   "attention_beside_load_us": round(m0.elapsed_time(m1) / 30 * 1e3, 2),
                                   "note": "scattered pool pages: staged, then one device page copy"}
    # ... and into 2048 consecutive pages (of a second pool, since the
    # decode pool has no free run that long): straight copies, no kernel.
    shape = (2048, hkv, 16, d)
    tensors = (torch.empty(shape, dtype=torch.bfloat16, device="cuda"),
               torch.empty(shape, dtype=torch.bfloat16, device="cuda"))
    mover2 = MV.Mover(B.make_pool(2048, hkv, d, *tensors), store, 4096)
    run_pages = np.arange(2048, dtype=np.int32)
    r_alone = events_ms(lambda: mover2.load_dma(run_pages, load_slots, pool_tensors=tensors), 3, torch, warm=1)
    torch.cuda.synchronize()
    side.wait_stream(main)
    s0.record(side)
    mover2.load_dma(run_pages, load_slots, stream=side.cuda_stream, pool_tensors=tensors)
    s1.record(side)
    m0.record(main)
    for _ in range(30):
        attn()
    m1.record(main)
    torch.cuda.synchronize()
    out["overlap_copy_engines_direct"] = {"load_alone_ms": round(r_alone, 3),
                                          "load_beside_attention_ms": round(s0.elapsed_time(s1), 3),
                                          "attention_beside_load_us": round(m0.elapsed_time(m1) / 30 * 1e3, 2),
                                          "note": "2048 consecutive pool pages: one copy per tensor"}
    # Paced: the staged load cut into n parts, part i waiting for the i-th
    # of n attention calls (the transfer spread over them).
    paced = {}
    for n in (64, 128, 256):
        torch.cuda.synchronize()
        side.wait_stream(main)
        events = []
        m0.record(main)
        for _ in range(n):
            attn()
            ev = torch.cuda.Event()
            ev.record(main)
            events.append(ev)
        m1.record(main)
        s0.record(side)
        mover.load_dma(load_pages, load_slots, stream=side.cuda_stream, after=events)
        s1.record(side)
        torch.cuda.synchronize()
        paced[str(n)] = {"load_ms": round(s0.elapsed_time(s1), 3),
                         "attention_beside_load_us": round(m0.elapsed_time(m1) / n * 1e3, 2)}
    a_alone2 = events_ms(attn, 64, torch)
    out["overlap_copy_engines_paced"] = {"parts_and_attention_calls": paced,
                                         "attention_alone_us": round(a_alone2 * 1e3, 2),
                                         "note": "the staged 134 MB load in n parts, part i after attention call i"}
    del ds, store, mover
    torch.cuda.empty_cache()
    return out


def traffic_from_profile(kind):
    """HBM bytes per launch from the committed counter summary, if it was
    taken with the kernel source as it is now; else None."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    src = os.path.join(ROOT, "paper_2608_25523_amd", "csrc", "pfx_kernels.hip")
    try:
        rec = json.load(open(path))
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != digest:
        return None
    return rec.get(kind, {}).get("bytes_per_step")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--replicas", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-extend", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="skip configs 1, 4 and 5 (about a minute)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip prefix movement, the rebuild of a preempted request and the service tables")
    ap.add_argument("--more", action="store_true", help="accepted for older command lines; the extras run by default")
    ap.add_argument("--no-engines", action="store_true",
                    help="skip the prefix-phase comparison of the two decode engines (counter passes over the rest)")
    ap.add_argument("--engines-only", action="store_true",
                    help="only the prefix-phase comparison of the two decode engines (for counter passes)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a 1 GiB device copy (counter calibration for rocprofv3 --pmc runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}), flush=True)
        sys.exit(2)

    import torch

    from paper_2608_25523_amd import binding as B
    from paper_2608_25523_amd import runner as RN
    from paper_2608_25523_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.engines_only:
        print(json.dumps({"prefix_phase_engines": bench_prefix_engines(args, torch, B, RN, W)}), flush=True)
        return
    if args.calib_copy:
        log(f"calibration copy: {copy_calibration(torch, B)} bytes moved per launch")
    copy_gbs = measured_copy_peak(torch, B)
    log(f"measured device page copy: {copy_gbs:.0f} GB/s (read + write)")
    log("decode-8B: building inputs")
    dec = bench_decode(args, torch, B, RN, W)
    log(f"decode-8B: {dec['ms'] * 1e3:.1f} us/step, attention {dec['attn_ms'] * 1e3:.1f} us "
        f"(vector-ALU engine {dec['valu_ms'] * 1e3:.1f} us)")
    ext = None
    if not args.no_extend:
        log("extend-8B: building inputs")
        ext = bench_extend(args, torch, B, RN, W)
        log(f"extend-8B: {ext['ms']:.3f} ms/step, attention {ext['attn_ms']:.3f} ms, "
            f"append {ext['append_ms']:.3f} ms")
    engines = None
    if not args.no_engines:
        log("decode-8B prefix phase on both decode engines")
        engines = bench_prefix_engines(args, torch, B, RN, W)
        log(f"prefix phase: MFMA {engines['mfma']['attn_us']} us, VALU {engines['valu']['attn_us']} us")
    configs = None
    if not args.no_configs:
        log("configs 1, 4, 5")
        configs = bench_configs(torch, B, RN, W, cpu=not args.no_cpu)
        log(f"config4 decode {configs['config4']['decode_attn_us']} us; config5 "
            f"decode {configs['config5']['decode']['ms_80_layers']} ms, extend "
            f"{configs['config5']['extend']['ms_80_layers']} ms (80 layers)")
    extras = None
    if not args.no_extras:
        log("movement, rebuild, service tables")
        extras = bench_extras(torch, B, RN, W)
    cpu = cpu_ext = None
    if not args.no_cpu:
        log("cpu baseline (oracle): decode-8B")
        cpu = cpu_baseline(dec, W)
        if ext is not None:
            log("cpu baseline (oracle): extend-8B")
            cpu_ext = cpu_baseline_extend(ext, W)

    u = dec["unique_bytes"]
    value = u / (dec["ms"] * 1e-3) / 1e9
    achieved = u / (dec["attn_ms"] * 1e-3) / 1e9
    st = dec["stats"]
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dec["ms"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16; lengths per the workload recipe)",
        "config": {"workload": "decode-8B: Hq32/Hkv8/d128, 4 prefixes x 2048, 64 decode reqs (16/agent, "
                               "suffix U[64,512]), 65536-page pool, random placement",
                   "unique_kv_bytes": u, "replicas": dec["replicas"], "prefix_items": st.num_prefix_items,
                   "suffix_items": st.num_suffix_items, "decode_steps": st.num_decode_steps,
                   "decode_pieces": st.num_decode_pieces},
        "roofline": {"bound": "hbm", "kernel": "pfx_attention: decode_kernel + merge_rows_kernel",
                     "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic_from_profile("decode"),
                     "measured_peak": round(copy_gbs, 1), "frac_measured": round(achieved / copy_gbs, 4),
                     "measured_peak_kind": "pfx_page_copy device to device, random 32 KiB pages, read + write",
                     "attn_us": round(dec["attn_ms"] * 1e3, 3), "attn_calls": dec["spread"]["calls"],
                     "attn_us_p10_p50_p90": [round(dec["spread"][k] * 1e3, 3) for k in ("p10", "p50", "p90")]},
        "decode_valu_engine": {
            "kernel": "pfx_attention with decode_engine = PFX_DECODE_VALU: decode_kernel on v_dot2_f32_bf16 "
                      "+ merge_rows_kernel",
            "attn_us": round(dec["valu_ms"] * 1e3, 3), "calls": dec["valu_spread"]["calls"],
            "GBs": round(u / (dec["valu_ms"] * 1e-3) / 1e9, 2),
            "frac": round(u / (dec["valu_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "vs_mfma": round(dec["valu_ms"] / dec["attn_ms"], 3)},
        "prefix_phase_engines": engines,
        "graph_ms_per_step": None if dec["graph_ms"] is None else round(dec["graph_ms"], 5),
        "step_parts": dec["side"],
        "cpu_baseline": cpu,
    }
    if ext is not None:
        tf = ext["flops"] / (ext["attn_ms"] * 1e-3) / 1e12
        out["extend"] = {
            "workload": "extend-8B: Hq32/Hkv8/d128, 3 prefixes x 4096, 32 reqs suffix U[256,2048]",
            "value": round(ext["flops"] / (ext["ms"] * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
            "ms_per_step": round(ext["ms"], 4), "steps": ext["steps"], "append_ms": round(ext["append_ms"], 4),
            "roofline": {"bound": "mfma", "kernel": "pfx_attention: extend_kernel", "achieved": round(tf, 2),
                         "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / BF16_PEAK_TFLOPS, 4),
                         "traffic": traffic_from_profile("extend"), "flops": ext["flops"],
                         "attn_ms": round(ext["attn_ms"], 4), "attn_calls": ext["spread"]["calls"],
                         "attn_ms_p10_p50_p90": [round(ext["spread"][k], 4) for k in ("p10", "p50", "p90")]},
            "cpu_baseline": cpu_ext,
        }
    if configs is not None:
        out.update(configs)
    if extras is not None:
        out["extras"] = extras
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
