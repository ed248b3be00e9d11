"""Scheduling events executed through the library on the GPU.

Five tasks flow through an A -> B -> C workflow (one agent per stage, static
prefixes of 700, 1200 and 400 tokens at the 8B layer shape).  The KV budget
(1700 tokens) never holds the A and B prefixes together, so the scheduler
has to move prefixes.  At each event the product scheduler decides (and
must match the plain reference); the engine moves prefixes between the pool
and a pinned host store, releases preempted requests, prefills admitted
ones (their prompt plus any tokens they must rebuild) and runs one decode
step for every running request.  Every prefill and decode output is checked
against the fp64 attention oracle over the logical [prefix ; suffix]
sequence, and resident prefix pages must equal the original bits after any
number of round trips.
"""

from __future__ import annotations

import copy

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from oracle import scheduler as OS  # noqa: E402
from paper_2608_25523_amd import engine as EN  # noqa: E402
from paper_2608_25523_amd import runner as RN  # noqa: E402
from paper_2608_25523_amd import scheduler as S  # noqa: E402
from paper_2608_25523_amd import workflows as WF  # noqa: E402
from paper_2608_25523_amd import workloads as W  # noqa: E402
import parity as PT  # noqa: E402

pytestmark = pytest.mark.gpu

HQ, HKV, D = 32, 8, 128
PREFIX = [700, 1200, 400]
MAX_NEW = 3


def announce(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def draw(rng, shape):
    return W.bf16_round(rng.standard_normal(size=shape, dtype=np.float32))


def check(label, q_bits, o, lse, k_seq, v_seq, positions):
    """GPU rows against oracle.attend_rows over the logical sequence."""
    ro, rl = oracle.attend_rows(oracle.bf16_bits_to_f64(q_bits), oracle.bf16_bits_to_f64(k_seq),
                                oracle.bf16_bits_to_f64(v_seq), positions, HQ, 1.0 / np.sqrt(D))
    got = oracle.bf16_bits_to_f64(RN.to_host_bits(o))
    err = float(np.max(np.abs(got - ro)))
    rel = float(np.linalg.norm(got - ro) / np.linalg.norm(ro))
    lerr = float(np.max(np.abs(lse.cpu().numpy() - rl)))
    assert err <= PT.MAX_ABS and rel <= PT.REL_L2 and lerr <= PT.LSE_ABS, (label, err, rel, lerr)
    return err


def test_scheduling_events_through_the_library():
    rng = np.random.default_rng(909)
    prefixes = [(draw(rng, (l, HKV, D)), draw(rng, (l, HKV, D))) for l in PREFIX]
    eng = EN.Engine(512, HQ, HKV, D, prefixes)
    dag = WF.chain(3)
    params = S.Params(budget=1700.0, mu=HKV * D * 4, b_swap=4e6, t_decode=0.02, beta=0.5, rho=0.5, h_age=2.0)
    # Task state kept by the test: stage statuses, and per task its current request.
    tasks = [{"id": t, "arrival": float(t), "stages": [{"status": "ready" if v == 0 else "pending", "served": 0.0}
                                                       for v in range(3)]} for t in range(5)]
    reqs = {}
    toks = {}      # request -> (k bits, v bits) of every token it has produced so far (prompt, then decoded)
    nxt = [0]

    def new_request(t, stage):
        rid = nxt[0]
        nxt[0] += 1
        prompt = int(rng.integers(20, 60))
        reqs[rid] = {"id": rid, "task": t, "stage": stage, "prompt": prompt, "d": prompt + MAX_NEW,
                     "d_hat": 0.5 + 0.01 * prompt, "running": False, "generated": 0, "credit": 0.0}
        toks[rid] = (draw(rng, (prompt, HKV, D)), draw(rng, (prompt, HKV, D)))

    for t in range(5):
        new_request(t, 0)
    moved_events, completed = 0, 0
    for ev in range(14):
        live = [r for r in reqs.values() if tasks[r["task"]]["stages"][r["stage"]]["status"] != "done"]
        if not live:
            break
        sc = {"dag": dag, "prefix_len": PREFIX, "profiles": [[1.0, 1.5, 2.0]] * 3, "tasks": copy.deepcopy(tasks),
              "requests": [{k: r[k] for k in ("id", "task", "stage", "d", "d_hat", "running", "generated", "credit")}
                           for r in live],
              "resident": sorted(eng.resident), "now": 10.0 + ev}
        dec = S.decide(sc, params)
        ref = OS.hierarchical_search(copy.deepcopy(sc), params)
        assert list(dec.running) == ref["running"] and list(dec.resident) == ref["resident"], (ev, dec, ref)
        announce(f"event {ev}: resident {sorted(eng.resident)} -> {list(dec.resident)}, running {list(dec.running)}, "
                 f"admitted {dec.admitted}, preempted {list(dec.preempted)}, score {dec.score:.3f}")
        before = set(eng.resident)
        eng.apply(dec)
        if set(eng.resident) != before:
            moved_events += 1
        torch.cuda.synchronize()
        for a, pages in eng.resident.items():
            k, v = eng.read_pages(pages)
            n = PREFIX[a]
            kk = k.transpose(0, 2, 1, 3).reshape(-1, HKV, D)[:n]
            vv = v.transpose(0, 2, 1, 3).reshape(-1, HKV, D)[:n]
            assert np.array_equal(kk, prefixes[a][0]) and np.array_equal(vv, prefixes[a][1]), f"prefix {a} bits"
        for r in dec.preempted:
            reqs[r]["running"] = False
            reqs[r]["credit"] = 0.0
        for r in dec.admitted:
            q = reqs[r]
            a = dag["agent"][q["stage"]]
            q["running"], q["credit"] = True, dec.credits[r]
            tasks[q["task"]]["stages"][q["stage"]]["status"] = "running"
            # prefill: the prompt plus the tokens decoded before a preemption (rebuilt by extend)
            kt, vt = toks[r]
            n = kt.shape[0]
            qb = draw(rng, (n, HQ, D))
            o, lse = eng.prefill(r, a, RN.to_device_bits(qb), RN.to_device_bits(kt), RN.to_device_bits(vt))
            B_sync()
            check(f"event {ev} prefill {r}", qb, o, lse, np.concatenate([prefixes[a][0], kt]),
                  np.concatenate([prefixes[a][1], vt]), [PREFIX[a] + i for i in range(n)])
        run = list(dec.running)
        if run:
            qb = draw(rng, (len(run), HQ, D))
            kb, vb = draw(rng, (len(run), HKV, D)), draw(rng, (len(run), HKV, D))
            o, lse = eng.decode(run, RN.to_device_bits(qb), RN.to_device_bits(kb), RN.to_device_bits(vb))
            B_sync()
            for i, r in enumerate(run):
                a = dag["agent"][reqs[r]["stage"]]
                kt = np.concatenate([toks[r][0], kb[i:i + 1]])
                vt = np.concatenate([toks[r][1], vb[i:i + 1]])
                toks[r] = (kt, vt)
                check(f"event {ev} decode {r}", qb[i:i + 1], o[i:i + 1], lse[i:i + 1],
                      np.concatenate([prefixes[a][0], kt]), np.concatenate([prefixes[a][1], vt]),
                      [PREFIX[a] + kt.shape[0] - 1])
                reqs[r]["generated"] += 1
                if reqs[r]["generated"] >= MAX_NEW:
                    # the stage completes; the task's next stage becomes ready
                    q = reqs[r]
                    st = tasks[q["task"]]["stages"]
                    st[q["stage"]]["status"] = "done"
                    st[q["stage"]]["served"] = 0.0
                    q["running"] = False
                    eng.release(r)
                    completed += 1
                    if q["stage"] + 1 < 3:
                        st[q["stage"] + 1]["status"] = "ready"
                        new_request(q["task"], q["stage"] + 1)
    announce(f"events done: {completed} requests completed, {moved_events} events moved prefixes, "
             f"{eng.moved_tokens} prefix tokens moved")
    assert completed >= 5 and moved_events >= 1


def B_sync():
    from paper_2608_25523_amd import binding as B
    B.pfx_sync_check()
