"""Preemption and re-admission on the same kernels (Sec. 4.2, Eq. (9) and the
paragraph before it: a preempted request's generated-token KV is discarded
and rebuilt by decoding it again).  Four requests of one agent (8B layer
shape) decode 24 tokens after a 200-token prompt; then request 0's generated
slots are overwritten and rebuilt, once by replaying its 24 decode steps
alone and once by a single extend call over the 24 tokens.

Pins: pool pages equal the oracle's append of every token, bit for bit,
after the original run and after each rebuild; the replayed decode steps
give request 0 the same outputs bit for bit (a column's scores, softmax and
merge never depend on the other columns of its step); the extend rebuild
matches the oracle within the stated tolerances."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_25523_amd import binding as B
from paper_2608_25523_amd import runner as RN
from paper_2608_25523_amd import workloads as W

pytestmark = pytest.mark.gpu

P, L0, Y, R = 2048, 200, 24, 4


def announce(msg):
    print(f"[gpu-test] {msg}", flush=True)


def step(pool, batch, k_rows, v_rows, q_rows, mode):
    """Append the batch's new tokens and run attention; returns (o bits, lse)."""
    plan = B.plan_from_batch(pool, batch, mode).upload()
    t = batch.num_tokens
    B.pfx_append_kv(pool, plan, RN.to_device_bits(k_rows), RN.to_device_bits(v_rows))
    o = torch.empty((t, batch.num_q_heads, batch.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((t, batch.num_q_heads), dtype=torch.float32, device="cuda")
    B.pfx_attention(pool, plan, RN.to_device_bits(q_rows), o, lse)
    B.pfx_sync_check()
    return RN.to_host_bits(o), lse.cpu().numpy()


@pytest.mark.timeout(300)
def test_preempted_request_rebuilt_by_decode_and_by_extend():
    announce(f"rebuild: 4 requests, prefix {P}, prompt {L0}, {Y} generated tokens; request 0 rebuilt twice")
    full = W.make_batch(4040, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=1024, prefix_len=[P],
                        agent=[0] * R, suffix_len=[L0 + Y] * R, n_rows=[L0 + Y] * R)
    hv = W.host_values_fast(full, 4041)          # every token's K/V: k_new row r * (L0 + Y) + t
    ds = RN.DeviceStep(full, hv)                 # prefix written, suffix slots poisoned
    hq, hkv, d = full.num_q_heads, full.num_kv_heads, full.head_dim
    rows = lambda r, t0, t1: np.arange(r * (L0 + Y) + t0, r * (L0 + Y) + t1)
    rng = np.random.Generator(np.random.PCG64(4042))
    q_steps = [W.bf16_round(rng.standard_normal((R, hq, d), dtype=np.float32)) for _ in range(Y)]

    # The prompts, then Y decode steps for all four requests.
    prompt = W.with_lengths(full, [L0] * R, [L0] * R)
    idx = np.concatenate([rows(r, 0, L0) for r in range(R)])
    step(ds.pool, prompt, hv.k_new[idx], hv.v_new[idx], hv.q[idx], B.PFX_MODE_EXTEND)
    out = []
    for k in range(Y):
        sb = W.with_lengths(full, [L0 + k + 1] * R, [1] * R)
        idx = np.array([r * (L0 + Y) + L0 + k for r in range(R)])
        out.append(step(ds.pool, sb, hv.k_new[idx], hv.v_new[idx], q_steps[k], B.PFX_MODE_DECODE))
    want_k, want_v = oracle.append_kv(hv.k_pages, hv.v_pages, [np.array([list(hv.pages).index(p) for p in sp])
                                                                for sp in full.suffix_pages],
                                      full.suffix_len, full.n_rows, hv.k_new, hv.v_new)
    gk, gv = ds.read_pages(hv.pages)
    assert np.array_equal(gk, want_k) and np.array_equal(gv, want_v), "pool after the original run"

    # Preempt request 0: its generated slots are reused.
    gen = [(int(full.suffix_pages[0][(L0 + k) // 16]), (L0 + k) % 16) for k in range(Y)]
    pg = torch.tensor([p for p, _ in gen], device="cuda")
    sl = torch.tensor([s for _, s in gen], device="cuda")

    def wipe():
        ds.k_pool.view(torch.int16)[pg, :, sl, :] = W.POISON_BF16
        ds.v_pool.view(torch.int16)[pg, :, sl, :] = W.POISON_BF16

    # Rebuild 1: replay request 0's decode steps alone.
    wipe()
    for k in range(Y):
        sb = W.with_lengths(full, [L0 + k + 1] + [L0 + Y] * (R - 1), [1] + [0] * (R - 1))
        o, lse = step(ds.pool, sb, hv.k_new[[L0 + k]], hv.v_new[[L0 + k]], q_steps[k][:1], B.PFX_MODE_DECODE)
        assert np.array_equal(o[0], out[k][0][0]), f"replayed decode step {k} differs"
        assert np.array_equal(lse[0], out[k][1][0])
    gk, gv = ds.read_pages(hv.pages)
    assert np.array_equal(gk, want_k) and np.array_equal(gv, want_v), "pool after the decode rebuild"

    # Rebuild 2: one extend call over the Y tokens.
    wipe()
    sb = W.with_lengths(full, [L0 + Y] * R, [Y] + [0] * (R - 1))
    qy = np.stack([q_steps[k][0] for k in range(Y)])
    o, lse = step(ds.pool, sb, hv.k_new[rows(0, L0, L0 + Y)], hv.v_new[rows(0, L0, L0 + Y)], qy, B.PFX_MODE_EXTEND)
    gk, gv = ds.read_pages(hv.pages)
    assert np.array_equal(gk, want_k) and np.array_equal(gv, want_v), "pool after the extend rebuild"
    index = {int(p): i for i, p in enumerate(hv.pages)}
    pp = [np.array([index[int(p)] for p in pl]) for pl in sb.prefix_pages]
    sp = [np.array([index[int(p)] for p in pl]) for pl in sb.suffix_pages]
    ro, rl = oracle.prefix_shared_attention(want_k, want_v, pp, sb.prefix_len, sb.agent, sp, sb.suffix_len,
                                            sb.n_rows, qy, hq)
    got = oracle.bf16_bits_to_f64(o)
    assert np.max(np.abs(got - ro)) <= 1e-2
    assert np.linalg.norm(got - ro) <= 2e-2 * np.linalg.norm(ro)
    assert np.max(np.abs(lse - rl)) <= 1e-2
    announce("rebuild: decode replay bit-identical, extend rebuild within tolerance, pages bit-exact")
