"""The allocation-free entry point through the C interface on the GPU: its
outputs and pools equal those of pfx_append_kv + pfx_attention on the same
plan bit for bit, and the oracle's within the stated tolerances, on two calls
in a row (the second with a smaller batch, so the static array still holds
the first call's tables and partial states)."""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_25523_amd import binding as B  # noqa: E402
from paper_2608_25523_amd import runner as RN  # noqa: E402
from paper_2608_25523_amd import workloads as W  # noqa: E402
import parity as PT  # noqa: E402

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"\n[gpu-case] {msg}", flush=True)


def small(seed, hq, hkv, d, plen, reqs):
    return W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=512, prefix_len=plen,
                        agent=[r[0] for r in reqs], suffix_len=[r[1] for r in reqs], n_rows=[r[2] for r in reqs])


def one_call(batch, hv, label, with_append=True):
    announce(f"noalloc {label}: tokens={batch.num_tokens} reqs={len(batch.agent)} pool={batch.num_pages}")
    # Reference: the existing entry points, plan uploaded into a torch workspace.
    ref = RN.DeviceStep(batch, hv)
    ref.step()
    B.pfx_sync_check()
    o_ref, l_ref = ref.outputs()
    pk_ref, pv_ref = ref.read_pages(hv.pages)
    plan = ref.plan
    # Same initial pool and inputs, the allocation-free call (the plan's own
    # workspace is left alone).
    ds = RN.DeviceStep(batch, hv)
    if not with_append:
        ds.append()
    ds.o.zero_()
    ds.lse.fill_(float("nan"))
    torch.cuda.synchronize()
    B.pfx_attention_noalloc(ds.pool, plan, ds.q, ds.o, ds.lse,
                            k_new=ds.k_new if with_append else None, v_new=ds.v_new if with_append else None)
    B.pfx_sync_check()
    o, l = ds.outputs()
    pk, pv = ds.read_pages(hv.pages)
    assert np.array_equal(pk, pk_ref) and np.array_equal(pv, pv_ref), f"{label}: pools differ"
    assert np.array_equal(o, o_ref), f"{label}: O differs from pfx_attention's"
    assert np.array_equal(l, l_ref), f"{label}: LSE differs from pfx_attention's"
    exp_k, exp_v = PT.expected_pools(batch, hv)
    assert np.array_equal(pk, exp_k) and np.array_equal(pv, exp_v), f"{label}: pool differs from the oracle's"
    o_or, l_or = PT.reference(batch, hv, (exp_k, exp_v))
    res = PT.compare(batch, o, l, o_or, l_or, label)
    announce(f"noalloc {label}: bit-identical; oracle max_abs={res[0]:.2e} rel={res[1]:.2e}")


def test_noalloc_matches_existing_entry_points_twice():
    big = W.config_batch(2)                       # 640 decode pieces, 5.8 MB of tables + partial states
    one_call(big, W.host_values_fast(big, 2002), "decode-8B")
    smaller = small(12, 32, 8, 128, [100, 0, 37],
                    [(0, 70, 1), (2, 1, 1), (1, 40, 40), (0, 65, 1), (2, 17, 4), (-1, 31, 1)])
    one_call(smaller, W.host_values(smaller, 62), "small mixed")
    one_call(smaller, W.host_values(smaller, 63), "small mixed, attention only", with_append=False)


def test_noalloc_rejects_oversized_plan_before_running():
    b = W.make_batch(14, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=65536, prefix_len=[30000],
                     agent=[0] * 120, suffix_len=[40] * 120, n_rows=[1] * 120)
    hv = W.host_values_fast(b, 15)
    ds = RN.DeviceStep(b, hv)
    plan = B.plan_from_batch(ds.pool, b, B.PFX_MODE_DECODE, piece_steps=1)
    assert plan.workspace_bytes() > B.PFX_NOALLOC_MAX_WORKSPACE
    before = ds.read_pages(hv.pages)
    ds.o.zero_()
    with pytest.raises(B.PfxError) as e:
        B.pfx_attention_noalloc(ds.pool, plan, ds.q, ds.o, ds.lse, k_new=ds.k_new, v_new=ds.v_new)
    assert e.value.code == B.PFX_ENOMEM
    B.pfx_sync_check()
    after = ds.read_pages(hv.pages)
    assert all(np.array_equal(x, y) for x, y in zip(before, after)), "a rejected call wrote the pool"
    assert not ds.o.view(torch.int16).any(), "a rejected call wrote O"
