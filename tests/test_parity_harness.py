"""The parity harness on the CPU: the parallel oracle checker accepts the
oracle's own result rounded to bf16 and rejects planted errors, on all rows
and on sampled rows (no GPU involved)."""

from __future__ import annotations

import numpy as np
import pytest

import parity as PT
from paper_2608_25523_amd import workloads as W


def _case():
    b = W.make_batch(77, num_q_heads=8, num_kv_heads=2, head_dim=64, num_pages=128, prefix_len=[90, 40],
                     agent=[0, 1, -1, 0, 1], suffix_len=[30, 17, 12, 5, 40], n_rows=[30, 1, 12, 1, 3])
    hv = W.host_values(b, 78)
    kp, vp = PT.expected_pools(b, hv)
    o_ref, l_ref = PT.reference(b, hv, (kp, vp))
    o_bits = W.bf16_round(o_ref.astype(np.float32))
    return b, hv, kp, vp, o_bits, l_ref.astype(np.float32)


@pytest.fixture(scope="module")
def ck():
    c = PT.OracleChecker(workers=2)
    yield c
    c.close()


def test_checker_accepts_oracle_result(ck):
    b, hv, kp, vp, o_bits, lse = _case()
    rows = PT.all_rows(b)
    h = ck.submit(b, hv.pages, kp, vp, PT.gather_rows(hv.q, b, rows), PT.gather_rows(o_bits, b, rows),
                  PT.gather_rows(lse, b, rows), rows)
    max_abs, rel, lerr, n = ck.collect(h, "oracle vs itself")
    assert n == b.num_tokens and max_abs <= PT.MAX_ABS and lerr < 1e-5


@pytest.mark.parametrize("split", [True, False])
def test_checker_rejects_planted_errors(ck, split):
    b, hv, kp, vp, o_bits, lse = _case()
    rows = {0: [3, 29], 2: [0, 11], 4: [1]}
    bad = o_bits.copy()
    q_indptr = b.q_indptr()
    t = q_indptr[2] + 11
    bad[t, 5, 7] = W.bf16_round(np.float32(0.05) + np.float32(1.0))  # ~1 off at one element
    h = ck.submit(b, hv.pages, kp, vp, PT.gather_rows(hv.q, b, rows), PT.gather_rows(bad, b, rows),
                  PT.gather_rows(lse, b, rows), rows, split_heads=split)
    with pytest.raises(AssertionError, match="max-abs"):
        ck.collect(h, "planted O error")
    wrong_lse = lse.copy()
    wrong_lse[q_indptr[4] + 1, 3] += 0.05
    h = ck.submit(b, hv.pages, kp, vp, PT.gather_rows(hv.q, b, rows), PT.gather_rows(o_bits, b, rows),
                  PT.gather_rows(wrong_lse, b, rows), rows, split_heads=split)
    with pytest.raises(AssertionError, match="LSE"):
        ck.collect(h, "planted LSE error")


def test_checker_with_scale_and_no_lse(ck):
    b, hv, kp, vp, _, _ = _case()
    o_ref, _ = PT.reference(b, hv, (kp, vp), scale=0.3)
    o_bits = W.bf16_round(o_ref.astype(np.float32))
    rows = PT.all_rows(b)
    h = ck.submit(b, hv.pages, kp, vp, PT.gather_rows(hv.q, b, rows), PT.gather_rows(o_bits, b, rows), None,
                  rows, scale=0.3)
    ck.collect(h, "explicit scale")
    h = ck.submit(b, hv.pages, kp, vp, PT.gather_rows(hv.q, b, rows), PT.gather_rows(o_bits, b, rows), None,
                  rows, scale=0.2)
    with pytest.raises(AssertionError):
        ck.collect(h, "wrong scale")


def test_one_hot_values_select_one_value_row():
    """The planted one-hot queries: the oracle's every output row is one of
    the value rows of its KV head (the generator aimed q at one key)."""
    b, hv, *_ = _case()
    h2 = W.plant_one_hot(b, hv, 5, alpha_log2=4)
    kp, vp = PT.expected_pools(b, h2)
    o, _ = PT.reference(b, h2, (kp, vp))
    allv = PT.oracle.bf16_bits_to_f64(vp).transpose(1, 0, 2, 3).reshape(b.num_kv_heads, -1, b.head_dim)
    for t in range(o.shape[0]):
        for h in range(b.num_q_heads):
            assert np.nanmin(np.abs(allv[h // b.group] - o[t, h]).max(axis=1)) < 1e-9
