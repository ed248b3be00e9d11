"""Shared helpers for GPU parity tests: run a step on the device, recompute it
with the fp64 oracle, and compare to the stated tolerances."""

from __future__ import annotations

import numpy as np

import oracle

# Tolerances for bf16 inputs with fp32 accumulation, bf16 output.
MAX_ABS = 1e-2       # every output element
REL_L2 = 2e-2        # ||O_gpu - O_ref||_2 / ||O_ref||_2, per request
LSE_ABS = 1e-2


def compact_ids(batch, pages):
    """Relabel page ids as indices into the compact page arrays."""
    index = {int(p): i for i, p in enumerate(pages)}
    pp = [np.array([index[int(p)] for p in pl], np.int64) for pl in batch.prefix_pages]
    sp = [np.array([index[int(p)] for p in pl], np.int64) for pl in batch.suffix_pages]
    return pp, sp


def expected_pools(batch, hv):
    """Oracle's pool contents (compact) after the step's append."""
    _, sp = compact_ids(batch, hv.pages)
    return oracle.append_kv(hv.k_pages, hv.v_pages, sp, batch.suffix_len, batch.n_rows, hv.k_new, hv.v_new)


def reference(batch, hv, pools=None, rows=None, scale=None):
    pp, sp = compact_ids(batch, hv.pages)
    kp, vp = pools if pools is not None else expected_pools(batch, hv)
    return oracle.prefix_shared_attention(kp, vp, pp, batch.prefix_len, batch.agent, sp, batch.suffix_len,
                                          batch.n_rows, hv.q, batch.num_q_heads, scale=scale, rows=rows)


def compare(batch, o_bits, lse, o_ref, lse_ref, label=""):
    """Check GPU outputs against the oracle on every row the oracle computed.
    Returns (max_abs, worst_rel, max_lse_err)."""
    o = oracle.bf16_bits_to_f64(o_bits)
    have = ~np.isnan(o_ref[:, 0, 0])
    assert have.any(), "no reference rows"
    assert not np.isnan(o[have]).any(), f"{label}: NaN in GPU output"
    assert not np.isnan(lse[have]).any(), f"{label}: NaN in GPU LSE"
    err = np.abs(o[have] - o_ref[have])
    max_abs = float(err.max())
    lse_err = float(np.abs(lse[have] - lse_ref[have]).max())
    worst_rel = 0.0
    q_indptr = batch.q_indptr()
    for r in range(len(batch.agent)):
        sl = slice(q_indptr[r], q_indptr[r + 1])
        m = have[sl]
        if not m.any():
            continue
        ref = o_ref[sl][m]
        rel = np.linalg.norm(o[sl][m] - ref) / max(np.linalg.norm(ref), 1e-30)
        worst_rel = max(worst_rel, float(rel))
    assert max_abs <= MAX_ABS, f"{label}: max-abs {max_abs:.3e}"
    assert worst_rel <= REL_L2, f"{label}: relative error {worst_rel:.3e}"
    assert lse_err <= LSE_ABS, f"{label}: LSE error {lse_err:.3e}"
    return max_abs, worst_rel, lse_err
