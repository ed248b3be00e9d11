"""Service-time uses (Sec. 4.2 after Eq. (4); Eq. (9)): the oracle pinned by
closed cases, and the product's table checked against the oracle on CPU
(the table is built from given numbers here; tests/test_gpu_service.py
measures one)."""

import pytest

from oracle import service as OS
from paper_2608_25523_amd import service as SV


def test_oracle_closed_cases():
    # no new tokens: the estimate is the prefill alone; no prefill cost: decode alone
    assert OS.fallback_estimate(lambda n: 3e-3, 2e-5, 1000, 0) == 3e-3
    assert OS.fallback_estimate(lambda n: 0.0, 2e-5, 1000, 250) == pytest.approx(5e-3)
    # nothing to rebuild discards nothing; rebuild work adds over requests
    assert OS.j_redo(2e-5, []) == 0.0
    assert OS.j_redo(2e-5, [10, 0, 30]) == pytest.approx(OS.j_redo(2e-5, [10]) + OS.j_redo(2e-5, [30]))


def test_table_interpolates_and_matches_oracle():
    tab = SV.ServiceTable({256: 1e-4, 1024: 4e-4, 4096: 2e-3}, t_decode=2.5e-5)
    assert tab.t_prefill(1024) == pytest.approx(4e-4)            # at a measured length
    assert tab.t_prefill(640) == pytest.approx(2.5e-4)           # halfway between 256 and 1024
    assert tab.t_prefill(8192) == pytest.approx(2e-3 + (8192 - 4096) * (2e-3 - 4e-4) / 3072)  # last segment extended
    for n, new in ((300, 0), (2048, 17), (5000, 400)):
        assert tab.estimate(n, new) == pytest.approx(OS.fallback_estimate(tab.t_prefill, 2.5e-5, n, new))
    assert tab.j_redo([5, 7]) == pytest.approx(OS.j_redo(2.5e-5, [5, 7]))
