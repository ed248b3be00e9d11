"""Service-time tables measured on the GPU (Sec. 4.2: profiled T_prefill and
T_decode).  Properties the method fixes: prefill time grows with the input,
and one grouped decode step for 64 requests of an agent costs far less than
64 single-request steps, since the prefix is read once for the group."""

import pytest

from paper_2608_25523_amd import service as SV

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(300)
def test_service_tables():
    print("[gpu-test] service tables: prefill over a 4096-token prefix, decode steps over 2048", flush=True)
    pre = SV.profile_prefill([256, 1024, 4096], prefix_len=4096, reps=3)
    assert pre[256] < pre[1024] < pre[4096]
    dec = SV.profile_decode([1, 64], prefix_len=2048, suffix_len=288, reps=10)
    assert 0 < dec[1] and dec[64] < 16 * dec[1]
    tab = SV.ServiceTable(pre, dec[64])
    assert tab.estimate(1024, 100) == pytest.approx(pre[1024] + 100 * dec[64])
