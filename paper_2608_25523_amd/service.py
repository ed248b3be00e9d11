"""Service-time tables from this build's kernels.

The paper's scheduler estimates a request's LLM service, before it has
observations for the agent-stage pair, as T_prefill(|input|) +
T_decode * max_new (Sec. 4.2, the text after Eq. (4)), and charges the decode
work discarded by a preemption as T_decode times the tokens to rebuild
(Eq. (9)).  Both T's are profiled.  Here they are measured on the attention
path of one layer at a given shape: T_prefill(L) is one extend call for a
request of L new tokens over its agent's resident prefix, T_decode(B) one
decode step (one new token for each of B requests of one agent).  A model's
figure is the layer figure times its layer count plus the non-attention
work, which this library does not run.

Product side: the binding, the runner and the input generators only.
"""

from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from . import runner as RN
from . import workloads as W


def _time_call(fn, reps: int) -> float:
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / reps


def _step(prefix_len: int, suffix_len, n_rows, hq: int, hkv: int, d: int, seed: int) -> RN.DeviceStep:
    r = len(suffix_len)
    pages = (prefix_len + 15) // 16 + sum((int(l) + 15) // 16 for l in suffix_len) + 64
    b = W.make_batch(seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, num_pages=pages,
                     prefix_len=[prefix_len], agent=[0] * r, suffix_len=suffix_len, n_rows=n_rows)
    return RN.DeviceStep(b, W.host_values_fast(b, seed), poison=False)


def profile_prefill(lengths, prefix_len: int, hq: int = 32, hkv: int = 8, d: int = 128, reps: int = 5) -> dict:
    """T_prefill(L) in seconds: one extend call, L new tokens over the prefix."""
    out = {}
    for i, L in enumerate(lengths):
        ds = _step(prefix_len, [int(L)], [int(L)], hq, hkv, d, 500 + i)
        out[int(L)] = _time_call(lambda: B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse), reps)
        del ds
    return out


def profile_decode(batch_sizes, prefix_len: int, suffix_len: int, hq: int = 32, hkv: int = 8, d: int = 128,
                   reps: int = 20) -> dict:
    """T_decode(B) in seconds: one decode step for B requests of one agent,
    each with suffix_len tokens of its own (the new one included)."""
    out = {}
    for i, nb in enumerate(batch_sizes):
        ds = _step(prefix_len, [int(suffix_len)] * int(nb), [1] * int(nb), hq, hkv, d, 700 + i)
        out[int(nb)] = _time_call(lambda: B.pfx_attention(ds.pool, ds.plan, ds.q, ds.o, ds.lse), reps)
        del ds
    return out


class ServiceTable:
    """Measured T_prefill(L) and T_decode, with the two uses Sec. 4.2 makes
    of them.  T_prefill is interpolated linearly between measured lengths
    (and extended along the last segment); T_decode is one value."""

    def __init__(self, prefill: dict, t_decode: float):
        self.lengths = np.array(sorted(prefill), dtype=np.float64)
        self.times = np.array([prefill[k] for k in sorted(prefill)], dtype=np.float64)
        self.t_decode = float(t_decode)

    def t_prefill(self, length: float) -> float:
        x, y = self.lengths, self.times
        if len(x) == 1:
            return float(y[0] * length / x[0])
        j = int(np.clip(np.searchsorted(x, length) - 1, 0, len(x) - 2))
        return float(y[j] + (y[j + 1] - y[j]) * (length - x[j]) / (x[j + 1] - x[j]))

    def estimate(self, input_len: float, max_new: int) -> float:
        """Fallback service estimate: T_prefill(|input|) + T_decode * max_new."""
        return self.t_prefill(input_len) + self.t_decode * max_new

    def j_redo(self, rebuild_tokens) -> float:
        """Eq. (9): decode work discarded by preempting requests that must
        rebuild y_r generated tokens each."""
        return self.t_decode * float(np.sum(rebuild_tokens))
