"""Service estimates that the scheduler derives from profiled times.

TEST INFRASTRUCTURE ONLY: imported by tests, never by the product path.

Sec. 4.2, after Eq. (4): a request with no observations for its agent-stage
pair is estimated to need T_prefill(|input|) + T_decode * max_new of LLM
service.  Sec. 4.2, Eq. (9): preempting the requests P discards
sum over r in P of T_decode * y_r, y_r being the generated tokens that must be
rebuilt by decoding.
"""

from __future__ import annotations

from typing import Callable, Iterable


def fallback_estimate(t_prefill: Callable[[float], float], t_decode: float, input_len: float, max_new: int) -> float:
    return t_prefill(input_len) + t_decode * max_new


def j_redo(t_decode: float, rebuild_tokens: Iterable[int]) -> float:
    return sum(t_decode * y for y in rebuild_tokens)
