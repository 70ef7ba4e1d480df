"""Closed-form statement of the deficit token-budget rule (Sangam paper,
Sec. 4.1, Alg. 1), one iteration at a time.

TEST INFRASTRUCTURE ONLY: the tests use it to check the library's native
admission; nothing on the product path imports it.

It restates what the rule decides rather than walking the queue step by
step. Let B = tau - D_t + S_{t-1} be the iteration's prefill budget (D_t the
tokens of the decodes, which are always seated; S_{t-1} the carried
deficit), and c_k the token count of the first k waiting prefills in arrival
order (c_0 = 0; prefills are indivisible and each holds at least one token,
so c_k grows strictly with k). Then:

  - with no prefill waiting, nothing is admitted and the carry becomes 0;
  - the admitted prefills are the longest head of the queue that fits the
    budget: k* = max{k : c_k <= B} (0 when B < 0);
  - a microbatch holding no decode takes the head prefill even when it does
    not fit (so that a prefill larger than tau is served): k* >= 1 then;
  - the carry is what the budget leaves, floored at zero: max(B - c_{k*}, 0).
"""
from typing import Sequence, Tuple

import numpy as np


def admit(tau: int, decode_tokens: Sequence[int], waiting: Sequence[int],
          deficit: int) -> Tuple[int, int]:
    """One iteration: returns (number of head prefills admitted, new deficit).
    decode_tokens lists the in-flight decodes' token counts."""
    if len(waiting) == 0:
        return 0, 0
    budget = int(tau) - int(np.sum(np.asarray(decode_tokens, np.int64))) + int(deficit)
    prefix = np.concatenate([[0], np.cumsum(np.asarray(waiting, np.int64))])
    k = int(np.searchsorted(prefix, budget, side="right")) - 1  # largest k with prefix[k] <= budget
    k = max(k, 0)
    if len(decode_tokens) == 0:
        k = max(k, 1)
    return k, max(budget - int(prefix[k]), 0)
