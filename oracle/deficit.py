"""Plain Python transcription of the deficit token-budget rule (Sangam
paper, Sec. 4.1, Alg. 1), one iteration at a time.

TEST INFRASTRUCTURE ONLY: the tests use it to check the library's native
admission; nothing on the product path imports it.

The steps, in the algorithm's order:
  - no prefill waiting: decode-only iteration, the deficit is reset to 0;
  - budget = tau - Tokens(decodes) + deficit; the microbatch starts as the
    decodes (they are never displaced);
  - walk the waiting queue from its head (arrival order): the head is moved
    into the microbatch when its tokens fit the budget, or when the
    microbatch is still empty (the idle rule); otherwise the walk stops;
  - the deficit carried on is max(budget, 0).
"""
from typing import List, Sequence, Tuple


def admit(tau: int, decode_tokens: Sequence[int], waiting: Sequence[int],
          deficit: int) -> Tuple[int, int]:
    """One iteration: returns (number of head prefills admitted, new deficit).
    decode_tokens lists the in-flight decodes' token counts."""
    if len(waiting) == 0:
        return 0, 0
    budget = tau - sum(decode_tokens) + deficit
    microbatch: List[str] = ["decode"] * len(decode_tokens)
    queue = list(waiting)
    admitted = 0
    while queue:
        p = queue[0]
        idle = len(microbatch) == 0
        if p <= budget or idle:
            microbatch.append("prefill")
            queue.pop(0)
            budget -= p
            admitted += 1
        else:
            break
    return admitted, max(budget, 0)
