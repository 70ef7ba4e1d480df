"""Binding of the deficit token-budget admission (include/sangam_sched.h)."""
from __future__ import annotations

import ctypes
from typing import Sequence, Tuple

import numpy as np

from ._lib import check, lib


def admit(tau: int, decode_tokens: int, num_decodes: int, waiting: Sequence[int],
          deficit: int) -> Tuple[int, int]:
    """sangam_deficit_admit: how many waiting prefills (from the head, in
    arrival order) join this iteration, and the deficit carried on."""
    w = np.ascontiguousarray(np.asarray(waiting, dtype=np.int64))
    d = ctypes.c_int64(int(deficit))
    n = ctypes.c_int32(0)
    check(lib.sangam_deficit_admit(int(tau), int(decode_tokens), int(num_decodes),
                                   w.ctypes.data if len(w) else None, len(w), ctypes.byref(d),
                                   ctypes.byref(n)))
    return int(n.value), int(d.value)
