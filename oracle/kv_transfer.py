"""Paged-KV export / import written out as plain gathers and scatters, one
request and one position at a time (Sangam paper, Sec. 4.3 and its hybrid
architecture figure: a prefill worker's KV is handed to a decode-role worker;
Sec. 5: the cache is paged, page size 16, and moved over torch.distributed).

TEST INFRASTRUCTURE ONLY: the tests and the benchmark's CPU-baseline leg use
it; nothing on the product path imports it.

Definitions (bf16 values are handled as their uint16 bit patterns, so every
result is exact):
  position p of request i lives in page page_ids[page_indptr[i] + p // 16],
  slot p % 16, of a pool [pages, Hkv, 16, D];
  the packed buffers are [sum L_i, Hkv, D]; position p of request i is row
  kv_indptr[i] + p, kv_indptr the exclusive prefix sum of kv_len.
  export: packed row of (i, p) <- pool (page(i, p), :, slot(p), :)
  import: pool (page(i, p), :, slot(p), :) <- packed row of (i, p)
Positions p >= L_i do not exist: import leaves those slots of the last page,
and every page no request lists, as they were.
"""
from typing import Sequence, Tuple

import numpy as np

PAGE = 16


def kv_indptr(kv_len: Sequence[int]) -> np.ndarray:
    out = np.zeros(len(kv_len) + 1, np.int64)
    out[1:] = np.cumsum(np.asarray(kv_len, np.int64))
    return out


def _place(i: int, p: int, page_indptr, page_ids) -> Tuple[int, int]:
    """(page, slot) of position p of request i."""
    return int(page_ids[page_indptr[i] + p // PAGE]), p % PAGE


def export(pool_k: np.ndarray, pool_v: np.ndarray, kv_len, page_indptr, page_ids) -> Tuple[np.ndarray, np.ndarray]:
    """The packed K and V of the listed requests."""
    ind = kv_indptr(kv_len)
    rows = int(ind[-1])
    k = np.empty((rows,) + pool_k.shape[1:2] + pool_k.shape[3:], pool_k.dtype)
    v = np.empty_like(k)
    for i, L in enumerate(kv_len):
        for p in range(int(L)):
            page, slot = _place(i, p, page_indptr, page_ids)
            k[ind[i] + p] = pool_k[page, :, slot, :]
            v[ind[i] + p] = pool_v[page, :, slot, :]
    return k, v


def import_(k_packed: np.ndarray, v_packed: np.ndarray, pool_k: np.ndarray, pool_v: np.ndarray, kv_len,
            page_indptr, page_ids) -> Tuple[np.ndarray, np.ndarray]:
    """Copies of the pools after the packed rows are written into them."""
    ind = kv_indptr(kv_len)
    pk, pv = pool_k.copy(), pool_v.copy()
    for i, L in enumerate(kv_len):
        for p in range(int(L)):
            page, slot = _place(i, p, page_indptr, page_ids)
            pk[page, :, slot, :] = k_packed[ind[i] + p]
            pv[page, :, slot, :] = v_packed[ind[i] + p]
    return pk, pv
