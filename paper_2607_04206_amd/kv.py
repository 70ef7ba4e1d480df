"""Python face of the paged-KV export / import (include/sangam_kv.h): plan,
export and import over torch tensors. Argument marshalling only: the copies
run in the HIP kernels of libsangam_attn.so."""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np
import torch

from . import _lib
from ._lib import KvDesc, check, lib


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


@dataclass
class KvPlan:
    host: np.ndarray             # uint8 blob (host)
    dev: Optional[torch.Tensor]  # the same bytes on the device
    rows: int                    # rows of the packed buffers (sum of L_i)
    num_kv_heads: int
    head_dim: int
    num_pool_pages: int

    def host_ptr(self) -> int:
        return self.host.ctypes.data

    def to(self, device) -> "KvPlan":
        self.dev = torch.from_numpy(self.host).to(device)
        return self


def plan(*, kv_len, page_indptr, page_ids, num_kv_heads, head_dim, num_pool_pages, page_size=16,
         device=None) -> KvPlan:
    """sangam_kv_plan: validate the batch and list its pages (host only)."""
    arrays = [_i32(x) for x in (kv_len, page_indptr, page_ids)]
    d = KvDesc()
    d.num_items = int(len(arrays[0]))
    d.num_kv_heads = int(num_kv_heads)
    d.head_dim = int(head_dim)
    d.page_size = int(page_size)
    d.num_pool_pages = int(num_pool_pages)
    d.kv_len, d.page_indptr, d.page_ids = (a.ctypes.data for a in arrays)
    used = ctypes.c_size_t(0)
    st = lib.sangam_kv_plan(ctypes.byref(d), None, 0, ctypes.byref(used))
    if st not in (_lib.SANGAM_OK, -5):  # -5: buffer too small, *used holds the size
        check(st)
    buf = np.zeros(int(used.value), np.uint8)
    check(lib.sangam_kv_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used)))
    del arrays
    p = KvPlan(host=buf, dev=None, rows=int(lib.sangam_kv_plan_rows(buf.ctypes.data)),
               num_kv_heads=int(num_kv_heads), head_dim=int(head_dim), num_pool_pages=int(num_pool_pages))
    if device is not None:
        p.to(device)
    return p


def _check_pool(p: KvPlan, t: torch.Tensor, name: str, dev) -> None:
    if not isinstance(t, torch.Tensor) or t.dtype != torch.bfloat16 or not t.is_contiguous() or t.device != dev:
        raise ValueError(f"{name} must be a contiguous bfloat16 tensor on {dev}")
    if tuple(t.shape) != (p.num_pool_pages, p.num_kv_heads, 16, p.head_dim):
        raise ValueError(f"{name} must be [{p.num_pool_pages}, {p.num_kv_heads}, 16, {p.head_dim}], "
                         f"got {tuple(t.shape)}")


def _check_packed(p: KvPlan, t: torch.Tensor, name: str, dev) -> None:
    if not isinstance(t, torch.Tensor) or t.dtype != torch.bfloat16 or not t.is_contiguous() or t.device != dev:
        raise ValueError(f"{name} must be a contiguous bfloat16 tensor on {dev}")
    if tuple(t.shape) != (p.rows, p.num_kv_heads, p.head_dim):
        raise ValueError(f"{name} must be [{p.rows}, {p.num_kv_heads}, {p.head_dim}], got {tuple(t.shape)}")


def _prep(p: KvPlan, dev, stream):
    if dev.type != "cuda":
        raise ValueError("the KV copies need device tensors (a ROCm GPU)")
    if p.dev is None or p.dev.device != dev:
        p.to(dev)
    return (stream if stream is not None else torch.cuda.current_stream(dev)).cuda_stream


def kv_export(p: KvPlan, k_cache: torch.Tensor, v_cache: torch.Tensor, k_packed: Optional[torch.Tensor] = None,
              v_packed: Optional[torch.Tensor] = None,
              stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """sangam_kv_export on the current (or given) stream; allocates the packed
    buffers with torch when they are not passed."""
    dev = k_cache.device
    _check_pool(p, k_cache, "k_cache", dev)
    _check_pool(p, v_cache, "v_cache", dev)
    shape = (p.rows, p.num_kv_heads, p.head_dim)
    if k_packed is None:
        k_packed = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    if v_packed is None:
        v_packed = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    _check_packed(p, k_packed, "k_packed", dev)
    _check_packed(p, v_packed, "v_packed", dev)
    s = _prep(p, dev, stream)
    check(lib.sangam_kv_export(p.host_ptr(), p.dev.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                               k_packed.data_ptr(), v_packed.data_ptr(), s))
    return k_packed, v_packed


def kv_import(p: KvPlan, k_packed: torch.Tensor, v_packed: torch.Tensor, k_cache: torch.Tensor,
              v_cache: torch.Tensor, stream: Optional[torch.cuda.Stream] = None) -> None:
    """sangam_kv_import on the current (or given) stream: writes the listed
    pages' slots [0, L_i) of k_cache / v_cache in place."""
    dev = k_cache.device
    _check_pool(p, k_cache, "k_cache", dev)
    _check_pool(p, v_cache, "v_cache", dev)
    _check_packed(p, k_packed, "k_packed", dev)
    _check_packed(p, v_packed, "v_packed", dev)
    s = _prep(p, dev, stream)
    check(lib.sangam_kv_import(p.host_ptr(), p.dev.data_ptr(), k_packed.data_ptr(), v_packed.data_ptr(),
                               k_cache.data_ptr(), v_cache.data_ptr(), s))
