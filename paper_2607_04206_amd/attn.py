"""Python face of the C ABI: the same two calls, plan and forward, over torch
tensors. Argument marshalling only: every step of the attention call runs in
the HIP kernels of libsangam_attn.so; PyTorch supplies device memory and the
stream."""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Tuple, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import AttnDesc, PlanInfo, SangamError, check, lib


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


@dataclass
class Plan:
    host: np.ndarray                 # uint8 blob (host)
    dev: Optional[torch.Tensor]      # the same bytes on the device (None before upload)
    info: PlanInfo
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    total_q: int
    num_pool_pages: int = 0  # pool size the plan's page ids were checked against
    total_pages: int = 0     # entries of page_ids the kernels read
    upload_stream: Optional[torch.cuda.Stream] = None  # the stream the device copy was issued on
    upload_done: Optional[torch.cuda.Event] = None     # recorded on it after the copy

    @property
    def workspace_bytes(self) -> int:
        return int(self.info.workspace_bytes)

    def host_ptr(self) -> int:
        return self.host.ctypes.data

    def item_splits(self, item: int):
        n = ctypes.c_int32(0)
        check(lib.sangam_plan_item_splits(self.host_ptr(), item, ctypes.byref(n), None, 0))
        starts = np.zeros(n.value + 1, np.int32)
        check(lib.sangam_plan_item_splits(self.host_ptr(), item, ctypes.byref(n),
                                          starts.ctypes.data, len(starts)))
        return starts

    def to(self, device) -> "Plan":
        """Copy the blob to device memory (the caller's H2D copy of plan_dev):
        staged through pinned host memory and copied without blocking on the
        device's current stream, after which an event is recorded there.
        Launches on that stream follow the copy; a forward on another stream
        waits for the event first. torch's pinned-memory pool keeps the
        staging buffer until the copy is done."""
        dev = torch.device(device)
        pinned = torch.from_numpy(self.host).pin_memory()
        self.dev = torch.empty(pinned.shape, dtype=pinned.dtype, device=dev)
        self.upload_stream = torch.cuda.current_stream(dev)
        self.dev.copy_(pinned, non_blocking=True)
        self.upload_done = torch.cuda.Event()
        self.upload_done.record(self.upload_stream)
        return self

    def order_after_upload(self, stream: torch.cuda.Stream) -> None:
        """Make `stream` wait for the plan's device copy when the copy was
        issued on another stream. Under graph capture nothing is waited for
        (a wait on an event recorded outside the capture is not allowed):
        the plan must then be resident before the capture starts, e.g. after
        a synchronisation or an eager call on the capturing stream."""
        if self.upload_done is None or stream == self.upload_stream:
            return
        if torch.cuda.is_current_stream_capturing():
            return
        stream.wait_event(self.upload_done)


def make_desc(*, q_indptr, q_offset, kv_len, page_indptr, page_ids, num_q_heads, num_kv_heads,
              head_dim, num_pool_pages, sm_scale, page_size=16, force_kv_splits=0, num_cus=0,
              q_pos=None):
    arrays = [_i32(x) for x in (q_indptr, q_offset, kv_len, page_indptr, page_ids)]
    if q_pos is not None:
        arrays.append(_i32(q_pos))
    d = AttnDesc()
    d.num_items = int(len(arrays[1]))
    d.num_q_heads = int(num_q_heads)
    d.num_kv_heads = int(num_kv_heads)
    d.head_dim = int(head_dim)
    d.page_size = int(page_size)
    d.force_kv_splits = int(force_kv_splits)
    d.num_pool_pages = int(num_pool_pages)
    d.sm_scale = float(np.float32(sm_scale))
    d.num_cus = int(num_cus)
    d.q_indptr, d.q_offset, d.kv_len, d.page_indptr, d.page_ids = (a.ctypes.data for a in arrays[:5])
    d.q_pos = arrays[5].ctypes.data if q_pos is not None else None
    return d, arrays  # keep arrays alive while d is used


_plan_cap = 1 << 16  # bytes of the first planning buffer; grows with the largest plan seen


def plan(*, q_indptr, q_offset, kv_len, page_indptr, page_ids, num_q_heads, num_kv_heads, head_dim,
         num_pool_pages, sm_scale, page_size=16, force_kv_splits=0, num_cus=0, q_pos=None,
         device=None) -> Plan:
    """sangam_attn_plan: validate the batch and build its launch plan (host only).
    q_pos: optional per-row positions (per-token cached decodes). With
    ``device`` the blob is also copied to that device."""
    d, keep = make_desc(q_indptr=q_indptr, q_offset=q_offset, kv_len=kv_len,
                        page_indptr=page_indptr, page_ids=page_ids, num_q_heads=num_q_heads,
                        num_kv_heads=num_kv_heads, head_dim=head_dim,
                        num_pool_pages=num_pool_pages, sm_scale=sm_scale, page_size=page_size,
                        force_kv_splits=force_kv_splits, num_cus=num_cus, q_pos=q_pos)
    global _plan_cap
    used = ctypes.c_size_t(0)
    # one planning pass in the common case: a buffer sized from earlier plans,
    # a second pass only when this batch needs more (-5: *used holds the size)
    buf = np.empty(_plan_cap, np.uint8)
    st = lib.sangam_attn_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used))
    if st == -5:
        _plan_cap = max(_plan_cap, 2 * int(used.value))
        buf = np.empty(int(used.value), np.uint8)
        st = lib.sangam_attn_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used))
    check(st)
    buf = buf[:int(used.value)].copy() if buf.nbytes > 4 * int(used.value) else buf[:int(used.value)]
    info = PlanInfo()
    check(lib.sangam_plan_get_info(buf.ctypes.data, ctypes.byref(info)))
    del keep
    p = Plan(host=buf, dev=None, info=info, num_q_heads=int(num_q_heads),
             num_kv_heads=int(num_kv_heads), head_dim=int(head_dim),
             total_q=int(info.total_q_rows), num_pool_pages=int(num_pool_pages),
             total_pages=int(_i32(page_indptr)[-1]))
    if device is not None:
        p.to(device)
    return p


def _need(t: torch.Tensor, name: str, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")


def c_args(p: Plan, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, k_cache: torch.Tensor,
           v_cache: torch.Tensor, page_ids: torch.Tensor, out: torch.Tensor, lse: Optional[torch.Tensor],
           workspace: Optional[torch.Tensor], stream) -> tuple:
    """The argument list of sangam_attn_forward for already checked tensors."""
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    return (p.host_ptr(), p.dev.data_ptr(), q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
            k_cache.data_ptr(), v_cache.data_ptr(), int(k_cache.shape[0]), page_ids.data_ptr(),
            int(page_ids.numel()), out.data_ptr(), lse.data_ptr() if lse is not None else None, ws_ptr,
            ws_len, stream.cuda_stream)


def forward(p: Plan, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
            k_cache: torch.Tensor, v_cache: torch.Tensor, page_ids: torch.Tensor,
            out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
            workspace: Optional[torch.Tensor] = None, want_lse: bool = True,
            stream: Optional[torch.cuda.Stream] = None,
            launch_events: Optional[Sequence[torch.cuda.Event]] = None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """sangam_attn_forward on the current (or given) stream. Allocates out,
    lse and the workspace with torch when they are not passed. With six
    timing events, calls sangam_attn_forward_timed instead: events 2k and
    2k + 1 travel in the dispatch of launch k (prefill-shaped, decode-shaped,
    merge), so their elapsed time is that kernel's execution alone."""
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("forward needs device tensors (a ROCm GPU)")
    T, Hq, Hkv, D = p.total_q, p.num_q_heads, p.num_kv_heads, p.head_dim
    _need(q, "q", torch.bfloat16, (T, Hq, D), dev)
    _need(k_new, "k_new", torch.bfloat16, (T, Hkv, D), dev)
    _need(v_new, "v_new", torch.bfloat16, (T, Hkv, D), dev)
    _need(k_cache, "k_cache", torch.bfloat16, None, dev)
    _need(v_cache, "v_cache", torch.bfloat16, tuple(k_cache.shape), dev)
    if k_cache.dim() != 4 or k_cache.shape[1] != Hkv or k_cache.shape[2] != 16 or k_cache.shape[3] != D:
        raise ValueError("k_cache must be [num_pool_pages, Hkv, 16, D]")
    if k_cache.shape[0] < p.num_pool_pages:
        raise ValueError(f"the plan addresses {p.num_pool_pages} pool pages, k_cache holds {k_cache.shape[0]}")
    _need(page_ids, "page_ids", torch.int32, None, dev)
    if page_ids.dim() != 1 or page_ids.numel() < p.total_pages:
        raise ValueError(f"page_ids must be a 1-D tensor of at least {p.total_pages} entries "
                         "(the plan's page table, on the device)")
    if p.dev is None or p.dev.device != dev:
        p.to(dev)
    if out is None:
        out = torch.empty((T, Hq, D), dtype=torch.bfloat16, device=dev)
    _need(out, "out", torch.bfloat16, (T, Hq, D), dev)
    if lse is None and want_lse:
        lse = torch.empty((T, Hq), dtype=torch.float32, device=dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, (T, Hq), dev)
    wsb = p.workspace_bytes
    if wsb > 0 and workspace is None:
        workspace = torch.empty((wsb,), dtype=torch.uint8, device=dev)
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    p.order_after_upload(s)
    args = c_args(p, q, k_new, v_new, k_cache, v_cache, page_ids, out, lse, workspace, s)
    if launch_events is None:
        check(lib.sangam_attn_forward(*args))
    else:
        if len(launch_events) != 6:
            raise ValueError("launch_events needs 6 events (start and stop of 3 launches)")
        evs = (ctypes.c_void_p * 6)(*[e.cuda_event for e in launch_events])
        check(lib.sangam_attn_forward_timed(*args, evs))
    return out, lse


def forward_noalloc(p: Plan, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                    k_cache: torch.Tensor, v_cache: torch.Tensor, page_ids: torch.Tensor,
                    out: torch.Tensor, lse: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """sangam_attn_forward_noalloc: the forward with split partials in the
    library's own device array, for callers that cannot allocate. out (and
    lse, when wanted) are the caller's; the plan must already be on the
    device (Plan.to) and its workspace within sangam_noalloc_scratch_bytes()."""
    dev = q.device
    T, Hq, Hkv, D = p.total_q, p.num_q_heads, p.num_kv_heads, p.head_dim
    _need(q, "q", torch.bfloat16, (T, Hq, D), dev)
    _need(k_new, "k_new", torch.bfloat16, (T, Hkv, D), dev)
    _need(v_new, "v_new", torch.bfloat16, (T, Hkv, D), dev)
    _need(k_cache, "k_cache", torch.bfloat16, None, dev)
    _need(v_cache, "v_cache", torch.bfloat16, tuple(k_cache.shape), dev)
    if k_cache.dim() != 4 or k_cache.shape[1] != Hkv or k_cache.shape[2] != 16 or k_cache.shape[3] != D:
        raise ValueError("k_cache must be [num_pool_pages, Hkv, 16, D]")
    _need(page_ids, "page_ids", torch.int32, None, dev)
    _need(out, "out", torch.bfloat16, (T, Hq, D), dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, (T, Hq), dev)
    if p.dev is None or p.dev.device != dev:
        raise ValueError("the plan is not on the device: call Plan.to(device) first")
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    p.order_after_upload(s)
    args = c_args(p, q, k_new, v_new, k_cache, v_cache, page_ids, out, lse, None, s)
    # the same arguments without the workspace pointer and size
    check(lib.sangam_attn_forward_noalloc(*args[:12], args[14]))
    return out, lse
