"""ctypes binding of the fp64 CPU oracle (``attn_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg use it; the product path never imports it. It reads the
logical, unpaged per-item arrays that ``workloads.py`` draws and never the
page table.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Iterable, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "attn_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP). Always recompiles when force."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra",
               "-o", tmp, SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=True)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        L.oracle_attn.argtypes = [i32, i32, i32, i32, f32, P, P, P, P, P, P, P, P, P, P, P, i64, P, P]
        L.oracle_attn.restype = ctypes.c_int
        L.oracle_weights.argtypes = [i32, i32, i32, i32, f32, P, P, P, P, P, P, P, P, P, P, i64, i32, P]
        L.oracle_weights.restype = ctypes.c_int
        L.oracle_expected_kv.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, P, i32, P, P]
        L.oracle_expected_kv.restype = ctypes.c_int
        L.oracle_threads.argtypes = [ctypes.c_int]
        L.oracle_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def threads(n: int = 0) -> int:
    return lib().oracle_threads(n)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _bits(t) -> np.ndarray:
    """bf16 torch tensor -> contiguous uint16 numpy array of its bit patterns."""
    import torch
    return np.ascontiguousarray(t.contiguous().view(torch.int16).numpy().view(np.uint16))


class Call:
    """Packed arrays of one oracle call (a subset of a workload's items)."""

    def __init__(self, wl, items: Optional[Sequence[int]] = None, heads: Optional[Sequence[int]] = None):
        """heads: optional query heads; the call then holds only those (in that
        order), each paired with its own copy of its KV head g = h // G
        (G = 1 in the reduced call), so every (row, head) result is the one
        of the full call, without drawing the other heads' values."""
        self.items = list(range(wl.num_items)) if items is None else list(items)
        self.hq, self.hkv, self.d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
        qh = kvh = None
        if heads is not None:
            G = wl.num_q_heads // wl.num_kv_heads
            qh = [int(h) for h in heads]
            kvh = [h // G for h in qh]
            self.hq = self.hkv = len(qh)
        self.sm_scale = wl.sm_scale
        n = [wl.n(i) for i in self.items]
        self.q_indptr = np.zeros(len(n) + 1, np.int32)
        self.q_indptr[1:] = np.cumsum(n)
        self.q_offset = np.asarray([wl.q_offset[i] for i in self.items], np.int32)
        # per-row positions (None: rows of item i sit at q_offset[i] + r)
        self.q_pos = None
        if getattr(wl, "q_pos", None) is not None:
            self.q_pos = np.concatenate([wl.positions(i) for i in self.items]).astype(np.int32)
        self.kv_len = np.asarray([wl.kv_len[i] for i in self.items], np.int32)
        z = np.zeros((0,), np.uint16)
        empty = (lambda: z)
        self.q = np.concatenate([_bits(wl.q(i, heads=qh)).reshape(-1) for i in self.items] or [empty()])
        self.k_new = np.concatenate([_bits(wl.k_new(i, heads=kvh)).reshape(-1) for i in self.items] or [empty()])
        self.v_new = np.concatenate([_bits(wl.v_new(i, heads=kvh)).reshape(-1) for i in self.items] or [empty()])
        kc, vc, ctx = [], [], [0]
        for i in self.items:
            k = wl.k_ctx(i, heads=kvh)
            if k is None:
                ctx.append(ctx[-1])
                continue
            kc.append(_bits(k).reshape(-1))
            vc.append(_bits(wl.v_ctx(i, heads=kvh)).reshape(-1))
            ctx.append(ctx[-1] + int(wl.kv_len[i]))
        self.ctx_indptr = np.asarray(ctx, np.int64)
        self.k_ctx = np.concatenate(kc) if kc else np.zeros((1,), np.uint16)
        self.v_ctx = np.concatenate(vc) if vc else np.zeros((1,), np.uint16)

    def args(self):
        return (len(self.items), self.hq, self.hkv, self.d, ctypes.c_float(self.sm_scale),
                _ptr(self.q_indptr), _ptr(self.q_offset), _ptr(self.q_pos), _ptr(self.kv_len),
                _ptr(self.ctx_indptr),
                _ptr(self.q), _ptr(self.k_new), _ptr(self.v_new), _ptr(self.k_ctx), _ptr(self.v_ctx))


def selection(call: Call, rows: Optional[Dict[int, Iterable[int]]] = None,
              heads: Optional[Sequence[int]] = None):
    """(row, head) pair list of a call: per item its chosen local rows (default
    all) and heads (default all). Returns (sel array, {item: (rows, base)}, heads)."""
    hq = call.hq
    hs = list(range(hq)) if heads is None else list(heads)
    sel, layout = [], {}
    for k, i in enumerate(call.items):
        n = int(call.q_indptr[k + 1] - call.q_indptr[k])
        rr = np.arange(n) if rows is None or i not in rows else np.asarray(list(rows[i]), np.int64)
        base = len(sel)
        for r in rr:
            for h in hs:
                sel.append((int(call.q_indptr[k]) + int(r)) * hq + h)
        layout[i] = (rr, base)
    return np.asarray(sel, np.int64), layout, hs


def run(call: Call, sel: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """The C oracle over prepared arrays: out [len(sel), D], lse [len(sel)]."""
    out = np.empty((len(sel), call.d), np.float64)
    lse = np.empty((len(sel),), np.float64)
    rc = lib().oracle_attn(*call.args(), _ptr(sel), len(sel), _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError(f"oracle_attn rejected the call (code {rc})")
    return out, lse


def attention(wl, items: Optional[Sequence[int]] = None,
              rows: Optional[Dict[int, Iterable[int]]] = None,
              heads: Optional[Sequence[int]] = None) -> Dict[int, Tuple[np.ndarray, np.ndarray, np.ndarray]]:
    """fp64 attention for the chosen items.

    rows: optional {item: local row indices}; default every row.
    heads: optional list of query heads; default all.
    Returns {item: (local_rows, out [len(rows), len(heads), D], lse [len(rows), len(heads)])}.
    """
    # only the chosen heads' values are drawn (the reduced call holds them in order)
    call = Call(wl, items, heads=heads)
    sel, layout, hs = selection(call, rows, None)
    out, lse = run(call, sel)
    res = {}
    for i, (rr, base) in layout.items():
        cnt = len(rr) * len(hs)
        res[i] = (rr, out[base:base + cnt].reshape(len(rr), len(hs), call.d),
                  lse[base:base + cnt].reshape(len(rr), len(hs)))
    return res


def attention_all(wl) -> Tuple[np.ndarray, np.ndarray]:
    """Every row and head of the call: out [sum n, Hq, D], lse [sum n, Hq]."""
    call = Call(wl)
    T = int(call.q_indptr[-1])
    out = np.empty((T, call.hq, call.d), np.float64)
    lse = np.empty((T, call.hq), np.float64)
    rc = lib().oracle_attn(*call.args(), None, 0, _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError(f"oracle_attn rejected the call (code {rc})")
    return out, lse


def weights(wl, row: int, head: int) -> np.ndarray:
    """Normalized softmax weights of one packed row / head over its item's L keys."""
    call = Call(wl)
    T = int(call.q_indptr[-1])
    if not (0 <= row < T):
        raise IndexError(row)
    item = int(np.searchsorted(call.q_indptr, row, side="right") - 1)
    w = np.empty((int(call.kv_len[item]),), np.float64)
    rc = lib().oracle_weights(*call.args(), row, head, _ptr(w))
    if rc != 0:
        raise ValueError(f"oracle_weights rejected the call (code {rc})")
    return w


def expected_kv(wl, item: int) -> Tuple[np.ndarray, np.ndarray]:
    """Cache content of an item after the call: (k, v) uint16 bf16 bits [L, Hkv, D]."""
    call = Call(wl, [item])
    L = int(call.kv_len[0])
    k = np.empty((L, call.hkv, call.d), np.uint16)
    v = np.empty_like(k)
    rc = lib().oracle_expected_kv(1, call.hkv, call.d, _ptr(call.q_indptr), _ptr(call.q_offset),
                                  _ptr(call.q_pos), _ptr(call.kv_len), _ptr(call.ctx_indptr), _ptr(call.k_new),
                                  _ptr(call.v_new), _ptr(call.k_ctx), _ptr(call.v_ctx), 0,
                                  _ptr(k), _ptr(v))
    if rc != 0:
        raise ValueError(f"oracle_expected_kv rejected the call (code {rc})")
    return k, v
