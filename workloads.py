"""Seeded synthetic workloads for the mixed block-decode / prefill attention call.

This module only draws inputs. It holds none of the attention arithmetic, so
both the fp64 oracle (``oracle/``) and the HIP path may use it.

Shapes follow the paper's setting: bf16 serving (Sec. 6.1), KV pages of 16
tokens and decode blocks of 32 positions (Sec. 6.1), prompts followed by the
whole appended masked response (Sec. 6.1, trace setup), LLaDA-8B (MHA) and
Dream-7B (GQA) head layouts (Sec. 6.1, Sec. 6.3). The paper's traces are not
used: prompt lengths are drawn from lognormals whose medians and spreads stand
in for Table 1.

Recipe (one for every workload):

1. ``numpy.random.default_rng(seed)`` draws, in this order, prompt lengths,
   decode block indices and the page permutation.
2. Prompt length ``P = clip(rint(exp(N(ln median, sigma))), lo, hi)``; context
   length ``L = P + R`` (R = appended response length).
3. A block decode at block index ``b`` has ``n = 32`` query rows at
   positions ``o = P + 32 b``; a prefill has ``o = 0``, ``n = L``.
4. Page ids are ``rng.permutation(pool)[:needed]``, handed out in item order.
5. Values come from a counter-based generator, so any piece can be drawn on
   the CPU or directly in device memory with identical bits: element ``c`` of
   piece (seed, item, kind) is ``T[(h(mul(c) + key) >> 8) & 0xFFFF]`` where
   ``h`` is the lowbias32 integer hash (C. Wellons, "Prospecting for hash
   functions", 2018), ``mul`` multiplies by an odd constant mod 2^32, ``key``
   hashes (seed, item, kind), and ``T`` holds the 65536 quantiles
   ``Phi^-1((i + 0.5) / 65536)`` of N(0, 1), rounded to bf16 (RNE). Only
   integer arithmetic runs per element, so CPU and GPU draws agree bit for
   bit. The bf16 bytes are the ground truth both sides read.
6. Batch order: decodes first, then prefills (the microbatch order of the
   deficit scheduler, Alg. 1).
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np
import torch

PAGE_SIZE = 16
BLOCK = 32

# kinds of value tensors, used to derive per-piece seeds
KIND_Q, KIND_KCTX, KIND_VCTX, KIND_KNEW, KIND_VNEW = range(5)


@dataclasses.dataclass
class Workload:
    """Descriptor of one attention call plus deterministic value generators."""

    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    q_indptr: np.ndarray  # int32 [n+1]
    q_offset: np.ndarray  # int32 [n]
    kv_len: np.ndarray  # int32 [n]
    is_prefill: np.ndarray  # bool [n]
    page_indptr: np.ndarray  # int32 [n+1]
    page_ids: np.ndarray  # int32 [page_indptr[-1]]
    num_pool_pages: int
    sm_scale: float  # float32 value
    q_scale: float = 1.0  # stress variant multiplies Q by this before rounding
    # optional overrides: item -> callable(kind) -> fp32 tensor
    value_fn: Optional[Callable[[int, int], torch.Tensor]] = None
    page_size: int = PAGE_SIZE
    # optional per-row positions, int32 [sum n]: row r of item i sits at
    # q_pos[q_indptr[i] + r] instead of q_offset[i] + r (per-token cached
    # decodes that recompute scattered positions)
    q_pos: Optional[np.ndarray] = None

    @property
    def num_items(self) -> int:
        return int(self.q_offset.shape[0])

    @property
    def total_q(self) -> int:
        return int(self.q_indptr[-1])

    def n(self, i: int) -> int:
        return int(self.q_indptr[i + 1] - self.q_indptr[i])

    def positions(self, i: int) -> np.ndarray:
        """Sequence positions of item i's rows (int64 [n_i])."""
        if self.q_pos is not None:
            return self.q_pos[self.q_indptr[i]:self.q_indptr[i + 1]].astype(np.int64)
        return np.arange(int(self.q_offset[i]), int(self.q_offset[i]) + self.n(i), dtype=np.int64)

    # ------------------------------------------------------------------ values
    def _draw(self, item: int, kind: int, shape: Tuple[int, ...], device="cpu",
              heads: Optional[Sequence[int]] = None) -> torch.Tensor:
        """Piece (item, kind) of shape [rows, H, D]; with ``heads``, only those
        entries of axis 1 ([rows, len(heads), D]), drawn without the others."""
        if self.value_fn is not None:
            t = self.value_fn(item, kind)
            if t is not None:
                assert tuple(t.shape) == tuple(shape), (t.shape, shape)
                if heads is not None:
                    t = t[:, list(heads)]
                return t.to(torch.bfloat16).to(device)
        scale = self.q_scale if kind == KIND_Q else 1.0
        if heads is None:
            return counter_normal_bf16(self.seed, item, kind, shape, device=device, scale=scale)
        return counter_normal_bf16_heads(self.seed, item, kind, shape, heads, device=device, scale=scale)

    def q(self, i: int, device="cpu", heads=None) -> torch.Tensor:
        """Query rows of item i, bf16 [n_i, Hq, D] (or only the listed heads)."""
        return self._draw(i, KIND_Q, (self.n(i), self.num_q_heads, self.head_dim), device, heads)

    def k_new(self, i: int, device="cpu", heads=None) -> torch.Tensor:
        """Fresh keys of item i (positions o_i .. o_i+n_i-1), bf16 [n_i, Hkv, D]."""
        return self._draw(i, KIND_KNEW, (self.n(i), self.num_kv_heads, self.head_dim), device, heads)

    def v_new(self, i: int, device="cpu", heads=None) -> torch.Tensor:
        return self._draw(i, KIND_VNEW, (self.n(i), self.num_kv_heads, self.head_dim), device, heads)

    def k_ctx(self, i: int, device="cpu", heads=None) -> Optional[torch.Tensor]:
        """Cache content before the call for positions [0, L_i), bf16 [L_i, Hkv, D].

        None for a prefill (it brings its whole sequence as fresh rows). Rows
        [o_i, o_i+n_i) hold stale values that the call must overwrite."""
        if self.is_prefill[i]:
            return None
        return self._draw(i, KIND_KCTX, (int(self.kv_len[i]), self.num_kv_heads, self.head_dim), device,
                          heads)

    def v_ctx(self, i: int, device="cpu", heads=None) -> Optional[torch.Tensor]:
        if self.is_prefill[i]:
            return None
        return self._draw(i, KIND_VCTX, (int(self.kv_len[i]), self.num_kv_heads, self.head_dim), device,
                          heads)

    # ------------------------------------------------------- packed views
    def packed_q(self, device="cpu") -> torch.Tensor:
        return torch.cat([self.q(i, device) for i in range(self.num_items)], 0)

    def packed_k_new(self, device="cpu") -> torch.Tensor:
        return torch.cat([self.k_new(i, device) for i in range(self.num_items)], 0)

    def packed_v_new(self, device="cpu") -> torch.Tensor:
        return torch.cat([self.v_new(i, device) for i in range(self.num_items)], 0)

    def item_pages(self, i: int) -> np.ndarray:
        return self.page_ids[self.page_indptr[i]:self.page_indptr[i + 1]]

    def fill_paged_cache(self, k_pool: torch.Tensor, v_pool: torch.Tensor, items=None) -> None:
        """Scatter each decode item's pre-call context into its pages.

        Pool layout [num_pool_pages, Hkv, page_size, D]: position p of item i
        lives in page page_ids[page_indptr[i] + p // page_size], slot
        p % page_size. Values are drawn on the pool's device. Slots >= L_i of
        an item's last page keep whatever the pool held."""
        S = self.page_size
        dev = k_pool.device
        for i in range(self.num_items) if items is None else items:
            if self.is_prefill[i]:
                continue
            L = int(self.kv_len[i])
            pages = torch.from_numpy(self.item_pages(i).astype(np.int64)).to(dev)
            npg = pages.numel()
            full = L // S  # whole pages
            for ctx, pool in ((self.k_ctx(i, dev), k_pool), (self.v_ctx(i, dev), v_pool)):
                if full:
                    blk = ctx[:full * S].view(full, S, self.num_kv_heads, self.head_dim)
                    pool[pages[:full]] = blk.permute(0, 2, 1, 3)
                r = L - full * S
                if r:
                    pool[pages[npg - 1], :, :r] = ctx[full * S:].permute(1, 0, 2)

    def flops(self) -> float:
        """Algorithmic flops: QK^T and PV, non-causal, 4*n*L*D*Hq per item."""
        n = np.diff(self.q_indptr).astype(np.float64)
        return float(np.sum(4.0 * n * self.kv_len.astype(np.float64) * self.head_dim * self.num_q_heads))

    def hbm_bytes(self) -> float:
        """Algorithmic HBM bytes: K and V read once per item, the cache write of
        the fresh rows, Q read, O write, page ids and the LSE write."""
        n = np.diff(self.q_indptr).astype(np.float64)
        L = self.kv_len.astype(np.float64)
        D, Hq, Hkv = self.head_dim, self.num_q_heads, self.num_kv_heads
        per = 2.0 * (2 * L * Hkv * D + 2 * n * Hkv * D + 2 * n * Hq * D)
        per += 4.0 * np.ceil(L / self.page_size) + 4.0 * n * Hq
        return float(np.sum(per))



# ------------------------------------------------------- counter generator
_M32 = 0xFFFFFFFF
_TABLES = {}


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for int64 tensors holding values < 2^32, without
    overflowing int64 (16-bit halves)."""
    lo = (x & 0xFFFF) * c
    hi = (((x >> 16) * c) & 0xFFFF) << 16
    return (lo + hi) & _M32


def _lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    return x ^ (x >> 16)


def _hash_u32_np(idx: np.ndarray, key: int) -> np.ndarray:
    """The same element hash as the torch path, on uint32 numpy arrays, whose
    multiplications wrap modulo 2^32 by themselves (host draws)."""
    with np.errstate(over="ignore"):
        x = idx.astype(np.uint32, copy=True)
        x *= np.uint32(0x27D4EB2F)
        x += np.uint32(key)
        x ^= x >> np.uint32(16)
        x *= np.uint32(0x7FEB352D)
        x ^= x >> np.uint32(15)
        x *= np.uint32(0x846CA68B)
        x ^= x >> np.uint32(16)
    return x


_HOST_POOL = None
_HOST_CHUNK = 1 << 18


def _draw_host(key: int, idx: np.ndarray, table: torch.Tensor) -> torch.Tensor:
    """Table entries at the hashed indices, drawn in parallel pieces (numpy
    releases the interpreter lock in its element loops)."""
    global _HOST_POOL
    bits = table.view(torch.int16).numpy()
    out = np.empty(idx.shape[0], np.int16)

    def piece(a, b):
        h = _hash_u32_np(idx[a:b], key)
        h >>= np.uint32(8)
        h &= np.uint32(0xFFFF)
        np.take(bits, h, out=out[a:b])

    n = idx.shape[0]
    if n <= _HOST_CHUNK:
        piece(0, n)
    else:
        if _HOST_POOL is None:
            from concurrent.futures import ThreadPoolExecutor
            _HOST_POOL = ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0))))
        list(_HOST_POOL.map(lambda a: piece(a, min(n, a + _HOST_CHUNK)), range(0, n, _HOST_CHUNK)))
    return torch.from_numpy(out).view(torch.bfloat16)


def normal_table(device="cpu", scale: float = 1.0) -> torch.Tensor:
    """65536 bf16 quantiles of N(0, 1) (times scale, before rounding)."""
    key = (str(device), float(scale))
    if key not in _TABLES:
        i = torch.arange(65536, dtype=torch.float64)
        t = torch.special.ndtri((i + 0.5) / 65536.0) * scale
        _TABLES[key] = t.to(torch.bfloat16).to(device)
    return _TABLES[key]


def piece_key(seed: int, item: int, kind: int) -> int:
    k = torch.tensor([(seed * 0x9E3779B1 + item * 0x85EBCA77 + kind * 0xC2B2AE3D) & _M32],
                     dtype=torch.int64)
    k = _lowbias32(_lowbias32(k) ^ ((seed >> 32) & _M32))
    return int(k.item())


def counter_normal_bf16(seed: int, item: int, kind: int, shape, device="cpu", scale: float = 1.0,
                        chunk: int = 1 << 24) -> torch.Tensor:
    """Element c of piece (seed, item, kind): T[(h(mul(c) + key) >> 8) & 0xFFFF]."""
    n = int(np.prod(shape)) if len(shape) else 1
    if n >= (1 << 32):
        raise ValueError("a piece must have fewer than 2^32 elements")
    key = piece_key(seed, item, kind)
    table = normal_table(device, scale)
    out = torch.empty(n, dtype=torch.bfloat16, device=device)
    host = torch.device(device).type == "cpu"
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        if host:
            out[c0:c1] = _draw_host(key, np.arange(c0, c1, dtype=np.uint32), table)
            continue
        idx = torch.arange(c0, c1, dtype=torch.int64, device=device)
        h = _lowbias32((_mul32(idx, 0x27D4EB2F) + key) & _M32)
        out[c0:c1] = table[(h >> 8) & 0xFFFF]
    return out.view(*shape)


def counter_normal_bf16_heads(seed: int, item: int, kind: int, shape, heads: Sequence[int], device="cpu",
                              scale: float = 1.0, chunk: int = 1 << 24) -> torch.Tensor:
    """The entries [:, heads, :] of piece (seed, item, kind) of shape [rows, H,
    D], drawn from their own counters (c = (row * H + h) * D + d) without the
    other heads: bitwise the same values as slicing the whole piece."""
    rows, H, D = (int(x) for x in shape)
    hs = torch.as_tensor(list(heads), dtype=torch.int64, device=device)
    if hs.numel() and (int(hs.min()) < 0 or int(hs.max()) >= H):
        raise IndexError("head out of range")
    if rows * H * D >= (1 << 32):
        raise ValueError("a piece must have fewer than 2^32 elements")
    key = piece_key(seed, item, kind)
    table = normal_table(device, scale)
    per_row = hs.numel() * D
    out = torch.empty(rows * per_row, dtype=torch.bfloat16, device=device)
    inner = (hs[:, None] * D + torch.arange(D, dtype=torch.int64, device=device)[None, :]).reshape(-1)
    step = max(1, chunk // max(per_row, 1))
    host = torch.device(device).type == "cpu"
    inner_np = inner.cpu().numpy().astype(np.uint32) if host else None
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        if host:
            idx_np = (np.arange(r0, r1, dtype=np.uint32)[:, None] * np.uint32(H * D) + inner_np[None, :]).reshape(-1)
            out[r0 * per_row:r1 * per_row] = _draw_host(key, idx_np, table)
            continue
        idx = (torch.arange(r0, r1, dtype=torch.int64, device=device)[:, None] * (H * D) + inner[None, :]).reshape(-1)
        h = _lowbias32((_mul32(idx, 0x27D4EB2F) + key) & _M32)
        out[r0 * per_row:r1 * per_row] = table[(h >> 8) & 0xFFFF]
    return out.view(rows, hs.numel(), D)

# ---------------------------------------------------------------- builders
def _lognormal_lengths(rng, count, median, sigma, lo, hi) -> np.ndarray:
    x = rng.normal(math.log(median), sigma, size=count)
    return np.clip(np.rint(np.exp(x)), lo, hi).astype(np.int64)


def make_workload(name: str, seed: int, *, hq: int, hkv: int, d: int,
                  decodes: List[Tuple[int, int]], prefills: List[int],
                  rng: Optional[np.random.Generator] = None, pool_pages: Optional[int] = None,
                  q_scale: float = 1.0, page_size: int = PAGE_SIZE,
                  sm_scale: Optional[float] = None,
                  pos_decodes: Sequence[Tuple[Sequence[int], int]] = ()) -> Workload:
    """decodes: list of (o, L) for 32-row block decodes (n = min(32, L - o)),
    or (o, L, n) for a block of n rows at positions o .. o+n-1 over a cached
    context (n may exceed 32: a larger decode block);
    pos_decodes: list of (positions, L) for decodes that recompute the given
    strictly increasing positions (placed after the block decodes);
    prefills: list of L. Pages are drawn from ``rng`` (default: seeded by seed)."""
    if rng is None:
        rng = np.random.default_rng(seed)
    q_off, kv_len, n_rows, pre, pos = [], [], [], [], []
    for dec in decodes:
        o, L = dec[0], dec[1]
        n = dec[2] if len(dec) > 2 else min(BLOCK, L - o)
        assert 1 <= n and o >= 0 and o + n <= L, dec
        q_off.append(o)
        kv_len.append(L)
        n_rows.append(n)
        pre.append(False)
        pos.append(np.arange(o, o + n_rows[-1]))
    for (pp, L) in pos_decodes:
        pp = np.asarray(pp, dtype=np.int64)
        assert len(pp) >= 1 and (np.diff(pp) > 0).all() and pp[0] >= 0 and pp[-1] < L
        q_off.append(int(pp[0]))
        kv_len.append(L)
        n_rows.append(len(pp))
        pre.append(False)
        pos.append(pp)
    for L in prefills:
        q_off.append(0)
        kv_len.append(L)
        n_rows.append(L)
        pre.append(True)
        pos.append(np.arange(L))
    kv_len_a = np.asarray(kv_len, dtype=np.int32)
    npages = (kv_len_a.astype(np.int64) + page_size - 1) // page_size
    needed = int(npages.sum())
    pool = pool_pages if pool_pages is not None else max(2 * needed, 1)
    perm = rng.permutation(pool)[:needed].astype(np.int32)
    page_indptr = np.zeros(len(kv_len) + 1, dtype=np.int32)
    page_indptr[1:] = np.cumsum(npages)
    q_indptr = np.zeros(len(kv_len) + 1, dtype=np.int32)
    q_indptr[1:] = np.cumsum(n_rows)
    if sm_scale is None:
        sm_scale = float(np.float32(1.0 / math.sqrt(d)))
    return Workload(name=name, seed=seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                    q_indptr=q_indptr, q_offset=np.asarray(q_off, dtype=np.int32),
                    kv_len=kv_len_a, is_prefill=np.asarray(pre, dtype=bool),
                    page_indptr=page_indptr, page_ids=perm, num_pool_pages=pool,
                    sm_scale=sm_scale, q_scale=q_scale, page_size=page_size,
                    q_pos=np.concatenate(pos).astype(np.int32) if pos_decodes else None)


def _decodes_from_prompts(rng, prompts, resp) -> List[Tuple[int, int]]:
    blocks = rng.integers(0, resp // BLOCK, size=len(prompts))
    return [(int(P) + BLOCK * int(b), int(P) + resp) for P, b in zip(prompts, blocks)]


def tiny_mixed(seed: int = 0) -> Workload:
    """Single request, one layer: MHA 4/4, D 64, prompt 96 + 32 masked response
    positions (L = 128). Item 0 is the block decode of rows 96..127 over all 128
    cached positions; item 1 is the whole 128-token prefill. The decode's cache
    is the prefill's K/V and its query / fresh K/V rows are the prefill's rows
    96..127, so decode rows must equal prefill rows 96..127."""
    w = make_workload("tiny_mixed", seed, hq=4, hkv=4, d=64, decodes=[(96, 128)], prefills=[128])
    base = Workload(**{f.name: getattr(w, f.name) for f in dataclasses.fields(w)})
    base.value_fn = None

    def value_fn(item, kind):
        # everything is drawn as item 1 (the prefill); item 0 views into it
        if item == 1:
            return None
        if kind == KIND_Q:
            return base.q(1)[96:128].float()
        if kind == KIND_KNEW:
            return base.k_new(1)[96:128].float()
        if kind == KIND_VNEW:
            return base.v_new(1)[96:128].float()
        if kind == KIND_KCTX:
            return base.k_new(1).float()
        if kind == KIND_VCTX:
            return base.v_new(1).float()
        return None

    w.value_fn = value_fn
    return w


def llada_decode(seed: int = 0) -> Workload:
    """LLaDA-8B-shaped layer, decode only: MHA 32/32, D 128; 32 block decodes,
    prompts ~ LN(300, 0.8) in [16, 2048] + 256 response, block index 0..7."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, 32, 300, 0.8, 16, 2048)
    dec = _decodes_from_prompts(rng, P, 256)
    return make_workload("llada_decode", seed, hq=32, hkv=32, d=128, decodes=dec, prefills=[], rng=rng)


def dream_mixed(seed: int = 0) -> Workload:
    """Dream-7B-shaped layer, mixed batch: GQA 28/4, D 128; 48 block decodes
    (prompts ~ LN(500, 0.8) in [16, 4096] + 256) plus two whole prefills of
    L = 2304 and 3328."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, 48, 500, 0.8, 16, 4096)
    dec = _decodes_from_prompts(rng, P, 256)
    return make_workload("dream_mixed", seed, hq=28, hkv=4, d=128, decodes=dec,
                         prefills=[2304, 3328], rng=rng)


def dream_decode(seed: int = 0) -> Workload:
    """The 48 block decodes of dream_mixed(seed) alone (the same lengths and
    block offsets; GQA 28/4, D 128): a decode-only batch whose whole-group
    tiles leave CUs idle unless its contexts are cut."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, 48, 500, 0.8, 16, 4096)
    dec = _decodes_from_prompts(rng, P, 256)
    return make_workload("dream_decode", seed, hq=28, hkv=4, d=128, decodes=dec, prefills=[], rng=rng)


def dream_prefill(seed: int = 0) -> Workload:
    """The two whole prefills of dream_mixed (L = 2304 and 3328; GQA 28/4,
    D 128) alone: the batch's compute-bound part, profiled apart from its
    block decodes."""
    rng = np.random.default_rng(seed)
    _lognormal_lengths(rng, 48, 500, 0.8, 16, 4096)  # the same draws as dream_mixed, so the same pages
    rng.integers(0, 256 // BLOCK, size=48)
    return make_workload("dream_prefill", seed, hq=28, hkv=4, d=128, decodes=[], prefills=[2304, 3328], rng=rng)


def prefill_heavy(seed: int = 0) -> Workload:
    """Long-document prefills: GQA 28/4, D 128; 8 whole prefills with prompts
    ~ LN(6000, 0.5) in [1024, 16384] + 256 response; KV written to pages."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, 8, 6000, 0.5, 1024, 16384)
    return make_workload("prefill_heavy", seed, hq=28, hkv=4, d=128, decodes=[],
                         prefills=[int(p) + 256 for p in P], rng=rng)


LONG_DECODE_POOL_PAGES = 262_144  # 64 GiB of K+V pages at MHA 32 heads, D 128


def long_decode(seed: int = 0) -> Workload:
    """High-concurrency long-context decode: MHA 32/32, D 128; 256 block
    decodes, prompts ~ LN(1200, 1.0) in [16, 32768] + 512 response, block index
    0..15, pages scattered over a 64 GiB pool (262,144 pages)."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, 256, 1200, 1.0, 16, 32768)
    dec = _decodes_from_prompts(rng, P, 512)
    return make_workload("long_decode", seed, hq=32, hkv=32, d=128, decodes=dec, prefills=[],
                         rng=rng, pool_pages=LONG_DECODE_POOL_PAGES)


WORKLOADS = {
    "tiny_mixed": tiny_mixed,
    "llada_decode": llada_decode,
    "dream_mixed": dream_mixed,
    "dream_decode": dream_decode,
    "dream_prefill": dream_prefill,
    "prefill_heavy": prefill_heavy,
    "long_decode": long_decode,
}


def token_cache_decodes(seed: int, *, hq: int, hkv: int, d: int, count: int, median: int = 500,
                        sigma: float = 0.8, resp: int = 256, rows: int = 32,
                        prefills: Sequence[int] = ()) -> Workload:
    """Per-token cached decodes (the dKV-Cache-PD reading of Sec. 2.2): each of
    `count` requests, prompt ~ LN(median, sigma) + `resp` response positions,
    recomputes `rows` positions drawn without replacement from its response
    (sorted) and reuses the cache everywhere else; optional whole prefills
    join the batch."""
    rng = np.random.default_rng(seed)
    P = _lognormal_lengths(rng, count, median, sigma, 16, 4096)
    pos = []
    for p in P:
        pp = np.sort(rng.choice(resp, size=rows, replace=False)) + int(p)
        pos.append((pp, int(p) + resp))
    return make_workload(f"token_cache_{hq}_{hkv}_{d}", seed, hq=hq, hkv=hkv, d=d, decodes=[],
                         prefills=list(prefills), rng=rng, pos_decodes=pos)


@dataclasses.dataclass
class TraceRequest:
    """One request of a synthetic serving trace."""
    rid: int
    arrival: int             # iteration at which it arrives
    prompt: int              # prompt tokens P
    resp: int                # appended masked response tokens R (R / 32 blocks)
    steps: List[int]         # denoising steps of each block (block decodes per block)


def serving_trace(seed: int, iterations: int, rate: float, *, median: int = 500, sigma: float = 0.8,
                  resp: int = 256, min_steps: int = 2, max_steps: int = 8) -> List[TraceRequest]:
    """Synthetic request stream for a serving loop (stands in for the paper's
    traces, Sec. 6.1): Poisson arrivals at `rate` requests per iteration,
    prompts ~ LN(median, sigma) in [16, 4096], `resp` appended masks in blocks
    of 32, and per block a number of denoising steps (block decodes) drawn
    uniformly from [min_steps, max_steps] (the confidence-threshold sampler
    unmasks a variable number of tokens per step, Sec. 3.2)."""
    rng = np.random.default_rng(seed)
    reqs: List[TraceRequest] = []
    for t in range(iterations):
        for _ in range(int(rng.poisson(rate))):
            P = int(_lognormal_lengths(rng, 1, median, sigma, 16, 4096)[0])
            steps = [int(x) for x in rng.integers(min_steps, max_steps + 1, size=resp // BLOCK)]
            reqs.append(TraceRequest(len(reqs), t, P, resp, steps))
    return reqs


SWEEP_SHAPES = {"llada": (32, 32), "dream": (28, 4)}


def token_cache(seed: int = 0) -> Workload:
    """LLaDA-8B-shaped per-token cached decodes: MHA 32/32, D 128; 32 requests
    (prompts ~ LN(300, 0.8) in [16, 4096] + 256 response), each recomputing 32
    scattered response positions over its whole cached context."""
    return token_cache_decodes(seed, hq=32, hkv=32, d=128, count=32, median=300, sigma=0.8)


def decode_sweep(shape: str, batch: int, seed: int = 0, L: int = 1024) -> Workload:
    """Decode-batch sweep point: `batch` block decodes of one model shape (LLaDA
    32/32 or Dream 28/4 heads, D 128), every request with L = 1024 cached
    positions and its 32-row block at a random block index of the last 256."""
    hq, hkv = SWEEP_SHAPES[shape]
    rng = np.random.default_rng(seed)
    blocks = rng.integers(0, 8, size=batch)
    dec = [(L - 256 + 32 * int(b), L) for b in blocks]
    return make_workload(f"decode_sweep_{shape}_{batch}", seed, hq=hq, hkv=hkv, d=128, decodes=dec,
                         prefills=[], rng=rng)


def ragged_small(seed: int, *, hq: int, hkv: int, d: int, q_scale: float = 1.0) -> Workload:
    """Small ragged mixed batch spanning several tiles and ragged tails: block
    decodes with partial last pages and short / odd-length prefills."""
    rng = np.random.default_rng(1000 + seed)
    dec = []
    for L in (37, 130, 333, 700, 64, 1025):
        o = int(rng.integers(0, max(1, L - 8)))
        dec.append((o, L))
    pre = [1, 19, 150, 301]
    return make_workload(f"ragged_small_{hq}_{hkv}_{d}", seed, hq=hq, hkv=hkv, d=d,
                         decodes=dec, prefills=pre, rng=rng, q_scale=q_scale)


def device_inputs(wl: Workload, device, fill: Optional[float] = float("nan")) -> dict:
    """Device tensors of one call: packed q / k_new / v_new, the paged pools with
    every decode item's pre-call context scattered in, and the page table.
    Pool slots that hold no context are set to ``fill`` (NaN by default, so a
    read of an unowned slot shows up in the output); ``fill=None`` leaves them
    uninitialised."""
    shape = (wl.num_pool_pages, wl.num_kv_heads, wl.page_size, wl.head_dim)
    if fill is None:
        k_cache = torch.empty(shape, dtype=torch.bfloat16, device=device)
        v_cache = torch.empty(shape, dtype=torch.bfloat16, device=device)
    else:
        k_cache = torch.full(shape, fill, dtype=torch.bfloat16, device=device)
        v_cache = torch.full(shape, fill, dtype=torch.bfloat16, device=device)
    wl.fill_paged_cache(k_cache, v_cache)
    return dict(q=wl.packed_q(device), k_new=wl.packed_k_new(device), v_new=wl.packed_v_new(device),
                k_cache=k_cache, v_cache=v_cache,
                page_ids=torch.from_numpy(np.ascontiguousarray(wl.page_ids)).to(device))


def gather_item_cache(wl: Workload, pool: torch.Tensor, i: int) -> torch.Tensor:
    """Positions [0, L_i) of item i read back from a pool, [L_i, Hkv, D]."""
    pages = torch.from_numpy(wl.item_pages(i).astype(np.int64)).to(pool.device)
    blk = pool[pages].permute(0, 2, 1, 3).reshape(-1, wl.num_kv_heads, wl.head_dim)
    return blk[:int(wl.kv_len[i])]


@dataclasses.dataclass
class KvTransferCase:
    """A batch of requests to move between two paged pools: the source page
    table (sender's pool) and an unrelated destination page table (receiver's
    pool), with the source pool's contents as bf16 bit patterns."""
    name: str
    kv_len: np.ndarray       # [n] int32
    page_indptr: np.ndarray  # [n + 1] int32
    src_pages: np.ndarray    # [total pages] int32, pages of the source pool
    dst_pages: np.ndarray    # [total pages] int32, pages of the destination pool
    num_pool_pages: int
    num_kv_heads: int
    head_dim: int
    pool_k: np.ndarray       # [num_pool_pages, Hkv, 16, D] uint16
    pool_v: np.ndarray

    @property
    def rows(self) -> int:
        return int(self.kv_len.sum())


def kv_transfer_case(name: str, seed: int, kv_len: Sequence[int], *, hkv: int, d: int,
                     spare_pages: int = 3) -> KvTransferCase:
    """Requests of the given lengths laid out on random pages of a pool with
    `spare_pages` unused pages per used one; both page tables are drawn
    without replacement from the same pool size. Pool values: standard normal
    draws rounded to bf16 (every slot, listed or not)."""
    rng = np.random.default_rng(seed)
    kv_len = np.asarray(kv_len, np.int32)
    counts = (kv_len.astype(np.int64) + 15) // 16
    page_indptr = np.zeros(len(kv_len) + 1, np.int32)
    page_indptr[1:] = np.cumsum(counts)
    total = int(page_indptr[-1])
    pool = max(total * (1 + spare_pages), 1)
    src = rng.permutation(pool)[:total].astype(np.int32)
    dst = rng.permutation(pool)[:total].astype(np.int32)
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (pool, hkv, 16, d)
    pk = torch.randn(shape, generator=g).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    pv = torch.randn(shape, generator=g).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return KvTransferCase(name, kv_len, page_indptr, src, dst, pool, hkv, d, pk, pv)
