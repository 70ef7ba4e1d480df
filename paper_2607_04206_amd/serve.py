"""A serving loop around the attention call: requests move through the
cached-dLLM cycle (whole prefill of prompt + masked response, then block
decodes of one 32-token block until it is resolved, then a re-prefill that
refreshes the cache at the block boundary; Sec. 2.2, Sec. 4.3), each
iteration's microbatch is composed by the deficit token-budget rule
(Sec. 4.1, Alg. 1) and served by one sangam_attn_forward call over a paged KV
pool (Sec. 5).

Only one attention layer is run per iteration (the model around it is out of
scope), with synthetic Q / K / V values: the loop exercises batch composition,
planning and the kernels on real mixed batches."""
from __future__ import annotations

import dataclasses
import time
from typing import List, Optional

import numpy as np
import torch

from . import attn, sched

BLOCK = 32
PAGE = 16


class PagePool:
    """Free list of KV pages of one pool (host side)."""

    def __init__(self, num_pages: int):
        self.num_pages = num_pages
        self._free = list(range(num_pages - 1, -1, -1))

    def take(self, n: int) -> List[int]:
        if n > len(self._free):
            raise MemoryError(f"KV pool exhausted: {n} pages wanted, {len(self._free)} free")
        return [self._free.pop() for _ in range(n)]

    def give(self, pages: List[int]) -> None:
        self._free.extend(reversed(pages))

    @property
    def free(self) -> int:
        return len(self._free)


@dataclasses.dataclass
class _State:
    req: object                 # workloads.TraceRequest
    pages: Optional[List[int]] = None
    block: int = 0              # block being decoded (or to decode after the prefill)
    steps_left: int = 0
    phase: str = "waiting"      # waiting (for a prefill), decoding, done
    queued_at: int = 0

    @property
    def L(self) -> int:
        return self.req.prompt + self.req.resp


@dataclasses.dataclass
class Iteration:
    t: int
    decodes: int
    prefills: int
    prefill_tokens: int
    waiting_after: int
    deficit: int
    plan_ms: float
    events: Optional[tuple] = None  # (start, end) torch events around the call
    # start / stop events in the dispatch of each launch that ran (prefill-
    # shaped, decode-shaped, merge): kernel execution without host gaps
    launch_events: Optional[list] = None
    queue_waits: List[int] = dataclasses.field(default_factory=list)
    captured: Optional[dict] = None
    batch: Optional[list] = None  # (request id, kind) of each item, in batch order


class ServingLoop:
    """Drive a list of trace requests through iterations of one GPU."""

    def __init__(self, requests, *, hq: int, hkv: int, d: int, tau: int, device,
                 num_pool_pages: Optional[int] = None, max_rows: int = 1 << 15, seed: int = 0):
        self.reqs = [_State(r) for r in sorted(requests, key=lambda r: (r.arrival, r.rid))]
        self.hq, self.hkv, self.d, self.tau = hq, hkv, d, tau
        self.dev = device
        need = sum(-(-(s.L) // PAGE) for s in self.reqs)
        self.pool = PagePool(num_pool_pages if num_pool_pages is not None else max(need, 1))
        self.max_rows = max_rows
        if device is not None:  # device None: plan every batch but run nothing (host checks)
            g = torch.Generator(device="cpu").manual_seed(seed)
            shape = (self.pool.num_pages, hkv, PAGE, d)
            self.k_cache = torch.randn(shape, generator=g).to(torch.bfloat16).to(device)
            self.v_cache = torch.randn(shape, generator=g).to(torch.bfloat16).to(device)
            self.q = torch.randn((max_rows, hq, d), generator=g).to(torch.bfloat16).to(device)
            self.k_new = torch.randn((max_rows, hkv, d), generator=g).to(torch.bfloat16).to(device)
            self.v_new = torch.randn((max_rows, hkv, d), generator=g).to(torch.bfloat16).to(device)
            self.out = torch.empty((max_rows, hq, d), dtype=torch.bfloat16, device=device)
            self.lse = torch.empty((max_rows, hq), dtype=torch.float32, device=device)
        self.deficit = 0
        self.next_arrival = 0
        self.waiting: List[_State] = []  # arrival order of the requests (re-prefills keep their place)
        self.sm_scale = float(np.float32(1.0 / np.sqrt(d)))

    def _arrive(self, t: int) -> None:
        while self.next_arrival < len(self.reqs) and self.reqs[self.next_arrival].req.arrival <= t:
            s = self.reqs[self.next_arrival]
            s.queued_at = t
            self.waiting.append(s)
            self.next_arrival += 1
        self.waiting.sort(key=lambda s: (s.req.arrival, s.req.rid))

    def busy(self) -> bool:
        return self.next_arrival < len(self.reqs) or any(s.phase != "done" for s in self.reqs)

    def step(self, t: int, timed: bool = True, capture: bool = False) -> Optional[Iteration]:
        """One iteration: compose the microbatch, run the call, advance states.
        capture: keep the call's descriptor and a copy of its inputs (the
        pages' pre-call content included) on the record, for checking."""
        self._arrive(t)
        decodes = [s for s in self.reqs if s.phase == "decoding"]
        n_adm, self.deficit = sched.admit(self.tau, BLOCK * len(decodes), len(decodes),
                                          [s.L for s in self.waiting], self.deficit)
        admitted = self.waiting[:n_adm]
        del self.waiting[:n_adm]
        if not decodes and not admitted:
            return None
        for s in admitted:
            if s.pages is None:  # a request's pages live from its first prefill to its end
                s.pages = self.pool.take(-(-s.L // PAGE))
        items = decodes + admitted
        nd = len(decodes)
        n = [BLOCK] * nd + [s.L for s in admitted]
        o = [s.req.prompt + BLOCK * s.block for s in decodes] + [0] * len(admitted)
        rows = int(np.sum(n))
        if rows > self.max_rows:
            raise ValueError(f"iteration {t}: {rows} rows exceed the {self.max_rows}-row buffers")
        q_indptr = np.zeros(len(items) + 1, np.int32)
        q_indptr[1:] = np.cumsum(n)
        kv_len = np.asarray([s.L for s in items], np.int32)
        page_indptr = np.zeros(len(items) + 1, np.int32)
        page_indptr[1:] = np.cumsum([len(s.pages) for s in items])
        page_ids = np.concatenate([np.asarray(s.pages, np.int32) for s in items])
        t0 = time.perf_counter()
        p = attn.plan(q_indptr=q_indptr, q_offset=np.asarray(o, np.int32), kv_len=kv_len,
                      page_indptr=page_indptr, page_ids=page_ids, num_q_heads=self.hq,
                      num_kv_heads=self.hkv, head_dim=self.d, num_pool_pages=self.pool.num_pages,
                      sm_scale=self.sm_scale, device=self.dev)
        plan_ms = (time.perf_counter() - t0) * 1e3
        if self.dev is None:
            timed = capture = False
        else:
            self._nd = nd
            self._desc = (q_indptr, np.asarray(o, np.int32), kv_len, page_indptr)
            self._run(p, page_ids, rows, timed, capture)
        rec = Iteration(t=t, decodes=len(decodes), prefills=len(admitted),
                        prefill_tokens=int(sum(s.L for s in admitted)), waiting_after=len(self.waiting),
                        deficit=self.deficit, plan_ms=plan_ms, events=self._ev if timed else None,
                        launch_events=self._lev if timed else None,
                        queue_waits=[t - s.queued_at for s in admitted])
        rec.captured = self._snap if capture else None
        rec.batch = [(s.req.rid, "decode" if k < nd else "prefill") for k, s in enumerate(items)]
        self._advance(t, decodes, admitted)
        return rec

    def _run(self, p, page_ids, rows, timed, capture):
        pid = torch.from_numpy(page_ids).to(self.dev, non_blocking=True)
        stream = torch.cuda.current_stream(self.dev)
        snap = None
        nd = self._nd
        if capture:
            q_indptr, q_offset, kv_len, page_indptr = self._desc
            snap = dict(q_indptr=q_indptr, q_offset=q_offset, kv_len=kv_len,
                        page_indptr=page_indptr, page_ids=page_ids, sm_scale=self.sm_scale,
                        q=self.q[:rows].clone(), k_new=self.k_new[:rows].clone(),
                        v_new=self.v_new[:rows].clone(),
                        k_pages=self.k_cache[pid.long()].clone(), v_pages=self.v_cache[pid.long()].clone(),
                        decodes=nd)
        ev = lev = used = None
        if timed:
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            lev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
            for e in lev:  # torch reads elapsed time only from events it has recorded
                e.record(stream)
            i = p.info
            used = (i.num_prefill_tiles > 0, i.num_decode_tiles > 0, i.num_split_items > 0)
            ev[0].record(stream)
        attn.forward(p, self.q[:rows], self.k_new[:rows], self.v_new[:rows], self.k_cache, self.v_cache,
                     pid, out=self.out[:rows], lse=self.lse[:rows], launch_events=lev)
        if timed:
            ev[1].record(stream)
            lev = [(lev[2 * k], lev[2 * k + 1]) for k in range(3) if used[k]]
        if capture:
            snap["out"] = self.out[:rows].clone()
            snap["lse"] = self.lse[:rows].clone()
        self._ev, self._lev, self._snap = ev, lev, snap

    def _advance(self, t, decodes, admitted):
        # advance: a prefill starts (or resumes at) its block; a decode step
        # may resolve the block, which sends the request back for a re-prefill
        for s in admitted:
            s.phase = "decoding"
            s.steps_left = s.req.steps[s.block]
        for s in decodes:
            s.steps_left -= 1
            if s.steps_left == 0:
                s.block += 1
                if s.block == len(s.req.steps):
                    s.phase = "done"
                    self.pool.give(s.pages)
                    s.pages = None
                else:
                    s.phase = "waiting"
                    s.queued_at = t + 1
                    self.waiting.append(s)
        self.waiting.sort(key=lambda s: (s.req.arrival, s.req.rid))

    def run(self, max_iterations: int, timed: bool = True) -> List[Iteration]:
        log = []
        for t in range(max_iterations):
            if not self.busy():
                break
            rec = self.step(t, timed)
            if rec is not None:
                log.append(rec)
        return log
