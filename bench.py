#!/usr/bin/env python3
"""Benchmark of the mixed block-decode / prefill attention call on one MI355X.

A step is one whole call: the prefill-shaped and the decode-shaped attention
launches (which also write the fresh K/V rows back into their pages) and the
split merge, over one batch whose inputs are already resident in HBM. Prints
one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--seed S]

Protocol:
- the plan is timed on the host (median of 5);
- W warm-up steps;
- a per-launch breakdown (events in each launch's dispatch; null for a
  launch that has no work);
- the timed region: K steps back to back, bracketed by device
  synchronisation, with events only on the dominant attention launch;
  ms_per_step is host wall time over those K steps, and the roofline figure
  is that launch's mean duration (median and min beside it);
- R flushed steps (--flushed-reps): before each, a 1 GiB read outside the
  timing evicts the previous step's data from the 256 MB Infinity Cache; the
  step and the dominant launch are timed with events (median and min);
- the chip's measured ceilings (a 4 GiB streaming read, an MFMA-only loop),
  against which the fractions are reported beside the spec-sheet peaks;
- the oracle on a bounded CPU sample (median of 3 after a warm-up).

Work counts are algorithmic: F = sum 4 n L D Hq flops (QK^T and PV, no causal
halving) and B = K/V read once per item + cache write of the fresh rows + Q
read + O write + page ids + LSE write.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attention TFLOP/s + KV HBM GB/s (frac. of roofline), mixed decode/prefill batch"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PHASES = ("prefill_attn", "decode_attn", "merge")


def split_work(wl, fused_decodes=False):
    """Algorithmic flops / bytes of each attention launch of the call.
    fused_decodes: the plan runs the block decodes inside the prefill-shaped
    launch. Each launch also writes back the fresh rows of its items."""
    import numpy as np
    n = np.diff(wl.q_indptr).astype(np.float64)
    L = wl.kv_len.astype(np.float64)
    D, Hq, Hkv = wl.head_dim, wl.num_q_heads, wl.num_kv_heads
    pre = n > 32
    flops = 4.0 * n * L * D * Hq
    # K/V read once, Q read, O write, LSE write, page ids (decode), and the
    # fresh rows written into their pages
    attn_b = 2.0 * (2 * L * Hkv * D + 2 * n * Hq * D) + 4.0 * n * Hq
    attn_b += np.where(pre, 0.0, 4.0 * np.ceil(L / 16))
    attn_b += 2.0 * (2 * n * Hkv * D)
    in_pre = np.ones_like(pre) if fused_decodes else pre
    return {
        "prefill_attn": (float(flops[in_pre].sum()), float(attn_b[in_pre].sum())),
        "decode_attn": (float(flops[~in_pre].sum()), float(attn_b[~in_pre].sum())),
    }


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def _oracle_sample(wl, target_flops, row_flops):
    """Rows of a bounded sample: whole block decodes first, then evenly spaced
    rows of each prefill, up to about target_flops."""
    import numpy as np
    dec = [i for i in range(wl.num_items) if wl.n(i) <= 32]
    pre = [i for i in range(wl.num_items) if wl.n(i) > 32]
    rows, acc = {}, 0.0
    for i in dec:
        if acc + wl.n(i) * row_flops(i) > target_flops and rows:
            break
        rows[i] = np.arange(wl.n(i))
        acc += wl.n(i) * row_flops(i)
    left = max(target_flops - acc, 0.0)
    if pre:
        per_item = left / len(pre)
        for i in pre:
            k = int(min(wl.n(i), max(1, per_item // row_flops(i))))
            rows[i] = np.linspace(0, wl.n(i) - 1, k).astype(np.int64)
            acc += k * row_flops(i)
    return rows, acc


def cpu_baseline(wl, budget_s, single_thread=True):
    """The oracle (as it stands) on the host cores, on a bounded sample of the
    same workload: every block decode, then evenly spaced rows of each prefill,
    sized so that one run takes about budget_s / 3. A calibration run serves as
    the warm-up; then three timed runs, whose median gives the rate. Input
    drawing is not timed. Also one thread on the single-request workload
    (whole call) and on a sample of the LLaDA decode batch."""
    import numpy as np

    import workloads
    from oracle import oracle
    all_threads = len(os.sched_getaffinity(0))
    threads = oracle.threads(all_threads)
    D, Hq = wl.head_dim, wl.num_q_heads

    def timed(call, sel):
        t0 = time.perf_counter()
        oracle.run(call, sel)
        return time.perf_counter() - t0

    def rate_of(w, budget, row_flops):
        # calibrate on a piece large enough to keep the threads busy
        dec = [i for i in range(w.num_items) if w.n(i) <= 32]
        cal_items = dec[:4] if dec else [i for i in range(w.num_items)][:1]
        cal_rows = {i: np.arange(w.n(i) if w.n(i) <= 32 else min(w.n(i), 64)) for i in cal_items}
        call = oracle.Call(w, sorted(cal_rows))
        sel, _, _ = oracle.selection(call, cal_rows)
        cal = sum(len(r) * row_flops(i) for i, r in cal_rows.items()) / max(timed(call, sel), 1e-6)
        return cal * budget

    row_flops = lambda i: 4.0 * int(wl.kv_len[i]) * D * Hq
    rows, acc = _oracle_sample(wl, rate_of(wl, budget_s / 3, row_flops), row_flops)
    call = oracle.Call(wl, sorted(rows))
    sel, _, _ = oracle.selection(call, rows)
    times = [timed(call, sel) for _ in range(3)]
    dt = float(np.median(times))
    n_dec = sum(1 for i in rows if wl.n(i) <= 32)
    n_pre_rows = sum(len(rows[i]) for i in rows if wl.n(i) > 32)
    total_dec = sum(1 for i in range(wl.num_items) if wl.n(i) <= 32)
    total_pre_rows = sum(wl.n(i) for i in range(wl.num_items) if wl.n(i) > 32)
    model = cpu_model()
    sample = (f"{n_dec} of {total_dec} block decodes (all rows, all heads) and {n_pre_rows} of "
              f"{total_pre_rows} prefill rows, evenly spaced (all heads), of {wl.name} seed {wl.seed}: "
              f"{acc / 1e9:.1f} GFLOP, median of 3 runs after a warm-up "
              f"({', '.join(f'{x:.2f}' for x in times)} s), fp64, {threads} threads on {model}, "
              f"input drawing excluded")

    # one thread: the single-request workload whole, and LLaDA block decodes
    one = []
    oracle.threads(1)
    try:
        for w, budget in ((workloads.tiny_mixed(0), None), (workloads.llada_decode(0), 3.0)) if single_thread else ():
            rf = lambda i, w=w: 4.0 * int(w.kv_len[i]) * w.head_dim * w.num_q_heads
            if budget is None:
                r1 = {i: np.arange(w.n(i)) for i in range(w.num_items)}
                a1 = sum(w.n(i) * rf(i) for i in range(w.num_items))
            else:
                r1, a1 = _oracle_sample(w, rate_of(w, budget, rf), rf)
            c1 = oracle.Call(w, sorted(r1))
            s1, _, _ = oracle.selection(c1, r1)
            timed(c1, s1)
            t1 = float(np.median([timed(c1, s1) for _ in range(3)]))
            one.append({"workload": w.name, "value": a1 / t1 / 1e12, "unit": "TFLOP/s", "cores": 1,
                        "sample": f"{len(r1)} of {w.num_items} items ({a1 / 1e9:.2f} GFLOP), median of 3 "
                                  f"after a warm-up: {t1:.3f} s"})
    finally:
        oracle.threads(all_threads)
    return {"value": acc / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": sample, "seconds": dt, "cpu": model, "single_thread": one or None}


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in ("attn_fwd.hip", "plan.cpp", "plan_format.h"):
        with open(os.path.join(ROOT, "paper_2607_04206_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, or None when there is none or the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != kernel_source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def decode_sweep(args):
    """Decode iteration time against batch size (the attention-only analogue
    of the paper's decode-batch measurement): each point is one call over B
    block decodes at L = 1024, timed over `steps` back-to-back calls; the
    dominant launch is timed with dispatch-attached events."""
    import ctypes
    import numpy as np
    import torch

    import workloads
    from paper_2607_04206_amd import attn
    from paper_2607_04206_amd._lib import check, lib

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    for shape in ("llada", "dream"):
        for B in [int(b) for b in args.sweep_batches.split(",")]:
            wl = workloads.decode_sweep(shape, B, args.seed)
            t = workloads.device_inputs(wl, dev, fill=None)
            p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len,
                          page_indptr=wl.page_indptr, page_ids=wl.page_ids,
                          num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                          head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages,
                          sm_scale=wl.sm_scale, device=dev)
            out = torch.empty((wl.total_q, wl.num_q_heads, wl.head_dim), dtype=torch.bfloat16, device=dev)
            lse = torch.empty((wl.total_q, wl.num_q_heads), dtype=torch.float32, device=dev)
            ws = torch.empty((max(p.workspace_bytes, 16),), dtype=torch.uint8, device=dev)
            args_c = attn.c_args(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                                 t["page_ids"], out, lse, ws, stream)
            for _ in range(args.warmup):
                check(lib.sangam_attn_forward(*args_c))
            K = args.steps
            evs = []
            for _ in range(K):
                e = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
                for x in e:
                    x.record(stream)
                evs.append((e, (ctypes.c_void_p * 6)(*[x.cuda_event for x in e])))
            torch.cuda.synchronize()
            w0 = time.perf_counter()
            for k in range(K):
                check(lib.sangam_attn_forward(*args_c))
            torch.cuda.synchronize()
            ms = (time.perf_counter() - w0) * 1e3 / K
            for k in range(K):
                check(lib.sangam_attn_forward_timed(*args_c, evs[k][1]))
            torch.cuda.synchronize()
            launches = np.mean([[e[2 * j].elapsed_time(e[2 * j + 1]) for j in range(3)] for e, _ in evs], 0)
            F, Bytes = wl.flops(), wl.hbm_bytes()
            # the launch that holds the block decodes: prefill-shaped heads-across
            # tiles for a small GQA batch, else the decode-shaped launch
            fused = int(p.info.num_fused_decode_tiles) > 0
            kern = float(launches[0] if fused else launches[1])
            print(json.dumps({
                "sweep": "decode_batch", "shape": shape, "num_q_heads": wl.num_q_heads,
                "num_kv_heads": wl.num_kv_heads, "batch": B, "kv_len": 1024, "ms_per_call": ms,
                "decode_kernel_ms": kern, "merge_ms": float(launches[2]) if p.info.num_split_items > 0 else None,
                "tflops": F / (ms / 1e3) / 1e12, "hbm_gbs": Bytes / (ms / 1e3) / 1e9,
                "kernel_hbm_frac": Bytes / (kern / 1e3) / (PEAK_HBM_GBS * 1e9),
                "kernel_mfma_frac": F / (kern / 1e3) / (PEAK_BF16_TFLOPS * 1e12),
                "decode_launch": "prefill-shaped (heads across)" if fused else "decode-shaped",
                "splits": int(p.info.num_split_items),
                "tiles": int(p.info.num_prefill_tiles if fused else p.info.num_decode_tiles),
                "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(wl, args.sweep_cpu_budget, False)}),
                  flush=True)
            del t, out, lse, ws


def serve_trace(args):
    """Serving loop over a synthetic trace (Dream 28/4 heads, D 128): per
    iteration the deficit rule admits whole prefills next to the in-flight
    block decodes, the host plans the batch and one attention call runs.
    Prints one JSON line with per-iteration call times (HIP events) split by
    iteration kind, admitted prefill tokens against tau, and prefill
    queueing delays."""
    import numpy as np
    import torch

    import workloads
    from paper_2607_04206_amd.serve import ServingLoop

    dev = torch.device("cuda:0")
    reqs = workloads.serving_trace(args.seed, args.trace_iters, args.trace_rate)
    loop = ServingLoop(reqs, hq=28, hkv=4, d=128, tau=args.tau, device=dev, seed=args.seed)
    log = loop.run(args.trace_iters * 8)
    torch.cuda.synchronize()
    ms = np.asarray([r.events[0].elapsed_time(r.events[1]) for r in log])
    kern = np.asarray([sum(a.elapsed_time(b) for a, b in r.launch_events) for r in log])
    mixed = np.asarray([r.prefills > 0 for r in log])
    waits = [w for r in log for w in r.queue_waits]
    def pct(x, q):
        return float(np.percentile(x, q)) if len(x) else None
    res = {
        "trace": "serving_loop", "heads": "28/4", "head_dim": 128, "tau": args.tau,
        "requests": len(reqs), "iterations": len(log), "rate_per_iteration": args.trace_rate,
        "finished": sum(1 for s in loop.reqs if s.phase == "done"),
        "mixed_iterations": int(mixed.sum()), "decode_only_iterations": int((~mixed).sum()),
        "call_ms_mean": float(ms.mean()), "call_ms_p50": pct(ms, 50), "call_ms_p99": pct(ms, 99),
        "decode_only_ms_mean": float(ms[~mixed].mean()) if (~mixed).any() else None,
        "mixed_ms_mean": float(ms[mixed].mean()) if mixed.any() else None,
        "mixed_ms_p99": pct(ms[mixed], 99),
        # the same from events in the launches' dispatches: kernel time, no host gaps
        "kernel_ms_mean": float(kern.mean()), "kernel_ms_p99": pct(kern, 99),
        "decode_only_kernel_ms_mean": float(kern[~mixed].mean()) if (~mixed).any() else None,
        "mixed_kernel_ms_mean": float(kern[mixed].mean()) if mixed.any() else None,
        "mixed_kernel_ms_p99": pct(kern[mixed], 99),
        "prefill_tokens_per_busy_iteration": float(np.mean([r.prefill_tokens for r in log])),
        "prefill_tokens_max": int(max(r.prefill_tokens for r in log)),
        "decodes_mean": float(np.mean([r.decodes for r in log])),
        "prefill_wait_iterations_mean": float(np.mean(waits)) if waits else None,
        "prefill_wait_iterations_p99": pct(waits, 99),
        "plan_ms_mean": float(np.mean([r.plan_ms for r in log])),
    }
    print(json.dumps(res), flush=True)


def kv_cpu_baseline(pool_k, pool_v, kv_len, page_indptr, page_ids, hkv, d, budget_s):
    """The export oracle (as it stands, one position at a time) on the first
    requests of the batch, as many as take about budget_s; their pages are
    copied to host memory first (not timed). Rate in the GPU lines' unit:
    K and V of every exported position read once and written once."""
    import numpy as np
    import torch

    from oracle import kv_transfer as okv

    def sample(n_req):
        lens = [int(x) for x in kv_len[:n_req]]
        pages = page_ids[page_indptr[0]:page_indptr[n_req]]
        idx = torch.as_tensor(pages.astype(np.int64), device=pool_k.device)
        hk = pool_k.index_select(0, idx).view(torch.int16).cpu().numpy()
        hv = pool_v.index_select(0, idx).view(torch.int16).cpu().numpy()
        local = np.arange(len(pages), dtype=np.int64)  # pages renumbered in sample order
        ind = np.asarray(page_indptr[:n_req + 1], np.int64) - int(page_indptr[0])
        t = time.perf_counter()
        okv.export(hk, hv, lens, ind, local)
        return sum(lens), time.perf_counter() - t

    rows1, dt1 = sample(1)
    per_row = dt1 / max(rows1, 1)
    n_req, acc = 0, 0
    while n_req < len(kv_len) and (acc + int(kv_len[n_req])) * per_row <= budget_s:
        acc += int(kv_len[n_req])
        n_req += 1
    n_req = max(n_req, 1)
    rows, dt = sample(n_req)
    moved = 2 * 2 * rows * hkv * d * 2
    return {"value": moved / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"export of {rows} positions ({n_req} of {len(kv_len)} requests) in {dt:.2f} s, "
                      f"pure Python, one thread"}


def kv_transfer(args):
    """Paged-KV export and import (the hand-off of requests' KV between workers
    in the hybrid configuration) over the cached contexts of the LLaDA decode
    batch (32 requests, 32 KV heads), the Dream mixed batch (50 requests, 4 KV
    heads) and the long decode batch (256 requests, 32 KV heads). Each copy is
    one launch; times are HIP events around it on the launch stream. Bytes
    moved = every position's K and V read once and written once."""
    import numpy as np
    import torch

    import workloads
    from paper_2607_04206_amd import kv

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    for name in ("llada_decode", "dream_mixed", "long_decode"):
        wl = getattr(workloads, name)(args.seed)
        hkv, d = wl.num_kv_heads, wl.head_dim
        rng = np.random.default_rng(args.seed)
        counts = (wl.kv_len.astype(np.int64) + 15) // 16
        indptr = np.zeros(len(counts) + 1, np.int32)
        indptr[1:] = np.cumsum(counts)
        pool = int(indptr[-1]) * 2
        src = rng.permutation(pool)[:indptr[-1]].astype(np.int32)
        dst = rng.permutation(pool)[:indptr[-1]].astype(np.int32)
        ps = kv.plan(kv_len=wl.kv_len, page_indptr=indptr, page_ids=src, num_kv_heads=hkv, head_dim=d,
                     num_pool_pages=pool, device=dev)
        pd = kv.plan(kv_len=wl.kv_len, page_indptr=indptr, page_ids=dst, num_kv_heads=hkv, head_dim=d,
                     num_pool_pages=pool, device=dev)
        shape = (pool, hkv, 16, d)
        ka = torch.randn(shape, device=dev).to(torch.bfloat16)
        va = torch.randn(shape, device=dev).to(torch.bfloat16)
        kb, vb = torch.empty_like(ka), torch.empty_like(va)
        pk = torch.empty((ps.rows, hkv, d), dtype=torch.bfloat16, device=dev)
        pv = torch.empty_like(pk)
        res = {"bench": "kv_transfer", "batch": name, "requests": int(wl.num_items), "kv_heads": hkv,
               "head_dim": d, "positions": ps.rows}
        moved = 2 * 2 * ps.rows * hkv * d * 2  # K and V, read and written
        for op, call in (("export", lambda: kv.kv_export(ps, ka, va, pk, pv)),
                         ("import", lambda: kv.kv_import(pd, pk, pv, kb, vb))):
            for _ in range(args.warmup):
                call()
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(args.steps)]
            torch.cuda.synchronize()
            for a, b in evs:
                a.record(stream)
                call()
                b.record(stream)
            torch.cuda.synchronize()
            us = float(np.mean([a.elapsed_time(b) for a, b in evs])) * 1e3
            res[f"{op}_us"] = us
            res[f"{op}_gbs"] = moved / (us / 1e6) / 1e9
            res[f"{op}_hbm_frac"] = res[f"{op}_gbs"] / PEAK_HBM_GBS
        res["bytes_moved_per_copy"] = moved
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = kv_cpu_baseline(ka, va, wl.kv_len, indptr, src, hkv, d, args.kv_cpu_budget)
        print(json.dumps(res), flush=True)
        del ka, va, kb, vb, pk, pv
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="dream_mixed",
                    choices=["tiny_mixed", "llada_decode", "dream_mixed", "dream_decode", "dream_prefill",
                             "prefill_heavy", "long_decode", "token_cache"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep-batches", default="1,2,4,8,16,32,64",
                    help="comma-separated batch sizes (--decode-sweep)")
    ap.add_argument("--sweep-cpu-budget", type=float, default=1.0,
                    help="seconds of oracle work per point (--decode-sweep)")
    ap.add_argument("--kv-cpu-budget", type=float, default=2.0,
                    help="seconds of oracle work per batch (--kv-transfer)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="run one device-to-device copy of this many MiB before warm-up, as the "
                         "reference kernel that scales the HBM traffic counters")
    ap.add_argument("--decode-sweep", action="store_true",
                    help="instead of one workload: block-decode batches of 1..64 requests at L = 1024 "
                         "for the LLaDA (32/32) and Dream (28/4) head shapes, one JSON line each")
    ap.add_argument("--serve-trace", action="store_true",
                    help="instead of one workload: a serving loop over a synthetic request trace, each "
                         "iteration's microbatch composed by the deficit token-budget rule (Dream 28/4 heads)")
    ap.add_argument("--tau", type=int, default=4096, help="token budget per iteration (--serve-trace)")
    ap.add_argument("--trace-iters", type=int, default=600, help="iterations (--serve-trace)")
    ap.add_argument("--trace-rate", type=float, default=0.3, help="requests per iteration (--serve-trace)")
    ap.add_argument("--kv-transfer", action="store_true",
                    help="time the paged-KV export / import of three batches' cached contexts")
    ap.add_argument("--flushed-reps", type=int, default=50,
                    help="steps timed after the timed region, each after a 1 GiB read (outside the "
                         "timing) that evicts the previous step's data from the 256 MB Infinity "
                         "Cache; reported as median and min. A read, not a write: written lines "
                         "would be written back to HBM during the next step")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the measured HBM-read and MFMA ceilings")
    ap.add_argument("--ceiling-reps", type=int, default=5)
    ap.add_argument("--ceilings", action="store_true",
                    help="instead of a workload: print the measured ceilings as one JSON line")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1).", file=sys.stderr)
        sys.exit(2)
    if args.decode_sweep:
        decode_sweep(args)
        return
    if args.serve_trace:
        serve_trace(args)
        return
    if args.kv_transfer:
        kv_transfer(args)
        return
    if args.ceilings:
        print(json.dumps({"ceilings": measure_ceilings(args)}), flush=True)
        return

    bench_workload(args)


def measure_ceilings(args):
    """Measured ceilings of the chip (HIP events around one probe launch,
    median of the reps): a streaming read of a 4 GiB buffer (16 times the
    256 MB Infinity Cache, so the figure is HBM) and a matrix-core loop of
    independent bf16 MFMAs."""
    import numpy as np
    import torch

    from paper_2607_04206_amd._lib import check, lib

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    res = {}
    nbytes = 4 << 30
    buf = torch.ones((nbytes // 4,), dtype=torch.int32, device=dev)
    grid = 8192
    sink = torch.empty((grid,), dtype=torch.int32, device=dev)
    times = []
    for r in range(3 + args.ceiling_reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        check(lib.sangam_probe_hbm_read(buf.data_ptr(), nbytes, sink.data_ptr(), grid, stream.cuda_stream))
        b.record(stream)
        b.synchronize()
        if r >= 3:
            times.append(a.elapsed_time(b) / 1e3)
    res["hbm_read_gbs"] = nbytes / float(np.median(times)) / 1e9
    res["hbm_read"] = "4 GiB streaming read, 16-byte loads, 8192 work-groups of 256 threads"
    del buf, sink
    grid, iters = 2048, 2048
    sinkf = torch.empty((grid,), dtype=torch.float32, device=dev)
    flops = grid * 4 * iters * 8 * 32768.0
    times = []
    for r in range(2 + args.ceiling_reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        check(lib.sangam_probe_mfma_bf16(sinkf.data_ptr(), grid, iters, stream.cuda_stream))
        b.record(stream)
        b.synchronize()
        if r >= 2:
            times.append(a.elapsed_time(b) / 1e3)
    res["mfma_bf16_tflops"] = flops / float(np.median(times)) / 1e12
    res["mfma"] = "v_mfma_f32_32x32x16_bf16, 8 independent chains per wave, 2048 work-groups of 4 waves"
    return res


def bench_workload(args):
    """One workload: warm-up, a per-launch breakdown, the timed region of K
    back-to-back steps, then R flushed steps (each after a 1 GiB read) timed
    with events, the measured ceilings and the oracle on a CPU sample."""
    import ctypes

    import numpy as np
    import torch

    import workloads
    from paper_2607_04206_amd import attn
    from paper_2607_04206_amd._lib import check, lib

    dev = torch.device("cuda:0")
    wl = getattr(workloads, args.workload)(args.seed)
    print(f"[bench] {wl.name} seed {wl.seed}: drawing inputs", file=sys.stderr, flush=True)
    t = workloads.device_inputs(wl, dev, fill=None)

    plan_kw = dict(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                   page_ids=wl.page_ids, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                   head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale, q_pos=wl.q_pos)
    attn.plan(**plan_kw)  # first call sizes the binding's planning buffer
    plan_times = []
    for _ in range(5):
        t0 = time.perf_counter()
        p = attn.plan(**plan_kw)
        plan_times.append((time.perf_counter() - t0) * 1e3)
    plan_ms = float(np.median(plan_times))
    p.to(dev)
    T, Hq, D = wl.total_q, wl.num_q_heads, wl.head_dim
    out = torch.empty((T, Hq, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((T, Hq), dtype=torch.float32, device=dev)
    ws = torch.empty((max(p.workspace_bytes, 16),), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    args_c = attn.c_args(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"],
                         out, lse, ws, stream)
    ran = {"prefill_attn": p.info.num_prefill_tiles > 0, "decode_attn": p.info.num_decode_tiles > 0,
           "merge": p.info.num_split_items > 0}

    def make_events(which=range(3)):
        """Start / stop event pairs of the three launches; launches outside
        `which` get NULL entries (no timestamps)."""
        evs = [torch.cuda.Event(enable_timing=True) if j // 2 in which else None for j in range(6)]
        for e in evs:
            if e is not None:
                e.record(stream)  # creates the HIP event
        arr = (ctypes.c_void_p * 6)(*[e.cuda_event if e is not None else None for e in evs])
        return evs, arr

    flush_buf = torch.ones((1 << 28,), dtype=torch.float32, device=dev)  # 1 GiB, read between flushed steps
    if args.copy_calib_mib > 0:
        src = torch.ones((args.copy_calib_mib << 20,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        check(lib.sangam_attn_forward(*args_c))
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    # per-launch breakdown, outside the timed region: events on all three
    # launches; a launch with no work reports null
    K = args.steps
    n_phase = max(3, min(K, 10))
    evsets = [make_events() for _ in range(n_phase)]
    torch.cuda.synchronize()
    for k in range(n_phase):
        check(lib.sangam_attn_forward_timed(*args_c, evsets[k][1]))
    torch.cuda.synchronize()
    phase_ms = {}
    for j, name in enumerate(PHASES):
        phase_ms[name] = (float(np.mean([evsets[k][0][2 * j].elapsed_time(evsets[k][0][2 * j + 1])
                                         for k in range(n_phase)])) if ran[name] else None)
    work = split_work(wl, fused_decodes=int(p.info.num_fused_decode_tiles) > 0)
    dom = max((n for n in ("prefill_attn", "decode_attn") if ran[n]), key=lambda n: phase_ms[n])
    jd = PHASES.index(dom)

    # timed region: K whole steps back to back; only the dominant launch
    # carries events (in its dispatch)
    evsets = [make_events((jd,)) for _ in range(K)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(K):
        check(lib.sangam_attn_forward_timed(*args_c, evsets[k][1]))
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - w0) * 1e3 / K
    dom_all = np.array([evsets[k][0][2 * jd].elapsed_time(evsets[k][0][2 * jd + 1]) for k in range(K)])
    print(f"[bench] timed {K} steps: {ms_per_step:.4f} ms/step", file=sys.stderr, flush=True)

    # flushed protocol: before each rep a 1 GiB read (outside the timing)
    # evicts the previous rep's data from the 256 MB Infinity Cache; the step
    # and the dominant launch are timed with events
    R = max(args.flushed_reps, 0)
    evsets = [make_events((jd,)) for _ in range(R)]
    step_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(R)]
    torch.cuda.synchronize()
    for k in range(R):
        flush_buf.sum()
        step_ev[k][0].record(stream)
        check(lib.sangam_attn_forward_timed(*args_c, evsets[k][1]))
        step_ev[k][1].record(stream)
    torch.cuda.synchronize()
    fl_step = np.array([a.elapsed_time(b) for a, b in step_ev])
    fl_dom = np.array([evsets[k][0][2 * jd].elapsed_time(evsets[k][0][2 * jd + 1]) for k in range(R)])
    if R:
        print(f"[bench] flushed {R} steps: median {np.median(fl_step):.4f} ms", file=sys.stderr, flush=True)
    del flush_buf

    F, B = wl.flops(), wl.hbm_bytes()
    sec = ms_per_step / 1e3
    tflops, gbs = F / sec / 1e12, B / sec / 1e9
    t_star = max(F / (PEAK_BF16_TFLOPS * 1e12), B / (PEAK_HBM_GBS * 1e9))

    ceil = None
    if not args.no_ceilings:
        print("[bench] measuring the chip's ceilings", file=sys.stderr, flush=True)
        ceil = measure_ceilings(args)

    f_d, b_d = work[dom]
    dom_ms = float(dom_all.mean())
    t_d = dom_ms / 1e3
    intensity = f_d / max(b_d, 1.0)
    if intensity >= PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": f_d / t_d / 1e12, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
        rate = lambda ms: f_d / (ms / 1e3) / 1e12
        measured_peak = ceil["mfma_bf16_tflops"] if ceil else None
    else:
        roof = {"bound": "hbm", "achieved": b_d / t_d / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
        rate = lambda ms: b_d / (ms / 1e3) / 1e9
        measured_peak = ceil["hbm_read_gbs"] if ceil else None
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = measured_traffic(args.workload, dom)  # summaries are named by the --workload value
    roof["kernel"] = dom
    roof["kernel_ms"] = dom_ms
    roof["kernel_ms_median"] = float(np.median(dom_all))
    roof["kernel_ms_min"] = float(dom_all.min())
    roof["flushed"] = None
    if R:
        roof["flushed"] = {"kernel_ms_median": float(np.median(fl_dom)), "kernel_ms_min": float(fl_dom.min()),
                           "achieved_median": rate(float(np.median(fl_dom))),
                           "frac_median": rate(float(np.median(fl_dom))) / roof["peak"],
                           "step_ms_median": float(np.median(fl_step)), "step_ms_min": float(fl_step.min()),
                           "reps": R, "flush": "1 GiB read between reps, outside the timing"}
    if measured_peak:
        roof["measured_peak"] = measured_peak
        roof["frac_of_measured"] = roof["achieved"] / measured_peak
        if R:
            roof["flushed"]["frac_of_measured_median"] = roof["flushed"]["achieved_median"] / measured_peak
    roof["algorithmic_flops"] = f_d
    roof["algorithmic_bytes"] = b_d

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on a CPU sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, args.cpu_budget)

    n_dec = int((np.diff(wl.q_indptr) <= 32).sum())
    res = {
        "metric": METRIC,
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "seed": wl.seed, "block_decodes": n_dec,
                   "prefills": wl.num_items - n_dec, "num_q_heads": wl.num_q_heads,
                   "num_kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim, "page_size": 16,
                   "query_rows": T, "context_tokens": int(wl.kv_len.sum()),
                   "parallelism": "1 GPU"},
        "tflops": tflops,
        "hbm_gbs": gbs,
        "mfma_frac": tflops / PEAK_BF16_TFLOPS,
        "hbm_frac": gbs / PEAK_HBM_GBS,
        "roofline_frac": t_star / sec,
        "algorithmic_flops": F,
        "algorithmic_bytes": B,
        "flushed_step_ms_median": float(np.median(fl_step)) if R else None,
        "flushed_step_ms_min": float(fl_step.min()) if R else None,
        "phase_ms": phase_ms,
        "plan_ms": plan_ms,
        "kernel_source_hash": kernel_source_hash(),
        "ceilings": ceil,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)

if __name__ == "__main__":
    main()
