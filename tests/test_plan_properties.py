"""Randomised planner properties (hypothesis): for arbitrary ragged batches
(block decodes, cached blocks of more than 32 rows, per-token position
lists, prefills), head shapes, forced
split counts and CU counts, the plan's work-groups tile every (query head,
row, key) of every item exactly once, respect the range limit of tiles that
read cached rows, list exactly the rows of split items for the merge, and
keep the split partial buffers inside the workspace. Host only."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import workloads
from tests.test_plan import HEADS_ACROSS, parse

MAX_CACHED_RANGE = 8192
SHAPES = [(4, 4), (8, 4), (12, 4), (28, 4), (32, 8), (16, 2), (11, 1), (8, 1), (6, 6), (24, 8)]


@st.composite
def batches(draw):
    hq, hkv = draw(st.sampled_from(SHAPES))
    d = draw(st.sampled_from([64, 128]))
    n_dec = draw(st.integers(0, 6))
    n_pos = draw(st.integers(0, 2))
    n_pre = draw(st.integers(0 if n_dec + n_pos else 1, 3))
    decodes = []
    for _ in range(n_dec):
        L = draw(st.integers(1, 20000))
        o = draw(st.integers(0, L - 1))
        decodes.append((o, L))
    pos = []
    for _ in range(n_pos):
        L = draw(st.integers(2, 3000))
        k = draw(st.integers(1, min(32, L - 1)))
        p = sorted(draw(st.sets(st.integers(0, L - 1), min_size=k, max_size=k)))
        pos.append((p, L))
    for _ in range(draw(st.integers(0, 2))):  # cached blocks of more than 32 rows
        L = draw(st.integers(34, 20000))
        n = draw(st.integers(33, min(300, L)))
        decodes.append((draw(st.integers(0, L - n)), L, n))
    prefills = [draw(st.integers(1, 700)) for _ in range(n_pre)]
    force = draw(st.sampled_from([0, 0, 0, 1, 2, 3, 7]))
    cus = draw(st.sampled_from([0, 8, 64, 256]))
    seed = draw(st.integers(0, 1000))
    wl = workloads.make_workload("prop", seed, hq=hq, hkv=hkv, d=d, decodes=decodes, prefills=prefills,
                                 pos_decodes=pos)
    return wl, force, cus


def check_plan(wl, force, cus):
    from paper_2607_04206_amd import attn
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                  page_ids=wl.page_ids, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                  head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale,
                  force_kv_splits=force, num_cus=cus, q_pos=wl.q_pos)
    h, items, dec, pre, mer = parse(p)
    G = wl.num_q_heads // wl.num_kv_heads
    qw, rows_pt = int(h["decode_qw"]), int(h["prefill_rows"])
    waves = rows_pt // 32
    # rectangles (row range x key range) per (item, query head)
    rects = {}

    def add(i, hd, r0, r1, k0, k1):
        assert 0 <= r0 < r1 <= wl.n(i) and 0 <= k0 < k1 <= int(wl.kv_len[i])
        rects.setdefault((i, hd), []).append((r0, r1, k0, k1))

    for t in dec:
        i = int(t["item"])
        assert wl.n(i) <= 32 and int(t["row0"]) == 0 and not t["flags"] & HEADS_ACROSS
        for hd in range(int(t["q_head0"]), int(t["q_head0"]) + qw):
            assert hd // G == t["kv_head"]
            add(i, hd, 0, wl.n(i), int(t["kv_begin"]), int(t["kv_end"]))
    for t in pre:
        i = int(t["item"])
        hd0 = int(t["q_head0"])
        assert hd0 // G == t["kv_head"]
        if t["flags"] & HEADS_ACROSS:
            assert wl.n(i) <= 32 and G >= 4
            for hd in range(hd0, min(hd0 + waves, (int(t["kv_head"]) + 1) * G)):
                add(i, hd, 0, wl.n(i), int(t["kv_begin"]), int(t["kv_end"]))
        else:
            assert wl.n(i) > 32
            r0 = int(t["row0"])
            add(i, hd0, r0, min(r0 + rows_pt, wl.n(i)), int(t["kv_begin"]), int(t["kv_end"]))
    for t in np.concatenate([dec, pre]):
        it = items[int(t["item"])]
        all_fresh = int(it["o"]) == 0 and int(it["n"]) == int(it["L"])
        if not all_fresh:
            assert int(t["kv_end"]) - int(t["kv_begin"]) <= MAX_CACHED_RANGE
        # the tile's range is its split's chunk
        s = int(t["split"])
        assert int(t["kv_begin"]) == s * int(it["split_len"])
        assert int(t["kv_end"]) == min(int(it["L"]), (s + 1) * int(it["split_len"]))
    # exact partition: inside the domain, pairwise disjoint, areas add up
    for i in range(wl.num_items):
        n, L = wl.n(i), int(wl.kv_len[i])
        for hd in range(wl.num_q_heads):
            rs = sorted(rects.get((i, hd), []))
            area = sum((r1 - r0) * (k1 - k0) for r0, r1, k0, k1 in rs)
            assert area == n * L, (i, hd, area, n * L)
            for a in range(len(rs)):
                for b in range(a + 1, len(rs)):
                    ra, rb = rs[a], rs[b]
                    overlap = min(ra[1], rb[1]) > max(ra[0], rb[0]) and min(ra[3], rb[3]) > max(ra[2], rb[2])
                    assert not overlap, (i, hd, ra, rb)
    # merge rows: exactly the rows of split items, in item order
    want = [(i, r) for i in range(wl.num_items) if items[i]["num_splits"] > 1 for r in range(wl.n(i))]
    assert [(int(m["item"]), int(m["row"])) for m in mer] == want
    # split partials inside the workspace and disjoint
    spans = []
    for it in items:
        S = int(it["num_splits"])
        assert S * int(it["split_len"]) >= int(it["L"]) > (S - 1) * int(it["split_len"])
        assert int(it["split_len"]) % 64 == 0 or S == 1
        if S > 1:
            spans.append((int(it["ws_o"]), int(it["ws_o"]) + S * int(it["n"]) * wl.num_q_heads * wl.head_dim))
            spans.append((int(it["ws_lse"]), int(it["ws_lse"]) + S * int(it["n"]) * wl.num_q_heads))
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    if spans:
        assert spans[-1][1] * 4 <= p.workspace_bytes
    if force > 0:
        # one 64-aligned chunk length from min(force, ceil(L / 64)) chunks,
        # unless the range limit of cached keys asks for more
        for i, it in enumerate(items):
            L, S = int(it["L"]), int(it["num_splits"])
            k = min(force, -(-L // 64))
            all_fresh = int(it["o"]) == 0 and int(it["n"]) == L
            if not all_fresh:
                k = max(k, -(-L // MAX_CACHED_RANGE))
            want_len = -(-(-(-L // k)) // 64) * 64
            assert int(it["split_len"]) == (want_len if S > 1 else int(it["split_len"]))
            assert S == -(-L // want_len), (L, force, S)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(batches())
def test_plan_partitions_every_item(case):
    wl, force, cus = case
    check_plan(wl, force, cus)
