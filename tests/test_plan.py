"""Host planner: descriptor validation, tile coverage, split rules, ordering.
Runs without a GPU (the planner makes no HIP call)."""
import ctypes

import numpy as np
import pytest

import workloads
from paper_2607_04206_amd import attn
from paper_2607_04206_amd._lib import SangamError, lib

# Internal blob layout (plan_format.h), read here only to check coverage.
HEADER = np.dtype([
    ("magic", "<u4"), ("version", "<u4"), ("total_bytes", "<u8"),
    ("num_items", "<i4"), ("hq", "<i4"), ("hkv", "<i4"), ("d", "<i4"), ("group", "<i4"),
    ("page_size", "<i4"), ("sm_scale", "<f4"), ("scale_log2", "<f4"),
    ("num_pool_pages", "<i8"), ("total_q", "<i8"), ("total_pages", "<i8"),
    ("n_decode_tiles", "<i4"), ("decode_qw", "<i4"), ("decode_kw", "<i4"), ("decode_nb", "<i4"),
    ("n_prefill_tiles", "<i4"), ("prefill_nb", "<i4"), ("n_merge_rows", "<i4"),
    ("num_split_items", "<i4"), ("max_splits", "<i4"), ("prefill_rows", "<i4"),
    ("n_fused_decode_tiles", "<i4"), ("reserved", "<i4"), ("workspace_bytes", "<i8"),
    ("off_items", "<u8"), ("off_decode_tiles", "<u8"), ("off_prefill_tiles", "<u8"), ("off_merge", "<u8"),
    ("off_positions", "<u8"), ("off_page_info", "<u8"),
])
ITEM = np.dtype([("q_start", "<i4"), ("n", "<i4"), ("o", "<i4"), ("L", "<i4"), ("page_start", "<i4"),
                 ("num_splits", "<i4"), ("split_len", "<i4"), ("merge_base", "<i4"),
                 ("ws_o", "<i8"), ("ws_lse", "<i8"), ("flags", "<i4"), ("pos_start", "<i4")])
POS_LIST = 1
TILE = np.dtype([("item", "<i4"), ("kv_head", "<i4"), ("q_head0", "<i4"), ("row0", "<i4"),
                 ("kv_begin", "<i4"), ("kv_end", "<i4"), ("split", "<i4"), ("flags", "<i4")])
HEADS_ACROSS = 1
MERGE = np.dtype([("item", "<i4"), ("row", "<i4")])


def parse(p):
    b = p.host
    h = np.frombuffer(b, HEADER, count=1)[0]
    items = np.frombuffer(b, ITEM, count=int(h["num_items"]), offset=int(h["off_items"]))
    dec = np.frombuffer(b, TILE, count=int(h["n_decode_tiles"]), offset=int(h["off_decode_tiles"]))
    pre = np.frombuffer(b, TILE, count=int(h["n_prefill_tiles"]), offset=int(h["off_prefill_tiles"]))
    mer = np.frombuffer(b, MERGE, count=int(h["n_merge_rows"]), offset=int(h["off_merge"]))
    return h, items, dec, pre, mer


def plan_of(wl, **kw):
    return attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len,
                     page_indptr=wl.page_indptr, page_ids=wl.page_ids,
                     num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                     head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages,
                     sm_scale=wl.sm_scale, q_pos=wl.q_pos, **kw)


def test_header_size_matches():
    # plan_format.h static_asserts the same sizes on the C side
    p = plan_of(workloads.tiny_mixed(0))
    h, *_ = parse(p)
    assert h["magic"] == 0x50414753 and h["version"] == 4
    assert h["total_bytes"] == p.host.nbytes
    assert HEADER.itemsize == 176 and ITEM.itemsize == 56 and TILE.itemsize == 32


def coverage(wl, p):
    """Count how often each (item, q-head, row, key) is covered by a tile."""
    h, items, dec, pre, _ = parse(p)
    G = wl.num_q_heads // wl.num_kv_heads
    qw = int(h["decode_qw"])
    rows = int(h["prefill_rows"])
    cover = {}
    for i in range(wl.num_items):
        cover[i] = np.zeros((wl.num_q_heads, wl.n(i), int(wl.kv_len[i])), np.int32)
    for t in dec:
        i = int(t["item"])
        assert wl.n(i) <= 32
        for hd in range(int(t["q_head0"]), int(t["q_head0"]) + qw):
            assert hd // G == t["kv_head"]
            cover[i][hd, :, t["kv_begin"]:t["kv_end"]] += 1
    waves = rows // 32
    for t in pre:
        i = int(t["item"])
        hd = int(t["q_head0"])
        assert hd // G == t["kv_head"]
        if t["flags"] & HEADS_ACROSS:
            # a block decode in the prefill launch: one head per wave, only
            # those inside the tile's GQA group
            assert wl.n(i) <= 32 and t["row0"] == 0
            for h2 in range(hd, min(hd + waves, (int(t["kv_head"]) + 1) * G)):
                cover[i][h2, :, t["kv_begin"]:t["kv_end"]] += 1
            continue
        assert wl.n(i) > 32 and t["flags"] == 0
        r0 = int(t["row0"])
        cover[i][hd, r0:r0 + rows, t["kv_begin"]:t["kv_end"]] += 1
    return cover


@pytest.mark.parametrize("mk", [
    lambda: workloads.tiny_mixed(0),
    lambda: workloads.ragged_small(0, hq=4, hkv=4, d=64),
    lambda: workloads.ragged_small(0, hq=28, hkv=4, d=128),
    lambda: workloads.ragged_small(0, hq=8, hkv=4, d=128),
    lambda: workloads.ragged_small(0, hq=18, hkv=2, d=64),
    lambda: workloads.ragged_small(0, hq=11, hkv=1, d=128),
    lambda: workloads.llada_decode(1),
    lambda: workloads.dream_mixed(2),
    lambda: workloads.make_workload("g7", 3, hq=28, hkv=4, d=128, decodes=[(0, 9000), (64, 300)],
                                    prefills=[200]),
    lambda: workloads.make_workload("g2", 4, hq=8, hkv=4, d=64, decodes=[(32, 700)], prefills=[100]),
    lambda: workloads.token_cache_decodes(2, hq=8, hkv=8, d=64, count=5),
    lambda: workloads.token_cache_decodes(3, hq=28, hkv=4, d=128, count=4, prefills=[150]),
    lambda: workloads.make_workload("mb", 5, hq=28, hkv=4, d=128, prefills=[150],
                                    decodes=[(100, 500, 64), (37, 300, 33), (1500, 9000, 200), (20, 700)]),
    lambda: workloads.make_workload("mbm", 6, hq=8, hkv=8, d=64, prefills=[],
                                    decodes=[(0, 2000, 300), (4500, 9000, 100), (8190, 8400, 150)]),
])
@pytest.mark.parametrize("force", [0, 1, 3, 8])
def test_every_row_head_key_covered_once(mk, force):
    wl = mk()
    p = plan_of(wl, force_kv_splits=force)
    for i, c in coverage(wl, p).items():
        assert c.min() == 1 and c.max() == 1, f"item {i}"


def test_block_decodes_fuse_into_prefill_launch():
    # GQA groups of >= 4 heads: a mixed batch runs its block decodes as
    # heads-across tiles of the prefill launch, unsplit below 8192 keys
    wl = workloads.dream_mixed(0)
    p = plan_of(wl)
    h, items, dec, pre, mer = parse(p)
    n_dec = sum(1 for i in range(wl.num_items) if wl.n(i) <= 32)
    G = wl.num_q_heads // wl.num_kv_heads
    assert len(dec) == 0 and len(mer) == 0 and p.workspace_bytes == 0
    fused = pre[(pre["flags"] & HEADS_ACROSS) != 0]
    assert len(fused) == h["n_fused_decode_tiles"] == p.info.num_fused_decode_tiles
    assert len(fused) == n_dec * wl.num_kv_heads * -(-G // 4)
    # longest first: every prefill tile is at least as long as any fused one
    cost = (pre["kv_end"] - pre["kv_begin"]).astype(np.int64) * 4
    assert np.all(np.diff(cost) <= 0)
    # a decode context over 8192 keys is still split (and merged)
    wl2 = workloads.make_workload("g7", 3, hq=28, hkv=4, d=128, decodes=[(0, 9000), (64, 300)],
                                  prefills=[200])
    p2 = plan_of(wl2)
    _, items2, dec2, pre2, mer2 = parse(p2)
    assert len(dec2) == 0
    assert items2[0]["num_splits"] == 2 and items2[1]["num_splits"] == 1
    assert len(mer2) == wl2.n(0)
    # pure decode batches and small groups keep the decode launch
    for wl3 in (workloads.llada_decode(0),
                workloads.make_workload("g2", 4, hq=8, hkv=4, d=64, decodes=[(32, 700)], prefills=[100])):
        p3 = plan_of(wl3)
        _, _, dec3, pre3, _ = parse(p3)
        assert len(dec3) > 0 and not np.any(pre3["flags"] & HEADS_ACROSS)
        assert p3.info.num_fused_decode_tiles == 0


def test_small_decode_only_gqa_batch_fuses():
    # a decode-only batch of 28/4-head block decodes too small to fill the CUs
    # takes heads-across tiles, its contexts cut to about two work-groups per
    # CU; a large one keeps the whole-group decode tiles
    for B, fused in ((1, True), (8, True), (16, True), (64, False)):
        wl = workloads.decode_sweep("dream", B, 0)
        p = plan_of(wl)
        h, items, dec, pre, mer = parse(p)
        if fused:
            assert len(dec) == 0 and len(pre) == p.info.num_fused_decode_tiles > 0
            assert np.all(pre["flags"] & HEADS_ACROSS)
            n_tiles = sum(int(it["num_splits"]) for it in items) * wl.num_kv_heads * 2
            assert len(pre) == n_tiles
            assert 128 <= n_tiles <= 2 * 256 or B == 1
            assert np.all(items["split_len"] >= 256)
        else:
            assert len(pre) == 0 and len(dec) > 0 and p.info.decode_q_waves == 7


def test_underfilled_decode_launch_cut_to_resident_work_groups():
    # a decode-only batch whose whole-context tiles leave resident slots idle
    # (two MHA or one GQA whole-group work-group per CU) is cut with the
    # shortest chunk (from the floor: 256 keys MHA, 512 GQA; 64-aligned)
    # whose tiles still fit in those slots
    def cdiv(a, b):
        return -(-a // b)

    def tiles_at(wl, c):
        return sum(wl.num_kv_heads * cdiv(int(L), c) for L in wl.kv_len)

    base = workloads.dream_mixed(0)
    dec = [(int(base.q_offset[i]), int(base.kv_len[i])) for i in range(base.num_items) if not base.is_prefill[i]]
    cases = [(workloads.make_workload("dreamdec", 0, hq=28, hkv=4, d=128, decodes=dec, prefills=[]), 256),
             (workloads.decode_sweep("dream", 32, 0), 256), (workloads.decode_sweep("dream", 32, 0), 200)]
    cases += [(workloads.decode_sweep("llada", B, 0), 256) for B in (1, 6, 8, 12, 15)]
    for wl, cus in cases:
        p = plan_of(wl, num_cus=cus)
        h, items, dec_t, pre, mer = parse(p)
        mha = wl.num_q_heads == wl.num_kv_heads
        assert len(pre) == 0 and p.info.decode_q_waves == (1 if mha else 7)
        slots = cus * (2 if mha else 1)
        assert wl.num_items * wl.num_q_heads // p.info.decode_q_waves < slots  # underfilled without splits
        floor = 256 if mha else 512
        chunk = max(floor, next(c for c in range(floor, 8192 + 1, 64) if tiles_at(wl, c) <= slots))
        for it, L in zip(items, wl.kv_len):
            pieces = cdiv(int(L), chunk)
            length = 64 * cdiv(cdiv(int(L), pieces), 64)  # 64-aligned piece length
            assert int(it["num_splits"]) == cdiv(int(L), length), (int(L), chunk)
        assert len(dec_t) == sum(wl.num_kv_heads * int(it["num_splits"]) for it in items) <= slots
    # one LLaDA decode still takes its four 256-key pieces (the floor binds)
    assert plan_of(workloads.decode_sweep("llada", 1, 0), num_cus=256).info.num_decode_tiles == 4 * 32
    # the uniform 32-decode batch keeps its two pieces per context at 256 CUs
    p = plan_of(workloads.decode_sweep("dream", 32, 0), num_cus=256)
    assert p.info.num_split_items == 32 and p.info.num_decode_tiles == 256


def test_splits_and_merge_rows():
    wl = workloads.make_workload("long", 0, hq=4, hkv=4, d=128,
                                 decodes=[(100, 9000), (0, 8192), (5, 300)], prefills=[20000])
    p = plan_of(wl)
    h, items, dec, pre, mer = parse(p)
    # a decode context over 8192 keys is always split; chunks are 64-aligned
    assert items[0]["num_splits"] >= 2
    assert items[0]["split_len"] % 64 == 0 and items[0]["split_len"] <= 8192
    assert items[1]["split_len"] <= 8192
    # prefill-shaped items are not split by default
    assert items[3]["num_splits"] == 1
    # merge rows list exactly the rows of split items
    want = [(i, r) for i in range(4) if items[i]["num_splits"] > 1 for r in range(wl.n(i))]
    assert [(int(m["item"]), int(m["row"])) for m in mer] == want
    # partial buffers do not overlap and fit in the workspace
    spans = []
    for it in items:
        if it["num_splits"] > 1:
            S, n = int(it["num_splits"]), int(it["n"])
            spans.append((int(it["ws_o"]), int(it["ws_o"]) + S * n * 4 * 128))
            spans.append((int(it["ws_lse"]), int(it["ws_lse"]) + S * n * 4))
    spans.sort()
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] * 4 <= p.workspace_bytes
    starts = p.item_splits(0)
    assert starts[0] == 0 and starts[-1] == 9000 and np.all(np.diff(starts) > 0)


def test_forced_split_count():
    wl = workloads.llada_decode(0)
    for k in (1, 2, 4, 8):
        p = plan_of(wl, force_kv_splits=k)
        _, items, *_ = parse(p)
        for i, it in enumerate(items):
            L = int(wl.kv_len[i])
            assert it["num_splits"] == min(k, -(-L // 64)) or it["num_splits"] <= k
            assert it["num_splits"] * it["split_len"] >= L > (it["num_splits"] - 1) * it["split_len"]
        if k == 1:
            assert p.workspace_bytes == 0


XCDS = 8


def xcd_slots(h, num_cus=256):
    """Work-group slots per XCD of the prefill-shaped launch."""
    return max(1, num_cus // XCDS) * (1 if int(h["prefill_rows"]) == 256 else 2)


def undo_xcd_order(tiles, C):
    """The launch order of a long prefill-shaped launch gives XCD x (blocks
    b = x mod 8) the C consecutive tiles [x C, (x + 1) C) of every chunk of
    8 C tiles of the longest-first list (a last, partial chunk of M tiles
    keeps the same layout over M // 8 and its remainder in order). Returns
    the longest-first list."""
    out = np.empty_like(tiles)
    for base in range(0, len(tiles), XCDS * C):
        M = min(XCDS * C, len(tiles) - base)
        c = M // XCDS
        for q in range(M):
            src = base + XCDS * (q % c) + q // c if q < XCDS * c else base + q
            out[base + q] = tiles[src]
    return out


def prefill_costs(h, items, pre):
    # cost = keys x waves holding rows (a fused block decode keeps all four busy)
    waves = int(h["prefill_rows"]) // 32
    rows = np.minimum(int(h["prefill_rows"]), items["n"][pre["item"]] - pre["row0"])
    return (pre["kv_end"] - pre["kv_begin"]) * np.where(pre["flags"] & HEADS_ACROSS, waves, (rows + 31) // 32)


def test_longest_first():
    for wl in (workloads.dream_mixed(0), workloads.llada_decode(0),
               workloads.make_workload("m", 5, hq=8, hkv=8, d=128, decodes=[(0, 3000), (32, 900)],
                                       prefills=[300, 1000])):
        p = plan_of(wl)
        h, items, dec, pre, _ = parse(p)
        dc = dec["kv_end"] - dec["kv_begin"]
        assert np.all(np.diff(dc) <= 0)
        assert len(pre) < 8 * XCDS * xcd_slots(h)  # a short launch: plain longest-first order
        assert np.all(np.diff(prefill_costs(h, items, pre)) <= 0)


def test_long_prefill_launch_takes_the_xcd_order():
    """prefill-heavy (26 rounds of wide tiles): undoing the XCD order gives a
    longest-first list, and within full chunks an XCD's 32 tiles are row
    blocks of at most three query heads (19-46 row blocks per head), all but
    the runs of each head's last, shorter row block, which longest-first
    order groups across heads."""
    wl = workloads.prefill_heavy(0)
    h, items, dec, pre, _ = parse(plan_of(wl))
    C = xcd_slots(h)
    assert len(pre) >= 8 * XCDS * C
    lpt = undo_xcd_order(pre, C)
    assert np.all(np.diff(prefill_costs(h, items, lpt)) <= 0)
    assert not np.array_equal(lpt, pre)
    # the tiles are those of the plain longest-first list, each once
    key = lambda t: (t["item"], t["q_head0"], t["row0"], t["kv_begin"])
    assert sorted(map(key, pre)) == sorted(map(key, lpt))
    runs = local = 0
    for base in range(0, len(pre) - XCDS * C + 1, XCDS * C):
        for x in range(XCDS):
            mine = pre[base + x: base + XCDS * C: XCDS]
            assert np.array_equal(mine, lpt[base + x * C: base + (x + 1) * C])
            runs += 1
            local += len(set(zip(mine["item"], mine["q_head0"]))) <= 3
    assert local >= 0.95 * runs, (local, runs)


@pytest.mark.parametrize("hq,xcd", [(8, False), (16, True)])
def test_xcd_order_threshold(hq, xcd):
    """Eight rounds of tiles per slot switch the order: one 2000-row prefill
    in wide tiles (8 row blocks per head) on 16 CUs (two slots per XCD) gives
    64 tiles (4 rounds) at 8 heads and 128 (8 rounds) at 16 heads."""
    wl = workloads.make_workload("xcd", 2, hq=hq, hkv=hq, d=128, decodes=[], prefills=[2000])
    h, items, dec, pre, _ = parse(plan_of(wl, num_cus=16))
    assert int(h["prefill_rows"]) == 256 and len(pre) == 8 * hq
    lpt = undo_xcd_order(pre, xcd_slots(h, 16)) if xcd else pre
    # longest first, ties in creation order (query head, then row block)
    cost = prefill_costs(h, items, lpt)
    assert np.array_equal(np.lexsort((lpt["row0"], lpt["q_head0"], -cost)), np.arange(len(lpt)))
    assert np.array_equal(lpt, pre) == (not xcd)


def test_deterministic_bytes():
    wl = workloads.dream_mixed(1)
    a = plan_of(wl).host
    b = plan_of(wl).host
    assert np.array_equal(a, b)


def test_decode_wave_shapes():
    for hq, hkv, qw, kw in [(32, 32, 1, 2), (8, 4, 2, 2), (28, 4, 7, 1), (24, 8, 3, 1),
                            (16, 1, 8, 1), (18, 2, 3, 1), (11, 1, 1, 2)]:
        wl = workloads.make_workload("s", 0, hq=hq, hkv=hkv, d=128, decodes=[(0, 64)], prefills=[])
        p = plan_of(wl)
        assert (p.info.decode_q_waves, p.info.decode_kv_waves) == (qw, kw), (hq, hkv)


# ---------------------------------------------------------------- validation
def _desc_kwargs(wl):
    return dict(q_indptr=wl.q_indptr.copy(), q_offset=wl.q_offset.copy(), kv_len=wl.kv_len.copy(),
                page_indptr=wl.page_indptr.copy(), page_ids=wl.page_ids.copy(),
                num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads, head_dim=wl.head_dim,
                num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale)


CODES = {"INVALID": -1, "UNSUPPORTED": -2, "PAGE_RANGE": -3, "PAGE_ALIAS": -4, "BUFFER": -5}


def _expect(code, **kw):
    with pytest.raises(SangamError) as e:
        attn.plan(**kw)
    assert e.value.status == CODES[code], str(e.value)
    assert len(lib.sangam_last_error()) > 0


def test_rejects_bad_descriptors():
    wl = workloads.ragged_small(0, hq=4, hkv=2, d=64)
    base = _desc_kwargs(wl)

    k = dict(base); k["head_dim"] = 96; _expect("UNSUPPORTED", **k)
    k = dict(base); k["num_kv_heads"] = 3; _expect("UNSUPPORTED", **k)
    k = dict(base); k["page_size"] = 32; _expect("UNSUPPORTED", **k)
    k = dict(base); k["sm_scale"] = float("nan"); _expect("INVALID", **k)
    k = dict(base); k["sm_scale"] = -1.0; _expect("INVALID", **k)
    k = dict(base); k["num_q_heads"] = 0; _expect("INVALID", **k)

    k = dict(base); qo = k["q_offset"].copy(); qo[0] = wl.kv_len[0]; k["q_offset"] = qo
    _expect("INVALID", **k)  # o + n > L
    k = dict(base); qo = k["q_offset"].copy(); qo[1] = -1; k["q_offset"] = qo
    _expect("INVALID", **k)
    k = dict(base); kl = k["kv_len"].copy(); kl[2] += 16; k["kv_len"] = kl
    _expect("INVALID", **k)  # page count no longer ceil(L/16)
    k = dict(base); qi = k["q_indptr"].copy(); qi[1] = qi[0]; k["q_indptr"] = qi
    _expect("INVALID", **k)  # n_0 = 0
    k = dict(base); pi = k["page_ids"].copy(); pi[3] = wl.num_pool_pages; k["page_ids"] = pi
    _expect("PAGE_RANGE", **k)
    k = dict(base); pi = k["page_ids"].copy(); pi[3] = -2; k["page_ids"] = pi
    _expect("PAGE_RANGE", **k)
    k = dict(base); pi = k["page_ids"].copy(); pi[5] = pi[1]; k["page_ids"] = pi
    _expect("PAGE_ALIAS", **k)


def test_zero_length_items_rejected():
    k = dict(q_indptr=[0, 1], q_offset=[0], kv_len=[0], page_indptr=[0, 0], page_ids=[],
             num_q_heads=1, num_kv_heads=1, head_dim=64, num_pool_pages=4, sm_scale=0.125)
    _expect("INVALID", **k)
    k = dict(q_indptr=[0], q_offset=[], kv_len=[], page_indptr=[0], page_ids=[],
             num_q_heads=1, num_kv_heads=1, head_dim=64, num_pool_pages=4, sm_scale=0.125)
    _expect("INVALID", **k)


def test_context_longer_than_2_30_rejected():
    """Tile key ranges are int32: a context past 2^30 positions is refused
    before its page table is read."""
    k = dict(q_indptr=[0, 32], q_offset=[0], kv_len=[(1 << 30) + 1], page_indptr=[0, 1], page_ids=[0],
             num_q_heads=1, num_kv_heads=1, head_dim=64, num_pool_pages=4, sm_scale=0.125)
    _expect("INVALID", **k)
    assert b"2^30" in lib.sangam_last_error()


def test_buffer_too_small_reports_size():
    from paper_2607_04206_amd._lib import SANGAM_OK
    wl = workloads.llada_decode(0)
    d, keep = attn.make_desc(**_desc_kwargs(wl))
    used = ctypes.c_size_t(0)
    st = lib.sangam_attn_plan(ctypes.byref(d), None, 0, ctypes.byref(used))
    assert st == CODES["BUFFER"] and used.value > 0
    buf = np.zeros(used.value - 1, np.uint8)
    st = lib.sangam_attn_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used))
    assert st == CODES["BUFFER"]
    buf = np.zeros(used.value, np.uint8)
    st = lib.sangam_attn_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used))
    assert st == SANGAM_OK
    del keep


def test_long_decode_plan_is_fast_and_sized():
    import time
    wl = workloads.long_decode(0)
    t = time.perf_counter()
    p = plan_of(wl)
    dt = time.perf_counter() - t
    assert dt < 2.0
    _, items, dec, pre, _ = parse(p)
    assert len(pre) == 0
    assert np.all(items["split_len"] <= 8192)
    assert np.all((items["L"] <= 8192) | (items["num_splits"] >= 2))


def test_decode_sweep_workloads():
    # decode-batch sweep points: B block decodes of 32 rows at L = 1024, block
    # index in the last 256 positions
    for shape in workloads.SWEEP_SHAPES:
        for B in (1, 64):
            wl = workloads.decode_sweep(shape, B)
            assert wl.num_items == B and (wl.kv_len == 1024).all()
            assert (np.diff(wl.q_indptr) == 32).all()
            assert ((wl.q_offset >= 768) & (wl.q_offset <= 992) & (wl.q_offset % 32 == 0)).all()


def test_underfilled_decode_launch_splits_finer():
    # fewer decode work-groups than two per CU: contexts are cut down to
    # 256-key chunks; a full launch keeps MHA chunks of at least 2048 keys
    small = plan_of(workloads.decode_sweep("llada", 1))
    h, items, dec, pre, mer = parse(small)
    assert len(pre) == 0 and items["num_splits"][0] == 4 and items["split_len"][0] == 256
    assert len(dec) == 32 * 4 and len(mer) == 32
    full = plan_of(workloads.decode_sweep("llada", 64))
    h, items, dec, pre, mer = parse(full)
    assert (items["num_splits"] == 1).all() and len(dec) == 64 * 32 and len(mer) == 0
    # the same batch on a 16-CU part counts as full
    h, items, dec, pre, mer = parse(plan_of(workloads.decode_sweep("llada", 1), num_cus=16))
    assert (items["num_splits"] == 1).all()


def test_position_list_items():
    # per-token cached decodes: scattered lists become kItemPosList items with
    # their positions and per-page slot masks in the blob; a contiguous list is
    # a plain block at its first position
    wl = workloads.make_workload("pl", 1, hq=4, hkv=2, d=64, decodes=[(40, 90)], prefills=[70],
                                 pos_decodes=[([3, 17, 18, 40, 95], 100), (range(10, 42), 60),
                                              ([0, 15, 16, 31, 32], 33)])
    p = plan_of(wl)
    h, items, dec, pre, mer = parse(p)
    assert [int(f) for f in items["flags"]] == [0, POS_LIST, 0, POS_LIST, 0]
    assert items["o"][2] == 10 and items["o"][1] == 3
    pos = np.frombuffer(p.host, np.int32, count=10, offset=int(h["off_positions"]))
    assert list(pos) == [3, 17, 18, 40, 95, 0, 15, 16, 31, 32]
    assert items["pos_start"][1] == 0 and items["pos_start"][3] == 5
    info = np.frombuffer(p.host, np.uint32, count=int(h["total_pages"]), offset=int(h["off_page_info"]))
    for i in (1, 3):
        listed = wl.positions(i)
        pages = range(int(wl.page_indptr[i]), int(wl.page_indptr[i + 1]))
        for k, e in enumerate(info[list(pages)]):
            slots = [int(x) - 16 * k for x in listed if x // 16 == k]
            assert int(e) & 0xFFFF == sum(1 << s_ for s_ in slots)
            assert int(e) >> 16 == int(np.sum(listed < 16 * k))
    # items without a list carry no page info
    for i in (0, 2, 4):
        assert not info[int(wl.page_indptr[i]):int(wl.page_indptr[i + 1])].any()


@pytest.mark.parametrize("pos,L,msg", [
    ([3, 3, 5], 10, "increase strictly"),
    ([5, 4], 10, "increase strictly"),
    ([2, 10], 10, "increase strictly"),
    ([-1, 4], 10, "increase strictly"),
    (list(range(0, 66, 2)), 70, "at most 32"),
])
def test_position_list_validation(pos, L, msg):
    wl = workloads.make_workload("bad", 0, hq=2, hkv=2, d=64, decodes=[(0, 40)], prefills=[],
                                 pos_decodes=[([1, 2, 7], 20)])
    q_pos = np.concatenate([wl.q_pos, np.asarray(pos, np.int32)])
    q_indptr = np.concatenate([wl.q_indptr, [wl.q_indptr[-1] + len(pos)]]).astype(np.int32)
    kv_len = np.concatenate([wl.kv_len, [L]]).astype(np.int32)
    npg = -(-L // 16)
    page_indptr = np.concatenate([wl.page_indptr, [wl.page_indptr[-1] + npg]]).astype(np.int32)
    page_ids = np.concatenate([wl.page_ids, np.arange(1000, 1000 + npg)]).astype(np.int32)
    with pytest.raises(SangamError, match=msg):
        attn.plan(q_indptr=q_indptr, q_offset=np.zeros(len(kv_len), np.int32), kv_len=kv_len,
                  page_indptr=page_indptr, page_ids=page_ids, num_q_heads=2, num_kv_heads=2,
                  head_dim=64, num_pool_pages=4096, sm_scale=0.125, q_pos=q_pos)


@pytest.mark.parametrize("hq,hkv", [(28, 4), (32, 32)])
def test_cached_multi_row_blocks_plan(hq, hkv):
    """A cached item with more than 32 rows (a larger decode block) runs in
    prefill-shaped tiles of 128 rows over its paged context; a context longer
    than the cached-range limit is cut into ranges of at most 8192 keys."""
    wl = workloads.make_workload("mb", 3, hq=hq, hkv=hkv, d=128, prefills=[],
                                 decodes=[(100, 500, 64), (1500, 9000, 200), (8190, 8400, 150)])
    h, items, dec, pre, mer = parse(plan_of(wl))
    assert len(dec) == 0
    assert [int(x) for x in items["num_splits"]] == [1, 2, 2]
    for t in pre:
        assert t["flags"] == 0 and t["kv_end"] - t["kv_begin"] <= 8192
    per_item = np.bincount(pre["item"], minlength=3)
    # item 0: 1 row block, items 1 and 2: 2 row blocks of 128, each split in two
    assert list(per_item) == [hq, 2 * 2 * hq, 2 * 2 * hq]
    assert len(mer) == 200 + 150


def test_wide_prefill_tiles_chosen():
    """256-row prefill-shaped tiles exactly when head_dim is 128, no block
    decode joins the prefill launch and every prefill-shaped item has at
    least 1024 rows."""
    def rows(wl):
        return int(parse(plan_of(wl))[0]["prefill_rows"])
    mk = lambda **kw: workloads.make_workload("w", 2, **kw)
    assert rows(workloads.prefill_heavy(0)) == 256
    assert rows(workloads.dream_prefill(0)) == 256
    assert rows(workloads.dream_mixed(0)) == 128           # fused block decodes
    assert rows(mk(hq=8, hkv=8, d=128, decodes=[(5, 900)], prefills=[2000])) == 256  # MHA decodes stay apart
    assert rows(mk(hq=28, hkv=4, d=128, decodes=[(5, 900)], prefills=[2000])) == 128  # GQA decodes fuse
    assert rows(mk(hq=8, hkv=8, d=128, decodes=[], prefills=[2000, 1023])) == 128     # a short prefill
    assert rows(mk(hq=8, hkv=8, d=64, decodes=[], prefills=[2000])) == 128            # head_dim 64
    assert rows(mk(hq=8, hkv=8, d=128, decodes=[(37, 9000, 1100)], prefills=[])) == 256  # long cached block
