"""Paged-KV export / import (the hand-off of a request's KV between workers in
the hybrid configuration, Sec. 4.3 and Sec. 5).

CPU: the plan's validation and records, and the oracle pinned against a
page-wise construction of each request's sequence, a round trip through an
unrelated page table, and planted slips. GPU: both kernels bit-exact against
the oracle on ragged batches and at the LLaDA and Dream decode batches' full
size, and attention over an imported pool bitwise equal to attention over the
source pool.
"""
import ctypes
import os

import numpy as np
import pytest
import torch

import workloads
from oracle import kv_transfer as kvo
from paper_2607_04206_amd import _lib, kv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

RECORD = np.dtype([("page", "<i4"), ("row0", "<i4"), ("nslots", "<i4"), ("item", "<i4")])

RAGGED = [1, 15, 16, 17, 33, 300, 2, 64]


def page_wise_sequence(pool: np.ndarray, pages: np.ndarray, L: int) -> np.ndarray:
    """A request's positions [0, L) built page by page: each page's [Hkv, 16, D]
    block turned into 16 rows [16, Hkv, D], the pages concatenated, the last
    page cut at L."""
    blocks = [np.transpose(pool[int(pg)], (1, 0, 2)) for pg in pages]
    return np.concatenate(blocks, axis=0)[:L]


# ---------------------------------------------------------------- plan (CPU)

def test_plan_records():
    c = workloads.kv_transfer_case("rec", 0, RAGGED, hkv=2, d=64)
    p = kv.plan(kv_len=c.kv_len, page_indptr=c.page_indptr, page_ids=c.src_pages, num_kv_heads=2,
                head_dim=64, num_pool_pages=c.num_pool_pages)
    assert p.rows == sum(RAGGED)
    recs = p.host[256:].view(RECORD)
    assert len(recs) == c.page_indptr[-1]
    row = 0
    for i, L in enumerate(RAGGED):
        for k in range(-(-L // 16)):
            r = recs[c.page_indptr[i] + k]
            assert (r["page"], r["row0"], r["nslots"], r["item"]) == (
                c.src_pages[c.page_indptr[i] + k], row + 16 * k, min(16, L - 16 * k), i)
        row += L


@pytest.mark.parametrize("bad,status", [
    (dict(kv_len=[]), -1),
    (dict(kv_len=[0]), -1),
    (dict(page_indptr=[0, 2]), -1),
    (dict(page_indptr=[1, 2], page_ids=[0, 1]), -1),
    (dict(page_ids=[7]), -3),
    (dict(page_ids=[-1]), -3),
    (dict(kv_len=[17, 3], page_indptr=[0, 2, 3], page_ids=[0, 1, 0]), -4),
    (dict(head_dim=96), -2),
    (dict(page_size=8), -2),
    (dict(num_kv_heads=0), -1),
])
def test_plan_rejects(bad, status):
    args = dict(kv_len=[5], page_indptr=[0, 1], page_ids=[3], num_kv_heads=2, head_dim=64, num_pool_pages=4)
    args.update(bad)
    with pytest.raises(_lib.SangamError) as e:
        kv.plan(**args)
    assert e.value.status == status


def test_plan_buffer_query_and_junk():
    d = _lib.KvDesc()
    kv_len = np.asarray([20], np.int32)
    ind = np.asarray([0, 2], np.int32)
    ids = np.asarray([1, 0], np.int32)
    d.num_items, d.num_kv_heads, d.head_dim, d.page_size, d.num_pool_pages = 1, 1, 64, 16, 2
    d.kv_len, d.page_indptr, d.page_ids = kv_len.ctypes.data, ind.ctypes.data, ids.ctypes.data
    used = ctypes.c_size_t(0)
    assert _lib.lib.sangam_kv_plan(ctypes.byref(d), None, 0, ctypes.byref(used)) == -5
    assert used.value == 256 + 2 * 16
    junk = np.zeros(512, np.uint8)
    assert _lib.lib.sangam_kv_plan_rows(junk.ctypes.data) == 0
    # the copies reject a junk plan, NULL and misaligned pointers before any HIP call
    f = _lib.lib.sangam_kv_export
    assert f(junk.ctypes.data, 4096, 4096, 4096, 4096, 4096, None) == -8
    buf = np.zeros(used.value, np.uint8)
    assert _lib.lib.sangam_kv_plan(ctypes.byref(d), buf.ctypes.data, buf.nbytes, ctypes.byref(used)) == 0
    assert f(buf.ctypes.data, 4096, None, 4096, 4096, 4096, None) == -1
    assert _lib.lib.sangam_kv_import(buf.ctypes.data, 4096, 4096, 4096, 4096 + 2, 4096, None) == -6


# ------------------------------------------------------------- oracle (CPU)

def _pins(mod):
    """The oracle's pins; raise AssertionError on any disagreement."""
    for hkv, d in ((2, 64), (3, 8), (1, 8)):
        c = workloads.kv_transfer_case(f"pin{hkv}", hkv, RAGGED, hkv=hkv, d=d)
        k, v = mod.export(c.pool_k, c.pool_v, c.kv_len, c.page_indptr, c.src_pages)
        ind = kvo.kv_indptr(c.kv_len)
        for i, L in enumerate(c.kv_len):
            pages = c.src_pages[c.page_indptr[i]:c.page_indptr[i + 1]]
            assert np.array_equal(k[ind[i]:ind[i + 1]], page_wise_sequence(c.pool_k, pages, L))
            assert np.array_equal(v[ind[i]:ind[i + 1]], page_wise_sequence(c.pool_v, pages, L))
        # round trip into an unrelated page table of a sentinel-filled pool
        sent = np.full_like(c.pool_k, 0x7FC1)
        bk, bv = mod.import_(k, v, sent, sent, c.kv_len, c.page_indptr, c.dst_pages)
        touched = np.zeros(c.pool_k.shape[:1] + (16,), bool)
        for i, L in enumerate(c.kv_len):
            pages = c.dst_pages[c.page_indptr[i]:c.page_indptr[i + 1]]
            src = c.src_pages[c.page_indptr[i]:c.page_indptr[i + 1]]
            assert np.array_equal(page_wise_sequence(bk, pages, L), page_wise_sequence(c.pool_k, src, L))
            assert np.array_equal(page_wise_sequence(bv, pages, L), page_wise_sequence(c.pool_v, src, L))
            for p in range(int(L)):
                touched[pages[p // 16], p % 16] = True
        untouched = ~touched
        assert (bk.transpose(0, 2, 1, 3)[untouched] == 0x7FC1).all()
        assert (bv.transpose(0, 2, 1, 3)[untouched] == 0x7FC1).all()


def test_oracle_pins():
    _pins(kvo)


MUTANTS = {
    "slot_from_page_index": ("p % PAGE", "p // PAGE % PAGE"),
    "page_index_from_slot": ("page_indptr[i] + p // PAGE", "page_indptr[i] + p % PAGE % max(1, (len(page_ids) - page_indptr[i]))"),
    "row_of_next_request": ("k[ind[i] + p] =", "k[ind[i + 1] - 1 - p] ="),
    "v_from_k_pool": ("v[ind[i] + p] = pool_v[page, :, slot, :]", "v[ind[i] + p] = pool_k[page, :, slot, :]"),
    "import_writes_whole_page": ("for p in range(int(L)):\n            page, slot = _place(i, p, page_indptr, page_ids)\n            pk[",
                                 "for p in range(-(-int(L) // PAGE) * PAGE):\n            page, slot = _place(i, p, page_indptr, page_ids)\n            pk["),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_oracle_pins_reject_mutant(name):
    src = open(kvo.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) >= 1, f"mutation anchor missing: {a}"
    ns = {}
    exec(compile(src.replace(a, b), f"<mutant {name}>", "exec"), ns)

    class M:
        export = staticmethod(ns["export"])
        import_ = staticmethod(ns["import_"])

    with pytest.raises((AssertionError, IndexError, ValueError)):
        _pins(M)


# ----------------------------------------------------------------- GPU

def _dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return torch.device("cuda:0")


def _t(a: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)


def _np(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _check_case(c, dev):
    print(f"[case] kv transfer {c.name}: {len(c.kv_len)} requests, {c.rows} rows, Hkv {c.num_kv_heads}, "
          f"D {c.head_dim}", flush=True)
    ps = kv.plan(kv_len=c.kv_len, page_indptr=c.page_indptr, page_ids=c.src_pages, num_kv_heads=c.num_kv_heads,
                 head_dim=c.head_dim, num_pool_pages=c.num_pool_pages, device=dev)
    pd = kv.plan(kv_len=c.kv_len, page_indptr=c.page_indptr, page_ids=c.dst_pages, num_kv_heads=c.num_kv_heads,
                 head_dim=c.head_dim, num_pool_pages=c.num_pool_pages, device=dev)
    gk, gv = kv.kv_export(ps, _t(c.pool_k, dev), _t(c.pool_v, dev))
    ek, ev = kvo.export(c.pool_k, c.pool_v, c.kv_len, c.page_indptr, c.src_pages)
    torch.cuda.synchronize()
    assert np.array_equal(_np(gk), ek) and np.array_equal(_np(gv), ev)
    # import the oracle's packed rows into a sentinel-filled pool
    sent = np.full_like(c.pool_k, 0x7FC1)
    bk, bv = _t(sent, dev), _t(sent, dev)
    kv.kv_import(pd, _t(ek, dev), _t(ev, dev), bk, bv)
    xk, xv = kvo.import_(ek, ev, sent, sent, c.kv_len, c.page_indptr, c.dst_pages)
    torch.cuda.synchronize()
    assert np.array_equal(_np(bk), xk) and np.array_equal(_np(bv), xv)


@pytest.mark.gpu
@pytest.mark.parametrize("hkv,d", [(2, 64), (4, 128), (1, 128), (3, 64), (32, 128)])
def test_kv_copies_match_oracle(hkv, d):
    dev = _dev()
    _check_case(workloads.kv_transfer_case(f"ragged_{hkv}_{d}", 7 + hkv, RAGGED, hkv=hkv, d=d), dev)


@pytest.mark.gpu
@pytest.mark.parametrize("which", ["llada_decode", "dream_mixed"])
def test_kv_copies_full_size(which):
    """The cached contexts of the LLaDA (32 decodes, 32 KV heads) and Dream (48
    decodes, 4 KV heads) batches, every byte compared."""
    dev = _dev()
    wl = getattr(workloads, which)(0)
    c = workloads.kv_transfer_case(which, 11, wl.kv_len, hkv=wl.num_kv_heads, d=wl.head_dim, spare_pages=1)
    _check_case(c, dev)


@pytest.mark.gpu
def test_attention_after_import_is_bitwise_unchanged():
    """Decodes continue on the receiving pool: the same call over the imported
    pages returns the same bits as over the sender's pages."""
    from paper_2607_04206_amd import attn
    dev = _dev()
    wl = workloads.ragged_small(3, hq=8, hkv=2, d=128)
    print(f"[case] attention after import: {wl.name}", flush=True)
    t = workloads.device_inputs(wl, dev)
    # the pool after the call: the receiver gets the post-write cache
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                  page_ids=wl.page_ids, num_q_heads=8, num_kv_heads=2, head_dim=128,
                  num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale, device=dev)
    out_a, lse_a = attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"])
    rng = np.random.default_rng(5)
    dst = rng.permutation(wl.num_pool_pages)[:len(wl.page_ids)].astype(np.int32)
    ps = kv.plan(kv_len=wl.kv_len, page_indptr=wl.page_indptr, page_ids=wl.page_ids, num_kv_heads=2,
                 head_dim=128, num_pool_pages=wl.num_pool_pages, device=dev)
    pd = kv.plan(kv_len=wl.kv_len, page_indptr=wl.page_indptr, page_ids=dst, num_kv_heads=2, head_dim=128,
                 num_pool_pages=wl.num_pool_pages, device=dev)
    pk, pv = kv.kv_export(ps, t["k_cache"], t["v_cache"])
    rk = torch.full_like(t["k_cache"], float("nan"))
    rv = torch.full_like(t["v_cache"], float("nan"))
    kv.kv_import(pd, pk, pv, rk, rv)
    p2 = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                   page_ids=dst, num_q_heads=8, num_kv_heads=2, head_dim=128,
                   num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale, device=dev)
    out_b, lse_b = attn.forward(p2, t["q"], t["k_new"], t["v_new"], rk, rv,
                                torch.from_numpy(dst).to(dev))
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(lse_a, lse_b)
    # and the receiver's cache equals the sender's at every position
    def seq(pool, pages, L):
        idx = torch.from_numpy(np.asarray(pages, np.int64)).to(dev)
        return pool[idx].permute(0, 2, 1, 3).reshape(-1, 2, 128)[:L]

    for i in range(wl.num_items):
        sl = slice(int(wl.page_indptr[i]), int(wl.page_indptr[i + 1]))
        L = int(wl.kv_len[i])
        for a, b in ((t["k_cache"], rk), (t["v_cache"], rv)):
            assert torch.equal(seq(a, wl.page_ids[sl], L).view(torch.int16), seq(b, dst[sl], L).view(torch.int16))
