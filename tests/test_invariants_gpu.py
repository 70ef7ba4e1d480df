"""Invariants of bidirectional attention (Sec. 2.1: no causal mask, so the
keys of an item form a set) checked on the HIP path's own outputs, next to
the oracle comparisons of test_parity.py:

- permuting a block's rows (Q, k_new, v_new jointly) permutes its outputs;
- permuting a whole prefill's tokens jointly permutes its outputs;
- permuting the items of a batch (each with its pages) leaves every item's
  outputs unchanged, bit for bit (each tile's arithmetic depends on its item
  alone);
- GQA with G query heads per KV head equals MHA whose KV heads repeat each
  KV head G times;
- the call writes nothing outside its outputs: guard rows around out and lse
  keep their contents.

A permutation reorders the keys a tile sums over, so results may differ by
rounding: those comparisons use the parity bar (max |delta| <= 1e-2, mean
<= 1e-3) and the LSE bar of test_parity.py.
"""
import numpy as np
import pytest
import torch

import workloads
from tests.test_parity import LSE_ABS, check_full, compare, run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2607_04206_amd  # noqa: F401
    return torch.device("cuda:0")


def with_values(wl, fn):
    """wl with its values replaced: fn(item, kind) -> fp32 tensor or None."""
    wl.value_fn = fn
    return wl


def drawn(wl):
    """Every value piece of a workload as drawn (bf16 widened to fp32)."""
    vals = {}
    for i in range(wl.num_items):
        vals[(i, workloads.KIND_Q)] = wl.q(i).float()
        vals[(i, workloads.KIND_KNEW)] = wl.k_new(i).float()
        vals[(i, workloads.KIND_VNEW)] = wl.v_new(i).float()
        if not wl.is_prefill[i]:
            vals[(i, workloads.KIND_KCTX)] = wl.k_ctx(i).float()
            vals[(i, workloads.KIND_VCTX)] = wl.v_ctx(i).float()
    return vals


def rows_close(tag, got, ref, got_lse, ref_lse):
    compare(tag, got.float().cpu().numpy(), ref.float().cpu().numpy().astype(np.float64),
            got_lse.cpu().numpy(), ref_lse.cpu().numpy().astype(np.float64))


@pytest.mark.parametrize("hq,hkv", [(32, 32), (28, 4), (8, 2)])
def test_block_row_permutation(dev, hq, hkv):
    dec = [(40, 300), (200, 1100), (64, 96), (1000, 9100)]
    mk = lambda: workloads.make_workload("permb", 5, hq=hq, hkv=hkv, d=128, decodes=dec, prefills=[257])
    base = mk()
    vals = drawn(base)
    _, _, out0, lse0 = run(with_values(mk(), lambda i, k: vals.get((i, k))), dev)
    rng = np.random.default_rng(hq)
    perms = {i: torch.from_numpy(rng.permutation(32)) for i in range(len(dec))}
    pv = dict(vals)
    for i, pi in perms.items():
        for kind in (workloads.KIND_Q, workloads.KIND_KNEW, workloads.KIND_VNEW):
            pv[(i, kind)] = vals[(i, kind)][pi]
    wl1 = with_values(mk(), lambda i, k: pv.get((i, k)))
    _, _, out1, lse1 = run(wl1, dev)
    check_full(wl1, out1, lse1)
    for i, pi in perms.items():
        b = int(base.q_indptr[i])
        rows_close(f"block rows of item {i}", out1[b:b + 32], out0[b:b + 32][pi.to(dev)],
                   lse1[b:b + 32], lse0[b:b + 32][pi.to(dev)])
    # the prefill is untouched by the decodes' permutation
    b = int(base.q_indptr[len(dec)])
    assert torch.equal(out1[b:], out0[b:])


@pytest.mark.parametrize("hq,hkv,L", [(28, 4, 300), (32, 32, 1000), (4, 4, 129)])
def test_prefill_token_permutation(dev, hq, hkv, L):
    mk = lambda: workloads.make_workload("permp", 6, hq=hq, hkv=hkv, d=128, decodes=[(10, 77)], prefills=[L])
    base = mk()
    vals = drawn(base)
    _, _, out0, lse0 = run(with_values(mk(), lambda i, k: vals.get((i, k))), dev)
    pi = torch.from_numpy(np.random.default_rng(L).permutation(L))
    pv = dict(vals)
    for kind in (workloads.KIND_Q, workloads.KIND_KNEW, workloads.KIND_VNEW):
        pv[(1, kind)] = vals[(1, kind)][pi]
    wl1 = with_values(mk(), lambda i, k: pv.get((i, k)))
    _, _, out1, lse1 = run(wl1, dev)
    check_full(wl1, out1, lse1)
    b = int(base.q_indptr[1])
    rows_close("prefill tokens", out1[b:], out0[b:][pi.to(dev)], lse1[b:], lse0[b:][pi.to(dev)])


@pytest.mark.parametrize("hq,hkv", [(28, 4), (32, 32)])
def test_batch_item_permutation(dev, hq, hkv):
    """Items reordered (values and pages travel with their item): each item's
    outputs are bitwise the same."""
    dec = [(40, 300), (200, 1100), (64, 96), (1000, 9100), (5, 37)]
    pre = [513, 64]
    wl0 = workloads.make_workload("permi", 7, hq=hq, hkv=hkv, d=128, decodes=dec, prefills=pre)
    vals = drawn(wl0)
    wl0.value_fn = lambda i, k: vals.get((i, k))
    _, _, out0, lse0 = run(wl0, dev)
    order = [3, 0, 4, 2, 1, 6, 5]  # decodes still before prefills, each group reordered
    items = [(dec + [(0, L) for L in pre])[j] for j in order]
    wl1 = workloads.make_workload("permi", 7, hq=hq, hkv=hkv, d=128,
                                  decodes=[x for x, j in zip(items, order) if j < len(dec)],
                                  prefills=[x[1] for x, j in zip(items, order) if j >= len(dec)])
    # pages and values follow the items
    pages = [wl0.item_pages(j) for j in order]
    wl1.page_ids = np.concatenate(pages).astype(np.int32)
    wl1.num_pool_pages = wl0.num_pool_pages
    wl1.value_fn = lambda i, k: vals.get((order[i], k))
    _, _, out1, lse1 = run(wl1, dev)
    for new, old in enumerate(order):
        a0, a1 = int(wl0.q_indptr[old]), int(wl0.q_indptr[old + 1])
        b0, b1 = int(wl1.q_indptr[new]), int(wl1.q_indptr[new + 1])
        assert torch.equal(out1[b0:b1], out0[a0:a1]), f"item {old}"
        assert torch.equal(lse1[b0:b1], lse0[a0:a1]), f"item {old}"


@pytest.mark.parametrize("hkv,G", [(4, 7), (2, 4), (8, 1)])
def test_gqa_equals_repeated_mha(dev, hkv, G):
    hq = hkv * G
    dec = [(40, 300), (200, 1100), (1000, 9100)]
    pre = [257]
    gqa = workloads.make_workload("gqa", 8, hq=hq, hkv=hkv, d=128, decodes=dec, prefills=pre)
    vals = drawn(gqa)
    gqa.value_fn = lambda i, k: vals.get((i, k))
    mha = workloads.make_workload("gqa", 8, hq=hq, hkv=hq, d=128, decodes=dec, prefills=pre)
    rep = {}
    for (i, k), v in vals.items():
        rep[(i, k)] = v if k == workloads.KIND_Q else v.repeat_interleave(G, 1)
    mha.value_fn = lambda i, k: rep.get((i, k))
    _, _, og, lg = run(gqa, dev)
    _, _, om, lm = run(mha, dev)
    check_full(gqa, og, lg)
    rows_close("GQA vs repeated MHA", og, om, lg, lm)


@pytest.mark.parametrize("force", [0, 2])
def test_guard_bands_around_outputs(dev, force):
    """out and lse are views into larger buffers whose guard rows hold a
    sentinel: after the call the guards are unchanged (the split merge
    included)."""
    from paper_2607_04206_amd import attn
    wl = workloads.ragged_small(5, hq=28, hkv=4, d=128)
    t = workloads.device_inputs(wl, dev)
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                  page_ids=wl.page_ids, num_q_heads=28, num_kv_heads=4, head_dim=128,
                  num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale, force_kv_splits=force, device=dev)
    T, G = wl.total_q, 64
    out_buf = torch.full((T + 2 * G, 28, 128), 12352.0, dtype=torch.bfloat16, device=dev)
    lse_buf = torch.full((T + 2 * G, 28), -777.0, dtype=torch.float32, device=dev)
    out, lse = out_buf[G:G + T], lse_buf[G:G + T]
    ws = None
    if p.workspace_bytes:
        ws_buf = torch.full((p.workspace_bytes + 2 * 4096,), 0x5A, dtype=torch.uint8, device=dev)
        ws = ws_buf[4096:4096 + p.workspace_bytes]
    before = (out_buf.clone(), lse_buf.clone())
    attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"], out=out,
                 lse=lse, workspace=ws)
    torch.cuda.synchronize()
    for sl in (slice(0, G), slice(G + T, T + 2 * G)):
        assert torch.equal(out_buf[sl].view(torch.int16), before[0][sl].view(torch.int16))
        assert torch.equal(lse_buf[sl], before[1][sl])
    if ws is not None:
        assert (ws_buf[:4096] == 0x5A).all() and (ws_buf[4096 + p.workspace_bytes:] == 0x5A).all()
    check_full(wl, out, lse)
