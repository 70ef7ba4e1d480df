"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.

Bar (bf16 inputs, fp32 accumulation): over all compared output elements
max |delta| <= 1e-2 and mean |delta| <= 1e-3, plus max |delta| <= 2e-2 * max|o|
(outputs shrink like 1/sqrt(L), which makes the absolute bounds loose at long
contexts); the cache write-back bit-exact; pool slots the batch does not own
untouched (they hold NaN, so a stray read or write shows).

LSE bound, derived from the arithmetic: the kernel rounds each softmax weight
p_j to bf16 (8 significant bits, RNE: relative error <= 2^-8) and sums the
rounded values, so the row sum l carries a relative error <= 2^-8 and ln l an
absolute error <= -ln(1 - 2^-8) = 3.9e-3; fp32 score rounding adds ~1e-6.
Bar: 4e-3.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import oracle

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS, REL_MAX, LSE_ABS = 1e-2, 1e-3, 2e-2, 4e-3


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2607_04206_amd  # noqa: F401  (fails loudly when the library is missing)
    return torch.device("cuda:0")


def run(wl, dev, force_splits=0, fill=float("nan"), want_lse=True, num_cus=0):
    from paper_2607_04206_amd import attn
    print(f"[case] {wl.name} seed={wl.seed} items={wl.num_items} force_splits={force_splits}",
          flush=True)
    t = workloads.device_inputs(wl, dev, fill=fill)
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len,
                  page_indptr=wl.page_indptr, page_ids=wl.page_ids, num_q_heads=wl.num_q_heads,
                  num_kv_heads=wl.num_kv_heads, head_dim=wl.head_dim,
                  num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale,
                  force_kv_splits=force_splits, q_pos=wl.q_pos, num_cus=num_cus, device=dev)
    out, lse = attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                            t["page_ids"], want_lse=want_lse)
    torch.cuda.synchronize()
    return p, t, out, lse


def compare(tag, got, ref, got_lse=None, ref_lse=None, max_abs=None, mean_abs=MEAN_ABS):
    got = np.asarray(got, np.float64)
    assert np.isfinite(got).all(), f"{tag}: non-finite output"
    d = np.abs(got - ref)
    mx, mean = d.max(), d.mean()
    bound = min(MAX_ABS, REL_MAX * np.abs(ref).max()) if max_abs is None else max_abs
    assert mx <= bound, f"{tag}: max |delta| {mx:.3e} > {bound:.3e}"
    assert mean <= mean_abs, f"{tag}: mean |delta| {mean:.3e} > {mean_abs:.3e}"
    if got_lse is not None:
        dl = np.abs(np.asarray(got_lse, np.float64) - ref_lse).max()
        assert dl <= LSE_ABS, f"{tag}: lse max |delta| {dl:.3e}"
    return mx, mean


def check_full(wl, out, lse):
    ref, ref_lse = oracle.attention_all(wl)
    return compare(wl.name, out.float().cpu().numpy(), ref,
                   None if lse is None else lse.cpu().numpy(), ref_lse)


def check_sampled(wl, out, lse, items, rows_per_item=None, heads=None):
    res = oracle.attention(wl, items=items, rows=rows_per_item, heads=heads)
    outc = out.float().cpu().numpy()
    lsec = lse.cpu().numpy()
    hs = list(range(wl.num_q_heads)) if heads is None else list(heads)
    g_all, r_all, gl_all, rl_all = [], [], [], []
    for i, (rr, ro, rl) in res.items():
        base = int(wl.q_indptr[i])
        g_all.append(outc[base + rr][:, hs])
        gl_all.append(lsec[base + rr][:, hs])
        r_all.append(ro)
        rl_all.append(rl)
    return compare(wl.name, np.concatenate([g.reshape(-1) for g in g_all]),
                   np.concatenate([r.reshape(-1) for r in r_all]),
                   np.concatenate([g.reshape(-1) for g in gl_all]),
                   np.concatenate([r.reshape(-1) for r in rl_all]))


def check_cache(wl, t, items=None):
    """Bit-exact write-back on [0, L_i); slots past L_i of the last page keep NaN."""
    kc, vc = t["k_cache"], t["v_cache"]
    for i in range(wl.num_items) if items is None else items:
        ek, ev = oracle.expected_kv(wl, i)
        gk = workloads.gather_item_cache(wl, kc, i).cpu().view(torch.int16).numpy().view(np.uint16)
        gv = workloads.gather_item_cache(wl, vc, i).cpu().view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(gk, ek), f"item {i}: K cache differs"
        assert np.array_equal(gv, ev), f"item {i}: V cache differs"
        L = int(wl.kv_len[i])
        if L % 16:
            last = int(wl.item_pages(i)[-1])
            assert torch.isnan(kc[last, :, L % 16:]).all() and torch.isnan(vc[last, :, L % 16:]).all()


def check_pool_untouched(wl, t):
    """Exactly the owned slots are finite: nothing outside [0, L_i) was written."""
    owned = int(np.sum(wl.kv_len.astype(np.int64))) * wl.num_kv_heads * wl.head_dim
    for pool in (t["k_cache"], t["v_cache"]):
        assert int((~torch.isnan(pool)).sum().item()) == owned


# ------------------------------------------------------------------- cases
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_mixed(dev, seed):
    wl = workloads.tiny_mixed(seed)
    p, t, out, lse = run(wl, dev)
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)
    # the block decode of rows 96..127 matches the prefill's rows 96..127
    o = out.float().cpu().numpy()
    assert np.abs(o[:32] - o[32 + 96:32 + 128]).max() <= 1e-2


SHAPES = [(4, 4, 64), (8, 2, 64), (18, 2, 64), (28, 4, 128), (32, 32, 128), (8, 4, 128), (11, 1, 128),
          (24, 8, 128), (1, 1, 64), (16, 1, 128), (64, 4, 128)]


@pytest.mark.parametrize("hq,hkv,d", SHAPES)
def test_ragged_small(dev, hq, hkv, d):
    wl = workloads.ragged_small(0, hq=hq, hkv=hkv, d=d)
    p, t, out, lse = run(wl, dev)
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("hq,hkv", [(16, 1), (64, 4)])
@pytest.mark.parametrize("force", [0, 3])
def test_large_gqa_group_decode_tiles(dev, hq, hkv, force):
    """Groups of 16 query heads per KV head in a decode-only batch on 8 CUs
    (so not the heads-across tiles of a small batch): each group runs as two
    decode-shaped work-groups of 8 waves, whose outputs take the direct
    stores (a wave's rows do not fit in LDS beside the stages)."""
    dec = [(40, 300), (200, 1100), (64, 96), (1000, 9100), (5, 37), (0, 33)]
    wl = workloads.make_workload("g16", 11, hq=hq, hkv=hkv, d=128, decodes=dec, prefills=[])
    p, t, out, lse = run(wl, dev, force_splits=force, num_cus=8)
    assert p.info.num_decode_tiles > 0 and p.info.decode_q_waves == 8 and p.info.num_fused_decode_tiles == 0
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("hq,hkv,d", [(4, 4, 64), (28, 4, 128), (32, 32, 128)])
@pytest.mark.parametrize("force", [1, 2, 4, 8])
def test_forced_splits(dev, hq, hkv, d, force):
    wl = workloads.ragged_small(1, hq=hq, hkv=hkv, d=d)
    p, t, out, lse = run(wl, dev, force_splits=force)
    check_full(wl, out, lse)
    check_cache(wl, t)


def test_split_count_independence(dev):
    wl = workloads.llada_decode(2)
    outs = [run(wl, dev, force_splits=k)[2].float() for k in (1, 2, 4, 8)]
    for o in outs[1:]:
        assert (o - outs[0]).abs().max().item() <= 1e-2


def test_q_stress(dev):
    """Q scaled by 4: a peaky softmax where few weights dominate, so the bf16
    rounding of P does not average out. Derived bound: each weight is rounded
    to bf16 (relative error <= 2^-8) and renormalised by the same rounded sum,
    so it errs by <= 2 * 2^-8 relative and |sum (w~ - w) v| <= 2^-7 max|V|;
    the bf16 output adds <= 2^-8 |o|: |delta| <= 1.5 * 2^-7 * max|V| (mean:
    the same with mean|V|)."""
    wl = workloads.ragged_small(2, hq=28, hkv=4, d=128, q_scale=4.0)
    p, t, out, lse = run(wl, dev)
    ref, ref_lse = oracle.attention_all(wl)
    vmax = max(float(wl.packed_v_new().float().abs().max()),
               max(float(wl.v_ctx(i).float().abs().max()) for i in range(wl.num_items)
                   if not wl.is_prefill[i]))
    vmean = float(wl.packed_v_new().float().abs().mean())
    compare(wl.name, out.float().cpu().numpy(), ref, lse.cpu().numpy(), ref_lse,
            max_abs=1.5 * 2 ** -7 * vmax, mean_abs=1.5 * 2 ** -7 * vmean)


def test_no_lse(dev):
    wl = workloads.ragged_small(3, hq=8, hkv=2, d=64)
    p, t, out, lse = run(wl, dev, want_lse=False)
    assert lse is None
    ref, _ = oracle.attention_all(wl)
    compare(wl.name, out.float().cpu().numpy(), ref)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_llada_decode(dev, seed):
    wl = workloads.llada_decode(seed)
    p, t, out, lse = run(wl, dev)
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dream_mixed(dev, seed):
    wl = workloads.dream_mixed(seed)
    p, t, out, lse = run(wl, dev)
    n_dec = int((~wl.is_prefill).sum())
    rng = np.random.default_rng(seed)
    rows = {}
    for i in range(n_dec, wl.num_items):
        n = wl.n(i)
        rows[i] = np.unique(np.r_[0, n - 1, 127, 128, rng.integers(0, n, 40)])
    check_sampled(wl, out, lse, items=list(range(wl.num_items)), rows_per_item=rows)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


def tile_rows(n, rng, tile=128):
    """One random row from every `tile`-row block of an item, plus its first
    and last rows."""
    picks = [int(rng.integers(b, min(n, b + tile))) for b in range(0, n, tile)]
    return np.unique(np.r_[0, n - 1, picks])


def spread_heads(rng, hq, hkv, count):
    """`count` query heads from distinct KV groups (as many as there are)."""
    G = hq // hkv
    groups = rng.permutation(hkv)[:count]
    if len(groups) < count:
        groups = np.r_[groups, rng.integers(0, hkv, count - len(groups))]
    return sorted({int(g) * G + int(rng.integers(0, G)) for g in groups})


def check_fresh_rows(wl, t, items):
    """The fresh rows of each item sit bit-exact at their positions in the pages."""
    for i in items:
        pos = wl.positions(i)
        pages = torch.from_numpy(wl.item_pages(i)[pos // 16].astype(np.int64)).to(t["k_cache"].device)
        slots = torch.from_numpy((pos % 16).astype(np.int64)).to(t["k_cache"].device)
        for pool, fresh in ((t["k_cache"], wl.k_new(i)), (t["v_cache"], wl.v_new(i))):
            got = pool[pages, :, slots].cpu()  # [n, Hkv, D]
            assert torch.equal(got.view(torch.int16), fresh.view(torch.int16)), f"item {i}: fresh rows"


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_prefill_heavy(dev, seed):
    """Every 128-row tile of every prefill is sampled (one random row each,
    plus the first and last row) on three query heads of distinct KV groups
    per item; the cache of every item is compared bit for bit."""
    wl = workloads.prefill_heavy(seed)
    p, t, out, lse = run(wl, dev)
    rng = np.random.default_rng(50 + seed)
    for i in range(wl.num_items):
        rows = {i: tile_rows(wl.n(i), rng)}
        heads = spread_heads(rng, wl.num_q_heads, wl.num_kv_heads, 3)
        check_sampled(wl, out, lse, items=[i], rows_per_item=rows, heads=heads)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_long_decode(dev, seed):
    """All 256 block decodes, every row, on four query heads spread over the
    KV heads (MHA: each its own group); the fresh rows of every item and the
    whole cache of the split items and eight others bit for bit."""
    wl = workloads.long_decode(seed)
    p, t, out, lse = run(wl, dev)
    order = np.argsort(-wl.kv_len)
    assert int(wl.kv_len[order[0]]) > 8192  # split-KV path exercised
    heads = [seed, 9 + seed, 18 + seed, 31 - seed]
    check_sampled(wl, out, lse, items=list(range(wl.num_items)), heads=heads)
    check_fresh_rows(wl, t, range(wl.num_items))
    rng = np.random.default_rng(70 + seed)
    split = [i for i in range(wl.num_items) if len(p.item_splits(i)) > 2]
    assert split
    full = sorted(set(split) | set(rng.choice(wl.num_items, 8, replace=False).tolist()))
    check_cache(wl, t, items=full)
    check_pool_untouched(wl, t)


# cached items with more than 32 rows (larger decode blocks): the rows run in
# prefill-shaped tiles over paged context; (o, L, n) with unaligned offsets, a
# block from position 0 under a cached tail, tiles spanning several 128-row
# blocks, and contexts past the 8192-key range limit whose split boundary a
# block straddles (L = 9000: chunks of 4544 keys)
CACHED_BLOCKS = [(100, 500, 64), (37, 300, 33), (0, 2000, 300), (1500, 9000, 200), (4500, 9000, 100),
                 (8190, 8400, 150)]


@pytest.mark.parametrize("hq,hkv,d", [(32, 32, 128), (28, 4, 128), (8, 2, 64)])
@pytest.mark.parametrize("with_decodes", [False, True])
@pytest.mark.parametrize("force", [0, 3])
def test_cached_multi_row_blocks(dev, hq, hkv, d, with_decodes, force):
    decodes = list(CACHED_BLOCKS) + ([(20, 700), (300, 333)] if with_decodes else [])
    wl = workloads.make_workload("cached_blocks", 31, hq=hq, hkv=hkv, d=d, decodes=decodes,
                                 prefills=[150] if with_decodes else [])
    p, t, out, lse = run(wl, dev, force_splits=force)
    assert p.info.num_prefill_tiles > 0
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("hq,hkv", [(28, 4), (32, 32), (8, 8)])
@pytest.mark.parametrize("force", [0, 2])
def test_wide_prefill_tiles(dev, hq, hkv, force):
    """The wide prefill-shaped tile (256 rows on eight waves, 128-key stages),
    which a batch of only long prefill-shaped items takes at head_dim 128:
    ragged row and key tails, a long cached block at an unaligned offset over
    a context past the cached-range limit, with and without forced splits;
    every row against the oracle, the cache bit for bit."""
    wl = workloads.make_workload("wide", 41, hq=hq, hkv=hkv, d=128, prefills=[1024, 1500, 2049],
                                 decodes=[(37, 9000, 1100), (0, 1300, 1029)])
    p, t, out, lse = run(wl, dev, force_splits=force)
    assert p.info.num_decode_tiles == 0 and p.info.num_fused_decode_tiles == 0
    from tests.test_plan import parse
    assert int(parse(p)[0]["prefill_rows"]) == 256
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


def test_sequential_prefill_then_decode(dev):
    """The cached-dLLM cycle in two calls (the single-request workload's
    sequential reading): a prefill call writes the request's pages, then a
    block decode call over those same pages reads them as its cache and
    refreshes rows 96..127. The decode matches the oracle (whose cache is the
    prefill's K/V) and the prefill's own rows 96..127."""
    from paper_2607_04206_amd import attn
    base = workloads.tiny_mixed(0)
    pre = workloads.make_workload("seq_prefill", 0, hq=4, hkv=4, d=64, decodes=[], prefills=[128])
    dec = workloads.make_workload("seq_decode", 0, hq=4, hkv=4, d=64, decodes=[(96, 128)], prefills=[])
    dec.page_ids = pre.page_ids.copy()
    dec.num_pool_pages = pre.num_pool_pages

    def pre_vals(item, kind):  # the prefill draws as the single-request workload's item 1
        return {workloads.KIND_Q: base.q(1), workloads.KIND_KNEW: base.k_new(1),
                workloads.KIND_VNEW: base.v_new(1)}[kind].float()

    def dec_vals(item, kind):  # the decode as its item 0 (cache = the prefill's K/V)
        return {workloads.KIND_Q: base.q(0), workloads.KIND_KNEW: base.k_new(0), workloads.KIND_VNEW: base.v_new(0),
                workloads.KIND_KCTX: base.k_ctx(0), workloads.KIND_VCTX: base.v_ctx(0)}[kind].float()

    pre.value_fn, dec.value_fn = pre_vals, dec_vals
    t = workloads.device_inputs(pre, dev)  # NaN pool: the decode reads only what the prefill wrote
    p1 = attn.plan(q_indptr=pre.q_indptr, q_offset=pre.q_offset, kv_len=pre.kv_len,
                   page_indptr=pre.page_indptr, page_ids=pre.page_ids, num_q_heads=4, num_kv_heads=4,
                   head_dim=64, num_pool_pages=pre.num_pool_pages, sm_scale=pre.sm_scale, device=dev)
    out1, lse1 = attn.forward(p1, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"])
    p2 = attn.plan(q_indptr=dec.q_indptr, q_offset=dec.q_offset, kv_len=dec.kv_len,
                   page_indptr=dec.page_indptr, page_ids=dec.page_ids, num_q_heads=4, num_kv_heads=4,
                   head_dim=64, num_pool_pages=dec.num_pool_pages, sm_scale=dec.sm_scale, device=dev)
    out2, lse2 = attn.forward(p2, dec.packed_q(dev), dec.packed_k_new(dev), dec.packed_v_new(dev),
                              t["k_cache"], t["v_cache"], t["page_ids"])
    torch.cuda.synchronize()
    check_full(pre, out1, lse1)
    check_full(dec, out2, lse2)
    check_cache(dec, t)
    check_pool_untouched(pre, t)
    # the decode's rows are the prefill's rows 96..127
    assert (out2.float() - out1[96:128].float()).abs().max().item() <= 1e-2
    # and the one-call reading (decode and prefill side by side on disjoint pages) agrees
    _, _, out_one, _ = run(base, dev)
    assert (out2.float() - out_one[:32].float()).abs().max().item() <= 1e-2


@pytest.mark.parametrize("hq,hkv,with_prefill,cus", [(8, 8, False, 0), (28, 4, False, 0), (28, 4, False, 8),
                                                     (28, 4, True, 0)])
def test_range_limit_boundary(dev, hq, hkv, with_prefill, cus):
    """Contexts at the longest range a tile may read from the cache (8192
    keys: 512 staged page ids, unsplit when one chunk per item is asked for)
    and one key past it (cut in two), block offsets at both ends; every row
    of these items against the oracle."""
    wl = workloads.make_workload("range_limit", 21, hq=hq, hkv=hkv, d=128,
                                 decodes=[(8192 - 32, 8192), (0, 8192), (8192 - 20, 8193), (4000, 8193)],
                                 prefills=[200] if with_prefill else [])
    p, t, out, lse = run(wl, dev, force_splits=1, num_cus=cus)
    assert [len(p.item_splits(i)) - 1 for i in range(4)] == [1, 1, 2, 2]
    # the MHA case and the 8-CU GQA case run decode-shaped tiles, the others heads-across tiles
    assert (p.info.num_decode_tiles > 0) == (hq == hkv or cus == 8)
    check_sampled(wl, out, lse, items=list(range(4)), heads=[0, hq // 2, hq - 1])
    check_cache(wl, t)
    check_pool_untouched(wl, t)


@pytest.mark.parametrize("shape", ["llada", "dream"])
@pytest.mark.parametrize("batch", [1, 64])
def test_decode_sweep_points(dev, shape, batch):
    """End points of the decode-batch sweep (block decodes at L = 1024)."""
    wl = workloads.decode_sweep(shape, batch, seed=1)
    p, t, out, lse = run(wl, dev)
    check_full(wl, out, lse)
    check_cache(wl, t)


@pytest.mark.parametrize("hq,hkv,d,prefills", [(8, 8, 64, ()), (32, 32, 128, ()), (28, 4, 128, ()),
                                               (28, 4, 128, (150, 301)), (8, 2, 64, (97,))])
@pytest.mark.parametrize("force", [0, 3])
def test_token_cache_decodes(dev, hq, hkv, d, prefills, force):
    """Per-token cached decodes: 32 rows at scattered response positions."""
    wl = workloads.token_cache_decodes(4, hq=hq, hkv=hkv, d=d, count=6, prefills=prefills)
    p, t, out, lse = run(wl, dev, force_splits=force)
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


def test_contiguous_list_is_the_block_decode(dev):
    blk = workloads.make_workload("blk", 3, hq=28, hkv=4, d=128, decodes=[(300, 700), (64, 96)], prefills=[])
    pos = workloads.make_workload("pos", 3, hq=28, hkv=4, d=128, decodes=[], prefills=[],
                                  pos_decodes=[(range(300, 332), 700), (range(64, 96), 96)])
    _, _, o1, l1 = run(blk, dev)
    _, _, o2, l2 = run(pos, dev)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_deterministic(dev):
    wl = workloads.dream_mixed(1)
    _, _, o1, l1 = run(wl, dev)
    _, _, o2, l2 = run(wl, dev)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_forward_with_launch_events(dev):
    """The timed entry point (events in each launch's dispatch) computes the
    same bits as the plain one, and each launch that ran reports a positive
    execution time."""
    from paper_2607_04206_amd import attn
    wl = workloads.ragged_small(3, hq=8, hkv=2, d=128)
    p, t, out0, lse0 = run(wl, dev, force_splits=2)
    stream = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for e in ev:
        e.record(stream)
    out, lse = attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"],
                            launch_events=ev)
    torch.cuda.synchronize()
    assert torch.equal(out, out0) and torch.equal(lse, lse0)
    i = p.info
    for k, ran in enumerate((i.num_prefill_tiles > 0, i.num_decode_tiles > 0, i.num_split_items > 0)):
        if ran:
            assert ev[2 * k].elapsed_time(ev[2 * k + 1]) > 0.0
    with pytest.raises(ValueError, match="6 events"):
        attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"],
                     launch_events=ev[:4])


def test_forward_checks_pool_and_page_table(dev):
    """The binding refuses a pool smaller than the plan's or a short device
    page table before any launch (the kernels would read past them)."""
    from paper_2607_04206_amd import attn
    wl = workloads.ragged_small(4, hq=4, hkv=2, d=64)
    t = workloads.device_inputs(wl, dev)
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                  page_ids=wl.page_ids, num_q_heads=4, num_kv_heads=2, head_dim=64,
                  num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale, device=dev)
    small = t["k_cache"][: wl.num_pool_pages - 1]
    with pytest.raises(ValueError, match="pool pages"):
        attn.forward(p, t["q"], t["k_new"], t["v_new"], small, small, t["page_ids"])
    with pytest.raises(ValueError, match="page_ids"):
        attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"][:-1])


def test_forward_on_another_stream_follows_the_plan_upload(dev):
    """The plan is copied to the device without blocking on the current
    stream; a forward issued right away on another stream waits for that
    copy (the binding orders it after the upload's event)."""
    from paper_2607_04206_amd import attn
    wl = workloads.ragged_small(6, hq=8, hkv=2, d=128)
    t = workloads.device_inputs(wl, dev)
    torch.cuda.synchronize()  # inputs ready: only the plan copy is left in flight
    side = torch.cuda.Stream(dev)
    for rep in range(3):
        p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len,
                      page_indptr=wl.page_indptr, page_ids=wl.page_ids, num_q_heads=8, num_kv_heads=2,
                      head_dim=128, num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale,
                      force_kv_splits=2, device=dev)
        with torch.cuda.stream(side):
            out, lse = attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                                    t["page_ids"], stream=side)
        side.synchronize()
        check_full(wl, out, lse)


def test_graph_capture_replays(dev):
    """The forward is only kernel launches on the caller's stream, so a HIP
    graph can hold it: every replay (with eager work on the same buffers in
    between) reproduces the eager call's bits, the split merge included."""
    from paper_2607_04206_amd import attn
    wl = workloads.ragged_small(2, hq=8, hkv=2, d=128)
    p, t, out0, lse0 = run(wl, dev, force_splits=2)
    assert p.workspace_bytes > 0
    check_full(wl, out0, lse0)
    out = torch.empty_like(out0)
    lse = torch.empty_like(lse0)
    ws = torch.empty((p.workspace_bytes,), dtype=torch.uint8, device=dev)
    args = (p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"])
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        attn.forward(*args, out=out, lse=lse, workspace=ws)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        attn.forward(*args, out=out, lse=lse, workspace=ws)
    for r in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        ws.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), out0.view(torch.int16)), f"replay {r}: out differs"
        assert torch.equal(lse, lse0), f"replay {r}: lse differs"
    check_cache(wl, t)


# --------------------------------------------------------------- invariants
def test_constant_v_and_equal_keys(dev):
    L, o = 700, 333
    c = torch.linspace(-2, 2, 128).bfloat16().float()
    vals = {
        (0, workloads.KIND_VCTX): c.expand(L, 4, 128).clone(),
        (0, workloads.KIND_VNEW): c.expand(32, 4, 128).clone(),
        (1, workloads.KIND_VNEW): c.expand(300, 4, 128).clone(),
    }
    wl = workloads.make_workload("const_v", 0, hq=28, hkv=4, d=128, decodes=[(o, L)], prefills=[300])
    wl.value_fn = lambda item, kind: vals.get((item, kind))
    _, _, out, _ = run(wl, dev)
    exp = c.to(torch.bfloat16).float().to(dev)
    assert (out.float() - exp).abs().max().item() == 0.0

    krow = torch.randn(1, 4, 128, generator=torch.Generator().manual_seed(0)).bfloat16().float()
    vals2 = {(0, workloads.KIND_KCTX): krow.expand(L, 4, 128).clone(),
             (0, workloads.KIND_KNEW): krow.expand(32, 4, 128).clone()}
    wl2 = workloads.make_workload("eq_k", 0, hq=28, hkv=4, d=128, decodes=[(o, L)], prefills=[])
    wl2.value_fn = lambda item, kind: vals2.get((item, kind))
    _, _, out2, _ = run(wl2, dev)
    V = wl2.v_ctx(0).double().clone()
    V[o:o + 32] = wl2.v_new(0).double()
    mean = V.mean(0)  # [4, 128]
    ref = mean.repeat_interleave(7, 0)[None].expand(32, 28, 128).numpy()
    compare("equal keys", out2.float().cpu().numpy(), ref)


def test_page_signature(dev):
    """All keys equal (uniform weights) and V[j, d] = 1 iff page(j) % D == d:
    o[d] is the fraction of the item's tokens on pages congruent to d, so a
    dropped or repeated page changes it by at least 1/L."""
    D = 64
    decodes = [(7, 900), (0, 33), (250, 2051)]
    wl = workloads.make_workload("pagesig", 3, hq=2, hkv=2, d=D, decodes=decodes, prefills=[])
    vals = {}
    for i in range(wl.num_items):
        L = int(wl.kv_len[i])
        o = int(wl.q_offset[i])
        pages = wl.item_pages(i)
        v = torch.zeros(L, 2, D)
        pos = np.arange(L)
        v[pos, :, pages[pos // 16] % D] = 1.0
        vals[(i, workloads.KIND_VCTX)] = v
        vals[(i, workloads.KIND_VNEW)] = v[o:o + wl.n(i)].clone()
        vals[(i, workloads.KIND_KCTX)] = torch.ones(L, 2, D)
        vals[(i, workloads.KIND_KNEW)] = torch.ones(wl.n(i), 2, D)
    wl.value_fn = lambda item, kind: vals.get((item, kind))
    _, _, out, _ = run(wl, dev)
    outc = out.float().cpu().numpy()
    for i in range(wl.num_items):
        L = int(wl.kv_len[i])
        pages = wl.item_pages(i)
        frac = np.bincount(pages[np.arange(L) // 16] % D, minlength=D) / L
        exp = torch.tensor(frac, dtype=torch.float32).bfloat16().float().numpy()
        base = int(wl.q_indptr[i])
        got = outc[base:base + wl.n(i)]
        assert np.abs(got - exp[None, None]).max() <= 2 ** -8 * max(exp.max(), 1e-3), f"item {i}"
