"""GPU parity on randomly drawn ragged batches (fixed seeds): head shapes from
MHA to 11 query heads per KV head, D 64 / 128, block decodes at random block
offsets (partial blocks and pages included), per-token position lists,
prefills, cached blocks of more than 32 rows, long prefills that take the
wide 256-row tile, forced split counts and small CU counts (which move small
decode-only GQA batches to heads-across tiles and change the split rules).
Each batch runs through the C ABI and is compared with the fp64 oracle on
every output element, LSE and written cache row."""
import numpy as np
import pytest
import torch

import workloads
from tests.test_parity import check_cache, check_full, check_pool_untouched
from tests.test_plan import parse

N_CASES = 300
SHAPES = [(4, 4), (8, 4), (12, 4), (28, 4), (32, 8), (16, 2), (11, 1), (8, 1), (6, 6), (24, 8)]


def random_batch(seed):
    rng = np.random.default_rng(7000 + seed)
    hq, hkv = SHAPES[int(rng.integers(len(SHAPES)))]
    d = int(rng.choice([64, 128]))
    decodes = []
    for _ in range(int(rng.integers(0, 6))):
        L = int(rng.integers(1, 3000))
        decodes.append((int(rng.integers(0, L)), L))
    pos = []
    for _ in range(int(rng.integers(0, 3))):
        L = int(rng.integers(2, 2000))
        k = int(rng.integers(1, min(32, L - 1) + 1))
        pos.append((np.sort(rng.choice(L, size=k, replace=False)), L))
    prefills = [int(rng.integers(1, 400)) for _ in range(int(rng.integers(0 if decodes or pos else 1, 3)))]
    force = int(rng.choice([0, 0, 0, 1, 2, 3, 7]))
    cus = int(rng.choice([0, 8, 64, 256]))
    # cached blocks of more than 32 rows (larger decode blocks, a block from 0
    # under a cached tail), or long prefills alone for the wide tile
    if rng.random() < 0.15:
        d = 128
        prefills = [int(rng.integers(1024, 2000)) for _ in range(int(rng.integers(1, 3)))]
        if hq // hkv >= 4:
            decodes, pos = [], []
    else:
        for _ in range(int(rng.integers(0, 3))):
            L = int(rng.integers(34, 3000))
            n = int(rng.integers(33, min(300, L) + 1))
            decodes.append((int(rng.integers(0, L - n + 1)), L, n))
    wl = workloads.make_workload(f"random_{seed}", seed, hq=hq, hkv=hkv, d=d, decodes=decodes,
                                 prefills=prefills, pos_decodes=pos, rng=rng)
    return wl, force, cus


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2607_04206_amd  # noqa: F401
    return torch.device("cuda:0")


@pytest.mark.gpu
@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_batch(dev, seed):
    from paper_2607_04206_amd import attn
    wl, force, cus = random_batch(seed)
    print(f"[case] random batch seed={seed}: items={wl.num_items} heads={wl.num_q_heads}/{wl.num_kv_heads} "
          f"d={wl.head_dim} force={force} cus={cus}", flush=True)
    t = workloads.device_inputs(wl, dev)
    p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                  page_ids=wl.page_ids, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                  head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale,
                  force_kv_splits=force, num_cus=cus, q_pos=wl.q_pos, device=dev)
    out, lse = attn.forward(p, t["q"], t["k_new"], t["v_new"], t["k_cache"], t["v_cache"], t["page_ids"])
    torch.cuda.synchronize()
    check_full(wl, out, lse)
    check_cache(wl, t)
    check_pool_untouched(wl, t)


def test_random_batches_reach_every_path():
    """The fixed seeds cover the launch shapes the planner can choose."""
    from paper_2607_04206_amd import attn
    seen = set()
    for seed in range(N_CASES):
        wl, force, cus = random_batch(seed)
        p = attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len, page_indptr=wl.page_indptr,
                      page_ids=wl.page_ids, num_q_heads=wl.num_q_heads, num_kv_heads=wl.num_kv_heads,
                      head_dim=wl.head_dim, num_pool_pages=wl.num_pool_pages, sm_scale=wl.sm_scale,
                      force_kv_splits=force, num_cus=cus, q_pos=wl.q_pos)
        i = p.info
        if i.num_decode_tiles:
            seen.add(f"decode_qw{i.decode_q_waves}_kw{i.decode_kv_waves}")
        if i.num_fused_decode_tiles:
            seen.add("fused" + ("_with_prefill" if i.num_prefill_tiles > i.num_fused_decode_tiles else "_alone"))
        if i.num_split_items:
            seen.add("split")
        if wl.q_pos is not None:
            seen.add("positions")
        if i.num_prefill_tiles > i.num_fused_decode_tiles:
            seen.add("prefill")
        if any(wl.n(k) > 32 and not wl.is_prefill[k] for k in range(wl.num_items)):
            seen.add("cached_block")
        if int(parse(p)[0]["prefill_rows"]) == 256:
            seen.add("wide")
    assert {"split", "positions", "prefill", "fused_with_prefill", "fused_alone", "cached_block",
            "wide"} <= seen, seen
    assert sum(s.startswith("decode_qw") for s in seen) >= 3, seen
