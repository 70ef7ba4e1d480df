"""Pins of the fp64 oracle against things other than itself.

Each pin would fail on a plausible slip in the oracle: a dropped scale, a wrong
sign, a wrong GQA index, a transposed operand, cache rows taken where fresh
rows belong (or the reverse), a wrong log base in the LSE.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import workloads
from oracle import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def custom(hq, hkv, d, decodes, prefills, values, sm_scale=None, seed=0):
    """Workload with explicit fp32 values: values[(item, kind)] -> tensor."""
    wl = workloads.make_workload("custom", seed, hq=hq, hkv=hkv, d=d, decodes=decodes,
                                 prefills=prefills, sm_scale=sm_scale)
    wl.value_fn = lambda item, kind: values.get((item, kind))
    return wl


def bf(x):
    return float(torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).float())


# ------------------------------------------------------------ brute force
def brute_force(wl):
    """Exact-rational scores, math.exp and math.fsum; assembles each item's
    sequence on its own (fresh row r at the row's position, cache rows
    elsewhere)."""
    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    G = hq // hkv
    sigma = Fraction(float(np.float32(wl.sm_scale)))
    outs, lses = [], []
    for i in range(wl.num_items):
        q = wl.q(i).float().numpy()
        kn, vn = wl.k_new(i).float().numpy(), wl.v_new(i).float().numpy()
        kc, vc = wl.k_ctx(i), wl.v_ctx(i)
        n, L = wl.n(i), int(wl.kv_len[i])
        row_at = {int(p): r for r, p in enumerate(wl.positions(i))}
        K, V = [], []
        for j in range(L):
            if j in row_at:
                K.append(kn[row_at[j]]); V.append(vn[row_at[j]])
            else:
                K.append(kc[j].float().numpy()); V.append(vc[j].float().numpy())
        out = np.zeros((n, hq, d))
        lse = np.zeros((n, hq))
        for r in range(n):
            for h in range(hq):
                g = h // G
                s = [sigma * sum(Fraction(float(q[r, h, e])) * Fraction(float(K[j][g, e])) for e in range(d))
                     for j in range(L)]
                m = max(s)
                w = [math.exp(float(sj - m)) for sj in s]
                Z = math.fsum(w)
                for e in range(d):
                    out[r, h, e] = math.fsum(w[j] * float(V[j][g, e]) for j in range(L)) / Z
                lse[r, h] = float(m) + math.log(Z)
        outs.append(out)
        lses.append(lse)
    return np.concatenate(outs), np.concatenate(lses)


def brute_force_kv(wl, i):
    """The item's cache after the call, assembled row by row on its own:
    bf16 bits [L, Hkv, D] of K and V."""
    row_at = {int(p): r for r, p in enumerate(wl.positions(i))}
    kn, vn = wl.k_new(i), wl.v_new(i)
    kc, vc = wl.k_ctx(i), wl.v_ctx(i)
    K = torch.stack([kn[row_at[j]] if j in row_at else kc[j] for j in range(int(wl.kv_len[i]))])
    V = torch.stack([vn[row_at[j]] if j in row_at else vc[j] for j in range(int(wl.kv_len[i]))])
    bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
    return bits(K), bits(V)


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2), (2, 1)])
def test_brute_force_positions(hq, hkv):
    # per-token cached decodes: scattered positions (first, last, adjacent,
    # isolated) next to a block decode and a prefill
    wl = workloads.make_workload("bfp", 8, hq=hq, hkv=hkv, d=8, decodes=[(2, 6)], prefills=[4],
                                 pos_decodes=[([1, 4, 5], 8), ([0, 6], 7), ([3], 9), ([0, 1, 2, 3, 4], 5)])
    out, lse = oracle.attention_all(wl)
    ref_out, ref_lse = brute_force(wl)
    assert np.abs(out - ref_out).max() <= 1e-14
    assert np.abs(lse - ref_lse).max() <= 1e-14
    for i in range(wl.num_items):
        k, v = oracle.expected_kv(wl, i)
        rk, rv = brute_force_kv(wl, i)
        assert np.array_equal(k, rk) and np.array_equal(v, rv), f"item {i}"


def test_contiguous_positions_equal_block_decode():
    # a position list that is a contiguous range describes the block decode
    blk = workloads.make_workload("blk", 4, hq=4, hkv=2, d=16, decodes=[(40, 100), (3, 35)], prefills=[])
    pos = workloads.make_workload("pos", 4, hq=4, hkv=2, d=16, decodes=[], prefills=[],
                                  pos_decodes=[(range(40, 72), 100), (range(3, 35), 35)])
    a, la = oracle.attention_all(blk)
    b, lb = oracle.attention_all(pos)
    assert np.array_equal(a, b) and np.array_equal(la, lb)
    for i in range(2):
        ka, va = oracle.expected_kv(blk, i)
        kb, vb = oracle.expected_kv(pos, i)
        assert np.array_equal(ka, kb) and np.array_equal(va, vb)


def test_refresh_with_cached_values_is_position_independent():
    # fresh rows equal to the cached rows they replace leave the result that
    # of the cache alone, whichever positions are refreshed; a wrong position
    # map would mix in rows from other positions
    L, n = 50, 6
    wls = []
    for k, pp in enumerate(([0, 7, 8, 30, 31, 49], [10, 11, 12, 13, 14, 15])):
        wl = workloads.make_workload(f"same{k}", 2, hq=4, hkv=4, d=16, decodes=[], prefills=[],
                                     pos_decodes=[(pp, L)])
        ctx_k, ctx_v = wl.k_ctx(0).float(), wl.v_ctx(0).float()
        q0 = workloads.make_workload("q", 2, hq=4, hkv=4, d=16, decodes=[], prefills=[],
                                     pos_decodes=[([0, 7, 8, 30, 31, 49], L)]).q(0).float()
        vals = {workloads.KIND_KNEW: ctx_k[pp].clone(), workloads.KIND_VNEW: ctx_v[pp].clone(),
                workloads.KIND_Q: q0}
        wl.value_fn = lambda item, kind, vals=vals: vals.get(kind)
        wls.append(wl)
    a, la = oracle.attention_all(wls[0])
    b, lb = oracle.attention_all(wls[1])
    assert np.array_equal(a, b) and np.array_equal(la, lb)
    # and it is the attention over the cached sequence itself
    K = wls[0].k_ctx(0).double().numpy()
    V = wls[0].v_ctx(0).double().numpy()
    q = wls[0].q(0).double().numpy()
    s = np.einsum("rhd,jhd->rhj", q, K) * float(np.float32(wls[0].sm_scale))
    w = np.exp(s - s.max(-1, keepdims=True))
    ref = np.einsum("rhj,jhd->rhd", w / w.sum(-1, keepdims=True), V)
    assert np.abs(a - ref).max() <= 1e-12


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2), (2, 1)])
def test_brute_force_tiny(hq, hkv):
    # decodes with stale cache rows in their block, a prefill, odd lengths
    wl = workloads.make_workload("bf", 7, hq=hq, hkv=hkv, d=8,
                                 decodes=[(2, 7), (0, 3), (5, 8)], prefills=[5, 1])
    out, lse = oracle.attention_all(wl)
    ref_out, ref_lse = brute_force(wl)
    assert np.abs(out - ref_out).max() <= 1e-14
    assert np.abs(lse - ref_lse).max() <= 1e-14


@pytest.mark.parametrize("hq,hkv", [(2, 2), (4, 2)])
def test_brute_force_multi_row_blocks(hq, hkv):
    # cached items with more than 32 query rows (a larger decode block, one
    # starting at 0 below a cached tail, one ending at the context's end) next
    # to a prefill: the fresh rows replace exactly their positions
    wl = workloads.make_workload("bfm", 6, hq=hq, hkv=hkv, d=4,
                                 decodes=[(3, 40, 34), (0, 37, 33), (2, 38, 36)], prefills=[3])
    assert [wl.n(i) for i in range(3)] == [34, 33, 36]
    out, lse = oracle.attention_all(wl)
    ref_out, ref_lse = brute_force(wl)
    assert np.abs(out - ref_out).max() <= 1e-14
    assert np.abs(lse - ref_lse).max() <= 1e-14
    for i in range(3):
        k, v = oracle.expected_kv(wl, i)
        rk, rv = brute_force_kv(wl, i)
        assert np.array_equal(k, rk) and np.array_equal(v, rv), f"item {i}"


@pytest.mark.parametrize("hq,hkv", [(28, 4), (8, 8)])
def test_head_subset_call_equals_full_call(hq, hkv):
    # the reduced call that draws only the chosen heads (each paired with its
    # own KV head) returns, bit for bit, the full call's values for them
    wl = workloads.make_workload("sub", 5, hq=hq, hkv=hkv, d=64, decodes=[(30, 200), (0, 45, 40)],
                                 prefills=[70])
    full, full_lse = oracle.attention_all(wl)
    heads = [hq - 1, 0, hq // 2, 1]
    res = oracle.attention(wl, heads=heads)
    for i, (rr, o, l) in res.items():
        base = int(wl.q_indptr[i])
        assert np.array_equal(o, full[base + rr][:, heads]), f"item {i}"
        assert np.array_equal(l, full_lse[base + rr][:, heads]), f"item {i}"


def test_brute_force_scale():
    wl = workloads.make_workload("bf", 3, hq=2, hkv=1, d=4, decodes=[(1, 6)], prefills=[4],
                                 sm_scale=0.3)
    out, lse = oracle.attention_all(wl)
    ref_out, ref_lse = brute_force(wl)
    assert np.abs(out - ref_out).max() <= 1e-14
    assert np.abs(lse - ref_lse).max() <= 1e-14


# ------------------------------------------------------- library routine
def sdpa_reference(wl):
    """torch float64 scaled_dot_product_attention, non-causal, KV heads
    repeated G times; the sequence assembled with torch indexing."""
    hq, hkv = wl.num_q_heads, wl.num_kv_heads
    G = hq // hkv
    outs = []
    for i in range(wl.num_items):
        o, n, L = int(wl.q_offset[i]), wl.n(i), int(wl.kv_len[i])
        if wl.is_prefill[i]:
            K, V = wl.k_new(i).double(), wl.v_new(i).double()
        else:
            K, V = wl.k_ctx(i).double().clone(), wl.v_ctx(i).double().clone()
            K[o:o + n] = wl.k_new(i).double()
            V[o:o + n] = wl.v_new(i).double()
        q = wl.q(i).double().permute(1, 0, 2)  # [hq, n, d]
        K = K.permute(1, 0, 2).repeat_interleave(G, 0)
        V = V.permute(1, 0, 2).repeat_interleave(G, 0)
        y = torch.nn.functional.scaled_dot_product_attention(
            q, K, V, is_causal=False, scale=float(np.float32(wl.sm_scale)))
        outs.append(y.permute(1, 0, 2).numpy())
    return np.concatenate(outs)


@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (4, 4, 64)])
def test_matches_torch_sdpa(hq, hkv, d):
    wl = workloads.make_workload("sdpa", 11, hq=hq, hkv=hkv, d=d,
                                 decodes=[(40, 300), (288, 320)], prefills=[257])
    out, _ = oracle.attention_all(wl)
    ref = sdpa_reference(wl)
    assert np.abs(out - ref).max() <= 1e-12


# ----------------------------------------------------------- closed forms
def test_golden_two_key():
    vals = {}
    with open(os.path.join(GOLDEN, "two_key_softmax.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    t = torch.tensor
    values = {
        (0, workloads.KIND_Q): t([[[1.0, 0.0]]]),
        (0, workloads.KIND_KNEW): t([[[1.0, 0.0]], [[0.0, 0.0]]]),
        (0, workloads.KIND_VNEW): t([[[1.0, 0.0]], [[0.0, 1.0]]]),
    }
    # a prefill of L = 2 has n = 2 query rows; give row 1 the same query
    values[(0, workloads.KIND_Q)] = t([[[1.0, 0.0]], [[1.0, 0.0]]])
    wl = custom(1, 1, 2, [], [2], values, sm_scale=1.0)
    out, lse = oracle.attention_all(wl)
    assert abs(out[0, 0, 0] - vals["o0"]) <= 1e-15
    assert abs(out[0, 0, 1] - vals["o1"]) <= 1e-15
    assert abs(lse[0, 0] - vals["lse"]) <= 1e-15


def test_two_keys_logistic_with_scale():
    rng = torch.Generator().manual_seed(5)
    d = 16
    q = torch.randn(2, 1, d, generator=rng).bfloat16().float()
    k = torch.randn(2, 1, d, generator=rng).bfloat16().float()
    v = torch.randn(2, 1, d, generator=rng).bfloat16().float()
    sig = 0.25
    wl = custom(1, 1, d, [], [2], {(0, workloads.KIND_Q): q, (0, workloads.KIND_KNEW): k,
                                   (0, workloads.KIND_VNEW): v}, sm_scale=sig)
    out, lse = oracle.attention_all(wl)
    qd, kd, vd = q.double().numpy(), k.double().numpy(), v.double().numpy()
    for r in range(2):
        s0 = sig * float(qd[r, 0] @ kd[0, 0])
        s1 = sig * float(qd[r, 0] @ kd[1, 0])
        lam = 1.0 / (1.0 + math.exp(-(s0 - s1)))
        exp_o = lam * vd[0, 0] + (1 - lam) * vd[1, 0]
        assert np.abs(out[r, 0] - exp_o).max() <= 1e-13
        assert abs(lse[r, 0] - (max(s0, s1) + math.log1p(math.exp(-abs(s0 - s1))))) <= 1e-13


def test_single_key():
    # L = 1: o = v0 and lse = s0
    wl = workloads.make_workload("one", 2, hq=4, hkv=2, d=64, decodes=[], prefills=[1])
    out, lse = oracle.attention_all(wl)
    q, k, v = wl.q(0).double(), wl.k_new(0).double(), wl.v_new(0).double()
    for h in range(4):
        g = h // 2
        assert np.abs(out[0, h] - v[0, g].numpy()).max() == 0.0
        s0 = float(np.float32(wl.sm_scale)) * float(q[0, h] @ k[0, g])
        assert abs(lse[0, h] - s0) <= 1e-12


def test_zero_query_gives_mean():
    # Q = 0: uniform weights, o = mean of the assembled V, lse = ln L
    L, o = 45, 13
    wl = workloads.make_workload("zq", 4, hq=2, hkv=2, d=32, decodes=[(o, L)], prefills=[])
    base_q = wl.q
    wl.value_fn = lambda item, kind: torch.zeros(32, 2, 32) if kind == workloads.KIND_Q else None
    out, lse = oracle.attention_all(wl)
    V = wl.v_ctx(0).double().clone()
    V[o:o + 32] = wl.v_new(0).double()
    mean = V.mean(0).numpy()  # [hkv, d]
    assert np.abs(out - mean[None]).max() <= 1e-14
    assert np.abs(lse - math.log(L)).max() <= 1e-14
    del base_q


def test_weights_sum_to_one():
    wl = workloads.ragged_small(0, hq=4, hkv=2, d=64)
    rows = [0, 5, wl.total_q - 1, int(wl.q_indptr[3]) + 2]
    for r in rows:
        for h in (0, 3):
            w = oracle.weights(wl, r, h)
            assert abs(w.sum() - 1.0) <= 1e-13
            assert (w >= 0).all()


def test_weights_match_softmax_of_exact_scores():
    # the debug entry's weights of every (packed row, head) against a softmax
    # taken here of exact-rational scores over the item's own assembled
    # sequence: a wrong row, head, KV group or position map shows
    wl = workloads.make_workload("w", 9, hq=4, hkv=2, d=8, decodes=[(3, 11), (0, 6, 5)], prefills=[7],
                                 pos_decodes=[([1, 6], 9)])
    G = 2
    sigma = Fraction(float(np.float32(wl.sm_scale)))
    for i in range(wl.num_items):
        q = wl.q(i).float().numpy()
        kn = wl.k_new(i).float().numpy()
        kc = wl.k_ctx(i)
        row_at = {int(p): r for r, p in enumerate(wl.positions(i))}
        L = int(wl.kv_len[i])
        K = [kn[row_at[j]] if j in row_at else kc[j].float().numpy() for j in range(L)]
        for r in range(wl.n(i)):
            for h in range(4):
                s = [sigma * sum(Fraction(float(q[r, h, e])) * Fraction(float(K[j][h // G, e])) for e in range(8))
                     for j in range(L)]
                m = max(s)
                e = [math.exp(float(sj - m)) for sj in s]
                Z = math.fsum(e)
                w = oracle.weights(wl, int(wl.q_indptr[i]) + r, h)
                assert np.abs(w - np.asarray(e) / Z).max() <= 1e-15, (i, r, h)


# -------------------------------------------------------------- invariants
def test_constant_v():
    L = 77
    c = torch.linspace(-3, 3, 64).bfloat16().float()
    vals = {(0, workloads.KIND_VCTX): c.expand(L, 2, 64).clone(),
            (0, workloads.KIND_VNEW): c.expand(32, 2, 64).clone(),
            (1, workloads.KIND_VNEW): c.expand(50, 2, 64).clone()}
    wl = custom(4, 2, 64, [(10, L)], [50], vals)
    out, _ = oracle.attention_all(wl)
    assert np.abs(out - c.double().numpy()).max() <= 1e-14


def test_equal_keys_give_mean_v():
    L, o = 90, 40
    krow = torch.randn(1, 2, 64, generator=torch.Generator().manual_seed(3)).bfloat16().float()
    vals = {(0, workloads.KIND_KCTX): krow.expand(L, 2, 64).clone(),
            (0, workloads.KIND_KNEW): krow.expand(32, 2, 64).clone()}
    wl = custom(6, 2, 64, [(o, L)], [], vals)
    out, lse = oracle.attention_all(wl)
    V = wl.v_ctx(0).double().clone()
    V[o:o + 32] = wl.v_new(0).double()
    mean = V.mean(0).numpy()
    G = 3
    for h in range(6):
        assert np.abs(out[:, h] - mean[h // G]).max() <= 1e-14


def test_block_row_permutation():
    wl = workloads.make_workload("perm", 8, hq=4, hkv=2, d=64, decodes=[(20, 200)], prefills=[])
    out, lse = oracle.attention_all(wl)
    perm = torch.randperm(32, generator=torch.Generator().manual_seed(1))
    q, kn, vn = wl.q(0).float(), wl.k_new(0).float(), wl.v_new(0).float()
    # permuting the query rows alone permutes the outputs
    wl2 = workloads.make_workload("perm", 8, hq=4, hkv=2, d=64, decodes=[(20, 200)], prefills=[])
    wl2.value_fn = lambda item, kind: q[perm] if kind == workloads.KIND_Q else None
    out2, lse2 = oracle.attention_all(wl2)
    assert np.abs(out2 - out[perm.numpy()]).max() <= 1e-14
    assert np.abs(lse2 - lse[perm.numpy()]).max() <= 1e-14
    # permuting block rows jointly (Q, K, V) permutes outputs too (the keys
    # move inside the bidirectional context, which the softmax ignores)
    wl3 = workloads.make_workload("perm", 8, hq=4, hkv=2, d=64, decodes=[(20, 200)], prefills=[])
    m = {workloads.KIND_Q: q[perm], workloads.KIND_KNEW: kn[perm], workloads.KIND_VNEW: vn[perm]}
    wl3.value_fn = lambda item, kind: m.get(kind)
    out3, lse3 = oracle.attention_all(wl3)
    assert np.abs(out3 - out[perm.numpy()]).max() <= 1e-13
    assert np.abs(lse3 - lse[perm.numpy()]).max() <= 1e-13


def test_prefill_token_permutation():
    L = 61
    wl = workloads.make_workload("pp", 9, hq=2, hkv=1, d=64, decodes=[], prefills=[L])
    out, lse = oracle.attention_all(wl)
    perm = torch.randperm(L, generator=torch.Generator().manual_seed(2))
    m = {workloads.KIND_Q: wl.q(0).float()[perm], workloads.KIND_KNEW: wl.k_new(0).float()[perm],
         workloads.KIND_VNEW: wl.v_new(0).float()[perm]}
    wl2 = workloads.make_workload("pp", 9, hq=2, hkv=1, d=64, decodes=[], prefills=[L])
    wl2.value_fn = lambda item, kind: m.get(kind)
    out2, lse2 = oracle.attention_all(wl2)
    assert np.abs(out2 - out[perm.numpy()]).max() <= 1e-13
    assert np.abs(lse2 - lse[perm.numpy()]).max() <= 1e-13


def test_batch_item_permutation():
    wl = workloads.ragged_small(1, hq=4, hkv=4, d=64)
    res = oracle.attention(wl)
    order = list(reversed(range(wl.num_items)))
    res2 = oracle.attention(wl, items=order)
    for i in range(wl.num_items):
        assert np.array_equal(res[i][1], res2[i][1])
        assert np.array_equal(res[i][2], res2[i][2])


def test_gqa_equals_repeated_mha():
    G = 7
    wl = workloads.make_workload("gqa", 12, hq=14, hkv=2, d=64, decodes=[(7, 100)], prefills=[33])
    out, lse = oracle.attention_all(wl)
    rep = {}
    for i in range(wl.num_items):
        rep[(i, workloads.KIND_Q)] = wl.q(i).float()
        for kind, fn in ((workloads.KIND_KNEW, wl.k_new), (workloads.KIND_VNEW, wl.v_new),
                         (workloads.KIND_KCTX, wl.k_ctx), (workloads.KIND_VCTX, wl.v_ctx)):
            t = fn(i)
            if t is not None:
                rep[(i, kind)] = t.float().repeat_interleave(G, 1)
    wl2 = custom(14, 14, 64, [(7, 100)], [33], rep)
    out2, lse2 = oracle.attention_all(wl2)
    assert np.array_equal(out, out2)
    assert np.array_equal(lse, lse2)


def test_decode_rows_equal_prefill_rows():
    # the single-request workload: decode of rows 96..127 over the prefill's KV
    wl = workloads.tiny_mixed(0)
    out, lse = oracle.attention_all(wl)
    assert np.abs(out[:32] - out[32 + 96:32 + 128]).max() <= 1e-14
    assert np.abs(lse[:32] - lse[32 + 96:32 + 128]).max() <= 1e-14


def test_expected_kv_assembly():
    wl = workloads.ragged_small(2, hq=2, hkv=2, d=64)
    for i in range(wl.num_items):
        k, v = oracle.expected_kv(wl, i)
        o, n, L = int(wl.q_offset[i]), wl.n(i), int(wl.kv_len[i])
        kn = wl.k_new(i).view(torch.int16).numpy().view(np.uint16)
        vn = wl.v_new(i).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(k[o:o + n], kn) and np.array_equal(v[o:o + n], vn)
        if not wl.is_prefill[i]:
            kc = wl.k_ctx(i).view(torch.int16).numpy().view(np.uint16)
            vc = wl.v_ctx(i).view(torch.int16).numpy().view(np.uint16)
            keep = np.r_[0:o, o + n:L]
            assert np.array_equal(k[keep], kc[keep]) and np.array_equal(v[keep], vc[keep])
            # the stale block rows really were different (the test can see a mix-up)
            assert not np.array_equal(kc[o:o + n], kn)


def test_rejects_invalid_calls():
    wl = workloads.make_workload("bad", 0, hq=2, hkv=2, d=8, decodes=[], prefills=[4])
    call = oracle.Call(wl)
    call.q_offset[0] = 1  # o + n > L
    out = np.empty((8, 8))
    lse = np.empty(8)
    rc = oracle.lib().oracle_attn(*call.args(), None, 0, oracle._ptr(out), oracle._ptr(lse))
    assert rc != 0


def test_sampled_rows_match_full():
    wl = workloads.ragged_small(3, hq=4, hkv=2, d=128)
    full, full_lse = oracle.attention_all(wl)
    rows = {0: [0, 3], 5: [1], 9: [0, 149]}
    res = oracle.attention(wl, items=[9, 0, 5], rows=rows, heads=[1, 3])
    for i, (rr, out, lse) in res.items():
        base = int(wl.q_indptr[i])
        for a, r in enumerate(rr):
            assert np.array_equal(out[a], full[base + r][[1, 3]])
            assert np.array_equal(lse[a], full_lse[base + r][[1, 3]])
