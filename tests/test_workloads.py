"""The seeded input generator: host and device draws agree bit for bit, and a
draw of some heads is the slice of the whole piece."""
import numpy as np
import pytest
import torch

import workloads


def torch_path(seed, item, kind, idx):
    """The torch integer path (the one device draws take), run on the CPU."""
    key = workloads.piece_key(seed, item, kind)
    h = workloads._lowbias32((workloads._mul32(idx, 0x27D4EB2F) + key) & workloads._M32)
    return workloads.normal_table("cpu")[(h >> 8) & 0xFFFF]


@pytest.mark.parametrize("seed,item,kind", [(0, 0, 0), (3, 17, 4), (2 ** 33 + 5, 255, 2)])
def test_host_draw_equals_torch_integer_path(seed, item, kind):
    n = 200_003
    got = workloads.counter_normal_bf16(seed, item, kind, (n,))
    ref = torch_path(seed, item, kind, torch.arange(n, dtype=torch.int64))
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
    # indices near 2^32 (the largest pieces): the wrap of the first multiply
    idx = torch.tensor([2 ** 32 - 1, 2 ** 32 - 2, 2 ** 31, 12345], dtype=torch.int64)
    key = workloads.piece_key(seed, item, kind)
    h = workloads._hash_u32_np(idx.numpy().astype(np.uint32), key)
    codes = torch.from_numpy(((h >> np.uint32(8)) & np.uint32(0xFFFF)).astype(np.int64))
    assert torch.equal(workloads.normal_table("cpu")[codes].view(torch.int16),
                       torch_path(seed, item, kind, idx).view(torch.int16))


def test_head_subset_is_slice():
    wl = workloads.make_workload("hs", 2, hq=12, hkv=4, d=32, decodes=[(5, 90)], prefills=[40])
    for i in range(wl.num_items):
        for f, hs in (("q", [11, 0, 5]), ("k_new", [3, 3, 1]), ("v_new", [2]), ("k_ctx", [0, 3]),
                      ("v_ctx", [1])):
            a = getattr(wl, f)(i)
            if a is None:
                continue
            b = getattr(wl, f)(i, heads=hs)
            assert torch.equal(a[:, hs].view(torch.int16), b.view(torch.int16)), (i, f)


def test_multi_row_blocks():
    wl = workloads.make_workload("mb", 1, hq=4, hkv=2, d=16, decodes=[(100, 500, 64), (0, 40, 33)],
                                 prefills=[7])
    assert [wl.n(i) for i in range(3)] == [64, 33, 7]
    assert list(wl.q_offset) == [100, 0, 0]
    assert list(wl.is_prefill) == [False, False, True]
    with pytest.raises(AssertionError):
        workloads.make_workload("bad", 1, hq=4, hkv=2, d=16, decodes=[(480, 500, 64)], prefills=[])
