"""The C-ABI library loads, exports every symbol its header declares, and its
forward entry point rejects bad arguments before touching the GPU."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import workloads
from paper_2607_04206_amd import _lib, attn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def declared_symbols():
    names = set()
    for f in os.listdir(INCLUDE):
        if f.endswith(".h"):
            src = open(os.path.join(INCLUDE, f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(sangam_[a-z_0-9]+)\s*\(", src))
    return names


def test_header_declares_the_boundary():
    names = declared_symbols()
    assert {"sangam_attn_plan", "sangam_attn_forward", "sangam_plan_workspace_bytes",
            "sangam_last_error"} <= names
    assert names == set(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (sangam_[a-z_0-9]+)$", out, flags=re.M))
    missing = declared_symbols() - exported
    assert not missing, missing
    for name in declared_symbols():
        assert hasattr(_lib.lib, name)


def test_version():
    assert _lib.lib.sangam_version() == 0x000100


def _plan():
    wl = workloads.ragged_small(0, hq=4, hkv=2, d=64)
    return attn.plan(q_indptr=wl.q_indptr, q_offset=wl.q_offset, kv_len=wl.kv_len,
                     page_indptr=wl.page_indptr, page_ids=wl.page_ids, num_q_heads=4,
                     num_kv_heads=2, head_dim=64, num_pool_pages=wl.num_pool_pages,
                     sm_scale=wl.sm_scale, force_kv_splits=2)


def _fwd(plan_host, plan_dev=4096, q=4096, kn=4096, vn=4096, kc=4096, vc=4096, pool=1 << 30, pid=4096,
         npid=1 << 30, out=4096, lse=None, ws=None, wsb=0):
    # fake device addresses: every check below fails before any HIP call
    return _lib.lib.sangam_attn_forward(plan_host, plan_dev, q, kn, vn, kc, vc, pool, pid, npid, out, lse,
                                        ws, wsb, None)


def test_forward_rejects_bad_plan():
    junk = np.zeros(256, np.uint8)
    assert _fwd(junk.ctypes.data) == -8
    assert _fwd(None) == -8
    assert b"plan" in _lib.lib.sangam_last_error()


def test_forward_rejects_null_and_misaligned():
    p = _plan()
    ws = p.workspace_bytes
    assert ws > 0
    assert _fwd(p.host_ptr(), q=None, ws=4096, wsb=ws) == -1
    assert _fwd(p.host_ptr(), out=None, ws=4096, wsb=ws) == -1
    assert _fwd(p.host_ptr(), q=4096 + 8, ws=4096, wsb=ws) == -6
    assert _fwd(p.host_ptr(), kc=4096 + 2, ws=4096, wsb=ws) == -6
    assert _fwd(p.host_ptr(), lse=4096 + 2, ws=4096, wsb=ws) == -6
    # workspace missing or too small
    assert _fwd(p.host_ptr(), ws=None, wsb=0) == -5
    assert _fwd(p.host_ptr(), ws=4096, wsb=ws - 1) == -5
    assert b"workspace" in _lib.lib.sangam_last_error()


def test_forward_rejects_small_pool_and_page_table():
    p = _plan()
    ws = p.workspace_bytes
    assert _fwd(p.host_ptr(), pool=p.num_pool_pages - 1, ws=4096, wsb=ws) == -5
    assert b"pool pages" in _lib.lib.sangam_last_error()
    assert _fwd(p.host_ptr(), npid=p.total_pages - 1, ws=4096, wsb=ws) == -5
    assert b"page ids" in _lib.lib.sangam_last_error()


def test_last_error_clears_on_success():
    _plan()
    assert _lib.lib.sangam_last_error() == b""


def test_plan_info_and_workspace_query():
    p = _plan()
    assert _lib.lib.sangam_plan_workspace_bytes(p.host_ptr()) == p.workspace_bytes
    junk = np.zeros(256, np.uint8)
    assert _lib.lib.sangam_plan_workspace_bytes(junk.ctypes.data) == 0
    info = _lib.PlanInfo()
    assert _lib.lib.sangam_plan_get_info(junk.ctypes.data, ctypes.byref(info)) == -8


def test_no_undefined_kernel_stubs():
    # hipcc can silently omit host launch stubs for kernel templates; the
    # library then fails to load with an undefined __device_stub__ symbol
    out = subprocess.run(["nm", "-D", "--undefined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    assert "__device_stub__" not in out
