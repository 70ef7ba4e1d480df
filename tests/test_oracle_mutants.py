"""The oracle's pins must catch plausible slips.

Each case copies the oracle's C source, plants one mistake by text
substitution, builds it on the CPU into a temporary library and checks that
the brute-force / closed-form comparisons reject it. The real oracle is never
modified.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import workloads
from oracle import oracle
from tests.test_oracle import brute_force, brute_force_kv

MUTANTS = {
    "scale_dropped": ("w[j] = sigma * dot;", "w[j] = dot;"),
    "exp_sign": ("w[j] = exp(w[j] - m);", "w[j] = exp(m - w[j]);"),
    "gqa_interleaved": ("const int32_t g = h / G;", "const int32_t g = h % c->hkv;"),
    "stale_block_rows": ("if (row >= 0) {", "if (row >= 0 && 0) {"),
    "positions_ignored": ("return c->q_pos ? c->q_pos[c->q_indptr[i] + r] : c->q_offset[i] + r;",
                          "return c->q_offset[i] + r;"),
    "fresh_row_shifted": ("c->fresh[base + row_pos(c, i, r)] = (int64_t)c->q_indptr[i] + r;",
                          "c->fresh[base + row_pos(c, i, r)] = (int64_t)c->q_indptr[i] + (r + 1) % "
                          "((int64_t)c->q_indptr[i + 1] - c->q_indptr[i]);"),
    "lse_log2": ("*lse = m + log(Z);", "*lse = m + log2(Z);"),
    "no_max_shift_sign": ("if (w[j] > m)", "if (w[j] < m)"),
    "value_transposed": ("out[e] += w[j] * widen(vrow[e]);",
                         "out[e] += w[j] * widen(seq_row(c, i, e % c->kv_len[i], g, 1)[j % c->d]);"),
}


def _build_mutant(tmp_path, name):
    src = open(oracle.SRC).read()
    a, b = MUTANTS[name]
    assert src.count(a) >= 1, f"mutation anchor missing: {a}"
    mut = src.replace(a, b)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(mut)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-w", "-o", str(so),
                    str(c), "-lm"], check=True)
    return str(so)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(tmp_path, monkeypatch, name):
    so = _build_mutant(tmp_path, name)
    real = oracle.lib()
    L = ctypes.CDLL(so)
    for fn in ("oracle_attn", "oracle_weights", "oracle_expected_kv", "oracle_threads"):
        getattr(L, fn).argtypes = getattr(real, fn).argtypes
        getattr(L, fn).restype = getattr(real, fn).restype
    monkeypatch.setattr(oracle, "_lib", L)
    # the brute-force pins on a tiny GQA batch with stale decode blocks and a
    # per-token decode
    wl = workloads.make_workload("mut", 5, hq=4, hkv=2, d=8, decodes=[(2, 7), (1, 9)],
                                 prefills=[5], sm_scale=0.5, pos_decodes=[([0, 3, 4], 6)])
    out, lse = oracle.attention_all(wl)
    ref_out, ref_lse = brute_force(wl)
    agrees = bool(np.all(np.abs(out - ref_out) <= 1e-6) and np.all(np.abs(lse - ref_lse) <= 1e-6))
    # and the cache after the call, assembled on its own (attention alone does
    # not see which fresh row sits at which position: keys carry no position)
    for i in range(wl.num_items):
        k, v = oracle.expected_kv(wl, i)
        rk, rv = brute_force_kv(wl, i)
        agrees = agrees and bool(np.array_equal(k, rk) and np.array_equal(v, rv))
    caught = not agrees  # NaN compares false, so a NaN result counts as caught
    assert caught, f"mutant {name} slipped through the brute-force pin"
