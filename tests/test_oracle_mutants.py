"""Planted mistakes in a copy of the oracle must fail its pins (no GPU).

Each mutant is a one-line edit of ``oracle/ssa_oracle.c`` of the kind a careless
transcription makes: a dropped term, a wrong sign, a wrong index, a transposed
operand.  The unmodified copy, built the same way, must pass the same battery.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

from dense_ref import NAN16, page_out
from oracle import oracle as orc
from test_oracle_pins import CASES, dense_all, draw_case, run_oracle

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle",
                   "ssa_oracle.c")

MUTANTS = {
    "dropped_scale": ("scores[t] = scale * dot;", "scores[t] = dot;"),
    "exp_sign": ("scores[t] = exp(scores[t] - m);", "scores[t] = exp(m - scores[t]);"),
    "gqa_index": ("int g = h / G;", "int g = h % Hkv;"),
    "no_normalise": ("for (int d = 0; d < D; ++d) o[d] /= sum;", ""),
    "v_transposed": ("return (((size_t)page * Hkv + h) * D + d) * P + slot;",
                     "return (((size_t)page * Hkv + h) * P + slot) * D + d;"),
    "self_key_dropped": ("int64_t pos = (int64_t)ctx_len[i] + j;",
                         "int64_t pos = (int64_t)ctx_len[i] + j - 1;"),
    "weight_dropped": ("o[d] += scores[t] * bf16_to_double(", "o[d] += bf16_to_double("),
    "append_page_index": ("block_table[(size_t)i * max_pages_per_req + t / P];",
                          "block_table[(size_t)i * max_pages_per_req + t % P];"),
    "append_position": ("int64_t t = (int64_t)ctx_len[i] + j;", "int64_t t = j;"),
    "request_start": ("    q_start[i] = s;\n    s += q_len[i];", "    s += q_len[i];\n    q_start[i] = s;"),
    "prefix_ignored": ("for (int64_t t = 0; t <= pos; ++t) {\n    int64_t page = bt[t / P];\n    int slot = (int)(t % P);\n    double dot",
                       "for (int64_t t = ctx_len[i]; t <= pos; ++t) {\n    int64_t page = bt[t / P];\n    int slot = (int)(t % P);\n    double dot"),
}


def build_variant(tmp_path, name, edit):
    src = open(SRC).read()
    if edit is not None:
        old, new = edit
        assert src.count(old) == 1, name
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    c.write_text(src)
    so = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o",
                           str(so), str(c), "-lm"])
    return str(so)


def battery(lib):
    """True iff every pin below holds for the oracle in ``lib``."""
    with np.errstate(all="ignore"):
        for hq, hkv, d, P, cu in CASES:
            scale = float(np.float32(1.0 / np.sqrt(d)))
            ks, vs, qs, rng = draw_case(hq, hkv, d, P, cu, seed=hq * 31 + d)
            out = run_oracle(hq, hkv, d, P, scale, cu, ks, vs, qs, rng, lib=lib)
            ref = dense_all(hq, hkv, d, scale, cu, ks, vs, qs)
            if out.shape != ref.shape or not np.allclose(out, ref, rtol=0, atol=1e-12):
                return False
        # kv_append image
        hq, hkv, d, P = 4, 2, 16, 4
        cu = [(5, 11), (1, 30), (9, 0), (0, 7), (1, 0)]
        ks, vs, _, rng = draw_case(hq, hkv, d, P, cu, seed=14)
        bt, kfull, vfull = page_out(ks, vs, hkv, d, P, rng, spare=3)
        kc, vc = kfull.copy(), vfull.copy()
        for i, (c, u) in enumerate(cu):
            for t in range(u, u + c):
                kc[bt[i, t // P], :, t % P, :] = NAN16
                vc[bt[i, t // P], :, :, t % P] = NAN16
        k_new = np.concatenate([k[u:] for (c, u), k in zip(cu, ks)])
        v_new = np.concatenate([v[u:] for (c, u), v in zip(cu, vs)])
        k2, v2 = orc.kv_append(hkv, d, P, np.array([c for c, _ in cu], np.int32),
                               np.array([u for _, u in cu], np.int32), bt, k_new, v_new, kc, vc,
                               lib=lib)
        return bool(np.array_equal(k2, kfull) and np.array_equal(v2, vfull))


def run_battery(tmp_path, name, edit):
    """Exit status of the battery run in a child process: 0 = every pin holds,
    1 = a pin fails, anything else = the variant crashed or hung (an index
    mutant can write outside its arrays)."""
    so = build_variant(tmp_path, name, edit)
    here = os.path.dirname(os.path.abspath(__file__))
    code = ("import sys; sys.path[:0] = [%r, %r]\n"
            "from oracle import oracle as orc\n"
            "import test_oracle_mutants as m\n"
            "sys.exit(0 if m.battery(orc.bind(%r)) else 1)\n") % (here, os.path.dirname(here), so)
    try:
        return subprocess.run([sys.executable, "-c", code], capture_output=True,
                              timeout=20).returncode
    except subprocess.TimeoutExpired:  # a variant that corrupted its heap and hung
        return -9


def test_unmodified_copy_passes_the_battery(tmp_path):
    assert run_battery(tmp_path, "control", None) == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    assert run_battery(tmp_path, name, MUTANTS[name]) != 0
