"""Planted mistakes in the oracle (on the CPU): each mutant of fa_oracle.c is
compiled to a scratch library and must fail at least one pin, while the
unmodified source passes them all.  This shows the pins can tell a correct
oracle from plausible wrong ones (dropped scale, wrong head map, top-left
mask, log2 lse, missing normalisation, flipped exponent sign, swapped
operand, off-by-one range)."""
import ctypes
import json
import math
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "fa_oracle.c")
GOLDEN = os.path.join(ROOT, "tests", "golden", "hand_examples.json")

MUTANTS = {
    "control": [],
    "dropped_scale": [("scores[j] = scale * dot;", "scores[j] = dot;")],
    "interleaved_head_map": [("const int g = h / G;", "const int g = h % Hkv;")],
    "top_left_mask": [("causal ? (long)i + (long)(Nk - Nq)", "causal ? (long)i")],
    "log2_lse": [("*out_lse = m + log(l);", "*out_lse = m + log2(l);")],
    "no_normalisation": [("for (int d = 0; d < D; ++d) out_row[d] /= l;", "")],
    "flipped_exponent": [("scores[j] = exp(scores[j] - m);", "scores[j] = exp(m - scores[j]);")],
    "values_from_keys": [("const double *vrow = v +", "const double *vrow = k +")],
    "off_by_one_last": [(": (long)Nk - 1;", ": (long)Nk - 2;")],
}


def build_variant(name, tmp_path):
    src = open(SRC).read()
    for old, new in MUTANTS[name]:
        assert old in src, (name, old)
        src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off", "-o",
                    str(so), str(c), "-lm"], check=True)
    lib = ctypes.CDLL(str(so))
    DP = ctypes.POINTER(ctypes.c_double)
    lib.fa_oracle_f64.argtypes = [DP] * 5 + [ctypes.c_int] * 7 + [ctypes.c_double]
    lib.fa_oracle_f64.restype = ctypes.c_int
    return lib


def run(lib, q, k, v, causal, scale):
    q, k, v = (np.ascontiguousarray(x, dtype=np.float64) for x in (q, k, v))
    B, Nq, Hq, D = q.shape
    Nk, Hkv = k.shape[1], k.shape[2]
    o = np.zeros((B, Nq, Hq, D))
    lse = np.zeros((B, Hq, Nq))
    DP = ctypes.POINTER(ctypes.c_double)
    rc = lib.fa_oracle_f64(*(a.ctypes.data_as(DP) for a in (q, k, v, o, lse)), B, Hq, Hkv, Nq,
                           Nk, D, int(causal), float(scale))
    assert rc == 0
    return o, lse


def pins_pass(lib) -> bool:
    ok = True
    for c in json.load(open(GOLDEN))["cases"]:
        o, lse = run(lib, np.array(c["q"]), np.array(c["k"]), np.array(c["v"]), c["causal"],
                     c["scale"])
        ok &= np.allclose(o, c["o"], atol=1e-12) and np.allclose(lse, c["lse"], atol=1e-12)
    # uniform closed form, causal with Nq < Nk, GQA
    r = np.random.default_rng(5)
    B, Hq, Hkv, Nq, Nk, D = 1, 4, 2, 3, 6, 2
    k = r.standard_normal((B, Nk, Hkv, D))
    v = r.standard_normal((B, Nk, Hkv, D))
    o, lse = run(lib, np.zeros((B, Nq, Hq, D)), k, v, True, 0.7)
    for h in range(Hq):
        for i in range(Nq):
            n = i + Nk - Nq + 1
            ok &= np.allclose(o[0, i, h], v[0, :n, h // 2].mean(0), atol=1e-12)
            ok &= abs(lse[0, h, i] - math.log(n)) < 1e-12
    # library cross-check (float64 softmax) on a random non-causal case
    q = r.standard_normal((1, 5, 2, 3))
    k = r.standard_normal((1, 7, 1, 3))
    v = r.standard_normal((1, 7, 1, 3))
    o, lse = run(lib, q, k, v, False, 0.6)
    s = np.einsum("bihd,bjd->bhij", q, k[:, :, 0]) * 0.6
    w = np.exp(s - s.max(-1, keepdims=True))
    w /= w.sum(-1, keepdims=True)
    ref = np.einsum("bhij,bjd->bihd", w, v[:, :, 0])
    ok &= np.allclose(o, ref, atol=1e-12)
    return bool(ok)


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_detect_planted_mistake(name, tmp_path):
    lib = build_variant(name, tmp_path)
    if name == "control":
        assert pins_pass(lib)
    else:
        assert not pins_pass(lib), f"mutant {name} was not detected"
