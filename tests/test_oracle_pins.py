"""Pins for the fp64 oracle: checks against what the paper and the mathematics
fix, independent of the oracle's own code.

Each test names the plausible oracle mistake it would catch.  The oracle is
the plain definition of Sec. 2 (softmax(q k^T * scale) v per head) with the
head map of Sec. 4.1.1; the streaming recurrence of Alg. 1 and the blocked
state carry of Alg. 2 are transcribed separately below and must reach the same
values by brute force on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def rnd(shape, seed, lo=None, hi=None):
    r = np.random.default_rng(seed)
    if lo is None:
        return r.standard_normal(shape)
    return r.uniform(lo, hi, shape)


def qkv(B, Hq, Hkv, Nq, Nk, D, seed=0):
    return (rnd((B, Nq, Hq, D), seed), rnd((B, Nk, Hkv, D), seed + 1),
            rnd((B, Nk, Hkv, D), seed + 2))


def visible(i, Nq, Nk, causal):
    return i + (Nk - Nq) + 1 if causal else Nk


# --------------------------------------------------------------- hand examples
@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_derived_examples(case):
    """Closed forms derived on paper (tests/golden): catches a dropped or
    misplaced scale, log2 instead of ln in lse, the wrong head map, a
    top-left causal mask, a missing normalisation."""
    q, k, v = (np.array(case[x], dtype=np.float64) for x in ("q", "k", "v"))
    o, lse = oracle.attention(q, k, v, bool(case["causal"]), case["scale"])
    np.testing.assert_allclose(o, np.array(case["o"]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, np.array(case["lse"]), rtol=0, atol=1e-14)


# ------------------------------------------------------------------ invariants
@pytest.mark.parametrize("causal", [False, True])
def test_weight_rows_sum_to_one(causal):
    """Softmax rows are distributions (catches a wrong normaliser)."""
    q, k, v = qkv(2, 4, 2, 7, 9, 5, seed=3)
    w = oracle.weights(q, k, v, causal, 0.7)
    assert np.all(w >= 0)
    np.testing.assert_allclose(w.sum(-1), 1.0, rtol=0, atol=1e-12)
    if causal:  # masked keys carry exactly zero weight (bottom-right)
        for i in range(7):
            assert np.all(w[:, :, i, visible(i, 7, 9, True):] == 0)


@pytest.mark.parametrize("causal", [False, True])
def test_weights_against_torch_softmax(causal):
    """The weight entry point against torch's float64 softmax of the scaled
    scores with an explicit bottom-right mask, per query head on its key/value
    head h // G (catches a wrong scale, a wrong head map or mask, or an
    unnormalised row in the weights the unfused path is checked against)."""
    import torch

    B, Hq, Hkv, Nq, Nk, D, scale = 2, 6, 2, 5, 8, 3, 0.8
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=21)
    w = oracle.weights(q, k, v, causal, scale)
    G = Hq // Hkv
    qt, kt = torch.from_numpy(q), torch.from_numpy(k)
    for b in range(B):
        for h in range(Hq):
            s = (qt[b, :, h, :] @ kt[b, :, h // G, :].T) * scale          # [Nq, Nk]
            if causal:
                i = torch.arange(Nq)[:, None]
                j = torch.arange(Nk)[None, :]
                s = s.masked_fill(j > i + (Nk - Nq), float("-inf"))
            ref = torch.softmax(s, dim=-1).numpy()
            np.testing.assert_allclose(w[b, h], ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_weights_times_values_is_the_output(causal):
    """sum_j w_ij v_j equals the attention output of the other entry point
    (catches the two entry points disagreeing on the head map, the mask or the
    normalisation)."""
    B, Hq, Hkv, Nq, Nk, D, scale = 2, 4, 2, 6, 7, 5, 1.1
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=22)
    w = oracle.weights(q, k, v, causal, scale)
    o, _ = oracle.attention(q, k, v, causal, scale)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            np.testing.assert_allclose(w[b, h] @ v[b, :, h // G, :], o[b, :, h, :], rtol=0, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_all_ones_values(causal):
    """V = 1 gives O = 1 for every row (catches missing division by l)."""
    q, k, _ = qkv(1, 3, 1, 6, 8, 4, seed=5)
    v = np.ones((1, 8, 1, 4))
    o, _ = oracle.attention(q, k, v, causal, 1.3)
    np.testing.assert_allclose(o, 1.0, rtol=0, atol=1e-14)


@pytest.mark.parametrize("causal,zero", [(False, "q"), (True, "q"), (False, "scale"),
                                         (True, "scale")])
def test_uniform_weights_closed_form(causal, zero):
    """q = 0 (or scale = 0) gives the mean of the visible V rows and
    lse = ln(#visible); with Nq < Nk this pins the bottom-right alignment and
    catches an off-by-one in the last visible key."""
    B, Hq, Hkv, Nq, Nk, D = 2, 4, 2, 5, 9, 3
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=11)
    scale = 0.9
    if zero == "q":
        q = np.zeros_like(q)
    else:
        scale = 0.0
    o, lse = oracle.attention(q, k, v, causal, scale)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            for i in range(Nq):
                n = visible(i, Nq, Nk, causal)
                np.testing.assert_allclose(o[b, i, h], v[b, :n, h // G].mean(0), rtol=0,
                                           atol=1e-13)
                assert abs(lse[b, h, i] - math.log(n)) < 1e-13


def test_dominant_score_selects_its_value_row():
    """q_i = alpha * k_j* with orthonormal key rows: the output tends to
    V[j*] with error at most (Nk-1) e^{-gap} max|V| (catches a sign error in the
    max subtraction or a transposed operand)."""
    Nk, D, alpha = 6, 8, 40.0
    basis, _ = np.linalg.qr(rnd((D, D), 21))
    k = basis[:Nk].reshape(1, Nk, 1, D)
    v = rnd((1, Nk, 1, D), 22)
    for jstar in range(Nk):
        q = (alpha * basis[jstar]).reshape(1, 1, 1, D)
        o, lse = oracle.attention(q, k, v, False, 1.0)
        gap = alpha  # s_j* = alpha, every other s_j = 0
        bound = (Nk - 1) * math.exp(-gap) * np.abs(v).max() * 2
        assert np.abs(o[0, 0, 0] - v[0, jstar, 0]).max() <= bound
        assert abs(lse[0, 0, 0] - (alpha + math.log1p((Nk - 1) * math.exp(-alpha)))) < 1e-12


def test_gqa_equals_mha_on_replicated_heads():
    """GQA with G = Hq/Hkv equals MHA on K/V heads repeated G times in
    contiguous groups (Sec. 4.1.1 replication); catches an interleaved head map."""
    B, Hq, Hkv, Nq, Nk, D = 2, 6, 2, 4, 7, 5
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=31)
    G = Hq // Hkv
    kr, vr = np.repeat(k, G, axis=2), np.repeat(v, G, axis=2)
    for causal in (False, True):
        o1, l1 = oracle.attention(q, k, v, causal, 0.4)
        o2, l2 = oracle.attention(q, kr, vr, causal, 0.4)
        np.testing.assert_array_equal(o1, o2)
        np.testing.assert_array_equal(l1, l2)


def test_mqa_equals_per_head_loop():
    """MQA (Hkv = 1): every query head attends the single K/V head; equals
    separate single-head calls."""
    B, Hq, Nq, Nk, D = 1, 5, 3, 6, 4
    q, k, v = qkv(B, Hq, 1, Nq, Nk, D, seed=41)
    o, lse = oracle.attention(q, k, v, True, 0.6)
    for h in range(Hq):
        oh, lh = oracle.attention(q[:, :, h:h + 1], k, v, True, 0.6)
        np.testing.assert_array_equal(o[:, :, h:h + 1], oh)
        np.testing.assert_array_equal(lse[:, h:h + 1], lh)


def test_causal_special_cases():
    """Row 0 of a square causal call is exactly V row 0; decode (Nq=1) causal
    equals non-causal; the last causal prefill row equals decode; every causal
    row equals non-causal attention over the truncated keys (bottom-right)."""
    B, H, N, D = 1, 2, 8, 4
    q, k, v = qkv(B, H, H, N, N, D, seed=51)
    o, lse = oracle.attention(q, k, v, True, 0.5)
    np.testing.assert_array_equal(o[:, 0], v[:, 0])
    od_c, ld_c = oracle.attention(q[:, -1:], k, v, True, 0.5)
    od_n, ld_n = oracle.attention(q[:, -1:], k, v, False, 0.5)
    np.testing.assert_array_equal(od_c, od_n)
    np.testing.assert_allclose(o[:, -1:], od_n, rtol=0, atol=1e-14)
    Nq = 3
    qs = q[:, :Nq]
    oc, lc = oracle.attention(qs, k, v, True, 0.5)
    for i in range(Nq):
        n = visible(i, Nq, N, True)
        oi, li = oracle.attention(qs[:, i:i + 1], k[:, :n], v[:, :n], False, 0.5)
        np.testing.assert_allclose(oc[:, i:i + 1], oi, rtol=0, atol=1e-14)
        np.testing.assert_allclose(lc[:, :, i:i + 1], li, rtol=0, atol=1e-14)


# ------------------------------------------------ independent transcriptions
def alg1_streaming_row(qrow, K, V, scale):
    """Per-key streaming softmax of Alg. 1: running maximum M, running sum,
    rescale factor ms = exp(M_old - M) applied to the accumulator when a new
    maximum arrives (strict >), weight vs = exp(S - M) otherwise, then one
    normalisation at the end.  Returns (o, lse)."""
    M = -math.inf
    Sum = 0.0
    VKQ = np.zeros(V.shape[1])
    for kr, vr in zip(K, V):
        S = float(np.dot(qrow, kr)) * scale
        M_old = M
        ms, vs = 1.0, 1.0
        if S > M:
            M = S
            ms = math.exp(M_old - M)
            VKQ = VKQ * ms
        else:
            vs = math.exp(S - M)
        VKQ = VKQ + vr * vs
        Sum = Sum * ms + vs
    return VKQ / Sum, M + math.log(Sum)


def blocked_rows(Q, K, V, scale, causal, Br, Bc, off):
    """Blocked form with state carried across key blocks (Alg. 2): for each
    block of Br query rows, running max / sum / accumulator are initialised
    at the first key block and updated block by block; the accumulator is
    normalised once after the last key block (the reading the design notes
    give for the normalisation placement)."""
    Nq, D = Q.shape
    Nk = K.shape[0]
    out = np.zeros((Nq, D))
    lse = np.zeros(Nq)
    for r0 in range(0, Nq, Br):
        rows = np.arange(r0, min(r0 + Br, Nq))
        m = np.full(len(rows), -math.inf)
        l = np.zeros(len(rows))
        acc = np.zeros((len(rows), D))
        for c0 in range(0, Nk, Bc):
            cols = np.arange(c0, min(c0 + Bc, Nk))
            S = (Q[rows] @ K[cols].T) * scale
            if causal:
                S = np.where(cols[None, :] <= rows[:, None] + off, S, -math.inf)
            m_new = np.maximum(m, S.max(axis=1))
            base = np.where(np.isinf(m_new), 0.0, m_new)  # fully masked so far
            alpha = np.exp(m - base)
            P = np.exp(S - base[:, None])
            l = l * alpha + P.sum(axis=1)
            acc = acc * alpha[:, None] + P @ V[cols]
            m = m_new
        out[rows] = acc / l[:, None]
        lse[rows] = m + np.log(l)
    return out, lse


@pytest.mark.parametrize("causal", [False, True])
def test_alg1_streaming_equals_direct(causal):
    """Alg. 1's per-key recurrence (transcribed above) matches the oracle to
    1e-12 relative, brute force over small shapes."""
    for Nq, Nk, D in [(1, 1, 1), (3, 5, 2), (4, 4, 3), (2, 9, 4)]:
        if causal and Nq > Nk:
            continue
        q, k, v = qkv(1, 2, 1, Nq, Nk, D, seed=61 + Nq * 10 + Nk)
        o, lse = oracle.attention(q, k, v, causal, 0.8)
        for h in range(2):
            for i in range(Nq):
                n = visible(i, Nq, Nk, causal)
                oi, li = alg1_streaming_row(q[0, i, h], k[0, :n, 0], v[0, :n, 0], 0.8)
                np.testing.assert_allclose(o[0, i, h], oi, rtol=1e-12, atol=1e-13)
                assert abs(lse[0, h, i] - li) <= 1e-12 * max(1.0, abs(li))


def test_blocked_tiling_equals_direct_brute_force():
    """Every block shape Br in [1, Nq], Bc in [1, Nk] of the blocked state
    carry reaches the oracle's value (Nq, Nk <= 9, D <= 4, causal both ways,
    G in {1, 2, 3})."""
    shapes = [(1, 1, 1), (3, 7, 2), (5, 5, 4), (9, 9, 3), (2, 9, 1), (7, 8, 2)]
    for (Nq, Nk, D), causal, G in itertools.product(shapes, (False, True), (1, 2, 3)):
        if causal and Nq > Nk:
            continue
        Hkv = 1
        q, k, v = qkv(1, G * Hkv, Hkv, Nq, Nk, D, seed=71 + Nq + 13 * Nk + D)
        o, lse = oracle.attention(q, k, v, causal, 0.55)
        for h in range(G):
            for Br in range(1, Nq + 1):
                for Bc in range(1, Nk + 1):
                    ob, lb = blocked_rows(q[0, :, h], k[0, :, 0], v[0, :, 0], 0.55, causal,
                                          Br, Bc, Nk - Nq)
                    np.testing.assert_allclose(o[0, :, h], ob, rtol=1e-12, atol=1e-13)
                    np.testing.assert_allclose(lse[0, h], lb, rtol=1e-12, atol=1e-13)


def merge_partials(parts):
    """Log-sum-exp merge of partial results over disjoint key ranges:
    lse = log sum_s exp(lse_s), o = sum_s exp(lse_s - lse) o_s."""
    lses = np.stack([p[1] for p in parts])
    top = lses.max(axis=0)
    lse = top + np.log(np.exp(lses - top).sum(axis=0))
    o = sum(np.exp(p[1] - lse)[..., None] * p[0] for p in parts)
    return o, lse


def test_split_kv_merge_equals_unsplit():
    """Decode split-KV: for every set of split points over a tiny key range,
    merging per-split (o_s, lse_s) by log-sum-exp gives the unsplit result
    and the unsplit lse."""
    B, Hq, Hkv, Nk, D = 2, 4, 2, 7, 3
    q, k, v = qkv(B, Hq, Hkv, 1, Nk, D, seed=81)
    o_ref, l_ref = oracle.attention(q, k, v, False, 0.9)
    for r in range(1, Nk):
        for cuts in itertools.combinations(range(1, Nk), r):
            edges = (0,) + cuts + (Nk,)
            parts = []
            for a, b in zip(edges[:-1], edges[1:]):
                o_s, l_s = oracle.attention(q, k[:, a:b], v[:, a:b], False, 0.9)
                parts.append((o_s[:, 0], l_s[..., 0].transpose(0, 1)))
            o_m, l_m = merge_partials([(p[0], p[1]) for p in parts])
            np.testing.assert_allclose(o_m, o_ref[:, 0], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(l_m, l_ref[..., 0], rtol=1e-12, atol=1e-13)


# ------------------------------------------------------ library cross-checks
@pytest.mark.parametrize("shape", [(1, 2, 2, 128, 128, 64, False), (1, 4, 1, 64, 96, 32, True),
                                   (2, 8, 2, 33, 33, 16, True)])
def test_matches_torch_softmax_float64(shape):
    """Reduction to library routines: torch float64 matmul + softmax with an
    explicit bottom-right mask (and logsumexp) match the oracle to 1e-12."""
    import torch

    B, Hq, Hkv, Nq, Nk, D, causal = shape
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=91)
    scale = 1.0 / math.sqrt(D)
    o, lse = oracle.attention(q, k, v, causal, scale)
    G = Hq // Hkv
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)                       # B H Nq D
    tk = torch.from_numpy(np.repeat(k, G, axis=2)).permute(0, 2, 1, 3)  # B H Nk D
    tv = torch.from_numpy(np.repeat(v, G, axis=2)).permute(0, 2, 1, 3)
    s = torch.matmul(tq, tk.transpose(-1, -2)) * scale
    if causal:
        i = torch.arange(Nq)[:, None]
        j = torch.arange(Nk)[None, :]
        s = s.masked_fill(j > i + (Nk - Nq), float("-inf"))
    ref = torch.matmul(torch.softmax(s, dim=-1), tv).permute(0, 2, 1, 3).numpy()
    ref_lse = torch.logsumexp(s, dim=-1).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)


def test_linearity_permutation_and_lse_brute_force():
    """Linear in V; jointly permuting K and V rows leaves non-causal output
    unchanged; exp(lse) equals the brute-force sum of exp(scores)."""
    B, Hq, Hkv, Nq, Nk, D = 1, 2, 1, 3, 6, 4
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=101)
    v2 = rnd(v.shape, 102)
    a, b = 1.7, -0.3
    o1, _ = oracle.attention(q, k, v, False, 0.7)
    o2, _ = oracle.attention(q, k, v2, False, 0.7)
    o3, lse = oracle.attention(q, k, a * v + b * v2, False, 0.7)
    np.testing.assert_allclose(o3, a * o1 + b * o2, rtol=1e-12, atol=1e-13)
    perm = np.random.default_rng(7).permutation(Nk)
    o4, l4 = oracle.attention(q, k[:, perm], v[:, perm], False, 0.7)
    np.testing.assert_allclose(o4, o1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l4, lse, rtol=1e-12, atol=1e-13)
    for h in range(Hq):
        for i in range(Nq):
            tot = sum(math.exp(0.7 * float(np.dot(q[0, i, h], k[0, j, 0]))) for j in range(Nk))
            assert abs(math.exp(lse[0, h, i]) - tot) <= 1e-12 * tot


# ------------------------------------------------------------- plumbing
def test_rows_entry_and_fanout_match_full_pass():
    """The row entry point and the process fan-out give bit-identical rows."""
    B, Hq, Hkv, Nq, Nk, D = 2, 4, 2, 9, 11, 8
    q, k, v = qkv(B, Hq, Hkv, Nq, Nk, D, seed=111)
    o, lse = oracle.attention(q, k, v, True, 0.3)
    o_p, l_p = oracle.attention_parallel(q, k, v, True, 0.3, workers=3)
    np.testing.assert_array_equal(o, o_p)
    np.testing.assert_array_equal(lse, l_p)
    rows = np.array([[1, 3, 8], [0, 0, 0], [1, 0, 4]])
    o_r, l_r = oracle.attention_rows(q, k, v, True, 0.3, rows)
    for n, (b, h, i) in enumerate(rows):
        np.testing.assert_array_equal(o_r[n], o[b, i, h])
        assert l_r[n] == lse[b, h, i]


@pytest.mark.parametrize("bad", ["ratio", "causal", "rows"])
def test_oracle_rejects_invalid_arguments(bad):
    q, k, v = qkv(1, 3, 2, 4, 4, 2, seed=1)
    with pytest.raises(ValueError):
        if bad == "ratio":
            oracle.attention(q, k, v, False, 1.0)  # Hq = 3 not a multiple of Hkv = 2
        elif bad == "causal":
            q2, k2, v2 = qkv(1, 2, 2, 5, 4, 2, seed=1)
            oracle.attention(q2, k2, v2, True, 1.0)  # causal with Nq > Nk
        else:
            q2, k2, v2 = qkv(1, 2, 2, 4, 4, 2, seed=1)
            oracle.attention_rows(q2, k2, v2, False, 1.0, [[0, 2, 0]])
