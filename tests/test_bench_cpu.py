"""Host-side checks of the benchmark's work counts (no GPU): the closed forms
bench.py divides by are compared with brute-force counts on small shapes."""
import itertools

import bench
from paper_2608_18656_amd.inputs import Workload


def _brute_visible(Nq, L, causal=True):
    # query i (the sequence's position L - Nq + i) sees key j iff j <= L - Nq + i
    return sum(1 for i, j in itertools.product(range(Nq), range(L)) if not causal or j <= L - Nq + i)


def test_chunked_visible_pairs_brute_force():
    for Nq, lens in [(1, [1]), (3, [3, 7]), (5, [5, 9, 64]), (16, [16, 17, 100])]:
        assert bench.chunked_visible_pairs(Nq, lens) == sum(_brute_visible(Nq, L) for L in lens)


def test_workload_visible_pairs_brute_force():
    for Nq, Nk, causal in [(1, 9, True), (7, 7, True), (5, 12, True), (6, 4, False), (13, 40, True)]:
        w = Workload("t", 1, 2, 1, Nq, Nk, 64, causal, "f16", 0)
        assert w.visible_pairs() == _brute_visible(Nq, Nk, causal)


def test_unfused_min_bytes_counts_each_array_once():
    B, Hq, Hkv, Nq, Nk, D, es = 2, 4, 2, 5, 9, 64, 2
    w = Workload("t", B, Hq, Hkv, Nq, Nk, D, True, "f16", 0)
    vis = B * Hq * w.visible_pairs()
    s_bytes, p_bytes = 4 * vis, 2 * vis                  # S and P, each written once and read once
    q_o = 2 * B * Nq * Hq * D * es                        # Q read, O written
    k_v = 2 * B * Nk * Hkv * D * es                       # K and V read
    assert bench.unfused_min_bytes(B, Hq, Hkv, Nq, Nk, D, w.visible_pairs(), es) == \
        2 * s_bytes + 2 * p_bytes + q_o + k_v
    # the headline workload: 12 x 67,141,632 visible scores + 20,971,520 bytes of Q, K, V, O
    assert bench.unfused_min_bytes(1, 32, 8, 2048, 2048, 64, 2048 * 2049 // 2, 2) == 826_671_104


def test_staged_kv_bytes_brute_force():
    """The packing ablation's staged K/V bytes: every workgroup (slots / heads
    row blocks of 32 rows, `heads` query heads) stages each key tile its last
    row reaches, K and V, counted here by enumerating rows and tiles."""
    import math

    for (B, Hq, Hkv, Nq, Nk, D, causal) in [(1, 8, 2, 100, 130, 64, True), (2, 16, 1, 70, 70, 128, True),
                                            (1, 4, 4, 33, 90, 64, False)]:
        w = Workload("t", B, Hq, Hkv, Nq, Nk, D, causal, "f16", 0)
        bc = 64 if D == 64 else 32
        G = Hq // Hkv
        for slots, heads in [(1, 1), (2, 1), (4, 1), (4, 2), (8, 1)]:
            if G % heads:
                continue
            rows = 32 * (slots // heads)
            total = 0
            for b in range(B):
                for g in range(Hkv):
                    for hg in range(G // heads):
                        for r0 in range(0, Nq, rows):
                            seen = max((min(Nk, i + Nk - Nq + 1) if causal else Nk)
                                       for i in range(r0, min(r0 + rows, Nq)))
                            total += math.ceil(seen / bc) * bc * D * 2 * 2
            assert bench.staged_kv_bytes(w, slots, heads) == total, (B, Hq, Hkv, Nq, Nk, D, slots, heads)


def test_more_than_one_gpu_is_refused_with_a_message():
    """The benchmark measures one GPU: --gpus above 1 (or a WORLD_SIZE above 1)
    exits with status 2 and says so, before touching a GPU."""
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for args, env in [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "4"})]:
        r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), *args], capture_output=True, text=True,
                           env={**os.environ, **env}, timeout=120)
        assert r.returncode == 2, (args, env, r.returncode)
        assert "one GPU" in r.stderr, r.stderr
