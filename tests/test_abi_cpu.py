"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/fa.h declares, and its argument validation returns
the documented status codes before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2608_18656_amd import _lib, validate, workspace_bytes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fa.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fa_[a-z0-9_]+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = _lib.load()
    names = declared_functions()
    assert len(names) >= 10
    assert set(names) == set(_lib.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.fa_version() == (0 << 16) | (1 << 8)


def test_status_strings():
    lib = _lib.load()
    for code, name in _lib.STATUS_NAMES.items():
        assert lib.fa_status_string(code).decode().startswith(name)


A = 1 << 20   # fake, 16-byte aligned, non-overlapping "device" addresses
GOOD = dict(q=A, k=9 * A, v=17 * A, o=25 * A, lse=33 * A)
DIMS = dict(B=1, Hq=4, Hkv=2, Nq=8, Nk=8, D=64, causal=1, scale=0.125)


def call(dt="f16", out=None, **over):
    p = dict(GOOD)
    p.update(DIMS)
    p.update(over)
    return validate(p["q"], p["k"], p["v"], p["o"], p["lse"], p["B"], p["Hq"], p["Hkv"], p["Nq"],
                    p["Nk"], p["D"], p["causal"], p["scale"], dt, out)


@pytest.mark.parametrize("over,code", [
    ({}, 0),
    ({"q": None}, 1), ({"k": None}, 1), ({"v": None}, 1), ({"o": None}, 1),
    ({"B": 0}, 2), ({"Hq": 0}, 2), ({"Nq": 0}, 2), ({"Nk": -1}, 2), ({"D": 0}, 2),
    ({"Hq": 6, "Hkv": 4}, 3),
    ({"D": 60}, 4), ({"D": 264}, 4),
    ({"Nq": 9, "Nk": 8}, 5),
    ({"scale": float("nan")}, 6), ({"scale": float("inf")}, 6),
    ({"q": A + 8}, 7), ({"o": 25 * A + 2}, 7), ({"lse": 33 * A + 2}, 7),
    ({"o": A + 64}, 8), ({"lse": 9 * A + 16}, 8), ({"lse": 25 * A}, 8),
])
def test_validation_status_codes(over, code):
    assert call(**over) == code


def test_validation_accepts_edge_shapes_and_scales():
    assert call(lse=None) == 0                      # lse optional
    assert call(causal=0, Nq=9, Nk=8) == 0          # non-causal Nq > Nk is fine
    assert call(scale=0.0) == 0 and call(scale=-2.0) == 0
    assert call(D=8) == 0 and call(D=256) == 0
    assert call(Hkv=1) == 0 and call(Hkv=4) == 0   # MQA and MHA


def test_validation_dtype_rules():
    assert call("bf16") == 0 and call("f32") == 0
    assert call("f16", "f32") == 0 and call("bf16", "f32") == 0   # fp32 verify output
    assert call("f16", "bf16") == 9 and call("f32", "f16") == 9
    assert call(7) == 9


def test_validation_rejects_size_overflow():
    assert call(B=1 << 30, Nq=1 << 30, Nk=1 << 30, causal=0) == 2


def test_workspace_bytes():
    # decode: B * Hq * S * (D + 2) floats; other shapes need none
    assert workspace_bytes(16, 32, 8, 1, 8192, 128, "bf16", 8) == 16 * 32 * 8 * 130 * 4
    assert workspace_bytes(16, 32, 8, 1, 8192, 128, "bf16", 0) > 0
    assert workspace_bytes(1, 32, 8, 2048, 2048, 64, "bf16") == 0
    assert workspace_bytes(1, 2, 2, 1, 128, 64, "f32") == 0
    assert workspace_bytes(1, 2, 2, 1, 128, 64, "f16", 300) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "absent.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(FileNotFoundError):
        _lib.load()


@pytest.mark.parametrize("packing,Hq,Hkv", [(3, 4, 2), (-1, 4, 2), (8, 8, 1), (4, 4, 2), (2, 6, 2)])
def test_packing_rejected_before_any_launch(packing, Hq, Hkv):
    """fa_fwd_packed checks heads_per_workgroup on the host (no HIP call):
    it must be 0, 1, 2 or 4 and divide Hq / Hkv."""
    lib = _lib.load()
    st = lib.fa_fwd_packed(GOOD["q"], GOOD["k"], GOOD["v"], GOOD["o"], GOOD["lse"], 1, Hq, Hkv,
                           8, 8, 64, 1, 0.125, None, 0, 0, packing)
    assert st == 13


def test_kvcache_sequence_lengths_checked_before_any_launch():
    """fa_fwd_kvcache: NULL, misaligned or output-overlapping seqlens_k are
    refused on the host (no HIP call)."""
    lib = _lib.load()
    def st(seqlens, o=GOOD["o"]):
        return lib.fa_fwd_kvcache(GOOD["q"], GOOD["k"], GOOD["v"], o, GOOD["lse"], seqlens, 2, 4, 2,
                                  8, 8, 64, 1, 0.125, None, 0, 0)
    assert st(None) == 1
    assert st(41 * A + 2) == 7
    assert st(25 * A + 64) == 8          # inside o


def test_q8_gemv_argument_errors_before_any_launch():
    """fa_q8_0_gemv's checks return before any HIP call (fake addresses)."""
    lib = _lib.load()
    W, X, Y = 1 << 20, 64 << 20, 96 << 20
    F16, BF16, F32 = _lib.FA_F16, _lib.FA_BF16, _lib.FA_F32

    def call(w=W, x=X, y=Y, M=8, K=64, xt=BF16, yt=BF16):
        return lib.fa_q8_0_gemv(w, x, y, M, K, xt, yt, None)

    assert call(w=None) == 1 and call(x=None) == 1 and call(y=None) == 1
    for M, K in [(0, 64), (-1, 64), (8, 0), (8, 16), (8, 48), (8, 33), (1, (1 << 30) + 32)]:
        assert call(M=M, K=K) == 2, (M, K)
    assert call(xt=3) == 9 and call(xt=F16, yt=BF16) == 9 and call(xt=F32, yt=F16) == 9
    assert call(yt=7) == 9
    assert call(w=W + 2) == 7                      # weights need 4-byte alignment
    assert call(x=X + 2) == 7 and call(x=X + 8) == 7   # x needs 16-byte alignment
    assert call(y=Y + 1) == 7 and call(xt=F32, yt=F32, y=Y + 2) == 7
    assert call(y=W + 100) == 8                    # y inside w (8 * 2 * 34 bytes)
    assert call(y=X + 64) == 8                     # y inside x
    assert call(y=W + 8 * 2 * 34) != 8             # y right after w: no overlap reported


def test_paged_argument_errors_before_any_launch():
    """fa_fwd_kvcache_paged's own checks (fake addresses, no HIP call)."""
    lib = _lib.load()
    Q, K, V, O, L, S, T = (k << 24 for k in (1, 2, 3, 4, 5, 6, 7))
    F16, BF16, F32 = _lib.FA_F16, _lib.FA_BF16, _lib.FA_F32

    def call(q=Q, k=K, v=V, o=O, lse=L, sl=S, bt=T, B=2, Hq=8, Hkv=2, Nq=1, D=64, ps=64, mp=4, npg=8,
             causal=0, scale=0.125, it=F16, ot=F16):
        return lib.fa_fwd_kvcache_paged(q, k, v, o, lse, sl, bt, B, Hq, Hkv, Nq, D, ps, mp, npg, causal,
                                        scale, None, it, ot)

    assert call(sl=None) == 1 and call(bt=None) == 1 and call(q=None) == 1
    for ps in (0, 32, 96, -64):
        assert call(ps=ps) == 2, ps
    assert call(mp=0) == 2 and call(npg=0) == 2 and call(ps=1 << 30, mp=4) == 2
    assert call(sl=S + 2) == 7 and call(bt=T + 1) == 7
    assert call(it=F32, ot=F32) == 9
    assert call(D=96) == 4 and call(D=256) == 4
    assert call(o=T) == 8                          # o overlaps the block table
    assert call(lse=S) == 8                        # lse overlaps the lengths
    assert call(o=K + 64) == 8                     # o inside the K pool (8 pages of 64 x 2 x 64 x 2 B)
    assert call(Hq=6, Hkv=4) == 3


def test_header_is_plain_c(tmp_path):
    """include/fa.h compiles as C11 (no C++ in the boundary) and declares
    every entry point with the signature the library exports."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    names = declared_functions()
    src = tmp_path / "uses_fa.c"
    body = "\n".join(f"    (void)&{n};" for n in names)
    src.write_text(
        '#include "fa.h"\n'
        "int main(void) {\n"
        f"{body}\n"
        "    fa_status_t s = FA_OK; fa_dtype_t t = FA_BF16; (void)s; (void)t;\n"
        "    return FA_MAX_SPLITS == 256 && FA_ERR_PACKING == 13 ? 0 : 1;\n"
        "}\n")
    out = tmp_path / "uses_fa.o"
    r = subprocess.run([cc, "-std=c11", "-Wall", "-Werror", "-pedantic", "-I",
                        os.path.join(ROOT, "include"), "-c", str(src), "-o", str(out)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_unfused_argument_errors_before_any_launch():
    """fa_fwd_unfused's own checks and fa_unfused_workspace_bytes (fake
    addresses, no HIP call)."""
    lib = _lib.load()
    Q, K, V, O, L, W = (k << 32 for k in (1, 2, 3, 4, 5, 6))
    F16, BF16, F32 = _lib.FA_F16, _lib.FA_BF16, _lib.FA_F32
    need = lib.fa_unfused_workspace_bytes(2, 8, 100, 130)
    assert need == 6 * 2 * 8 * 100 * 192                       # Nk rounded up to 64
    assert lib.fa_unfused_workspace_bytes(1, 1, 1, 1) == 6 * 64
    assert lib.fa_unfused_workspace_bytes(1, 1, 1, 64) == 6 * 64
    assert lib.fa_unfused_workspace_bytes(0, 8, 100, 130) == 0
    assert lib.fa_unfused_workspace_bytes(1, 8, -1, 130) == 0
    assert lib.fa_unfused_workspace_bytes(1 << 30, 1 << 30, 1 << 30, 1 << 30) == 0   # overflow

    def call(q=Q, k=K, v=V, o=O, lse=L, B=2, Hq=8, Hkv=2, Nq=100, Nk=130, D=64, causal=1,
             scale=0.125, it=F16, ot=F16, ws=W, wsb=None):
        return lib.fa_fwd_unfused(q, k, v, o, lse, B, Hq, Hkv, Nq, Nk, D, causal, scale, None, it, ot,
                                  ws, need if wsb is None else wsb)

    assert call(q=None) == 1 and call(ws=None) == 1
    assert call(Hq=6, Hkv=4) == 3 and call(Nq=200) == 5 and call(scale=float("nan")) == 6
    assert call(it=F32, ot=F32) == 9 and call(ot=BF16) == 9
    assert call(D=96) == 4 and call(D=32) == 4
    assert call(ws=W + 128) == 7                          # workspace not 256-byte aligned
    assert call(wsb=need - 1) == 10                       # workspace too small
    assert call(ws=Q) == 8                                 # workspace over q
    assert call(ws=O - 256) == 8                           # workspace runs into o
    assert call(o=Q + 64) == 8                             # the checks of fa_fwd come first
    assert call(B=1, Hq=2, Hkv=1, Nq=1, Nk=(1 << 23) + 1) == 2   # 32-bit offsets in a block of scores
    far = [k << 44 for k in range(1, 7)]                 # fake addresses that cannot overlap
    assert call(*far[:5], B=1 << 10, Hq=1 << 11, Hkv=1 << 11, Nq=1 << 10, Nk=1 << 10, causal=0,
                ws=far[5]) == 2                           # 2^31 rows of scores


def test_per_call_workspace_argument_errors_before_any_launch():
    """fa_fwd_ws / fa_fwd_kvcache_ws / fa_fwd_kvcache_paged_ws: a decode call's
    own workspace is checked (NULL, alignment, size, overlap) before any HIP
    call, after the checks of the call it extends (fake addresses)."""
    lib = _lib.load()
    Q, K, V, O, L, S, T, W = (k << 32 for k in range(1, 9))
    F16, BF16 = _lib.FA_F16, _lib.FA_BF16
    B, Hq, Hkv, Nk, D = 16, 32, 8, 8192, 128
    need = lib.fa_workspace_bytes(B, Hq, Hkv, 1, Nk, D, BF16, 0)
    assert need > 0 and need == lib.fa_workspace_bytes(B, Hq, Hkv, 1, Nk, D, BF16, 2)   # 2 splits
    assert lib.fa_workspace_bytes(B, Hq, Hkv, 1, Nk, D, BF16, 5) == B * Hq * 5 * (D + 2) * 4
    assert lib.fa_workspace_bytes(1, 4, 2, 64, 64, 64, F16, 0) == 0   # prefill takes none

    def fwd(ws=W, wsb=None, q=Q, o=O, Nq=1, splits=0, causal=0):
        return lib.fa_fwd_ws(q, K, V, o, L, B, Hq, Hkv, Nq, Nk, D, causal, 0.088, None, BF16, BF16,
                             splits, ws, need if wsb is None else wsb)

    assert fwd(ws=None) == 1                       # decode needs a workspace
    assert fwd(ws=W + 8) == 7                      # not 16-byte aligned
    assert fwd(wsb=need - 1) == 10                 # too small
    assert fwd(ws=K + 4096) == 8                   # inside k
    assert fwd(ws=O - 64) == 8                     # runs into o
    assert fwd(q=None) == 1 and fwd(splits=257) == 12   # the checks of fa_fwd_splitkv come first
    assert fwd(splits=5, wsb=need) == 10           # 5 splits need more than the default 2

    def kv(ws=W, wsb=None, sl=S):
        return lib.fa_fwd_kvcache_ws(Q, K, V, O, L, sl, B, Hq, Hkv, 1, Nk, D, 0, 0.088, None, BF16, BF16,
                                     ws, need if wsb is None else wsb)

    assert kv(ws=None) == 1 and kv(ws=W + 4) == 7 and kv(wsb=16) == 10 and kv(ws=V) == 8
    assert kv(sl=None) == 1                        # the lengths are checked first

    def paged(ws=W, wsb=None, bt=T):
        ps, mp, npg = 256, Nk // 256, B * (Nk // 256)
        return lib.fa_fwd_kvcache_paged_ws(Q, K, V, O, L, S, bt, B, Hq, Hkv, 1, D, ps, mp, npg, 0, 0.088,
                                           None, BF16, BF16, ws, need if wsb is None else wsb)

    assert paged(ws=None) == 1 and paged(ws=W + 2) == 7 and paged(wsb=need - 16) == 10
    assert paged(ws=O) == 8 and paged(bt=None) == 1


def test_noalloc_size_limit_before_any_launch():
    """fa_fwd_splitkv_noalloc refuses partial results beyond its 32 MiB
    scratch with FA_ERR_WORKSPACE, after the checks of fa_fwd_splitkv, before
    any HIP call (fake addresses)."""
    lib = _lib.load()
    far = [k << 40 for k in range(1, 6)]
    BF16 = _lib.FA_BF16
    # 256 * 64 * 16 * (128 + 2) * 4 B = 136 MB of partials
    assert lib.fa_fwd_splitkv_noalloc(*far, 256, 64, 8, 1, 65536, 128, 0, 0.088, None, BF16, BF16, 16) == 10
    assert lib.fa_workspace_bytes(256, 64, 8, 1, 65536, 128, BF16, 16) > (32 << 20)
    assert lib.fa_fwd_splitkv_noalloc(*far, 256, 64, 8, 1, 65536, 128, 0, 0.088, None, BF16, BF16, 300) == 12
    assert lib.fa_fwd_splitkv_noalloc(None, *far[1:], 2, 8, 2, 1, 100, 64, 0, 0.1, None, BF16, BF16, 0) == 1


def test_workgroup_layout_argument_errors():
    """fa_fwd_slots: slots 0, 1, 2, 4, 8; heads 0, 1, 2, 4, 8 dividing Hq / Hkv
    and the slots; anything else is FA_ERR_PACKING before any HIP call."""
    lib = _lib.load()
    Q, K, V, O, L = (k << 32 for k in range(1, 6))
    F16 = _lib.FA_F16

    def call(slots, heads, Hq=16, Hkv=2):
        return lib.fa_fwd_slots(Q, K, V, O, L, 1, Hq, Hkv, 64, 64, 64, 1, 0.125, None, F16, F16, slots, heads)

    for slots, heads in [(3, 0), (16, 0), (-1, 0), (4, 8), (2, 4), (1, 2), (8, 3), (8, 16)]:
        assert call(slots, heads) == 13, (slots, heads)
    assert call(8, 8, Hq=12, Hkv=3) == 13          # 8 heads do not divide the group of 4
    assert call(4, 2, Hq=6, Hkv=2) == 13           # nor 2 a group of 3
    assert lib.fa_fwd_packed(Q, K, V, O, L, 1, 16, 2, 64, 64, 64, 1, 0.125, None, F16, F16, 8) == 13
