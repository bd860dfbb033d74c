"""The C ABI used from plain C, without PyTorch: tests/c_client (built by
__graft_entry__.build()) reads inputs from a file, calls fa_fwd,
fa_q8_0_gemv and (fp16 / bf16) fa_fwd_unfused on device buffers and a
workspace it allocates itself, and writes the results; they are compared
with the fp64 oracles (attention in verify mode within 2e-3, the Q8_0
product within its derived fp32 bound)."""
import os
import struct
import subprocess
import sys

import numpy as np
import pytest

import oracle
from oracle import q8 as oracle_q8
from paper_2608_18656_amd.inputs import DTYPES, make_q8_0, make_qkv

from helpers import check_against

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c_client")
CODES = {"f16": 0, "bf16": 1, "f32": 2}


@pytest.mark.parametrize("case", [
    (1, 8, 2, 200, 200, 64, 1, "bf16"),
    (2, 16, 1, 1, 3000, 128, 0, "f16"),
    (1, 2, 2, 50, 90, 64, 0, "f32"),
], ids=["prefill_bf16", "decode_f16", "f32"])
def test_c_client_matches_oracle(case, tmp_path):
    import torch

    if not os.path.exists(EXE):
        pytest.fail("tests/c_client is not built (run __graft_entry__.build())")
    B, Hq, Hkv, Nq, Nk, D, causal, dt = case
    scale = D ** -0.5
    q, k, v = make_qkv(B, Hq, Hkv, Nq, Nk, D, dt, seed=606 + Nq)
    M, K = 300, 2048
    w, x = make_q8_0(M, K, seed=607, x_dtype="f32")
    inp = tmp_path / "in.bin"
    with open(inp, "wb") as f:
        f.write(struct.pack("<8i", B, Hq, Hkv, Nq, Nk, D, causal, CODES[dt]))
        f.write(struct.pack("<f", scale))
        for t in (q, k, v):
            f.write(t.contiguous().view(torch.uint8).numpy().tobytes())
        f.write(struct.pack("<2i", M, K))
        f.write(w.numpy().tobytes())
        f.write(x.numpy().astype(np.float32).tobytes())
    out = tmp_path / "out.bin"
    print(f"c_client case {case}", flush=True)
    r = subprocess.run([EXE, str(inp), str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    data = np.fromfile(out, dtype=np.float32)
    no, nl = B * Nq * Hq * D, B * Hq * Nq
    o = torch.from_numpy(data[:no].reshape(B, Nq, Hq, D).copy())
    lse = torch.from_numpy(data[no:no + nl].reshape(B, Hq, Nq).copy())
    y = data[no + nl:no + nl + M].astype(np.float64)
    o_ref, l_ref = oracle.attention(q, k, v, bool(causal), scale)
    check_against(o, lse, o_ref, l_ref, DTYPES[dt], True, f"c_client {case}")
    ref = oracle_q8.gemv(w.numpy(), x.numpy())
    nb = K // 32
    wn = w.numpy()
    d = np.abs(np.ascontiguousarray(wn[:, :, 0:2]).view(np.float16).reshape(M, nb).astype(np.float64))
    qa = np.abs(np.ascontiguousarray(wn[:, :, 2:]).view(np.int8).astype(np.float64))
    S = (d * (qa * np.abs(x.numpy().astype(np.float64)).reshape(1, nb, 32)).sum(axis=2)).sum(axis=1)
    assert np.all(np.abs(y - ref) <= (2 * nb + 64) * 2.0 ** -24 * S)
    rest = data[no + nl + M:]
    if dt == "f32":
        assert rest.size == 0
    else:
        assert rest.size == no + nl
        o2 = torch.from_numpy(rest[:no].reshape(B, Nq, Hq, D).copy())
        l2 = torch.from_numpy(rest[no:].reshape(B, Hq, Nq).copy())
        check_against(o2, l2, o_ref, l_ref, DTYPES[dt], True, f"c_client unfused {case}")
