"""HIP graph capture of the library's calls: prefill, split-KV decode (with
its merge kernel and workspace), decode against a paged cache, the unfused
path (three kernels through a caller workspace) and the Q8_0
matrix-vector product are captured once after a warm-up call and replayed
several times, with eager work and synchronisations between the replays;
every replay must equal the eager result bit for bit.  (The library issues no
memset and allocates nothing once the decode workspace exists.)
"""
import pytest
import torch

import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import make_q8_0, make_qkv

pytestmark = pytest.mark.gpu


def _capture(fn):
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_replays_equal_eager():
    # prefill (causal GQA, bf16) and decode (GQA, split-KV + merge)
    qp, kp, vp = (t.cuda() for t in make_qkv(1, 16, 4, 300, 300, 64, "bf16", seed=1))
    qd, kd, vd = (t.cuda() for t in make_qkv(4, 32, 8, 1, 3000, 128, "bf16", seed=2))
    # paged decode: pages of 64 in reverse order
    B, Nk, ps = 4, 3000 // 64 * 64, 64
    kpg = kd[:, :Nk].reshape(B * (Nk // ps), ps, 8, 128).flip(0).contiguous()
    vpg = vd[:, :Nk].reshape(B * (Nk // ps), ps, 8, 128).flip(0).contiguous()
    table = (B * (Nk // ps) - 1 - torch.arange(B * (Nk // ps), device="cuda")).reshape(B, -1).to(torch.int32)
    sl = torch.tensor([Nk, 1000, 64, 1], dtype=torch.int32, device="cuda")
    # Q8_0 product
    w8, x8 = (t.cuda() for t in make_q8_0(3000, 2048, seed=3, x_dtype="bf16"))
    # unfused path on the prefill inputs
    wsu = torch.empty(fa.unfused_workspace_bytes(1, 16, 300, 300), dtype=torch.uint8, device="cuda")

    outs = {
        "prefill": (torch.empty_like(qp), torch.empty((1, 16, 300), dtype=torch.float32, device="cuda")),
        "decode": (torch.empty_like(qd), torch.empty((4, 32, 1), dtype=torch.float32, device="cuda")),
        "paged": (torch.empty_like(qd), torch.empty((4, 32, 1), dtype=torch.float32, device="cuda")),
        "q8": (torch.empty(3000, dtype=torch.bfloat16, device="cuda"),),
        "unfused": (torch.empty_like(qp), torch.empty((1, 16, 300), dtype=torch.float32, device="cuda")),
    }

    def calls():
        fa.fwd(qp, kp, vp, causal=True, out=outs["prefill"][0], lse=outs["prefill"][1])
        fa.fwd(qd, kd, vd, out=outs["decode"][0], lse=outs["decode"][1])
        fa.fwd_kvcache_paged(qd, kpg, vpg, table, sl, out=outs["paged"][0], lse=outs["paged"][1])
        fa.q8_0_gemv(w8, x8, out=outs["q8"][0])
        fa.fwd_unfused(qp, kp, vp, causal=True, out=outs["unfused"][0], lse=outs["unfused"][1],
                       workspace=wsu)

    calls()
    torch.cuda.synchronize()
    eager = {k: [t.clone() for t in v] for k, v in outs.items()}
    g = _capture(calls)
    for rep in range(4):
        for v in outs.values():
            for t in v:
                t.fill_(0)
        # unrelated eager work between replays
        fa.fwd(qd, kd, vd)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            for a, b in zip(v, eager[k]):
                assert torch.equal(a, b), f"replay {rep}: {k} differs from the eager result"
