"""Decode workspaces on the GPU: calls running concurrently on two streams,
each with its own workspace (fa_fwd_ws, fa_fwd_kvcache_ws,
fa_fwd_kvcache_paged_ws) or with the library-owned buffer of its stream, give
bit for bit the results of the same calls run one after another, and agree
with the oracle; a graph captured before the library-owned buffer of its
stream is outgrown still replays correctly afterwards (the outgrown buffer is
kept); a decode call that would need a new buffer inside stream capture is
refused with FA_ERR_WORKSPACE."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_18656_amd as fa
from paper_2608_18656_amd.inputs import DTYPES, make_qkv

from helpers import check_against, default_scale

pytestmark = pytest.mark.gpu

# B, Hq, Hkv, Nk, D, dtype, forced splits
SHAPES = [(4, 32, 8, 3000, 128, "bf16", 0), (8, 16, 1, 2500, 64, "f16", 7)]


def _inputs(i):
    B, Hq, Hkv, Nk, D, dt, S = SHAPES[i]
    q, k, v = make_qkv(B, Hq, Hkv, 1, Nk, D, dt, seed=300 + i)
    return (q, k, v), tuple(t.cuda() for t in (q, k, v)), default_scale(D), S


def _ws_bytes(i):
    B, Hq, Hkv, Nk, D, dt, S = SHAPES[i]
    return fa.workspace_bytes(B, Hq, Hkv, 1, Nk, D, dt, S)


@pytest.mark.parametrize("own", [True, False], ids=["per_call", "library_per_stream"])
def test_two_streams_concurrently_equal_serial(own):
    cpu, dev, scales, splits = zip(*(_inputs(i) for i in range(2)))
    # serial reference, one call after the other on the current stream
    serial = [fa.fwd(*dev[i], scale=scales[i], num_splits=splits[i] or None, out_dtype=torch.float32)
              for i in range(2)]
    torch.cuda.synchronize()
    wss = [torch.empty(_ws_bytes(i), dtype=torch.uint8, device="cuda") for i in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [(torch.empty_like(serial[i][0]), torch.empty_like(serial[i][1])) for i in range(2)]
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    for _ in range(20):   # interleaved in host order so that the streams overlap on the GPU
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                fa.fwd(*dev[i], scale=scales[i], num_splits=splits[i] or None, out_dtype=torch.float32,
                       out=outs[i][0], lse=outs[i][1], workspace=wss[i] if own else None)
    torch.cuda.synchronize()
    for i in range(2):
        assert torch.equal(outs[i][0], serial[i][0]) and torch.equal(outs[i][1], serial[i][1]), i
        o_ref, l_ref = oracle.attention(*cpu[i], False, scales[i])
        check_against(outs[i][0], outs[i][1], o_ref, l_ref, DTYPES[SHAPES[i][5]], True, f"stream {i}")


def test_kvcache_calls_with_their_own_workspace():
    """fa_fwd_kvcache_ws and fa_fwd_kvcache_paged_ws on two streams at once,
    each with its own workspace, against the library-owned-workspace calls."""
    B, Hq, Hkv, Nk, D = 4, 16, 4, 2048, 128
    q, k, v = (t.cuda() for t in make_qkv(B, Hq, Hkv, 1, Nk, D, "bf16", seed=310))
    sl = torch.tensor([2048, 1000, 64, 1], dtype=torch.int32, device="cuda")
    ps = 256
    npg = B * (Nk // ps)
    perm = torch.randperm(npg, generator=torch.Generator().manual_seed(311)).cuda()
    kp = torch.empty((npg, ps, Hkv, D), dtype=k.dtype, device="cuda")
    vp = torch.empty_like(kp)
    kp[perm] = k.reshape(npg, ps, Hkv, D)
    vp[perm] = v.reshape(npg, ps, Hkv, D)
    table = perm.reshape(B, -1).to(torch.int32)
    ref_c = fa.fwd_kvcache(q, k, v, sl)
    ref_p = fa.fwd_kvcache_paged(q, kp, vp, table, sl)
    torch.cuda.synchronize()
    need = fa.workspace_bytes(B, Hq, Hkv, 1, Nk, D, "bf16", 0)
    ws = [torch.empty(need, dtype=torch.uint8, device="cuda") for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    oc = (torch.empty_like(ref_c[0]), torch.empty_like(ref_c[1]))
    op = (torch.empty_like(ref_p[0]), torch.empty_like(ref_p[1]))
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    for _ in range(10):
        with torch.cuda.stream(streams[0]):
            fa.fwd_kvcache(q, k, v, sl, out=oc[0], lse=oc[1], workspace=ws[0])
        with torch.cuda.stream(streams[1]):
            fa.fwd_kvcache_paged(q, kp, vp, table, sl, out=op[0], lse=op[1], workspace=ws[1])
    torch.cuda.synchronize()
    assert torch.equal(oc[0], ref_c[0]) and torch.equal(oc[1], ref_c[1])
    assert torch.equal(op[0], ref_p[0]) and torch.equal(op[1], ref_p[1])
    assert torch.equal(op[0], oc[0])   # the paged cache holds the same keys
    with pytest.raises(fa.FaError) as e:
        fa.fwd_kvcache(q, k, v, sl, workspace=ws[0][: need - 16])
    assert e.value.status == 10


def test_graph_captured_before_growth_replays_after():
    """A decode captured with the library-owned buffer of its stream keeps
    working after a larger eager call on that stream grew the buffer (the
    outgrown buffer is kept until release)."""
    (cpu, dev, scale, _) = _inputs(0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    out = torch.empty_like(dev[0])
    lse = torch.empty((dev[0].shape[0], dev[0].shape[2], 1), dtype=torch.float32, device="cuda")
    with torch.cuda.stream(s):
        fa.fwd(*dev, scale=scale, out=out, lse=lse)   # warm-up: the stream's buffer
    torch.cuda.synchronize()
    eager = (out.clone(), lse.clone())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fa.fwd(*dev, scale=scale, out=out, lse=lse)
    torch.cuda.synchronize()
    # a much larger decode on the same stream grows its buffer
    qb, kb, vb = (t.cuda() for t in make_qkv(16, 64, 8, 1, 2048, 128, "bf16", seed=320))
    with torch.cuda.stream(s):
        fa.fwd(qb, kb, vb, num_splits=64)
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(0)
        lse.fill_(0)
        with torch.cuda.stream(s):
            fa.fwd(qb, kb, vb, num_splits=64)   # eager work on the grown buffer between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager[0]) and torch.equal(lse, eager[1]), rep


def test_no_allocation_inside_capture():
    """A first decode call on a fresh stream inside stream capture would need a
    new buffer: it is refused with FA_ERR_WORKSPACE, the capture is left
    valid, and the same call with its own workspace is captured and replays
    correctly."""
    (cpu, dev, scale, _) = _inputs(1)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    need = _ws_bytes(1)
    B, Hq, Hkv, Nk, D, dt, S = SHAPES[1]
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    out = torch.empty_like(dev[0])
    ref = fa.fwd(*dev, scale=scale, num_splits=S)[0]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    refused = None
    with torch.cuda.graph(g, stream=s):
        try:
            fa.fwd(*dev, scale=scale, num_splits=S, out=out)
        except fa.FaError as e:
            refused = e.status
        fa.fwd(*dev, scale=scale, num_splits=S, out=out, workspace=ws)
    torch.cuda.synchronize()
    assert refused == 10
    for _ in range(3):
        out.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
    np.testing.assert_array_equal(out.float().cpu().numpy(), ref.float().cpu().numpy())
