"""fp64 CPU oracle for exact softmax attention (MHA / GQA / MQA).

TEST INFRASTRUCTURE ONLY: the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the product library and
its Python binding never do.  It shares no code with the GPU path.

The arithmetic lives in ``fa_oracle.c`` (plain C, double precision, one thread,
no fast-math, no contraction).  This module only builds that file with gcc,
loads it with ctypes, converts inputs exactly to float64, and optionally spreads
independent query rows over worker processes (each worker still runs the
single-threaded C routine on its rows; the result does not depend on the split).

Definition followed (Sec. 2, scaled dot-product attention; Sec. 4.1, per-head
N x D operands): o = softmax(scale * q k^T) v per query head, key/value head
g = h // (Hq // Hkv), bottom-right causal mask, lse = m + ln(l).
Layouts: q, o [B, Nq, Hq, D]; k, v [B, Nk, Hkv, D]; lse [B, Hq, Nq].
"""
from __future__ import annotations

import ctypes
import multiprocessing as mp
import os
import subprocess
import time
from typing import Iterable, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fa_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_DP = ctypes.POINTER(ctypes.c_double)
_IP = ctypes.POINTER(ctypes.c_int)


def build(force: bool = False) -> str:
    """Compile fa_oracle.c into liboracle.so with gcc (strict IEEE double)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off",
               "-fno-fast-math", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        common = [_DP, _DP, _DP]
        dims = [ctypes.c_int] * 7 + [ctypes.c_double]
        lib.fa_oracle_f64.argtypes = common + [_DP, _DP] + dims
        lib.fa_oracle_f64.restype = ctypes.c_int
        lib.fa_oracle_rows_f64.argtypes = common + dims + [_IP, ctypes.c_int, _DP, _DP]
        lib.fa_oracle_rows_f64.restype = ctypes.c_int
        lib.fa_oracle_weights_f64.argtypes = common + [_DP] + dims
        lib.fa_oracle_weights_f64.restype = ctypes.c_int
        _lib = lib
    return _lib


def to_f64(x) -> np.ndarray:
    """Exact conversion of a torch tensor (fp16 / bf16 / fp32 / fp64) or array
    to a C-contiguous float64 numpy array (every narrower float is exactly
    representable in double)."""
    if hasattr(x, "detach"):
        import torch  # local: plain numpy callers never need torch

        x = x.detach().to("cpu")
        if x.dtype in (torch.float16, torch.bfloat16):
            x = x.to(torch.float32)
        x = x.numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a: np.ndarray, typ=_DP):
    return a.ctypes.data_as(typ)


def _dims(q, k, v):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be 4-D [B, N, H, D]")
    B, Nq, Hq, D = q.shape
    Bk, Nk, Hkv, Dk = k.shape
    if k.shape != v.shape or Bk != B or Dk != D:
        raise ValueError("shape mismatch between q, k and v")
    return B, Hq, Hkv, Nq, Nk, D


def attention(q, k, v, causal: bool, scale: float):
    """Full output (o [B,Nq,Hq,D], lse [B,Hq,Nq]) in float64, one thread."""
    q, k, v = to_f64(q), to_f64(k), to_f64(v)
    B, Hq, Hkv, Nq, Nk, D = _dims(q, k, v)
    o = np.empty((B, Nq, Hq, D), dtype=np.float64)
    lse = np.empty((B, Hq, Nq), dtype=np.float64)
    rc = _load().fa_oracle_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, Hq, Hkv,
                               Nq, Nk, D, int(bool(causal)), float(scale))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return o, lse


def weights(q, k, v, causal: bool, scale: float) -> np.ndarray:
    """Normalised attention weights w [B, Hq, Nq, Nk] (tiny inputs only)."""
    q, k, v = to_f64(q), to_f64(k), to_f64(v)
    B, Hq, Hkv, Nq, Nk, D = _dims(q, k, v)
    w = np.empty((B, Hq, Nq, Nk), dtype=np.float64)
    rc = _load().fa_oracle_weights_f64(_ptr(q), _ptr(k), _ptr(v), _ptr(w), B, Hq, Hkv, Nq,
                                       Nk, D, int(bool(causal)), float(scale))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return w


# ---------------------------------------------------------------- row fan-out
_SHARED = {}


def _rows_call(q, k, v, causal, scale, rows: np.ndarray):
    B, Hq, Hkv, Nq, Nk, D = _dims(q, k, v)
    rows = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 3)
    n = rows.shape[0]
    o = np.empty((n, D), dtype=np.float64)
    lse = np.empty((n,), dtype=np.float64)
    rc = _load().fa_oracle_rows_f64(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, Nq, Nk, D,
                                    int(bool(causal)), float(scale), _ptr(rows, _IP), n,
                                    _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return o, lse


def _worker(chunk: np.ndarray):
    t0 = time.process_time()
    o, lse = _rows_call(_SHARED["q"], _SHARED["k"], _SHARED["v"], _SHARED["causal"],
                        _SHARED["scale"], chunk)
    return o, lse, time.process_time() - t0


def _visible(rows: np.ndarray, Nq: int, Nk: int, causal: bool) -> np.ndarray:
    if not causal:
        return np.full(rows.shape[0], Nk, dtype=np.int64)
    return rows[:, 2].astype(np.int64) + (Nk - Nq) + 1


def attention_rows(q, k, v, causal: bool, scale: float, rows: Sequence[Sequence[int]],
                   workers: int = 1, stats: dict | None = None):
    """Outputs for selected query rows (triples b, h, i).

    Returns (o_rows [n, D], lse_rows [n]).  With workers > 1, rows are split
    into contiguous chunks of about equal visible-key work and computed by
    forked worker processes, each running the single-threaded C routine.
    If ``stats`` is given it receives wall seconds, summed worker CPU seconds
    and the worker count actually used.
    """
    q, k, v = to_f64(q), to_f64(k), to_f64(v)
    B, Hq, Hkv, Nq, Nk, D = _dims(q, k, v)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int32).reshape(-1, 3))
    _load()
    t0 = time.perf_counter()
    if workers <= 1 or rows.shape[0] < 2:
        c0 = time.process_time()
        o, lse = _rows_call(q, k, v, causal, scale, rows)
        cpu = time.process_time() - c0
        used = 1
    else:
        work = _visible(rows, Nq, Nk, causal)
        cum = np.cumsum(work)
        nchunks = min(rows.shape[0], workers * 4)
        edges = np.searchsorted(cum, np.linspace(0, cum[-1], nchunks + 1)[1:-1])
        chunks = [c for c in np.split(rows, edges) if c.shape[0] > 0]
        _SHARED.update(q=q, k=k, v=v, causal=causal, scale=scale)
        try:
            ctx = mp.get_context("fork")
            used = min(workers, len(chunks))
            with ctx.Pool(used) as pool:
                parts = pool.map(_worker, chunks, chunksize=1)
        finally:
            _SHARED.clear()
        o = np.concatenate([p[0] for p in parts], axis=0)
        lse = np.concatenate([p[1] for p in parts], axis=0)
        cpu = float(sum(p[2] for p in parts))
    if stats is not None:
        stats.update(wall_s=time.perf_counter() - t0, cpu_s=cpu, workers=used)
    return o, lse


def all_rows(B: int, Hq: int, Nq: int) -> np.ndarray:
    """Every (b, h, i) triple, in (b, h, i) order."""
    b, h, i = np.meshgrid(np.arange(B), np.arange(Hq), np.arange(Nq), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), i.ravel()], axis=1).astype(np.int32)


def attention_parallel(q, k, v, causal: bool, scale: float, workers: int = 1,
                       stats: dict | None = None):
    """Full output computed through the row fan-out (same values as
    ``attention``; used where one thread would take minutes)."""
    q, k, v = to_f64(q), to_f64(k), to_f64(v)
    B, Hq, Hkv, Nq, Nk, D = _dims(q, k, v)
    rows = all_rows(B, Hq, Nq)
    o_rows, lse_rows = attention_rows(q, k, v, causal, scale, rows, workers, stats)
    o = o_rows.reshape(B, Hq, Nq, D).transpose(0, 2, 1, 3).copy()
    lse = lse_rows.reshape(B, Hq, Nq)
    return o, lse


def default_workers() -> int:
    """Worker processes for the row fan-out: the CPUs this process may run on
    (its affinity mask), limited by OMP_NUM_THREADS where the environment sets
    a CPU share that way."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    share = os.environ.get("OMP_NUM_THREADS", "")
    if share.isdigit() and int(share) > 0:
        n = min(n, int(share))
    return max(1, n)


__all__: Iterable[str] = ["build", "attention", "attention_rows", "attention_parallel",
                          "weights", "to_f64", "all_rows", "default_workers"]
