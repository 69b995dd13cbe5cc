"""CPU oracle for budgeted weight-space merging -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never touches it and shares no code with it.

This module is a thin ctypes wrapper over ``liboracle.so`` (plain C, see
``oracle.c``) that accepts numpy arrays.  fp32 checkpoints are float32
arrays; bf16 checkpoints are uint16 arrays of raw bfloat16 bit patterns.
"""

from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

from .build import LIB, build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        i64p = C.POINTER(C.c_int64)
        L.orc_num_blocks.restype = C.c_int64
        L.orc_num_blocks.argtypes = [C.c_int32, i64p, C.c_int64]
        L.orc_blocks.argtypes = [C.c_int32, i64p, C.c_int64, i64p, i64p, C.POINTER(C.c_int32), i64p]
        L.orc_index.argtypes = [C.c_int64, i64p, i64p, C.c_int32, C.c_void_p, C.POINTER(C.c_void_p),
                                C.c_int32, C.c_void_p]
        L.orc_plan.argtypes = [C.c_int64, i64p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                               C.c_uint64, C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_plan_tensors.argtypes = [C.c_int32, i64p, C.c_int64, C.c_int32, C.c_int32, C.c_void_p,
                                       C.c_uint64, C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_merge_avg.argtypes = [C.c_int64, i64p, i64p, C.c_int32, C.c_void_p, C.POINTER(C.c_void_p),
                                    C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_merge_avg_renorm.argtypes = L.orc_merge_avg.argtypes
        L.orc_merge_ties.argtypes = [C.c_int64, i64p, i64p, C.c_int32, C.c_void_p, C.POINTER(C.c_void_p),
                                     C.c_int32, C.c_void_p, C.c_double, C.c_float, C.c_void_p]
        L.orc_merge_dare.argtypes = [C.c_int64, i64p, i64p, C.POINTER(C.c_int32), i64p, C.c_int32,
                                     C.c_void_p, C.POINTER(C.c_void_p), C.c_int32, C.c_void_p,
                                     C.c_double, C.c_uint32, C.c_int32, C.c_void_p, C.c_float, C.c_void_p]
        L.orc_philox4x32_10.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_mix64.restype = C.c_uint64
        L.orc_mix64.argtypes = [C.c_uint64]
        L.orc_round_bf16.argtypes = [C.c_void_p, C.c_void_p, C.c_int64]
        L.orc_ties_thresholds.argtypes = [C.c_int64, i64p, i64p, C.c_int32, C.c_void_p, C.POINTER(C.c_void_p),
                                          C.c_int32, C.c_double, C.c_void_p]
        L.orc_ties_tensor_thresholds.argtypes = [C.c_int64, i64p, i64p, C.POINTER(C.c_int32), C.c_int32, C.c_int32,
                                                 C.c_void_p, C.POINTER(C.c_void_p), C.c_int32, C.c_void_p,
                                                 C.c_double, C.c_void_p]
        L.orc_merge_ties_tau.argtypes = [C.c_int64, i64p, i64p, C.c_int32, C.c_void_p, C.POINTER(C.c_void_p),
                                         C.c_int32, C.c_void_p, C.c_void_p, C.c_float, C.c_void_p]
        L.orc_lora_delta.argtypes = [C.c_int32, C.c_int64, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p,
                                     C.c_float, C.c_void_p]
        L.orc_ties_k.restype = C.c_int64
        L.orc_ties_k.argtypes = [C.c_int64, C.c_double]
        L.orc_num_threads.restype = C.c_int
        L.orc_set_num_threads.argtypes = [C.c_int]
        _lib = L
    return _lib


DTYPE = {"f32": 0, "bf16": 1}
EBYTES = {"f32": 4, "bf16": 2}


def _i64(a):
    a = np.ascontiguousarray(a, dtype=np.int64)
    return a, a.ctypes.data_as(C.POINTER(C.c_int64))


DELTA = 0x100  # experts hold Delta_i = W_i - W_0 (the explicit-delta source)


def _dt(dtype, delta=False):
    return (DTYPE[dtype] if isinstance(dtype, str) else int(dtype)) | (DELTA if delta else 0)


def _ptrs(arrs):
    arr = (C.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    return arr


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


class Blocks:
    """The block partition of a layout, as computed by the oracle."""

    def __init__(self, numel: Sequence[int], block_elems: int):
        L = lib()
        nt = len(numel)
        numel_a, numel_p = _i64(numel)
        G = L.orc_num_blocks(nt, numel_p, block_elems)
        if G < 0:
            raise ValueError("bad layout")
        self.off = np.zeros(G, np.int64)
        self.len = np.zeros(G, np.int64)
        self.tensor = np.zeros(G, np.int32)
        self.elem0 = np.zeros(G, np.int64)
        _check(L.orc_blocks(nt, numel_p, block_elems,
                            self.off.ctypes.data_as(C.POINTER(C.c_int64)),
                            self.len.ctypes.data_as(C.POINTER(C.c_int64)),
                            self.tensor.ctypes.data_as(C.POINTER(C.c_int32)),
                            self.elem0.ctypes.data_as(C.POINTER(C.c_int64))), "blocks")
        self.G = int(G)
        self.numel = np.ascontiguousarray(numel, np.int64)
        self.block_elems = int(block_elems)


def index(blocks: Blocks, dtype, base, experts, doff=None, ids=None, delta=False):
    """Sum of squared deltas per (block, expert); returns float32 [nb, K].

    ``ids`` restricts to a subset of blocks; ``doff`` overrides where each
    listed block's data starts in the (possibly compact) buffers."""
    L = lib()
    ids = np.arange(blocks.G) if ids is None else np.asarray(ids)
    doff = blocks.off[ids] if doff is None else np.asarray(doff)
    K = len(experts)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    out = np.zeros((len(ids), K), np.float32)
    _check(L.orc_index(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts), K,
                       out.ctypes.data), "index")
    return out


def plan(blocks: Blocks, dtype, K: int, sumsq, w, budget: int, flags: int = 0):
    """Algorithm 1; returns (mask uint32[G], stats dict).  sumsq None: no
    block catalog, the deterministic tensor-level fallback (orc_plan_tensors)."""
    L = lib()
    w = np.ascontiguousarray(w, np.float32)
    assert w.size == K
    mask = np.zeros(blocks.G, np.uint32)
    st = np.zeros(5, np.uint64)
    if sumsq is None:
        n_a, n_p = _i64(blocks.numel)
        _check(L.orc_plan_tensors(len(blocks.numel), n_p, blocks.block_elems, _dt(dtype), K, w.ctypes.data,
                                  int(budget), flags, mask.ctypes.data, st.ctypes.data), "plan (tensor level)")
        return mask, dict(cost=int(st[0]), n_selected=int(st[1]), full_bytes=int(st[2]),
                          digest=int(st[3]), n_units=int(st[4]))
    sumsq = np.ascontiguousarray(sumsq, np.float32).reshape(-1)
    assert sumsq.size == blocks.G * K
    l_a, l_p = _i64(blocks.len)
    _check(L.orc_plan(blocks.G, l_p, _dt(dtype), K, sumsq.ctypes.data, w.ctypes.data,
                      int(budget), flags, mask.ctypes.data, st.ctypes.data), "plan")
    return mask, dict(cost=int(st[0]), n_selected=int(st[1]), full_bytes=int(st[2]),
                      digest=int(st[3]), n_units=int(st[4]))


def _merge_args(blocks, ids, doff):
    ids = np.arange(blocks.G) if ids is None else np.asarray(ids)
    doff = blocks.off[ids] if doff is None else np.asarray(doff)
    return ids, doff


def merge_avg(blocks, dtype, base, experts, mask, alpha, out=None, ids=None, doff=None, delta=False):
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    out = np.empty_like(base) if out is None else out
    mask = np.ascontiguousarray(mask, np.uint32)
    alpha = np.ascontiguousarray(alpha, np.float32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    _check(L.orc_merge_avg(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts),
                           len(experts), mask.ctypes.data, alpha.ctypes.data, out.ctypes.data), "avg")
    return out


def merge_avg_renorm(blocks, dtype, base, experts, mask, alpha, out=None, ids=None, doff=None, delta=False):
    """Selected-only AVG: alpha renormalised over each block's selected experts."""
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    out = np.empty_like(base) if out is None else out
    mask = np.ascontiguousarray(mask, np.uint32)
    alpha = np.ascontiguousarray(alpha, np.float32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    _check(L.orc_merge_avg_renorm(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts),
                                  len(experts), mask.ctypes.data, alpha.ctypes.data, out.ctypes.data),
           "avg_renorm")
    return out


def merge_ties(blocks, dtype, base, experts, mask, density, lam, out=None, ids=None, doff=None, delta=False):
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    out = np.empty_like(base) if out is None else out
    mask = np.ascontiguousarray(mask, np.uint32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    _check(L.orc_merge_ties(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts),
                            len(experts), mask.ctypes.data, float(density), float(lam),
                            out.ctypes.data), "ties")
    return out


def ties_thresholds(blocks, dtype, base, experts, density, ids=None, doff=None, delta=False):
    """Per-unit TIES trim thresholds (uint32 fp32 patterns), [len(ids), K]."""
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    tau = np.zeros((len(ids), len(experts)), np.uint32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    _check(L.orc_ties_thresholds(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts),
                                 len(experts), float(density), tau.ctypes.data), "ties thresholds")
    return tau


def ties_tensor_thresholds(blocks, dtype, base, experts, mask, density, delta=False):
    """Per-tensor trim thresholds over the zero-completed masked deltas:
    uint32 [n_tensors, K] (see orc_ties_tensor_thresholds)."""
    L = lib()
    K = len(experts)
    T = int(blocks.tensor.max()) + 1 if blocks.G else 0
    mask = np.ascontiguousarray(mask, np.uint32)
    tau = np.zeros(T * K, np.uint32)
    d_a, d_p = _i64(blocks.off)
    l_a, l_p = _i64(blocks.len)
    t_a = np.ascontiguousarray(blocks.tensor, np.int32)
    _check(L.orc_ties_tensor_thresholds(blocks.G, d_p, l_p, t_a.ctypes.data_as(C.POINTER(C.c_int32)), T,
                                        _dt(dtype, delta), base.ctypes.data, _ptrs(experts), K, mask.ctypes.data,
                                        float(density), tau.ctypes.data), "ties_tensor_thresholds")
    return tau.reshape(T, K)


def expand_tensor_thresholds(blocks, tau_t):
    """Per-unit thresholds [G * K] from per-tensor ones: unit (g, i) takes its tensor's."""
    return np.ascontiguousarray(tau_t[blocks.tensor], np.uint32).reshape(-1)


def merge_ties_tau(blocks, dtype, base, experts, mask, tau, lam, out=None, ids=None, doff=None, delta=False):
    """TIES with given per-unit thresholds tau [len(ids), K]."""
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    out = np.empty_like(base) if out is None else out
    mask = np.ascontiguousarray(mask, np.uint32)
    tau = np.ascontiguousarray(tau, np.uint32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    _check(L.orc_merge_ties_tau(len(ids), d_p, l_p, _dt(dtype, delta), base.ctypes.data, _ptrs(experts),
                                len(experts), mask.ctypes.data, tau.ctypes.data, float(lam),
                                out.ctypes.data), "ties tau")
    return out


def merge_dare(blocks, dtype, base, experts, mask, p, seed, combine, alpha, lam,
               out=None, ids=None, doff=None, delta=False):
    """combine: 0 = linear, 1 = sign-elect."""
    L = lib()
    ids, doff = _merge_args(blocks, ids, doff)
    out = np.empty_like(base) if out is None else out
    mask = np.ascontiguousarray(mask, np.uint32)
    alpha = np.ascontiguousarray(alpha, np.float32)
    d_a, d_p = _i64(doff)
    l_a, l_p = _i64(blocks.len[ids])
    t_a = np.ascontiguousarray(blocks.tensor[ids], np.int32)
    e_a, e_p = _i64(blocks.elem0[ids])
    _check(L.orc_merge_dare(len(ids), d_p, l_p, t_a.ctypes.data_as(C.POINTER(C.c_int32)), e_p,
                            _dt(dtype, delta), base.ctypes.data, _ptrs(experts), len(experts),
                            mask.ctypes.data, float(p), int(seed) & 0xFFFFFFFF, int(combine),
                            alpha.ctypes.data, float(lam), out.ctypes.data), "dare")
    return out


def lora_delta(dtype, rows: int, cols: int, A, B, scale: float):
    """One adapted tensor's delta, [rows * cols] in the checkpoint dtype.

    A: [rank, cols], B: [rows, rank] (row-major, checkpoint dtype)."""
    A = np.ascontiguousarray(A)
    B = np.ascontiguousarray(B)
    rank = A.shape[0]
    if A.shape != (rank, cols) or B.shape != (rows, rank) or A.dtype != B.dtype:
        raise ValueError("adapter shapes do not match the tensor")
    out = np.zeros(rows * cols, A.dtype)
    _check(lib().orc_lora_delta(_dt(dtype), rows, cols, rank, A.ctypes.data, B.ctypes.data, float(scale),
                                out.ctypes.data), "lora delta")
    return out


def lora_materialize(blocks: Blocks, dtype, numel, loras, adapters, mask=None, fill=None):
    """Explicit delta checkpoints drawn from LoRA adapters (one per expert).

    ``loras``: records (tensor, rows, cols, rank, a_off, b_off, scale); expert
    i's A and B of a record lie at those element offsets of ``adapters[i]``.
    Tensors without a record have zero deltas.  Unit (g, i) is written when
    bit i of mask[g] is set (every unit when mask is None); the other
    elements keep ``fill[i]`` (zeros when fill is None)."""
    numel = [int(n) for n in numel]
    toff = np.concatenate([[0], np.cumsum(numel)]).astype(np.int64)
    P = int(toff[-1])
    out = []
    for i, ad in enumerate(adapters):
        ad = np.ascontiguousarray(ad)
        full = np.zeros(P, ad.dtype)
        for (t, rows, cols, rank, a_off, b_off, scale) in loras:
            A = ad[a_off:a_off + rank * cols].reshape(rank, cols)
            B = ad[b_off:b_off + rows * rank].reshape(rows, rank)
            full[toff[t]:toff[t] + rows * cols] = lora_delta(dtype, rows, cols, A, B, scale)
        d = np.zeros(P, ad.dtype) if fill is None else np.array(fill[i], copy=True)
        for g in range(blocks.G):
            if mask is None or (int(mask[g]) >> i) & 1:
                o, n = int(blocks.off[g]), int(blocks.len[g])
                d[o:o + n] = full[o:o + n]
        out.append(d)
    return out


def philox4x32_10(ctr, key):
    L = lib()
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    o = np.zeros(4, np.uint32)
    L.orc_philox4x32_10(c.ctypes.data, k.ctypes.data, o.ctypes.data)
    return o


def mix64(x: int) -> int:
    return int(lib().orc_mix64(int(x) & 0xFFFFFFFFFFFFFFFF))


def round_bf16(x):
    x = np.ascontiguousarray(x, np.float32)
    y = np.zeros(x.shape, np.uint16)
    lib().orc_round_bf16(x.ctypes.data, y.ctypes.data, x.size)
    return y


def ties_k(n: int, density: float) -> int:
    return int(lib().orc_ties_k(int(n), float(density)))


def num_threads() -> int:
    return int(lib().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (results do not
    depend on it)."""
    lib().orc_set_num_threads(int(n))


def full_bytes(blocks: Blocks, dtype, K: int) -> int:
    return int(blocks.len.sum()) * EBYTES[dtype if isinstance(dtype, str) else ("f32", "bf16")[dtype]] * K
