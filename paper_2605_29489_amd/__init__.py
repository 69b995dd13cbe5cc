"""Python binding of libmergepipe.so (budgeted weight-space merging on MI355X).

Argument marshalling only: every step of the path (index, plan, merge) runs
in the library's HIP kernels.  PyTorch is used for device/pinned memory and
streams.  The functions have the names of the C entry points declared in
``include/mergepipe.h``; they take torch tensors and raise ``MPError`` on a
non-zero status.

The library must have been built (``python -m paper_2605_29489_amd.build``
or ``__graft_entry__.build()``); importing this package without it raises
ImportError -- there is no fallback.
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmergepipe.so")

MP_OK = 0
MP_E_ARG = -1
MP_E_UNSUPPORTED = -2
MP_E_NOMEM = -3
MP_E_HIP = -4
MP_E_IO = -5
MP_F32, MP_BF16 = 0, 1
MP_DEVICE, MP_HOST_PINNED, MP_HOST_PAGEABLE, MP_HOST_FILE = 0, 1, 2, 3
MP_EXPERTS_DELTA = 16  # OR-ed into residency: experts hold W_i - W_0
MP_COMBINE_LINEAR, MP_COMBINE_SIGN_ELECT = 0, 1
MP_PLAN_PER_BYTE, MP_PLAN_SKIP_ZERO = 1, 2

EXPORTS = ("mp_layout_blocks", "mp_index_blocks", "mp_index_ties", "mp_ties_tensor_thresholds", "mp_plan",
           "mp_plan_noalloc", "mp_coverage", "mp_merge_avg", "mp_merge_avg_renorm",
           "mp_merge_ties",
           "mp_merge_ties_tau", "mp_merge_dare", "mp_lora_materialize", "mp_lora_merge_ties_tau", "mp_stream_copy",
           "mp_set_stage_bytes",
           "mp_set_workspace_limit", "mp_workspace_bytes", "mp_last_error", "mp_release")


class mp_layout(C.Structure):
    _fields_ = [("n_tensors", C.c_int32), ("dtype", C.c_int32),
                ("numel", C.POINTER(C.c_int64)), ("block_elems", C.c_int64)]


class mp_plan_stats(C.Structure):
    _fields_ = [("budget_bytes", C.c_uint64), ("cost_bytes", C.c_uint64), ("full_bytes", C.c_uint64),
                ("n_selected", C.c_uint64), ("n_units", C.c_uint64), ("digest", C.c_uint64)]

    def as_dict(self):
        return {f: int(getattr(self, f)) for f, _ in self._fields_}


class mp_io_stats(C.Structure):
    _fields_ = [("expert_bytes", C.c_uint64), ("base_bytes", C.c_uint64), ("out_bytes", C.c_uint64),
                ("h2d_bytes", C.c_uint64), ("expert_bytes_by_expert", C.c_uint64 * 32)]

    def as_dict(self):
        d = {f: int(getattr(self, f)) for f, _ in self._fields_[:4]}
        d["expert_bytes_by_expert"] = [int(x) for x in self.expert_bytes_by_expert]
        return d


class mp_lora_tensor(C.Structure):
    _fields_ = [("tensor", C.c_int32), ("rank", C.c_int32), ("rows", C.c_int64), ("cols", C.c_int64),
                ("a_off", C.c_int64), ("b_off", C.c_int64), ("scale", C.c_float)]


class MPError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mergepipe error {code}: {msg}")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    # Buffers come from torch, which ships its own HIP runtime.  Load that one
    # first, so this library binds to the same runtime: loaded the other way
    # round, the library's runtime does not know torch's allocations.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = C.CDLL(LIB_PATH)
    vp, i32, u32, u64 = C.c_void_p, C.c_int32, C.c_uint32, C.c_uint64
    lp = C.POINTER(mp_layout)
    L.mp_layout_blocks.argtypes = [lp, C.POINTER(C.c_int64)]
    L.mp_index_blocks.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, vp]
    L.mp_index_ties.argtypes = [lp, vp, C.POINTER(vp), i32, i32, C.c_double, vp, vp, vp]
    L.mp_plan.argtypes = [lp, i32, vp, C.POINTER(C.c_float), u64, u32, vp, C.POINTER(mp_plan_stats), vp]
    L.mp_plan_noalloc.argtypes = L.mp_plan.argtypes
    L.mp_merge_avg.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, C.POINTER(C.c_float), vp,
                               C.POINTER(mp_io_stats), vp]
    L.mp_merge_avg_renorm.argtypes = L.mp_merge_avg.argtypes
    L.mp_coverage.argtypes = [lp, i32, vp, C.POINTER(C.c_uint64), vp]
    L.mp_ties_tensor_thresholds.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, C.c_double, vp, vp]
    L.mp_merge_ties.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, C.c_double, C.c_float, vp,
                                C.POINTER(mp_io_stats), vp]
    L.mp_merge_ties_tau.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, vp, C.c_float, vp,
                                    C.POINTER(mp_io_stats), vp]
    L.mp_merge_dare.argtypes = [lp, vp, C.POINTER(vp), i32, i32, vp, C.c_double, u32, i32,
                                C.POINTER(C.c_float), C.c_float, vp, C.POINTER(mp_io_stats), vp]
    L.mp_lora_materialize.argtypes = [lp, C.POINTER(mp_lora_tensor), i32, C.POINTER(vp), i32, vp, C.POINTER(vp),
                                      vp]
    L.mp_lora_merge_ties_tau.argtypes = [lp, vp, C.POINTER(mp_lora_tensor), i32, C.POINTER(vp), i32, vp, vp,
                                         C.c_float, vp, vp]
    L.mp_last_error.restype = C.c_char_p
    L.mp_stream_copy.argtypes = [vp, vp, u64, vp]
    L.mp_set_stage_bytes.argtypes = [u64]
    L.mp_set_stage_bytes.restype = i32
    L.mp_set_workspace_limit.argtypes = [u64]
    L.mp_set_workspace_limit.restype = i32
    L.mp_workspace_bytes.argtypes = []
    L.mp_workspace_bytes.restype = u64
    L.mp_last_error.argtypes = []
    L.mp_release.argtypes = []
    for name in ("mp_layout_blocks", "mp_index_blocks", "mp_index_ties", "mp_ties_tensor_thresholds", "mp_plan",
                 "mp_plan_noalloc", "mp_coverage", "mp_merge_avg",
                 "mp_merge_avg_renorm", "mp_merge_ties",
                 "mp_merge_ties_tau",
                 "mp_merge_dare", "mp_lora_materialize", "mp_lora_merge_ties_tau", "mp_stream_copy"):
        getattr(L, name).restype = C.c_int
    return L


lib = _load()


@dataclass
class Layout:
    """Host-side mp_layout: tensor numels, block size and dtype code."""

    numel: Sequence[int]
    block_elems: int
    dtype: int  # MP_F32 or MP_BF16

    def __post_init__(self):
        self._numel = (C.c_int64 * max(len(self.numel), 1))(*[int(n) for n in self.numel])
        self._s = mp_layout(len(self.numel), int(self.dtype), C.cast(self._numel, C.POINTER(C.c_int64)),
                            int(self.block_elems))

    @property
    def ref(self):
        return C.byref(self._s)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == MP_F32 else 2

    @property
    def n_params(self) -> int:
        return int(sum(int(n) for n in self.numel))


def _check(rc: int):
    if rc != MP_OK:
        raise MPError(rc, lib.mp_last_error().decode())


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _ptrs(ts):
    """Array of expert pointers: tensors by address, file paths (MP_HOST_FILE)
    as NUL-terminated strings kept alive with the array."""
    keep, vals = [], []
    for t in ts:
        if isinstance(t, (str, bytes, os.PathLike)):
            b = C.create_string_buffer(os.fsencode(t))
            keep.append(b)
            vals.append(C.addressof(b))
        else:
            vals.append(_ptr(t))
    arr = (C.c_void_p * max(len(ts), 1))(*vals)
    arr._keep = keep
    return arr


def _floats(xs, K):
    if xs is None:
        return None
    xs = [float(x) for x in xs]
    if len(xs) != K:
        raise ValueError(f"expected {K} coefficients, got {len(xs)}")
    return (C.c_float * K)(*xs)


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def mp_layout_blocks(layout: Layout) -> int:
    g = C.c_int64(0)
    _check(lib.mp_layout_blocks(layout.ref, C.byref(g)))
    return int(g.value)


def mp_index_blocks(layout: Layout, base, experts, sumsq, residency: int = MP_DEVICE, stream=None,
                    delta: bool = False):
    _check(lib.mp_index_blocks(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta),
                               _ptr(sumsq), _stream(stream)))


def mp_index_ties(layout: Layout, base, experts, density: float, tau, sumsq=None, residency: int = MP_DEVICE,
                  stream=None, delta: bool = False):
    """Per-unit TIES thresholds (uint32 patterns in `tau`, G*K) and, if given, sumsq."""
    _check(lib.mp_index_ties(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta),
                             float(density),
                             _ptr(sumsq), _ptr(tau), _stream(stream)))


def mp_plan(layout: Layout, K: int, sumsq, w, budget_bytes: int, mask, flags: int = 0, stream=None) -> dict:
    st = mp_plan_stats()
    _check(lib.mp_plan(layout.ref, K, _ptr(sumsq), _floats(w, K), int(budget_bytes), flags, _ptr(mask),
                       C.byref(st), _stream(stream)))
    return st.as_dict()


def mp_plan_noalloc(layout: Layout, K: int, sumsq, w, budget_bytes: int, mask, flags: int = 0,
                    stream=None) -> dict:
    """mp_plan on the library's fixed device array (allocates nothing)."""
    st = mp_plan_stats()
    _check(lib.mp_plan_noalloc(layout.ref, K, _ptr(sumsq), _floats(w, K), int(budget_bytes), flags, _ptr(mask),
                               C.byref(st), _stream(stream)))
    return st.as_dict()


def _res(residency: int, delta: bool) -> int:
    return residency | (MP_EXPERTS_DELTA if delta else 0)


def _io(io):
    return C.byref(io) if io is not None else None


def mp_ties_tensor_thresholds(layout: Layout, base, experts, mask, density: float, tau,
                              residency: int = MP_DEVICE, stream=None, delta: bool = False):
    """Per-unit TIES thresholds at tensor scope for this mask (device uint32 [G*K])."""
    _check(lib.mp_ties_tensor_thresholds(layout.ref, _ptr(base), _ptrs(experts), len(experts),
                                         _res(residency, delta), _ptr(mask), float(density), _ptr(tau),
                                         _stream(stream)))


def mp_coverage(layout: Layout, K: int, mask, stream=None):
    """Touched elements per (tensor, expert) of a mask: numpy uint64 [n_tensors, K]."""
    import numpy as np
    cov = np.zeros(len(layout.numel) * K, np.uint64)
    _check(lib.mp_coverage(layout.ref, K, _ptr(mask), cov.ctypes.data_as(C.POINTER(C.c_uint64)), _stream(stream)))
    return cov.reshape(len(layout.numel), K)


def mp_merge_avg(layout: Layout, base, experts, mask, alpha, out, residency: int = MP_DEVICE,
                 io: bool = False, stream=None, delta: bool = False) -> Optional[dict]:
    st = mp_io_stats() if io else None
    _check(lib.mp_merge_avg(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta), _ptr(mask),
                            _floats(alpha, len(experts)), _ptr(out), _io(st), _stream(stream)))
    return st.as_dict() if io else None


def mp_merge_avg_renorm(layout: Layout, base, experts, mask, alpha, out, residency: int = MP_DEVICE,
                        io: bool = False, stream=None, delta: bool = False) -> Optional[dict]:
    """Selected-only AVG: alpha renormalised over each block's selected experts."""
    st = mp_io_stats() if io else None
    _check(lib.mp_merge_avg_renorm(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta),
                                   _ptr(mask),
                                   _floats(alpha, len(experts)), _ptr(out), _io(st), _stream(stream)))
    return st.as_dict() if io else None


def mp_merge_ties(layout: Layout, base, experts, mask, density: float, lam: float, out,
                  residency: int = MP_DEVICE, io: bool = False, stream=None, delta: bool = False) -> Optional[dict]:
    st = mp_io_stats() if io else None
    _check(lib.mp_merge_ties(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta), _ptr(mask),
                             float(density), float(lam), _ptr(out), _io(st), _stream(stream)))
    return st.as_dict() if io else None


def mp_merge_ties_tau(layout: Layout, base, experts, mask, tau, lam: float, out, residency: int = MP_DEVICE,
                      io: bool = False, stream=None, delta: bool = False) -> Optional[dict]:
    st = mp_io_stats() if io else None
    _check(lib.mp_merge_ties_tau(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta),
                                 _ptr(mask),
                                 _ptr(tau), float(lam), _ptr(out), _io(st), _stream(stream)))
    return st.as_dict() if io else None


def mp_merge_dare(layout: Layout, base, experts, mask, p: float, seed: int, combine: int, alpha, lam: float,
                  out, residency: int = MP_DEVICE, io: bool = False, stream=None,
                  delta: bool = False) -> Optional[dict]:
    st = mp_io_stats() if io else None
    a = _floats(alpha, len(experts)) if alpha is not None else None
    _check(lib.mp_merge_dare(layout.ref, _ptr(base), _ptrs(experts), len(experts), _res(residency, delta), _ptr(mask),
                             float(p), int(seed) & 0xFFFFFFFF, int(combine), a, float(lam), _ptr(out), _io(st),
                             _stream(stream)))
    return st.as_dict() if io else None


def mp_lora_materialize(layout: Layout, loras, adapters, deltas, mask=None, stream=None):
    """Explicit-delta checkpoints drawn from LoRA adapters (selected units only).

    ``loras``: records (tensor, rows, cols, rank, a_off, b_off, scale);
    ``adapters``/``deltas``: K device tensors each (adapters may be empty
    when there are no records)."""
    recs = (mp_lora_tensor * max(len(loras), 1))(
        *[mp_lora_tensor(int(t), int(rank), int(rows), int(cols), int(a), int(b), float(sc))
          for (t, rows, cols, rank, a, b, sc) in loras])
    K = len(deltas)
    _check(lib.mp_lora_materialize(layout.ref, recs, len(loras), _ptrs(adapters) if loras else None, K, _ptr(mask),
                                   _ptrs(deltas), _stream(stream)))


def mp_lora_merge_ties_tau(layout: Layout, base, loras, adapters, mask, tau, lam, out, stream=None):
    """Budgeted TIES from catalog thresholds with every selected delta drawn
    from the adapters inside the merge (no delta checkpoint): equal to
    ``mp_lora_materialize(mask)`` then ``mp_merge_ties_tau(delta=True)``.

    ``loras`` as for mp_lora_materialize; ``adapters``: K device tensors
    (K entries of None when there are no records); ``mask``: device
    int32[G]; ``tau``: device int32[G*K]."""
    recs = (mp_lora_tensor * max(len(loras), 1))(
        *[mp_lora_tensor(int(t), int(rank), int(rows), int(cols), int(a), int(b), float(sc))
          for (t, rows, cols, rank, a, b, sc) in loras])
    K = len(adapters)
    _check(lib.mp_lora_merge_ties_tau(layout.ref, _ptr(base), recs, len(loras), _ptrs(adapters) if loras else None,
                                      K, _ptr(mask),
                                      _ptr(tau), float(lam), _ptr(out), _stream(stream)))


def mp_last_error() -> str:
    return lib.mp_last_error().decode()


def mp_stream_copy(src, dst, stream=None):
    """Plain stream copy of src's bytes into dst (device tensors of equal
    byte size, a multiple of 16): a measurement aid for the HBM rate."""
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("src and dst differ in size")
    _check(lib.mp_stream_copy(_ptr(src), _ptr(dst), n, _stream(stream)))


def mp_set_stage_bytes(nbytes: int):
    _check(lib.mp_set_stage_bytes(int(nbytes)))


def mp_set_workspace_limit(nbytes: int):
    """Cap on the library's cached workspace in bytes (0: none)."""
    _check(lib.mp_set_workspace_limit(int(nbytes)))


def mp_workspace_bytes() -> int:
    return int(lib.mp_workspace_bytes())


def mp_release():
    lib.mp_release()
