"""The C ABI library loads, exports every entry point include/mergepipe.h
declares, and rejects invalid arguments before touching the GPU.  Runs on the
CPU: none of the calls below reaches a HIP runtime call."""

import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mergepipe.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mp_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def mp():
    import paper_2605_29489_amd as m
    return m


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("mp_layout_blocks", "mp_index_blocks", "mp_plan", "mp_merge_avg", "mp_merge_avg_renorm", "mp_merge_ties",
              "mp_merge_dare", "mp_last_error", "mp_release"):
        assert n in names


def test_every_declared_symbol_is_exported(mp):
    lib = C.CDLL(mp.LIB_PATH)
    for n in _declared():
        assert hasattr(lib, n), n
    assert set(mp.EXPORTS) <= set(_declared())


def test_struct_layouts_match_header(mp):
    # mp_layout: int32, int32, pointer, int64 -> 24 bytes on LP64
    assert C.sizeof(mp.mp_layout) == 24
    assert C.sizeof(mp.mp_plan_stats) == 48
    assert C.sizeof(mp.mp_io_stats) == 32 + 8 * 32  # four totals + per-expert bytes
    assert C.sizeof(mp.mp_lora_tensor) == 48  # int32 x2, int64 x4, float + tail padding


def test_lora_records_rejected_before_any_device_work(mp):
    lib = mp.lib
    L = mp.Layout([64 * 96, 512, 32 * 48], 256, mp.MP_BF16)
    ptrs = (C.c_void_p * 2)(None, None)

    def rc(recs, K=2, adapters=ptrs, deltas=ptrs):  # records in the C field order
        arr = (mp.mp_lora_tensor * max(len(recs), 1))(*[mp.mp_lora_tensor(*r) for r in recs])
        return lib.mp_lora_materialize(L.ref, arr, len(recs), adapters, K, None, deltas, None)

    good = (0, 16, 64, 96, 0, 16 * 96, 0.5)
    bad = [
        [(3, 16, 64, 96, 0, 0, 1.0)],            # no such tensor
        [good, (0, 8, 64, 96, 0, 0, 1.0)],       # two adapters for one tensor
        [(0, 0, 64, 96, 0, 0, 1.0)],             # rank 0
        [(0, 65, 64, 96, 0, 0, 1.0)],            # rank above 64
        [(0, 16, 96, 60, 0, 0, 1.0), (2, 4, 48, 32, 0, 0, 1.0)],  # shape does not match numel
        [(1, 4, 2, 256, 0, 0, 1.0), (2, 4, 16, 100, 0, 0, 1.0)],  # ok, then rows x cols != numel
        [(1, 4, 128, 4, 0, 0, 1.0), (0, 4, 64, 96, -1, 0, 1.0)],  # negative offset
        [(0, 4, 64, 96, 0, 0, float("inf"))],    # non-finite scale
        [(1, 4, 256, 2, 0, 0, 1.0)],             # cols not a multiple of 4
        [(0, 4, 1 << 40, 1 << 40, 0, 0, 1.0)],   # a product that overflows int64
        [(0, 4, 64, 96, 1 << 50, 0, 1.0)],       # offset beyond 2^48
    ]
    for recs in bad:
        assert rc(recs) == mp.MP_E_ARG, recs
    assert rc([good], K=0) == mp.MP_E_ARG
    assert rc([good], K=33) == mp.MP_E_ARG
    assert rc([good], adapters=None) == mp.MP_E_ARG
    assert rc([good], deltas=None) == mp.MP_E_ARG


def test_layout_blocks_counts(mp):
    from workloads import family_spec
    for name, G in (("qwen2.5-1.5b", 376989), ("llama3-8b", 1960513), ("qwen2.5-7b", 1859341), ("toy", 1024)):
        lay = family_spec(name).layout
        L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
        assert mp.mp_layout_blocks(L) == G
    assert mp.mp_layout_blocks(mp.Layout([], 4096, mp.MP_BF16)) == 0


@pytest.mark.parametrize("numel,be,dt", [
    ([4096], 4100, 1),   # block not a multiple of 8 bf16 elements
    ([4100], 4096, 1),   # tensor not 16-byte aligned
    ([4096], 0, 0),
    ([-8], 4096, 0),
    ([4096], 4096, 7),   # bad dtype
])
def test_layout_validation(mp, numel, be, dt):
    L = mp.Layout(numel, be, dt)
    with pytest.raises(mp.MPError) as e:
        mp.mp_layout_blocks(L)
    assert e.value.code == mp.MP_E_ARG
    assert mp.mp_last_error() != ""


def test_argument_errors_before_any_device_call(mp):
    L = mp.Layout([4096], 4096, mp.MP_BF16)
    lib = mp.lib
    ptrs = (C.c_void_p * 33)()
    # K out of range
    for K in (0, 33):
        assert lib.mp_index_blocks(L.ref, None, ptrs, K, 0, None, None) == mp.MP_E_ARG
        st = mp.mp_plan_stats()
        w = (C.c_float * 33)(*([1.0] * 33))
        assert lib.mp_plan(L.ref, K, None, w, 0, 0, None, C.byref(st), None) == mp.MP_E_ARG
    # bad residency
    assert lib.mp_index_blocks(L.ref, None, ptrs, 1, 5, None, None) == mp.MP_E_ARG
    # the explicit-delta bit combines with a valid residency only
    assert lib.mp_index_blocks(L.ref, None, ptrs, 1, mp.MP_EXPERTS_DELTA | 3, None, None) == mp.MP_E_ARG
    assert lib.mp_index_blocks(L.ref, None, ptrs, 1, 32, None, None) == mp.MP_E_ARG
    assert "residency" in mp.mp_last_error()
    # unsupported plan flags (bits other than per-byte and skip-zero)
    st = mp.mp_plan_stats()
    w = (C.c_float * 1)(1.0)
    for fl in (4, 8, 0x80000000, 4 | mp.MP_PLAN_PER_BYTE):
        assert lib.mp_plan(L.ref, 1, None, w, 0, fl, None, C.byref(st), None) == mp.MP_E_UNSUPPORTED
    # non-finite plan weight
    wn = (C.c_float * 1)(float("nan"))
    assert lib.mp_plan(L.ref, 1, None, wn, 0, 0, None, C.byref(st), None) == mp.MP_E_ARG
    # TIES density and DARE p/combine ranges
    assert lib.mp_merge_ties(L.ref, None, ptrs, 1, 0, None, 1.5, 1.0, None, None, None) == mp.MP_E_ARG
    assert lib.mp_merge_ties(L.ref, None, ptrs, 1, 0, None, -0.1, 1.0, None, None, None) == mp.MP_E_ARG
    a = (C.c_float * 1)(1.0)
    assert lib.mp_merge_dare(L.ref, None, ptrs, 1, 0, None, 1.0, 0, 0, a, 1.0, None, None, None) == mp.MP_E_ARG
    assert lib.mp_merge_dare(L.ref, None, ptrs, 1, 0, None, 0.5, 0, 9, a, 1.0, None, None, None) == mp.MP_E_ARG
    assert lib.mp_merge_dare(L.ref, None, ptrs, 1, 0, None, 0.5, 0, 0, None, 1.0, None, None, None) == mp.MP_E_ARG
    # AVG with NULL / non-finite alpha
    assert lib.mp_merge_avg(L.ref, None, ptrs, 1, 0, None, None, None, None, None) == mp.MP_E_ARG
    an = (C.c_float * 1)(float("inf"))
    assert lib.mp_merge_avg(L.ref, None, ptrs, 1, 0, None, an, None, None, None) == mp.MP_E_ARG
    assert lib.mp_merge_avg_renorm(L.ref, None, ptrs, 1, 0, None, None, None, None, None) == mp.MP_E_ARG
    assert lib.mp_merge_avg_renorm(L.ref, None, ptrs, 1, 0, None, an, None, None, None) == mp.MP_E_ARG
    # stream copy: sizes that are not a multiple of 16, or beyond 2^40
    assert lib.mp_stream_copy(None, None, 17, None) == mp.MP_E_ARG
    assert "multiple of 16" in mp.mp_last_error()
    assert lib.mp_stream_copy(None, None, 1 << 41, None) == mp.MP_E_ARG
    # unit ids must fit 32 bits: 2^28 blocks x 32 experts
    big = mp.Layout([4096 * (1 << 28)], 4096, mp.MP_BF16)
    assert lib.mp_index_blocks(big.ref, None, ptrs, 32, 0, None, None) == mp.MP_E_ARG
    assert "32-bit" in mp.mp_last_error()


def test_plan_noalloc_rejects_a_layout_beyond_its_fixed_array(mp):
    # 5 million blocks need 20 MB of block lengths, more than the plan's
    # fixed 16 MiB device array: refused on the host, before any device work,
    # with the sizes in the message (no GPU is touched)
    lib = mp.lib
    st = mp.mp_plan_stats()
    w = (C.c_float * 1)(1.0)
    L = mp.Layout([4096 * 1000] * 5000, 4096, mp.MP_BF16)
    rc = lib.mp_plan_noalloc(L.ref, 1, None, w, 0, 0, None, C.byref(st), None)
    assert rc == mp.MP_E_UNSUPPORTED
    msg = lib.mp_last_error().decode()
    need = int(msg.split(" needs ")[1].split()[0])
    assert "16777216" in msg and need > 16777216 and "5000000 blocks" in msg
    # the tensor-level plan (no catalog) refuses tensors of 2^32 or more elements
    L = mp.Layout([4096 * 2_000_000], 4096, mp.MP_BF16)
    assert lib.mp_plan_noalloc(L.ref, 1, None, w, 0, 0, None, C.byref(st), None) == mp.MP_E_UNSUPPORTED
    assert "2^32" in lib.mp_last_error().decode()
    # argument errors come first, as in mp_plan
    assert lib.mp_plan_noalloc(L.ref, 40, None, w, 0, 0, None, C.byref(st), None) == mp.MP_E_ARG
    assert lib.mp_plan_noalloc(L.ref, 1, None, w, 0, 8, None, C.byref(st), None) == mp.MP_E_UNSUPPORTED



def test_argument_errors_leave_host_outputs_untouched(mp):
    # On an argument error nothing is written: the host-side stats, coverage
    # and io records keep their contents (checked on the CPU, where the
    # errors are caught before any device call).
    lib = mp.lib
    L = mp.Layout([4096, 4096], 4096, mp.MP_BF16)
    ptrs = (C.c_void_p * 4)()
    sentinel = 0x5A5A5A5A5A5A5A5A
    st = mp.mp_plan_stats(*([sentinel] * 6))
    w = (C.c_float * 4)(*([1.0] * 4))
    wn = (C.c_float * 4)(*([float("nan")] * 4))
    for call in (lambda: lib.mp_plan(L.ref, 0, None, w, 0, 0, None, C.byref(st), None),
                 lambda: lib.mp_plan(L.ref, 4, None, wn, 0, 0, None, C.byref(st), None),
                 lambda: lib.mp_plan(L.ref, 4, None, w, 0, 16, None, C.byref(st), None),
                 lambda: lib.mp_plan_noalloc(L.ref, 4, None, wn, 0, 0, None, C.byref(st), None)):
        assert call() in (mp.MP_E_ARG, mp.MP_E_UNSUPPORTED)
        assert all(getattr(st, f) == sentinel for f, _ in st._fields_)
    cov = (C.c_uint64 * 8)(*([sentinel] * 8))
    assert lib.mp_coverage(L.ref, 0, None, cov, None) == mp.MP_E_ARG
    assert lib.mp_coverage(L.ref, 4, None, None, None) == mp.MP_E_ARG
    assert all(x == sentinel for x in cov)
    io = mp.mp_io_stats()
    io.expert_bytes = io.base_bytes = io.out_bytes = io.h2d_bytes = sentinel
    a = (C.c_float * 4)(*([float("inf")] * 4))
    assert lib.mp_merge_avg(L.ref, None, ptrs, 4, 0, None, a, None, C.byref(io), None) == mp.MP_E_ARG
    assert lib.mp_merge_ties(L.ref, None, ptrs, 4, 0, None, 2.0, 1.0, None, C.byref(io), None) == mp.MP_E_ARG
    assert lib.mp_merge_dare(L.ref, None, ptrs, 4, 0, None, 1.5, 0, 0, w, 1.0, None, C.byref(io), None) == mp.MP_E_ARG
    assert (io.expert_bytes, io.base_bytes, io.out_bytes, io.h2d_bytes) == (sentinel,) * 4
    # the workspace cap takes any value; its byte count reads without a GPU
    assert lib.mp_set_workspace_limit(0) == mp.MP_OK
    assert lib.mp_workspace_bytes() == 0
