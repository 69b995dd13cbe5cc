"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, on the
same seeded inputs.

Bars: index (sumsq), mask and plan statistics bit-exact; merged weights
within 1e-6 relative (fp32) or 1 bf16 ulp after the final rounding
(`assert_merge_equal`), and in fact bitwise equal: both sides fix the same
operation order, so any difference is reported; the expert bytes the merge
kernels load equal the plan's cost (Prop. 1: the executor reads only
selected blocks).
"""

import math
import os
import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_merge_equal, gather_blocks, to_dev, to_host, to_pinned
from workloads import FamilySpec, family_spec, make_family

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2605_29489_amd as m
    return m


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _mini_qwen(n_layers=2, K=4, dtype="bf16", be=4096):
    """Small family with the Qwen tensor pattern: full blocks, biases and
    norms (short blocks: 256 and 64 elements) and ragged tensor tails."""
    hidden, ffn, vocab = 256, 704, 520
    t = [("embed_tokens.weight", (vocab, hidden))]
    for l in range(n_layers):
        p = f"layers.{l}."
        t += [(p + "q.weight", (hidden, hidden)), (p + "q.bias", (hidden,)),
              (p + "k.weight", (64, hidden)), (p + "k.bias", (64,)),
              (p + "v.weight", (64, hidden)), (p + "v.bias", (64,)),
              (p + "o.weight", (hidden, hidden)),
              (p + "gate.weight", (ffn, hidden)), (p + "up.weight", (ffn, hidden)),
              (p + "down.weight", (hidden, ffn)),
              (p + "input_layernorm.weight", (hidden,)), (p + "post_attention_layernorm.weight", (hidden,))]
    t.append(("norm.weight", (hidden,)))
    return FamilySpec("mini-qwen", tuple(t), dtype, be, K, ())


def _ragged_f32(K=3):
    t = (("a", (3 * 4096 + 4,)), ("b", (8,)), ("c", (4096,)), ("d", (2052,)), ("e", (4, 1025)))
    return FamilySpec("ragged-f32", t, "f32", 4096, K, ())


def _expert_files(exps_np):
    """Writes each expert checkpoint to a file of its own; returns the paths."""
    import tempfile
    d = tempfile.mkdtemp(prefix="mp_experts_")
    paths = []
    for i, e in enumerate(exps_np):
        p = os.path.join(d, f"expert{i}.bin")
        np.ascontiguousarray(e).tofile(p)
        paths.append(p)
    return paths


def _lay(mp, spec):
    lay = spec.layout
    return mp.Layout(lay.numel, lay.block_elems, lay.dtype_code), lay


def _run_all(mp, spec, base_np, exps_np, op, budgets, w=None, residency=None, delta=False, **kw):
    """Index, plan and merge on the GPU and with the oracle; compare.  With
    residency MP_HOST_PINNED the experts stay in pinned host memory; with
    delta the expert arrays are explicit deltas (MP_EXPERTS_DELTA)."""
    import torch
    L, lay = _lay(mp, spec)
    K = len(exps_np)
    dtype = lay.dtype
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    res = mp.MP_DEVICE if residency is None else residency
    base = to_dev(base_np, dtype)
    if res == mp.MP_HOST_PINNED:
        exps = [to_pinned(e, dtype) for e in exps_np]
    elif res == mp.MP_HOST_PAGEABLE:  # ordinary host memory (the numpy arrays themselves)
        exps = [torch.from_numpy(e) for e in exps_np]
    elif res == mp.MP_HOST_FILE:  # files holding the flat checkpoints
        exps = _expert_files(exps_np)
    else:
        exps = [to_dev(e, dtype) for e in exps_np]
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    tau = None
    if op == "ties_tau":  # catalog pass: sums of squares and per-unit thresholds together
        tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
        mp.mp_index_ties(L, base, exps, kw["density"], tau, sumsq=sumsq, residency=res, delta=delta)
        t_orc = oracle.ties_thresholds(blocks, dtype, base_np, exps_np, kw["density"], delta=delta).reshape(-1)
        assert np.array_equal(tau.cpu().numpy().view(np.uint32), t_orc), "thresholds differ"
    else:
        mp.mp_index_blocks(L, base, exps, sumsq, residency=res, delta=delta)
    S_gpu = sumsq.cpu().numpy()
    S_orc = oracle.index(blocks, dtype, base_np, exps_np, delta=delta).reshape(-1)
    assert np.array_equal(S_gpu.view(np.uint32), S_orc.view(np.uint32)), "index differs"
    if w is None:
        w = [1.0 / K] * K if op in ("avg", "avg_renorm", "dare_lin") else [1.0] * K
    full = int(blocks.len.sum()) * lay.elem_bytes * K
    out = torch.empty_like(base)
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    results = []
    for f in budgets:
        B = int(f * full) if isinstance(f, float) else int(f)
        st = mp.mp_plan(L, K, sumsq, w, B, mask)
        m_gpu = mask.cpu().numpy().view(np.uint32)
        m_orc, st_orc = oracle.plan(blocks, dtype, K, S_orc, w, B)
        assert np.array_equal(m_gpu, m_orc), f"mask differs at B={B}"
        assert st["cost_bytes"] == st_orc["cost"] <= B
        assert st["n_selected"] == st_orc["n_selected"]
        assert st["full_bytes"] == st_orc["full_bytes"] == full
        assert st["digest"] == st_orc["digest"]
        assert st["n_units"] == G * K and st["budget_bytes"] == B
        if op == "avg":
            io = mp.mp_merge_avg(L, base, exps, mask, kw["alpha"], out, residency=res, io=True, delta=delta)
            want = oracle.merge_avg(blocks, dtype, base_np, exps_np, m_orc, kw["alpha"], delta=delta)
        elif op == "avg_renorm":
            io = mp.mp_merge_avg_renorm(L, base, exps, mask, kw["alpha"], out, residency=res, io=True, delta=delta)
            want = oracle.merge_avg_renorm(blocks, dtype, base_np, exps_np, m_orc, kw["alpha"], delta=delta)
        elif op == "ties":
            io = mp.mp_merge_ties(L, base, exps, mask, kw["density"], kw["lam"], out, residency=res, io=True,
                                  delta=delta)
            want = oracle.merge_ties(blocks, dtype, base_np, exps_np, m_orc, kw["density"], kw["lam"], delta=delta)
        elif op == "ties_tau":
            io = mp.mp_merge_ties_tau(L, base, exps, mask, tau, kw["lam"], out, residency=res, io=True, delta=delta)
            want = oracle.merge_ties(blocks, dtype, base_np, exps_np, m_orc, kw["density"], kw["lam"], delta=delta)
            # the in-merge trim gives the same bits
            out2 = torch.empty_like(base)
            mp.mp_merge_ties(L, base, exps, mask, kw["density"], kw["lam"], out2, residency=res, delta=delta)
            assert torch.equal(out.view(torch.int16) if out.dtype == torch.bfloat16 else out.view(torch.int32),
                               out2.view(torch.int16) if out2.dtype == torch.bfloat16 else out2.view(torch.int32))
        else:
            comb = 0 if op == "dare_lin" else 1
            io = mp.mp_merge_dare(L, base, exps, mask, kw["p"], kw["seed"], comb, kw.get("alpha"), kw["lam"],
                                  out, residency=res, io=True, delta=delta)
            want = oracle.merge_dare(blocks, dtype, base_np, exps_np, m_orc, kw["p"], kw["seed"], comb,
                                     kw.get("alpha", [1.0] * K), kw["lam"], delta=delta)
        got = to_host(out)
        nb = assert_merge_equal(got, want, base_np, dtype, f"{op} B={B}")
        assert nb == 0, f"{op} B={B}: {nb} values within tolerance but not bitwise equal"
        # the kernels read exactly the selected expert blocks (Prop. 1); TIES with
        # density 0 keeps nothing and reads no expert at all
        read = 0 if (op == "ties" and kw.get("density") == 0.0) else st["cost_bytes"]
        assert io["expert_bytes"] == read, "kernels loaded bytes outside the plan"
        if res == mp.MP_HOST_PINNED:  # only those blocks cross PCIe
            assert io["h2d_bytes"] == read
        elif res in (mp.MP_HOST_PAGEABLE, mp.MP_HOST_FILE):  # the staged copies are exactly the selected blocks
            assert io["h2d_bytes"] == st["cost_bytes"]
        else:
            assert io["h2d_bytes"] == 0
        results.append((B, st, nb))
        _say(f"  {spec.name} {op} B={B}: cost={st['cost_bytes']} sel={st['n_selected']} non-bitwise={nb}")
    return results


# ---------------------------------------------------------------- small families

@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_mini_qwen_bf16_all_ops(mp, op):
    spec = _mini_qwen()
    base, exps = make_family(spec, seed=1)
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
    _say(f"case mini-qwen bf16 {op}")
    _run_all(mp, spec, base, exps, op, [0, 0.1, 0.25, 0.5, 0.77, 1.0, 2.0, 12345], **kw)


@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_ragged_fp32_all_ops(mp, op):
    spec = _ragged_f32()
    base, exps = make_family(spec, seed=2)
    kw = dict(alpha=[0.5, 0.25, 0.25], density=0.1, lam=0.8, p=0.5, seed=3)
    _say(f"case ragged fp32 {op}")
    _run_all(mp, spec, base, exps, op, [0, 0.3, 0.6, 1.0], **kw)


@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_host_pinned_experts_all_ops(mp, op):
    # experts in pinned host memory: the kernels read the selected blocks
    # over PCIe; results are the same bits as with device-resident experts
    spec = _mini_qwen()
    base, exps = make_family(spec, seed=1)
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
    _say(f"case mini-qwen bf16 {op}, pinned host experts")
    _run_all(mp, spec, base, exps, op, [0, 0.3, 1.0], residency=mp.MP_HOST_PINNED, **kw)


def test_host_pinned_ragged_fp32_multi_group(mp):
    spec = _ragged_f32(K=6)
    base, exps = make_family(spec, K=6, seed=21)
    _say("case ragged fp32 K=6, pinned host experts")
    _run_all(mp, spec, base, exps, "ties", [0.5, 1.0], residency=mp.MP_HOST_PINNED, density=0.1, lam=0.8)
    _run_all(mp, spec, base, exps, "avg", [0.5], residency=mp.MP_HOST_PINNED, alpha=[1.0 / 6] * 6)


def test_host_pinned_rejects_device_and_pageable_experts(mp):
    import torch
    spec = _mini_qwen(n_layers=1)
    L, lay = _lay(mp, spec)
    base, exps = make_family(spec, seed=3)
    b = to_dev(base, "bf16")
    G = oracle.Blocks(lay.numel, lay.block_elems).G
    sumsq = torch.empty(G * 4, dtype=torch.float32, device="cuda")
    dev = [to_dev(e, "bf16") for e in exps]
    pageable = [torch.from_numpy(e.view(np.int16)).view(torch.bfloat16) for e in exps]
    for bad in (dev, pageable):
        with pytest.raises(mp.MPError) as err:
            mp.mp_index_blocks(L, b, bad, sumsq, residency=mp.MP_HOST_PINNED)
        assert err.value.code == mp.MP_E_ARG
    # exact-size pinned allocations one byte short of a checkpoint (torch's
    # pinned cache may hand out a larger block, which hides an undersized one)
    short = [_RawPinnedBuffer(e.nbytes - 1) for e in exps]
    try:
        with pytest.raises(mp.MPError) as err:
            mp.mp_index_blocks(L, b, short, sumsq, residency=mp.MP_HOST_PINNED)
        assert err.value.code == mp.MP_E_ARG
    finally:
        torch.cuda.synchronize()
        for x in short:
            x.free()


@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_host_pageable_experts_all_ops(mp, op):
    # experts in ordinary host memory: the selected blocks are packed into
    # pinned staging, copied to the device and merged chunk by chunk; same
    # bits as device-resident experts, and the staged bytes are the plan cost
    spec = _mini_qwen()
    base, exps = make_family(spec, seed=1)
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
    _say(f"case mini-qwen bf16 {op}, pageable host experts")
    _run_all(mp, spec, base, exps, op, [0, 0.3, 1.0], residency=mp.MP_HOST_PAGEABLE, **kw)


@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_host_file_experts_all_ops(mp, op):
    # experts in files (the paper's disk-resident regime): the selected
    # blocks are read with pread into pinned staging and merged from the
    # staged copy; same bits as device-resident experts, staged bytes == cost
    spec = _mini_qwen()
    base, exps = make_family(spec, seed=1)
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
    _say(f"case mini-qwen bf16 {op}, expert files")
    _run_all(mp, spec, base, exps, op, [0, 0.3, 1.0], residency=mp.MP_HOST_FILE, **kw)


def test_host_file_experts_small_staging_deltas_and_errors(mp):
    import torch
    mp.mp_set_stage_bytes(1 << 20)
    try:
        spec = _ragged_f32(K=3)
        base, exps = make_family(spec, seed=22)
        _say("case ragged fp32 expert files, 1 MiB staging, explicit deltas")
        _run_all(mp, spec, base, _as_deltas(base, exps, "f32"), "ties_tau", [0.2, 1.0], residency=mp.MP_HOST_FILE,
                 delta=True, density=0.3, lam=1.0)
    finally:
        mp.mp_set_stage_bytes(256 << 20)
    spec = _mini_qwen(n_layers=1)
    base_np, exps_np = make_family(spec, seed=23)
    L, lay = _lay(mp, spec)
    base = to_dev(base_np, lay.dtype)
    G = mp.mp_layout_blocks(L)
    sumsq = torch.empty(G * len(exps_np), dtype=torch.float32, device="cuda")
    paths = _expert_files(exps_np)
    with pytest.raises(mp.MPError) as e:
        mp.mp_index_blocks(L, base, paths[:-1] + [paths[-1] + ".missing"], sumsq, residency=mp.MP_HOST_FILE)
    assert e.value.code == mp.MP_E_IO
    with open(paths[0], "r+b") as f:  # one byte short of a checkpoint
        f.truncate(os.path.getsize(paths[0]) - 1)
    with pytest.raises(mp.MPError) as e:
        mp.mp_index_blocks(L, base, paths, sumsq, residency=mp.MP_HOST_FILE)
    assert e.value.code == mp.MP_E_ARG


def test_host_pageable_small_staging_many_chunks(mp):
    # 1 MiB staging buffers: the index (6.7 MB of experts) and the merges
    # cross many chunks, reusing both buffers several times; then ragged
    # fp32 blocks with K = 6 (groups of experts in the TIES kernel)
    mp.mp_set_stage_bytes(1 << 20)
    try:
        spec = _mini_qwen(n_layers=1)
        base, exps = make_family(spec, seed=4)
        kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
        for op in ("avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"):
            _say(f"case mini-qwen bf16 {op}, pageable host experts, 1 MiB staging")
            _run_all(mp, spec, base, exps, op, [0.1, 0.45, 1.0], residency=mp.MP_HOST_PAGEABLE, **kw)
        spec = _ragged_f32(K=6)
        base, exps = make_family(spec, K=6, seed=21)
        kw = dict(alpha=[1.0 / 6] * 6, density=0.3, lam=1.0, p=0.7, seed=11)
        for op in ("avg", "ties", "ties_tau", "dare_sign"):
            _say(f"case ragged fp32 K=6 {op}, pageable host experts, 1 MiB staging")
            _run_all(mp, spec, base, exps, op, [0.2, 0.65, 1.0], residency=mp.MP_HOST_PAGEABLE, **kw)
    finally:
        mp.mp_set_stage_bytes(256 << 20)


def test_host_pageable_rejects_device_experts_and_bad_staging(mp):
    import torch
    spec = _mini_qwen(n_layers=1)
    L, lay = _lay(mp, spec)
    base, exps = make_family(spec, seed=3)
    b = to_dev(base, "bf16")
    G = oracle.Blocks(lay.numel, lay.block_elems).G
    sumsq = torch.empty(G * 4, dtype=torch.float32, device="cuda")
    dev = [to_dev(e, "bf16") for e in exps]
    with pytest.raises(mp.MPError) as err:
        mp.mp_index_blocks(L, b, dev, sumsq, residency=mp.MP_HOST_PAGEABLE)
    assert err.value.code == mp.MP_E_ARG
    for n in (0, (1 << 20) - 1, (4 << 30) + 1):
        with pytest.raises(mp.MPError) as err:
            mp.mp_set_stage_bytes(n)
        assert err.value.code == mp.MP_E_ARG


def test_toy_config_avg_full_parity(mp):
    # the toy family: fp32 8 x (512x1024), K=4, AVG 1/K, B = 50%
    spec = family_spec("toy")
    base, exps = make_family(spec, seed=0)
    _say("case toy fp32 avg")
    _run_all(mp, spec, base, exps, "avg", [0.5, 0.25, 1.0], alpha=[0.25] * 4)


@pytest.mark.parametrize("K", [1, 2, 7, 32])
def test_expert_counts(mp, K):
    spec = _mini_qwen(n_layers=1, K=K)
    base, exps = make_family(spec, K=K, seed=10 + K)
    _say(f"case mini-qwen K={K}")
    _run_all(mp, spec, base, exps, "ties", [0.0, 0.4, 1.0], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "ties_tau", [0.4, 1.0], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "avg", [0.4], alpha=[1.0 / K] * K)
    _run_all(mp, spec, base, exps, "avg_renorm", [0.4, 1.0], alpha=[1.0 / K] * K)


@pytest.mark.parametrize("be", [1024, 2048, 512])
def test_block_sizes(mp, be):
    spec = _mini_qwen(n_layers=1, be=be)
    base, exps = make_family(spec, seed=4)
    _say(f"case block_elems={be}")
    _run_all(mp, spec, base, exps, "ties", [0.35, 1.0], density=0.3, lam=1.0)
    _run_all(mp, spec, base, exps, "ties_tau", [0.35, 1.0], density=0.3, lam=1.0)
    _run_all(mp, spec, base, exps, "dare_lin", [0.5], alpha=[0.3, 0.2, 0.4, 0.1], p=0.3, seed=11, lam=1.0)


@pytest.mark.parametrize("be", [1028, 4100])
def test_dare_fp32_blocks_starting_mid_draw(mp, be):
    # fp32 blocks of be = 4 (mod 8) elements: every other block of a tensor
    # starts in the middle of a Philox draw (eight elements per draw), so its
    # chunks take the draw's upper two words
    t = (("a", (3 * 4100 + 8,)), ("b", (12,)), ("c", (5000,)), ("d", (4, 1025)))
    spec = FamilySpec("fp32-mid-draw", t, "f32", be, 3, ())
    base, exps = make_family(spec, seed=5)
    _say(f"case fp32 DARE block_elems={be}")
    for op in ("dare_lin", "dare_sign"):
        _run_all(mp, spec, base, exps, op, [0.4, 1.0], alpha=[0.5, 0.25, 0.25], p=0.7, seed=13, lam=0.9)


def _as_deltas(base_np, exps_np, dtype):
    """Explicit-delta experts of a family: fl32(W_i - W_0) in the checkpoint
    dtype (any arrays of that dtype are valid deltas)."""
    if dtype == "f32":
        return [(e - base_np).astype(np.float32) for e in exps_np]
    f = lambda u: (u.astype(np.uint32) << 16).view(np.float32)
    return [oracle.round_bf16(f(e) - f(base_np)) for e in exps_np]


@pytest.mark.parametrize("op", ["avg", "avg_renorm", "ties", "ties_tau", "dare_lin", "dare_sign"])
def test_explicit_delta_experts_all_ops(mp, op):
    # experts given as stored deltas (MP_EXPERTS_DELTA): the index reads no
    # base, the merges add the merged delta to the base; bf16 and ragged fp32
    spec = _mini_qwen()
    base, exps = make_family(spec, seed=1)
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0, p=0.9, seed=7)
    _say(f"case mini-qwen bf16 {op}, explicit deltas")
    _run_all(mp, spec, base, _as_deltas(base, exps, "bf16"), op, [0, 0.3, 0.7, 1.0], delta=True, **kw)
    spec = _ragged_f32()
    base, exps = make_family(spec, seed=2)
    kw = dict(alpha=[0.5, 0.25, 0.25], density=0.1, lam=0.8, p=0.5, seed=3)
    _say(f"case ragged fp32 {op}, explicit deltas")
    _run_all(mp, spec, base, _as_deltas(base, exps, "f32"), op, [0.3, 1.0], delta=True, **kw)


def test_explicit_delta_experts_on_the_host(mp):
    # the delta flag combined with both host feeds
    spec = _mini_qwen(n_layers=1)
    base, exps = make_family(spec, seed=9)
    d = _as_deltas(base, exps, "bf16")
    kw = dict(alpha=[0.25] * 4, density=0.2, lam=1.0)
    for res in (mp.MP_HOST_PINNED, mp.MP_HOST_PAGEABLE):
        for op in ("avg", "ties_tau"):
            _say(f"case explicit deltas, residency {res}, {op}")
            _run_all(mp, spec, base, d, op, [0.4, 1.0], residency=res, delta=True, **kw)


def test_manifest_coverage_realized_reads_and_replay(mp):
    # Section 3's run record: mp_coverage equals the mask's touched elements
    # per (tensor, expert) by definition; the in-kernel per-expert read
    # counters equal the coverage bytes (N^run = A) on every feed; the plan
    # replays to the recorded digest and a tampered budget does not.
    import json
    import torch
    from paper_2605_29489_amd.manifest import build_manifest, dumps, replay
    spec = _mini_qwen(n_layers=1)
    base_np, exps_np = make_family(spec, seed=13)
    L, lay = _lay(mp, spec)
    K = len(exps_np)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    base = to_dev(base_np, lay.dtype)
    sumsq = torch.empty(blocks.G * K, dtype=torch.float32, device="cuda")
    mask = torch.empty(blocks.G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = int(blocks.len.sum()) * lay.elem_bytes * K
    for res in (mp.MP_DEVICE, mp.MP_HOST_PINNED, mp.MP_HOST_PAGEABLE):
        if res == mp.MP_HOST_PINNED:
            exps = [to_pinned(e, lay.dtype) for e in exps_np]
        elif res == mp.MP_HOST_PAGEABLE:
            exps = [torch.from_numpy(e) for e in exps_np]
        else:
            exps = [to_dev(e, lay.dtype) for e in exps_np]
        _say(f"case manifest, residency {res}")
        mp.mp_index_blocks(L, base, exps, sumsq, residency=res)
        st = mp.mp_plan(L, K, sumsq, [0.25] * K, int(0.37 * full), mask)
        io = mp.mp_merge_avg(L, base, exps, mask, [0.25] * K, out, residency=res, io=True)
        cov = mp.mp_coverage(L, K, mask)
        m_np = mask.cpu().numpy().view(np.uint32)
        want = np.zeros((len(lay.numel), K), np.uint64)
        for g in range(blocks.G):
            for i in range(K):
                if (m_np[g] >> i) & 1:
                    want[blocks.tensor[g], i] += blocks.len[g]
        assert np.array_equal(cov, want)
        assert [int(x) for x in io["expert_bytes_by_expert"][:K]] == [int(c) * lay.elem_bytes for c in want.sum(0)]
        assert all(x == 0 for x in io["expert_bytes_by_expert"][K:])
        man = build_manifest(L, K, st, io, cov, "avg", {"alpha": [0.25] * K},
                             tensor_names=[n for n, _ in spec.tensors], inputs={"family": spec.name, "seed": 13})
        assert man["realized"]["within_plan"] and man["realized"]["matches_coverage"]
        man = json.loads(dumps(man))
        assert replay(man, mp, L, K, sumsq, [0.25] * K, mask)["ok"]
        bad = json.loads(dumps(man))
        bad["plan"]["budget_bytes"] = int(0.5 * full)
        assert not replay(bad, mp, L, K, sumsq, [0.25] * K, mask)["ok"]


def _tensor_ties_case(mp, spec, base_np, exps_np, budgets, density, lam, residency=None, delta=False):
    """Tensor-scope TIES: per-unit thresholds from mp_ties_tensor_thresholds
    for each plan's mask, then the threshold merge; both against the oracle."""
    import torch
    L, lay = _lay(mp, spec)
    K = len(exps_np)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    res = mp.MP_DEVICE if residency is None else residency
    base = to_dev(base_np, lay.dtype)
    exps = [to_pinned(e, lay.dtype) for e in exps_np] if res == mp.MP_HOST_PINNED else \
        [to_dev(e, lay.dtype) for e in exps_np]
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq, residency=res, delta=delta)
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = int(blocks.len.sum()) * lay.elem_bytes * K
    for f in budgets:
        st = mp.mp_plan(L, K, sumsq, [1.0] * K, int(f * full), mask)
        mp.mp_ties_tensor_thresholds(L, base, exps, mask, density, tau, residency=res, delta=delta)
        m_np = mask.cpu().numpy().view(np.uint32)
        t_orc = oracle.expand_tensor_thresholds(
            blocks, oracle.ties_tensor_thresholds(blocks, lay.dtype, base_np, exps_np, m_np, density, delta=delta))
        assert np.array_equal(tau.cpu().numpy().view(np.uint32), t_orc), f"thresholds differ at B={f}"
        io = mp.mp_merge_ties_tau(L, base, exps, mask, tau, lam, out, residency=res, io=True, delta=delta)
        want = oracle.merge_ties_tau(blocks, lay.dtype, base_np, exps_np, m_np, t_orc, lam, delta=delta)
        nb = assert_merge_equal(to_host(out), want, base_np, lay.dtype, f"tensor TIES B={f}")
        assert nb == 0
        assert io["expert_bytes"] == st["cost_bytes"]
        _say(f"  {spec.name} tensor TIES rho={density} B={f}: sel={st['n_selected']}")


def test_ties_tensor_scope(mp):
    # the per-tensor trim: every density edge, both dtypes, heavy tails
    spec = _mini_qwen(n_layers=2)
    base, exps = make_family(spec, seed=31)
    for dens in (0.2, 0.05, 1.0, 0.0, 1.0 / 4096):
        _say(f"case tensor-scope TIES mini-qwen bf16 rho={dens}")
        _tensor_ties_case(mp, spec, base, exps, [0.0, 0.15, 0.5, 1.0], dens, 1.0)
    spec = _ragged_f32(K=3)
    base, exps = make_family(spec, seed=32)
    _say("case tensor-scope TIES ragged fp32")
    _tensor_ties_case(mp, spec, base, exps, [0.3, 1.0], 0.3, 0.8)
    spec = _mini_qwen(n_layers=1, K=2)
    P = sum(int(np.prod(s)) for _, s in spec.tensors)
    rng = np.random.default_rng(33)
    b0 = oracle.round_bf16(rng.normal(0.0, 0.02, P).astype(np.float32))
    heavy = rng.normal(0.0, 1e-4, P)
    out_idx = rng.random(P) < 0.01
    heavy[out_idx] = rng.normal(0.0, 1.0, int(out_idx.sum()))
    ex = _bf16_family_from_deltas(b0, [heavy, rng.normal(0.0, 1e-3, P)])
    _say("case tensor-scope TIES heavy tails")
    _tensor_ties_case(mp, spec, b0, ex, [0.4, 1.0], 0.1, 1.0)


def test_ties_tensor_scope_deltas_and_pinned(mp):
    spec = _mini_qwen(n_layers=1)
    base, exps = make_family(spec, seed=34)
    _say("case tensor-scope TIES explicit deltas")
    _tensor_ties_case(mp, spec, base, _as_deltas(base, exps, "bf16"), [0.3, 1.0], 0.2, 1.0, delta=True)
    _say("case tensor-scope TIES pinned experts")
    _tensor_ties_case(mp, spec, base, exps, [0.3, 1.0], 0.2, 1.0, residency=mp.MP_HOST_PINNED)


def test_avg_renorm_coefficients(mp):
    # Selected-only AVG with unequal, non-dyadic coefficients (the quotients
    # alpha_i / s are inexact) and a zero coefficient: blocks whose only
    # selected expert has alpha 0 sum to s = 0 and keep the base.
    spec = _mini_qwen(n_layers=1)
    base, exps = make_family(spec, seed=6)
    _say("case avg_renorm coefficients")
    _run_all(mp, spec, base, exps, "avg_renorm", [0.0, 0.2, 0.55, 1.0], w=[1.0, 0.9, 0.8, 0.7],
             alpha=[0.3, 0.0, 0.11, 1.9])
    spec = _ragged_f32(K=3)
    base, exps = make_family(spec, seed=8)
    _run_all(mp, spec, base, exps, "avg_renorm", [0.15, 0.5, 1.0], alpha=[0.2, 0.7, 0.1])


def test_large_blocks_avg_dare_and_ties_unsupported(mp):
    import torch
    spec = _mini_qwen(n_layers=1, be=8192)
    base, exps = make_family(spec, seed=5)
    _say("case block_elems=8192")
    _run_all(mp, spec, base, exps, "avg", [0.5], alpha=[0.25] * 4)
    _run_all(mp, spec, base, exps, "dare_sign", [0.5], p=0.2, seed=1, lam=1.0)
    L, lay = _lay(mp, spec)
    b = to_dev(base, "bf16")
    e = [to_dev(x, "bf16") for x in exps]
    mask = torch.zeros(oracle.Blocks(lay.numel, 8192).G, dtype=torch.int32, device="cuda")
    with pytest.raises(mp.MPError) as err:
        mp.mp_merge_ties(L, b, e, mask, 0.2, 1.0, torch.empty_like(b))
    assert err.value.code == mp.MP_E_UNSUPPORTED


def test_ties_and_zero_and_identical_experts(mp):
    # identical experts -> exact score ties (tie-break on uid); an all-zero
    # expert -> zero scores; heavy value ties inside blocks (coarse deltas)
    spec = _mini_qwen(n_layers=1, K=4)
    base, exps = make_family(spec, seed=6)
    exps = [exps[0], exps[0].copy(), base.copy(), exps[1]]
    _say("case identical/zero experts")
    _run_all(mp, spec, base, exps, "ties", [0.1, 0.3, 0.5, 0.74, 0.75, 0.76, 1.0], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "avg", [0.3, 0.6], alpha=[0.25] * 4)
    coarse = [base.copy() for _ in range(3)]
    rng = np.random.default_rng(0)
    for c in coarse:
        sel = rng.random(c.size) < 0.5
        c[sel] = (c[sel].astype(np.int32) + rng.integers(-2, 3, int(sel.sum()))).astype(np.uint16)
    _say("case coarse ties")
    _run_all(mp, spec, base, coarse, "ties", [0.5, 1.0], density=0.15, lam=1.0)
    _run_all(mp, spec, base, coarse, "ties_tau", [0.5, 1.0], density=0.15, lam=1.0)


def _bf16_family_from_deltas(base_np, deltas):
    """Experts W_i = bf16(fl32(W0 + d_i)) for the given fp32 deltas."""
    x0 = (base_np.astype(np.uint32) << 16).view(np.float32)
    return [oracle.round_bf16((x0 + d.astype(np.float32)).astype(np.float32)) for d in deltas]


def test_ties_threshold_search_paths(mp):
    # Delta distributions that drive every branch of the trim-threshold
    # search: uniform magnitudes (the k-th largest lies in the binade of the
    # block maximum), rare huge outliers (it lies far below the max), mostly
    # unchanged weights (fewer than k nonzero deltas: everything nonzero is
    # kept), bucket-dense values with distinct low bits, and densities that
    # give k = 1 and k = n.
    spec = _mini_qwen(n_layers=1, K=4)
    base, _ = make_family(spec, seed=12)
    P = base.size
    rng = np.random.default_rng(12)
    uni = rng.uniform(-0.01, 0.01, P)
    heavy = rng.normal(0.0, 1e-4, P)
    out_idx = rng.random(P) < 0.01
    heavy[out_idx] = rng.normal(0.0, 1.0, int(out_idx.sum()))
    sparse = np.where(rng.random(P) < 0.1, rng.normal(0.0, 1e-3, P), 0.0)
    dense = 1e-3 * (1.0 + rng.integers(0, 4, P) / 64.0) * np.sign(rng.normal(size=P))
    exps = _bf16_family_from_deltas(base, [uni, heavy, sparse, dense])
    for dens in (0.2, 0.05, 1.0 / 4096, 1.0, 0.0):
        _say(f"case threshold paths density={dens}")
        _run_all(mp, spec, base, exps, "ties", [0.5, 1.0], density=dens, lam=1.0)
        _run_all(mp, spec, base, exps, "ties_tau", [0.5, 1.0], density=dens, lam=1.0)


def test_ties_threshold_guess_above_tau(mp):
    # Both TIES selectors (the catalog's and the one inside the merge) first
    # count only values above a guess taken from the deltas' RMS.  Bimodal
    # deltas (a tenth near 1.0, the rest in [0.13, 0.2]) put that guess above
    # the k-th largest at density 0.2 while the k-th largest still lies in
    # the window below the maximum: the rest of the window must be counted
    # and the cut found there.  A normal expert takes the first pass.
    spec = _mini_qwen(n_layers=1, K=2)
    P = sum(int(np.prod(s)) for _, s in spec.tensors)
    rng = np.random.default_rng(19)
    base = oracle.round_bf16(rng.normal(0.0, 0.02, P).astype(np.float32))
    big = rng.random(P) < 0.1
    mag = np.where(big, rng.uniform(0.9, 1.1, P), rng.uniform(0.13, 0.2, P))
    bimodal = mag * np.sign(rng.normal(size=P))
    exps = _bf16_family_from_deltas(base, [bimodal, rng.normal(0.0, 0.01, P)])
    for dens in (0.2, 0.12, 0.5):
        _say(f"case guess above tau density={dens}")
        _run_all(mp, spec, base, exps, "ties_tau", [1.0], density=dens, lam=1.0)
        _run_all(mp, spec, base, exps, "ties", [0.5, 1.0], density=dens, lam=1.0)


def test_ties_subnormal_deltas(mp):
    # base weights near the bottom of the normal range, deltas subnormal in
    # fp32: the magnitude patterns and the keep test must treat them exactly
    spec = _mini_qwen(n_layers=1, K=3)
    P = sum(int(np.prod(s)) for _, s in spec.tensors)
    rng = np.random.default_rng(13)
    base = oracle.round_bf16(rng.normal(0.0, 2e-38, P).astype(np.float32))
    deltas = [rng.normal(0.0, s, P) for s in (1e-39, 5e-39, 3e-40)]
    exps = _bf16_family_from_deltas(base, deltas)
    _say("case subnormal deltas")
    _run_all(mp, spec, base, exps, "ties", [0.4, 1.0], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "ties_tau", [0.4, 1.0], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "ties", [1.0], density=0.3, lam=0.5)


def test_ties_infinite_masses(mp):
    # deltas near the top of the fp32 range, some infinite: kept masses of
    # several entries overflow, and the mean must be IEEE's (inf / count is
    # inf) in both TIES paths; density 0 keeps none of them
    spec = _mini_qwen(n_layers=1, K=4)
    P = sum(int(np.prod(s)) for _, s in spec.tensors)
    rng = np.random.default_rng(17)
    base = oracle.round_bf16(rng.normal(0.0, 1e36, P).astype(np.float32))
    deltas = [np.clip(rng.normal(0.0, s, P), -3e38, 3e38) for s in (1.2e38, 1.5e38, 1.0e38, 1.3e38)]
    exps = _bf16_family_from_deltas(base, deltas)
    for i, e in enumerate(exps):
        e[rng.choice(P, 40, replace=False)] = np.uint16(0x7F80 if i % 2 == 0 else 0xFF80)
    _say("case infinite masses")
    _run_all(mp, spec, base, exps, "ties", [1.0, 0.6], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "ties_tau", [1.0, 0.6], density=0.2, lam=1.0)
    _run_all(mp, spec, base, exps, "ties_tau", [1.0], density=0.0, lam=1.0)


def _near_cancellation_deltas(rng, P, K, dt):
    """Explicit deltas where most elements hold, over three of the experts,
    an order of (a, -a, +-a * 2^-25), (a, -a, a * 2^-23) or (a, -a, a * 2^-24)
    (a with a 3-bit mantissa, so every value is exact in bf16); the rest are
    normal.  With K = 5 the triple sits on experts 0-2 for even elements and
    on experts 2-4 for odd ones; the other experts hold zeros there."""
    a = np.ldexp(1.0 + rng.integers(0, 8, P) / 8.0, rng.integers(-12, -4, P)) * rng.choice([-1.0, 1.0], P)
    small = a * np.ldexp(1.0, rng.choice([-25, -25, -25, -23, -24], P)) * rng.choice([-1.0, 1.0], P)
    trip = np.stack([a, -a, small])  # [3, P]
    order = np.argsort(rng.random((3, P)), axis=0)
    trip = np.take_along_axis(trip, order, axis=0)
    D = np.zeros((K, P))
    first = np.where((np.arange(P) % 2 == 1) & (K >= 5), 2, 0)
    for r in range(3):
        D[first + r, np.arange(P)] = trip[r]
    normal = rng.random(P) < 0.3
    D[:, normal] = rng.normal(0.0, 1e-3, (K, int(normal.sum())))
    if dt == "bf16":
        return [oracle.round_bf16(d.astype(np.float32)) for d in D]
    return [d.astype(np.float32) for d in D]


@pytest.mark.parametrize("dt,K", [("bf16", 3), ("f32", 5)])
def test_ties_election_near_cancellation(mp, dt, K):
    # The election compares the rounded one-signed masses fl32(P) and
    # -fl32(N): for kept (a, -a, a * 2^-25) it elects nothing, although the
    # exact mass is nonzero.  Both TIES routes and DARE's sign-elect combine
    # match the oracle bit for bit on families built from such triples (the
    # deltas are explicit, so they reach the kernels exactly).
    spec = _mini_qwen(n_layers=1, K=K) if dt == "bf16" else _ragged_f32(K=K)
    P = sum(int(np.prod(s)) for _, s in spec.tensors)
    rng = np.random.default_rng(29)
    base = rng.normal(0.0, 0.02, P).astype(np.float32)
    base = oracle.round_bf16(base) if dt == "bf16" else base
    deltas = _near_cancellation_deltas(rng, P, K, dt)
    # the data reach the discriminating case: at density 1 and a full mask,
    # elements whose exact kept mass is nonzero but elect no sign
    lay = spec.layout
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    full = np.full(blocks.G, (1 << K) - 1, np.uint32)
    zero_base = np.zeros_like(base)
    out0 = oracle.merge_ties(blocks, dt, zero_base, deltas, full, 1.0, 1.0, delta=True)
    D = np.stack([oracle_f32(d, dt) for d in deltas]).astype(np.float64)
    hidden = (oracle_f32(out0, dt) == 0) & (D.sum(0) != 0)
    _say(f"case election near cancellation {dt} K={K}: {int(hidden.sum())} of {P} elements elect none "
         f"with a nonzero exact mass")
    assert hidden.sum() > P // 10
    for dens in (1.0, 0.5):
        _run_all(mp, spec, base, deltas, "ties", [1.0, 0.5], density=dens, lam=1.0, delta=True)
        _run_all(mp, spec, base, deltas, "ties_tau", [1.0, 0.5], density=dens, lam=1.0, delta=True)
    for p in (0.0, 0.3):
        _run_all(mp, spec, base, deltas, "dare_sign", [1.0, 0.5], p=p, seed=7, lam=1.0, delta=True)


def oracle_f32(a, dt):
    """fp32 values of a checkpoint array (bf16 patterns widened exactly)."""
    if dt == "bf16":
        return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32)
    return np.asarray(a, np.float32)


def test_skip_zero_full_budget_merges_equal_full_merges(mp):
    # With the skip-zero option, units whose block equals the base (S = 0:
    # the family's untouched blocks) are never selected; at full budget every
    # merge operator still gives the full merge bit for bit, and reads
    # exactly the nonzero units' bytes.
    import torch
    spec = _mini_qwen(K=4)
    base_np, exps_np = make_family(spec, seed=5)
    L, lay = _lay(mp, spec)
    K = len(exps_np)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    base = to_dev(base_np, lay.dtype)
    exps = [to_dev(e, lay.dtype) for e in exps_np]
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq)
    S = sumsq.cpu().numpy()
    assert (S == 0).sum() > 0, "the family has untouched blocks"
    full = int(blocks.len.sum()) * lay.elem_bytes * K
    m_all = torch.empty(G, dtype=torch.int32, device="cuda")
    m_nz = torch.empty(G, dtype=torch.int32, device="cuda")
    mp.mp_plan(L, K, sumsq, [1.0] * K, full, m_all)
    st = mp.mp_plan(L, K, sumsq, [1.0] * K, full, m_nz, flags=mp.MP_PLAN_SKIP_ZERO)
    nz_cost = sum(int(blocks.len[u // K]) * lay.elem_bytes for u in np.nonzero(S != 0)[0])
    assert st["cost_bytes"] == nz_cost and st["n_selected"] == int((S != 0).sum())
    _say("case skip-zero at full budget")
    o1, o2 = torch.empty_like(base), torch.empty_like(base)
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    mp.mp_index_ties(L, base, exps, 0.2, tau)
    runs = [
        lambda m, o: mp.mp_merge_avg(L, base, exps, m, [0.25] * K, o, io=True),
        lambda m, o: mp.mp_merge_ties(L, base, exps, m, 0.2, 1.0, o, io=True),
        lambda m, o: mp.mp_merge_ties_tau(L, base, exps, m, tau, 1.0, o, io=True),
        lambda m, o: mp.mp_merge_dare(L, base, exps, m, 0.9, 7, 0, [0.25] * K, 1.0, o, io=True),
        lambda m, o: mp.mp_merge_dare(L, base, exps, m, 0.9, 7, 1, None, 1.0, o, io=True),
    ]
    for run in runs:
        run(m_all, o1)
        io = run(m_nz, o2)
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
        assert io["expert_bytes"] == nz_cost


def test_plan_many_rounds(mp):
    # Many distinct block lengths, scores with deliberate ties (equal sums
    # of squares, equal weights) and zero scores: after the first cut, the
    # cheaper candidates above it are planned in later rounds.  Mask, cost,
    # count and digest match the oracle's literal sort + greedy at every
    # budget, including budgets where many rounds remain.
    import torch
    numel = [4096 * 3 + 64, 4096 + 512, 2048, 1024 + 256, 4096 * 2 + 1536, 768, 4096, 384, 128, 4096 + 2560]
    L = mp.Layout(numel, 4096, mp.MP_BF16)
    blocks = oracle.Blocks(numel, 4096)
    K = 5
    G = blocks.G
    rng = np.random.default_rng(23)
    S = rng.choice(np.array([0.0, 1e-4, 2.5e-3, 2.5e-3, 7e-2, 1.0, 3.0], np.float32), size=G * K)
    S = (S * rng.choice(np.array([1.0, 1.0, 0.5], np.float32), size=G * K)).astype(np.float32)
    sumsq = torch.from_numpy(S).cuda()
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    full = int(blocks.len.sum()) * 2 * K
    lens = sorted(set(int(x) for x in blocks.len))
    assert len(lens) >= 8
    _say(f"case plan rounds: G={G}, {len(lens)} distinct lengths")
    budgets = sorted(set([0, 1, 127, 128, 129, full // 7, full // 3, full // 2, full - 1, full, full + 5]
                         + [int(x) for x in rng.integers(0, full, 40)]))
    # flags: 0 literal, 1 per-byte scores, 2 skip zero units, 3 both
    for flags in (0, mp.MP_PLAN_PER_BYTE, mp.MP_PLAN_SKIP_ZERO, mp.MP_PLAN_PER_BYTE | mp.MP_PLAN_SKIP_ZERO):
        for w in ([1.0] * K, [0.5, 1.0, 1.0, 0.25, 2.0]):
            for B in budgets:
                st = mp.mp_plan(L, K, sumsq, w, B, mask, flags=flags)
                m_orc, st_orc = oracle.plan(blocks, "bf16", K, S, w, B, flags=flags)
                assert np.array_equal(mask.cpu().numpy().view(np.uint32), m_orc), \
                    f"mask differs at B={B} w={w} flags={flags}"
                assert st["cost_bytes"] == st_orc["cost"] <= B
                assert st["n_selected"] == st_orc["n_selected"]
                assert st["digest"] == st_orc["digest"]
                assert st["full_bytes"] == st_orc["full_bytes"] and st["n_units"] == G * K


def _assert_tensor_plan(mp, L, blocks, dtype, K, w, B, flags, mask):
    st = mp.mp_plan(L, K, None, w, B, mask, flags=flags)
    m = mask.cpu().numpy().view(np.uint32)
    m_orc, st_orc = oracle.plan(blocks, dtype, K, None, w, B, flags=flags)
    assert np.array_equal(m, m_orc), f"tensor-level mask differs at B={B} w={w} flags={flags}"
    assert st["cost_bytes"] == st_orc["cost"] <= B and st["n_selected"] == st_orc["n_selected"]
    assert st["digest"] == st_orc["digest"] and st["full_bytes"] == st_orc["full_bytes"]
    assert st["n_units"] == blocks.G * K
    # no tensor is split: every block of a tensor carries the same word
    first = np.concatenate([[True], blocks.tensor[1:] != blocks.tensor[:-1]])
    starts = np.nonzero(first)[0]
    word = np.repeat(m[starts], np.diff(np.concatenate([starts, [blocks.G]])))
    assert np.array_equal(m, word)
    return st


def test_plan_without_catalog(mp):
    # no block catalog (sumsq NULL): Section 3's tensor-level plan, bit-exact
    # against the oracle at every budget, weight vector and flag, no tensor
    # split; then a merge over that mask
    import torch
    spec = _mini_qwen(n_layers=2)
    base_np, exps_np = make_family(spec, seed=35)
    L, lay = _lay(mp, spec)
    K = len(exps_np)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    mask = torch.empty(blocks.G, dtype=torch.int32, device="cuda")
    full = int(blocks.len.sum()) * lay.elem_bytes * K
    rng = np.random.default_rng(36)
    budgets = sorted(set([0, 1, full // 3, full // 2, full - 1, full, full + 7] +
                         [int(x) for x in rng.integers(0, full, 12)]))
    for flags in (0, mp.MP_PLAN_PER_BYTE, mp.MP_PLAN_SKIP_ZERO):
        for w in ([1.0] * K, [0.5, 2.0, 1.0, 1.5]):
            for B in budgets:
                _assert_tensor_plan(mp, L, blocks, lay.dtype, K, w, B, flags, mask)
    _say(f"  tensor-level plans: {len(budgets)} budgets x 2 weights x 3 flags equal")
    B = int(0.4 * full)
    _assert_tensor_plan(mp, L, blocks, lay.dtype, K, [1.0] * K, B, 0, mask)
    m_orc, _ = oracle.plan(blocks, lay.dtype, K, None, [1.0] * K, B)
    base = to_dev(base_np, lay.dtype)
    exps = [to_dev(e, lay.dtype) for e in exps_np]
    out = torch.empty_like(base)
    mp.mp_merge_ties(L, base, exps, mask, 0.2, 1.0, out)
    want = oracle.merge_ties(blocks, lay.dtype, base_np, exps_np, m_orc, 0.2, 1.0)
    assert assert_merge_equal(to_host(out), want, base_np, lay.dtype, "ties without catalog") == 0


@pytest.mark.parametrize("name,K", [("qwen2.5-1.5b", 4), ("llama3-8b", 16)])
def test_plan_without_catalog_full_layouts(mp, name, K):
    # the tensor-level plan on the full tensor lists (338 and 291 tensors,
    # many distinct sizes, hence many plan rounds), against the oracle
    import torch
    lay = family_spec(name).layout
    L = mp.Layout(lay.numel, lay.block_elems, mp.MP_BF16)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    mask = torch.empty(blocks.G, dtype=torch.int32, device="cuda")
    full = lay.n_params * 2 * K
    rng = np.random.default_rng(37)
    w = [float(x) for x in rng.choice([0.25, 0.5, 1.0], K)]
    for flags in (0, mp.MP_PLAN_PER_BYTE):
        for f in (1.0 / K, 0.1, 0.25, 0.5, 0.77, 1.0):
            _assert_tensor_plan(mp, L, blocks, "bf16", K, w, int(f * full), flags, mask)
    _say(f"  {name} K={K}: tensor-level plans equal")


def test_budget_boundaries_exact(mp):
    # budgets at the exact cost of a greedy prefix, one byte below and above
    spec = _mini_qwen(n_layers=1)
    base, exps = make_family(spec, seed=8)
    lay = spec.layout
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    S = oracle.index(blocks, "bf16", base, exps).reshape(-1)
    _, st = oracle.plan(blocks, "bf16", 4, S, [1.0] * 4, int(0.37 * int(blocks.len.sum()) * 8))
    c = st["cost"]
    _say("case budget boundaries")
    _run_all(mp, spec, base, exps, "ties", [c - 1, c, c + 1, 1, 511, 512, 513], density=0.2, lam=1.0)


def test_empty_layout(mp):
    import torch
    L = mp.Layout([], 4096, mp.MP_BF16)
    base = torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    exps = [torch.zeros(8, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    sumsq = torch.zeros(1, dtype=torch.float32, device="cuda")
    mask = torch.zeros(1, dtype=torch.int32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq)
    st = mp.mp_plan(L, 2, sumsq, [1.0, 1.0], 100, mask)
    assert st["cost_bytes"] == 0 and st["n_units"] == 0 and st["n_selected"] == 0
    assert st["digest"] == oracle.mix64(0)
    mp.mp_merge_ties(L, base, exps, mask, 0.2, 1.0, torch.empty_like(base))


def test_non_anticipation_and_determinism(mp):
    # P3: changing unselected expert blocks leaves the output bitwise unchanged;
    # two runs are bit-identical.
    import torch
    spec = _mini_qwen(n_layers=1)
    base_np, exps_np = make_family(spec, seed=9)
    L, lay = _lay(mp, spec)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    base = to_dev(base_np, "bf16")
    exps = [to_dev(e, "bf16") for e in exps_np]
    sumsq = torch.empty(blocks.G * 4, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq)
    mask = torch.empty(blocks.G, dtype=torch.int32, device="cuda")
    full = int(blocks.len.sum()) * 2 * 4
    mp.mp_plan(L, 4, sumsq, [1.0] * 4, full // 3, mask)
    m = mask.cpu().numpy().view(np.uint32)
    outs = {}
    for op in ("ties", "avg", "dare_sign"):
        o1, o2 = torch.empty_like(base), torch.empty_like(base)
        run = {
            "ties": lambda ex, o: mp.mp_merge_ties(L, base, ex, mask, 0.2, 1.0, o),
            "avg": lambda ex, o: mp.mp_merge_avg(L, base, ex, mask, [0.25] * 4, o),
            "dare_sign": lambda ex, o: mp.mp_merge_dare(L, base, ex, mask, 0.9, 7, 1, None, 1.0, o),
        }[op]
        run(exps, o1)
        junk = [e.clone() for e in exps]
        for i in range(4):
            for g in np.nonzero(((m >> i) & 1) == 0)[0]:
                junk[i][blocks.off[g]:blocks.off[g] + blocks.len[g]] = 7.0
        run(junk, o2)
        o3 = torch.empty_like(base)
        run(exps, o3)
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), op
        assert torch.equal(o1.view(torch.int16), o3.view(torch.int16)), op


class _RawDeviceBuffer:
    """An exact-size hipMalloc allocation (torch's caching allocator may hand
    out a slice of a larger segment, which hides an undersized buffer)."""

    def __init__(self, nbytes):
        import ctypes
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._p = ctypes.c_void_p()
        assert self._hip.hipMalloc(ctypes.byref(self._p), ctypes.c_size_t(nbytes)) == 0
        self.nbytes = nbytes

    def data_ptr(self):
        return self._p.value

    def free(self):
        self._hip.hipFree(self._p)


class _RawPinnedBuffer:
    """An exact-size hipHostMalloc allocation."""

    def __init__(self, nbytes):
        import ctypes
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._p = ctypes.c_void_p()
        assert self._hip.hipHostMalloc(ctypes.byref(self._p), ctypes.c_size_t(nbytes), ctypes.c_uint(0)) == 0
        self.nbytes = nbytes

    def data_ptr(self):
        return self._p.value

    def free(self):
        self._hip.hipHostFree(self._p)


def test_invalid_device_arguments_rejected(mp):
    import torch
    spec = _mini_qwen(n_layers=1)
    L, lay = _lay(mp, spec)
    P = lay.n_params
    base = torch.zeros(P, dtype=torch.bfloat16, device="cuda")
    exps = [torch.zeros(P, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    G = oracle.Blocks(lay.numel, lay.block_elems).G
    mask = torch.zeros(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    host = torch.zeros(P, dtype=torch.bfloat16)
    with pytest.raises(mp.MPError):  # host buffer where device memory is required
        mp.mp_merge_avg(L, host, exps, mask, [0.5, 0.5], out)
    with pytest.raises(mp.MPError):  # output aliases an expert
        mp.mp_merge_avg(L, base, exps, mask, [0.5, 0.5], exps[1])
    with pytest.raises(mp.MPError):  # pageable host expert with MP_HOST_PINNED
        mp.mp_merge_avg(L, base, [host, host], mask, [0.5, 0.5], out, residency=mp.MP_HOST_PINNED)
    small_out = _RawDeviceBuffer(P)  # half the bytes a bf16 checkpoint needs
    small_mask = _RawDeviceBuffer(2 * G)
    small_sumsq = _RawDeviceBuffer(4 * G)
    try:
        with pytest.raises(mp.MPError):
            mp.mp_merge_avg(L, base, exps, mask, [0.5, 0.5], small_out)
        with pytest.raises(mp.MPError):
            mp.mp_merge_ties(L, base, exps, small_mask, 0.2, 1.0, out)
        with pytest.raises(mp.MPError):
            mp.mp_index_blocks(L, base, exps, small_sumsq)
    finally:
        torch.cuda.synchronize()
        for b in (small_out, small_mask, small_sumsq):
            b.free()


def test_stream_copy(mp):
    # the measurement aid copies every byte, ragged sizes included, writes
    # nothing past the end, and refuses overlapping or non-device buffers
    import torch
    g = torch.Generator(device="cuda").manual_seed(5)
    for n in (16, 1008, 1024, 1040, (1 << 20) + 48, 3 * (1 << 24) + 16):
        src = torch.randint(-2**31, 2**31 - 1, (n // 4,), dtype=torch.int32, device="cuda", generator=g)
        dst = torch.full((n // 4 + 64,), -1, dtype=torch.int32, device="cuda")
        mp.mp_stream_copy(src, dst[:n // 4])
        torch.cuda.synchronize()
        assert torch.equal(src, dst[:n // 4]), n
        assert bool((dst[n // 4:] == -1).all()), n
    buf = torch.zeros(4096, dtype=torch.int32, device="cuda")
    with pytest.raises(mp.MPError):
        mp._check(mp.lib.mp_stream_copy(mp._ptr(buf), mp._ptr(buf[16:]), 4096, None))
    host = torch.zeros(4096, dtype=torch.int32)  # ordinary host memory: not a device buffer
    with pytest.raises(mp.MPError):
        mp._check(mp.lib.mp_stream_copy(mp._ptr(buf), host.data_ptr(), 4096, None))
