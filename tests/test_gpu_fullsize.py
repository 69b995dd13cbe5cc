"""Parity at the workload shapes, in the launch configuration the benchmark
times.

* Qwen2.5-1.5B-shaped family, K = 4, TIES (device-resident experts): the
  oracle runs on host copies of the whole family.  The index, the catalog
  thresholds, the mask and plan statistics at every budget, and the merged
  checkpoint of both TIES routes are compared bit for bit in full; the oracle
  plans from its own index.  The tensor-scope thresholds are compared on
  every (tensor, expert) pair for a seeded mask.
* Llama-3-8B-shaped families cut to two layers (real hidden, FFN and vocab:
  the embedding and output head, the largest tensors, are whole):
  K = 8 AVG with experts in pinned host memory at ten budgets (merged
  checkpoint compared in full), and K = 16 TIES (density 0.1, 0-80% untouched
  blocks) with experts in pageable host memory at six budgets (merged blocks
  compared on a sample holding the first and last block of every tensor,
  every short block and random blocks of the embedding, the head and the
  rest).  Index and plan are compared in full.
* Qwen2.5-7B-shaped family, K = 8, DARE with sign election: index, merged
  blocks on samples, plan in full (from the GPU index, which the samples
  verified).
"""

import gc
import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_merge_equal, gather_blocks, to_host
from workloads import family_spec, make_family_device

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


def _assert_bitwise(got, want, what):
    """Merged checkpoints equal bit for bit; on a mismatch, report how far
    apart the differing values are (the 1-ulp bar first)."""
    if np.array_equal(got, want):
        return
    d = np.flatnonzero(got != want)
    assert_merge_equal(got[d], want[d], None, "bf16", what)
    raise AssertionError(f"{what}: {d.size} values within 1 ulp but not bitwise equal (first at {d[:5].tolist()})")


def _sample_ids(blocks, n_random, seed, n_big=0):
    """First and last block of every tensor, every short block, n_big random
    blocks of each of the two largest tensors and n_random random blocks."""
    rng = np.random.default_rng(seed)
    t = blocks.tensor
    first = np.flatnonzero(np.r_[True, t[1:] != t[:-1]])
    last = np.r_[first[1:] - 1, blocks.G - 1]
    short = np.flatnonzero(blocks.len < blocks.block_elems)
    parts = [first, last, short, rng.choice(blocks.G, n_random, replace=False)]
    if n_big:
        for tt in np.argsort(-blocks.numel, kind="stable")[:2]:
            parts.append(rng.integers(first[tt], last[tt] + 1, n_big))
    return np.unique(np.concatenate(parts))


def _elem_index(blocks, ids):
    return np.concatenate([np.arange(blocks.off[g], blocks.off[g] + blocks.len[g]) for g in ids])


def _index_full(mp, L, blocks, base, exps, b_h, e_h, res, what):
    """GPU index against the oracle's over every block; returns both (the
    GPU's on the device, the oracle's on the host)."""
    import torch
    K = len(exps)
    sumsq = torch.empty(blocks.G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq, residency=res)
    S_orc = oracle.index(blocks, "bf16", b_h, e_h)
    assert np.array_equal(sumsq.cpu().numpy().view(np.uint32), S_orc.reshape(-1).view(np.uint32)), \
        f"{what}: index differs"
    _say(f"  index equal on all {blocks.G} x {K} units")
    return sumsq, S_orc


def _plan_both(mp, L, blocks, K, sumsq, S_orc, w, B, mask, full):
    st = mp.mp_plan(L, K, sumsq, w, B, mask)
    m_orc, st_orc = oracle.plan(blocks, "bf16", K, S_orc, w, B)
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), m_orc), f"mask differs at B={B}"
    assert st["cost_bytes"] == st_orc["cost"] <= B and st["digest"] == st_orc["digest"]
    assert st["n_selected"] == st_orc["n_selected"] and st["full_bytes"] == full == st_orc["full_bytes"]
    return st, m_orc


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def test_headline_qwen15b_ties_full_compare(mp):
    import torch
    spec = family_spec("qwen2.5-1.5b")
    lay = spec.layout
    K, dens, lam = 4, 0.2, 1.0
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case qwen2.5-1.5b full compare: P={lay.n_params} G={G} K={K} TIES density {dens}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda")
    b_h = to_host(base)
    e_h = [to_host(e) for e in exps]
    _say("  host copies made")
    sumsq, S_orc = _index_full(mp, L, blocks, base, exps, b_h, e_h, mp.MP_DEVICE, "qwen2.5-1.5b")
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    sumsq2 = torch.empty_like(sumsq)
    mp.mp_index_ties(L, base, exps, dens, tau, sumsq=sumsq2)
    assert torch.equal(sumsq2.view(torch.int32), sumsq.view(torch.int32)), "catalog sums of squares differ"
    del sumsq2
    t_orc = oracle.ties_thresholds(blocks, "bf16", b_h, e_h, dens)
    assert np.array_equal(tau.cpu().numpy().view(np.uint32), t_orc.reshape(-1)), "thresholds differ"
    _say(f"  catalog thresholds equal on all {G} x {K} units")
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = lay.n_params * 2 * K
    w = [1.0] * K
    for f in (0.25, 0.5, 1.0):
        B = int(f * full)
        st, m_orc = _plan_both(mp, L, blocks, K, sumsq, S_orc, w, B, mask, full)
        want = oracle.merge_ties_tau(blocks, "bf16", b_h, e_h, m_orc, t_orc, lam)
        io = mp.mp_merge_ties(L, base, exps, mask, dens, lam, out, io=True)
        assert io["expert_bytes"] == st["cost_bytes"]
        _assert_bitwise(to_host(out), want, f"in-merge TIES B={f}")
        io = mp.mp_merge_ties_tau(L, base, exps, mask, tau, lam, out, io=True)
        assert io["expert_bytes"] == st["cost_bytes"]
        _assert_bitwise(to_host(out), want, f"threshold TIES B={f}")
        _say(f"  B={f}: cost={st['cost_bytes']} selected={st['n_selected']}: both TIES routes equal in full")
        del want
    del base, exps, out, b_h, e_h
    _free()


def test_headline_qwen15b_tensor_ties_thresholds(mp):
    """Tensor-scope TIES thresholds at the headline shape, in the launch
    configuration the tensor-scope benchmark times (runs of 16 blocks, every
    XCD's range of (run, expert) pairs): a seeded mask holding about half of
    the units, with expert t mod K taking no block of every third tensor t;
    every (tensor, expert) threshold compared with the oracle's."""
    import torch
    spec = family_spec("qwen2.5-1.5b")
    lay = spec.layout
    K, dens = 4, 0.2
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case qwen2.5-1.5b tensor-scope TIES thresholds: G={G} K={K} density {dens}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda")
    b_h = to_host(base)
    e_h = [to_host(e) for e in exps]
    rng = np.random.default_rng(41)
    m = rng.integers(0, 1 << K, size=G, dtype=np.uint32)
    t = np.asarray(blocks.tensor, np.int64)
    left = t % 3 == 0
    m[left] &= ~(np.uint32(1) << (t[left] % K).astype(np.uint32))
    mask = torch.from_numpy(m.view(np.int32)).cuda()
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    mp.mp_ties_tensor_thresholds(L, base, exps, mask, dens, tau)
    got = tau.cpu().numpy().view(np.uint32)
    _say("  GPU thresholds done; oracle")
    want = oracle.expand_tensor_thresholds(blocks, oracle.ties_tensor_thresholds(blocks, "bf16", b_h, e_h, m, dens))
    assert np.array_equal(got, want), f"{int(np.count_nonzero(got != want))} unit thresholds differ"
    _say(f"  thresholds equal on all {G} x {K} units")
    del base, exps, b_h, e_h
    _free()


def test_llama3_8b_two_layers_k8_avg_pinned(mp):
    """Llama-3-8B shapes (two layers), K = 8, AVG, experts in pinned host
    memory: ten budgets, everything compared in full."""
    import torch
    spec = family_spec("llama3-8b", n_layers=2)
    lay = spec.layout
    K = spec.K
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case llama3-8b x2 layers K={K} AVG pinned: P={lay.n_params} G={G}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda", experts_on_host="pinned")
    b_h = to_host(base)
    e_h = [to_host(e) for e in exps]  # views of the pinned buffers
    sumsq, S_orc = _index_full(mp, L, blocks, base, exps, b_h, e_h, mp.MP_HOST_PINNED, "llama3-8b x2")
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = lay.n_params * 2 * K
    a = [1.0 / K] * K
    for f in [x / 10 for x in range(1, 11)]:
        B = int(f * full)
        st, m_orc = _plan_both(mp, L, blocks, K, sumsq, S_orc, a, B, mask, full)
        io = mp.mp_merge_avg(L, base, exps, mask, a, out, residency=mp.MP_HOST_PINNED, io=True)
        assert io["expert_bytes"] == st["cost_bytes"] == io["h2d_bytes"]
        want = oracle.merge_avg(blocks, "bf16", b_h, e_h, m_orc, a)
        _assert_bitwise(to_host(out), want, f"AVG pinned B={f}")
        _say(f"  B={f}: cost={st['cost_bytes']} selected={st['n_selected']}: merged checkpoint equal in full")
        del want
    del base, exps, out, b_h, e_h
    _free()


def test_llama3_8b_two_layers_k16_ties_pageable(mp):
    """Llama-3-8B shapes (two layers), K = 16, TIES density 0.1, 0-80%
    untouched blocks per expert, experts in pageable host memory (staged):
    six budgets; index and plan in full, merged blocks on a sample that
    covers every tensor's ends, the short blocks, the embedding and head."""
    import torch
    spec = family_spec("llama3-8b-k16", n_layers=2)
    lay = spec.layout
    K = spec.K
    dens, lam = 0.1, 1.0
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case llama3-8b-k16 x2 layers K={K} TIES pageable: P={lay.n_params} G={G}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda", experts_on_host="pageable")
    b_h = to_host(base)
    e_h = [to_host(e) for e in exps]  # views of the host tensors
    sumsq, S_orc = _index_full(mp, L, blocks, base, exps, b_h, e_h, mp.MP_HOST_PAGEABLE, "llama3-8b-k16 x2")
    ids = _sample_ids(blocks, 2048, 321, n_big=1024)
    idx = _elem_index(blocks, ids)
    idx_t = torch.from_numpy(idx).cuda()
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    want = np.zeros_like(b_h)
    full = lay.n_params * 2 * K
    w = [1.0] * K
    for f in (1 / 16, 0.1, 0.25, 0.5, 0.75, 1.0):
        B = int(f * full)
        st, m_orc = _plan_both(mp, L, blocks, K, sumsq, S_orc, w, B, mask, full)
        io = mp.mp_merge_ties(L, base, exps, mask, dens, lam, out, residency=mp.MP_HOST_PAGEABLE, io=True)
        assert io["expert_bytes"] == st["cost_bytes"]
        oracle.merge_ties(blocks, "bf16", b_h, e_h, m_orc[ids], dens, lam, out=want, ids=ids)
        _assert_bitwise(to_host(out[idx_t]), want[idx], f"TIES pageable B={f}")
        _say(f"  B={f:.4f}: cost={st['cost_bytes']} selected={st['n_selected']}: "
             f"{len(ids)} sampled blocks equal")
    del base, exps, out, b_h, e_h, want
    _free()


def test_qwen7b_dare_sign_elect_fullsize(mp):
    import torch
    spec = family_spec("qwen2.5-7b")
    lay = spec.layout
    K, p, seed, lam = 8, 0.9, 7, 1.0
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case qwen2.5-7b full size: P={lay.n_params} G={G} K={K} DARE sign-elect")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda")
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq)
    S = sumsq.cpu().numpy()
    ids = _sample_ids(blocks, 96, 123)
    b_np, doff = gather_blocks(base, blocks, ids)
    e_np = [gather_blocks(e, blocks, ids)[0] for e in exps]
    S_orc = oracle.index(blocks, "bf16", b_np, e_np, doff=doff, ids=ids)
    assert np.array_equal(S.reshape(G, K)[ids].view(np.uint32), S_orc.view(np.uint32)), "index differs on samples"
    _say(f"  index ok on {len(ids)} sampled blocks")
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = lay.n_params * 2 * K
    w = [1.0] * K
    B = int(0.3 * full)
    st = mp.mp_plan(L, K, sumsq, w, B, mask)
    m_orc, st_orc = oracle.plan(blocks, "bf16", K, S, w, B)
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), m_orc), "mask differs"
    assert st["cost_bytes"] == st_orc["cost"] <= B and st["digest"] == st_orc["digest"]
    assert st["n_selected"] == st_orc["n_selected"] and st["full_bytes"] == full
    io = mp.mp_merge_dare(L, base, exps, mask, p, seed, 1, None, lam, out, io=True)
    assert io["expert_bytes"] == st["cost_bytes"]
    want = oracle.merge_dare(blocks, "bf16", b_np, e_np, m_orc[ids], p, seed, 1, [1.0] * K, lam,
                             ids=ids, doff=doff)
    got, _ = gather_blocks(out, blocks, ids)
    _assert_bitwise(got, want, "DARE sign-elect B=0.3")
    _say(f"  B=0.3: cost={st['cost_bytes']} selected={st['n_selected']}: {len(ids)} sampled blocks equal")
    del base, exps, out
    _free()
