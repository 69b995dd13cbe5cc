"""Full-size parity on the workload shapes, in the launch configuration the
benchmark times (device-resident experts, one call per step stage).

The index is compared bit for bit on sampled blocks (the oracle recomputes
them from host copies of the same bytes); the plan is compared bit for bit in
full (the oracle plans all units from the GPU's index, which the samples
verified); merged outputs are compared on the sampled blocks.  Samples cover
the first and last blocks, every short block and a seeded random set.
"""

import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_merge_equal, gather_blocks
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


def _sample_ids(blocks, n_random, seed):
    rng = np.random.default_rng(seed)
    short = np.nonzero(blocks.len < blocks.len.max())[0]
    ids = np.unique(np.concatenate([[0, 1, blocks.G - 1], short[:64], rng.choice(blocks.G, n_random, replace=False)]))
    return ids


def _full_run(mp, name, K, op, budgets, n_random=192, **kw):
    import torch
    spec = family_spec(name)
    lay = spec.layout
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    _say(f"case {name} full size: P={lay.n_params} G={G} K={K} op={op}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda")
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, exps, sumsq)
    S = sumsq.cpu().numpy()
    ids = _sample_ids(blocks, n_random, 123)
    b_np, doff = gather_blocks(base, blocks, ids)
    e_np = [gather_blocks(e, blocks, ids)[0] for e in exps]
    S_orc = oracle.index(blocks, "bf16", b_np, e_np, doff=doff, ids=ids)
    assert np.array_equal(S.reshape(G, K)[ids].view(np.uint32), S_orc.view(np.uint32)), "index differs on samples"
    _say(f"  index ok on {len(ids)} sampled blocks")
    tau = None
    if op == "ties":  # catalog thresholds (and the same sums of squares) in one pass
        tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
        sumsq2 = torch.empty_like(sumsq)
        mp.mp_index_ties(L, base, exps, kw["density"], tau, sumsq=sumsq2)
        assert torch.equal(sumsq2.view(torch.int32), sumsq.view(torch.int32)), "catalog sums of squares differ"
        t_orc = oracle.ties_thresholds(blocks, "bf16", b_np, e_np, kw["density"], ids=ids, doff=doff)
        assert np.array_equal(tau.cpu().numpy().view(np.uint32).reshape(G, K)[ids], t_orc), "thresholds differ"
        _say(f"  thresholds ok on {len(ids)} sampled blocks")
        del sumsq2
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = lay.n_params * 2 * K
    w = kw.get("w", [1.0] * K)
    for f in budgets:
        B = int(f * full)
        st = mp.mp_plan(L, K, sumsq, w, B, mask)
        m_gpu = mask.cpu().numpy().view(np.uint32)
        m_orc, st_orc = oracle.plan(blocks, "bf16", K, S, w, B)
        assert np.array_equal(m_gpu, m_orc), f"mask differs at B={B}"
        assert st["cost_bytes"] == st_orc["cost"] <= B and st["digest"] == st_orc["digest"]
        assert st["n_selected"] == st_orc["n_selected"] and st["full_bytes"] == full
        if op == "ties":
            io = mp.mp_merge_ties(L, base, exps, mask, kw["density"], kw["lam"], out, io=True)
            want = oracle.merge_ties(blocks, "bf16", b_np, e_np, m_orc[ids], kw["density"], kw["lam"],
                                     ids=ids, doff=doff)
            # catalog thresholds: the same bits for the whole checkpoint
            out2 = torch.empty_like(out)
            io2 = mp.mp_merge_ties_tau(L, base, exps, mask, tau, kw["lam"], out2, io=True)
            assert io2["expert_bytes"] == st["cost_bytes"]
            assert torch.equal(out.view(torch.int16), out2.view(torch.int16)), f"catalog-threshold TIES differs at B={f}"
            del out2
        else:
            io = mp.mp_merge_dare(L, base, exps, mask, kw["p"], kw["seed"], 1, None, kw["lam"], out, io=True)
            want = oracle.merge_dare(blocks, "bf16", b_np, e_np, m_orc[ids], kw["p"], kw["seed"], 1,
                                     [1.0] * K, kw["lam"], ids=ids, doff=doff)
        assert io["expert_bytes"] == st["cost_bytes"]
        got, _ = gather_blocks(out, blocks, ids)
        nb = assert_merge_equal(got, want, None, "bf16", f"{name} {op} B={f}")
        assert nb == 0, f"{name} {op} B={f}: {nb} sampled values within tolerance but not bitwise equal"
        _say(f"  B={f}: cost={st['cost_bytes']} selected={st['n_selected']} sampled non-bitwise={nb}")
    del base, exps, out
    torch.cuda.empty_cache()


def test_headline_qwen15b_ties_fullsize(mp):
    _full_run(mp, "qwen2.5-1.5b", 4, "ties", (0.25, 0.5, 1.0), density=0.2, lam=1.0)


def test_qwen7b_dare_sign_elect_fullsize(mp):
    _full_run(mp, "qwen2.5-7b", 8, "dare", (0.3,), n_random=96, p=0.9, seed=7, lam=1.0)
