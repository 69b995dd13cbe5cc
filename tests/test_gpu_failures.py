"""Failure handling on the GPU, forced from the host: a cap on the library's
workspace gives MP_E_NOMEM before anything is enqueued (the output keeps
its contents); an injected pack failure at chunk n of a staged call gives
MP_E_IO; argument errors write no output.  Every kernel that runs exits
normally; after each failure the same call succeeds and matches the oracle."""

import os
import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import to_dev, to_host
from workloads import FamilySpec, make_family

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


def _family(K=3):
    # 4.6 M parameters: 9 MB per bf16 checkpoint, so 1 MiB staging chunks
    # give a merge at half budget about a dozen chunks and the index about 27
    t = (("a", (1024 * 4096 + 512,)), ("b", (96, 4096)), ("c", (2048,)))
    spec = FamilySpec("fail-test", t, "bf16", 4096, K, ())
    base, exps = make_family(spec, seed=91)
    return spec, base, exps


def _setup(mp, spec, base_np, exps_np):
    import torch
    lay = spec.layout
    L = mp.Layout(lay.numel, lay.block_elems, mp.MP_BF16)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    K = len(exps_np)
    S = oracle.index(blocks, "bf16", base_np, exps_np).reshape(-1)
    full = lay.n_params * 2 * K
    m_np, _ = oracle.plan(blocks, "bf16", K, S, [1.0 / K] * K, full // 2)
    mask = torch.from_numpy(m_np.view(np.int32)).cuda()
    return L, blocks, K, mask, m_np


def _sentinel_out(base):
    out = base.clone()
    out.view(torch_int16()).fill_(0x1234)
    return out


def torch_int16():
    import torch
    return torch.int16


def test_workspace_limit_gives_nomem_and_writes_nothing(mp):
    import torch
    spec, base_np, exps_np = _family()
    L, blocks, K, mask, m_np = _setup(mp, spec, base_np, exps_np)
    base = to_dev(base_np, "bf16")
    exps = [to_dev(e, "bf16") for e in exps_np]
    alpha = [1.0 / K] * K
    want = oracle.merge_avg(blocks, "bf16", base_np, exps_np, m_np, alpha)
    try:
        torch.cuda.synchronize()  # nothing in flight when the workspace is released
        mp.mp_release()
        assert mp.mp_workspace_bytes() == 0
        mp.mp_set_workspace_limit(1)
        out = _sentinel_out(base)
        before = out.clone()
        with pytest.raises(mp.MPError) as ei:
            mp.mp_merge_avg(L, base, exps, mask, alpha, out)
        assert ei.value.code == mp.MP_E_NOMEM
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), before.view(torch.int16))
        assert mp.mp_workspace_bytes() == 0
        with pytest.raises(mp.MPError) as ei:  # the plan needs its scratch too
            st = mp.mp_plan(L, K, None, alpha, 10**9, mask)
        assert ei.value.code == mp.MP_E_NOMEM
        # no cap: the same call succeeds and matches the oracle
        mp.mp_set_workspace_limit(0)
        mp.mp_merge_avg(L, base, exps, mask, alpha, out)
        assert np.array_equal(to_host(out), want)
        held = mp.mp_workspace_bytes()
        assert held > 0
        _say(f"  workspace held after one device merge: {held} bytes")
        # a cap above the device workspace but below the staging buffers:
        # the host-pageable merge (pinned staging) is refused, nothing written
        mp.mp_set_workspace_limit(held + (1 << 20))
        out2 = _sentinel_out(base)
        before2 = out2.clone()
        host = [torch.from_numpy(e) for e in exps_np]
        with pytest.raises(mp.MPError) as ei:
            mp.mp_merge_avg(L, base, host, mask, alpha, out2, residency=mp.MP_HOST_PAGEABLE)
        assert ei.value.code == mp.MP_E_NOMEM
        torch.cuda.synchronize()
        assert torch.equal(out2.view(torch.int16), before2.view(torch.int16))
        assert mp.mp_workspace_bytes() == held
        mp.mp_set_workspace_limit(0)
        mp.mp_merge_avg(L, base, host, mask, alpha, out2, residency=mp.MP_HOST_PAGEABLE)
        assert np.array_equal(to_host(out2), want)
    finally:
        mp.mp_set_workspace_limit(0)


def test_pack_failure_at_chunk_n_gives_io_error(mp):
    import torch
    spec, base_np, exps_np = _family()
    L, blocks, K, mask, m_np = _setup(mp, spec, base_np, exps_np)
    base = to_dev(base_np, "bf16")
    host = [torch.from_numpy(e) for e in exps_np]
    alpha = [1.0 / K] * K
    sumsq = torch.empty(blocks.G * K, dtype=torch.float32, device="cuda")
    out = torch.empty_like(base)
    try:
        mp.mp_set_stage_bytes(1 << 20)  # 1 MiB chunks: a few dozen chunks for this family
        for n in (0, 2, 5):
            os.environ["MP_FAULT_PACK_CHUNK"] = str(n)
            with pytest.raises(mp.MPError) as ei:
                mp.mp_merge_avg(L, base, host, mask, alpha, out, residency=mp.MP_HOST_PAGEABLE)
            assert ei.value.code == mp.MP_E_IO
            with pytest.raises(mp.MPError) as ei:
                mp.mp_index_blocks(L, base, host, sumsq, residency=mp.MP_HOST_PAGEABLE)
            assert ei.value.code == mp.MP_E_IO
            torch.cuda.synchronize()  # the chunks before n ran normally
        _say("  injected pack failures at chunks 0, 2, 5: MP_E_IO for the merge and the index")
        del os.environ["MP_FAULT_PACK_CHUNK"]
        mp.mp_index_blocks(L, base, host, sumsq, residency=mp.MP_HOST_PAGEABLE)
        S = oracle.index(blocks, "bf16", base_np, exps_np).reshape(-1)
        assert np.array_equal(sumsq.cpu().numpy().view(np.uint32), S.view(np.uint32))
        io = mp.mp_merge_avg(L, base, host, mask, alpha, out, residency=mp.MP_HOST_PAGEABLE, io=True)
        assert np.array_equal(to_host(out), oracle.merge_avg(blocks, "bf16", base_np, exps_np, m_np, alpha))
        assert io["h2d_bytes"] == io["expert_bytes"]
    finally:
        os.environ.pop("MP_FAULT_PACK_CHUNK", None)
        mp.mp_set_stage_bytes(256 << 20)


def test_argument_errors_write_no_output(mp):
    import torch
    spec, base_np, exps_np = _family()
    L, blocks, K, mask, m_np = _setup(mp, spec, base_np, exps_np)
    base = to_dev(base_np, "bf16")
    exps = [to_dev(e, "bf16") for e in exps_np]
    out = _sentinel_out(base)
    before = out.clone()
    sumsq = torch.full((blocks.G * K,), 7.0, dtype=torch.float32, device="cuda")
    tau = torch.full((blocks.G * K,), 7, dtype=torch.int32, device="cuda")
    m2 = torch.full_like(mask, 5)
    calls = [
        lambda: mp.mp_merge_avg(L, base, exps, mask, [float("nan")] * K, out),
        lambda: mp.mp_merge_ties(L, base, exps, mask, 1.5, 1.0, out),
        lambda: mp.mp_merge_ties_tau(L, base, exps, mask, tau, float("inf"), out),
        lambda: mp.mp_merge_dare(L, base, exps, mask, 1.0, 7, 0, [0.5] * K, 1.0, out),
        lambda: mp.mp_merge_avg(L, base, exps, mask, [0.5] * K, exps[0]),  # output aliases an expert
        lambda: mp.mp_index_ties(L, base, exps, 2.0, tau, sumsq=sumsq),
        lambda: mp.mp_plan(L, K, sumsq, [1.0] * K, 10**9, m2, flags=64),
        lambda: mp.mp_plan(L, K, sumsq, [float("nan")] * K, 10**9, m2),
    ]
    for c in calls:
        with pytest.raises(mp.MPError) as ei:
            c()
        assert ei.value.code in (mp.MP_E_ARG, mp.MP_E_UNSUPPORTED)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), before.view(torch.int16))
    assert bool((sumsq == 7.0).all()) and bool((tau == 7).all()) and bool((m2 == 5).all())


def test_tensor_thresholds_report_no_cut_and_serialise_streams(mp):
    # the selection's "no cut" branch (never reached by real data) is forced
    # from the host: the kernels finish normally, the call reads the error
    # word and returns MP_E_HIP; without the hook, calls on two streams that
    # share the device scratch give the oracle's thresholds back to back
    import torch
    spec, base_np, exps_np = _family()
    L, blocks, K, mask, m_np = _setup(mp, spec, base_np, exps_np)
    base = to_dev(base_np, "bf16")
    exps = [to_dev(e, "bf16") for e in exps_np]
    tau = torch.empty(blocks.G * K, dtype=torch.int32, device="cuda")
    try:
        os.environ["MP_FAULT_TENSOR_NO_CUT"] = "1"
        with pytest.raises(mp.MPError) as ei:
            mp.mp_ties_tensor_thresholds(L, base, exps, mask, 0.2, tau)
        assert ei.value.code == mp.MP_E_HIP and "internal error" in str(ei.value)
    finally:
        os.environ.pop("MP_FAULT_TENSOR_NO_CUT", None)
    full = np.full(blocks.G, (1 << K) - 1, np.uint32)
    mask_full = torch.from_numpy(full.view(np.int32)).cuda()
    want_half = oracle.expand_tensor_thresholds(
        blocks, oracle.ties_tensor_thresholds(blocks, "bf16", base_np, exps_np, m_np, 0.2))
    want_full = oracle.expand_tensor_thresholds(
        blocks, oracle.ties_tensor_thresholds(blocks, "bf16", base_np, exps_np, full, 0.1))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    tau2 = torch.empty_like(tau)
    torch.cuda.synchronize()  # inputs made on the current stream are ready for s1 and s2
    for _ in range(3):
        mp.mp_ties_tensor_thresholds(L, base, exps, mask, 0.2, tau, stream=s1)
        mp.mp_ties_tensor_thresholds(L, base, exps, mask_full, 0.1, tau2, stream=s2)
        torch.cuda.synchronize()
        assert np.array_equal(tau.cpu().numpy().view(np.uint32), want_half)
        assert np.array_equal(tau2.cpu().numpy().view(np.uint32), want_full)
    _say("  forced no-cut: MP_E_HIP; two streams in turn: both thresholds equal the oracle's")
