"""GPU parity of the low-rank adapter delta source (mp_lora_materialize)
against the oracle, and of the budgeted path run on the deltas it writes.

Bars: on the dyadic grid (every rank sum exact in fp32) the materialised
deltas are bitwise equal to the oracle's for any summation order, and so is
everything downstream (index, plan, merge).  On normal-distributed adapters
the matrix cores' fp32 accumulation may differ from the correctly rounded
sum: bf16 deltas may then differ by 1 ulp, fp32 ones by at most
(rank + 2) * 2^-24 * |scale| * sum_k |B[r][k] A[k][c]|.
"""

import sys

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_merge_equal, to_dev, to_host
from workloads import FamilySpec, family_spec, lora_records, make_family, make_family_device, make_lora_adapters

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


def _awkward(dtype, be=512):
    """Adapted matrices with rows and columns off the 64 x 128 tile grid
    (44 columns: rows of A not 16-byte aligned in bf16), blocks that cut
    rows, and tensors without an adapter in between."""
    t = (("w0", (200, 136)), ("v0", (64,)), ("w1", (130, 264)), ("w2", (96, 8)), ("v1", (520,)),
         ("w3", (72, 1000)), ("w4", (64, 128)), ("e", (40, 48)), ("w5", (30, 44)))
    return FamilySpec("awkward", t, dtype, be, 3, ())


def _sentinel(P, dtype, i):
    v = np.float32(7.0 + i)
    if dtype == "bf16":
        return np.full(P, oracle.round_bf16(np.array([v]))[0], np.uint16)
    return np.full(P, v, np.float32)


def _f32(x, dtype):
    return (x.astype(np.uint32) << 16).view(np.float32) if dtype == "bf16" else x


def _assert_close(got, want, A, B, scale, dtype, what):
    """|got - want| <= (rank + 2) 2^-24 |scale| sum_k |B A| (the fp32
    accumulation bound), plus one ulp of the dtype for the final rounding."""
    r = A.shape[0]
    Af, Bf = np.abs(_f32(A, dtype).astype(np.float64)), np.abs(_f32(B, dtype).astype(np.float64))
    bound = (r + 2) * 2.0**-24 * abs(scale) * (Bf @ Af).reshape(-1)
    g, w = _f32(got, dtype).astype(np.float64), _f32(want, dtype).astype(np.float64)
    if dtype == "bf16":
        bound = bound + np.spacing(np.maximum(np.abs(g), np.abs(w)).astype(np.float32)).astype(np.float64) * 65536
    err = np.abs(g - w)
    assert (err <= bound + 1e-45).all(), f"{what}: {int((err > bound + 1e-45).sum())} deltas beyond the bound"
    return int((got != want).sum())


def _materialize(mp, spec, recs, ads_np, mask_np=None, prefill=True):
    import torch
    lay = spec.layout
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    K = len(ads_np)
    ads = [to_dev(a, lay.dtype) for a in ads_np] if recs else []
    outs = [to_dev(_sentinel(lay.n_params, lay.dtype, i), lay.dtype) for i in range(K)] if prefill else \
        [torch.empty(lay.n_params, dtype=torch.bfloat16 if lay.dtype == "bf16" else torch.float32, device="cuda")
         for _ in range(K)]
    mask = None if mask_np is None else torch.from_numpy(np.ascontiguousarray(mask_np, np.uint32).view(np.int32)).cuda()
    mp.mp_lora_materialize(L, recs, ads, outs, mask=mask)
    torch.cuda.synchronize()
    return L, outs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank", [1, 7, 16, 33, 64])
def test_lora_materialize_exact_grid_bitwise(mp, dtype, rank):
    spec = _awkward(dtype)
    lay = spec.layout
    recs, n = lora_records(spec, rank, 0.5, targets=("w0", "w1", "w2", "w3", "w4", "w5"))
    ads = make_lora_adapters(n, 3, dtype, seed=rank, grid=True)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    rng = np.random.default_rng(rank)
    for mask in (None, rng.integers(0, 8, blocks.G).astype(np.uint32), np.zeros(blocks.G, np.uint32)):
        _say(f"case lora exact {dtype} rank={rank} mask={'all' if mask is None else int(mask.sum())}")
        _, outs = _materialize(mp, spec, recs, ads, mask)
        fill = [_sentinel(lay.n_params, dtype, i) for i in range(3)]
        want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads, mask=mask, fill=fill)
        for i in range(3):
            got = to_host(outs[i])
            assert np.array_equal(got, want[i]), f"expert {i}: {int((got != want[i]).sum())} elements differ"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("route", ["row-lists", "operand-copy"])
def test_lora_masked_pull_row_lists(mp, dtype, route):
    # Masked pulls: sparse masks (most rows of most tensors unselected), a
    # mask selecting every block, and two masked pulls with one layout and
    # record set issued on two streams without a synchronisation between them
    # (they share the table's scratch).  With a bf16 tensor whose rows are not
    # whole 16-byte chunks (w5, 44 columns) the pull lists the rows meeting a
    # selected block and computes only those; otherwise it runs on the
    # operand-order copy and skips the wave tiles with nothing selected.
    import torch
    spec = _awkward(dtype)
    lay = spec.layout
    targets = ("w0", "w1", "w2", "w3", "w4") + (("w5",) if route == "row-lists" else ())
    if dtype == "f32" and route == "row-lists":
        pytest.skip("fp32 rows are always whole 16-byte chunks")
    recs, n = lora_records(spec, 16, 0.5, targets=targets)
    ads = make_lora_adapters(n, 3, dtype, seed=41, grid=True)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    rng = np.random.default_rng(41)
    fill = [_sentinel(lay.n_params, dtype, i) for i in range(3)]
    sparse = np.where(rng.random((blocks.G, 3)) < 0.05, 1, 0).astype(np.uint32)
    sparse = (sparse << np.arange(3, dtype=np.uint32)).sum(1).astype(np.uint32)
    full = np.full(blocks.G, 7, np.uint32)
    for name, mask in (("sparse", sparse), ("full", full)):
        _say(f"case lora row lists {dtype} {name}")
        _, outs = _materialize(mp, spec, recs, ads, mask)
        want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads, mask=mask, fill=fill)
        for i in range(3):
            got = to_host(outs[i])
            assert np.array_equal(got, want[i]), f"{name} expert {i}: {int((got != want[i]).sum())} differ"
    _say(f"case lora row lists {dtype} two streams")
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    ads_d = [to_dev(a, dtype) for a in ads]
    masks = [sparse, rng.integers(0, 8, blocks.G).astype(np.uint32)]
    outs = [[to_dev(_sentinel(lay.n_params, dtype, i), dtype) for i in range(3)] for _ in masks]
    mdev = [torch.from_numpy(m.view(np.int32)).cuda() for m in masks]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for o, m, st in zip(outs, mdev, streams):
        mp.mp_lora_materialize(L, recs, ads_d, o, mask=m, stream=st)
    torch.cuda.synchronize()
    for o, m in zip(outs, masks):
        want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads, mask=m, fill=fill)
        for i in range(3):
            got = to_host(o[i])
            assert np.array_equal(got, want[i]), f"two streams expert {i}: {int((got != want[i]).sum())} differ"


@pytest.mark.parametrize("rank", [8, 16, 64])
def test_lora_materialize_exact_grid_bitwise_aligned_rows(mp, rank):
    # bf16 with every row of A 16-byte aligned: the 16-byte loads of A
    spec = _awkward("bf16")
    lay = spec.layout
    recs, n = lora_records(spec, rank, 0.5, targets=("w0", "w1", "w2", "w3", "w4"))
    assert all(r[4] % 8 == 0 and r[2] % 8 == 0 for r in recs)
    ads = make_lora_adapters(n, 3, "bf16", seed=rank + 1, grid=True)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    rng = np.random.default_rng(rank + 1)
    for mask in (None, rng.integers(0, 8, blocks.G).astype(np.uint32), np.zeros(blocks.G, np.uint32)):
        _say(f"case lora exact aligned rank={rank} mask={'all' if mask is None else int(mask.sum())}")
        _, outs = _materialize(mp, spec, recs, ads, mask)
        fill = [_sentinel(lay.n_params, "bf16", i) for i in range(3)]
        want = oracle.lora_materialize(blocks, "bf16", lay.numel, recs, ads, mask=mask, fill=fill)
        for i in range(3):
            got = to_host(outs[i])
            assert np.array_equal(got, want[i]), f"expert {i}: {int((got != want[i]).sum())} elements differ"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("be", [8, 64, 112, 120])
def test_lora_materialize_short_blocks_bitwise(mp, dtype, be):
    # blocks shorter than a lane's 116-column span (several blocks per lane
    # and tile row) and just above it
    spec = _awkward(dtype, be=be)
    lay = spec.layout
    recs, n = lora_records(spec, 16, 0.5, targets=("w0", "w1", "w3", "w4"))
    ads = make_lora_adapters(n, 3, dtype, seed=be, grid=True)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    mask = np.random.default_rng(be).integers(0, 8, blocks.G).astype(np.uint32)
    _say(f"case lora short blocks {dtype} be={be} G={blocks.G}")
    _, outs = _materialize(mp, spec, recs, ads, mask)
    fill = [_sentinel(lay.n_params, dtype, i) for i in range(3)]
    want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads, mask=mask, fill=fill)
    for i in range(3):
        got = to_host(outs[i])
        assert np.array_equal(got, want[i]), f"expert {i}: {int((got != want[i]).sum())} elements differ"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank", [16, 64])
def test_lora_materialize_normal_adapters_within_bound(mp, dtype, rank):
    spec = _awkward(dtype)
    lay = spec.layout
    recs, n = lora_records(spec, rank, 2.0, targets=("w0", "w1", "w3"))
    ads = make_lora_adapters(n, 2, dtype, seed=100 + rank, std=0.05)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    _say(f"case lora normal {dtype} rank={rank}")
    _, outs = _materialize(mp, spec, recs, ads)
    want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads)
    toff = np.concatenate([[0], np.cumsum(lay.numel)])
    for i in range(2):
        got = to_host(outs[i])
        af = ads[i]
        nb = 0
        for (t, rows, cols, r, a_off, b_off, sc) in recs:
            sl = slice(toff[t], toff[t] + rows * cols)
            nb += _assert_close(got[sl], want[i][sl], af[a_off:a_off + r * cols].reshape(r, cols),
                                af[b_off:b_off + rows * r].reshape(rows, r), sc, dtype, f"tensor {t}")
        _say(f"  expert {i}: {nb} of {got.size} deltas differ from the correctly rounded ones")
        rest = np.ones(lay.n_params, bool)
        for (t, rows, cols, *_r) in recs:
            rest[toff[t]:toff[t] + rows * cols] = False
        assert not got[rest].any(), "a tensor without an adapter has nonzero deltas"


def _mini(dtype, n_layers=2, be=4096):
    hidden, ffn, vocab = 256, 704, 520
    t = [("embed_tokens.weight", (vocab, hidden))]
    for l in range(n_layers):
        p = f"layers.{l}."
        t += [(p + "self_attn.q_proj.weight", (hidden, hidden)), (p + "self_attn.q_proj.bias", (hidden,)),
              (p + "self_attn.k_proj.weight", (64, hidden)), (p + "self_attn.v_proj.weight", (64, hidden)),
              (p + "self_attn.o_proj.weight", (hidden, hidden)),
              (p + "mlp.gate_proj.weight", (ffn, hidden)), (p + "mlp.up_proj.weight", (ffn, hidden)),
              (p + "mlp.down_proj.weight", (hidden, ffn)), (p + "input_layernorm.weight", (hidden,))]
    t.append(("norm.weight", (hidden,)))
    return FamilySpec("mini-lora", tuple(t), dtype, be, 4, ())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_lora_budgeted_ties_and_avg_on_materialised_deltas(mp, dtype):
    # Algorithm 2 with the adapter source: catalog from the full deltas, a plan
    # per budget, then only the selected units materialised and merged.
    import torch
    spec = _mini(dtype)
    lay = spec.layout
    K = 4
    recs, n = lora_records(spec, 16, 0.5)
    ads = make_lora_adapters(n, K, dtype, seed=5, grid=True)
    base_np, _ = make_family(spec, K=1, seed=3)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    G = blocks.G
    L, full = _materialize(mp, spec, recs, ads)
    d_orc = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads)
    for i in range(K):
        assert np.array_equal(to_host(full[i]), d_orc[i])
    base = to_dev(base_np, dtype)
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_blocks(L, base, full, sumsq, delta=True)
    S_orc = oracle.index(blocks, dtype, base_np, d_orc, delta=True).reshape(-1)
    assert np.array_equal(sumsq.cpu().numpy().view(np.uint32), S_orc.view(np.uint32))
    del full
    fb = oracle.full_bytes(blocks, dtype, K)
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    for f in (0.25, 0.5, 1.0):
        B = int(f * fb)
        for op, w in (("ties", [1.0] * K), ("avg", [0.25] * K)):
            _say(f"case lora pipeline {dtype} {op} B={f}")
            st = mp.mp_plan(L, K, sumsq, w, B, mask, flags=mp.MP_PLAN_SKIP_ZERO)
            m_orc, st_orc = oracle.plan(blocks, dtype, K, S_orc, w, B, flags=2)
            m_gpu = mask.cpu().numpy().view(np.uint32)
            assert np.array_equal(m_gpu, m_orc) and st["digest"] == st_orc["digest"]
            # only the selected units are pulled; the rest of the buffers stay garbage
            _, sel = _materialize(mp, spec, recs, ads, m_gpu, prefill=False)
            if op == "ties":
                io = mp.mp_merge_ties(L, base, sel, mask, 0.2, 1.0, out, io=True, delta=True)
                want = oracle.merge_ties(blocks, dtype, base_np, d_orc, m_orc, 0.2, 1.0, delta=True)
            else:
                io = mp.mp_merge_avg(L, base, sel, mask, w, out, io=True, delta=True)
                want = oracle.merge_avg(blocks, dtype, base_np, d_orc, m_orc, w, delta=True)
            nb = assert_merge_equal(to_host(out), want, base_np, dtype, f"lora {op} B={f}")
            assert nb == 0
            assert io["expert_bytes"] == st["cost_bytes"]


def test_lora_without_records_writes_zeros_and_rejects_bad_buffers(mp):
    import torch
    spec = _awkward("bf16")
    lay = spec.layout
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    mask = np.random.default_rng(9).integers(0, 4, blocks.G).astype(np.uint32)
    _say("case lora no records")
    L, outs = _materialize(mp, spec, [], [None, None], mask)
    for i in range(2):
        want = _sentinel(lay.n_params, "bf16", i)
        for g in range(blocks.G):
            if (mask[g] >> i) & 1:
                want[blocks.off[g]:blocks.off[g] + blocks.len[g]] = 0
        assert np.array_equal(to_host(outs[i]), want)
    recs, n = lora_records(spec, 8, 1.0, targets=("w0",))
    from tests.test_gpu_parity import _RawDeviceBuffer
    small = _RawDeviceBuffer(2 * (n - 1))  # one element short
    dl = [torch.zeros(lay.n_params, dtype=torch.bfloat16, device="cuda")]
    try:
        with pytest.raises(mp.MPError) as e:
            mp.mp_lora_materialize(L, recs, [small], dl)
        assert e.value.code == mp.MP_E_ARG
    finally:
        small.free()
    buf = torch.zeros(lay.n_params + n, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(mp.MPError) as e:  # the delta buffer overlaps the adapter
        mp.mp_lora_materialize(L, recs, [buf[lay.n_params // 2:]], [buf[:lay.n_params]])
    assert e.value.code == mp.MP_E_ARG
    with pytest.raises(mp.MPError) as e:  # two experts share one delta buffer
        mp.mp_lora_materialize(L, recs, [buf, buf], [dl[0], dl[0]])
    assert e.value.code == mp.MP_E_ARG


def test_lora_fullsize_qwen_layout_sampled_tensors(mp):
    # Qwen2.5-1.5B shapes, rank-16 adapters on every projection of every
    # layer, four experts: the whole model is materialised on the GPU and
    # whole tensors spread over the model are checked against the oracle.
    import torch
    spec = family_spec("qwen2.5-1.5b")
    lay = spec.layout
    K = 4
    recs, n = lora_records(spec, 16, 2.0)
    ads_np = make_lora_adapters(n, K, "bf16", seed=11, std=0.05)
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    ads = [to_dev(a, "bf16") for a in ads_np]
    outs = [torch.empty(lay.n_params, dtype=torch.bfloat16, device="cuda") for _ in range(K)]
    _say("case lora fullsize qwen2.5-1.5b rank 16")
    mp.mp_lora_materialize(L, recs, ads, outs)
    torch.cuda.synchronize()
    toff = np.concatenate([[0], np.cumsum(lay.numel)])
    names = [nm for nm, _ in spec.tensors]
    picks = [r for r in recs if names[r[0]].startswith(("layers.0.", "layers.13.", "layers.27."))]
    assert len(picks) == 21
    for (t, rows, cols, r, a_off, b_off, sc) in picks:
        for i in (0, K - 1):
            A = ads_np[i][a_off:a_off + r * cols].reshape(r, cols)
            B = ads_np[i][b_off:b_off + rows * r].reshape(rows, r)
            want = oracle.lora_delta("bf16", rows, cols, A, B, sc)
            got = to_host(outs[i][int(toff[t]):int(toff[t]) + rows * cols])
            nb = _assert_close(got, want, A, B, sc, "bf16", f"{names[t]} expert {i}")
            _say(f"  {names[t]} expert {i}: {nb} of {got.size} deltas differ from the correctly rounded ones")
    # tensors without an adapter: zeros
    for t in (0, len(lay.numel) - 1):
        assert not outs[0][int(toff[t]):int(toff[t + 1])].view(torch.int16).any().item()


# ------------------------------------------------------------ fused adapter TIES merge
def _fused(mp, spec, recs, ads_d, base_d, mask_np, tau_d, lam, K):
    import torch
    lay = spec.layout
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    mask = torch.from_numpy(np.ascontiguousarray(mask_np, np.uint32).view(np.int32)).cuda()
    out = torch.empty_like(base_d)
    mp.mp_lora_merge_ties_tau(L, base_d, recs, ads_d if recs else [None] * K, mask, tau_d, lam, out)
    torch.cuda.synchronize()
    return to_host(out)


def _fused_targets(dtype):
    # bf16 needs whole 16-byte chunks per row: w5 (44 columns) only in fp32
    return ("w0", "w1", "w2", "w3", "w4") + (("w5",) if dtype == "f32" else ())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank", [1, 7, 16, 33, 64])
def test_lora_fused_ties_exact_grid_bitwise(mp, dtype, rank):
    # The fused merge against the oracle's pull then TIES from thresholds,
    # on dyadic adapters (every rank sum exact): bitwise, at random, full and
    # empty masks, with tensors off the tile grid and without adapters.
    import torch
    spec = _awkward(dtype)
    lay = spec.layout
    K = 3
    recs, n = lora_records(spec, rank, 0.5, targets=_fused_targets(dtype))
    ads = make_lora_adapters(n, K, dtype, seed=200 + rank, grid=True)
    base_np, _ = make_family(spec, K=1, seed=rank)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    d_full = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads)
    tau = oracle.ties_thresholds(blocks, dtype, base_np, d_full, 0.3, delta=True)
    tau_d = torch.from_numpy(np.ascontiguousarray(tau, np.uint32).reshape(-1).view(np.int32)).cuda()
    ads_d = [to_dev(a, dtype) for a in ads]
    base_d = to_dev(base_np, dtype)
    rng = np.random.default_rng(rank)
    for name, mask in (("random", rng.integers(0, 8, blocks.G).astype(np.uint32)),
                       ("full", np.full(blocks.G, 7, np.uint32)), ("empty", np.zeros(blocks.G, np.uint32))):
        for lam in (1.0, 0.7):
            _say(f"case lora fused exact {dtype} rank={rank} mask={name} lam={lam}")
            got = _fused(mp, spec, recs, ads_d, base_d, mask, tau_d, lam, K)
            want = oracle.merge_ties_tau(blocks, dtype, base_np, d_full, mask, tau, lam, delta=True)
            assert assert_merge_equal(got, want, base_np, dtype, f"fused {name} lam={lam}") == 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("be", [8, 64, 112, 4096])
def test_lora_fused_ties_block_sizes_bitwise(mp, dtype, be):
    # blocks shorter than a tile row segment (several blocks per lane and
    # tile) up to blocks holding many rows
    import torch
    spec = _awkward(dtype, be=be)
    lay = spec.layout
    K = 3
    recs, n = lora_records(spec, 16, 0.5, targets=_fused_targets(dtype))
    ads = make_lora_adapters(n, K, dtype, seed=be, grid=True)
    base_np, _ = make_family(spec, K=1, seed=be)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    d_full = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads)
    tau = oracle.ties_thresholds(blocks, dtype, base_np, d_full, 0.2, delta=True)
    tau_d = torch.from_numpy(np.ascontiguousarray(tau, np.uint32).reshape(-1).view(np.int32)).cuda()
    mask = np.random.default_rng(be).integers(0, 8, blocks.G).astype(np.uint32)
    _say(f"case lora fused blocks {dtype} be={be} G={blocks.G}")
    got = _fused(mp, spec, recs, [to_dev(a, dtype) for a in ads], to_dev(base_np, dtype), mask, tau_d, 1.0, K)
    want = oracle.merge_ties_tau(blocks, dtype, base_np, d_full, mask, tau, 1.0, delta=True)
    assert assert_merge_equal(got, want, base_np, dtype, f"fused be={be}") == 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank", [16, 64])
def test_lora_fused_ties_equals_pull_then_merge(mp, dtype, rank):
    # Normal-distributed adapters (fp32 accumulation not exact): the fused
    # merge equals the library's own pull of the selected units followed by
    # the threshold merge, bit for bit, with the thresholds from the
    # library's catalog pass over the full pull.
    import torch
    spec = _awkward(dtype)
    lay = spec.layout
    K = 4
    recs, n = lora_records(spec, rank, 2.0, targets=_fused_targets(dtype))
    ads = make_lora_adapters(n, K, dtype, seed=300 + rank, std=0.05)
    base_np, _ = make_family(spec, K=1, seed=300 + rank)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    L, full = _materialize(mp, spec, recs, ads, prefill=False)
    base_d = to_dev(base_np, dtype)
    tau_d = torch.empty(blocks.G * K, dtype=torch.int32, device="cuda")
    mp.mp_index_ties(L, base_d, full, 0.2, tau_d, delta=True)
    ads_d = [to_dev(a, dtype) for a in ads]
    rng = np.random.default_rng(rank)
    out = torch.empty_like(base_d)
    for f in (0.1, 0.5, 1.0):
        mask = np.where(rng.random((blocks.G, K)) < f, 1, 0).astype(np.uint32)
        mask = (mask << np.arange(K, dtype=np.uint32)).sum(1).astype(np.uint32)
        _say(f"case lora fused vs pull {dtype} rank={rank} f={f}")
        _, sel = _materialize(mp, spec, recs, ads, mask, prefill=False)
        mdev = torch.from_numpy(mask.view(np.int32)).cuda()
        mp.mp_merge_ties_tau(L, base_d, sel, mdev, tau_d, 1.0, out, delta=True)
        torch.cuda.synchronize()
        want = to_host(out)
        got = _fused(mp, spec, recs, ads_d, base_d, mask, tau_d, 1.0, K)
        assert np.array_equal(got, want), f"f={f}: {int((got != want).sum())} elements differ"


def test_lora_fused_ties_without_records_and_bad_arguments(mp):
    import torch
    spec = _awkward("bf16")
    lay = spec.layout
    K = 2
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    base_np, _ = make_family(spec, K=1, seed=7)
    base_d = to_dev(base_np, "bf16")
    mask = np.random.default_rng(7).integers(0, 4, blocks.G).astype(np.uint32)
    tau = np.full(blocks.G * K, 0x3c000000, np.uint32)
    tau_d = torch.from_numpy(tau.view(np.int32)).cuda()
    _say("case lora fused no records")
    got = _fused(mp, spec, [], None, base_d, mask, tau_d, 0.5, K)
    zeros = [np.zeros(lay.n_params, np.uint16) for _ in range(K)]
    want = oracle.merge_ties_tau(blocks, "bf16", base_np, zeros, mask, tau.reshape(blocks.G, K), 0.5, delta=True)
    assert np.array_equal(got, want)
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    mdev = torch.from_numpy(mask.view(np.int32)).cuda()
    recs, n = lora_records(spec, 8, 1.0, targets=("w0", "w5"))
    ads = [torch.zeros(n, dtype=torch.bfloat16, device="cuda") for _ in range(K)]
    out = torch.empty_like(base_d)
    with pytest.raises(mp.MPError) as e:  # w5: 44 bf16 columns, rows not whole 16-byte chunks
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads, mdev, tau_d, 1.0, out)
    assert e.value.code == mp.MP_E_UNSUPPORTED
    recs, n = lora_records(spec, 8, 1.0, targets=("w0",))
    with pytest.raises(mp.MPError) as e:  # out is the base
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads, mdev, tau_d, 1.0, base_d)
    assert e.value.code == mp.MP_E_ARG
    with pytest.raises(mp.MPError) as e:  # thresholds in host memory
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads, mdev, torch.from_numpy(tau.view(np.int32)), 1.0, out)
    assert e.value.code == mp.MP_E_ARG
    with pytest.raises(mp.MPError) as e:
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads, mdev, tau_d, float("nan"), out)
    assert e.value.code == mp.MP_E_ARG


def test_lora_fused_fullsize_qwen_layout(mp):
    # The Qwen2.5-1.5B layout with rank-16 adapters on every projection, four
    # experts, in the launch configuration the benchmark times: catalog from
    # the full pull, skip-zero plans at two budgets, then the fused merge.
    # Dyadic adapters keep every delta exact, so the whole output equals the
    # two-call route and whole tensors equal the oracle (thresholds included).
    import torch
    spec = family_spec("qwen2.5-1.5b")
    lay = spec.layout
    K = 4
    P = lay.n_params
    recs, n = lora_records(spec, 16, 2.0)
    ads_np = make_lora_adapters(n, K, "bf16", seed=23, grid=True)
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    G = mp.mp_layout_blocks(L)
    base, ex = make_family_device(spec, K=1, seed=5)
    del ex
    ads = [to_dev(a, "bf16") for a in ads_np]
    deltas = [torch.empty(P, dtype=torch.bfloat16, device="cuda") for _ in range(K)]
    _say("case lora fused fullsize: catalog")
    mp.mp_lora_materialize(L, recs, ads, deltas)
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mp.mp_index_ties(L, base, deltas, 0.2, tau, sumsq=sumsq, delta=True)
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    out2 = torch.empty_like(base)
    names = [nm for nm, _ in spec.tensors]
    toff = np.concatenate([[0], np.cumsum(lay.numel)]).astype(np.int64)
    nblk = [(int(x) + lay.block_elems - 1) // lay.block_elems for x in lay.numel]
    g0s = np.concatenate([[0], np.cumsum(nblk)]).astype(np.int64)
    by_t = {r[0]: r for r in recs}
    picks = [names.index(x) for x in ("layers.0.self_attn.q_proj.weight", "layers.13.mlp.down_proj.weight",
                                      "layers.27.self_attn.v_proj.weight", "layers.27.mlp.up_proj.weight",
                                      "norm.weight")]
    tau_h = tau.cpu().numpy().view(np.uint32).reshape(G, K)
    for f in (0.25, 1.0):
        _say(f"case lora fused fullsize B={f}")
        mp.mp_plan(L, K, sumsq, [1.0] * K, int(f * P * 2 * K), mask, flags=mp.MP_PLAN_SKIP_ZERO)
        mp.mp_lora_merge_ties_tau(L, base, recs, ads, mask, tau, 1.0, out)
        mp.mp_lora_materialize(L, recs, ads, deltas, mask=mask)
        mp.mp_merge_ties_tau(L, base, deltas, mask, tau, 1.0, out2, delta=True)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), out2.view(torch.int16)), "fused and two-call outputs differ"
        mask_h = mask.cpu().numpy().view(np.uint32)
        for t in picks:
            a, b = int(toff[t]), int(toff[t + 1])
            sub = oracle.Blocks([b - a], lay.block_elems)
            b_np = to_host(base[a:b])
            if t in by_t:
                _, rows, cols, r, a_off, b_off, sc = by_t[t]
                d_t = [oracle.lora_delta("bf16", rows, cols, ads_np[i][a_off:a_off + r * cols].reshape(r, cols),
                                         ads_np[i][b_off:b_off + rows * r].reshape(rows, r), sc) for i in range(K)]
            else:
                d_t = [np.zeros(b - a, np.uint16) for _ in range(K)]
            g0, g1 = int(g0s[t]), int(g0s[t + 1])
            tau_t = oracle.ties_thresholds(sub, "bf16", b_np, d_t, 0.2, delta=True)
            assert np.array_equal(tau_h[g0:g1], tau_t), f"{names[t]}: thresholds differ from the oracle's"
            want = oracle.merge_ties_tau(sub, "bf16", b_np, d_t, mask_h[g0:g1], tau_t, 1.0, delta=True)
            got = to_host(out[a:b])
            assert np.array_equal(got, want), f"{names[t]} B={f}: {int((got != want).sum())} elements differ"


def test_lora_fused_two_streams_and_workspace_cap(mp):
    # Two fused merges with one layout and record set but different adapters,
    # issued on two streams with no synchronisation between them: they share
    # the table's operand-order copies, so the second call's copy must wait
    # for the first call's merge.  Then a workspace cap: MP_E_NOMEM before
    # anything is enqueued, the output untouched.
    import torch
    spec = _awkward("bf16")
    lay = spec.layout
    K = 3
    recs, n = lora_records(spec, 16, 0.5, targets=_fused_targets("bf16"))
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    L = mp.Layout(lay.numel, lay.block_elems, lay.dtype_code)
    base_np, _ = make_family(spec, K=1, seed=51)
    base_d = to_dev(base_np, "bf16")
    rng = np.random.default_rng(51)
    cases = []
    for j in range(2):
        ads = make_lora_adapters(n, K, "bf16", seed=60 + j, grid=True)
        d_full = oracle.lora_materialize(blocks, "bf16", lay.numel, recs, ads)
        tau = oracle.ties_thresholds(blocks, "bf16", base_np, d_full, 0.2, delta=True)
        mask = rng.integers(0, 8, blocks.G).astype(np.uint32)
        want = oracle.merge_ties_tau(blocks, "bf16", base_np, d_full, mask, tau, 1.0, delta=True)
        cases.append(([to_dev(a, "bf16") for a in ads],
                      torch.from_numpy(mask.view(np.int32)).cuda(),
                      torch.from_numpy(np.ascontiguousarray(tau, np.uint32).reshape(-1).view(np.int32)).cuda(),
                      torch.empty_like(base_d), want))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    _say("case lora fused two streams")
    for (ads_d, m_d, t_d, out, _), st in zip(cases, streams):
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads_d, m_d, t_d, 1.0, out, stream=st)
    torch.cuda.synchronize()
    for j, (_, _, _, out, want) in enumerate(cases):
        got = to_host(out)
        assert np.array_equal(got, want), f"stream {j}: {int((got != want).sum())} elements differ"
    _say("case lora fused workspace cap")
    ads_d, m_d, t_d, _, want = cases[0]
    try:
        mp.mp_release()
        mp.mp_set_workspace_limit(1)
        out = torch.full_like(base_d, 3.0)
        before = out.clone()
        with pytest.raises(mp.MPError) as ei:
            mp.mp_lora_merge_ties_tau(L, base_d, recs, ads_d, m_d, t_d, 1.0, out)
        assert ei.value.code == mp.MP_E_NOMEM
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), before.view(torch.int16))
        mp.mp_set_workspace_limit(0)
        mp.mp_lora_merge_ties_tau(L, base_d, recs, ads_d, m_d, t_d, 1.0, out)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(out), want)
    finally:
        mp.mp_set_workspace_limit(0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_lora_fused_and_pulls_with_32_experts(mp, dtype):
    # The widest expert set (K = 32: every bit of a mask word is an expert):
    # the full and masked pulls on the operand-order copy and the fused
    # merge, against the oracle on the dyadic grid.
    import torch
    spec = _awkward(dtype)
    lay = spec.layout
    K = 32
    recs, n = lora_records(spec, 8, 0.5, targets=_fused_targets(dtype))
    ads = make_lora_adapters(n, K, dtype, seed=320, grid=True)
    base_np, _ = make_family(spec, K=1, seed=320)
    blocks = oracle.Blocks(lay.numel, lay.block_elems)
    rng = np.random.default_rng(320)
    mask = rng.integers(0, 1 << 32, blocks.G, dtype=np.uint64).astype(np.uint32)
    mask[::7] = 0xFFFFFFFF
    mask[3::7] = 0
    _say(f"case lora K=32 {dtype} pulls")
    d_full = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads)
    _, outs = _materialize(mp, spec, recs, ads)
    for i in (0, 17, 31):
        assert np.array_equal(to_host(outs[i]), d_full[i]), f"full pull, expert {i}"
    fill = [_sentinel(lay.n_params, dtype, i) for i in range(K)]
    _, outs = _materialize(mp, spec, recs, ads, mask)
    want = oracle.lora_materialize(blocks, dtype, lay.numel, recs, ads, mask=mask, fill=fill)
    for i in (0, 5, 17, 31):
        assert np.array_equal(to_host(outs[i]), want[i]), f"masked pull, expert {i}"
    del outs
    _say(f"case lora K=32 {dtype} fused")
    tau = oracle.ties_thresholds(blocks, dtype, base_np, d_full, 0.3, delta=True)
    tau_d = torch.from_numpy(np.ascontiguousarray(tau, np.uint32).reshape(-1).view(np.int32)).cuda()
    got = _fused(mp, spec, recs, [to_dev(a, dtype) for a in ads], to_dev(base_np, dtype), mask, tau_d, 0.9, K)
    want = oracle.merge_ties_tau(blocks, dtype, base_np, d_full, mask, tau, 0.9, delta=True)
    assert assert_merge_equal(got, want, base_np, dtype, "fused K=32") == 0
