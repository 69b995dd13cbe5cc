"""The plan entry point that allocates nothing (mp_plan_noalloc), through the
C ABI, against mp_plan on the same inputs: masks and stats bit for bit, on
two calls in a row, the second over a smaller layout, so nothing of the
first call's contents of the fixed device array may leak into it."""

import sys

import numpy as np
import pytest

import oracle
from workloads import family_spec

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


def _compare(mp, L, K, sumsq, w, B, flags, blocks=None, S=None):
    import torch
    G = int(sum((n + L.block_elems - 1) // L.block_elems for n in L.numel))
    m1 = torch.full((G,), -1, dtype=torch.int32, device="cuda")
    m2 = torch.full((G,), -7, dtype=torch.int32, device="cuda")
    st1 = mp.mp_plan(L, K, sumsq, w, B, m1, flags=flags)
    st2 = mp.mp_plan_noalloc(L, K, sumsq, w, B, m2, flags=flags)
    assert torch.equal(m1, m2), f"mask differs at B={B} flags={flags}"
    assert st1 == st2, (st1, st2)
    if blocks is not None:
        m_orc, st_orc = oracle.plan(blocks, "bf16", K, S, w, B, flags=flags)
        assert np.array_equal(m2.cpu().numpy().view(np.uint32), m_orc)
        assert st2["cost_bytes"] == st_orc["cost"] and st2["digest"] == st_orc["digest"]
    return st2


def test_plan_noalloc_equals_plan_on_two_calls(mp):
    import torch
    # call 1: the Qwen2.5-1.5B-shaped layout at full size (376,989 blocks, K = 4)
    lay = family_spec("qwen2.5-1.5b").layout
    L = mp.Layout(lay.numel, lay.block_elems, mp.MP_BF16)
    K = 4
    G = len(lay.block_lengths())
    rng = np.random.default_rng(61)
    S = rng.lognormal(-14.0, 2.0, G * K).astype(np.float32)
    S[rng.random(G * K) < 0.2] = 0.0
    sumsq = torch.from_numpy(S).cuda()
    full = lay.n_params * 2 * K
    for f in (0.25, 0.5, 1.0):
        st = _compare(mp, L, K, sumsq, [1.0] * K, int(f * full), 0)
        _say(f"  full layout B={f}: cost={st['cost_bytes']} sel={st['n_selected']}")
    # call 2: a smaller layout with ten block lengths (many plan rounds),
    # K = 5, sums of squares with ties and zeros, every flag, and the
    # fallback without a catalog
    numel = [4096 * 3 + 64, 4096 + 512, 2048, 1024 + 256, 4096 * 2 + 1536, 768, 4096, 384, 128, 4096 + 2560]
    L2 = mp.Layout(numel, 4096, mp.MP_BF16)
    blocks = oracle.Blocks(numel, 4096)
    K2 = 5
    S2 = rng.choice(np.array([0.0, 1e-4, 2.5e-3, 2.5e-3, 7e-2, 1.0, 3.0], np.float32), size=blocks.G * K2)
    s2 = torch.from_numpy(S2).cuda()
    full2 = int(blocks.len.sum()) * 2 * K2
    for flags in (0, mp.MP_PLAN_PER_BYTE, mp.MP_PLAN_SKIP_ZERO, 3):
        for w in ([1.0] * K2, [0.5, 1.0, 1.0, 0.25, 2.0]):
            for B in (0, 129, full2 // 7, full2 // 2, full2 - 1, full2, full2 + 5):
                _compare(mp, L2, K2, s2, w, B, flags, blocks, S2)
    for B in (full2 // 3, full2):
        _compare(mp, L2, K2, None, [1.0, 2.0, 1.0, 1.0, 0.5], B, 0, blocks, None)
    _say("  small layout: every flag, budget and the fallback equal")
