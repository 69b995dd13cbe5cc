"""Pins for the CPU oracle: published values, closed forms, invariants the
paper proves, special cases and brute force on tiny inputs.

None of these compares the oracle with a re-typed copy of itself; each fails
for a plausible mistake (a dropped term, a wrong sign or index, a transposed
operand, the wrong greedy semantics, a wrong tie-break).
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _bits_bf16(x):
    return oracle.round_bf16(np.asarray(x, np.float32))


def _f32_of_bf16(u16):
    return (np.asarray(u16, np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# building blocks: published known answers
# --------------------------------------------------------------------------

def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLD, "philox4x32_10_kat.txt")) if l.strip() and l[0] != "#"]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        got = oracle.philox4x32_10(v[0:4], v[4:6])
        assert [int(x) for x in got] == v[6:10]


def test_splitmix64_published_outputs():
    want = [int(l, 16) for l in open(os.path.join(GOLD, "splitmix64_seed0.txt")) if l.strip() and l[0] != "#"]
    gamma = 0x9E3779B97F4A7C15
    got = [oracle.mix64((n * gamma) & (2**64 - 1)) for n in range(len(want))]
    assert got == want


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * np.float32(0.02),
        rng.standard_normal(1000).astype(np.float32) * np.float32(1e30),
        rng.standard_normal(1000).astype(np.float32) * np.float32(1e-38),  # subnormal range
        np.array([0.0, -0.0, 1.0, 1.00390625, 1.0078125, 1.01171875, -1.00390625, 3.0e38], np.float32),
    ])
    # exact halfway cases: mantissa low 16 bits == 0x8000
    u = rng.integers(0, 2**32, 5000, dtype=np.uint64).astype(np.uint32)
    u = (u & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    u = u[(u & np.uint32(0x7F800000)) != np.uint32(0x7F800000)]
    x = np.concatenate([x, u.view(np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.round_bf16(x)
    assert np.array_equal(got, want)


def test_ties_k_rounding():
    assert oracle.ties_k(4096, 0.2) == 820  # 819.2 -> 820
    assert oracle.ties_k(4096, 0.1) == 410  # 409.6 -> 410
    assert oracle.ties_k(4096, 0.25) == 1024  # exact, no ceil bump
    assert oracle.ties_k(4096, 1.0) == 4096
    assert oracle.ties_k(4096, 0.0) == 0
    assert oracle.ties_k(256, 0.2) == 52  # 51.2
    assert oracle.ties_k(1536, 0.2) == 308  # 307.2


# --------------------------------------------------------------------------
# Section 2: block partition
# --------------------------------------------------------------------------

def test_block_partition_is_disjoint_and_tensor_local():
    numel = [8192, 1536, 256, 4096 * 3 + 8, 8, 4096]
    b = oracle.Blocks(numel, 4096)
    # closed-form count: sum of ceilings
    assert b.G == sum(-(-n // 4096) for n in numel) == 2 + 1 + 1 + 4 + 1 + 1
    # blocks tile [0, P) in order with no gap/overlap
    assert b.off[0] == 0
    assert np.array_equal(b.off[1:], b.off[:-1] + b.len[:-1])
    assert b.off[-1] + b.len[-1] == sum(numel)
    starts = np.concatenate([[0], np.cumsum(numel)[:-1]])
    for g in range(b.G):
        t = b.tensor[g]
        assert starts[t] <= b.off[g] and b.off[g] + b.len[g] <= starts[t] + numel[t]
        assert b.elem0[g] == b.off[g] - starts[t]
        assert b.elem0[g] % 4096 == 0
        # only the last block of a tensor may be short
        if b.len[g] < 4096:
            assert b.off[g] + b.len[g] == starts[t] + numel[t]


@pytest.mark.parametrize("name,G,short", [
    ("qwen2.5-1.5b", 376989, 141), ("llama3-8b", 1960513, 0), ("qwen2.5-7b", 1859341, 141), ("toy", 1024, 0)])
def test_block_counts_of_the_workload_shapes(name, G, short):
    from workloads import family_spec
    lay = family_spec(name).layout
    b = oracle.Blocks(lay.numel, lay.block_elems)
    assert b.G == G
    assert int((b.len < lay.block_elems).sum()) == short


# --------------------------------------------------------------------------
# index: canonical fp32 sum of squares
# --------------------------------------------------------------------------

def _blocks_for(numel, be=4096):
    return oracle.Blocks(numel, be)


def test_index_closed_form_constant_delta():
    # bf16: base 0.5, expert 0.5 + 2^-8 -> d = 2^-8 exactly, S = n * 2^-16 exactly
    numel = [4096, 1536, 256, 4096]
    b = _blocks_for(numel)
    P = sum(numel)
    base = _bits_bf16(np.full(P, 0.5))
    ex = _bits_bf16(np.full(P, 0.5 + 2**-8))
    S = oracle.index(b, "bf16", base, [ex, base])
    assert np.array_equal(S[:, 0], (b.len * 2.0**-16).astype(np.float32))
    assert np.all(S[:, 1] == 0.0)
    # fp32: d = 2^-10 -> S = n * 2^-20
    base32 = np.full(P, 0.25, np.float32)
    S32 = oracle.index(b, "f32", base32, [base32 + np.float32(2**-10), base32 - np.float32(2**-10)])
    assert np.array_equal(S32[:, 0], (b.len * 2.0**-20).astype(np.float32))
    assert np.array_equal(S32[:, 1], S32[:, 0])  # sign of the delta does not matter


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_index_counts_every_position_once(dtype):
    # 128 blocks x 32 experts: expert k of block g carries one nonzero delta at
    # position (g*32 + k) of its block, so all 4096 positions are hit once.
    nblk, K = 128, 32
    b = _blocks_for([4096] * nblk)
    P = 4096 * nblk
    base = np.zeros(P, np.float32)
    exps = []
    vals = np.zeros((nblk, K), np.float64)
    for k in range(K):
        e = np.zeros(P, np.float32)
        for g in range(nblk):
            pos = g * K + k
            v = np.float32(1.0 + (pos % 7) / 8.0) * np.float32(2.0 ** -(pos % 5))
            e[g * 4096 + pos] = v
            vals[g, k] = float(v) ** 2
        exps.append(e)
    if dtype == "bf16":
        base = _bits_bf16(base)
        exps = [_bits_bf16(e) for e in exps]
    S = oracle.index(b, dtype, base, exps)
    assert np.array_equal(S.astype(np.float64), vals)


def test_index_short_block_tail_positions():
    # short blocks (1536, 256 elements): a nonzero at each tail position is counted
    for n in (1536, 256, 8, 24):
        b = _blocks_for([n], 4096)
        for pos in sorted({0, n - 1, n // 2, max(0, n - 8)}):
            base = np.zeros(n, np.float32)
            e = base.copy()
            e[pos] = 3.0
            S = oracle.index(b, "f32", base, [e])
            assert S[0, 0] == 9.0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_index_within_rounding_bound_of_exact(dtype):
    from workloads import family_spec, make_family
    spec = family_spec("qwen2.5-1.5b", n_layers=1, vocab=64)
    lay = spec.layout
    base, exps = make_family(spec, K=3, seed=5)
    if dtype == "f32":
        base = _f32_of_bf16(base)
        exps = [_f32_of_bf16(e) for e in exps]
    b = oracle.Blocks(lay.numel, lay.block_elems)
    S = oracle.index(b, dtype, base, exps).astype(np.float64)
    b32 = base.astype(np.float32) if dtype == "f32" else _f32_of_bf16(base)
    u = 2.0**-24
    for i, e in enumerate(exps):
        e32 = e if dtype == "f32" else _f32_of_bf16(e)
        d = (e32 - b32).astype(np.float64)  # the fp32 subtraction is exact here? use fp32 result
        d = (e32 - b32).astype(np.float32).astype(np.float64)
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            exact = float(np.sum(d[o:o + n] ** 2))
            V = 4 if dtype == "f32" else 8
            chain = -(-n // (64 * V)) * V + 6
            gam = chain * u / (1 - chain * u)
            assert abs(S[g, i] - exact) <= gam * exact + 1e-45


def test_index_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(3)
    b = _blocks_for([4096, 4096, 520])
    P = 4096 * 2 + 520
    base = rng.standard_normal(P).astype(np.float32)
    d = (rng.standard_normal(P) * 1e-3).astype(np.float32)
    S1 = oracle.index(b, "f32", np.zeros(P, np.float32), [d])
    S2 = oracle.index(b, "f32", np.zeros(P, np.float32), [d * np.float32(2.0)])
    assert np.array_equal(S2, S1 * np.float32(4.0))


# --------------------------------------------------------------------------
# Algorithm 1 (PlanGen)
# --------------------------------------------------------------------------

def test_plan_worked_example():
    ex = json.load(open(os.path.join(GOLD, "plan_worked_example.json")))
    b = oracle.Blocks(ex["numel"], ex["block_elems"])
    assert list(b.len * 4) == ex["block_cost_bytes"]
    K = ex["K"]
    S = np.array(ex["sumsq"], np.float32)
    for c in ex["cases"]:
        mask, st = oracle.plan(b, ex["dtype"], K, S, c["w"], c["budget"])
        assert list(mask) == c["mask"], c["notes"]
        assert st["cost"] == c["cost"] and st["n_selected"] == c["n_selected"]
        assert st["full_bytes"] == 160 and st["n_units"] == 6
        # digest definition: mix64(sum_g mix64(g<<32 | mask_g) xor cost)
        D = sum(oracle.mix64((g << 32) | int(m)) for g, m in enumerate(mask)) & (2**64 - 1)
        assert st["digest"] == oracle.mix64(D ^ st["cost"])


def test_plan_per_byte_worked_example():
    # Per-byte scores (flag 1): fp32 blocks of 8, 2 and 2 elements cost 32, 8
    # and 8 bytes; K = 1, S = (4, 3, 2.5), w = 1.  Plain scores 4 > 3 > 2.5
    # put the big block first; per-byte scores 4/32 = 0.125, 3/8 = 0.375,
    # 2.5/8 = 0.3125 put it last.
    b = oracle.Blocks([8, 2, 2], 8)
    S = np.array([4.0, 3.0, 2.5], np.float32)
    for B, plain, per_byte in ((32, [1, 0, 0], [0, 1, 1]), (40, [1, 1, 0], [0, 1, 1]),
                               (48, [1, 1, 1], [1, 1, 1]), (12, [0, 1, 0], [0, 1, 0])):
        m0, st0 = oracle.plan(b, "f32", 1, S, [1.0], B)
        m1, st1 = oracle.plan(b, "f32", 1, S, [1.0], B, flags=1)
        assert list(m0) == plain and list(m1) == per_byte
        assert st1["cost"] == sum(c for c, t in zip((32, 8, 8), per_byte) if t) <= B
        assert st1["n_units"] == 3 and st1["full_bytes"] == 48


def test_plan_per_byte_with_uniform_power_of_two_costs_is_the_plain_plan():
    # dividing every score by the same power of two (exact for normal
    # values) keeps the order, so the mask is the plain one
    rng = np.random.default_rng(31)
    for trial in range(60):
        G, K = int(rng.integers(1, 40)), int(rng.integers(1, 6))
        b = oracle.Blocks([16] * G, 16)
        S = (rng.integers(0, 5, G * K) * rng.random(G * K) + 1e-3).astype(np.float32)
        S[rng.random(G * K) < 0.2] = 0.0
        w = (rng.random(K) + 0.5).astype(np.float32)
        full = 16 * 4 * G * K
        for B in (0, 64, full // 3, full // 2, full):
            m0, st0 = oracle.plan(b, "f32", K, S, w, B)
            m1, st1 = oracle.plan(b, "f32", K, S, w, B, flags=1)
            assert np.array_equal(m0, m1) and st0 == st1


def test_plan_skip_zero_drops_exactly_the_zero_units():
    # Units with S = 0 score 0 and come last in the plain order, so the
    # greedy decides every positive unit the same way with or without them:
    # flag 2's mask is the plain mask without the zero units, at any budget.
    rng = np.random.default_rng(37)
    for trial in range(200):
        G, K = int(rng.integers(1, 15)), int(rng.integers(1, 5))
        b = oracle.Blocks(list(rng.choice([16, 8, 4, 12], size=G)), 16)
        S = (rng.random(G * K) * 10 + 0.01).astype(np.float32)
        S[rng.random(G * K) < 0.3] = 0.0
        w = (rng.random(K) + 0.5).astype(np.float32)
        full = int(b.len.sum()) * 4 * K
        B = int(rng.integers(0, full + 20))
        m0, st0 = oracle.plan(b, "f32", K, S, w, B)
        m2, st2 = oracle.plan(b, "f32", K, S, w, B, flags=2)
        zero = np.zeros(G, np.uint32)
        for u in np.nonzero(S == 0)[0]:
            zero[u // K] |= np.uint32(1 << (u % K))
        assert np.array_equal(m2, m0 & ~zero)
        cost = sum(int(b.len[g]) * 4 for g in range(G) for i in range(K) if (int(m2[g]) >> i) & 1)
        assert st2["cost"] == cost and st2["n_selected"] == int(sum(bin(int(x)).count("1") for x in m2))
        assert st2["full_bytes"] == full and st2["n_units"] == G * K
    # all-zero experts: nothing is a candidate
    m, st = oracle.plan(oracle.Blocks([16], 16), "f32", 2, np.zeros(2, np.float32), [1.0, 1.0], 10**6, flags=2)
    assert int(m[0]) == 0 and st["cost"] == 0 and st["n_selected"] == 0


def test_plan_tensor_fallback_worked_examples():
    # Section 3's tensor-level fallback, hand-worked cases
    ex = json.load(open(os.path.join(GOLD, "plan_tensor_fallback.json")))
    b = oracle.Blocks(ex["numel"], ex["block_elems"])
    for c in ex["cases"]:
        m, st = oracle.plan(b, ex["dtype"], c["K"], None, c["w"], c["budget"], flags=c["flags"])
        assert [int(x) for x in m] == c["mask"], c["name"]
        assert st["cost"] == c["cost"] and st["n_selected"] == c["n_selected"], c["name"]
        assert st["full_bytes"] == c["full_bytes"] and st["n_units"] == b.G * c["K"]
        D = sum(oracle.mix64((g << 32) | int(m[g])) for g in range(b.G)) % (1 << 64)
        assert st["digest"] == oracle.mix64(D ^ st["cost"])


def _block_units_fallback(b, K, w, budget, s):
    # planted mistake: the greedy over (expert, block) units with statistic 1
    order = sorted(range(b.G * K), key=lambda u: (-(np.float32(w[u % K]) * np.float32(w[u % K])), u))
    m = np.zeros(b.G, np.uint32)
    C = 0
    for u in order:
        c = int(b.len[u // K]) * s
        if C + c <= budget:
            m[u // K] |= np.uint32(1 << (u % K))
            C += c
    return m


def test_plan_tensor_fallback_never_splits_a_tensor_and_is_sound():
    # At every budget: each tensor's blocks carry one selection word (no
    # tensor is split), C(A) <= B (Prop. 1), and every unselected (expert,
    # tensor) unit overflows the final cost (skip-and-continue).  Ranking:
    # a heavier expert's tensor before a lighter one's; equal weights in
    # tensor order.  The block-unit greedy fails the first property.
    rng = np.random.default_rng(71)
    split_seen = False
    for trial in range(60):
        T = int(rng.integers(1, 7))
        numel = [int(x) * 4 for x in rng.integers(0, 9, T)]
        be = 8
        b = oracle.Blocks(numel, be)
        K = int(rng.integers(1, 5))
        w = [float(x) for x in rng.choice([0.5, 1.0, 1.0, 2.0], K)]
        flags = int(rng.integers(0, 4))
        full = sum(numel) * 4 * K
        for B in sorted(set([0, full, full + 1] + [int(x) for x in rng.integers(0, full + 1, 8)])):
            m, st = oracle.plan(b, "f32", K, None, w, B, flags=flags)
            assert st["cost"] <= B
            words = {}
            for g in range(b.G):
                words.setdefault(int(b.tensor[g]), set()).add(int(m[g]))
            assert all(len(v) == 1 for v in words.values())
            tsel = {t: v.pop() for t, v in words.items()}
            cost = sum(numel[t] * 4 * bin(x).count("1") for t, x in tsel.items())
            assert cost == st["cost"]
            for t, x in tsel.items():
                for i in range(K):
                    if not (x >> i) & 1:
                        assert st["cost"] + numel[t] * 4 > B
            bad = _block_units_fallback(b, K, w, B, 4)
            for t in range(T):
                gs = [g for g in range(b.G) if b.tensor[g] == t]
                if len(set(int(bad[g]) for g in gs)) > 1:
                    split_seen = True
    assert split_seen  # the planted block-unit greedy does split tensors


def test_plan_tensor_fallback_weight_order():
    # Equal tensor sizes: with weights (1, 2) every tensor of expert 1 comes
    # before any tensor of expert 0, and within an expert tensors go in
    # layout order, so a budget of n tensors selects expert 1's first n.
    numel = [32] * 5
    b = oracle.Blocks(numel, 8)
    c = 32 * 2
    for n in range(0, 11):
        m, st = oracle.plan(b, "bf16", 2, None, [1.0, 2.0], n * c + c // 2)
        t_e1 = [t for t in range(5) if (int(m[4 * t]) >> 1) & 1]
        t_e0 = [t for t in range(5) if int(m[4 * t]) & 1]
        assert t_e1 == list(range(min(n, 5)))
        assert t_e0 == list(range(max(0, n - 5)))
        assert st["cost"] == n * c


def _random_plan_case(rng, G, K, uniform, ties=False):
    if uniform:
        numel = [16] * G
    else:
        numel = list(rng.choice([16, 8, 4, 12], size=G))
    b = oracle.Blocks(numel, 16)
    if ties:
        S = rng.integers(0, 3, size=G * K).astype(np.float32)
    else:
        S = (rng.random(G * K) * 10).astype(np.float32)
        S[rng.random(G * K) < 0.2] = 0.0
    w = (rng.random(K) + 0.5).astype(np.float32)
    return b, S, w


def test_plan_budget_soundness_and_maximality():
    # Prop. 1: C(A) <= B.  Skip-and-continue greedy: every unselected unit
    # overflows the final cost.
    rng = np.random.default_rng(7)
    for trial in range(300):
        G, K = int(rng.integers(1, 12)), int(rng.integers(1, 5))
        b, S, w = _random_plan_case(rng, G, K, uniform=bool(trial % 2), ties=bool(trial % 3 == 0))
        full = int(b.len.sum()) * 4 * K
        B = int(rng.integers(0, full + 20))
        mask, st = oracle.plan(b, "f32", K, S, w, B)
        cost = sum(int(b.len[g]) * 4 for g in range(b.G) for i in range(K) if (mask[g] >> i) & 1)
        assert cost == st["cost"] <= B
        assert st["full_bytes"] == full
        for g in range(b.G):
            for i in range(K):
                if not (mask[g] >> i) & 1:
                    assert st["cost"] + int(b.len[g]) * 4 > B
        if B >= full:
            assert np.all(mask == (1 << K) - 1)


def test_plan_uniform_costs_brute_force_optimal():
    # Eq. 6 with equal costs: the greedy maximises the retained score, the
    # cost is floor(B/c)*c, and the selected set is the top of the
    # (score desc, uid asc) order.
    rng = np.random.default_rng(11)
    for trial in range(120):
        G, K = int(rng.integers(1, 5)), int(rng.integers(1, 4))
        nu = G * K
        if nu > 12:
            continue
        b, S, w = _random_plan_case(rng, G, K, uniform=True, ties=bool(trial % 2))
        c = 64
        B = int(rng.integers(0, nu * c + 1))
        mask, st = oracle.plan(b, "f32", K, S, w, B)
        m = min(B // c, nu)
        assert st["cost"] == m * c and st["n_selected"] == m
        score = [float(np.float32(np.float32(w[u % K] * w[u % K]) * S[u])) for u in range(nu)]
        best = 0.0
        for r in range(m + 1):
            for comb in itertools.combinations(range(nu), r):
                best = max(best, sum(score[u] for u in comb))
        got = sum(score[u] for u in range(nu) if (mask[u // K] >> (u % K)) & 1)
        assert math.isclose(got, best, rel_tol=1e-12, abs_tol=1e-12)
        order = sorted(range(nu), key=lambda u: (-score[u], u))
        sel = {u for u in range(nu) if (mask[u // K] >> (u % K)) & 1}
        assert sel == set(order[:m])


def test_plan_ties_prefer_lower_uid():
    b = oracle.Blocks([16] * 3, 16)
    S = np.ones(6, np.float32)
    for m in range(7):
        mask, st = oracle.plan(b, "f32", 2, S, [1.0, 1.0], m * 64)
        sel = [u for u in range(6) if (mask[u // 2] >> (u % 2)) & 1]
        assert sel == list(range(m))


def test_plan_digest_sensitive_to_every_bit():
    b = oracle.Blocks([16] * 5, 16)
    rng = np.random.default_rng(2)
    S = rng.random(20).astype(np.float32)
    _, st0 = oracle.plan(b, "f32", 4, S, [1, 1, 1, 1], 5 * 64)
    digests = {st0["digest"]}
    for u in range(20):
        S2 = S.copy()
        S2[u] = 100.0  # forces u into the selection, changing the mask
        m2, st2 = oracle.plan(b, "f32", 4, S2, [1, 1, 1, 1], 5 * 64)
        digests.add(st2["digest"])
    assert len(digests) > 15


# --------------------------------------------------------------------------
# AVG
# --------------------------------------------------------------------------

def _tiny_family(rng, numel, K, dtype="f32", scale=1e-2):
    P = sum(numel)
    base = rng.standard_normal(P).astype(np.float32) * np.float32(0.02)
    exps = [base + (rng.standard_normal(P) * scale).astype(np.float32) for _ in range(K)]
    if dtype == "bf16":
        base = _bits_bf16(base)
        exps = [_bits_bf16(e) for e in exps]
    return base, exps


def test_avg_empty_mask_is_base_bitwise():
    rng = np.random.default_rng(0)
    for dtype in ("f32", "bf16"):
        numel = [4096, 1536, 256]
        b = oracle.Blocks(numel, 4096)
        base, exps = _tiny_family(rng, numel, 3, dtype)
        out = oracle.merge_avg(b, dtype, base, exps, np.zeros(b.G, np.uint32), [1 / 3] * 3)
        assert np.array_equal(out, base)


def test_avg_one_hot_alpha_reproduces_that_expert():
    rng = np.random.default_rng(1)
    numel = [4096, 1536, 256, 4096]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 4, "bf16", scale=1e-3)
    full = np.full(b.G, 15, np.uint32)
    for i in range(4):
        a = np.zeros(4, np.float32)
        a[i] = 1.0
        out = oracle.merge_avg(b, "bf16", base, exps, full, a)
        assert np.array_equal(out, exps[i]), i


def test_avg_closed_form_two_experts():
    rng = np.random.default_rng(2)
    numel = [4096, 520]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 2, "f32")
    out = oracle.merge_avg(b, "f32", base, exps, np.full(b.G, 3, np.uint32), [0.5, 0.5])
    want = base.astype(np.float64) + 0.5 * ((exps[0].astype(np.float64) - base) + (exps[1].astype(np.float64) - base))
    err = np.abs(out.astype(np.float64) - want)
    # each fp32 rounding is relative to the operand it rounds: x0, d_i, acc, y
    mag = np.maximum.reduce([np.abs(base), np.abs(exps[0] - base), np.abs(exps[1] - base),
                             np.abs(want).astype(np.float32)])
    assert np.all(err <= 4 * np.spacing(mag).astype(np.float64))


def test_avg_additive_identity_and_omission_bound_all_masks():
    # Prop. 2: M_full - M_A = sum_i (1-A_i) alpha_i Delta_i and
    # ||M_full - M_A|| <= sqrt(sum q^2) <= sum q, for every mask of a tiny
    # family.  Values are dyadic so every fp32 operation is exact and the
    # identity must hold with equality.
    rng = np.random.default_rng(3)
    numel = [8, 8, 4]
    b = oracle.Blocks(numel, 8)
    K = 3
    P = sum(numel)
    base = (rng.integers(-64, 64, P) / 1024.0).astype(np.float32)
    deltas = [(rng.integers(-16, 16, P) / 4096.0).astype(np.float32) for _ in range(K)]
    exps = [base + d for d in deltas]
    alpha = np.array([0.25, 0.5, 0.25], np.float32)
    full_mask = np.full(b.G, 7, np.uint32)
    Mf = oracle.merge_avg(b, "f32", base, exps, full_mask, alpha).astype(np.float64)
    nu = b.G * K
    for bits in range(1 << nu):
        A = np.array([[(bits >> (g * K + i)) & 1 for i in range(K)] for g in range(b.G)])
        mask = np.array([sum(int(A[g, i]) << i for i in range(K)) for g in range(b.G)], np.uint32)
        MA = oracle.merge_avg(b, "f32", base, exps, mask, alpha).astype(np.float64)
        diff = Mf - MA
        ident = np.zeros(P)
        q = np.zeros(b.G)
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            for i in range(K):
                if not A[g, i]:
                    ident[o:o + n] += float(alpha[i]) * deltas[i][o:o + n].astype(np.float64)
                    q[g] += abs(float(alpha[i])) * np.linalg.norm(deltas[i][o:o + n].astype(np.float64))
        assert np.array_equal(diff, ident)
        lhs = np.linalg.norm(diff)
        assert lhs <= math.sqrt(np.sum(q**2)) * (1 + 1e-12) + 1e-15
        assert math.sqrt(np.sum(q**2)) <= np.sum(q) * (1 + 1e-12) + 1e-15


def test_avg_non_anticipatory():
    # Section 2: the output depends only on the selected entries.
    rng = np.random.default_rng(4)
    numel = [4096, 1536, 256, 4096]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 4, "bf16")
    mask = rng.integers(0, 16, b.G).astype(np.uint32)
    out1 = oracle.merge_avg(b, "bf16", base, exps, mask, [0.25] * 4)
    junk = [e.copy() for e in exps]
    for g in range(b.G):
        for i in range(4):
            if not (mask[g] >> i) & 1:
                junk[i][b.off[g]:b.off[g] + b.len[g]] = rng.integers(0, 2**15, b.len[g]).astype(np.uint16)
    out2 = oracle.merge_avg(b, "bf16", base, junk, mask, [0.25] * 4)
    assert np.array_equal(out1, out2)


# --------------------------------------------------------------------------
# selected-only (renormalised) AVG, Appendix A.1's coefficient-drift variant
# --------------------------------------------------------------------------

def test_avg_renorm_single_selected_expert_is_that_expert():
    # With one selected expert a block's coefficient is alpha_i / alpha_i = 1
    # whatever alpha_i is, so the block is that expert's block; a block with
    # nothing selected is the base.
    rng = np.random.default_rng(21)
    numel = [4096, 1536, 256, 4096, 4096]
    b = oracle.Blocks(numel, 4096)
    for dtype in ("f32", "bf16"):
        base, exps = _tiny_family(rng, numel, 4, dtype, scale=1e-3)
        pick = rng.integers(-1, 4, b.G)
        mask = np.array([0 if i < 0 else 1 << i for i in pick], np.uint32)
        out = oracle.merge_avg_renorm(b, dtype, base, exps, mask, [0.3, 0.7, 0.1, 1.9])
        for g in range(b.G):
            sl = slice(b.off[g], b.off[g] + b.len[g])
            want = base[sl] if pick[g] < 0 else exps[pick[g]][sl]
            assert np.array_equal(out[sl], want), (dtype, g)


def test_avg_renorm_invariant_to_power_of_two_scaling_of_alpha():
    # beta = alpha_i / sum(selected alpha) is unchanged, exactly, when every
    # alpha is scaled by a power of two; plain AVG is not.
    rng = np.random.default_rng(22)
    numel = [4096, 1536, 256, 4096]
    b = oracle.Blocks(numel, 4096)
    for dtype in ("f32", "bf16"):
        base, exps = _tiny_family(rng, numel, 3, dtype)
        mask = rng.integers(0, 8, b.G).astype(np.uint32)
        alpha = np.array([0.3, 0.45, 0.11], np.float32)
        ref = oracle.merge_avg_renorm(b, dtype, base, exps, mask, alpha)
        for sc in (8.0, 1.0 / 16):
            got = oracle.merge_avg_renorm(b, dtype, base, exps, mask, alpha * np.float32(sc))
            assert np.array_equal(got, ref), (dtype, sc)
        plain = oracle.merge_avg(b, dtype, base, exps, mask, alpha * np.float32(8.0))
        assert not np.array_equal(plain, ref)


def test_avg_renorm_full_mask_with_unit_sum_is_avg():
    # alpha summing to exactly 1 in fp32 and every expert selected: beta =
    # alpha, so the selected-only merge is the (pinned) full-read AVG.
    rng = np.random.default_rng(23)
    numel = [4096, 1536, 256]
    b = oracle.Blocks(numel, 4096)
    for dtype, alpha in (("bf16", [0.125, 0.375, 0.5]), ("f32", [0.25, 0.25, 0.25, 0.25])):
        K = len(alpha)
        base, exps = _tiny_family(rng, numel, K, dtype)
        full = np.full(b.G, (1 << K) - 1, np.uint32)
        assert np.array_equal(oracle.merge_avg_renorm(b, dtype, base, exps, full, alpha),
                              oracle.merge_avg(b, dtype, base, exps, full, alpha))


def test_avg_renorm_is_a_convex_combination_of_the_selected_experts():
    # Positive alpha: the betas are positive and sum to 1 (to rounding), so
    # each output lies between the selected experts' values there.
    rng = np.random.default_rng(24)
    numel = [4096, 1536, 256, 4096]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 4, "f32")
    mask = rng.integers(1, 16, b.G).astype(np.uint32)
    out = oracle.merge_avg_renorm(b, "f32", base, exps, mask, [0.1, 0.2, 0.3, 0.4])
    for g in range(b.G):
        sl = slice(b.off[g], b.off[g] + b.len[g])
        sel = np.stack([exps[i][sl] for i in range(4) if (mask[g] >> i) & 1])
        lo, hi = sel.min(axis=0), sel.max(axis=0)
        tol = 4 * np.spacing(np.maximum(np.abs(lo), np.abs(hi)))
        assert np.all(out[sl] >= lo - tol) and np.all(out[sl] <= hi + tol), g


def test_avg_renorm_coefficient_drift_identity_and_bound_all_masks():
    # Appendix A.1: M_full - M_A = sum_i (alpha_i - beta_i(A)) Delta_i with
    # beta_i(A) = 0 where A_i = 0, and ||M_full - M_A|| <= (sum_b r_b^2)^(1/2),
    # r_b = sum_i |alpha_i - beta_i| ||Delta_i,b||.  beta is taken exactly
    # (fp64) from its definition; the oracle's fp32 rounding is the slack.
    rng = np.random.default_rng(25)
    numel = [8, 8, 4]
    b = oracle.Blocks(numel, 8)
    K = 3
    P = sum(numel)
    base = (rng.integers(-64, 64, P) / 1024.0).astype(np.float32)
    deltas = [(rng.integers(-16, 16, P) / 4096.0).astype(np.float32) for _ in range(K)]
    exps = [base + d for d in deltas]
    alpha = np.array([0.2, 0.5, 0.3], np.float32)
    Mf = oracle.merge_avg(b, "f32", base, exps, np.full(b.G, 7, np.uint32), alpha).astype(np.float64)
    mag = np.abs(base).astype(np.float64) + sum(np.abs(d).astype(np.float64) for d in deltas)
    slack = 8 * np.spacing(mag.astype(np.float32)).astype(np.float64)
    nu = b.G * K
    for bits in range(1 << nu):
        A = np.array([[(bits >> (g * K + i)) & 1 for i in range(K)] for g in range(b.G)])
        mask = np.array([sum(int(A[g, i]) << i for i in range(K)) for g in range(b.G)], np.uint32)
        MA = oracle.merge_avg_renorm(b, "f32", base, exps, mask, alpha).astype(np.float64)
        ident = np.zeros(P)
        r = np.zeros(b.G)
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            s = sum(float(alpha[i]) for i in range(K) if A[g, i])
            for i in range(K):
                beta = float(alpha[i]) / s if (A[g, i] and s != 0.0) else 0.0
                dd = deltas[i][o:o + n].astype(np.float64)
                ident[o:o + n] += (float(alpha[i]) - beta) * dd
                r[g] += abs(float(alpha[i]) - beta) * np.linalg.norm(dd)
        diff = Mf - MA
        assert np.all(np.abs(diff - ident) <= slack), bits
        assert np.linalg.norm(diff) <= math.sqrt(np.sum(r**2)) + np.linalg.norm(slack), bits


# --------------------------------------------------------------------------
# TIES with a per-tensor trim scope
# --------------------------------------------------------------------------

def _mag_f32(dtype, x):
    return _f32_of_bf16(x) if dtype == "bf16" else np.asarray(x, np.float32)


def test_ties_tensor_thresholds_are_kth_largest_of_the_zero_completed_tensor():
    # Definition by a library selection: per (tensor, expert) the tensor's
    # |d| with unselected blocks set to zero, and np.partition's k-th largest.
    rng = np.random.default_rng(41)
    numel = [4096 * 3 + 8, 1536, 16, 4096 * 2]
    b = oracle.Blocks(numel, 4096)
    for dtype in ("f32", "bf16"):
        base, exps = _tiny_family(rng, numel, 3, dtype)
        for dens in (0.2, 0.05, 0.6, 1.0, 0.0):
            mask = rng.integers(0, 8, b.G).astype(np.uint32)
            tau = oracle.ties_tensor_thresholds(b, dtype, base, exps, mask, dens)
            x0 = _mag_f32(dtype, base)
            for t in range(len(numel)):
                gs = np.nonzero(b.tensor == t)[0]
                lo, hi = b.off[gs[0]], b.off[gs[-1]] + b.len[gs[-1]]
                for i in range(3):
                    mag = np.zeros(hi - lo, np.float32)
                    for g in gs:
                        if (mask[g] >> i) & 1:
                            sl = slice(b.off[g], b.off[g] + b.len[g])
                            mag[b.off[g] - lo:b.off[g] - lo + b.len[g]] = np.abs(_mag_f32(dtype, exps[i][sl]) - x0[sl])
                    k = oracle.ties_k(hi - lo, dens)
                    want = 0xFFFFFFFF if k == 0 else int(np.partition(mag, mag.size - k)[mag.size - k].view(np.uint32))
                    assert int(tau[t, i]) == want, (dtype, dens, t, i)


def test_ties_tensor_scope_on_single_block_tensors_is_the_block_scope():
    # when every tensor is one block the two trim scopes coincide: thresholds
    # and the full-mask merge equal the (pinned) per-block TIES
    rng = np.random.default_rng(42)
    numel = [4096, 1536, 256, 4000]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 4, "bf16")
    full = np.full(b.G, 15, np.uint32)
    for dens in (0.2, 0.5):
        tt = oracle.ties_tensor_thresholds(b, "bf16", base, exps, full, dens)
        tu = oracle.expand_tensor_thresholds(b, tt)
        assert np.array_equal(tu, oracle.ties_thresholds(b, "bf16", base, exps, dens).reshape(-1))
        assert np.array_equal(oracle.merge_ties_tau(b, "bf16", base, exps, full, tu, 1.0),
                              oracle.merge_ties(b, "bf16", base, exps, full, dens, 1.0))


def test_ties_from_catalog_thresholds_equals_ties_on_any_mask():
    # the per-unit threshold depends on the unit's own block only, so TIES
    # from thresholds computed over the whole checkpoint equals TIES that
    # trims the selected units itself, whatever the mask (the in-merge route
    # recomputes exactly the catalog value)
    rng = np.random.default_rng(44)
    numel = [4096 * 3 + 100, 1536, 256, 4096 * 2]
    b = oracle.Blocks(numel, 4096)
    for dtype in ("f32", "bf16"):
        base, exps = _tiny_family(rng, numel, 5, dtype, scale=1e-3)
        for dens in (0.1, 0.2, 0.7):
            tau = oracle.ties_thresholds(b, dtype, base, exps, dens)
            for _ in range(4):
                m = rng.integers(0, 32, b.G).astype(np.uint32)
                assert np.array_equal(oracle.merge_ties_tau(b, dtype, base, exps, m, tau, 1.0),
                                      oracle.merge_ties(b, dtype, base, exps, m, dens, 1.0)), (dtype, dens)


def test_ties_tensor_thresholds_non_anticipatory():
    rng = np.random.default_rng(43)
    numel = [4096 * 3, 1536]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 3, "bf16")
    mask = np.array([5, 0, 3, 6], np.uint32)
    t1 = oracle.ties_tensor_thresholds(b, "bf16", base, exps, mask, 0.3)
    junk = [e.copy() for e in exps]
    for g in range(b.G):
        for i in range(3):
            if not (mask[g] >> i) & 1:
                junk[i][b.off[g]:b.off[g] + b.len[g]] = rng.integers(0, 2**15, b.len[g]).astype(np.uint16)
    assert np.array_equal(t1, oracle.ties_tensor_thresholds(b, "bf16", base, junk, mask, 0.3))


# --------------------------------------------------------------------------
# experts stored as explicit deltas (Section 3's executor sources)
# --------------------------------------------------------------------------

def _dyadic_family(rng, numel, K):
    # base and deltas on a coarse dyadic grid: W_i = W_0 + Delta_i and
    # W_i - W_0 are exact in fp32, so both expert forms carry the same deltas
    P = sum(numel)
    base = (rng.integers(-2048, 2048, P) / 2.0**16).astype(np.float32)
    deltas = [(rng.integers(-512, 512, P) / 2.0**18).astype(np.float32) for _ in range(K)]
    return base, deltas, [base + d for d in deltas]


def test_delta_experts_equal_weight_experts_when_exact():
    rng = np.random.default_rng(31)
    numel = [4096, 1536, 256, 4096, 2052]
    b = oracle.Blocks(numel, 4096)
    K = 4
    base, deltas, weights = _dyadic_family(rng, numel, K)
    assert all(np.array_equal(w - base, d) for w, d in zip(weights, deltas))
    mask = rng.integers(0, 16, b.G).astype(np.uint32)
    assert np.array_equal(oracle.index(b, "f32", base, deltas, delta=True), oracle.index(b, "f32", base, weights))
    assert np.array_equal(oracle.ties_thresholds(b, "f32", base, deltas, 0.2, delta=True),
                          oracle.ties_thresholds(b, "f32", base, weights, 0.2))
    runs = [
        lambda ex, dl: oracle.merge_avg(b, "f32", base, ex, mask, [0.1, 0.2, 0.3, 0.4], delta=dl),
        lambda ex, dl: oracle.merge_avg_renorm(b, "f32", base, ex, mask, [0.1, 0.2, 0.3, 0.4], delta=dl),
        lambda ex, dl: oracle.merge_ties(b, "f32", base, ex, mask, 0.3, 0.9, delta=dl),
        lambda ex, dl: oracle.merge_dare(b, "f32", base, ex, mask, 0.6, 5, 0, [0.25] * 4, 1.0, delta=dl),
        lambda ex, dl: oracle.merge_dare(b, "f32", base, ex, mask, 0.6, 5, 1, [1.0] * 4, 0.7, delta=dl),
    ]
    for r in runs:
        assert np.array_equal(r(deltas, True), r(weights, False))


def test_delta_experts_index_does_not_read_the_base():
    # With explicit deltas the sums of squares and trim thresholds are
    # functions of the deltas alone; the merged output moves with the base.
    rng = np.random.default_rng(32)
    numel = [4096, 1536, 256]
    b = oracle.Blocks(numel, 4096)
    base, deltas, _ = _dyadic_family(rng, numel, 3)
    other = (rng.standard_normal(sum(numel)) * 3.0).astype(np.float32)
    assert np.array_equal(oracle.index(b, "f32", base, deltas, delta=True),
                          oracle.index(b, "f32", other, deltas, delta=True))
    assert np.array_equal(oracle.ties_thresholds(b, "f32", base, deltas, 0.25, delta=True),
                          oracle.ties_thresholds(b, "f32", other, deltas, 0.25, delta=True))
    full = np.full(b.G, 7, np.uint32)
    zero = np.zeros_like(base)
    # base 0: the AVG output is the weighted delta sum itself; base W_0 adds W_0 (exact here)
    acc = oracle.merge_avg(b, "f32", zero, deltas, full, [0.25, 0.25, 0.5], delta=True)
    got = oracle.merge_avg(b, "f32", base, deltas, full, [0.25, 0.25, 0.5], delta=True)
    assert np.array_equal(got, base + acc)


def test_delta_experts_bf16_constant_delta_closed_form():
    # A constant bf16 delta c = 2^-5 in every element: S = n c^2 exactly.
    numel = [4096, 1536, 520]
    b = oracle.Blocks(numel, 4096)
    P = sum(numel)
    base = _bits_bf16(np.random.default_rng(33).standard_normal(P).astype(np.float32))
    d = _bits_bf16(np.full(P, 2.0**-5, np.float32))
    S = oracle.index(b, "bf16", base, [d], delta=True).reshape(-1)
    assert np.array_equal(S, (b.len * 2.0**-10).astype(np.float32))


# --------------------------------------------------------------------------
# LoRA adapters as a delta source (Section 3, Executor)
# --------------------------------------------------------------------------

def _round_f32_exact(fr):
    # the fp32 nearest to the rational fr, ties to even: float(fr) is within
    # one fp32 ulp of it, so the answer is that value or a neighbour
    from fractions import Fraction
    x = np.float32(float(fr))
    cands = [np.nextafter(x, np.float32(-np.inf)), x, np.nextafter(x, np.float32(np.inf))]
    return min(cands, key=lambda c: (abs(Fraction(float(c)) - fr), int(np.float32(c).view(np.uint32)) & 1))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lora_delta_brute_force_exact_sum(dtype):
    # Each element is the exact rational sum of the rank products, rounded
    # once to fp32, times the scale in fp32, stored in the dtype.  A 5 x 6
    # tensor with rank 3 (no square shapes: a transposed operand fails).
    from fractions import Fraction
    rng = np.random.default_rng(51)
    rows, cols, rank = 5, 6, 3
    A = (rng.standard_normal((rank, cols)) * np.exp(rng.uniform(-8, 8, (rank, cols)))).astype(np.float32)
    B = (rng.standard_normal((rows, rank)) * np.exp(rng.uniform(-8, 8, (rows, rank)))).astype(np.float32)
    scale = np.float32(0.7)
    if dtype == "bf16":
        A, B = _bits_bf16(A), _bits_bf16(B)
        Af, Bf = _f32_of_bf16(A), _f32_of_bf16(B)
    else:
        Af, Bf = A, B
    got = oracle.lora_delta(dtype, rows, cols, A, B, scale)
    want = np.zeros(rows * cols, np.float32)
    for r in range(rows):
        for c in range(cols):
            fr = sum(Fraction(float(Bf[r, k])) * Fraction(float(Af[k, c])) for k in range(rank))
            want[r * cols + c] = scale * _round_f32_exact(fr)
    if dtype == "bf16":
        want = _bits_bf16(want)
    assert np.array_equal(got, want)


def test_lora_delta_rank_one_and_identity_factors():
    # rank 1: scale * outer(u, v); A = I (rank = cols): scale * B;
    # B = I (rank = rows): scale * A.  Dyadic values make every sum exact.
    rng = np.random.default_rng(52)
    rows, cols = 7, 12
    u = (rng.integers(-64, 64, rows) / 64.0).astype(np.float32)
    v = (rng.integers(-64, 64, cols) / 32.0).astype(np.float32)
    got = oracle.lora_delta("f32", rows, cols, v.reshape(1, cols), u.reshape(rows, 1), 0.5)
    assert np.array_equal(got, (0.5 * np.outer(u, v)).astype(np.float32).reshape(-1))
    B = (rng.integers(-100, 100, (rows, cols)) / 16.0).astype(np.float32)
    got = oracle.lora_delta("f32", rows, cols, np.eye(cols, dtype=np.float32), B, 2.0)
    assert np.array_equal(got, (2.0 * B).reshape(-1))
    A = (rng.integers(-100, 100, (rows, cols)) / 16.0).astype(np.float32)
    got = oracle.lora_delta("f32", rows, cols, A, np.eye(rows, dtype=np.float32), 0.25)
    assert np.array_equal(got, (0.25 * A).reshape(-1))
    # the same in bf16 (the values are bf16-exact)
    got = oracle.lora_delta("bf16", rows, cols, _bits_bf16(A), _bits_bf16(np.eye(rows, dtype=np.float32)), 0.25)
    assert np.array_equal(got, _bits_bf16(0.25 * A).reshape(-1))


def test_lora_delta_is_additive_over_rank_components():
    # Stacking two adapters along the rank gives the sum of their deltas
    # (every sum exact on this grid): no rank term is dropped.
    rng = np.random.default_rng(53)
    rows, cols, r1, r2 = 9, 20, 5, 11
    def grid(shape):
        return (rng.integers(-16, 16, shape) / 16.0).astype(np.float32)
    A1, A2, B1, B2 = grid((r1, cols)), grid((r2, cols)), grid((rows, r1)), grid((rows, r2))
    d1 = oracle.lora_delta("f32", rows, cols, A1, B1, 1.0)
    d2 = oracle.lora_delta("f32", rows, cols, A2, B2, 1.0)
    d = oracle.lora_delta("f32", rows, cols, np.vstack([A1, A2]), np.hstack([B1, B2]), 1.0)
    assert np.array_equal(d, d1 + d2)
    assert np.array_equal(d.reshape(rows, cols), B1 @ A1 + B2 @ A2)


def _lora_family(rng, numel, shapes, K, rank, dtype="f32"):
    # adapters on a dyadic grid: every rank sum is exact, so W_i = W_0 + d
    # is exact too; records pack A then B per tensor
    loras, off = [], 0
    for t, (rows, cols) in shapes.items():
        loras.append((t, rows, cols, rank, off, off + rank * cols, 0.5))
        off += rank * (rows + cols)
    ads = [(rng.integers(-8, 8, off) / 64.0).astype(np.float32) for _ in range(K)]
    if dtype == "bf16":
        ads = [_bits_bf16(a) for a in ads]
    return loras, ads


def test_lora_materialize_masks_fill_and_unadapted_tensors():
    rng = np.random.default_rng(54)
    numel = [24 * 40, 520, 16 * 72, 4096]
    b = oracle.Blocks(numel, 256)
    K = 3
    loras, ads = _lora_family(rng, numel, {0: (24, 40), 2: (16, 72)}, K, 6)
    full = oracle.lora_materialize(b, "f32", numel, loras, ads)
    toff = np.concatenate([[0], np.cumsum(numel)])
    for i in range(K):
        assert not full[i][toff[1]:toff[2]].any() and not full[i][toff[3]:].any()  # no adapter: zero
        A = ads[i][0:6 * 40].reshape(6, 40)
        B = ads[i][6 * 40:6 * 64].reshape(24, 6)
        assert np.array_equal(full[i][:960], (0.5 * (B @ A)).astype(np.float32).reshape(-1))
    mask = rng.integers(0, 8, b.G).astype(np.uint32)
    fill = [np.full(sum(numel), 9.0, np.float32) for _ in range(K)]
    part = oracle.lora_materialize(b, "f32", numel, loras, ads, mask=mask, fill=fill)
    for i in range(K):
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            want = full[i][o:o + n] if (mask[g] >> i) & 1 else fill[i][o:o + n]
            assert np.array_equal(part[i][o:o + n], want)


def test_lora_deltas_merge_like_the_weights_they_define():
    # The merge only sees deltas: adapters materialised as explicit deltas
    # give the merge of the checkpoints W_i = W_0 + scale * B A, here exact.
    rng = np.random.default_rng(55)
    numel = [32 * 48, 16, 40 * 64, 520]
    b = oracle.Blocks(numel, 512)
    K = 4
    loras, ads = _lora_family(rng, numel, {0: (32, 48), 2: (40, 64)}, K, 8)
    base = (rng.integers(-2048, 2048, sum(numel)) / 2.0**10).astype(np.float32)
    deltas = oracle.lora_materialize(b, "f32", numel, loras, ads)
    weights = [base + d for d in deltas]
    assert all(np.array_equal(w - base, d) for w, d in zip(weights, deltas))
    mask = rng.integers(0, 16, b.G).astype(np.uint32)
    assert np.array_equal(oracle.merge_ties(b, "f32", base, deltas, mask, 0.3, 1.0, delta=True),
                          oracle.merge_ties(b, "f32", base, weights, mask, 0.3, 1.0))
    assert np.array_equal(oracle.merge_avg(b, "f32", base, deltas, mask, [0.25] * 4, delta=True),
                          oracle.merge_avg(b, "f32", base, weights, mask, [0.25] * 4))


# --------------------------------------------------------------------------
# TIES
# --------------------------------------------------------------------------

def test_ties_worked_example():
    ex = json.load(open(os.path.join(GOLD, "ties_worked_example.json")))
    b = oracle.Blocks(ex["numel"], ex["block_elems"])
    for case in ex["cases"]:
        deltas = [np.array(d, np.float32) for d in case["deltas"]]
        for run in case["runs"]:
            base = np.full(8, run["base"], np.float32)
            exps = [base + d for d in deltas]
            mask = np.array(case["mask"], np.uint32)
            want = np.array(run["out"], np.float32)
            out = oracle.merge_ties(b, "f32", base, exps, mask, case["density"], run["lambda"])
            assert np.array_equal(out, want), case["name"]
            # the catalog route (thresholds, then the merge) gives the same bits
            tau = oracle.ties_thresholds(b, "f32", base, exps, case["density"])
            out = oracle.merge_ties_tau(b, "f32", base, exps, mask, tau, run["lambda"])
            assert np.array_equal(out, want), case["name"]
            if case["density"] == 1.0:
                # DARE's sign-elect combine with nothing dropped (p = 0) elects
                # and averages the same way
                out = oracle.merge_dare(b, "f32", base, exps, mask, 0.0, 7, 1, [0.0] * len(exps), run["lambda"])
                assert np.array_equal(out, want), case["name"]


def _sign_elect_running_sum(ts):
    # the rejected reading: the sign of a running fp32 sum in expert order
    s = np.float32(0)
    for v in ts:
        s = np.float32(s + np.float32(v))
    agree = [np.float32(v) for v in ts if v != 0 and np.sign(v) == np.sign(s)]
    if s == 0 or not agree:
        return np.float32(0)
    m = np.float32(0)
    for v in agree:
        m = np.float32(m + v)
    return np.float32(m / np.float32(len(agree)))


def test_ties_election_compares_rounded_masses():
    # Every order of (1, -1, 2^-25) over three experts: fl32(P) = fl32(1 + 2^-25)
    # = 1 = -N, so nothing is elected for any order, although the exact kept
    # mass is +2^-25.  A running fp32 sum in expert order (planted below)
    # elects + for two of the six orders, and fails.
    import itertools
    b = oracle.Blocks([8], 8)
    base = np.zeros(8, np.float32)
    trip = (1.0, -1.0, 2.0 ** -25)
    perms = list(itertools.permutations(range(3)))
    ds = np.zeros((3, 8), np.float32)
    for j, pm in enumerate(perms):
        ds[:, j] = [trip[r] for r in pm]
    ds[:, 6] = (2.0 ** -23, -1.0, 1.0)  # P = 1 + 2^-23 > 1: +, mean 0.5 + 2^-24
    ds[:, 7] = (-1.0, 2.0 ** -24, 1.0)  # P = fl32(1 + 2^-24) = 1 (tie to even): none
    out = oracle.merge_ties(b, "f32", base, list(ds), np.full(1, 7, np.uint32), 1.0, 1.0)
    want = np.zeros(8, np.float32)
    want[6] = 0.5 + 2.0 ** -24
    assert np.array_equal(out, want)
    planted = np.array([_sign_elect_running_sum(ds[:, j]) for j in range(8)], np.float32)
    assert not np.array_equal(planted, want)
    # mirrored: all signs flipped flips the result
    out = oracle.merge_ties(b, "f32", base, list(-ds), np.full(1, 7, np.uint32), 1.0, 1.0)
    assert np.array_equal(out, -want)


def test_ties_trim_keeps_exactly_top_k():
    # K=1, lambda=1, base 0, continuous deltas (all magnitudes distinct): the
    # output is nonzero exactly on the k largest-|d| positions of each block.
    rng = np.random.default_rng(5)
    numel = [4096, 4096, 1536, 256, 24]
    b = oracle.Blocks(numel, 4096)
    P = sum(numel)
    base = np.zeros(P, np.float32)
    d = rng.standard_normal(P).astype(np.float32)
    for rho in (0.2, 0.1, 0.5, 0.013):
        out = oracle.merge_ties(b, "f32", base, [d], np.ones(b.G, np.uint32), rho, 1.0)
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            k = min(n, math.ceil(rho * n))
            top = set(np.argsort(-np.abs(d[o:o + n]), kind="stable")[:k].tolist())
            nz = set(np.nonzero(out[o:o + n])[0].tolist())
            assert nz == top
            assert np.array_equal(out[o:o + n][list(top)], d[o:o + n][list(top)])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ties_thresholds_are_kth_largest_magnitudes(dtype):
    # the per-unit threshold is the k-th largest |d| (numpy partition of the
    # fp32 deltas), all ones (a NaN pattern: nothing kept) when k = 0; ragged
    # and short blocks included
    rng = np.random.default_rng(41)
    numel = [4096, 1536, 256, 24, 4096]
    b = oracle.Blocks(numel, 1024)
    P = sum(numel)
    K = 3
    if dtype == "f32":
        base = rng.standard_normal(P).astype(np.float32)
        exps = [(base + rng.standard_normal(P).astype(np.float32) * s).astype(np.float32) for s in (1e-3, 1e-2, 0.0)]
        f = lambda a: a
    else:
        base = _bits_bf16(rng.normal(0, 0.02, P))
        exps = [_bits_bf16(_f32_of_bf16(base) + rng.normal(0, s, P)) for s in (1e-3, 3e-4, 0.0)]
        f = _f32_of_bf16
    for rho in (0.0, 0.2, 0.013, 1.0):
        tau = oracle.ties_thresholds(b, dtype, base, exps, rho)
        assert tau.shape == (b.G, K)
        for g in range(b.G):
            o, n = b.off[g], b.len[g]
            k = min(n, math.ceil(rho * n))
            for i in range(K):
                m = np.abs((f(exps[i][o:o + n]) - f(base[o:o + n])).astype(np.float32))
                want = 0xFFFFFFFF if k == 0 else int(np.partition(m, n - k)[n - k].view(np.uint32))
                assert int(tau[g, i]) == want


def test_ties_with_thresholds_equals_ties():
    # merging with the per-unit thresholds reproduces the TIES merge bit for
    # bit, for every mask of a tiny family and for random masks of a larger one
    rng = np.random.default_rng(42)
    numel = [2048, 512, 40]
    b = oracle.Blocks(numel, 512)
    P = sum(numel)
    base = _bits_bf16(rng.normal(0, 0.02, P))
    exps = [_bits_bf16(_f32_of_bf16(base) + rng.normal(0, s, P)) for s in (1e-3, 2e-3, 5e-4, 1e-3)]
    for rho, lam in ((0.2, 1.0), (0.05, 0.7), (1.0, 1.0), (0.0, 1.0)):
        tau = oracle.ties_thresholds(b, "bf16", base, exps, rho)
        for trial in range(6):
            mask = rng.integers(0, 16, b.G).astype(np.uint32)
            want = oracle.merge_ties(b, "bf16", base, exps, mask, rho, lam)
            got = oracle.merge_ties_tau(b, "bf16", base, exps, mask, tau, lam)
            assert np.array_equal(got, want)
    # infinite deltas: density 0 keeps none of them either way, and a larger
    # density keeps them and gives an infinite mean
    b1 = oracle.Blocks([8], 8)
    x0 = np.zeros(8, np.float32)
    e1 = np.array([np.inf, -np.inf, 1, -1, 2, 0, 0, 0], np.float32)
    for rho in (0.0, 0.25, 1.0):
        tau = oracle.ties_thresholds(b1, "f32", x0, [e1], rho)
        want = oracle.merge_ties(b1, "f32", x0, [e1], np.ones(1, np.uint32), rho, 1.0)
        got = oracle.merge_ties_tau(b1, "f32", x0, [e1], np.ones(1, np.uint32), tau, 1.0)
        assert np.array_equal(got, want)
        if rho == 0.0:
            assert np.array_equal(want, x0)
        else:
            assert np.isinf(want[0]) and np.isinf(want[1])


def test_ties_threshold_ties_all_kept_and_zeros_never():
    b = oracle.Blocks([16], 16)
    d = np.array([3, 3, 3, 3, 2, 2, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0], np.float32)
    base = np.zeros(16, np.float32)
    # k = ceil(0.125*16) = 2 -> tau = 3 -> all four 3s kept
    out = oracle.merge_ties(b, "f32", base, [d], np.ones(1, np.uint32), 0.125, 1.0)
    assert np.array_equal(out, np.where(d == 3, d, 0))
    # k = 16 > nnz: tau = 0, zeros never kept -> all nonzeros
    out = oracle.merge_ties(b, "f32", base, [d], np.ones(1, np.uint32), 1.0, 1.0)
    assert np.array_equal(out, d)
    # density 0 keeps nothing
    out = oracle.merge_ties(b, "f32", base, [d], np.ones(1, np.uint32), 0.0, 1.0)
    assert np.array_equal(out, base)


def test_ties_single_expert_full_density_is_that_expert():
    rng = np.random.default_rng(6)
    numel = [4096, 1536, 256]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 1, "bf16", scale=1e-3)
    out = oracle.merge_ties(b, "bf16", base, exps, np.ones(b.G, np.uint32), 1.0, 1.0)
    assert np.array_equal(out, exps[0])
    # two identical experts: disjoint mean of equal entries is that entry
    out = oracle.merge_ties(b, "bf16", base, [exps[0], exps[0]], np.full(b.G, 3, np.uint32), 1.0, 1.0)
    assert np.array_equal(out, exps[0])


def test_ties_negation_symmetry():
    rng = np.random.default_rng(7)
    numel = [4096, 1536]
    b = oracle.Blocks(numel, 4096)
    P = sum(numel)
    base = np.zeros(P, np.float32)
    ds = [(rng.standard_normal(P) * 1e-3).astype(np.float32) for _ in range(4)]
    mask = rng.integers(0, 16, b.G).astype(np.uint32)
    o1 = oracle.merge_ties(b, "f32", base, ds, mask, 0.2, 1.0)
    o2 = oracle.merge_ties(b, "f32", base, [-d for d in ds], mask, 0.2, 1.0)
    assert np.array_equal(o2, -o1)


def test_ties_elected_sign_and_mean_bounds():
    # the merged delta has the sign of the (trimmed) sum and lies within the
    # range of the agreeing entries.
    rng = np.random.default_rng(8)
    numel = [4096]
    b = oracle.Blocks(numel, 4096)
    base = np.zeros(4096, np.float32)
    ds = [(rng.standard_normal(4096) * 1e-3).astype(np.float32) for _ in range(5)]
    out = oracle.merge_ties(b, "f32", base, ds, np.full(1, 31, np.uint32), 1.0, 1.0).astype(np.float64)
    D = np.stack(ds).astype(np.float64)
    s = D.sum(0)
    assert np.all(np.sign(out) == np.sign(s))
    pos = np.where(D > 0, D, np.nan)
    neg = np.where(D < 0, D, np.nan)
    with np.errstate(all="ignore"):
        lo = np.where(s > 0, np.nanmin(pos, 0), np.nanmin(neg, 0))
        hi = np.where(s > 0, np.nanmax(pos, 0), np.nanmax(neg, 0))
    sel = s != 0
    assert np.all((out[sel] >= np.minimum(lo, hi)[sel] - 1e-9) & (out[sel] <= np.maximum(lo, hi)[sel] + 1e-9))


def test_ties_lambda_zero_is_base_and_non_anticipatory():
    rng = np.random.default_rng(9)
    numel = [4096, 256]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 3, "bf16")
    mask = np.array([5, 2], np.uint32)
    assert np.array_equal(oracle.merge_ties(b, "bf16", base, exps, mask, 0.2, 0.0), base)
    o1 = oracle.merge_ties(b, "bf16", base, exps, mask, 0.2, 1.0)
    junk = [e.copy() for e in exps]
    junk[1][:4096] = 0x3F80  # expert 1 not selected in block 0
    junk[0][4096:] = 0x4000  # expert 0 not selected in block 1
    junk[2][4096:] = 0x4000
    o2 = oracle.merge_ties(b, "bf16", base, junk, mask, 0.2, 1.0)
    assert np.array_equal(o1, o2)


# --------------------------------------------------------------------------
# DARE
# --------------------------------------------------------------------------

def test_dare_p0_linear_equals_avg_bitwise():
    rng = np.random.default_rng(10)
    numel = [4096, 1536, 256, 4096]
    b = oracle.Blocks(numel, 4096)
    for dtype in ("bf16", "f32"):
        base, exps = _tiny_family(rng, numel, 4, dtype)
        mask = rng.integers(0, 16, b.G).astype(np.uint32)
        alpha = np.array([0.25, 0.125, 0.5, 0.3], np.float32)
        a = oracle.merge_avg(b, dtype, base, exps, mask, alpha)
        d = oracle.merge_dare(b, dtype, base, exps, mask, 0.0, 123, 0, alpha, 1.0)
        assert np.array_equal(a, d)


def test_dare_p0_sign_elect_equals_ties_full_density():
    rng = np.random.default_rng(11)
    numel = [4096, 1536, 256]
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 5, "bf16")
    mask = rng.integers(0, 32, b.G).astype(np.uint32)
    t = oracle.merge_ties(b, "bf16", base, exps, mask, 1.0, 0.7)
    d = oracle.merge_dare(b, "bf16", base, exps, mask, 0.0, 9, 1, np.ones(5, np.float32), 0.7)
    assert np.array_equal(t, d)


def _const_delta_family(numel, K, c=1.0):
    P = sum(numel)
    base = np.zeros(P, np.float32)
    return base, [base + np.float32(c) for _ in range(K)]


def test_dare_keep_rate_and_rescale():
    numel = [1 << 20]
    b = oracle.Blocks(numel, 4096)
    base, exps = _const_delta_family(numel, 1)
    for p in (0.9, 0.5, 0.1):
        out = oracle.merge_dare(b, "f32", base, exps, np.ones(b.G, np.uint32), p, 7, 0, [1.0], 1.0)
        s = np.float32(1.0 / (1.0 - p))
        kept = out != 0
        assert np.all(out[kept] == s)  # kept entries rescaled by 1/(1-p)
        n = out.size
        frac = kept.mean()
        assert abs(frac - (1 - p)) < 6 * math.sqrt(p * (1 - p) / n)
        # unbiased: the mean rescaled delta estimates the delta (1.0)
        assert abs(out.astype(np.float64).mean() - 1.0) < 6 * float(s) * math.sqrt(p * (1 - p) / n)


def test_dare_masks_independent_across_experts_tensors_and_lanes():
    numel = [1 << 18, 1 << 18]
    b = oracle.Blocks(numel, 4096)
    base, exps = _const_delta_family(numel, 2)
    p = 0.5
    # expert 0 alone and expert 1 alone
    k0 = oracle.merge_dare(b, "f32", base, exps, np.full(b.G, 1, np.uint32), p, 3, 0, [1.0, 1.0], 1.0) != 0
    k1 = oracle.merge_dare(b, "f32", base, exps, np.full(b.G, 2, np.uint32), p, 3, 0, [1.0, 1.0], 1.0) != 0
    n = k0.size
    sd = math.sqrt(0.25 * 0.75 / n)
    assert abs((k0 & k1).mean() - 0.25) < 6 * sd  # experts draw independent masks
    half = numel[0]
    assert abs((k0[:half] == k0[half:]).mean() - 0.5) < 6 * math.sqrt(0.25 / half)  # tensors differ
    g8 = k0.reshape(-1, 8)
    all_eq = (g8.all(1) | (~g8).all(1)).mean()
    assert abs(all_eq - 1 / 128) < 6 * math.sqrt(1 / 128 * 127 / 128 / g8.shape[0])  # the 8 draws of a call differ
    lo = k0.reshape(-1, 2)
    assert abs((lo[:, 0] == lo[:, 1]).mean() - 0.5) < 6 * math.sqrt(0.25 / lo.shape[0])  # a word's two halves differ
    # a different seed gives a different mask
    k0b = oracle.merge_dare(b, "f32", base, exps, np.full(b.G, 1, np.uint32), p, 4, 0, [1.0, 1.0], 1.0) != 0
    assert abs((k0 == k0b).mean() - 0.5) < 6 * math.sqrt(0.25 / n)


def test_dare_drop_decision_follows_counter_mapping():
    # element e of tensor t of expert i uses the 16-bit half e%8 of the
    # Philox output for counter (e//8, 0, t, 0) under key (seed, i): word
    # (e%8)//2, its low half for even e; dropped iff half < floor(p*2^16).
    # Tensors of 64, 4096+64 and 4100 elements: fp32 blocks of 4100 start
    # at element 0 only, so every block starts a draw; the 4100-element
    # block size below puts a second block of tensor 2 at element 4100,
    # the middle of draw 512.
    for numel, be in (([64, 4096 + 64], 4096), ([8200, 20], 4100)):
        b = oracle.Blocks(numel, be)
        base, exps = _const_delta_family(numel, 3)
        for p, seed in ((0.5, 0xDEADBEEF), (0.9, 7), (0.3, 0)):
            out = oracle.merge_dare(b, "f32", base, exps, np.full(b.G, 4, np.uint32), p, seed, 0,
                                    [0.0, 0.0, 1.0], 1.0)
            T = math.floor(p * 2**16)
            start = 0
            for t, n in enumerate(numel):
                probe = sorted({e for e in list(range(0, 20)) + [n - 1, n - 5, n - 8, 4096 + 3, 4100, 4101, 4103,
                                                                 4104] if 0 <= e < n})
                for e in probe:
                    w = int(oracle.philox4x32_10([e // 8, 0, t, 0], [seed, 2])[(e % 8) // 2])
                    u = (w >> 16) if e % 2 else (w & 0xFFFF)
                    assert (out[start + e] == 0) == (u < T), (numel, p, t, e)
                start += n


def test_dare_non_anticipatory_drop_mask():
    # the drop mask of a selected expert does not depend on which other
    # experts are selected (omega is fixed by (seed, expert, element)).
    numel = [4096, 1536]
    rng = np.random.default_rng(12)
    b = oracle.Blocks(numel, 4096)
    base, exps = _tiny_family(rng, numel, 3, "f32")
    alpha = np.array([0.5, 0.25, 0.25], np.float32)
    only2 = oracle.merge_dare(b, "f32", base, exps, np.full(b.G, 4, np.uint32), 0.9, 7, 0, alpha, 1.0)
    zeroed = [base.copy(), base.copy(), exps[2]]  # experts 0,1 have zero delta
    all3 = oracle.merge_dare(b, "f32", base, zeroed, np.full(b.G, 7, np.uint32), 0.9, 7, 0, alpha, 1.0)
    assert np.array_equal(only2, all3)


def test_oracle_results_do_not_depend_on_the_thread_count():
    # Each per-block computation is sequential, so the oracle's results are
    # bitwise the same on one thread and on several (the parallel loops only
    # split the blocks among threads).
    rng = np.random.default_rng(81)
    numel = [4096 * 9 + 512, 4096 * 4, 1536, 256, 4096 * 7 + 64]
    b = oracle.Blocks(numel, 4096)
    K = 4
    base, exps = _tiny_family(rng, numel, K, "bf16", scale=1e-3)
    full = sum(numel) * 2 * K
    w = [0.25] * K

    def run():
        S = oracle.index(b, "bf16", base, exps)
        tau = oracle.ties_thresholds(b, "bf16", base, exps, 0.2)
        m, st = oracle.plan(b, "bf16", K, S, [1.0] * K, full // 2)
        mt, stt = oracle.plan(b, "bf16", K, None, w, full // 3)
        return [S, tau, m, mt, np.array([st["digest"], stt["digest"]], np.uint64),
                oracle.merge_avg(b, "bf16", base, exps, m, w),
                oracle.merge_avg_renorm(b, "bf16", base, exps, m, w),
                oracle.merge_ties(b, "bf16", base, exps, m, 0.2, 1.0),
                oracle.merge_ties_tau(b, "bf16", base, exps, m, tau, 1.0),
                oracle.merge_dare(b, "bf16", base, exps, m, 0.9, 7, 0, w, 1.0),
                oracle.merge_dare(b, "bf16", base, exps, m, 0.9, 7, 1, w, 1.0),
                oracle.ties_tensor_thresholds(b, "bf16", base, exps, m, 0.2)]

    n = oracle.num_threads()
    try:
        oracle.set_num_threads(1)
        assert oracle.num_threads() == 1
        one = run()
        oracle.set_num_threads(max(n, 8))
        many = run()
    finally:
        oracle.set_num_threads(n)
    for a, c in zip(one, many):
        assert np.array_equal(np.asarray(a).view(np.uint8), np.asarray(c).view(np.uint8))
