#!/usr/bin/env python3
"""Benchmark of the budgeted-merge hot path on one MI355X.

Workload: a synthetic Qwen2.5-1.5B-shaped bf16 checkpoint family (28 layers,
hidden 1536, FFN 8960, 12 q / 2 kv heads x 128, vocab 151936, tied
embeddings; P = 1,543,714,304 parameters, G = 376,989 blocks of 4096) with
K = 4 experts, merged with budgeted TIES (keep density 0.2, lambda 1) at
B = 25%, 50% and 100% of the expert bytes.

One step = index the expert deltas once, then for each budget: plan
(Algorithm 1) + TIES merge; the plans of the second and third budgets run on
a second stream while the previous budget's merge runs.  Two routes compute
the same bits:
  catalog (default): the index pass also stores every unit's TIES trim
      threshold (mask-independent), and each merge reads it;
  in-merge: the index pass stores the squared norms only, and each merge
      finds the thresholds of its selected units itself.
All inputs are resident in HBM before the timed region.  The metric is
merged parameters per second (3 P per step); effective HBM GB/s and the
roofline fraction come from HIP events around each kernel-launching call on
the stream the kernels run on.  After the timed region the other route's
merges are timed once for reference.

The CPU baseline is the oracle (test infrastructure) on a bounded sample of
the same family: every 2nd block, the same route (index, thresholds for the
catalog route, plan and TIES at the three budgets), on all host cores.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from workloads import CONFIGS  # noqa: E402  (shape tables only; no GPU work at import)

METRIC = "merged params/sec + effective HBM GB/s, budgeted TIES merge at B=25/50/100%"
HBM_PEAK = 8.0e12  # MI355X published HBM3E bandwidth, bytes/s
BUDGETS = (0.25, 0.5, 1.0)
TRAFFIC_PROFILES = {
    "catalog": os.path.join(ROOT, "profiles", "ties_threshold_merge_qwen2.5-1.5b_counters.md"),
    "in-merge": os.path.join(ROOT, "profiles", "ties_merge_qwen2.5-1.5b_counters.md"),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


_CSRC = "paper_2605_29489_amd/csrc/"
# the sources each route's merge kernel is built from: a committed counter
# profile is used only while their hash matches the one it records
KERNEL_SOURCES = {
    "catalog": tuple(_CSRC + f for f in ("k_merge.hip", "merge_src.h", "device_common.h")),
    "in-merge": tuple(_CSRC + f for f in ("k_merge_ties.hip", "merge_src.h", "device_common.h", "ties_select.h")),
}


def kernel_source_hash(route="catalog") -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES[route]:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


LORA_SOURCES = ("paper_2605_29489_amd/csrc/k_lora.hip", "paper_2605_29489_amd/csrc/device_common.h")
LORA_TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "lora_ties_qwen2.5-1.5b_counters.md")


def lora_source_hash() -> str:
    h = hashlib.sha256()
    for p in LORA_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_lora_traffic():
    """HBM bytes of one fused adapter TIES merge launch (k_lora_ties, the
    mean over the three budgets) from the committed counter profile, or None
    if it is missing or was taken on a different kernel source."""
    if not os.path.exists(LORA_TRAFFIC_PROFILE):
        return None
    kv = {}
    for line in open(LORA_TRAFFIC_PROFILE):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            kv[k.strip()] = v.strip().strip("`")
    if kv.get("kernel_source_sha256_16") != lora_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_fused_launch"])
    except (KeyError, ValueError):
        return None


def stored_traffic(route):
    """HBM bytes per merge launch of the route from the committed counter
    profile, or None if it is missing or was taken on a different kernel
    source."""
    path = TRAFFIC_PROFILES[route]
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            kv[k.strip()] = v.strip().strip("`")
    if kv.get("kernel_source_sha256_16") != kernel_source_hash(route):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(spec, base, exps, route, blocks_stride=8):
    """Time the oracle on every `blocks_stride`-th block (bounded sample)."""
    import numpy as np
    import torch

    import oracle

    lay = spec.layout
    blk = oracle.Blocks(lay.numel, lay.block_elems)
    ids = np.arange(0, blk.G, blocks_stride)
    idx = np.concatenate([np.arange(blk.off[g], blk.off[g] + blk.len[g]) for g in ids])
    ti = torch.from_numpy(idx).cuda()
    host = lambda t: t[ti].view(torch.int16).cpu().numpy().view(np.uint16)
    b_np = host(base)
    e_np = [host(e) for e in exps]
    del ti
    doff = np.concatenate([[0], np.cumsum(blk.len[ids])[:-1]]).astype(np.int64)
    # a sub-family made of the sampled blocks: same lengths, tensors, offsets
    sub = oracle.Blocks([int(n) for n in blk.len[ids]], lay.block_elems)
    K = len(exps)
    nparams = int(blk.len[ids].sum())
    full = nparams * 2 * K
    t0 = time.perf_counter()
    S = oracle.index(blk, "bf16", b_np, e_np, doff=doff, ids=ids).reshape(-1)
    tau = oracle.ties_thresholds(blk, "bf16", b_np, e_np, 0.2, ids=ids, doff=doff) if route == "catalog" else None
    for f in BUDGETS:
        mask, _ = oracle.plan(sub, "bf16", K, S, [1.0] * K, int(f * full))
        if route == "catalog":
            oracle.merge_ties_tau(blk, "bf16", b_np, e_np, mask, tau, 1.0, ids=ids, doff=doff)
        else:
            oracle.merge_ties(blk, "bf16", b_np, e_np, mask, 0.2, 1.0, ids=ids, doff=doff)
    dt = time.perf_counter() - t0
    return {
        "value": 3 * nparams / dt,
        "unit": "params/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"every {blocks_stride}th block ({len(ids)} blocks, {nparams} params, all {K} experts): "
                  f"index{' + thresholds' if route == 'catalog' else ''} + plan + TIES at B=25/50/100% "
                  f"of the sample's expert bytes; {dt:.2f} s",
    }


PCIE_PEAK = 64.0e9  # PCIe Gen5 x16, one direction, nominal bytes/s


def host_cpu():
    """The host the CPU baseline ran on: model name and socket count from
    /proc/cpuinfo, and the CPUs this process may use."""
    model, sockets = None, set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name") and model is None:
                    model = line.split(":", 1)[1].strip()
                elif line.startswith("physical id"):
                    sockets.add(line.split(":", 1)[1].strip())
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    return {"cpu_model": model, "sockets": len(sockets) or None, "nproc": nproc}


def one_thread(fn):
    """Run fn with the oracle on one thread, then restore its thread count."""
    import oracle
    n = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        return fn()
    finally:
        oracle.set_num_threads(n)


def fidelity(out, m_full, blen, n_sel, n_units):
    """Fidelity of a budgeted merge against the full-read one (reporting only,
    outside every timed region): Rel. l2 = ||M_A - M_full|| / ||M_full|| over
    the checkpoint, P95 block = the 95th percentile over blocks of
    ||M_A - M_full|| / ||M_full|| per block, Touched = selected units / (K G).
    fp64, in block-aligned chunks of about 2^27 elements."""
    import torch
    ends = torch.cumsum(blen, 0)
    num_all, den_all = [], []
    g0, e0, G = 0, 0, int(blen.numel())
    while g0 < G:
        g1 = int(torch.searchsorted(ends, e0 + (1 << 27), right=True))
        g1 = max(g1, g0 + 1)
        e1 = int(ends[g1 - 1])
        a = out[e0:e1].double()
        b = m_full[e0:e1].double()
        a.sub_(b).square_()
        b.square_()
        num_all.append(torch.segment_reduce(a, "sum", lengths=blen[g0:g1]))
        den_all.append(torch.segment_reduce(b, "sum", lengths=blen[g0:g1]))
        del a, b
        g0, e0 = g1, e1
    num, den = torch.cat(num_all), torch.cat(den_all)
    rel = float(num.sum().sqrt() / den.sum().sqrt())
    ok = den > 0
    blk = (num[ok] / den[ok]).sqrt().float()
    p95 = float(torch.quantile(blk, 0.95)) if blk.numel() else 0.0
    return {"rel_l2": rel, "p95_block": p95, "touched": n_sel / n_units}


def write_expert_files(exps, P):
    """Writes each (device) expert to a file under $MP_BENCH_DIR (default /tmp),
    frees the device copies, and returns the paths with a function that asks
    the kernel to drop the files from the page cache, so that reads come from
    storage."""
    import tempfile
    import torch
    d = tempfile.mkdtemp(prefix="mp_experts_", dir=os.environ.get("MP_BENCH_DIR", "/tmp"))
    paths = []
    for i in range(len(exps)):
        p = os.path.join(d, f"expert{i}.bin")
        with open(p, "wb") as f:
            for c0 in range(0, P, 1 << 27):
                f.write(exps[i][c0:c0 + (1 << 27)].view(torch.int16 if exps[i].dtype == torch.bfloat16
                                                       else torch.int32).cpu().numpy().tobytes())
            f.flush()
            os.fsync(f.fileno())
        exps[i] = None
        paths.append(p)
        log(f"wrote {p}")
    torch.cuda.empty_cache()

    def drop():
        for p in paths:
            fd = os.open(p, os.O_RDONLY)
            os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
            os.close(fd)

    return paths, drop


def cpu_baseline_lora(spec, recs, ads_np, base, cfg, n_layers=5):
    """Time the oracle on the whole LoRA step for the adapted tensors of the
    first n_layers layers (a bounded sample): pull every unit, index, then per
    budget plan, pull the selected units and merge."""
    import numpy as np
    import torch

    import oracle

    lay = spec.layout
    K = len(ads_np)
    toff = np.concatenate([[0], np.cumsum(lay.numel)]).astype(np.int64)
    names = [n for n, _ in spec.tensors]
    pick = [r for r in recs if names[r[0]].startswith(tuple(f"layers.{l}." for l in range(n_layers)))]
    numel = [r[1] * r[2] for r in pick]
    sub = oracle.Blocks(numel, lay.block_elems)
    b_np = np.concatenate([base[int(toff[r[0]]):int(toff[r[0]]) + r[1] * r[2]].view(torch.int16).cpu().numpy()
                           .view(np.uint16) for r in pick])
    sub_recs = [(j,) + tuple(r[1:]) for j, r in enumerate(pick)]  # tensor ids of the sub-layout
    nparams = int(sum(numel))
    full = nparams * 2 * K
    t0 = time.perf_counter()
    d_all = oracle.lora_materialize(sub, lay.dtype, numel, sub_recs, ads_np)
    S = oracle.index(sub, lay.dtype, b_np, d_all, delta=True).reshape(-1)
    tau = oracle.ties_thresholds(sub, lay.dtype, b_np, d_all, cfg["density"], delta=True)
    for f in cfg["budgets"]:
        mask, _ = oracle.plan(sub, lay.dtype, K, S, [1.0] * K, int(f * full), flags=2)
        d = oracle.lora_materialize(sub, lay.dtype, numel, sub_recs, ads_np, mask=mask)
        oracle.merge_ties_tau(sub, lay.dtype, b_np, d, mask, tau, cfg["lam"], delta=True)
    dt = time.perf_counter() - t0
    return {
        "value": len(cfg["budgets"]) * nparams / dt,
        "unit": "params/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"the {len(pick)} adapted tensors of layers 0-{n_layers - 1} ({nparams} params, all {K} experts): "
                  f"pull of every unit + "
                  f"index and thresholds + per budget (B=25/50/100% of the sample's expert bytes) plan, pull of "
                  f"the selected units and TIES from the thresholds; {dt:.2f} s",
    }


def run_lora(args):
    """Experts given as low-rank adapters: the catalog materialises every
    expert's deltas once and indexes them (sums of squares and every unit's
    TIES trim threshold); each budget then plans and merges with the stored
    thresholds, drawing the selected units' deltas from the adapters inside
    the merge (matrix-core contraction, no delta checkpoint).  The two-call
    route (pull the selected units, then merge them) is timed beside it and
    must give the same bits."""
    import numpy as np
    import torch

    import paper_2605_29489_amd as mp
    from workloads import family_spec, lora_records, make_family_device, make_lora_adapters

    cfg = CONFIGS[args.workload]
    torch.cuda.set_device(0)
    spec = family_spec(cfg["family"], n_layers=args.layers)
    lay = spec.layout
    K = spec.K
    P = lay.n_params
    es = lay.elem_bytes
    dt = mp.MP_F32 if lay.dtype == "f32" else mp.MP_BF16
    L = mp.Layout(lay.numel, lay.block_elems, dt)
    G = mp.mp_layout_blocks(L)
    recs, n_ad = lora_records(spec, cfg["rank"], cfg["scale"])
    adapted = sum(r[1] * r[2] for r in recs)
    log(f"generating {spec.description}: P={P} G={G}; rank-{cfg['rank']} adapters on {len(recs)} tensors "
        f"({adapted} params), {n_ad} adapter elements per expert")
    base, _ = make_family_device(spec, K=1, seed=0, device="cuda")
    tdt = torch.bfloat16 if lay.dtype == "bf16" else torch.float32
    ads = []
    ads_np = make_lora_adapters(n_ad, K, lay.dtype, seed=0, std=0.02)
    for a in ads_np:
        t = torch.from_numpy(a.view(np.int16) if lay.dtype == "bf16" else a).cuda()
        ads.append(t.view(tdt) if lay.dtype == "bf16" else t)
    deltas = [torch.empty(P, dtype=tdt, device="cuda") for _ in range(K)]
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    full = P * es * K
    w = [1.0] * K
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        r = fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b), r

    def med(fn):
        for _ in range(max(0, args.warmup)):
            fn()
        return float(np.median([timed(fn)[0] for _ in range(max(1, args.steps))]))

    pull_all_ms = med(lambda: mp.mp_lora_materialize(L, recs, ads, deltas, stream=stream))
    # the catalog of the pulled deltas: sums of squares and every unit's TIES
    # trim threshold (the headline's route: thresholds depend on the unit only)
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    idx_ms = med(lambda: mp.mp_index_ties(L, base, deltas, cfg["density"], tau, sumsq=sumsq, stream=stream,
                                          delta=True))
    flags = mp.MP_PLAN_SKIP_ZERO  # tensors without an adapter have zero deltas: never worth a read
    mp.mp_plan(L, K, sumsq, w, full, mask, flags=flags, stream=stream)
    rows = []
    out2 = torch.empty_like(base)
    ity = torch.int16 if lay.dtype == "bf16" else torch.int32
    # bytes one fused launch must move: the base read and the output written
    # once, the adapters, the mask and the thresholds
    fused_alg = 2 * P * es + K * n_ad * es + 4 * G + 4 * G * K
    for f in cfg["budgets"]:
        B = int(f * full)
        plan_ms, st = timed(lambda: mp.mp_plan(L, K, sumsq, w, B, mask, flags=flags, stream=stream))
        # the merge with every selected delta drawn from the adapters inside it
        fused_ms = med(lambda: mp.mp_lora_merge_ties_tau(L, base, recs, ads, mask, tau, cfg["lam"], out,
                                                         stream=stream))
        # for comparison, the two-call route on the same plan: pull the
        # selected units into delta checkpoints, then merge them
        pull_ms = med(lambda: mp.mp_lora_materialize(L, recs, ads, deltas, mask=mask, stream=stream))
        merge = lambda io=False: mp.mp_merge_ties_tau(L, base, deltas, mask, tau, cfg["lam"], out2, io=io,
                                                  stream=stream, delta=True)
        io = merge(io=True)
        assert io["expert_bytes"] == st["cost_bytes"]
        ms = med(merge)
        torch.cuda.synchronize()
        assert torch.equal(out.view(ity), out2.view(ity)), "the fused merge differs from pull + merge"
        rows.append({"budget_frac": f, "budget_bytes": B, "cost_bytes": st["cost_bytes"],
                     "n_selected": st["n_selected"], "plan_ms": round(plan_ms, 4), "fused_ms": round(fused_ms, 4),
                     "fused_effective_GBps": fused_alg / (fused_ms * 1e-3) / 1e9,
                     "two_call": {"pull_ms": round(pull_ms, 4), "merge_ms": round(ms, 4),
                                  "pull_effective_GBps": (st["cost_bytes"] + K * n_ad * es) / (pull_ms * 1e-3) / 1e9,
                                  "merge_effective_GBps": (2 * P * es + st["cost_bytes"] + 4 * G + 4 * st["n_selected"])
                                  / (ms * 1e-3) / 1e9}})
    step_ms = pull_all_ms + idx_ms + sum(r["plan_ms"] + r["fused_ms"] for r in rows)
    if args.calibration_copy:  # an empty-mask AVG launch copies the base: a copy of known size for byte counters
        mask.zero_()
        mp.mp_merge_avg(L, base, deltas, mask, [1.0 / K] * K, out, stream=stream, delta=True)
        torch.cuda.synchronize()
    # the dominant kernel: the fused merge, one launch per budget (each reads
    # the base and writes the whole output)
    fused_mean = float(np.mean([r["fused_ms"] for r in rows]))
    achieved = fused_alg / (fused_mean * 1e-3)
    result = {
        "metric": "merged params/sec, budgeted TIES merge of LoRA-adapter experts",
        "value": len(rows) * P / (step_ms * 1e-3), "unit": "params/s", "n_gpus": 1, "steps": max(1, args.steps),
        "warmup": args.warmup, "ms_per_step": round(step_ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{spec.description}; {cfg}", "storage_dtype": lay.dtype, "params": P,
                   "adapted_params": adapted, "adapter_elems_per_expert": n_ad, "blocks": G, "K": K,
                   "experts": "device (adapters)", "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "k_lora_ties, mean over the budgets",
                     "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": achieved / HBM_PEAK,
                     "traffic": stored_lora_traffic() if lay.dtype == "bf16" and args.layers is None else None,
                     "note": "bytes moved are the base read and the output written once; the kernel is bound by "
                             "vector-ALU issue (the TIES fold of every element for each selected expert, 8 "
                             "instructions per delta), not by HBM"},
        "breakdown": {"pull_all_ms": round(pull_all_ms, 4), "index_ms": round(idx_ms, 4),
                      "pull_all_GBps": (K * P * es + K * n_ad * es) / (pull_all_ms * 1e-3) / 1e9,
                      "per_budget": rows},
    }
    if not args.no_cpu_baseline and lay.dtype == "bf16":
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline_lora(spec, recs, ads_np, base, cfg)
    print(json.dumps(result), flush=True)


def cpu_baseline_sweep(spec, base, exps, cfg, flags, dl, target_elems=100_000_000):
    """Time the oracle on a sweep workload: index, then per budget plan and
    merge, over every n-th block (a bounded sample of about target_elems
    expert elements in all).  None for ops the sample cannot express
    (tensor-scope thresholds need whole tensors)."""
    import numpy as np
    import torch

    import oracle

    op = cfg["op"]
    if op not in ("avg", "avg_renorm", "ties", "dare"):
        return None
    lay = spec.layout
    blk = oracle.Blocks(lay.numel, lay.block_elems)
    stride = max(1, lay.n_params * len(exps) // target_elems)
    ids = np.arange(0, blk.G, stride)
    idx = torch.from_numpy(np.concatenate([np.arange(blk.off[g], blk.off[g] + blk.len[g]) for g in ids]))

    def host(t):
        x = t[idx.to(t.device)]
        return x.view(torch.int16).cpu().numpy().view(np.uint16) if x.dtype == torch.bfloat16 else x.cpu().numpy()

    b_np = host(base)
    e_np = [host(e) for e in exps]
    doff = np.concatenate([[0], np.cumsum(blk.len[ids])[:-1]]).astype(np.int64)
    sub = oracle.Blocks([int(n) for n in blk.len[ids]], lay.block_elems)
    K = len(exps)
    nparams = int(blk.len[ids].sum())
    full = nparams * lay.elem_bytes * K
    linear = op in ("avg", "avg_renorm") or (op == "dare" and cfg.get("combine") == "linear")
    w = [1.0 / K] * K if linear else [1.0] * K
    dt_name = lay.dtype
    t0 = time.perf_counter()
    S = oracle.index(blk, dt_name, b_np, e_np, doff=doff, ids=ids, delta=dl).reshape(-1)
    for f in cfg["budgets"]:
        mask, _ = oracle.plan(sub, dt_name, K, S, w, int(f * full), flags=flags)
        kw = dict(ids=ids, doff=doff, delta=dl)
        if op == "avg":
            oracle.merge_avg(blk, dt_name, b_np, e_np, mask, w, **kw)
        elif op == "avg_renorm":
            oracle.merge_avg_renorm(blk, dt_name, b_np, e_np, mask, w, **kw)
        elif op == "ties":
            oracle.merge_ties(blk, dt_name, b_np, e_np, mask, cfg["density"], cfg["lam"], **kw)
        else:
            comb = 1 if cfg["combine"] == "sign_elect" else 0
            oracle.merge_dare(blk, dt_name, b_np, e_np, mask, cfg["p"], cfg["seed"], comb, w, cfg["lam"], **kw)
    dt = time.perf_counter() - t0
    return {
        "value": len(cfg["budgets"]) * nparams / dt,
        "unit": "params/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"every n-th block, n = {stride} ({len(ids)} blocks, {nparams} params, all {K} experts): "
                  f"index + plan + "
                  f"{op} at each budget of the sweep (fractions of the sample's expert bytes); {dt:.2f} s",
    }


def run_sweep(args):
    """One of the other workload shapes: index once, then plan + merge at each
    budget of its sweep.  Experts are device-resident, stay in pinned host
    memory (kernels read the selected blocks over PCIe), or stay in ordinary
    host memory (the selected blocks are staged and copied over PCIe)."""
    import numpy as np
    import torch

    import paper_2605_29489_amd as mp
    from workloads import family_spec, make_family_device

    cfg = CONFIGS[args.workload]
    torch.cuda.set_device(0)
    spec = family_spec(cfg["family"], n_layers=args.layers)
    lay = spec.layout
    K = spec.K
    P = lay.n_params
    where = {"config": cfg["residency"], "device": "device", "pinned": "host_pinned",
             "pageable": "host_pageable", "file": "host_file"}[args.residency]
    pinned = where == "host_pinned"
    pageable = where == "host_pageable"
    files = where == "host_file"
    host = pinned or pageable or files  # experts cross PCIe: that link (or the storage) bounds the merge
    res = mp.MP_HOST_PINNED if pinned else (mp.MP_HOST_PAGEABLE if pageable else
                                            (mp.MP_HOST_FILE if files else mp.MP_DEVICE))
    dt = mp.MP_F32 if lay.dtype == "f32" else mp.MP_BF16
    L = mp.Layout(lay.numel, lay.block_elems, dt)
    G = mp.mp_layout_blocks(L)
    where_txt = {"host_pinned": "pinned host", "host_pageable": "pageable host",
                 "host_file": "files"}.get(where, "device")
    log(f"generating {spec.description}: P={P} G={G} experts {where_txt}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda",
                                    experts_on_host="pinned" if pinned else ("pageable" if pageable else None))
    dl = bool(args.experts_delta)
    if dl:  # the experts as stored deltas fl32(W_i - W_0) in the checkpoint dtype (set-up, not timed)
        if pinned or pageable:
            sys.exit("bench.py: --experts-delta supports device-resident experts or files only")
        for e in exps:
            for c0 in range(0, P, 1 << 28):
                c1 = min(P, c0 + (1 << 28))
                e[c0:c1] = (e[c0:c1].float() - base[c0:c1].float()).to(e.dtype)
    torch.cuda.synchronize()
    drop = None
    if files:  # one file per expert (set-up); the page cache is dropped before every timed call
        exps, drop = write_expert_files(exps, P)
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    mask = torch.empty(G, dtype=torch.int32, device="cuda")
    out = torch.empty_like(base)
    es = lay.elem_bytes
    full = P * es * K
    op = cfg["op"]
    linear = op in ("avg", "avg_renorm") or (op == "dare" and cfg.get("combine") == "linear")
    w = [1.0 / K] * K if linear else [1.0] * K  # the plan weighs units by the merge coefficients
    stream = torch.cuda.current_stream()
    tau_t = torch.empty(G * K, dtype=torch.int32, device="cuda") if op == "ties_tensor" else None
    blen_np = np.asarray(lay.block_lengths(), np.int64)

    def merge(io=False):
        if op == "avg":
            return mp.mp_merge_avg(L, base, exps, mask, [1.0 / K] * K, out, residency=res, io=io, stream=stream,
                                   delta=dl)
        if op == "avg_renorm":
            return mp.mp_merge_avg_renorm(L, base, exps, mask, [1.0 / K] * K, out, residency=res, io=io,
                                          stream=stream, delta=dl)
        if op == "ties":
            return mp.mp_merge_ties(L, base, exps, mask, cfg["density"], cfg["lam"], out, residency=res, io=io,
                                    stream=stream, delta=dl)
        if op == "ties_tensor":  # thresholds at tensor scope for this mask, then the threshold merge
            mp.mp_ties_tensor_thresholds(L, base, exps, mask, cfg["density"], tau_t, residency=res, stream=stream,
                                         delta=dl)
            return mp.mp_merge_ties_tau(L, base, exps, mask, tau_t, cfg["lam"], out, residency=res, io=io,
                                        stream=stream, delta=dl)
        comb = mp.MP_COMBINE_SIGN_ELECT if cfg["combine"] == "sign_elect" else mp.MP_COMBINE_LINEAR
        alpha = None if comb == mp.MP_COMBINE_SIGN_ELECT else [1.0 / K] * K
        return mp.mp_merge_dare(L, base, exps, mask, cfg["p"], cfg["seed"], comb, alpha, cfg["lam"], out,
                                residency=res, io=io, stream=stream, delta=dl)

    def timed(fn):
        if drop is not None:
            drop()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        r = fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b), r

    reps = max(1, args.steps)
    for _ in range(max(0, args.warmup)):
        mp.mp_index_blocks(L, base, exps, sumsq, residency=res, stream=stream, delta=dl)
    idx_ms = float(np.median([timed(lambda: mp.mp_index_blocks(L, base, exps, sumsq, residency=res,
                                                                stream=stream, delta=dl))[0] for _ in range(reps)]))
    rows = []
    flags = {"none": 0, "per_byte": mp.MP_PLAN_PER_BYTE, "skip_zero": mp.MP_PLAN_SKIP_ZERO,
             "both": mp.MP_PLAN_PER_BYTE | mp.MP_PLAN_SKIP_ZERO}[args.plan_flags]
    mp.mp_plan(L, K, sumsq, w, full, mask, flags=flags, stream=stream)  # first call sets up the workspace
    m_full = None
    if args.fidelity:  # the full-read merge M_full, for the fidelity metrics
        merge()
        m_full = out.clone()
        blen = torch.from_numpy(np.asarray(lay.block_lengths(), np.int64)).to(base.device)
    for f in cfg["budgets"]:
        B = int(f * full)
        plan_ms, st = timed(lambda: mp.mp_plan(L, K, sumsq, w, B, mask, flags=flags, stream=stream))
        io = merge(io=True)
        assert io["expert_bytes"] == st["cost_bytes"]
        for _ in range(max(0, args.warmup)):
            merge()
        ms = float(np.median([timed(merge)[0] for _ in range(reps)]))
        fid = fidelity(out, m_full, blen, st["n_selected"], K * G) if args.fidelity else None
        alg = 2 * P * es + st["cost_bytes"] + 4 * G if not host else st["cost_bytes"]
        pass_bytes = 0
        if op == "ties_tensor":  # three digit passes, each reading every selected expert block and, once, the base under it
            m_np = mask.cpu().numpy()
            pass_bytes = 3 * (st["cost_bytes"] + (0 if dl else int(blen_np[m_np != 0].sum()) * es))
            alg += pass_bytes
        rows.append({"budget_frac": round(f, 4), "budget_bytes": B, "cost_bytes": st["cost_bytes"],
                     "h2d_bytes": io["h2d_bytes"], "n_selected": st["n_selected"], "plan_ms": round(plan_ms, 4),
                     "merge_ms": round(ms, 4), "merge_params_per_s": P / (ms * 1e-3),
                     ("h2d_GBps" if host else "merge_effective_GBps"): alg / (ms * 1e-3) / 1e9})
        if op == "ties_tensor":
            rows[-1]["threshold_pass_bytes"] = pass_bytes
        if fid is not None:
            rows[-1]["fidelity"] = fid
    step_ms = idx_ms + sum(r["plan_ms"] + r["merge_ms"] for r in rows)
    dma = None
    fread = None
    if files:  # measured peak: sequential read of one expert file (up to 1 GiB) after a cache drop
        import time
        drop()
        n = min(P * es, 1 << 30)
        buf = bytearray(64 << 20)
        t0 = time.perf_counter()
        with open(exps[0], "rb", buffering=0) as f:
            got = 0
            while got < n:
                r = f.readinto(buf)
                if not r:
                    break
                got += r
        fread = got / (time.perf_counter() - t0)
    if pinned or pageable:  # measured peak: pinned host -> device with the copy engine (1 GiB, or one expert)
        n = P if pinned else min(P, (1 << 30) // es)
        src = exps[0] if pinned else exps[0][:n].pin_memory()
        dst = torch.empty(n, dtype=base.dtype, device=base.device)
        dst.copy_(src[:n], non_blocking=True)
        dma_ms, _ = timed(lambda: dst.copy_(src[:n], non_blocking=True))
        dma = n * es / (dma_ms * 1e-3)
        del dst, src
    tot_bytes = sum(r["cost_bytes"] if host else 2 * P * es + r["cost_bytes"] + 4 * G for r in rows)
    if op == "ties_tensor":
        tot_bytes += sum(r["threshold_pass_bytes"] for r in rows)
    tot_ms = sum(r["merge_ms"] for r in rows)
    achieved = tot_bytes / (tot_ms * 1e-3)
    peak = PCIE_PEAK if host else HBM_PEAK
    if files and fread:  # storage bounds it: the measured sequential read rate is the peak
        peak = fread
    result = {
        "metric": f"merged params/sec, budgeted {op.upper()} merge sweep",
        "value": len(rows) * P / (step_ms * 1e-3), "unit": "params/s", "n_gpus": 1, "steps": reps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{spec.description}; {op} {cfg}", "plan_flags": args.plan_flags,
                   "experts_form": "explicit deltas" if dl else "fine-tuned weights",
                   "storage_dtype": lay.dtype, "params": P,
                   "blocks": G, "K": K, "experts": where_txt,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "storage" if files else ("pcie" if host else "hbm"), "achieved": achieved / 1e9,
                     "peak": peak / 1e9,
                     "unit": "GB/s", "frac": achieved / peak, "traffic": None,
                     "measured_dma_h2d_GBps": None if dma is None else dma / 1e9,
                     "measured_file_read_GBps": None if fread is None else fread / 1e9},
        "breakdown": {"index_ms": round(idx_ms, 4), "per_budget": rows},
    }
    if not args.no_cpu_baseline and not files:
        log("timing the CPU oracle on a sample")
        cb = cpu_baseline_sweep(spec, base, exps, cfg, flags, dl)
        if cb is not None:
            cb["host"] = host_cpu()
            if P * K <= 100_000_000:  # the whole family fits the sample: time it on one thread too
                cb1 = one_thread(lambda: cpu_baseline_sweep(spec, base, exps, cfg, flags, dl))
                cb["one_thread"] = {"value": cb1["value"], "unit": cb1["unit"], "cores": cb1["cores"],
                                    "sample": cb1["sample"]}
            result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-stride", type=int, default=2)
    ap.add_argument("--workload", default="qwen2.5-1.5b", choices=sorted(CONFIGS),
                    help="the headline (default) or one of the other workload shapes")
    ap.add_argument("--layers", type=int, default=None,
                    help="other workloads: keep only this many transformer layers (host memory)")
    ap.add_argument("--residency", default="config", choices=("config", "device", "pinned", "pageable", "file"),
                    help="other workloads: where the experts live (default: the workload's own)")
    ap.add_argument("--ties", default="catalog", choices=("catalog", "in-merge"),
                    help="where the TIES trim thresholds are found: in the index pass (catalog) or in each merge")
    ap.add_argument("--plan-flags", default="none", choices=("none", "per_byte", "skip_zero", "both"),
                    help="other workloads: mp_plan options (default: the literal Algorithm 1)")
    ap.add_argument("--experts-delta", action="store_true",
                    help="other workloads: pass the experts as stored deltas W_i - W_0 (MP_EXPERTS_DELTA)")
    ap.add_argument("--fidelity", action="store_true",
                    help="other workloads: also report Rel. l2, P95 block and Touched against the full merge")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="after the timed region, run the AVG merge once with an empty mask: a plain copy "
                         "of the base (reads 2P + 4G bytes, writes 2P) for scaling hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures one GPU only; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if CONFIGS.get(args.workload, {}).get("op") == "lora_ties":
        return run_lora(args)
    if args.workload != "qwen2.5-1.5b":
        return run_sweep(args)

    import numpy as np
    import torch

    import paper_2605_29489_amd as mp
    from workloads import family_spec, make_family_device

    torch.cuda.set_device(0)
    spec = family_spec("qwen2.5-1.5b")
    lay = spec.layout
    K = spec.K
    P = lay.n_params
    L = mp.Layout(lay.numel, lay.block_elems, mp.MP_BF16)
    G = mp.mp_layout_blocks(L)
    log(f"generating {spec.description}: P={P} G={G}")
    base, exps = make_family_device(spec, K=K, seed=0, device="cuda")
    torch.cuda.synchronize()
    sumsq = torch.empty(G * K, dtype=torch.float32, device="cuda")
    tau = torch.empty(G * K, dtype=torch.int32, device="cuda")
    masks = [torch.empty(G, dtype=torch.int32, device="cuda") for _ in BUDGETS]
    catalog = args.ties == "catalog"
    out = torch.empty_like(base)
    full = P * 2 * K
    budgets = [int(f * full) for f in BUDGETS]
    stream = torch.cuda.current_stream()

    ev = lambda: torch.cuda.Event(enable_timing=True)

    # The plans of the second and third budgets need only the index, so they
    # run on a second stream while the previous budget's merge streams HBM;
    # each merge waits for its own plan.  (Both streams at default priority.)
    pstream = torch.cuda.Stream()

    def step(rec):
        e_i0, e_i1 = ev(), ev()
        e_i0.record(stream)
        if catalog:
            mp.mp_index_ties(L, base, exps, 0.2, tau, sumsq=sumsq, stream=stream)
        else:
            mp.mp_index_blocks(L, base, exps, sumsq, stream=stream)
        e_i1.record(stream)
        pstream.wait_event(e_i1)
        stats = []
        plan_ev = []
        merge_ev = []
        for j, (B, m) in enumerate(zip(budgets, masks)):
            ps = stream if j == 0 else pstream
            a, b = ev(), ev()
            a.record(ps)
            stats.append(mp.mp_plan(L, K, sumsq, [1.0] * K, B, m, stream=ps))
            b.record(ps)
            plan_ev.append((a, b))
            if j > 0:
                stream.wait_event(b)
            a, b = ev(), ev()
            a.record(stream)
            if catalog:
                mp.mp_merge_ties_tau(L, base, exps, m, tau, 1.0, out, stream=stream)
            else:
                mp.mp_merge_ties(L, base, exps, m, 0.2, 1.0, out, stream=stream)
            b.record(stream)
            merge_ev.append((a, b))
        if rec is not None:
            rec.append((e_i0, e_i1, plan_ev, merge_ev, stats))

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    recs = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(recs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall / args.steps * 1e3

    idx_ms = np.mean([a.elapsed_time(b) for a, b, _, _, _ in recs])
    plan_ms = np.array([[a.elapsed_time(b) for a, b in r[2]] for r in recs]).mean(0)
    merge_ms = np.array([[a.elapsed_time(b) for a, b in r[3]] for r in recs]).mean(0)
    stats = recs[-1][4]
    if catalog:
        io = mp.mp_merge_ties_tau(L, base, exps, masks[0], tau, 1.0, out, io=True, stream=stream)
    else:
        io = mp.mp_merge_ties(L, base, exps, masks[0], 0.2, 1.0, out, io=True, stream=stream)
    assert io["expert_bytes"] == stats[0]["cost_bytes"]
    # the run's manifest for the first budget (after the timed region): coverage
    # per (tensor, expert), realized reads per expert, plan replay
    from paper_2605_29489_amd.manifest import build_manifest, replay
    a, b = ev(), ev()
    a.record(stream)
    cov = mp.mp_coverage(L, K, masks[0], stream=stream)
    b.record(stream)
    torch.cuda.synchronize()
    man = build_manifest(L, K, stats[0], io, cov, "ties", {"density": 0.2, "lambda": 1.0})
    rp = replay(man, mp, L, K, sumsq, [1.0] * K, masks[0], stream=stream)
    manifest_check = {"coverage_ms": round(a.elapsed_time(b), 4), "within_plan": man["realized"]["within_plan"],
                      "reads_match_coverage": man["realized"]["matches_coverage"], "replay_ok": rp["ok"]}
    # the other route, once, for reference (its own index pass first)
    if catalog:
        mp.mp_index_blocks(L, base, exps, sumsq, stream=stream)
    else:
        mp.mp_index_ties(L, base, exps, 0.2, tau, sumsq=sumsq, stream=stream)
    alt = []
    for m in masks:
        a, b = ev(), ev()
        a.record(stream)
        if catalog:
            mp.mp_merge_ties(L, base, exps, m, 0.2, 1.0, out, stream=stream)
        else:
            mp.mp_merge_ties_tau(L, base, exps, m, tau, 1.0, out, stream=stream)
        b.record(stream)
        alt.append((a, b))
    torch.cuda.synchronize()
    alt_ms = [a.elapsed_time(b) for a, b in alt]
    # measured copy rate: the library's plain stream copy of the base into the
    # output (reads and writes 2P bytes with the merges' access pattern);
    # median of five launches after one
    copy_ms = []
    for _ in range(6):
        a, b = ev(), ev()
        a.record(stream)
        mp.mp_stream_copy(base, out, stream=stream)
        b.record(stream)
        copy_ms.append((a, b))
    torch.cuda.synchronize()
    copy_ms = float(np.median([a.elapsed_time(b) for a, b in copy_ms[1:]]))
    copy_GBps = 4 * P / (copy_ms * 1e-3) / 1e9
    # and the HIP runtime's own device-to-device copy of the base (reads and
    # writes 2P bytes), median of five
    rt_ms = []
    for _ in range(6):
        a, b = ev(), ev()
        a.record(stream)
        out.copy_(base)
        b.record(stream)
        rt_ms.append((a, b))
    torch.cuda.synchronize()
    rt_ms = float(np.median([a.elapsed_time(b) for a, b in rt_ms[1:]]))
    rt_GBps = 4 * P / (rt_ms * 1e-3) / 1e9
    if args.calibration_copy:  # the AVG kernel with an empty mask copies the base:
        # a copy of known size (reads 2P + 4G, writes 2P) for the byte counters
        empty = torch.zeros(G, dtype=torch.int32, device="cuda")
        mp.mp_merge_avg(L, base, exps, empty, [0.25] * K, out, stream=stream)
        torch.cuda.synchronize()

    ckpt = P * 2
    per_budget = []
    alg_bytes = []
    for f, st, pm, mm in zip(BUDGETS, stats, plan_ms, merge_ms):
        # base + selected expert blocks + output + mask (+ one threshold per selected unit)
        byts = 2 * ckpt + st["cost_bytes"] + 4 * G + (4 * st["n_selected"] if catalog else 0)
        alg_bytes.append(byts)
        per_budget.append({
            "budget_frac": f, "budget_bytes": st["budget_bytes"], "cost_bytes": st["cost_bytes"],
            "n_selected": st["n_selected"], "plan_ms": round(float(pm), 4),
            "plan_stream": "main" if f == BUDGETS[0] else "second (overlaps the previous budget's merge)",
            "merge_ms": round(float(mm), 4),
            "merge_params_per_s": P / (mm * 1e-3),
            "merge_effective_GBps": byts / (mm * 1e-3) / 1e9,
            "merge_hbm_frac": byts / (mm * 1e-3) / HBM_PEAK,
            "digest": hex(st["digest"]),
        })
    idx_bytes = (K + 1) * ckpt + (8 if catalog else 4) * G * K
    achieved = sum(alg_bytes) / (sum(merge_ms) * 1e-3)
    traffic = stored_traffic(args.ties)
    result = {
        "metric": METRIC,
        "value": 3 * P / (ms_step * 1e-3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "qwen2.5-1.5b-shaped bf16 family, K=4, index + (plan + TIES rho=0.2 lambda=1) "
                        "at B=25/50/100% per step",
            "ties_route": args.ties,
            "storage_dtype": "bf16", "params": P, "blocks": G, "block_elems": lay.block_elems, "K": K,
            "budgets_bytes": budgets, "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": achieved / HBM_PEAK,
            "traffic": traffic,
            "kernel": ("k_merge_elem<bf16, TIES from catalog thresholds>" if catalog else "k_merge_ties<bf16>")
                      + " (device-resident experts)",
            "measured_copy": {"GBps": copy_GBps, "frac_of_peak": copy_GBps * 1e9 / HBM_PEAK,
                              "ms": round(copy_ms, 4),
                              "kernel": "mp_stream_copy of the base (reads and writes 2P bytes; 16-byte "
                                        "non-temporal loads and stores, one chunk per lane)"},
            "frac_of_measured_copy": achieved / (copy_GBps * 1e9),
            "measured_runtime_copy": {"GBps": rt_GBps, "frac_of_peak": rt_GBps * 1e9 / HBM_PEAK,
                                      "ms": round(rt_ms, 4),
                                      "kernel": "the HIP runtime's device-to-device copy of the base "
                                                "(reads and writes 2P bytes)"},
        },
        "breakdown": {
            "index_ms": round(float(idx_ms), 4),
            "index_kernel": "k_index_ties<bf16> (sums of squares + thresholds)" if catalog else "k_index<bf16>",
            "index_effective_GBps": idx_bytes / (idx_ms * 1e-3) / 1e9,
            "index_hbm_frac": idx_bytes / (idx_ms * 1e-3) / HBM_PEAK,
            "per_budget": per_budget,
            "other_route": {"route": "in-merge" if catalog else "catalog",
                            "merge_ms": [round(float(x), 4) for x in alt_ms]},
            "manifest_B0": manifest_check,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cb = cpu_baseline(spec, base, exps, args.ties, args.cpu_stride)
        log("timing the CPU oracle on one thread (a smaller sample)")
        cb1 = one_thread(lambda: cpu_baseline(spec, base, exps, args.ties, 16 * args.cpu_stride))
        cb["host"] = host_cpu()
        cb["one_thread"] = {"value": cb1["value"], "unit": cb1["unit"], "cores": cb1["cores"],
                            "sample": cb1["sample"]}
        result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
