"""Run manifest and replay check.

The executor of the paper records, per run, the touched blocks, the
contributing experts and the realized I/O in a manifest (Section 3), and the
plan carries a digest of its selected blocks (Algorithm 1).  This module
assembles that record from what the library returns -- mp_plan's stats, a
merge's io stats (in-kernel counters of the expert bytes actually loaded,
split by expert) and mp_coverage's per-(tensor, expert) touched elements --
and replays a plan to check that it reproduces.  It computes nothing of the
merge itself.
"""

import json
from typing import Optional, Sequence

FORMAT = "mergepipe-manifest/1"


def build_manifest(layout, K: int, plan_stats: dict, io_stats: dict, coverage, op: str, params: dict,
                   tensor_names: Optional[Sequence[str]] = None, inputs: Optional[dict] = None) -> dict:
    """A JSON-serialisable manifest of one budgeted merge.

    layout: the binding's Layout; coverage: mp_coverage's [n_tensors, K]
    array; inputs: caller-supplied identities of the base and experts
    (lineage), recorded as given."""
    numel = [int(n) for n in layout.numel]
    es = 4 if int(layout.dtype) == 0 else 2
    P = sum(numel)
    by_expert = [int(x) for x in io_stats["expert_bytes_by_expert"][:K]]
    cov_bytes = [sum(int(coverage[t][i]) for t in range(len(numel))) * es for i in range(K)]
    tensors = []
    for t, n in enumerate(numel):
        row = [int(coverage[t][i]) for i in range(K)]
        tensors.append({
            "name": tensor_names[t] if tensor_names is not None else str(t),
            "numel": n,
            "touched_elements": row,
            "contributing_experts": [i for i in range(K) if row[i] > 0],
        })
    return {
        "format": FORMAT,
        "op": op,
        "params": params,
        "K": K,
        "layout": {"n_tensors": len(numel), "params": P, "block_elems": int(layout.block_elems),
                   "dtype": "f32" if es == 4 else "bf16"},
        "plan": {
            "budget_bytes": int(plan_stats["budget_bytes"]),
            "cost_bytes": int(plan_stats["cost_bytes"]),
            "full_bytes": int(plan_stats["full_bytes"]),
            "n_selected": int(plan_stats["n_selected"]),
            "n_units": int(plan_stats["n_units"]),
            "digest": "0x%016x" % int(plan_stats["digest"]),
        },
        "realized": {
            "expert_bytes": int(io_stats["expert_bytes"]),
            "expert_bytes_by_expert": by_expert,
            "h2d_bytes": int(io_stats["h2d_bytes"]),
            "base_bytes": int(io_stats["base_bytes"]),
            "out_bytes": int(io_stats["out_bytes"]),
            # Prop. 1: the loaded expert bytes are those of the selected units
            "within_plan": int(io_stats["expert_bytes"]) <= int(plan_stats["cost_bytes"]),
            "matches_coverage": by_expert == cov_bytes,
        },
        "touched": {
            "units": int(plan_stats["n_selected"]) / max(int(plan_stats["n_units"]), 1),
            "elements_by_expert": [c / es / P if P else 0.0 for c in cov_bytes],
        },
        "tensors": tensors,
        "inputs": inputs or {},
    }


def dumps(manifest: dict) -> str:
    return json.dumps(manifest, indent=1, sort_keys=True)


def replay(manifest: dict, mp, layout, K: int, sumsq, w, mask, flags: int = 0, stream=None) -> dict:
    """Re-runs the manifest's plan (same catalog sums sumsq, weights w and
    flags) into the device buffer mask and compares it with the record."""
    st = mp.mp_plan(layout, K, sumsq, w, manifest["plan"]["budget_bytes"], mask, flags=flags, stream=stream)
    got = {"cost_bytes": int(st["cost_bytes"]), "n_selected": int(st["n_selected"]),
           "digest": "0x%016x" % int(st["digest"])}
    want = {k: manifest["plan"][k] for k in got}
    return {"ok": got == want, "replayed": got, "recorded": want}
