"""Host logic of the run manifest (no GPU): the record it assembles from
plan stats, realized-read counters and coverage."""

import json

import numpy as np

from paper_2605_29489_amd import Layout, MP_BF16
from paper_2605_29489_amd.manifest import FORMAT, build_manifest, dumps


def _inputs():
    lay = Layout([8192, 4100, 16], 4096, MP_BF16)  # blocks: 2, 2 (4096 + 4), 1
    K = 3
    # mask per block (bit i = expert i): t0 b0 {0,2}, t0 b1 {0}, t1 b0 {1}, t1 b1 {}, t2 b0 {2}
    cov = np.array([[8192, 0, 4096], [0, 4096, 0], [0, 0, 16]], np.uint64)
    plan = dict(budget_bytes=40000, cost_bytes=2 * (8192 + 4096 + 4096 + 16), full_bytes=2 * 3 * 12308,
                n_selected=5, n_units=15, digest=0x1234)
    by = [2 * 8192, 2 * 4096, 2 * (4096 + 16)] + [0] * 29
    io = dict(expert_bytes=sum(by), expert_bytes_by_expert=by, h2d_bytes=0, base_bytes=2 * 12308,
              out_bytes=2 * 12308)
    return lay, K, plan, io, cov


def test_manifest_records_coverage_and_realized_reads():
    lay, K, plan, io, cov = _inputs()
    m = build_manifest(lay, K, plan, io, cov, "avg", {"alpha": [1 / 3] * 3}, tensor_names=["a", "b", "c"],
                       inputs={"base": "b0"})
    assert m["format"] == FORMAT
    assert [t["contributing_experts"] for t in m["tensors"]] == [[0, 2], [1], [2]]
    assert m["tensors"][1]["touched_elements"] == [0, 4096, 0]
    assert m["realized"]["within_plan"] and m["realized"]["matches_coverage"]
    assert m["touched"]["units"] == 5 / 15
    assert np.allclose(m["touched"]["elements_by_expert"], [8192 / 12308, 4096 / 12308, 4112 / 12308])
    assert m["plan"]["digest"] == "0x0000000000001234"
    assert json.loads(dumps(m)) == json.loads(json.dumps(m))


def test_manifest_flags_reads_that_disagree_with_the_mask():
    lay, K, plan, io, cov = _inputs()
    io = dict(io)
    by = list(io["expert_bytes_by_expert"])
    by[1] += 2 * 16  # a block of expert 1 the mask does not select was read
    io["expert_bytes_by_expert"] = by
    io["expert_bytes"] = sum(by)
    m = build_manifest(lay, K, plan, io, cov, "avg", {})
    assert not m["realized"]["matches_coverage"]
    assert not m["realized"]["within_plan"]
