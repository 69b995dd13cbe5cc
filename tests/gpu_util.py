"""Helpers for the GPU parity tests: moving checkpoint arrays between numpy
(fp32 arrays, or uint16 arrays of raw bfloat16 patterns) and torch device
tensors, and the merge tolerance."""

import numpy as np


def to_dev(a, dtype, device="cuda"):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device)


def to_pinned(a, dtype):
    """A new pinned host tensor holding the array (allocated pinned, never
    registered after the fact)."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    return t.pin_memory()


def to_host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def gather_blocks(t, blocks, ids):
    """Copy the listed blocks of a device checkpoint into one compact host
    array; returns (array, doff) with doff the element offset of each block."""
    import torch
    idx = np.concatenate([np.arange(blocks.off[g], blocks.off[g] + blocks.len[g]) for g in ids])
    sel = t[torch.from_numpy(idx).to(t.device)]
    doff = np.concatenate([[0], np.cumsum(blocks.len[ids])[:-1]]).astype(np.int64)
    return to_host(sel), doff


def assert_merge_equal(got, want, base, dtype, what=""):
    """The merge tolerance: fp32 |g - o| <= 1e-6 * max(|o|, |base|); bf16 at
    most 1 ulp apart after the final rounding.  Returns the number of
    elements that are not bitwise equal."""
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape
    if dtype == "bf16":
        g = got.view(np.int16).astype(np.int32)
        w = want.view(np.int16).astype(np.int32)
        # ulp distance on the sign-magnitude patterns
        gm = np.where(g < 0, -(g & 0x7FFF), g)
        wm = np.where(w < 0, -(w & 0x7FFF), w)
        dist = np.abs(gm - wm)
        bad = dist > 1
        assert not bad.any(), f"{what}: {int(bad.sum())} bf16 elements differ by > 1 ulp (max {int(dist.max())})"
        return int((got != want).sum())
    gf = got.astype(np.float64)
    wf = want.astype(np.float64)
    bf = np.asarray(base).astype(np.float64)
    tol = 1e-6 * np.maximum(np.abs(wf), np.abs(bf))
    bad = np.abs(gf - wf) > tol
    assert not bad.any(), f"{what}: {int(bad.sum())} fp32 elements outside 1e-6 relative"
    return int((got.view(np.uint32) != want.view(np.uint32)).sum())
