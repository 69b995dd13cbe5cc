"""Shape tables and the seeded value recipe for synthetic checkpoint families.

A checkpoint is one flat buffer holding its tensors back to back, each tensor
flattened row-major, in the order listed by the shape table.  The paper's
checkpoints are experts obtained by fine-tuning one common base model
(Sections 1 and 2); the recipe below imitates that structure:

* base weights ~ N(0, 0.02^2); normalisation weights 1 + N(0, 0.02^2);
  generated in fp32, then rounded to the family dtype;
* expert i, per consecutive run of ``block_elems`` elements of a tensor
  ("data block"): with probability-free exact count, ``round(zeta_i * G)``
  data blocks (chosen by a seeded permutation) are left untouched, the rest
  get a delta d ~ N(0, s^2) with s = exp(ln 1e-3 + xi), xi ~ N(0, 1)
  (log-normal per block);
* W_i = round_to_dtype(float32(W_0 + d)); untouched blocks copy W_0 bitwise.

The data blocks here are only a property of the *input distribution* (the
per-block scale of the synthetic fine-tune); how the merge method partitions
a checkpoint is computed independently by each implementation.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

DTYPE_CODES = {"f32": 0, "bf16": 1}
DTYPE_BYTES = {"f32": 4, "bf16": 2}


@dataclass(frozen=True)
class Layout:
    """Tensor numels of a flat checkpoint plus block size and dtype."""

    numel: Tuple[int, ...]
    block_elems: int
    dtype: str  # "f32" or "bf16"

    @property
    def n_params(self) -> int:
        return int(sum(self.numel))

    @property
    def elem_bytes(self) -> int:
        return DTYPE_BYTES[self.dtype]

    @property
    def dtype_code(self) -> int:
        return DTYPE_CODES[self.dtype]

    @property
    def ckpt_bytes(self) -> int:
        return self.n_params * self.elem_bytes

    def block_lengths(self) -> List[int]:
        """Element counts of the blocks in order (each tensor cut into
        block_elems runs, the last one short)."""
        out = []
        for n in self.numel:
            full, tail = divmod(int(n), self.block_elems)
            out += [self.block_elems] * full + ([tail] if tail else [])
        return out


@dataclass(frozen=True)
class FamilySpec:
    name: str
    tensors: Tuple[Tuple[str, Tuple[int, ...]], ...]
    dtype: str
    block_elems: int = 4096
    K: int = 4
    zero_frac: Tuple[float, ...] = ()
    description: str = ""

    @property
    def layout(self) -> Layout:
        numel = tuple(int(np.prod(s)) for _, s in self.tensors)
        return Layout(numel=numel, block_elems=self.block_elems, dtype=self.dtype)

    def zeta(self, i: int) -> float:
        if self.zero_frac:
            return float(self.zero_frac[i])
        return 0.2


def _qwen_like(n_layers, hidden, ffn, n_q, n_kv, head_dim, vocab, tied):
    q = n_q * head_dim
    kv = n_kv * head_dim
    t: List[Tuple[str, Tuple[int, ...]]] = [("embed_tokens.weight", (vocab, hidden))]
    for l in range(n_layers):
        p = f"layers.{l}."
        t += [
            (p + "self_attn.q_proj.weight", (q, hidden)),
            (p + "self_attn.q_proj.bias", (q,)),
            (p + "self_attn.k_proj.weight", (kv, hidden)),
            (p + "self_attn.k_proj.bias", (kv,)),
            (p + "self_attn.v_proj.weight", (kv, hidden)),
            (p + "self_attn.v_proj.bias", (kv,)),
            (p + "self_attn.o_proj.weight", (hidden, q)),
            (p + "mlp.gate_proj.weight", (ffn, hidden)),
            (p + "mlp.up_proj.weight", (ffn, hidden)),
            (p + "mlp.down_proj.weight", (hidden, ffn)),
            (p + "input_layernorm.weight", (hidden,)),
            (p + "post_attention_layernorm.weight", (hidden,)),
        ]
    t.append(("norm.weight", (hidden,)))
    if not tied:
        t.append(("lm_head.weight", (vocab, hidden)))
    return tuple(t)


def _llama_like(n_layers, hidden, ffn, n_q, n_kv, head_dim, vocab, tied):
    q = n_q * head_dim
    kv = n_kv * head_dim
    t: List[Tuple[str, Tuple[int, ...]]] = [("embed_tokens.weight", (vocab, hidden))]
    for l in range(n_layers):
        p = f"layers.{l}."
        t += [
            (p + "self_attn.q_proj.weight", (q, hidden)),
            (p + "self_attn.k_proj.weight", (kv, hidden)),
            (p + "self_attn.v_proj.weight", (kv, hidden)),
            (p + "self_attn.o_proj.weight", (hidden, q)),
            (p + "mlp.gate_proj.weight", (ffn, hidden)),
            (p + "mlp.up_proj.weight", (ffn, hidden)),
            (p + "mlp.down_proj.weight", (hidden, ffn)),
            (p + "input_layernorm.weight", (hidden,)),
            (p + "post_attention_layernorm.weight", (hidden,)),
        ]
    t.append(("norm.weight", (hidden,)))
    if not tied:
        t.append(("lm_head.weight", (vocab, hidden)))
    return tuple(t)


def _toy():
    return tuple((f"w{j}", (512, 1024)) for j in range(8))


def family_spec(name: str, n_layers: Optional[int] = None, vocab: Optional[int] = None) -> FamilySpec:
    """Return the family spec ``name``; ``n_layers``/``vocab`` truncate the
    shape for small parity cases (same tensor shapes, fewer of them)."""
    if name == "toy":
        return FamilySpec("toy", _toy(), "f32", 4096, 4, (),
                          "fp32 toy: 8 x (512x1024), K=4")
    if name == "qwen2.5-1.5b":
        L = 28 if n_layers is None else n_layers
        V = 151936 if vocab is None else vocab
        return FamilySpec(name, _qwen_like(L, 1536, 8960, 12, 2, 128, V, True), "bf16", 4096, 4, (),
                          f"Qwen2.5-1.5B-shaped bf16, {L} layers, vocab {V}, tied, K=4")
    if name == "llama3-8b":
        L = 32 if n_layers is None else n_layers
        V = 128256 if vocab is None else vocab
        return FamilySpec(name, _llama_like(L, 4096, 14336, 32, 8, 128, V, False), "bf16", 4096, 8, (),
                          f"Llama-3-8B-shaped bf16, {L} layers, vocab {V}, untied, K=8")
    if name == "qwen2.5-7b":
        L = 28 if n_layers is None else n_layers
        V = 152064 if vocab is None else vocab
        return FamilySpec(name, _qwen_like(L, 3584, 18944, 28, 4, 128, V, False), "bf16", 4096, 8, (),
                          f"Qwen2.5-7B-shaped bf16, {L} layers, vocab {V}, untied, K=8")
    if name == "llama3-8b-k16":
        L = 32 if n_layers is None else n_layers
        V = 128256 if vocab is None else vocab
        z = tuple(0.8 * i / 15.0 for i in range(16))
        return FamilySpec(name, _llama_like(L, 4096, 14336, 32, 8, 128, V, False), "bf16", 4096, 16, z,
                          f"Llama-3-8B-shaped bf16, {L} layers, K=16, 0-80% zero blocks")
    raise KeyError(name)


# The five workloads and the operator settings each is quoted with.
CONFIGS = {
    "toy": dict(family="toy", op="avg", budgets=(0.5,), residency="device"),
    "qwen2.5-1.5b": dict(family="qwen2.5-1.5b", op="ties", density=0.2, lam=1.0,
                         budgets=(0.25, 0.5, 1.0), residency="device"),
    "qwen2.5-1.5b-ties-sweep": dict(family="qwen2.5-1.5b", op="ties", density=0.2, lam=1.0,
                                    budgets=(1.0, 0.9, 0.8, 0.7, 0.6, 0.5), residency="device"),
    "qwen2.5-1.5b-ties-tensor": dict(family="qwen2.5-1.5b", op="ties_tensor", density=0.2, lam=1.0,
                                     budgets=(0.25, 0.5, 1.0), residency="device"),
    "qwen2.5-1.5b-lora-ties": dict(family="qwen2.5-1.5b", op="lora_ties", rank=16, scale=2.0, density=0.2,
                                   lam=1.0, budgets=(0.25, 0.5, 1.0), residency="device"),
    "qwen2.5-1.5b-avg-renorm": dict(family="qwen2.5-1.5b", op="avg_renorm", budgets=(0.25, 0.5, 1.0),
                                    residency="device"),
    "llama3-8b": dict(family="llama3-8b", op="avg", budgets=tuple(x / 10 for x in range(1, 11)),
                      residency="host_pinned"),
    "qwen2.5-7b": dict(family="qwen2.5-7b", op="dare", p=0.9, seed=7, combine="sign_elect", lam=1.0,
                       budgets=(0.3,), residency="device"),
    "qwen2.5-7b-dare-sweep": dict(family="qwen2.5-7b", op="dare", p=0.9, seed=7, combine="sign_elect", lam=1.0,
                                  budgets=(0.1, 0.3, 0.6), residency="device"),
    "qwen2.5-1.5b-avg": dict(family="qwen2.5-1.5b", op="avg", budgets=(0.25, 0.5, 1.0), residency="device"),
    "qwen2.5-1.5b-dare-lin": dict(family="qwen2.5-1.5b", op="dare", p=0.9, seed=7, combine="linear", lam=1.0,
                                  budgets=(0.25, 0.5, 1.0), residency="device"),
    "llama3-8b-k16": dict(family="llama3-8b-k16", op="ties", density=0.1, lam=1.0,
                          budgets=(1 / 16, 0.1, 0.25, 0.5, 0.75, 1.0), residency="host_pinned"),
}


def _is_norm(name: str) -> bool:
    return "layernorm" in name or name.startswith("norm.")


def _data_blocks(n: int, be: int) -> int:
    return (n + be - 1) // be


def _expert_block_scales(torch, spec: FamilySpec, i: int, seed: int, device):
    """Per data-block delta scale for expert i (0 for untouched blocks)."""
    lay = spec.layout
    nblk = sum(_data_blocks(n, lay.block_elems) for n in lay.numel)
    g = torch.Generator(device="cpu")
    g.manual_seed(1_000_003 * (seed + 1) + 7919 * (i + 1))
    xi = torch.randn(nblk, generator=g, dtype=torch.float64)
    sig = torch.exp(math.log(1e-3) + xi).to(torch.float32)
    nz = int(round(spec.zeta(i) * nblk))
    if nz > 0:
        perm = torch.randperm(nblk, generator=g)
        sig[perm[:nz]] = 0.0
    return sig.to(device)


def _fill(torch, spec: FamilySpec, K: int, seed: int, device, out_base, out_experts, tensor_filter=None):
    lay = spec.layout
    tdt = torch.float32 if lay.dtype == "f32" else torch.bfloat16
    be = lay.block_elems
    gb = torch.Generator(device=device)
    scales = [_expert_block_scales(torch, spec, i, seed, device) for i in range(K)]
    gens = []
    for i in range(K):
        ge = torch.Generator(device=device)
        ge.manual_seed(97 * (seed + 1) + 131 * (i + 1) + 17)
        gens.append(ge)
    gb.manual_seed(seed * 7 + 3)
    off = 0
    blk = 0
    for (name, shape), n in zip(spec.tensors, lay.numel):
        nb = _data_blocks(n, be)
        w0 = torch.randn(n, generator=gb, device=device, dtype=torch.float32) * 0.02
        if _is_norm(name):
            w0 = w0 + 1.0
        w0q = w0.to(tdt)
        out_base[off:off + n].copy_(w0q)
        w0f = w0q.to(torch.float32)
        for i in range(K):
            s = scales[i][blk:blk + nb]
            s_el = torch.repeat_interleave(s, be)[:n]
            d = torch.randn(n, generator=gens[i], device=device, dtype=torch.float32) * s_el
            wi = (w0f + d).to(tdt)
            out_experts[i][off:off + n].copy_(wi)
        off += n
        blk += nb
    return out_base, out_experts


def make_family(spec: FamilySpec, K: Optional[int] = None, seed: int = 0):
    """Generate base + K experts on the CPU; returns numpy arrays.

    fp32 families come back as float32 arrays, bf16 families as uint16 arrays
    holding the raw bfloat16 bit patterns.
    """
    import torch

    K = spec.K if K is None else K
    lay = spec.layout
    tdt = torch.float32 if lay.dtype == "f32" else torch.bfloat16
    P = lay.n_params
    base = torch.empty(P, dtype=tdt)
    experts = [torch.empty(P, dtype=tdt) for _ in range(K)]
    _fill(torch, spec, K, seed, "cpu", base, experts)
    if lay.dtype == "f32":
        return base.numpy(), [e.numpy() for e in experts]
    return base.view(torch.int16).numpy().view(np.uint16), [e.view(torch.int16).numpy().view(np.uint16) for e in experts]


def pinned_empty(n: int, dtype_name: str):
    """A CPU tensor of n elements whose storage is an exact-size hipHostMalloc
    allocation (pinned host memory), freed when the tensor is collected.

    torch's own pinned allocator rounds every request up to a power of two,
    which doubles the footprint of 16 GB experts."""
    import ctypes
    import weakref

    import torch

    hip = ctypes.CDLL("libamdhip64.so")
    es = DTYPE_BYTES[dtype_name]
    ptr = ctypes.c_void_p()
    rc = hip.hipHostMalloc(ctypes.byref(ptr), ctypes.c_size_t(max(n * es, 1)), ctypes.c_uint(0))
    if rc != 0 or not ptr.value:
        raise MemoryError(f"hipHostMalloc of {n * es} bytes failed (error {rc})")
    raw = (ctypes.c_uint8 * (n * es)).from_address(ptr.value)
    arr = np.frombuffer(raw, dtype=np.int16 if es == 2 else np.float32, count=n)
    t = torch.from_numpy(arr)
    if dtype_name == "bf16":
        t = t.view(torch.bfloat16)
    weakref.finalize(arr, hip.hipHostFree, ptr)
    t._pinned_owner = arr  # keeps the allocation alive as long as the tensor
    return t


def make_family_device(spec: FamilySpec, K: Optional[int] = None, seed: int = 0, device="cuda",
                       experts_on_host_pinned: bool = False, experts_on_host: Optional[str] = None):
    """Generate base + K experts as torch tensors on ``device``.

    ``experts_on_host`` = "pinned" (or ``experts_on_host_pinned``) or
    "pageable": the experts are generated on the device one at a time and
    copied into pinned, or ordinary, host tensors (the base stays on device).
    The values depend on the device's RNG, so families generated on different
    devices differ; consumers that need the same bytes copy them.
    """
    import torch

    K = spec.K if K is None else K
    lay = spec.layout
    tdt = torch.float32 if lay.dtype == "f32" else torch.bfloat16
    P = lay.n_params
    host = experts_on_host or ("pinned" if experts_on_host_pinned else None)
    if host not in (None, "pinned", "pageable"):
        raise ValueError(f"experts_on_host must be 'pinned' or 'pageable', not {host!r}")
    base = torch.empty(P, dtype=tdt, device=device)
    if host is None:
        experts = [torch.empty(P, dtype=tdt, device=device) for _ in range(K)]
        _fill(torch, spec, K, seed, device, base, experts)
        return base, experts
    # one device scratch expert at a time, then copy to host memory
    experts = []
    scratch = torch.empty(P, dtype=tdt, device=device)
    # generate base once with K=0 then each expert with the same per-expert streams
    _fill(torch, spec, 0, seed, device, base, [])
    for i in range(K):
        _fill_one_expert(torch, spec, i, seed, device, base, scratch)
        h = pinned_empty(P, lay.dtype) if host == "pinned" else torch.empty(P, dtype=tdt)
        h.copy_(scratch)
        experts.append(h)
    del scratch
    return base, experts


def _fill_one_expert(torch, spec: FamilySpec, i: int, seed: int, device, base, out):
    """Regenerate expert i exactly as ``_fill`` would (same RNG streams)."""
    lay = spec.layout
    tdt = torch.float32 if lay.dtype == "f32" else torch.bfloat16
    be = lay.block_elems
    s_all = _expert_block_scales(torch, spec, i, seed, device)
    ge = torch.Generator(device=device)
    ge.manual_seed(97 * (seed + 1) + 131 * (i + 1) + 17)
    off = 0
    blk = 0
    for n in lay.numel:
        nb = _data_blocks(n, be)
        w0f = base[off:off + n].to(torch.float32)
        s_el = torch.repeat_interleave(s_all[blk:blk + nb], be)[:n]
        d = torch.randn(n, generator=ge, device=device, dtype=torch.float32) * s_el
        out[off:off + n].copy_((w0f + d).to(tdt))
        off += n
        blk += nb
    return out


# ---------------------------------------------------------------- low-rank adapter experts

LORA_TARGETS = ("q_proj.weight", "k_proj.weight", "v_proj.weight", "o_proj.weight",
                "gate_proj.weight", "up_proj.weight", "down_proj.weight")


def lora_records(spec: FamilySpec, rank: int, scale: float, targets=LORA_TARGETS):
    """Adapter records for the spec's 2-D tensors whose names end with one of
    ``targets`` (None: every 2-D tensor): tuples (tensor, rows, cols, rank,
    a_off, b_off, scale), with A (rank x cols) then B (rows x rank) packed per
    tensor in layout order.  Returns (records, elements per adapter buffer)."""
    recs, off = [], 0
    for t, (name, shape) in enumerate(spec.tensors):
        if len(shape) != 2 or (targets is not None and not name.endswith(tuple(targets))):
            continue
        rows, cols = shape
        recs.append((t, rows, cols, rank, off, off + rank * cols, float(scale)))
        off += rank * (rows + cols)
    return recs, off


def make_lora_adapters(n: int, K: int, dtype: str, seed: int = 0, grid: bool = False, std: float = 0.02):
    """K adapter buffers of n elements, as numpy arrays (float32, or uint16
    bfloat16 patterns).  grid=True draws j/64 with j uniform in [-8, 8): on
    that grid every rank sum of products is exact in fp32.  Otherwise
    N(0, std^2), rounded to the dtype."""
    import torch

    rng = np.random.default_rng(seed)
    out = []
    for _ in range(K):
        if grid:
            x = (rng.integers(-8, 8, n) / 64.0).astype(np.float32)
        else:
            x = (rng.standard_normal(n) * std).astype(np.float32)
        if dtype == "bf16":
            x = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        out.append(x)
    return out
