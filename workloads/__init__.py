"""Seeded synthetic checkpoint families for the budgeted-merge path.

This package only *produces inputs*: tensor shape tables shaped like the
paper's Qwen and Llama merge workloads (Section 4 evaluates Qwen3 and
Llama-3 families, which are not available here) and a seeded value recipe
for a base checkpoint and K fine-tuned experts.  It holds none of the merge
method's arithmetic (no deltas, norms, plans or merges); the CPU oracle and
the GPU library both consume the bytes generated here.
"""

from .families import (  # noqa: F401
    CONFIGS,
    FamilySpec,
    Layout,
    family_spec,
    make_family,
    make_family_device,
    lora_records,
    make_lora_adapters,
)
