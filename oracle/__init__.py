"""CPU oracle for one sequence-parallel rank's attention shard.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product library and
its Python binding never do, and the two share no code.

Plain, slow, float64 (numpy) implementations written from the paper
(arXiv 2505.22296): masked attention forward / backward for a rank's shard
(Sections 3.2, 4, 5.2), Dummy-Head Ulysses pad/unpad and the pack/unpack
around the Ulysses all-to-all with the summing unpack of replicated GQA K/V
gradients (Section 4.1, Listing 1), and the Ring-Attention
log-sum-exp merge (Section 2.1, Table 1), and the all-rank USP simulation
(Ulysses inside, zigzag ring outside; Table 1); `loss`: the SP-aware loss
reduction (token log-probabilities, SFT / DPO over all-reduced sums, the
all-reduce's gradient; Sections 3.3 and 5.1).  See each module's docstring.
"""
from . import loss
from .attention import (bf16_bits_to_f64, segment_ids, allowed_mask, local_heads,
                        attn_forward, attn_backward, attn_dq_rows, attn_dkdv_keys)
from .sp import (pad_heads, unpad_heads, ulysses_pack, ulysses_unpack, ulysses_unpack_add,
                 ulysses_unpack_add_bf16, f32_to_bf16_bits, all_to_all, lse_merge,
                 ring_forward, ring_backward, ulysses_simulate, ulysses_simulate_backward,
                 usp_simulate)

__all__ = [
    "bf16_bits_to_f64", "segment_ids", "allowed_mask", "local_heads", "attn_forward",
    "attn_backward", "attn_dq_rows", "attn_dkdv_keys", "pad_heads", "unpad_heads",
    "ulysses_pack", "ulysses_unpack", "ulysses_unpack_add", "ulysses_unpack_add_bf16",
    "f32_to_bf16_bits", "all_to_all", "lse_merge", "ring_forward", "ring_backward",
    "ulysses_simulate", "ulysses_simulate_backward", "usp_simulate", "loss",
]
