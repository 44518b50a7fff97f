"""MI355X (gfx950) per-rank attention for Dummy-Head Ulysses and Ring-Attention
sequence parallelism (arXiv 2505.22296), behind the C ABI of include/sp_attn.h.

The Python surface mirrors the C entry points one to one; see `_lib`.
"""
from ._lib import (Desc, SpError, load, status_string, sp_attn_workspace_size, sp_attn_schedule,
                   sp_ulysses_pack, sp_ulysses_unpack, sp_ulysses_unpack_add, sp_attn_fwd,
                   sp_attn_fwd_static, STATIC_SCRATCH_BYTES,
                   sp_attn_bwd, sp_ring_step, sp_lse_merge, sp_f32_to_bf16, sp_profile_events,
                   sp_token_logprob, sp_token_logprob_bwd, sp_loss_reduce, SP_LOSS_SFT, SP_LOSS_DPO,
                   SP_KERNEL_TOKEN_LOGPROB, SP_KERNEL_TOKEN_LOGPROB_BWD,
                   SP_OK, SP_ERR_INVALID_ARG, SP_ERR_UNSUPPORTED, SP_ERR_WORKSPACE, SP_ERR_HIP,
                   SP_OP_FWD, SP_OP_BWD, SP_OP_RING_STEP, SP_DESC_SINGLE_SEQUENCE, SP_DESC_ROWSTATS_READY,
                   SP_DESC_DQ_ACC_INIT,
                   EXPORTED,
                   LIB_PATH, SP_KERNEL_ATTN_FWD, SP_KERNEL_ATTN_DQ, SP_KERNEL_ATTN_DKDV,
                   SP_KERNEL_PACK, SP_KERNEL_UNPACK, SP_KERNEL_LSE_MERGE, SP_KERNEL_UNPACK_ADD)

__all__ = [
    "Desc", "SpError", "load", "status_string", "sp_attn_workspace_size", "sp_attn_schedule",
    "sp_ulysses_pack", "sp_ulysses_unpack", "sp_ulysses_unpack_add", "sp_attn_fwd",
    "sp_attn_fwd_static", "STATIC_SCRATCH_BYTES",
    "sp_attn_bwd", "sp_ring_step", "sp_lse_merge", "sp_f32_to_bf16", "sp_profile_events",
    "sp_token_logprob", "sp_token_logprob_bwd", "sp_loss_reduce", "SP_LOSS_SFT", "SP_LOSS_DPO",
    "SP_KERNEL_TOKEN_LOGPROB", "SP_KERNEL_TOKEN_LOGPROB_BWD",
    "SP_OK", "SP_ERR_INVALID_ARG", "SP_ERR_UNSUPPORTED", "SP_ERR_WORKSPACE", "SP_ERR_HIP",
    "SP_OP_FWD", "SP_OP_BWD", "SP_OP_RING_STEP", "SP_DESC_SINGLE_SEQUENCE",
    "SP_DESC_ROWSTATS_READY", "SP_DESC_DQ_ACC_INIT", "EXPORTED",
    "LIB_PATH", "SP_KERNEL_ATTN_FWD", "SP_KERNEL_ATTN_DQ", "SP_KERNEL_ATTN_DKDV", "SP_KERNEL_PACK",
    "SP_KERNEL_UNPACK", "SP_KERNEL_LSE_MERGE", "SP_KERNEL_UNPACK_ADD",
]
