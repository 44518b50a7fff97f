"""Helpers shared by the tests: building library descriptors and oracle
keyword arguments from one problem description, moving bf16 bits to the GPU,
and error metrics.  Torch's GPU context is only touched inside functions."""
from __future__ import annotations

import math
import os
import re

import numpy as np

from workloads import Shard

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Tolerances for bf16 attention outputs and gradients vs the fp64 oracle.
MAX_ABS = 2e-2
REL_L2 = 5e-3
LSE_MAX_ABS = 1e-3


def header_functions():
    """Function names declared in include/sp_attn.h."""
    with open(os.path.join(ROOT, "include", "sp_attn.h")) as f:
        txt = f.read()
    return sorted(set(re.findall(r"^\s*(?:sp_status|const char\*|int32_t)\s+(sp_\w+)\s*\(", txt, re.M)))


def oracle_kw(sh: Shard, pos_q=None, pos_k=None, causal=None):
    # pieces of one sequence are one segment for the oracle (its mask then
    # depends on positions alone)
    cu_q = np.array([0, sh.cu_q[-1]]) if sh.single_sequence else sh.cu_q
    cu_k = np.array([0, sh.cu_k[-1]]) if sh.single_sequence else sh.cu_k
    return dict(cu_q=cu_q, cu_k=cu_k,
                pos_q=sh.pos_q if pos_q is None else pos_q,
                pos_k=sh.pos_k if pos_k is None else pos_k,
                H_loc=sh.H_loc, head_offset=sh.head_offset, num_real_heads=sh.num_real_heads,
                gqa_group=sh.gqa_group, kv_head_offset=sh.kv_head_offset, scale=sh.scale,
                causal=sh.causal if causal is None else causal)


def lib_desc(sh: Shard, pos_q=None, pos_k=None, causal=None, T_k=None, rowstats_ready=False,
             dq_acc_init=False):
    from paper_2505_22296_amd import Desc
    return Desc(T_q=sh.T_q, T_k=sh.T_k if T_k is None else T_k, head_dim=sh.D, H_loc=sh.H_loc,
                head_offset=sh.head_offset, num_real_heads=sh.num_real_heads,
                num_padded_heads=sh.num_padded_heads, gqa_group=sh.gqa_group,
                Hkv_loc=sh.Hkv_loc, kv_head_offset=sh.kv_head_offset, cu_seqlens_q=sh.cu_q,
                cu_seqlens_k=sh.cu_k, position_ids_q=sh.pos_q if pos_q is None else pos_q,
                position_ids_k=sh.pos_k if pos_k is None else pos_k,
                causal=sh.causal if causal is None else causal, softmax_scale=sh.scale,
                single_sequence=sh.single_sequence, rowstats_ready=rowstats_ready,
                dq_acc_init=dq_acc_init)


def to_dev(bits: np.ndarray):
    """uint16 bf16 bits -> torch.bfloat16 tensor on cuda:0 (same bits)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to("cuda:0")


def from_dev(t) -> np.ndarray:
    """GPU tensor -> float64 numpy (bf16 decoded exactly)."""
    import torch
    return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)


def bits_from_dev(t) -> np.ndarray:
    import torch
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def errs(gpu: np.ndarray, ref: np.ndarray):
    d = np.abs(gpu - ref)
    mx = float(d.max()) if d.size else 0.0
    nr = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(gpu - ref) / nr) if nr > 0 else float(np.linalg.norm(gpu - ref))
    return mx, rel


# Magnitude past which one bf16 rounding step (ulp 2^-5 on [4, 8)) alone
# exceeds half of MAX_ABS.
SCALED_FROM = 4.0


def scaled_max_abs(ref) -> float:
    """Absolute bar for bf16 results: MAX_ABS while the largest reference
    magnitude is at most SCALED_FROM; past it, two bf16 ulps of the largest
    reference value (2^-7 of it), where one rounding step alone exceeds half
    of MAX_ABS.  rel-L2 keeps REL_L2 either way."""
    m = float(np.abs(ref).max()) if np.size(ref) else 0.0
    if m <= SCALED_FROM:
        return MAX_ABS
    return max(MAX_ABS, 2.0 ** -7 * m)


def widened(ref) -> bool:
    """Whether scaled_max_abs(ref) is above the flat MAX_ABS bar."""
    return scaled_max_abs(ref) > MAX_ABS


def assert_close(gpu, ref, what, max_abs=MAX_ABS, rel_l2=REL_L2):
    mx, rel = errs(gpu, ref)
    assert mx <= max_abs and rel <= rel_l2, f"{what}: max_abs={mx:.3e} rel_l2={rel:.3e}"
    return mx, rel


def make_shard(name, T_q, T_k, D, H_loc, head_offset, num_real, num_padded, gqa, Hkv_loc,
               kv_off, seg_q, seg_k=None, pos_q=None, pos_k=None, causal=True, seed_base=0,
               single_sequence=False):
    """Explicit small problem (segments given as lengths; positions default to
    0.. per segment)."""
    cu_q = np.concatenate([[0], np.cumsum(seg_q)]).astype(np.int32)
    cu_k = cu_q.copy() if seg_k is None else np.concatenate([[0], np.cumsum(seg_k)]).astype(np.int32)

    def ramp(cu, T):
        p = np.zeros(T, np.int32)
        for s in range(len(cu) - 1):
            p[cu[s]:cu[s + 1]] = np.arange(cu[s + 1] - cu[s])
        return p

    return Shard(name=name, T_q=T_q, T_k=T_k, D=D, H_loc=H_loc, head_offset=head_offset,
                 num_real_heads=num_real, num_padded_heads=num_padded, gqa_group=gqa,
                 Hkv_loc=Hkv_loc, kv_head_offset=kv_off, cu_q=cu_q, cu_k=cu_k,
                 pos_q=ramp(cu_q, T_q) if pos_q is None else np.asarray(pos_q, np.int32),
                 pos_k=ramp(cu_k, T_k) if pos_k is None else np.asarray(pos_k, np.int32),
                 causal=causal, seed_base=seed_base, single_sequence=single_sequence)
