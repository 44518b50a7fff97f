"""ctypes binding of libspattn.so (argument marshalling only).

Every computation happens in the HIP library; this module only turns torch
tensors into device pointers, the current torch stream into a hipStream_t,
and allocates outputs/workspaces with torch's caching allocator.  If the
compiled library is missing, loading fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspattn.so")

SP_OK, SP_ERR_INVALID_ARG, SP_ERR_UNSUPPORTED, SP_ERR_WORKSPACE, SP_ERR_HIP = range(5)
SP_OP_FWD, SP_OP_BWD, SP_OP_RING_STEP = 0, 1, 2
SP_DESC_SINGLE_SEQUENCE = 1
SP_DESC_ROWSTATS_READY = 4
SP_DESC_DQ_ACC_INIT = 8
SCHED_ITEM_INTS = 8

_i32p = ctypes.POINTER(ctypes.c_int32)


class SpAttnDesc(ctypes.Structure):
    _fields_ = [
        ("T_q", ctypes.c_int32), ("T_k", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("H_loc", ctypes.c_int32), ("head_offset", ctypes.c_int32),
        ("num_real_heads", ctypes.c_int32), ("num_padded_heads", ctypes.c_int32),
        ("gqa_group", ctypes.c_int32), ("Hkv_loc", ctypes.c_int32),
        ("kv_head_offset", ctypes.c_int32), ("num_seqs", ctypes.c_int32),
        ("causal", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
        ("flags", ctypes.c_int32),
        ("cu_seqlens_q", _i32p), ("cu_seqlens_k", _i32p),
        ("position_ids_q", _i32p), ("position_ids_k", _i32p),
    ]


class SpError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib = None


def load() -> ctypes.CDLL:
    """Load libspattn.so (after torch, so the library binds to the HIP
    runtime torch already loaded)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (HIP runtime first)
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} not built; run `python -m paper_2505_22296_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(SpAttnDesc)
    sig = {
        "sp_status_string": (ctypes.c_char_p, [i32]),
        "sp_version": (i32, []),
        "sp_ulysses_pack": (i32, [vp, i32, i32, i32, i32, i32, _i32p, vp, vp]),
        "sp_ulysses_unpack": (i32, [vp, i32, i32, i32, i32, _i32p, i32, vp, vp]),
        "sp_ulysses_unpack_add": (i32, [vp, i32, i32, i32, i32, _i32p, i32, vp, vp]),
        "sp_token_logprob": (i32, [vp, vp, i32, i32, i32, _i32p, i32, vp, vp, vp, vp]),
        "sp_token_logprob_bwd": (i32, [vp, vp, vp, i32, i32, i32, _i32p, i32, vp, vp, vp]),
        "sp_loss_reduce": (i32, [vp, vp, i32, i32, i32, ctypes.c_float, vp, vp, vp]),
        "sp_attn_workspace_size": (i32, [D, i32, ctypes.POINTER(sz)]),
        "sp_attn_fwd": (i32, [D, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sp_attn_fwd_static": (i32, [D, vp, vp, vp, vp, vp, vp]),
        "sp_attn_bwd": (i32, [D, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "sp_ring_step": (i32, [D, vp, vp, vp, vp, vp, i32, vp, vp, sz, vp]),
        "sp_lse_merge": (i32, [vp, vp, vp, i32, vp, i32, i32, i32, vp, vp]),
        "sp_f32_to_bf16": (i32, [vp, vp, ctypes.c_int64, vp]),
        "sp_attn_schedule": (i32, [D, i32, _i32p, i32, _i32p]),
        "sp_profile_events": (i32, [i32, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


EXPORTED = ["sp_status_string", "sp_version", "sp_ulysses_pack", "sp_ulysses_unpack",
            "sp_ulysses_unpack_add", "sp_token_logprob", "sp_token_logprob_bwd", "sp_loss_reduce",
            "sp_attn_workspace_size", "sp_attn_fwd", "sp_attn_fwd_static", "sp_attn_bwd", "sp_ring_step",
            "sp_lse_merge", "sp_f32_to_bf16", "sp_attn_schedule", "sp_profile_events"]

SP_KERNEL_ATTN_FWD, SP_KERNEL_ATTN_DQ, SP_KERNEL_ATTN_DKDV = 1, 2, 3
SP_KERNEL_PACK, SP_KERNEL_UNPACK, SP_KERNEL_LSE_MERGE, SP_KERNEL_UNPACK_ADD = 4, 5, 6, 7
SP_KERNEL_TOKEN_LOGPROB, SP_KERNEL_TOKEN_LOGPROB_BWD = 8, 9
SP_LOSS_SFT, SP_LOSS_DPO = 0, 1


def status_string(s: int) -> str:
    return load().sp_status_string(int(s)).decode()


def _check(status: int, where: str):
    if status != SP_OK:
        raise SpError(status, where)


class Desc:
    """Owns an sp_attn_desc and the host arrays it points to."""

    def __init__(self, *, T_q, T_k, head_dim, H_loc, head_offset, num_real_heads,
                 num_padded_heads, gqa_group, Hkv_loc, kv_head_offset, cu_seqlens_q,
                 cu_seqlens_k, position_ids_q=None, position_ids_k=None, causal=True,
                 softmax_scale=None, single_sequence=False, rowstats_ready=False,
                 dq_acc_init=False):
        self._keep = []

        def arr(x):
            if x is None:
                return None
            a = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
            self._keep.append(a)
            return a.ctypes.data_as(_i32p)

        cq = np.asarray(cu_seqlens_q, dtype=np.int32)
        # the C ABI reads these host arrays by the counts in the descriptor
        if len(np.asarray(cu_seqlens_k)) != len(cq):
            raise ValueError("cu_seqlens_q and cu_seqlens_k need the same length (num_seqs + 1)")
        for name, pos, T in (("position_ids_q", position_ids_q, T_q),
                             ("position_ids_k", position_ids_k, T_k)):
            if pos is not None and len(np.asarray(pos)) < T:
                raise ValueError(f"{name} has fewer than {T} entries")
        self.c = SpAttnDesc(
            T_q=T_q, T_k=T_k, head_dim=head_dim, H_loc=H_loc, head_offset=head_offset,
            num_real_heads=num_real_heads, num_padded_heads=num_padded_heads,
            gqa_group=gqa_group, Hkv_loc=Hkv_loc, kv_head_offset=kv_head_offset,
            num_seqs=max(0, len(cq) - 1), causal=1 if causal else 0,
            softmax_scale=(1.0 / math.sqrt(head_dim)) if softmax_scale is None else softmax_scale,
            flags=((SP_DESC_SINGLE_SEQUENCE if single_sequence else 0)
                   | (SP_DESC_ROWSTATS_READY if rowstats_ready else 0)
                   | (SP_DESC_DQ_ACC_INIT if dq_acc_init else 0)),
            cu_seqlens_q=arr(cu_seqlens_q), cu_seqlens_k=arr(cu_seqlens_k),
            position_ids_q=arr(position_ids_q), position_ids_k=arr(position_ids_k))

    @property
    def ref(self):
        return ctypes.byref(self.c)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _alloc_on(stream=None):
    """Context for the wrapper's own allocations (outputs, workspace): on the
    stream the kernels are launched on.  torch's caching allocator ties a
    block to the stream current at allocation and, once the tensor is
    dropped, hands it to the next allocation on that stream without waiting
    for other streams; a workspace allocated on the current stream but read
    by kernels queued on `stream` could be reused while they still run."""
    import contextlib
    import torch
    if stream is None:
        return contextlib.nullcontext()
    return torch.cuda.stream(stream)


def sp_attn_workspace_size(desc: Desc, op: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().sp_attn_workspace_size(desc.ref, op, ctypes.byref(n)), "sp_attn_workspace_size")
    return n.value


def _workspace(desc: Desc, op: int, device, ws=None):
    import torch
    need = sp_attn_workspace_size(desc, op)
    if ws is not None and ws.numel() >= need:
        return ws, ws.numel()
    return torch.empty(need, dtype=torch.uint8, device=device), need


def sp_attn_schedule(desc: Desc, op: int) -> np.ndarray:
    """Host-side work list: [n_items, 8] int32 (see include/sp_attn.h)."""
    lib = load()
    n = ctypes.c_int32(0)
    _check(lib.sp_attn_schedule(desc.ref, op, None, 0, ctypes.byref(n)), "sp_attn_schedule")
    out = np.zeros((max(1, n.value), SCHED_ITEM_INTS), dtype=np.int32)
    _check(lib.sp_attn_schedule(desc.ref, op, out.ctypes.data_as(_i32p), n.value, ctypes.byref(n)),
           "sp_attn_schedule")
    return out[: n.value]


def sp_ulysses_pack(src, sp: int, H_dst_loc: int, head_map: Sequence[int], dst=None, stream=None):
    """src [T_loc, H_src, D] bf16 -> dst [sp, T_loc, H_dst_loc, D] bf16."""
    import torch
    T, Hs, D = src.shape
    if dst is None:
        with _alloc_on(stream):
            dst = torch.empty((sp, T, H_dst_loc, D), dtype=src.dtype, device=src.device)
    m = np.ascontiguousarray(np.asarray(head_map, dtype=np.int32))
    _check(load().sp_ulysses_pack(_ptr(src), T, Hs, D, sp, H_dst_loc, m.ctypes.data_as(_i32p),
                                  _ptr(dst), _stream(stream)), "sp_ulysses_pack")
    return dst


def sp_ulysses_unpack(src, head_map: Sequence[int], H_dst: int, dst=None, stream=None):
    """src [sp, T_loc, H_src_loc, D] bf16 -> dst [T_loc, H_dst, D] bf16."""
    import torch
    sp, T, Hs, D = src.shape
    if dst is None:
        with _alloc_on(stream):
            dst = torch.empty((T, H_dst, D), dtype=src.dtype, device=src.device)
    m = np.ascontiguousarray(np.asarray(head_map, dtype=np.int32))
    _check(load().sp_ulysses_unpack(_ptr(src), T, Hs, D, sp, m.ctypes.data_as(_i32p), H_dst,
                                    _ptr(dst), _stream(stream)), "sp_ulysses_unpack")
    return dst


def sp_ulysses_unpack_add(src, head_map: Sequence[int], H_dst: int, dst=None, stream=None):
    """src [sp, T_loc, H_src_loc, D] bf16 -> dst [T_loc, H_dst, D] bf16: the
    copies of a head that several slots name are summed (float32, ascending
    slot order, one rounding to bf16)."""
    import torch
    sp, T, Hs, D = src.shape
    if dst is None:
        with _alloc_on(stream):
            dst = torch.empty((T, H_dst, D), dtype=src.dtype, device=src.device)
    m = np.ascontiguousarray(np.asarray(head_map, dtype=np.int32))
    _check(load().sp_ulysses_unpack_add(_ptr(src), T, Hs, D, sp, m.ctypes.data_as(_i32p), H_dst,
                                        _ptr(dst), _stream(stream)), "sp_ulysses_unpack_add")
    return dst


def _cu(cu_seqlens):
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    return cu, len(cu) - 1


def sp_token_logprob(logits, labels, cu_seqlens, ignore_index: int = -100, logp=None, lse=None,
                     seq_sum=None, stream=None):
    """logits [T, V] bf16, labels [T] int32 (device) -> (logp [T], lse [T],
    seq_sum [num_seqs]) float32."""
    import torch
    T, V = logits.shape
    cu, n = _cu(cu_seqlens)
    dev = logits.device
    with _alloc_on(stream):
        logp = torch.empty(T, dtype=torch.float32, device=dev) if logp is None else logp
        lse = torch.empty(T, dtype=torch.float32, device=dev) if lse is None else lse
        if seq_sum is None:
            seq_sum = torch.empty(max(n, 0), dtype=torch.float32, device=dev)
    _check(load().sp_token_logprob(_ptr(logits), _ptr(labels), T, V, ignore_index,
                                   cu.ctypes.data_as(_i32p), n, _ptr(logp), _ptr(lse),
                                   _ptr(seq_sum) if n > 0 else None, _stream(stream)),
           "sp_token_logprob")
    return logp, lse, seq_sum


def sp_token_logprob_bwd(logits, labels, lse, cu_seqlens, grad_seq, ignore_index: int = -100,
                         dlogits=None, stream=None):
    """-> dlogits [T, V] bf16 = g (onehot(label) - softmax(logits)) per
    counted token, g = grad_seq[its sequence]."""
    import torch
    T, V = logits.shape
    cu, n = _cu(cu_seqlens)
    if dlogits is None:
        with _alloc_on(stream):
            dlogits = torch.empty_like(logits)
    _check(load().sp_token_logprob_bwd(_ptr(logits), _ptr(labels), _ptr(lse), T, V, ignore_index,
                                       cu.ctypes.data_as(_i32p), n, _ptr(grad_seq), _ptr(dlogits),
                                       _stream(stream)), "sp_token_logprob_bwd")
    return dlogits


def sp_loss_reduce(partial_sums, kind: int, coef: float, ref_partial_sums=None, loss=None,
                   grad=None, stream=None):
    """partial_sums [sp, n] float32 -> (loss [1], grad [sp, n]): the loss over
    the ranks' all-reduced sums and each rank's upstream gradient."""
    import torch
    spn, n = partial_sums.shape
    dev = partial_sums.device
    with _alloc_on(stream):
        loss = torch.empty(1, dtype=torch.float32, device=dev) if loss is None else loss
        grad = torch.empty((spn, n), dtype=torch.float32, device=dev) if grad is None else grad
    _check(load().sp_loss_reduce(_ptr(partial_sums), _ptr(ref_partial_sums), spn, n, kind,
                                 float(coef), _ptr(loss), _ptr(grad), _stream(stream)),
           "sp_loss_reduce")
    return loss, grad


def sp_attn_fwd(desc: Desc, q, k, v, o=None, lse=None, workspace=None, stream=None):
    import torch
    c = desc.c
    with _alloc_on(stream):
        if o is None:
            o = torch.empty((c.T_q, c.H_loc, c.head_dim), dtype=q.dtype, device=q.device)
        if lse is None:
            lse = torch.empty((c.H_loc, c.T_q), dtype=torch.float32, device=q.device)
        ws, nb = _workspace(desc, SP_OP_FWD, q.device, workspace)
        _check(load().sp_attn_fwd(desc.ref, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                  _ptr(ws), nb, _stream(stream)), "sp_attn_fwd")
    return o, lse


STATIC_SCRATCH_BYTES = 1 << 20


def sp_attn_fwd_static(desc: Desc, q, k, v, o, lse, stream=None):
    """Allocation-free forward: outputs must be given (o [T_q, H_loc, D]
    bf16, lse [H_loc, T_q] float32); the work list lives in the library's
    fixed device array (STATIC_SCRATCH_BYTES per GPU)."""
    _check(load().sp_attn_fwd_static(desc.ref, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                     _stream(stream)), "sp_attn_fwd_static")
    return o, lse


def sp_attn_bwd(desc: Desc, q, k, v, o, lse, dout, dq=None, dq_acc=None, dk=None, dv=None,
                workspace=None, stream=None):
    import torch
    with _alloc_on(stream):
        if dq is None and dq_acc is None:
            dq = torch.empty_like(q)
        if dk is None:
            dk = torch.empty_like(k)
        if dv is None:
            dv = torch.empty_like(v)
        ws, nb = _workspace(desc, SP_OP_BWD, q.device, workspace)
        _check(load().sp_attn_bwd(desc.ref, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                  _ptr(dout), _ptr(dq), _ptr(dq_acc), _ptr(dk), _ptr(dv),
                                  _ptr(ws), nb, _stream(stream)), "sp_attn_bwd")
    return (dq if dq is not None else dq_acc), dk, dv


def sp_ring_step(desc: Desc, q, k_chunk, v_chunk, o_acc, lse_acc, init: bool, o_out=None,
                 workspace=None, stream=None):
    with _alloc_on(stream):
        ws, nb = _workspace(desc, SP_OP_RING_STEP, q.device, workspace)
        _check(load().sp_ring_step(desc.ref, _ptr(q), _ptr(k_chunk), _ptr(v_chunk), _ptr(o_acc),
                                   _ptr(lse_acc), 1 if init else 0, _ptr(o_out), _ptr(ws), nb,
                                   _stream(stream)), "sp_ring_step")
    return o_acc, lse_acc


def sp_lse_merge(o_acc, lse_acc, o_part, lse_part, o_out=None, stream=None):
    import torch
    T, H, D = o_acc.shape
    is_bf16 = 1 if o_part.dtype == torch.bfloat16 else 0
    _check(load().sp_lse_merge(_ptr(o_acc), _ptr(lse_acc), _ptr(o_part), is_bf16, _ptr(lse_part),
                               T, H, D, _ptr(o_out), _stream(stream)), "sp_lse_merge")
    return o_acc, lse_acc


def sp_f32_to_bf16(src, dst=None, stream=None):
    import torch
    if dst is None:
        with _alloc_on(stream):
            dst = torch.empty(src.shape, dtype=torch.bfloat16, device=src.device)
    _check(load().sp_f32_to_bf16(_ptr(src), _ptr(dst), src.numel(), _stream(stream)),
           "sp_f32_to_bf16")
    return dst


def sp_profile_events(kernel_id: int, start=None, stop=None):
    """Arm (or with None, disarm) the per-thread timer of one kernel with
    torch.cuda.Event objects (enable_timing=True; recorded once beforehand so
    the underlying hipEvent exists)."""
    _check(load().sp_profile_events(kernel_id, None if start is None else start.cuda_event,
                                    None if stop is None else stop.cuda_event),
           "sp_profile_events")
