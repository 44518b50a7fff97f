#!/usr/bin/env python3
"""Benchmark of one sequence-parallel rank's attention shard on MI355X.

Metric: attention forward+backward TFLOP/s counting real heads only
(14 * D * allowed_pairs * H_real per step), and its fraction of the MI355X
bf16 dense MFMA peak (2.5 PFLOP/s).

A step is one pass of the rank's hot path over one batch of synthetic input
already resident in HBM:
  Ulysses shard: pack Q, K, V (dummy-head zero fill) -> attention forward ->
      unpack O -> pack dO -> attention backward -> unpack dQ (MHA: dK, dV too;
      GQA: summing unpack of the dK, dV copies received from the ranks that
      share each KV head)
  packed varlen shard: attention forward -> backward
  ring rank r: r+1 fused ring steps (LSE merge in the epilogue, bf16 O on the
      last) -> per-chunk backward into an fp32 dQ accumulator -> dQ to bf16
  USP rank (Ulysses inside a zigzag-ring group): the Ulysses pack of Q, K, V
      and dO and unpack of O, dQ (summing unpack of dK, dV) around the zigzag
      ring steps and their backward
The all-to-all itself is not run (one GPU).

Output: ONE JSON line on stdout (driver contract), with a `roofline` object
for the dominant kernel (HIP-event timed on the library's stream) and a
`cpu_baseline` object (the fp64 oracle on a bounded sample on host cores).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from workloads import (allowed_pairs, ring_chunk_positions, shard_inputs, randn_bf16_bits,  # noqa: E402
                       ulysses_kv_head_map, ulysses_q_head_map, workload, WORKLOADS,
                       zigzag_inputs, zigzag_step_positions)

METRIC = "attn fwd+bwd TFLOP/s (real heads) per SP-rank shard; % of bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, published
# the largest single-GPU shard: ring rank 4 of 8 over a 131072-token
# sequence (Q chunk of 16384 against KV chunks 0..4), 28 query / 4 KV heads
DEFAULT_WORKLOAD = "ring_L131072_8chunks_r4_q28kv4_d128"
# shards with dummy slots, for the dummy-head overhead (1 of 4 and 2 of 3)
DUMMY_WORKLOADS = ("ulysses_tiny_L1024_mha7of8_sp2_r1_d64",
                   "ulysses_long_L131072_4x32768_q40kv8_sp16_r13_d128")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class KernelTimers:
    """Event pairs armed around individual library kernels (sp_profile_events)."""

    def __init__(self, sp, torch):
        self.sp, self.torch = sp, torch
        self.pool, self.used, self.on = [], [], False
        self.only = None  # set of kernel ids to time (None: every kernel)

    def reserve(self, n):
        """Create (and record once) n event pairs ahead of the timed region."""
        while len(self.pool) < n:
            a = self.torch.cuda.Event(enable_timing=True)
            b = self.torch.cuda.Event(enable_timing=True)
            a.record()
            b.record()
            self.pool.append((a, b))

    def arm(self, kid, flops, nbytes=0.0):
        if not self.on or (self.only is not None and kid not in self.only):
            return
        self.reserve(len(self.used) + 1)
        pair = self.pool[len(self.used)]
        self.used.append((kid, flops, nbytes, pair))
        self.sp.sp_profile_events(kid, *pair)

    def disarm(self):
        for kid in KNAMES:
            self.sp.sp_profile_events(kid, None, None)

    def summary(self):
        out = {}
        for kid, flops, nbytes, (a, b) in self.used:
            ms = a.elapsed_time(b)
            s = out.setdefault(kid, {"ms": 0.0, "n": 0, "flops": 0.0, "bytes": 0.0, "all": []})
            s["ms"] += ms
            s["n"] += 1
            s["flops"] += flops
            s["bytes"] += nbytes
            s["all"].append(ms)
        return out


KNAMES = {1: "attn_fwd_kernel", 2: "attn_dq_kernel", 3: "attn_dkdv_kernel", 4: "pack_kernel",
          5: "unpack_kernel", 6: "merge_kernel", 7: "unpack_add_kernel"}


def lib_desc(sp, sh, pos_k=None, rowstats_ready=False, dq_acc_init=False):
    return sp.Desc(rowstats_ready=rowstats_ready, dq_acc_init=dq_acc_init, T_q=sh.T_q, T_k=sh.T_k,
                   head_dim=sh.D, H_loc=sh.H_loc,
                   head_offset=sh.head_offset, num_real_heads=sh.num_real_heads,
                   num_padded_heads=sh.num_padded_heads, gqa_group=sh.gqa_group,
                   Hkv_loc=sh.Hkv_loc, kv_head_offset=sh.kv_head_offset,
                   cu_seqlens_q=sh.cu_q, cu_seqlens_k=sh.cu_k, position_ids_q=sh.pos_q,
                   position_ids_k=sh.pos_k if pos_k is None else pos_k, causal=sh.causal,
                   softmax_scale=sh.scale, single_sequence=sh.single_sequence)


def to_dev(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


class Step:
    """Buffers and the launch sequence of one step for a workload."""

    def __init__(self, sp, torch, sh, timers):
        self.sp, self.torch, self.sh, self.t = sp, torch, sh, timers
        dev = "cuda"
        D = sh.D
        self.ring = sh.ring_chunks > 0
        nr = sh.n_real_loc
        if self.ring and sh.zigzag_sp:
            # zigzag ring: the rank's two chunks against the two chunks of each step
            self.descs = [lib_desc(sp, sh, zigzag_step_positions(sh, s))
                          for s in range(sh.ring_chunks)]
            # backward: the row statistics formed by step 0's call are reused;
            # step 0 starts the dQ accumulator
            self.descs_b = [lib_desc(sp, sh, zigzag_step_positions(sh, s), rowstats_ready=s > 0,
                                     dq_acc_init=s == 0)
                            for s in range(sh.ring_chunks)]
            self.pairs = [allowed_pairs(sh.cu_q, sh.cu_k, sh.pos_q, zigzag_step_positions(sh, s),
                                        single_sequence=True) for s in range(sh.ring_chunks)]
            q, do = zigzag_inputs(sh)
            self.q, self.do = to_dev(torch, q), to_dev(torch, do)
            self.k, self.v = [], []
            for s in range(sh.ring_chunks):
                k, v = zigzag_inputs(sh, s)
                self.k.append(to_dev(torch, k))
                self.v.append(to_dev(torch, v))
        elif self.ring:
            self.descs = [lib_desc(sp, sh, ring_chunk_positions(sh, c)) for c in range(sh.ring_chunks)]
            self.descs_b = [lib_desc(sp, sh, ring_chunk_positions(sh, c), rowstats_ready=c > 0,
                                     dq_acc_init=c == 0)
                            for c in range(sh.ring_chunks)]
            self.pairs = [allowed_pairs(sh.cu_q, sh.cu_k, sh.pos_q, ring_chunk_positions(sh, c))
                          for c in range(sh.ring_chunks)]
            q, _, _, do = shard_inputs(sh, chunk=0)
            self.q, self.do = to_dev(torch, q), to_dev(torch, do)
            self.k, self.v = [], []
            for c in range(sh.ring_chunks):
                _, k, v, _ = shard_inputs(sh, chunk=c)
                self.k.append(to_dev(torch, k))
                self.v.append(to_dev(torch, v))
        if self.ring:
            self.o_acc = torch.empty((sh.T_q, sh.H_loc, D), dtype=torch.float32, device=dev)
            self.lse_acc = torch.empty((sh.H_loc, sh.T_q), dtype=torch.float32, device=dev)
            self.o = torch.empty((sh.T_q, sh.H_loc, D), dtype=torch.bfloat16, device=dev)
            self.dq_acc = torch.empty((sh.T_q, sh.H_loc, D), dtype=torch.float32, device=dev)
            self.dq = torch.empty((sh.T_q, sh.H_loc, D), dtype=torch.bfloat16, device=dev)
            self.dk = [torch.empty_like(x) for x in self.k]
            self.dv = [torch.empty_like(x) for x in self.v]
            self.ws_f = torch.empty(max(sp.sp_attn_workspace_size(d, sp.SP_OP_RING_STEP)
                                        for d in self.descs), dtype=torch.uint8, device=dev)
            self.ws_b = torch.empty(max(sp.sp_attn_workspace_size(d, sp.SP_OP_BWD)
                                        for d in self.descs), dtype=torch.uint8, device=dev)
            self._ulysses_setup(sh)  # USP: Ulysses exchange inside the ring group
        else:
            self.desc = lib_desc(sp, sh)
            self.pairs = [allowed_pairs(sh.cu_q, sh.cu_k, sh.pos_q, sh.pos_k)]
            q, k, v, do = shard_inputs(sh)
            self.q, self.k, self.v, self.do = (to_dev(torch, x) for x in (q, k, v, do))
            self.o = torch.empty_like(self.q)
            self.lse = torch.empty((sh.H_loc, sh.T_q), dtype=torch.float32, device=dev)
            self.dq = torch.empty_like(self.q)
            self.dk = torch.empty_like(self.k)
            self.dv = torch.empty_like(self.v)
            self.ws_f = torch.empty(sp.sp_attn_workspace_size(self.desc, sp.SP_OP_FWD),
                                    dtype=torch.uint8, device=dev)
            self.ws_b = torch.empty(sp.sp_attn_workspace_size(self.desc, sp.SP_OP_BWD),
                                    dtype=torch.uint8, device=dev)
            self._ulysses_setup(sh)
        H = nr * D
        self.flops_fwd = [4.0 * H * p for p in self.pairs]
        self.flops_dq = [6.0 * H * p for p in self.pairs]
        self.flops_dkdv = [8.0 * H * p for p in self.pairs]  # S, dV, dP, dK
        self.flops_metric = 14.0 * H * sum(self.pairs)
        self.flops_strict = 12.0 * H * sum(self.pairs)
        sh_ = sh
        self.pack_bytes = 0
        if self.ulysses:
            el = 2 * sh_.D
            Tl = self.Tl
            self.pack_bytes = Tl * sh_.hs * el + sh_.sp * Tl * sh_.H_loc * el


    def _ulysses_setup(self, sh):
        """Buffers of the Ulysses exchange around attention: the rank's
        pre-all-to-all token slices, head maps, send buffers, and the
        reverse-side outputs."""
        torch, dev, D = self.torch, "cuda", sh.D
        self.ulysses = sh.sp > 1
        if self.ulysses:
            Tl = sh.T_q // sh.sp
            self.Tl = Tl
            sb = sh.seed_base + 50
            # the rank's pre-all-to-all token slice of every head
            self.q_pre = to_dev(torch, randn_bf16_bits((Tl, sh.hs, D), sb))
            self.do_pre = to_dev(torch, randn_bf16_bits((Tl, sh.hs, D), sb + 1))
            self.k_pre = to_dev(torch, randn_bf16_bits((Tl, sh.hkv, D), sb + 2))
            self.v_pre = to_dev(torch, randn_bf16_bits((Tl, sh.hkv, D), sb + 3))
            self.qmap = ulysses_q_head_map(sh.hs, sh.sp)
            self.mha = sh.hkv == sh.hs
            self.kmap = self.qmap if self.mha else ulysses_kv_head_map(sh.hs, sh.hkv, sh.sp)
            self.kw = len(self.kmap) // sh.sp
            # algorithmic bytes of each copy: named slots read, every slot
            # (dummies as zeros) written; the unpacks read named slots only
            row = Tl * D * 2
            named_q, named_kv = int(np.sum(self.qmap >= 0)), int(np.sum(self.kmap >= 0))
            self.bytes_pack_q = row * (named_q + len(self.qmap))
            self.bytes_pack_kv = row * (named_kv + len(self.kmap))
            self.bytes_unpack_q = row * 2 * named_q
            self.bytes_unpack_add = row * (named_kv + sh.hkv)
            self.send_q = torch.empty((sh.sp, Tl, sh.H_loc, D), dtype=torch.bfloat16, device=dev)
            self.send_do = torch.empty_like(self.send_q)
            self.send_k = torch.empty((sh.sp, Tl, self.kw, D), dtype=torch.bfloat16, device=dev)
            self.send_v = torch.empty_like(self.send_k)
            self.o_pre = torch.empty((Tl, sh.hs, D), dtype=torch.bfloat16, device=dev)
            self.dq_pre = torch.empty_like(self.o_pre)
            self.dk_pre = torch.empty((Tl, sh.hkv, D), dtype=torch.bfloat16, device=dev)
            self.dv_pre = torch.empty_like(self.dk_pre)
            if not self.mha:
                # reverse all-to-all receive buffers of dK / dV: chunk j is
                # what rank j returns for the KV heads it was sent (the
                # other ranks' gradients are synthetic here: one GPU)
                self.recv_dk = to_dev(torch, randn_bf16_bits((sh.sp, Tl, self.kw, D), sb + 4))
                self.recv_dv = to_dev(torch, randn_bf16_bits((sh.sp, Tl, self.kw, D), sb + 5))

    def run(self):
        sp, t, sh = self.sp, self.t, self.sh
        if self.ulysses:
            t.arm(sp.SP_KERNEL_PACK, 0.0, self.bytes_pack_q)
            sp.sp_ulysses_pack(self.q_pre, sh.sp, sh.H_loc, self.qmap, dst=self.send_q)
            t.arm(sp.SP_KERNEL_PACK, 0.0, self.bytes_pack_kv)
            sp.sp_ulysses_pack(self.k_pre, sh.sp, self.kw, self.kmap, dst=self.send_k)
            t.arm(sp.SP_KERNEL_PACK, 0.0, self.bytes_pack_kv)
            sp.sp_ulysses_pack(self.v_pre, sh.sp, self.kw, self.kmap, dst=self.send_v)
        if self.ring:
            n = len(self.descs)
            for c in range(n):
                t.arm(sp.SP_KERNEL_ATTN_FWD, self.flops_fwd[c])
                sp.sp_ring_step(self.descs[c], self.q, self.k[c], self.v[c], self.o_acc,
                                self.lse_acc, init=(c == 0), o_out=self.o if c == n - 1 else None,
                                workspace=self.ws_f)
        else:
            t.arm(sp.SP_KERNEL_ATTN_FWD, self.flops_fwd[0])
            sp.sp_attn_fwd(self.desc, self.q, self.k, self.v, self.o, self.lse,
                           workspace=self.ws_f)
        if self.ulysses:
            t.arm(sp.SP_KERNEL_UNPACK, 0.0, self.bytes_unpack_q)
            sp.sp_ulysses_unpack(self.o.view(sh.sp, self.Tl, sh.H_loc, sh.D), self.qmap, sh.hs,
                                 dst=self.o_pre)
            t.arm(sp.SP_KERNEL_PACK, 0.0, self.bytes_pack_q)
            sp.sp_ulysses_pack(self.do_pre, sh.sp, sh.H_loc, self.qmap, dst=self.send_do)
        if self.ring:
            # the first chunk starts the fp32 dQ accumulator, the last one
            # writes the bf16 dQ from it (no clearing, no separate cast)
            for c in range(n):
                t.arm(sp.SP_KERNEL_ATTN_DQ, self.flops_dq[c])
                t.arm(sp.SP_KERNEL_ATTN_DKDV, self.flops_dkdv[c])
                sp.sp_attn_bwd(self.descs_b[c], self.q, self.k[c], self.v[c], self.o, self.lse_acc,
                               self.do, dq=self.dq if c == n - 1 else None, dq_acc=self.dq_acc,
                               dk=self.dk[c], dv=self.dv[c], workspace=self.ws_b)
        else:
            t.arm(sp.SP_KERNEL_ATTN_DQ, self.flops_dq[0])
            t.arm(sp.SP_KERNEL_ATTN_DKDV, self.flops_dkdv[0])
            sp.sp_attn_bwd(self.desc, self.q, self.k, self.v, self.o, self.lse, self.do,
                           dq=self.dq, dk=self.dk, dv=self.dv, workspace=self.ws_b)
        if self.ulysses:
            t.arm(sp.SP_KERNEL_UNPACK, 0.0, self.bytes_unpack_q)
            sp.sp_ulysses_unpack(self.dq.view(sh.sp, self.Tl, sh.H_loc, sh.D), self.qmap, sh.hs,
                                 dst=self.dq_pre)
            if self.mha and not self.ring:
                t.arm(sp.SP_KERNEL_UNPACK, 0.0, self.bytes_unpack_q)
                sp.sp_ulysses_unpack(self.dk.view(sh.sp, self.Tl, sh.H_loc, sh.D), self.qmap,
                                     sh.hkv, dst=self.dk_pre)
                t.arm(sp.SP_KERNEL_UNPACK, 0.0, self.bytes_unpack_q)
                sp.sp_ulysses_unpack(self.dv.view(sh.sp, self.Tl, sh.H_loc, sh.D), self.qmap,
                                     sh.hkv, dst=self.dv_pre)
            elif not self.mha:
                t.arm(sp.SP_KERNEL_UNPACK_ADD, 0.0, self.bytes_unpack_add)
                sp.sp_ulysses_unpack_add(self.recv_dk, self.kmap, sh.hkv, dst=self.dk_pre)
                t.arm(sp.SP_KERNEL_UNPACK_ADD, 0.0, self.bytes_unpack_add)
                sp.sp_ulysses_unpack_add(self.recv_dv, self.kmap, sh.hkv, dst=self.dv_pre)


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def monolithic_problem(sh):
    """The shard as one attention problem for the oracle: bf16 bits of Q, K,
    V, dO and its oracle keyword arguments (ring / zigzag: the rank's rows
    against the concatenated keys of all its steps, positions deciding
    visibility), plus the pairs-per-head counter of a row subset."""
    import oracle
    if sh.ring_chunks and sh.zigzag_sp:
        q, do = zigzag_inputs(sh)
        kv = [zigzag_inputs(sh, s) for s in range(sh.ring_chunks)]
        k = np.concatenate([a for a, _ in kv])
        v = np.concatenate([b for _, b in kv])
        pos_k = np.concatenate([zigzag_step_positions(sh, s) for s in range(sh.ring_chunks)])
        cu_q, cu_k = np.array([0, sh.T_q]), np.array([0, len(pos_k)])
    elif sh.ring_chunks:
        q, _, _, do = shard_inputs(sh, chunk=0)
        kv = [shard_inputs(sh, chunk=c)[1:3] for c in range(sh.ring_chunks)]
        k = np.concatenate([a for a, _ in kv])
        v = np.concatenate([b for _, b in kv])
        pos_k = np.concatenate([ring_chunk_positions(sh, c) for c in range(sh.ring_chunks)])
        cu_q, cu_k = np.array([0, sh.T_q]), np.array([0, len(pos_k)])
    else:
        q, k, v, do = shard_inputs(sh)
        pos_k, cu_q, cu_k = sh.pos_k, sh.cu_q, sh.cu_k
    kw = dict(cu_q=cu_q, cu_k=cu_k, pos_q=sh.pos_q, pos_k=pos_k, H_loc=sh.H_loc,
              head_offset=sh.head_offset, num_real_heads=sh.num_real_heads,
              gqa_group=sh.gqa_group, kv_head_offset=sh.kv_head_offset, scale=sh.scale,
              causal=sh.causal)
    seg_q = oracle.segment_ids(cu_q, sh.T_q)
    seg_k = oracle.segment_ids(cu_k, len(pos_k))

    def pairs(rows):
        n = 0
        for b0 in range(0, len(rows), 256):
            n += int(oracle.allowed_mask(rows[b0:b0 + 256], seg_q, seg_k, np.asarray(sh.pos_q),
                                         np.asarray(pos_k), sh.causal).sum())
        return n
    return (q, k, v, do), kw, seg_q, pairs


def cpu_baseline(sh, st, budget_s=15.0):
    """The fp64 oracle as it stands (forward, then its analytic backward) on a
    bounded sample of the shard, on every host core this process may use:
    evenly spaced query rows of the rank (a 32-row probe first, then as many
    rows as fit the time budget), every real head, against all keys the
    shard gives them.  Reported as the oracle's rate in the metric's unit
    (14 D per allowed pair per real head over the sample), with the full
    shard's oracle time extrapolated at that rate."""
    import oracle
    from threadpoolctl import threadpool_limits
    cores = len(os.sched_getaffinity(0))
    bits, kw, seg_q, pairs = monolithic_problem(sh)
    q, k, v, do = (oracle.bf16_bits_to_f64(x) for x in bits)
    valid = np.nonzero(seg_q >= 0)[0]

    def run(m):
        rows = valid[np.unique(np.linspace(0, len(valid) - 1, m).astype(np.int64))]
        cu = np.concatenate([[0], np.cumsum(np.bincount(seg_q[rows], minlength=len(kw["cu_q"]) - 1))])
        sub = dict(kw, cu_q=cu, pos_q=np.asarray(kw["pos_q"])[rows])
        with threadpool_limits(limits=cores):
            t0 = time.perf_counter()
            o, lse = oracle.attn_forward(q[rows], k, v, **sub)
            oracle.attn_backward(q[rows], k, v, do[rows], o=o, lse=lse, **sub)
            dt = time.perf_counter() - t0
        return rows, dt

    m = min(32, len(valid))
    rows, dt = run(m)
    if dt < budget_s / 4 and m < len(valid):
        m = int(min(len(valid), max(m + 1, m * budget_s / max(dt, 1e-3) * 0.8)))
        rows, dt = run(m)
    flops = 14.0 * sh.D * pairs(rows) * sh.n_real_loc
    rate = flops / dt
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": (f"fp64 oracle forward + analytic backward on {len(rows)} evenly spaced of "
                       f"the {len(valid)} query rows, {sh.n_real_loc} real heads, against all "
                       f"{len(kw['pos_k'])} keys of the shard, D={sh.D}: {flops:.3e} FLOP "
                       f"(14 D per allowed pair) in {dt:.1f} s"),
            "cpu_model": cpu_model(), "seconds": round(dt, 2),
            "full_shard_seconds_extrapolated": round(st.flops_metric / rate, 1)}


def measure(sp, torch, name, steps, warmup, per_kernel=True, warmup_s=1.5, kernel_steps=10):
    """Times `steps` steps after a warmup.  Returns the step time, the
    dominant kernel's event timings over the timed steps (the warmup names
    the dominant kernel; only its launches carry events in the timed region,
    since every event pair adds ~11 us to a step), and every kernel's
    timings from `kernel_steps` further, untimed steps."""
    sh = workload(name)
    timers = KernelTimers(sp, torch)
    st = Step(sp, torch, sh, timers)
    # Every timing event is created and recorded once before the timed
    # region (fresh events record slowly), and nothing but one synchronize
    # separates the last warmup step from the first timed one: the GPU
    # clock drops within milliseconds of idling and takes ~20 ms to recover.
    timers.on = per_kernel
    timers.reserve(8 * (steps + warmup))
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    for m in marks:
        m.record()
    # W warmup steps, continued until ~1.5 s of GPU work so clocks settle
    t_w = time.perf_counter()
    n_w = 0
    while n_w < warmup or time.perf_counter() - t_w < warmup_s:
        if n_w == max(1, warmup // 2):
            timers.used = []  # re-use the pool from the start
        st.run()
        n_w += 1
        if n_w % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    warm = timers.summary()
    dom = max(warm, key=lambda k: warm[k]["ms"]) if warm else None
    timers.used = []
    timers.disarm()
    timers.only = {dom} if dom is not None else set()
    t0 = time.perf_counter()
    for i in range(steps):
        marks[i].record()
        st.run()
    marks[steps].record()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ks_dom = timers.summary()
    # every kernel, from further untimed steps
    timers.used = []
    timers.disarm()
    timers.only = None
    for _ in range(kernel_steps if per_kernel else 0):
        st.run()
    torch.cuda.synchronize()
    ks_all = timers.summary()
    timers.on = False
    timers.disarm()
    ms = dt * 1e3 / steps
    per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(steps))
    return sh, st, ms, ks_dom, ks_all, per_step


def measured_traffic(kernel, workload_name):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (profiles/traffic_<kernel>_<workload>.json), or None when any of
    the kernel's source files changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload_name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for src in rec["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != rec["sources_sha256"]:
        return None
    return rec["hbm_bytes_per_launch"]


def copy_calibration(torch, nbytes=1 << 30):
    """One plain device-to-device copy of known size, for scaling the
    FETCH_SIZE / WRITE_SIZE counters of a profiling run."""
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda").random_(0, 255)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    log(f"copy calibration: {nbytes} bytes read, {nbytes} bytes written")
    del a, b


def bandwidth(sp, torch, reps=24):
    """GB/s of the bandwidth kernels at the workloads' shapes: the Ulysses
    pack/unpack and the summing K/V-gradient unpack of the 7B-like and the
    long Ulysses shards, the loss path's token log-probs and their backward
    (4096 tokens x 152064 vocabulary), and the fp32 LSE merge of the ring
    rank's Q chunk.  Buffer sets rotate (>= 4 sets, > 1 GB in
    total) so that the 256 MB last-level cache cannot serve repeats.  GB/s
    comes from batches of back-to-back calls between one HIP event pair (as
    the calls run inside a step, each launch's dispatch overlapping the
    previous call); the single-call event median, which adds one dispatch
    gap per call, is reported beside it."""
    out = []
    HBM_PEAK = PEAK_HBM_GBS

    def run(label, nbytes, sets, call, batch=16):
        n = max(4, -(-(1 << 30) // max(nbytes, 1)) + 1)
        bufs = [sets() for _ in range(n)]
        for i in range(5):
            call(bufs[i % n])
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            a.record()
            call(bufs[i % n])
            b.record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) for a, b in ev)
        med = ts[len(ts) // 2]
        # back to back, as inside a step: `batch` calls over the rotating
        # sets between one event pair (the per-launch dispatch gap overlaps
        # the previous call), median over reps of the per-call average
        evb = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(evb):
            a.record()
            for k in range(batch):
                call(bufs[(i * batch + k) % n])
            b.record()
        torch.cuda.synchronize()
        tb = sorted(a.elapsed_time(b) / batch for a, b in evb)
        medb = tb[len(tb) // 2]
        gbs = nbytes / (medb * 1e-3) / 1e9
        out.append({"bandwidth_kernel": label, "bytes": int(nbytes), "buffer_sets": n,
                    "ms_per_call_back_to_back": round(medb, 4), "calls_per_batch": batch,
                    "ms_median_single_call": round(med, 4), "ms_min_single_call": round(ts[0], 4),
                    "GB_per_s": round(gbs, 1), "frac_of_hbm_peak": round(gbs / HBM_PEAK, 4),
                    "GB_per_s_single_call": round(nbytes / (med * 1e-3) / 1e9, 1)})
        del bufs

    for name in ("ulysses_7b_L32768_q28kv4_sp8_r6_d128", "ulysses_long_L131072_4x32768_q40kv8_sp16_r13_d128"):
        sh = workload(name)
        Tl, hs, spn, Hl, D = sh.T_q // sh.sp, sh.hs, sh.sp, sh.H_loc, sh.D
        hmap = ulysses_q_head_map(hs, spn)
        el = 2 * D
        rd, wr = Tl * hs * el, Tl * spn * Hl * el

        def mk_pack(Tl=Tl, hs=hs, spn=spn, Hl=Hl, D=D):
            src = torch.empty((Tl, hs, D), dtype=torch.bfloat16, device="cuda").normal_()
            return src, torch.empty((spn, Tl, Hl, D), dtype=torch.bfloat16, device="cuda")

        run(f"pack {name} [{Tl},{hs},{D}] -> [{spn},{Tl},{Hl},{D}]", rd + wr, mk_pack,
            lambda b, spn=spn, Hl=Hl, hmap=hmap: sp.sp_ulysses_pack(b[0], spn, Hl, hmap, dst=b[1]))

        def mk_unpack(Tl=Tl, hs=hs, spn=spn, Hl=Hl, D=D):
            src = torch.empty((spn, Tl, Hl, D), dtype=torch.bfloat16, device="cuda").normal_()
            return src, torch.empty((Tl, hs, D), dtype=torch.bfloat16, device="cuda")

        run(f"unpack {name} [{spn},{Tl},{Hl},{D}] -> [{Tl},{hs},{D}]", 2 * rd, mk_unpack,
            lambda b, hs=hs, hmap=hmap: sp.sp_ulysses_unpack(b[0], hmap, hs, dst=b[1]))

        # summing unpack of the dK (or dV) copies the ranks return (GQA)
        kmap = ulysses_kv_head_map(hs, sh.hkv, spn)
        kw_ = len(kmap) // spn
        ua_bytes = (int(np.sum(kmap >= 0)) * Tl + Tl * sh.hkv) * el  # named slots read

        def mk_unpack_add(Tl=Tl, spn=spn, kw_=kw_, D=D, hkv=sh.hkv):
            src = torch.empty((spn, Tl, kw_, D), dtype=torch.bfloat16, device="cuda").normal_()
            return src, torch.empty((Tl, hkv, D), dtype=torch.bfloat16, device="cuda")

        run(f"unpack_add {name} [{spn},{Tl},{kw_},{D}] -> [{Tl},{sh.hkv},{D}]", ua_bytes,
            mk_unpack_add, lambda b, kmap=kmap, hkv=sh.hkv: sp.sp_ulysses_unpack_add(
                b[0], kmap, hkv, dst=b[1]))

    # loss path: token log-probs (reads the logits once) and their backward
    # (reads them again, writes dlogits) at the loss workload's shape
    from workloads import LOSS_WORKLOAD
    Tl_, V_ = LOSS_WORKLOAD["T"], LOSS_WORKLOAD["V"]
    cu_ = np.linspace(0, Tl_, LOSS_WORKLOAD["n_seqs"] + 1).astype(np.int32)

    def mk_loss():
        x = torch.empty((Tl_, V_), dtype=torch.bfloat16, device="cuda").normal_(0.0, 2.0)
        lab = torch.randint(0, V_, (Tl_,), dtype=torch.int32, device="cuda")
        lse = torch.empty(Tl_, dtype=torch.float32, device="cuda")
        lp = torch.empty_like(lse)
        ss = torch.empty(len(cu_) - 1, dtype=torch.float32, device="cuda")
        g = torch.full((len(cu_) - 1,), 1.0 / Tl_, dtype=torch.float32, device="cuda")
        sp.sp_token_logprob(x, lab, cu_, logp=lp, lse=lse, seq_sum=ss)
        return x, lab, lse, lp, ss, g, torch.empty_like(x)

    run(f"token_logprob {LOSS_WORKLOAD['name']} [{Tl_},{V_}] bf16", Tl_ * V_ * 2, mk_loss,
        lambda b: sp.sp_token_logprob(b[0], b[1], cu_, logp=b[3], lse=b[2], seq_sum=b[4]))
    run(f"token_logprob_bwd {LOSS_WORKLOAD['name']} [{Tl_},{V_}] bf16", 2 * Tl_ * V_ * 2, mk_loss,
        lambda b: sp.sp_token_logprob_bwd(b[0], b[1], b[2], cu_, b[5], dlogits=b[6]))

    sh = workload("ring_L131072_8chunks_r4_q28kv4_d128")
    T, H, D = sh.chunk, sh.H_loc, sh.D
    mb = T * H * (D * 4 * 2 + D * 4 + 12)

    def mk_merge():
        o = torch.empty((T, H, D), dtype=torch.float32, device="cuda").normal_()
        lse = torch.empty((H, T), dtype=torch.float32, device="cuda").normal_()
        op = torch.empty((T, H, D), dtype=torch.float32, device="cuda").normal_()
        lp = torch.empty((H, T), dtype=torch.float32, device="cuda").normal_()
        return o, lse, op, lp

    run(f"lse_merge ring_L131072_8chunks_r4_q28kv4_d128 fp32 partial [{T},{H},{D}]", mb, mk_merge,
        lambda b: sp.sp_lse_merge(b[0], b[1], b[2], b[3]))
    return out


def recorded_workloads(path):
    """Workloads that already have a line in the JSONL file `path` (none if
    the file is absent); a line cut short by an interrupted run is ignored."""
    done = set()
    if path and os.path.exists(path):
        with open(path) as f:
            for line in f:
                try:
                    done.add(json.loads(line)["config"]["workload"])
                except (ValueError, KeyError, TypeError):
                    pass
    return done


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=WORKLOADS)
    ap.add_argument("--all", action="store_true", help="one JSON line per workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dummy-overhead", action="store_true",
                    help="skip the dummy-slot overhead measurement (tiny and long Ulysses shards)")
    ap.add_argument("--warmup-seconds", type=float, default=1.5,
                    help="keep warming up until this much time has passed")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 1 GiB device copy first (counter scaling)")
    ap.add_argument("--bandwidth", action="store_true",
                    help="only measure the pack / unpack / LSE-merge kernels (one JSON line each)")
    ap.add_argument("--jsonl", default=None,
                    help="also append each workload's line to this file; workloads already "
                         "recorded there are skipped, so a rerun resumes an interrupted --all")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(one SP rank's shard per GPU); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2505_22296_amd as sp
    sp.load()
    if args.copy_calibration:
        copy_calibration(torch)
    if args.bandwidth:
        for rec in bandwidth(sp, torch):
            print(json.dumps(rec), flush=True)
        return
    names = WORKLOADS if args.all else [args.workload]
    done = recorded_workloads(args.jsonl)
    for name in names:
        if name in done:
            log(f"{name}: already in {args.jsonl}, skipped")
            continue
        kernel_steps = 10
        sh, st, ms, ks_dom, ks, per_step = measure(sp, torch, name, args.steps, args.warmup,
                                                   warmup_s=args.warmup_seconds,
                                                   kernel_steps=kernel_steps)
        value = st.flops_metric / (ms * 1e-3) / 1e12
        # dominant kernel (most time per step), timed over the timed steps
        dom = max(ks_dom.items(), key=lambda kv: kv[1]["ms"]) if ks_dom else None
        roof = None
        kern = {}
        for kid, s in ks.items():
            avg = s["ms"] / s["n"]
            med = sorted(s["all"])[len(s["all"]) // 2]
            kern[KNAMES[kid]] = {"avg_ms": round(avg, 4), "median_ms": round(med, 4),
                                 "launches_per_step": s["n"] / kernel_steps,
                                 "tflops": round(s["flops"] / s["n"] / (avg * 1e-3) / 1e12, 1)
                                 if s["flops"] else None,
                                 "tflops_at_median": round(s["flops"] / s["n"] / (med * 1e-3) / 1e12, 1)
                                 if s["flops"] else None,
                                 "gb_per_s": round(s["bytes"] / s["n"] / (avg * 1e-3) / 1e9, 1)
                                 if s["bytes"] else None}
        if dom and dom[1]["flops"] > 0:
            kid, s = dom
            avg_s = s["ms"] / s["n"] * 1e-3
            ach = s["flops"] / s["n"] / avg_s / 1e12
            roof = {"bound": "mfma", "kernel": KNAMES[kid], "achieved": round(ach, 1),
                    "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                    "traffic": measured_traffic(KNAMES[kid], name),
                    "avg_launch_ms": round(s["ms"] / s["n"], 4),
                    "flops_per_launch": s["flops"] / s["n"]}
        elif dom:  # a copy kernel dominates (launch-bound shapes): HBM roofline
            kid, s = dom
            avg_s = s["ms"] / s["n"] * 1e-3
            ach = s["bytes"] / s["n"] / avg_s / 1e9
            roof = {"bound": "hbm", "kernel": KNAMES[kid], "achieved": round(ach, 1),
                    "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                    "traffic": measured_traffic(KNAMES[kid], name),
                    "avg_launch_ms": round(s["ms"] / s["n"], 4),
                    "bytes_per_launch": s["bytes"] / s["n"]}
        out = {
            "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded N(0,1) bf16; shapes of the paper's workloads)",
            "config": {"workload": name, "T_q": sh.T_q, "T_k": sh.T_k, "D": sh.D,
                       "H_loc": sh.H_loc, "H_real": sh.n_real_loc, "Hkv_loc": sh.Hkv_loc,
                       "segments": int(len(sh.cu_q) - 1), "ring_chunks": sh.ring_chunks,
                       "sp": sh.sp, "rank": sh.rank, "pairs_per_head": int(sum(st.pairs)),
                       "flops_per_step": st.flops_metric,
                       **({"ulysses_rank": sh.hp_rank} if sh.zigzag_sp and sh.sp > 1 else {})},
            "pct_of_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
            "strict_12D_tflops": round(st.flops_strict / (ms * 1e-3) / 1e12, 2),
            # per-step GPU times (events between steps); `value` uses the mean
            "ms_per_step_median": round(per_step[len(per_step) // 2], 4),
            "ms_per_step_min": round(per_step[0], 4),
            "tflops_at_median_step": round(st.flops_metric / (per_step[len(per_step) // 2] * 1e-3) / 1e12, 2),
            # every kernel, from further untimed steps with all kernels timed
            "kernels": kern,
            "kernels_steps": kernel_steps,
            "roofline": roof,
        }
        if not args.no_dummy_overhead and name == names[0]:
            log("timing the dummy-slot overhead ...")
            out["dummy_overhead"] = dummy_overhead(sp, torch)
        if not args.no_cpu_baseline and name == names[0]:
            log("timing the CPU oracle baseline ...")
            cb = cpu_baseline(sh, st)
            cb["gpu_speedup_at_this_rate"] = round(value / cb["value"], 1) if cb["value"] else None
            out["cpu_baseline"] = cb
        print(json.dumps(out), flush=True)
        if args.jsonl:
            with open(args.jsonl, "a") as f:
                f.write(json.dumps(out) + "\n")


def dummy_overhead(sp, torch, names=DUMMY_WORKLOADS, target_s=0.6):
    """Dummy-slot cost: attention fwd+bwd of a shard with dummy slots against
    the same real heads described without them (same inputs), each call
    pair timed with HIP events, the two variants alternating; medians."""
    out = {}
    for name in names:
        sh = workload(name)
        if sh.n_real_loc >= sh.H_loc:
            continue
        runs = {}
        for tag, s in (("with_dummies", sh), ("without", sh.without_dummies())):
            desc = lib_desc(sp, s)
            q, k, v, do = (to_dev(torch, x) for x in shard_inputs(s))
            o = torch.empty_like(q)
            lse = torch.empty((s.H_loc, s.T_q), dtype=torch.float32, device="cuda")
            dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
            wf = torch.empty(sp.sp_attn_workspace_size(desc, sp.SP_OP_FWD), dtype=torch.uint8,
                             device="cuda")
            wb = torch.empty(sp.sp_attn_workspace_size(desc, sp.SP_OP_BWD), dtype=torch.uint8,
                             device="cuda")

            def run(desc=desc, q=q, k=k, v=v, do=do, o=o, lse=lse, dq=dq, dk=dk, dv=dv, wf=wf,
                    wb=wb):
                sp.sp_attn_fwd(desc, q, k, v, o, lse, workspace=wf)
                sp.sp_attn_bwd(desc, q, k, v, o, lse, do, dq=dq, dk=dk, dv=dv, workspace=wb)
            runs[tag] = run
        for _ in range(5):
            for r in runs.values():
                r()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        runs["with_dummies"]()
        torch.cuda.synchronize()
        one = time.perf_counter() - t0
        reps = int(max(20, min(2000, target_s / max(one, 1e-5) / 2)))
        ev = {tag: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for _ in range(reps)] for tag in runs}
        for i in range(reps):
            order = ("with_dummies", "without") if i % 2 == 0 else ("without", "with_dummies")
            for tag in order:
                a, b = ev[tag][i]
                a.record()
                runs[tag]()
                b.record()
        torch.cuda.synchronize()
        med = {}
        for tag in runs:
            ts = sorted(a.elapsed_time(b) for a, b in ev[tag])
            med[tag] = ts[len(ts) // 2]
        out[name] = {"with_dummies_ms": round(med["with_dummies"], 4),
                     "without_ms": round(med["without"], 4), "reps": reps,
                     "dummy_slots": sh.H_loc - sh.n_real_loc, "slots": sh.H_loc,
                     "overhead_pct": round(100.0 * (med["with_dummies"] / med["without"] - 1.0), 2)}
    return out


if __name__ == "__main__":
    main()
