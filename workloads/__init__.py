"""Seeded synthetic workloads for one sequence-parallel rank's attention shard.

This module is shared by the CPU oracle's tests, the GPU parity tests and the
benchmark.  It holds NO attention arithmetic: only shapes, head bookkeeping,
segment layouts, position IDs, pair counting for FLOP accounting, and seeded
bf16 input bits.  Both sides consume the very same uint16 bit patterns.

The shapes follow the paper's workloads: Qwen2.5-style GQA head counts under
Dummy-Head Ulysses (Section 4, Listing 1: heads padded at the end of the head
axis up to a multiple of the SP size), neat-packed varlen batches (Section 3.2,
block-diagonal causal mask), and one Ring-Attention rank (Section 2.1 / Table 1
ring row).  The paper's datasets are not available; N(0,1) inputs of the same
shapes stand in for them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

__all__ = [
    "Shard", "WORKLOADS", "workload", "padded_heads", "bf16_bits_from_f32",
    "randn_bf16_bits", "varlen_lengths", "shard_inputs", "allowed_pairs",
    "ulysses_q_head_map", "ulysses_kv_head_map", "usp_shard", "loss_inputs", "LOSS_WORKLOAD",
]


def padded_heads(hs: int, sp: int) -> int:
    """Head count after dummy-head padding (Section 4.1): add sp - hs % sp
    heads when hs is not a multiple of sp, else none."""
    rem = hs % sp
    return hs if rem == 0 else hs + (sp - rem)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even) and return the
    16-bit patterns as uint16.  Inputs must be finite."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def randn_bf16_bits(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    """i.i.d. N(0, scale^2) drawn in float32 from PCG64(seed), rounded to bf16."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x = x * np.float32(scale)
    return bf16_bits_from_f32(x)


def varlen_lengths(total: int, seed: int = 0, median: int = 4096, sigma: float = 1.0,
                   lo: int = 512, hi: int = 16384) -> List[int]:
    """Neat-packing segment lengths: lognormal(ln median, sigma) rounded and
    clipped to [lo, hi], drawn in order until `total` tokens are filled; the
    draw that would overflow is replaced by the remainder (so the last segment
    may be shorter than lo)."""
    rng = np.random.default_rng(seed)
    out: List[int] = []
    left = total
    while left > 0:
        n = int(np.clip(np.rint(rng.lognormal(math.log(median), sigma)), lo, hi))
        n = min(n, left)
        out.append(n)
        left -= n
    return out


def ulysses_q_head_map(hs: int, sp: int) -> np.ndarray:
    """Pack map for Q (and MHA K/V): slot j*H_loc + h carries global head
    j*H_loc + h when it is a real head, else -1 (a zero dummy head)."""
    hs_new = padded_heads(hs, sp)
    m = np.arange(hs_new, dtype=np.int32)
    m[m >= hs] = -1
    return m


def ulysses_kv_head_map(hs: int, hkv: int, sp: int) -> np.ndarray:
    """GQA K/V pack map: rank j receives the contiguous KV heads its real Q
    heads read, in slots 0.., padded with -1 up to the widest rank."""
    hs_new = padded_heads(hs, sp)
    hloc = hs_new // sp
    g = hs // hkv
    ranges = []
    for j in range(sp):
        real = [h for h in range(j * hloc, (j + 1) * hloc) if h < hs]
        ranges.append((real[0] // g, real[-1] // g + 1) if real else (0, 0))
    width = max(b - a for a, b in ranges)
    m = np.full(sp * width, -1, dtype=np.int32)
    for j, (a, b) in enumerate(ranges):
        m[j * width: j * width + (b - a)] = np.arange(a, b, dtype=np.int32)
    return m


@dataclasses.dataclass
class Shard:
    """One SP rank's attention problem (the shapes the rank's kernels see).

    Layout of every activation is [T, H, D] with D innermost (bf16); LSE is
    [H, T] float32.  `cu_q`/`cu_k` delimit segments; segment s of Q attends
    to segment s of K only.  Positions are per-token IDs (a +1 ramp inside
    each segment)."""
    name: str
    T_q: int
    T_k: int
    D: int
    H_loc: int
    head_offset: int
    num_real_heads: int
    num_padded_heads: int
    gqa_group: int
    Hkv_loc: int
    kv_head_offset: int
    cu_q: np.ndarray
    cu_k: np.ndarray
    pos_q: np.ndarray
    pos_k: np.ndarray
    causal: bool = True
    seed_base: int = 0
    # Ulysses bookkeeping (pack/unpack shapes); sp=1 means no pack step.
    sp: int = 1
    rank: int = 0
    hs: int = 0
    hkv: int = 0
    # Ring bookkeeping: number of KV chunks this rank loops over (0 = not ring).
    ring_chunks: int = 0
    chunk: int = 0
    # Zigzag ring (Section 3.2): the sequence is cut into 2*zigzag_sp chunks,
    # rank r holds chunks r and 2*zigzag_sp-1-r, and ring step s brings the
    # two chunks of rank (r - s) mod zigzag_sp.  Q and each step's KV are
    # pieces of one sequence (single_sequence).
    zigzag_sp: int = 0
    single_sequence: bool = False
    # USP (Ulysses inside zigzag-ring groups): the Ulysses rank inside the
    # ring group (sp = Ulysses size, rank = ring rank, zigzag_sp = ring size).
    hp_rank: int = 0

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    @property
    def n_real_loc(self) -> int:
        return max(0, min(self.H_loc, self.num_real_heads - self.head_offset))

    def kv_of(self, h: int) -> int:
        return (self.head_offset + h) // self.gqa_group - self.kv_head_offset

    def without_dummies(self) -> "Shard":
        """The same real heads reading the same KV heads, described as a shard
        with no dummy slots (for timing the cost of the dummy slots)."""
        nr = self.n_real_loc
        kvs = [self.kv_of(h) for h in range(nr)]
        if self.gqa_group == 1:
            g, off = 1, -kvs[0]
        elif len(set(kvs)) == 1:
            g, off = nr, -kvs[0]
        else:
            raise ValueError("real heads span several KV heads under GQA")
        return dataclasses.replace(self, name=self.name + "_nodummy", H_loc=nr, head_offset=0,
                                   num_real_heads=nr, num_padded_heads=nr, gqa_group=g,
                                   kv_head_offset=off if off >= 0 else 0, sp=1,
                                   seed_base=self.seed_base)


def _ramp_positions(cu: np.ndarray, T: int, base: int = 0) -> np.ndarray:
    pos = np.zeros(T, dtype=np.int32)
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        pos[a:b] = base + np.arange(b - a, dtype=np.int32)
    return pos


def _ulysses(name, L, D, hs, hkv, sp, rank, seg_lens, seed_base) -> Shard:
    hs_new = padded_heads(hs, sp)
    hloc = hs_new // sp
    off = rank * hloc
    g = hs // hkv
    real = [h for h in range(off, off + hloc) if h < hs]
    if hkv == hs:  # MHA: K/V padded and split exactly like Q
        kvloc, kvoff = hloc, off
    elif real:
        kvoff = real[0] // g
        kvloc = real[-1] // g + 1 - kvoff
    else:
        kvoff, kvloc = 0, 1
    cu = np.concatenate([[0], np.cumsum(seg_lens)]).astype(np.int32)
    pos = _ramp_positions(cu, L)
    return Shard(name=name, T_q=L, T_k=L, D=D, H_loc=hloc, head_offset=off,
                 num_real_heads=hs, num_padded_heads=hs_new, gqa_group=g,
                 Hkv_loc=kvloc, kv_head_offset=kvoff, cu_q=cu, cu_k=cu.copy(),
                 pos_q=pos, pos_k=pos.copy(), causal=True, seed_base=seed_base,
                 sp=sp, rank=rank, hs=hs, hkv=hkv)


def _packed(name, T, D, hq, hkv, seg_lens, seed_base) -> Shard:
    cu = np.concatenate([[0], np.cumsum(seg_lens)]).astype(np.int32)
    pos = _ramp_positions(cu, T)
    return Shard(name=name, T_q=T, T_k=T, D=D, H_loc=hq, head_offset=0,
                 num_real_heads=hq, num_padded_heads=hq, gqa_group=hq // hkv,
                 Hkv_loc=hkv, kv_head_offset=0, cu_q=cu, cu_k=cu.copy(),
                 pos_q=pos, pos_k=pos.copy(), causal=True, seed_base=seed_base,
                 hs=hq, hkv=hkv)


def _ring(name, L, n_chunks, rank, D, hq, hkv, seed_base) -> Shard:
    C = L // n_chunks
    cu = np.array([0, C], dtype=np.int32)
    # Q chunk positions; each KV chunk c gets positions c*C.. when stepped.
    return Shard(name=name, T_q=C, T_k=C, D=D, H_loc=hq, head_offset=0,
                 num_real_heads=hq, num_padded_heads=hq, gqa_group=hq // hkv,
                 Hkv_loc=hkv, kv_head_offset=0, cu_q=cu, cu_k=cu.copy(),
                 pos_q=_ramp_positions(cu, C, rank * C), pos_k=_ramp_positions(cu, C, 0),
                 causal=True, seed_base=seed_base, hs=hq, hkv=hkv,
                 ring_chunks=rank + 1, chunk=C, rank=rank, sp=1)


def _zigzag(name, L, sp, rank, D, hq, hkv, seed_base) -> Shard:
    C = L // (2 * sp)
    cu = np.array([0, C, 2 * C], dtype=np.int32)
    a, b = zigzag_chunks(rank, sp)
    pos_q = np.concatenate([a * C + np.arange(C), b * C + np.arange(C)]).astype(np.int32)
    return Shard(name=name, T_q=2 * C, T_k=2 * C, D=D, H_loc=hq, head_offset=0,
                 num_real_heads=hq, num_padded_heads=hq, gqa_group=hq // hkv,
                 Hkv_loc=hkv, kv_head_offset=0, cu_q=cu, cu_k=cu.copy(), pos_q=pos_q,
                 pos_k=pos_q.copy(), causal=True, seed_base=seed_base, hs=hq, hkv=hkv,
                 ring_chunks=sp, chunk=C, rank=rank, sp=1, zigzag_sp=sp, single_sequence=True)


def usp_shard(name, L, hp, cp, r_cp, j_hp, D, hs, hkv, seed_base) -> Shard:
    """USP rank (ring rank r_cp of cp, Ulysses rank j_hp of hp): after the
    Ulysses all-to-all inside its ring group it holds the group's zigzag
    share (chunks r_cp and 2*cp-1-r_cp of 2*cp) over the heads Ulysses rank
    j_hp receives, and runs the zigzag ring over the shares of the other
    ring groups' rank j_hp."""
    C = L // (2 * cp)
    hs_new = padded_heads(hs, hp)
    hloc = hs_new // hp
    off = j_hp * hloc
    g = hs // hkv
    real = [h for h in range(off, off + hloc) if h < hs]
    if hkv == hs:
        kvloc, kvoff = hloc, off
    elif real:
        kvoff = real[0] // g
        kvloc = real[-1] // g + 1 - kvoff
    else:
        kvoff, kvloc = 0, 1
    cu = np.array([0, C, 2 * C], dtype=np.int32)
    a, b = zigzag_chunks(r_cp, cp)
    pos_q = np.concatenate([a * C + np.arange(C), b * C + np.arange(C)]).astype(np.int32)
    return Shard(name=name, T_q=2 * C, T_k=2 * C, D=D, H_loc=hloc, head_offset=off,
                 num_real_heads=hs, num_padded_heads=hs_new, gqa_group=g, Hkv_loc=kvloc,
                 kv_head_offset=kvoff, cu_q=cu, cu_k=cu.copy(), pos_q=pos_q, pos_k=pos_q.copy(),
                 causal=True, seed_base=seed_base, hs=hs, hkv=hkv, ring_chunks=cp, chunk=C,
                 rank=r_cp, sp=hp, zigzag_sp=cp, single_sequence=True, hp_rank=j_hp)


def zigzag_chunks(rank: int, sp: int):
    """The two sequence chunks (of 2*sp) a zigzag rank holds, in position order."""
    return rank, 2 * sp - 1 - rank


def zigzag_step_chunks(sh: Shard, s: int):
    """Sequence chunks of the KV that zigzag ring step s brings to the rank."""
    return zigzag_chunks((sh.rank - s) % sh.zigzag_sp, sh.zigzag_sp)


def zigzag_step_positions(sh: Shard, s: int) -> np.ndarray:
    C = sh.chunk
    a, b = zigzag_step_chunks(sh, s)
    return np.concatenate([a * C + np.arange(C), b * C + np.arange(C)]).astype(np.int32)


def zigzag_inputs(sh: Shard, s: int = None):
    """bf16 bits of a zigzag shard: (q, do) for the rank's two chunks when s
    is None, else (k, v) of ring step s.  Every sequence chunk has its own
    seeds, so a chunk's data is the same wherever it appears."""
    C, sb = sh.chunk, sh.seed_base

    def piece(c, off, H):
        return randn_bf16_bits((C, H, sh.D), sb + off + 16 * (c + 1))
    if s is None:
        chunks = zigzag_chunks(sh.rank, sh.zigzag_sp)
        q = np.concatenate([piece(c, 0, sh.H_loc) for c in chunks])
        do = np.concatenate([piece(c, 3, sh.H_loc) for c in chunks])
        q[:, sh.n_real_loc:] = 0   # dummy slots arrive zero from the pack
        do[:, sh.n_real_loc:] = 0
        return q, do
    chunks = zigzag_step_chunks(sh, s)
    k = np.concatenate([piece(c, 1, sh.Hkv_loc) for c in chunks])
    v = np.concatenate([piece(c, 2, sh.Hkv_loc) for c in chunks])
    return k, v


def ring_chunk_positions(sh: Shard, c: int) -> np.ndarray:
    """Positions of KV chunk c under the contiguous ring split."""
    return _ramp_positions(sh.cu_k, sh.T_k, c * sh.chunk)


def workload(name: str) -> Shard:
    """Build a named workload.  Names state the shape they describe."""
    if name == "ulysses_tiny_L1024_mha7of8_sp2_r1_d64":
        return _ulysses(name, 1024, 64, 7, 7, 2, 1, [1024], 0)
    if name == "ulysses_7b_L32768_q28kv4_sp8_r6_d128":
        return _ulysses(name, 32768, 128, 28, 4, 8, 6, [32768], 100)
    if name == "packed_varlen_T65536_q4kv1_d128":
        return _packed(name, 65536, 128, 4, 1, varlen_lengths(65536, seed=0), 200)
    if name == "ring_L131072_8chunks_r4_q28kv4_d128":
        return _ring(name, 131072, 8, 4, 128, 28, 4, 300)
    if name == "ulysses_long_L131072_4x32768_q40kv8_sp16_r13_d128":
        return _ulysses(name, 131072, 128, 40, 8, 16, 13, [32768] * 4, 400)
    if name == "zigzag_ring_L131072_sp8_r4_q28kv4_d128":
        return _zigzag(name, 131072, 8, 4, 128, 28, 4, 500)
    if name == "usp_L131072_hp4_cp2_r1_j2_q28kv4_d128":
        return usp_shard(name, 131072, 4, 2, 1, 2, 128, 28, 4, 600)
    raise KeyError(name)


WORKLOADS = [
    "ulysses_tiny_L1024_mha7of8_sp2_r1_d64",
    "ulysses_7b_L32768_q28kv4_sp8_r6_d128",
    "packed_varlen_T65536_q4kv1_d128",
    "ring_L131072_8chunks_r4_q28kv4_d128",
    "ulysses_long_L131072_4x32768_q40kv8_sp16_r13_d128",
    "zigzag_ring_L131072_sp8_r4_q28kv4_d128",
    "usp_L131072_hp4_cp2_r1_j2_q28kv4_d128",
]


def shard_inputs(sh: Shard, peaky: float = 1.0, chunk: Optional[int] = None):
    """bf16 bits for Q [T_q,H_loc,D], K/V [T_k,Hkv_loc,D], dO [T_q,H_loc,D].

    Dummy Q-head slots are zero (they arrive zero-padded from the pack), and
    for MHA shards the KV slots of dummy heads are zero as well.  For ring
    workloads `chunk` selects the KV chunk (seeds differ per chunk)."""
    sb = sh.seed_base
    kvs = 0 if chunk is None else 16 * (chunk + 1)
    q = randn_bf16_bits((sh.T_q, sh.H_loc, sh.D), sb + 0, peaky)
    k = randn_bf16_bits((sh.T_k, sh.Hkv_loc, sh.D), sb + 1 + kvs)
    v = randn_bf16_bits((sh.T_k, sh.Hkv_loc, sh.D), sb + 2 + kvs)
    do = randn_bf16_bits((sh.T_q, sh.H_loc, sh.D), sb + 3)
    nr = sh.n_real_loc
    q[:, nr:, :] = 0
    do[:, nr:, :] = 0
    if sh.gqa_group == 1:
        gk = sh.kv_head_offset + np.arange(sh.Hkv_loc)
        dummy_kv = gk >= sh.num_real_heads
        k[:, dummy_kv, :] = 0
        v[:, dummy_kv, :] = 0
    return q, k, v, do


def allowed_pairs(cu_q, cu_k, pos_q, pos_k, causal: bool = True,
                  single_sequence: bool = False) -> int:
    """Number of (query, key) pairs the mask allows, per head: same segment
    index (any valid row / key for pieces of one sequence) and, when causal,
    pos_k <= pos_q.  Positions must be +1 ramps inside each segment (and
    increase strictly over all pieces of one sequence)."""
    if single_sequence:
        nq, nk = int(cu_q[-1]), int(cu_k[-1])
        if not causal:
            return nq * nk
        return int(np.searchsorted(np.asarray(pos_k[:nk], np.int64),
                                   np.asarray(pos_q[:nq], np.int64), side="right").sum())
    total = 0
    for s in range(len(cu_q) - 1):
        qa, qb = int(cu_q[s]), int(cu_q[s + 1])
        ka, kb = int(cu_k[s]), int(cu_k[s + 1])
        nq, nk = qb - qa, kb - ka
        if nq <= 0 or nk <= 0:
            continue
        if not causal:
            total += nq * nk
            continue
        # row i (0-based in segment) sees keys j with kbase + j <= qbase + i
        d = int(pos_q[qa]) - int(pos_k[ka])
        for_rows = np.clip(np.arange(nq, dtype=np.int64) + d + 1, 0, nk)
        total += int(for_rows.sum())
    return total


# Loss path of one rank: the 7B-like shard's token slice (32768 tokens over
# SP 8 = 4096 tokens) against a 152064-entry vocabulary (Qwen2.5's padded
# vocabulary, from the public model config; the paper names the models, not
# their vocabulary), two sequences (a DPO chosen / rejected pair).
LOSS_WORKLOAD = dict(name="loss_T4096_V152064_dpo_pair", T=4096, V=152064, n_seqs=2, seed=700)


def loss_inputs(T: int, V: int, n_seqs: int, seed: int, prompt_frac: float = 0.25,
                logit_scale: float = 2.0, rows_per_block: int = 256):
    """bf16 logit bits [T, V] (N(0, logit_scale^2), rows drawn in blocks of
    rows_per_block with seed + block index), labels [T] int32 uniform in
    [0, V) with the first prompt_frac of each sequence set to -100 (prompt
    tokens are not scored), and cu_seqlens splitting T evenly into n_seqs."""
    bits = np.empty((T, V), dtype=np.uint16)
    for b0 in range(0, T, rows_per_block):
        b1 = min(T, b0 + rows_per_block)
        bits[b0:b1] = randn_bf16_bits((b1 - b0, V), seed + b0 // rows_per_block, logit_scale)
    rng = np.random.default_rng(seed + 100000)
    labels = rng.integers(0, V, T).astype(np.int32)
    cu = np.linspace(0, T, n_seqs + 1).astype(np.int32)
    for s in range(n_seqs):
        a, b = int(cu[s]), int(cu[s + 1])
        labels[a:a + int((b - a) * prompt_frac)] = -100
    return bits, labels, cu
