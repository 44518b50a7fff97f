"""Sequence-parallel data movement and merges (CPU oracle, float64 / uint16).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this.

  * pad_heads / unpad_heads: Dummy-Head Ulysses (Section 4.1, Listing 1):
    when hs % sp != 0, append sp - hs % sp zero heads at the END of the head
    axis; unpad keeps the first hs heads.
  * ulysses_pack / ulysses_unpack: the send/receive layouts around the
    Ulysses all-to-all (Section 4: [bs, L/sp, hs, d] <-> [bs, L, hs/sp, d]),
    written as index maps over a head map (-1 = zero dummy head).
  * ulysses_unpack_add: the backward of the GQA K/V pack.  The pack
    replicates a KV head to every rank whose real query heads read it, so on
    the way back the gradients the ranks return for one KV head are summed
    (the adjoint of the replication).  A bfloat16 variant fixes the order and
    precision the library uses: float32 sum in ascending slot order, one
    rounding to bfloat16.
  * all_to_all: the collective itself, simulated as an index permutation.
  * lse_merge / ring_forward: Ring-Attention (Section 2.1, Table 1): the
    rank's Q chunk is run against each KV chunk and the partial results are
    combined through log-sum-exp.
  * ulysses_simulate / ulysses_simulate_backward: every rank of a DHU
    layer, end to end, forward and backward.
  * usp_simulate: USP (the paper's 2-D comparison method, Table 1): Ulysses
    inside groups of sp_hp ranks, zigzag Ring-Attention across sp_cp groups.
"""
from __future__ import annotations

import numpy as np

from .attention import attn_forward, attn_backward

NEG_INF = -np.inf


def pad_heads(x: np.ndarray, sp: int) -> np.ndarray:
    """x: [bs, L, hs, d] -> [bs, L, hs_new, d], zero heads appended."""
    hs = x.shape[2]
    rem = hs % sp
    if rem == 0:
        return x
    pad = np.zeros(x.shape[:2] + (sp - rem,) + x.shape[3:], dtype=x.dtype)
    return np.concatenate([x, pad], axis=2)


def unpad_heads(x: np.ndarray, hs: int) -> np.ndarray:
    return x[:, :, :hs, :]


def ulysses_pack(src: np.ndarray, sp: int, H_dst_loc: int, head_map) -> np.ndarray:
    """dst[j, t, h, :] = src[t, head_map[j*H_dst_loc + h], :], or 0 where the
    map entry is -1.  src: [T_loc, H_src, D] -> dst: [sp, T_loc, H_dst_loc, D].
    Works on raw bit patterns (any dtype); zero is the all-zero pattern."""
    T_loc, _, D = src.shape
    dst = np.zeros((sp, T_loc, H_dst_loc, D), dtype=src.dtype)
    for j in range(sp):
        for h in range(H_dst_loc):
            g = int(head_map[j * H_dst_loc + h])
            if g >= 0:
                dst[j, :, h, :] = src[:, g, :]
    return dst


def ulysses_unpack(src: np.ndarray, head_map, H_dst: int) -> np.ndarray:
    """Inverse of the pack: dst[t, head_map[j*H + h], :] = src[j, t, h, :] for
    entries != -1 (dummy slots are dropped).  Every destination head must be
    named exactly once."""
    sp, T_loc, H_src_loc, D = src.shape
    dst = np.zeros((T_loc, H_dst, D), dtype=src.dtype)
    seen = np.zeros(H_dst, dtype=np.int64)
    for j in range(sp):
        for h in range(H_src_loc):
            g = int(head_map[j * H_src_loc + h])
            if g >= 0:
                dst[:, g, :] = src[j, :, h, :]
                seen[g] += 1
    assert np.all(seen == 1), "unpack map must name every destination head once"
    return dst


def ulysses_unpack_add(src: np.ndarray, head_map, H_dst: int) -> np.ndarray:
    """Adjoint of ulysses_pack: dst[t, g, :] = sum of src[j, t, h, :] over the
    slots j*H + h whose map entry is g, in ascending slot order; -1 slots are
    dropped; a head named by no slot is zero.  src: [sp, T_loc, H, D] (float
    values) -> dst: [T_loc, H_dst, D]."""
    sp, T_loc, H_src_loc, D = src.shape
    dst = np.zeros((T_loc, H_dst, D), dtype=np.float64)
    for j in range(sp):
        for h in range(H_src_loc):
            g = int(head_map[j * H_src_loc + h])
            if g >= 0:
                dst[:, g, :] += src[j, :, h, :]
    return dst


def f32_to_bf16_bits(x) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest, ties to even
    (finite inputs): add 0x7fff plus the lowest kept bit, drop 16 bits."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def ulysses_unpack_add_bf16(src_bits: np.ndarray, head_map, H_dst: int) -> np.ndarray:
    """ulysses_unpack_add on bfloat16 bit patterns as the library defines it:
    each input decoded to float32 (exact), the sum formed in float32 one term
    at a time in ascending slot order (rank j, then slot h), rounded once to
    bfloat16 (nearest-even).  Returns uint16 bits [T_loc, H_dst, D]."""
    sp, T_loc, H_src_loc, D = src_bits.shape
    vals = (np.asarray(src_bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    acc = np.zeros((T_loc, H_dst, D), dtype=np.float32)
    for j in range(sp):
        for h in range(H_src_loc):
            g = int(head_map[j * H_src_loc + h])
            if g >= 0:
                acc[:, g, :] = acc[:, g, :] + vals[j, :, h, :]
    return f32_to_bf16_bits(acc)


def all_to_all(send):
    """send[r][j] is what rank r sends to rank j; returns recv[j][r]."""
    sp = len(send)
    return [[send[r][j] for r in range(sp)] for j in range(sp)]


def lse_merge(o_acc, lse_acc, o_part, lse_part):
    """Combine two partial attention results over disjoint key sets.
    o: [T, H, D], lse: [H, T] (natural log).  L = logaddexp(L_a, L_b);
    O = e^(L_a - L) O_a + e^(L_b - L) O_b; (-inf, -inf) gives (0, -inf)."""
    la, lb = lse_acc, lse_part
    L = np.logaddexp(la, lb)
    fin = np.isfinite(L)
    Ls = np.where(fin, L, 0.0)
    wa = np.where(fin & np.isfinite(la), np.exp(np.where(np.isfinite(la), la, 0.0) - Ls), 0.0)
    wb = np.where(fin & np.isfinite(lb), np.exp(np.where(np.isfinite(lb), lb, 0.0) - Ls), 0.0)
    o = wa.T[:, :, None] * o_acc + wb.T[:, :, None] * o_part
    return o, np.where(fin, L, NEG_INF)


def ring_forward(q, kv_chunks, *, q_pos, kv_pos, H_loc, head_offset, num_real_heads,
                 gqa_group, kv_head_offset, scale, causal=True):
    """One ring rank: fold (O_c, LSE_c) of Q against each KV chunk c, in
    order, with lse_merge.  kv_chunks: [(k_c, v_c)], kv_pos: [pos_c]."""
    Tq = q.shape[0]
    D = q.shape[2]
    o = np.zeros((Tq, H_loc, D))
    lse = np.full((H_loc, Tq), NEG_INF)
    for (kc, vc), pk in zip(kv_chunks, kv_pos):
        oc, lc = attn_forward(q, kc, vc, cu_q=np.array([0, Tq]), cu_k=np.array([0, kc.shape[0]]),
                              pos_q=q_pos, pos_k=pk, H_loc=H_loc, head_offset=head_offset,
                              num_real_heads=num_real_heads, gqa_group=gqa_group,
                              kv_head_offset=kv_head_offset, scale=scale, causal=causal)
        o, lse = lse_merge(o, lse, oc, lc)
    return o, lse


def ring_backward(q, kv_chunks, do, o, lse, *, q_pos, kv_pos, H_loc, head_offset,
                  num_real_heads, gqa_group, kv_head_offset, scale, causal=True):
    """Gradients of one ring rank: each chunk's backward uses the FINAL
    (merged) O and LSE; dQ sums over chunks, each chunk has its own dK, dV."""
    Tq = q.shape[0]
    dq = np.zeros_like(q)
    dks, dvs = [], []
    for (kc, vc), pk in zip(kv_chunks, kv_pos):
        a, b, c = attn_backward(q, kc, vc, do, cu_q=np.array([0, Tq]),
                                cu_k=np.array([0, kc.shape[0]]), pos_q=q_pos, pos_k=pk,
                                H_loc=H_loc, head_offset=head_offset,
                                num_real_heads=num_real_heads, gqa_group=gqa_group,
                                kv_head_offset=kv_head_offset, scale=scale, causal=causal,
                                o=o, lse=lse)
        dq += a
        dks.append(b)
        dvs.append(c)
    return dq, dks, dvs


def _dhu_layout(hs, hs_new, hkv, sp, gqa_group):
    """Head maps of one DHU layer, given the padded head count hs_new that
    Listing 1's pad produced: Q map, K/V map, K/V slots per rank and each
    rank's first KV head.  MHA pads K/V like Q; under GQA only Q is padded
    and rank j receives the contiguous KV heads its real Q heads read."""
    assert hs_new % sp == 0 and hs_new >= hs
    hloc = hs_new // sp
    qmap = np.array([h if h < hs else -1 for h in range(hs_new)])
    if hkv == hs:
        return qmap, qmap, hloc, [j * hloc for j in range(sp)], hloc, hs_new
    rng = []
    for j in range(sp):
        real = [h for h in range(j * hloc, (j + 1) * hloc) if h < hs]
        rng.append((real[0] // gqa_group, real[-1] // gqa_group + 1) if real else (0, 0))
    kvw = max(1, max(b - a for a, b in rng))
    kmap = np.full(sp * kvw, -1)
    for j, (a, b) in enumerate(rng):
        kmap[j * kvw: j * kvw + b - a] = np.arange(a, b)
    return qmap, kmap, kvw, [a for a, _ in rng], hloc, hs_new


def _dhu_scatter(q_full, k_full, v_full, sp, gqa_group, extra=()):
    """Pad, split sequentially, pack and exchange: per rank the full-sequence
    tensors over its heads ([L, H_loc, D] each), plus the layout."""
    L, hs, D = q_full.shape
    hkv = k_full.shape[1]
    assert L % sp == 0
    Tl = L // sp
    qp = pad_heads(q_full[None], sp)[0]
    qmap, kmap, kvw, kv_off, hloc, hs_new = _dhu_layout(hs, qp.shape[1], hkv, sp, gqa_group)
    mha = hkv == hs
    kp, vp = ((pad_heads(k_full[None], sp)[0], pad_heads(v_full[None], sp)[0]) if mha
              else (k_full, v_full))
    kv_pack_map = np.arange(hs_new) if mha else kmap

    def exchange(x, width, m):
        sends = [ulysses_pack(x[r * Tl:(r + 1) * Tl], sp, width, m) for r in range(sp)]
        recv = all_to_all(sends)
        # sequential split: source chunks in rank order are the whole sequence
        return [np.concatenate(recv[j], axis=0) for j in range(sp)]

    qs = exchange(qp, hloc, np.arange(hs_new))
    ks = exchange(kp, kvw, kv_pack_map)
    vs = exchange(vp, kvw, kv_pack_map)
    xs = [exchange(pad_heads(x[None], sp)[0], hloc, np.arange(hs_new)) for x in extra]
    return qs, ks, vs, xs, (qmap, kmap, kvw, kv_off, hloc, hs_new, Tl, mha)


def _dhu_gather(per_rank, sp, Tl, hloc, hs_new, hs):
    """Reverse exchange of [L, H_loc, D] per-rank results, unpack, unpad."""
    back = all_to_all([list(np.split(per_rank[j], sp, axis=0)) for j in range(sp)])
    return np.concatenate([
        unpad_heads(ulysses_unpack(np.stack(back[r]), np.arange(hs_new), hs_new)[None], hs)[0]
        for r in range(sp)], axis=0)


def ulysses_simulate(q_full, k_full, v_full, sp, *, scale, cu, pos, gqa_group=1):
    """Every rank of one Dummy-Head Ulysses attention layer (batch 1).

    q_full: [L, hs, D]; k_full, v_full: [L, hkv, D] (hkv = hs / gqa_group).
    Per Listing 1, Q (and for MHA also K, V) is padded with zero heads at the
    end of the head axis; the sequence is split sequentially over sp ranks;
    the all-to-all gives rank j the full sequence over heads j*H_loc..; each
    rank attends over its heads; the reverse all-to-all and unpad return
    [L, hs, D].  For GQA only Q is padded and rank j receives the KV heads
    its real Q heads read.  Returns (O [L, hs, D], per-rank LSE)."""
    L, hs, D = q_full.shape
    qs, ks, vs, _, lay = _dhu_scatter(q_full, k_full, v_full, sp, gqa_group)
    qmap, kmap, kvw, kv_off, hloc, hs_new, Tl, mha = lay
    outs, lses = [], []
    for j in range(sp):
        oj, lj = attn_forward(qs[j], ks[j], vs[j], cu_q=cu, cu_k=cu, pos_q=pos, pos_k=pos,
                              H_loc=hloc, head_offset=j * hloc, num_real_heads=hs,
                              gqa_group=gqa_group, kv_head_offset=kv_off[j], scale=scale)
        outs.append(oj)
        lses.append(lj)
    return _dhu_gather(outs, sp, Tl, hloc, hs_new, hs), lses


def ulysses_simulate_backward(q_full, k_full, v_full, do_full, sp, *, scale, cu, pos,
                              gqa_group=1):
    """Gradients of one DHU layer over every rank (batch 1), for the loss
    sum(dO * O).  dO reaches each rank through the same pad + all-to-all as Q
    (its dummy heads are zero); each rank differentiates its own heads; dQ
    goes back through the reverse all-to-all and unpad (the backward of the
    pad drops the dummy heads).  K/V: for MHA the same as dQ; under GQA the
    reverse all-to-all returns each rank's dK/dV of the KV heads it received
    and ulysses_unpack_add sums the copies of a KV head that several ranks
    held.  Returns dQ [L, hs, D], dK and dV [L, hkv, D]."""
    L, hs, D = q_full.shape
    hkv = k_full.shape[1]
    qs, ks, vs, (dos,), lay = _dhu_scatter(q_full, k_full, v_full, sp, gqa_group, (do_full,))
    qmap, kmap, kvw, kv_off, hloc, hs_new, Tl, mha = lay
    dqs, dks, dvs = [], [], []
    for j in range(sp):
        a, b, c = attn_backward(qs[j], ks[j], vs[j], dos[j], cu_q=cu, cu_k=cu, pos_q=pos,
                                pos_k=pos, H_loc=hloc, head_offset=j * hloc,
                                num_real_heads=hs, gqa_group=gqa_group,
                                kv_head_offset=kv_off[j], scale=scale)
        dqs.append(a)
        dks.append(b)
        dvs.append(c)
    dq = _dhu_gather(dqs, sp, Tl, hloc, hs_new, hs)
    if mha:
        return dq, _dhu_gather(dks, sp, Tl, hloc, hs_new, hs), _dhu_gather(dvs, sp, Tl, hloc,
                                                                            hs_new, hs)

    def kv_back(per_rank):
        back = all_to_all([list(np.split(per_rank[j], sp, axis=0)) for j in range(sp)])
        return np.concatenate([ulysses_unpack_add(np.stack(back[r]), kmap, hkv)
                               for r in range(sp)], axis=0)

    return dq, kv_back(dks), kv_back(dvs)


def usp_simulate(q_full, k_full, v_full, do_full, sp_hp, sp_cp, *, scale, gqa_group=1):
    """Every rank of a USP attention layer (batch 1, one causal sequence).

    Ranks form sp_cp ring groups of sp_hp Ulysses ranks.  The sequence is cut
    into 2*sp_cp chunks; ring rank r holds chunks r and 2*sp_cp-1-r (zigzag),
    split sequentially over its sp_hp Ulysses ranks.  Inside a ring group the
    DHU all-to-all gives Ulysses rank j the group's whole share over heads
    j*H_loc..; across groups, rank (r, j) runs the zigzag ring over the
    shares of ranks (r - s mod sp_cp, j), s = 0..sp_cp-1, merging partials
    by log-sum-exp; the backward uses the merged O / LSE, and each step's dK,
    dV are summed at the rank that owns those keys before the reverse
    all-to-all (summing unpack under GQA).  Returns O, dQ [L, hs, D], dK, dV
    [L, hkv, D] and the per-rank results {(r, j): dict(q_pos, o, lse, dq,
    kv_pos, dk, dv)} (dk / dv per ring step)."""
    L, hs, D = q_full.shape
    hkv = k_full.shape[1]
    n_ch = 2 * sp_cp
    assert L % n_ch == 0
    C = L // n_ch
    share = [np.concatenate([r * C + np.arange(C), (n_ch - 1 - r) * C + np.arange(C)])
             for r in range(sp_cp)]
    groups = [_dhu_scatter(q_full[share[r]], k_full[share[r]], v_full[share[r]], sp_hp, gqa_group,
                           (do_full[share[r]],)) for r in range(sp_cp)]
    qmap, kmap, kvw, kv_off, hloc, hs_new, Tl, mha = groups[0][4]
    per_rank = {}
    o_g = [[None] * sp_hp for _ in range(sp_cp)]
    dq_g = [[None] * sp_hp for _ in range(sp_cp)]
    dk_g = [[np.zeros_like(groups[r][1][j]) for j in range(sp_hp)] for r in range(sp_cp)]
    dv_g = [[np.zeros_like(groups[r][2][j]) for j in range(sp_hp)] for r in range(sp_cp)]
    for r in range(sp_cp):
        for j in range(sp_hp):
            steps = [(r - s) % sp_cp for s in range(sp_cp)]
            chunks = [(groups[r2][1][j], groups[r2][2][j]) for r2 in steps]
            kv_pos = [share[r2] for r2 in steps]
            kw = dict(q_pos=share[r], kv_pos=kv_pos, H_loc=hloc, head_offset=j * hloc,
                      num_real_heads=hs, gqa_group=gqa_group, kv_head_offset=kv_off[j],
                      scale=scale)
            q, do = groups[r][0][j], groups[r][3][0][j]
            o, lse = ring_forward(q, chunks, **kw)
            dq, dks, dvs = ring_backward(q, chunks, do, o, lse, **kw)
            for r2, a, b in zip(steps, dks, dvs):
                dk_g[r2][j] += a
                dv_g[r2][j] += b
            o_g[r][j], dq_g[r][j] = o, dq
            per_rank[(r, j)] = dict(q_pos=share[r], o=o, lse=lse, dq=dq, kv_pos=kv_pos,
                                    dk=dks, dv=dvs)

    def kv_back(per_j):
        if mha:
            return _dhu_gather(per_j, sp_hp, Tl, hloc, hs_new, hs)
        back = all_to_all([list(np.split(per_j[j], sp_hp, axis=0)) for j in range(sp_hp)])
        return np.concatenate([ulysses_unpack_add(np.stack(back[i]), kmap, hkv)
                               for i in range(sp_hp)], axis=0)

    O, dQ = np.zeros_like(q_full), np.zeros_like(q_full)
    dK, dV = np.zeros_like(k_full), np.zeros_like(v_full)
    for r in range(sp_cp):
        O[share[r]] = _dhu_gather(o_g[r], sp_hp, Tl, hloc, hs_new, hs)
        dQ[share[r]] = _dhu_gather(dq_g[r], sp_hp, Tl, hloc, hs_new, hs)
        dK[share[r]] = kv_back(dk_g[r])
        dV[share[r]] = kv_back(dv_g[r])
    return O, dQ, dK, dV, per_rank
