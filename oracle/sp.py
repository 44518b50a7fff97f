"""Sequence-parallel data movement and merges (CPU oracle, float64 / uint16).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this.

  * pad_heads / unpad_heads: Dummy-Head Ulysses (Section 4.1, Listing 1):
    when hs % sp != 0, append sp - hs % sp zero heads at the END of the head
    axis; unpad keeps the first hs heads.
  * ulysses_pack / ulysses_unpack: the send/receive layouts around the
    Ulysses all-to-all (Section 4: [bs, L/sp, hs, d] <-> [bs, L, hs/sp, d]),
    written as index maps over a head map (-1 = zero dummy head).
  * all_to_all: the collective itself, simulated as an index permutation.
  * lse_merge / ring_forward: Ring-Attention (Section 2.1, Table 1): the
    rank's Q chunk is run against each KV chunk and the partial results are
    combined through log-sum-exp.
  * ulysses_simulate: every rank of a DHU layer, end to end.
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
    hkv = k_full.shape[1]
    assert L % sp == 0
    Tl = L // sp
    qp = pad_heads(q_full[None], sp)[0]
    hs_new = qp.shape[1]
    hloc = hs_new // sp
    qmap = np.array([h if h < hs else -1 for h in range(hs_new)])
    if hkv == hs:
        kp, vp = pad_heads(k_full[None], sp)[0], pad_heads(v_full[None], sp)[0]
        kmap, kvw = qmap, hloc
        kv_off = [j * hloc for j in range(sp)]
    else:
        kp, vp = k_full, v_full
        rng = []
        for j in range(sp):
            real = [h for h in range(j * hloc, (j + 1) * hloc) if h < hs]
            rng.append((real[0] // gqa_group, real[-1] // gqa_group + 1) if real else (0, 0))
        kvw = max(1, max(b - a for a, b in rng))
        kmap = np.full(sp * kvw, -1)
        for j, (a, b) in enumerate(rng):
            kmap[j * kvw: j * kvw + b - a] = np.arange(a, b)
        kv_off = [a for a, _ in rng]
    # send side: each rank packs its token slice
    sends_q = [ulysses_pack(qp[r * Tl:(r + 1) * Tl], sp, hloc, np.arange(hs_new)) for r in range(sp)]
    sends_k = [ulysses_pack(kp[r * Tl:(r + 1) * Tl], sp, kvw, kmap if hkv != hs else np.arange(hs_new)) for r in range(sp)]
    sends_v = [ulysses_pack(vp[r * Tl:(r + 1) * Tl], sp, kvw, kmap if hkv != hs else np.arange(hs_new)) for r in range(sp)]
    rq, rk, rv = all_to_all(sends_q), all_to_all(sends_k), all_to_all(sends_v)
    outs, lses = [], []
    for j in range(sp):
        # sequential split: concatenating source chunks in rank order is [L, H, D]
        qj = np.concatenate(rq[j], axis=0)
        kj = np.concatenate(rk[j], axis=0)
        vj = np.concatenate(rv[j], axis=0)
        oj, lj = attn_forward(qj, kj, vj, cu_q=cu, cu_k=cu, pos_q=pos, pos_k=pos,
                              H_loc=hloc, head_offset=j * hloc, num_real_heads=hs,
                              gqa_group=gqa_group, kv_head_offset=kv_off[j], scale=scale)
        outs.append(np.stack(np.split(oj, sp, axis=0)))  # [sp, Tl, hloc, D]
        lses.append(lj)
    back = all_to_all([[outs[j][r] for r in range(sp)] for j in range(sp)])
    o = np.concatenate([
        unpad_heads(ulysses_unpack(np.stack(back[r]), np.arange(hs_new), hs_new)[None], hs)[0]
        for r in range(sp)], axis=0)
    return o, lses
