"""Plain fp64 masked attention, forward and analytic backward (CPU oracle).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this.

What is computed is the plain definition of scaled dot-product attention
under a block-diagonal causal mask.  Sequence parallelism (Ulysses head
sharding, Section 4; Ring-Attention chunking, Section 2.1) is an exact
re-partitioning of this computation: the paper's correctness experiment
(Section 6.1) finds forward log-probs identical with and without SP.  So the
oracle is the monolithic definition, evaluated for one rank's shard:

  * segments (neat packing, Section 3.2): query row i of segment s attends to
    keys of segment s only; rows past the last segment attend to nothing;
  * causal: key j is visible to row i iff pos_k[j] <= pos_q[i] (positions are
    the explicit position IDs of Section 5.2; the diagonal is included);
  * softmax scale is passed in (1/sqrt(D) by convention);
  * dummy heads (Section 4.1, padded at the end of the head axis) produce
    O = +0, LSE = -inf and zero gradients by definition;
  * GQA: local head i reads KV head (head_offset + i) // gqa_group minus
    kv_head_offset.

Softmax is evaluated exactly over the whole row (not online).  Rows are
processed in blocks only to bound memory; no other reordering.
"""
from __future__ import annotations

import numpy as np

NEG_INF = -np.inf


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bfloat16 bit patterns (uint16) to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def segment_ids(cu: np.ndarray, T: int) -> np.ndarray:
    """seg[i] = s for cu[s] <= i < cu[s+1]; -1 for rows past cu[-1]."""
    seg = np.full(T, -1, dtype=np.int64)
    for s in range(len(cu) - 1):
        seg[int(cu[s]):int(cu[s + 1])] = s
    return seg


def allowed_mask(rows, seg_q, seg_k, pos_q, pos_k, causal):
    """Boolean [len(rows), T_k]: which keys each listed query row may see."""
    sq = seg_q[rows][:, None]
    m = (sq >= 0) & (sq == seg_k[None, :])
    if causal:
        m &= pos_k[None, :].astype(np.int64) <= pos_q[rows][:, None].astype(np.int64)
    return m


def local_heads(H_loc, head_offset, num_real_heads, gqa_group, kv_head_offset):
    """[(local head, local kv head or None for a dummy head)]."""
    out = []
    for i in range(H_loc):
        g = head_offset + i
        out.append((i, g // gqa_group - kv_head_offset) if g < num_real_heads else (i, None))
    return out


def _row_stats(q_rows, k, mask, scale):
    """For a block of query rows against all keys of one KV head: the exact
    softmax P (zeros where masked / for rows without keys) and LSE."""
    S = scale * (q_rows @ k.T)
    S = np.where(mask, S, NEG_INF)
    m = S.max(axis=1) if S.shape[1] else np.full(S.shape[0], NEG_INF)
    has = np.isfinite(m)
    m_safe = np.where(has, m, 0.0)
    E = np.where(mask, np.exp(S - m_safe[:, None]), 0.0)
    den = E.sum(axis=1)
    P = np.where(has[:, None], E / np.where(has, den, 1.0)[:, None], 0.0)
    lse = np.where(has, m_safe + np.log(np.where(has, den, 1.0)), NEG_INF)
    return P, lse


def attn_forward(q, k, v, *, cu_q, cu_k, pos_q, pos_k, H_loc, head_offset,
                 num_real_heads, gqa_group, kv_head_offset, scale, causal=True,
                 rows=None, row_block=256):
    """O [n_rows, H_loc, D] (float64) and LSE [H_loc, n_rows] (natural log).

    q: [T_q, H_loc, D]; k, v: [T_k, Hkv_loc, D], all float64.  `rows`
    restricts the computation to the listed query rows (sampled parity)."""
    T_q = q.shape[0]
    T_k = k.shape[0]
    rows = np.arange(T_q) if rows is None else np.asarray(rows, dtype=np.int64)
    seg_q, seg_k = segment_ids(cu_q, T_q), segment_ids(cu_k, T_k)
    pos_q = np.asarray(pos_q, dtype=np.int64)
    pos_k = np.asarray(pos_k, dtype=np.int64)
    D = q.shape[2]
    O = np.zeros((len(rows), H_loc, D))
    LSE = np.full((H_loc, len(rows)), NEG_INF)
    for h, kv in local_heads(H_loc, head_offset, num_real_heads, gqa_group, kv_head_offset):
        if kv is None:
            continue  # dummy head: O = +0, LSE = -inf
        for b0 in range(0, len(rows), row_block):
            r = rows[b0:b0 + row_block]
            mask = allowed_mask(r, seg_q, seg_k, pos_q, pos_k, causal)
            P, lse = _row_stats(q[r, h, :], k[:, kv, :], mask, scale)
            O[b0:b0 + len(r), h, :] = P @ v[:, kv, :]
            LSE[h, b0:b0 + len(r)] = lse
    return O, LSE


def attn_backward(q, k, v, do, *, cu_q, cu_k, pos_q, pos_k, H_loc, head_offset,
                  num_real_heads, gqa_group, kv_head_offset, scale, causal=True,
                  o=None, lse=None, row_block=256):
    """Analytic gradients of sum(dO * O) w.r.t. Q, K, V (float64).

    With P the softmax of row i and D_i = sum_j P_ij dP_ij = dO_i . O_i:
      dP = dO V^T,  dS = P * (dP - D),  dQ = scale dS K,
      dK = scale dS^T Q,  dV = P^T dO   (GQA: summed over the group).
    `o`/`lse` may be supplied from a previous oracle forward (they are only
    used to form D and P); otherwise they are recomputed here."""
    T_q, T_k = q.shape[0], k.shape[0]
    seg_q, seg_k = segment_ids(cu_q, T_q), segment_ids(cu_k, T_k)
    pos_q = np.asarray(pos_q, dtype=np.int64)
    pos_k = np.asarray(pos_k, dtype=np.int64)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for h, kv in local_heads(H_loc, head_offset, num_real_heads, gqa_group, kv_head_offset):
        if kv is None:
            continue
        for b0 in range(0, T_q, row_block):
            r = np.arange(b0, min(T_q, b0 + row_block))
            mask = allowed_mask(r, seg_q, seg_k, pos_q, pos_k, causal)
            P, lse_r = _row_stats(q[r, h, :], k[:, kv, :], mask, scale)
            if lse is not None:
                # Use the given LSE: P = exp(S - LSE) on allowed pairs.
                S = scale * (q[r, h, :] @ k[:, kv, :].T)
                L = lse[h, r]
                fin = np.isfinite(L)
                P = np.where(mask & fin[:, None],
                             np.exp(np.where(mask, S, 0.0) - np.where(fin, L, 0.0)[:, None]), 0.0)
            o_r = (P @ v[:, kv, :]) if o is None else o[r, h, :]
            dO = do[r, h, :]
            Drow = (dO * o_r).sum(axis=1)
            dP = dO @ v[:, kv, :].T
            dS = P * (dP - Drow[:, None])
            dq[r, h, :] = scale * (dS @ k[:, kv, :])
            dk[:, kv, :] += scale * (dS.T @ q[r, h, :])
            dv[:, kv, :] += P.T @ dO
    return dq, dk, dv


def attn_dq_rows(q, k, v, do, rows, **kw):
    """dQ for the listed query rows only (sampled parity at large sizes)."""
    O, L = attn_forward(q, k, v, rows=rows, **kw)
    T_q, T_k = q.shape[0], k.shape[0]
    seg_q, seg_k = segment_ids(kw["cu_q"], T_q), segment_ids(kw["cu_k"], T_k)
    pq, pk = np.asarray(kw["pos_q"], np.int64), np.asarray(kw["pos_k"], np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), q.shape[1], q.shape[2]))
    for h, kv in local_heads(kw["H_loc"], kw["head_offset"], kw["num_real_heads"],
                             kw["gqa_group"], kw["kv_head_offset"]):
        if kv is None:
            continue
        mask = allowed_mask(rows, seg_q, seg_k, pq, pk, kw.get("causal", True))
        P, _ = _row_stats(q[rows, h, :], k[:, kv, :], mask, kw["scale"])
        dO = do[rows, h, :]
        Drow = (dO * O[:, h, :]).sum(axis=1)
        dS = P * (dO @ v[:, kv, :].T - Drow[:, None])
        out[:, h, :] = kw["scale"] * (dS @ k[:, kv, :])
    return out, O, L


def attn_dkdv_keys(q, k, v, do, keys, **kw):
    """dK, dV for the listed key rows only: every query row that sees any of
    those keys is evaluated exactly (its full softmax row)."""
    T_q, T_k = q.shape[0], k.shape[0]
    seg_q, seg_k = segment_ids(kw["cu_q"], T_q), segment_ids(kw["cu_k"], T_k)
    pq, pk = np.asarray(kw["pos_q"], np.int64), np.asarray(kw["pos_k"], np.int64)
    causal = kw.get("causal", True)
    keys = np.asarray(keys, dtype=np.int64)
    dk = np.zeros((len(keys), k.shape[1], k.shape[2]))
    dv = np.zeros_like(dk)
    # rows that see at least one listed key
    need = np.zeros(T_q, dtype=bool)
    for b0 in range(0, T_q, 4096):
        r = np.arange(b0, min(T_q, b0 + 4096))
        m = allowed_mask(r, seg_q, seg_k[keys], pq, pk[keys], causal)
        need[r] = m.any(axis=1)
    rows = np.nonzero(need)[0]
    for h, kv in local_heads(kw["H_loc"], kw["head_offset"], kw["num_real_heads"],
                             kw["gqa_group"], kw["kv_head_offset"]):
        if kv is None:
            continue
        for b0 in range(0, len(rows), 256):
            r = rows[b0:b0 + 256]
            mask = allowed_mask(r, seg_q, seg_k, pq, pk, causal)
            P, _ = _row_stats(q[r, h, :], k[:, kv, :], mask, kw["scale"])
            dO = do[r, h, :]
            o_r = P @ v[:, kv, :]
            Drow = (dO * o_r).sum(axis=1)
            Pk = P[:, keys]
            dS = Pk * (dO @ v[keys, kv, :].T - Drow[:, None])
            dk[:, kv, :] += kw["scale"] * (dS.T @ q[r, h, :])
            dv[:, kv, :] += Pk.T @ dO
    return dk, dv
