"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each pin takes the oracle's attention module `A` (and, where needed, its SP
module `S`) as an argument, so the mutation test can run the same pins
against deliberately broken copies of the oracle source.

Sources of truth used here:
  * closed forms (single visible key; all-zero queries give a uniform
    softmax over the visible keys);
  * a library routine: torch float64 scaled_dot_product_attention on the CPU
    with an explicit boolean mask, and torch autograd through it;
  * central finite differences of sum(dO * O);
  * the gradient identities sum_j dK_j = 0 and sum_j dV_j = sum_i dO_i that
    follow from softmax rows summing to one;
  * exact-decomposition invariants the paper relies on: the ring fold equals
    monolithic attention (Section 2.1), a packed batch equals its sequences
    run one by one (Section 3.2), and Dummy-Head Ulysses over all ranks
    equals attention without SP (Sections 4.1 and 6.1).
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

from workloads import padded_heads, ulysses_kv_head_map, ulysses_q_head_map


def _kw(T, H, Hkv, cu=None, pos_q=None, pos_k=None, head_offset=0, num_real=None,
        gqa=None, kv_off=0, scale=0.37, causal=True, Tk=None):
    Tk = T if Tk is None else Tk
    cu_q = np.array([0, T]) if cu is None else np.asarray(cu)
    cu_k = np.array([0, Tk]) if cu is None else np.asarray(cu)
    if pos_q is None:
        pos_q = np.zeros(T, np.int64)
        for s in range(len(cu_q) - 1):
            pos_q[cu_q[s]:cu_q[s + 1]] = np.arange(cu_q[s + 1] - cu_q[s])
    if pos_k is None:
        pos_k = np.zeros(Tk, np.int64)
        for s in range(len(cu_k) - 1):
            pos_k[cu_k[s]:cu_k[s + 1]] = np.arange(cu_k[s + 1] - cu_k[s])
    num_real = H if num_real is None else num_real
    gqa = (num_real // Hkv if num_real >= Hkv else 1) if gqa is None else gqa
    return dict(cu_q=cu_q, cu_k=cu_k, pos_q=pos_q, pos_k=pos_k, H_loc=H,
                head_offset=head_offset, num_real_heads=num_real, gqa_group=gqa,
                kv_head_offset=kv_off, scale=scale, causal=causal)


def _rand(rng, *shape):
    return rng.standard_normal(shape)


# ---------------------------------------------------------------- closed forms
def pin_single_visible_key(A):
    """Row 0 of a causal segment sees only key 0: O_0 = v_0, LSE_0 = s q0.k0."""
    rng = np.random.default_rng(1)
    T, H, D = 9, 2, 5
    q, k, v = _rand(rng, T, H, D), _rand(rng, T, 1, D), _rand(rng, T, 1, D)
    kw = _kw(T, H, 1)
    O, L = A.attn_forward(q, k, v, **kw)
    for h in range(H):
        assert np.allclose(O[0, h], v[0, 0], rtol=0, atol=1e-14)
        assert np.isclose(L[h, 0], kw["scale"] * q[0, h] @ k[0, 0], rtol=0, atol=1e-14)


def pin_zero_query_uniform(A):
    """Q = 0 makes every visible score 0: O_i = mean of visible v_j and
    LSE_i = log(number visible).  Varlen, offsets and padding rows included."""
    rng = np.random.default_rng(2)
    T, Tk, H, D = 23, 23, 3, 4
    cu = np.array([0, 7, 7, 16, 20])
    pos = np.zeros(T, np.int64)
    pos[0:7] = 5 + np.arange(7)       # segment 0 starts at position 5
    pos[7:16] = np.arange(9)
    pos[16:20] = 2 + np.arange(4)
    posk = pos.copy()
    posk[0:7] = 3 + np.arange(7)      # keys start two positions earlier
    q = np.zeros((T, H, D))
    k, v = _rand(rng, Tk, 1, D), _rand(rng, Tk, 1, D)
    kw = _kw(T, H, 1, cu=cu, pos_q=pos, pos_k=posk)
    O, L = A.attn_forward(q, k, v, **kw)
    seg = np.full(T, -1)
    for s in range(len(cu) - 1):
        seg[cu[s]:cu[s + 1]] = s
    for i in range(T):
        vis = [j for j in range(Tk) if seg[i] >= 0 and seg[j] == seg[i] and posk[j] <= pos[i]]
        for h in range(H):
            if vis:
                assert np.allclose(O[i, h], v[vis, 0].mean(axis=0), atol=1e-13)
                assert np.isclose(L[h, i], np.log(len(vis)), atol=1e-13)
            else:
                assert np.all(O[i, h] == 0) and L[h, i] == -np.inf


# ------------------------------------------------------------ library routine
def _torch_ref(q, k, v, do, kw):
    """torch float64 SDPA with an explicit boolean mask, plus autograd."""
    T, H, D = q.shape
    Tk = k.shape[0]
    seg_q = np.full(T, -1)
    seg_k = np.full(Tk, -1)
    for s in range(len(kw["cu_q"]) - 1):
        seg_q[kw["cu_q"][s]:kw["cu_q"][s + 1]] = s
        seg_k[kw["cu_k"][s]:kw["cu_k"][s + 1]] = s
    mask = (seg_q[:, None] >= 0) & (seg_q[:, None] == seg_k[None, :])
    if kw["causal"]:
        mask &= np.asarray(kw["pos_k"])[None, :] <= np.asarray(kw["pos_q"])[:, None]
    has = mask.any(axis=1)
    O = np.zeros_like(q)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for h in range(H):
        g = kw["head_offset"] + h
        if g >= kw["num_real_heads"]:
            continue
        kv = g // kw["gqa_group"] - kw["kv_head_offset"]
        tq = torch.tensor(q[has, h][None, None], requires_grad=True)
        tk = torch.tensor(k[:, kv][None, None], requires_grad=True)
        tv = torch.tensor(v[:, kv][None, None], requires_grad=True)
        m = torch.tensor(mask[has][None, None])
        o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m,
                                                             scale=kw["scale"])
        (o * torch.tensor(do[has, h][None, None])).sum().backward()
        O[has, h] = o[0, 0].detach().numpy()
        dq[has, h] = tq.grad[0, 0].numpy()
        dk[:, kv] += tk.grad[0, 0].numpy()
        dv[:, kv] += tv.grad[0, 0].numpy()
    return O, dq, dk, dv


def pin_torch_sdpa(A):
    """Forward and backward equal torch fp64 SDPA + autograd (GQA, dummy
    heads, varlen with padding rows, position offsets, non-causal)."""
    rng = np.random.default_rng(3)
    cases = [
        dict(T=37, H=4, Hkv=1, D=8, cu=[0, 37], num_real=4, gqa=4, kv_off=0, ho=0),
        dict(T=50, H=4, Hkv=2, D=6, cu=[0, 13, 13, 40, 47], num_real=7, gqa=2, kv_off=2, ho=4),
        dict(T=41, H=3, Hkv=3, D=5, cu=[0, 20, 41], num_real=5, gqa=1, kv_off=3, ho=3),
    ]
    for c in cases:
        T, H, Hkv, D = c["T"], c["H"], c["Hkv"], c["D"]
        q, k, v, do = _rand(rng, T, H, D), _rand(rng, T, Hkv, D), _rand(rng, T, Hkv, D), _rand(rng, T, H, D)
        for causal in (True, False):
            kw = _kw(T, H, Hkv, cu=c["cu"], head_offset=c["ho"], num_real=c["num_real"],
                     gqa=c["gqa"], kv_off=c["kv_off"], causal=causal)
            O, _ = A.attn_forward(q, k, v, **kw)
            dq, dk, dv = A.attn_backward(q, k, v, do, **kw)
            rO, rdq, rdk, rdv = _torch_ref(q, k, v, do, kw)
            for a, b in ((O, rO), (dq, rdq), (dk, rdk), (dv, rdv)):
                assert np.allclose(a, b, rtol=0, atol=1e-12), np.abs(a - b).max()
    # ring-style offsets: Q chunk at positions 40.., K chunk at 20..
    T = 24
    q, k, v, do = _rand(rng, T, 2, 4), _rand(rng, T, 1, 4), _rand(rng, T, 1, 4), _rand(rng, T, 2, 4)
    kw = _kw(T, 2, 1, pos_q=40 + np.arange(T), pos_k=30 + np.arange(T))
    O, _ = A.attn_forward(q, k, v, **kw)
    rO, rdq, rdk, rdv = _torch_ref(q, k, v, do, kw)
    dq, dk, dv = A.attn_backward(q, k, v, do, **kw)
    for a, b in ((O, rO), (dq, rdq), (dk, rdk), (dv, rdv)):
        assert np.allclose(a, b, rtol=0, atol=1e-12)


def pin_sampled_checkers(A):
    """The sampled checkers used at full size -- dQ of listed rows
    (attn_dq_rows, with its O and LSE) and dK / dV of listed keys
    (attn_dkdv_keys) -- equal torch fp64 SDPA + autograd restricted to the
    same rows / keys, on arbitrary row and key subsets: varlen with padding
    rows, GQA, dummy slots, ring-style position offsets, non-causal, and
    pieces of one sequence (positions jumping between pieces)."""
    rng = np.random.default_rng(13)
    cases = [
        (dict(T=37, H=4, Hkv=1, D=8, cu=[0, 37], num_real=4, gqa=4, kv_off=0, ho=0), None, None),
        (dict(T=50, H=4, Hkv=2, D=6, cu=[0, 13, 13, 40, 47], num_real=7, gqa=2, kv_off=2, ho=4),
         None, None),
        (dict(T=41, H=3, Hkv=3, D=5, cu=[0, 20, 41], num_real=5, gqa=1, kv_off=3, ho=3), None, None),
        # ring offsets: rows at positions 40.., keys at 30..
        (dict(T=24, H=2, Hkv=1, D=4, cu=[0, 24], num_real=2, gqa=2, kv_off=0, ho=0),
         40 + np.arange(24), 30 + np.arange(24)),
        # pieces of one sequence: positions strictly increasing with jumps
        (dict(T=30, H=3, Hkv=1, D=5, cu=[0, 30], num_real=3, gqa=3, kv_off=0, ho=0),
         np.r_[np.arange(10), 50 + np.arange(20)], np.r_[5 + np.arange(12), 40 + np.arange(18)]),
    ]
    for c, pq, pk in cases:
        T, H, Hkv, D = c["T"], c["H"], c["Hkv"], c["D"]
        q, k, v, do = _rand(rng, T, H, D), _rand(rng, T, Hkv, D), _rand(rng, T, Hkv, D), _rand(rng, T, H, D)
        for causal in (True, False):
            kw = _kw(T, H, Hkv, cu=c["cu"], pos_q=pq, pos_k=pk, head_offset=c["ho"],
                     num_real=c["num_real"], gqa=c["gqa"], kv_off=c["kv_off"], causal=causal)
            rO, rdq, rdk, rdv = _torch_ref(q, k, v, do, kw)
            for trial in range(3):
                rows = np.sort(rng.choice(T, size=int(rng.integers(1, T)), replace=False))
                keys = np.sort(rng.choice(T, size=int(rng.integers(1, T)), replace=False))
                dq, O, _ = A.attn_dq_rows(q, k, v, do, rows, **kw)
                assert np.allclose(dq, rdq[rows], rtol=0, atol=1e-12), np.abs(dq - rdq[rows]).max()
                assert np.allclose(O, rO[rows], rtol=0, atol=1e-12)
                dk, dv = A.attn_dkdv_keys(q, k, v, do, keys, **kw)
                assert np.allclose(dk, rdk[keys], rtol=0, atol=1e-12), np.abs(dk - rdk[keys]).max()
                assert np.allclose(dv, rdv[keys], rtol=0, atol=1e-12), np.abs(dv - rdv[keys]).max()


def pin_bf16_decode(A):
    """bf16_bits_to_f64 equals torch's bfloat16 -> float64 conversion on all
    65,536 bit patterns (NaNs compared as NaN)."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = A.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


# ------------------------------------------------------- finite differences
def pin_finite_differences(A):
    """Central differences of sum(dO * O) match the analytic backward."""
    rng = np.random.default_rng(4)
    T, H, Hkv, D = 11, 2, 1, 4
    cu = [0, 6, 11]
    q, k, v, do = _rand(rng, T, H, D), _rand(rng, T, Hkv, D), _rand(rng, T, Hkv, D), _rand(rng, T, H, D)
    kw = _kw(T, H, Hkv, cu=cu, gqa=2)
    dq, dk, dv = A.attn_backward(q, k, v, do, **kw)

    def loss(qq, kk, vv):
        return float((A.attn_forward(qq, kk, vv, **kw)[0] * do).sum())

    h = 1e-6
    for arr, grad, which in ((q, dq, 0), (k, dk, 1), (v, dv, 2)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args = [q.copy(), k.copy(), v.copy()]
            args[which][idx] += h
            fp = loss(*args)
            args[which][idx] -= 2 * h
            fm = loss(*args)
            num[idx] = (fp - fm) / (2 * h)
        err = np.abs(num - grad).max() / max(1e-12, np.abs(grad).max())
        assert err < 1e-6, (which, err)


# ------------------------------------------------------ gradient identities
def pin_gradient_sums(A):
    """Per KV head: sum_j dK_j = 0 and sum_j dV_j = sum over rows with keys
    of dO_i, for each segment separately."""
    rng = np.random.default_rng(5)
    T, H, Hkv, D = 45, 4, 2, 6
    cu = [0, 17, 30, 45]
    q, k, v, do = _rand(rng, T, H, D), _rand(rng, T, Hkv, D), _rand(rng, T, Hkv, D), _rand(rng, T, H, D)
    kw = _kw(T, H, Hkv, cu=cu, gqa=2)
    _, dk, dv = A.attn_backward(q, k, v, do, **kw)
    for s in range(3):
        a, b = cu[s], cu[s + 1]
        for kv in range(Hkv):
            assert np.allclose(dk[a:b, kv].sum(axis=0), 0, atol=1e-12)
            want = do[a:b, 2 * kv:2 * kv + 2].sum(axis=(0, 1))
            assert np.allclose(dv[a:b, kv].sum(axis=0), want, atol=1e-12)


# -------------------------------------------------------- SP decompositions
def pin_packed_equals_separate(A):
    """A packed batch equals its sequences run one by one (fwd and bwd)."""
    rng = np.random.default_rng(6)
    lens = [9, 1, 14, 6]
    T = sum(lens)
    cu = np.concatenate([[0], np.cumsum(lens)])
    H, Hkv, D = 2, 1, 4
    q, k, v, do = _rand(rng, T, H, D), _rand(rng, T, Hkv, D), _rand(rng, T, Hkv, D), _rand(rng, T, H, D)
    kw = _kw(T, H, Hkv, cu=cu)
    O, L = A.attn_forward(q, k, v, **kw)
    g = A.attn_backward(q, k, v, do, **kw)
    for s, n in enumerate(lens):
        a, b = cu[s], cu[s + 1]
        kws = _kw(n, H, Hkv)
        Os, Ls = A.attn_forward(q[a:b], k[a:b], v[a:b], **kws)
        gs = A.attn_backward(q[a:b], k[a:b], v[a:b], do[a:b], **kws)
        assert np.allclose(O[a:b], Os, atol=1e-13) and np.allclose(L[:, a:b], Ls, atol=1e-13)
        for x, y in zip(g, gs):
            assert np.allclose(x[a:b], y, atol=1e-13)


def pin_ring_fold(A, S):
    """Ring rank r: folding chunk partials with the LSE merge equals
    monolithic causal attention over the concatenated keys; its backward
    (per-chunk, with the final O/LSE) equals the monolithic backward."""
    rng = np.random.default_rng(7)
    C, n, r, H, Hkv, D = 8, 4, 2, 4, 2, 5
    L = C * n
    q_full, k_full, v_full, do_full = (_rand(rng, L, H, D), _rand(rng, L, Hkv, D),
                                       _rand(rng, L, Hkv, D), _rand(rng, L, H, D))
    q = q_full[r * C:(r + 1) * C]
    do = do_full[r * C:(r + 1) * C]
    chunks = [(k_full[c * C:(c + 1) * C], v_full[c * C:(c + 1) * C]) for c in range(r + 1)]
    pos = [c * C + np.arange(C) for c in range(r + 1)]
    common = dict(H_loc=H, head_offset=0, num_real_heads=H, gqa_group=2, kv_head_offset=0, scale=0.41)
    o, lse = S.ring_forward(q, chunks, q_pos=r * C + np.arange(C), kv_pos=pos, **common)
    Kc = k_full[:(r + 1) * C]
    Vc = v_full[:(r + 1) * C]
    mono = dict(cu_q=np.array([0, C]), cu_k=np.array([0, (r + 1) * C]),
                pos_q=r * C + np.arange(C), pos_k=np.arange((r + 1) * C), **common)
    Om, Lm = A.attn_forward(q, Kc, Vc, **mono)
    assert np.allclose(o, Om, atol=1e-12) and np.allclose(lse, Lm, atol=1e-12)
    dq, dks, dvs = S.ring_backward(q, chunks, do, o, lse, q_pos=r * C + np.arange(C), kv_pos=pos, **common)
    dqm, dkm, dvm = A.attn_backward(q, Kc, Vc, do, **mono)
    assert np.allclose(dq, dqm, atol=1e-12)
    assert np.allclose(np.concatenate(dks), dkm, atol=1e-12)
    assert np.allclose(np.concatenate(dvs), dvm, atol=1e-12)


def pin_zigzag_fold(A, S):
    """Zigzag ring (Section 3.2): the sequence cut into 2*sp chunks, rank r
    holding chunks r and 2*sp-1-r.  For every rank, folding its sp ring steps
    (each bringing the two chunks of rank (r - s) mod sp, positions jumping
    between the pieces) equals monolithic causal attention of its rows over
    the whole sequence; per-step dK/dV summed over all ranks and steps equal
    the monolithic dK/dV of every key."""
    rng = np.random.default_rng(12)
    sp, C, H, Hkv, D = 3, 6, 4, 2, 5
    L = 2 * sp * C
    q_full, k_full, v_full, do_full = (_rand(rng, L, H, D), _rand(rng, L, Hkv, D),
                                       _rand(rng, L, Hkv, D), _rand(rng, L, H, D))
    common = dict(H_loc=H, head_offset=0, num_real_heads=H, gqa_group=2, kv_head_offset=0, scale=0.41)
    full = dict(cu_q=np.array([0, L]), cu_k=np.array([0, L]), pos_q=np.arange(L), pos_k=np.arange(L),
                **common)
    Om, Lm = A.attn_forward(q_full, k_full, v_full, **full)
    dqm, dkm, dvm = A.attn_backward(q_full, k_full, v_full, do_full, **full)
    dk_sum, dv_sum = np.zeros_like(k_full), np.zeros_like(v_full)
    for r in range(sp):
        rows = np.r_[r * C + np.arange(C), (2 * sp - 1 - r) * C + np.arange(C)]
        steps = [(r - s) % sp for s in range(sp)]
        keys = [np.r_[j * C + np.arange(C), (2 * sp - 1 - j) * C + np.arange(C)] for j in steps]
        chunks = [(k_full[kk], v_full[kk]) for kk in keys]
        o, lse = S.ring_forward(q_full[rows], chunks, q_pos=rows, kv_pos=keys, **common)
        assert np.allclose(o, Om[rows], atol=1e-12) and np.allclose(lse, Lm[:, rows], atol=1e-12)
        dq, dks, dvs = S.ring_backward(q_full[rows], chunks, do_full[rows], o, lse, q_pos=rows,
                                       kv_pos=keys, **common)
        assert np.allclose(dq, dqm[rows], atol=1e-12)
        for kk, a, b in zip(keys, dks, dvs):
            dk_sum[kk] += a
            dv_sum[kk] += b
    assert np.allclose(dk_sum, dkm, atol=1e-12) and np.allclose(dv_sum, dvm, atol=1e-12)


def pin_merge_identity(S):
    """(0, -inf) is the merge identity; the merge is commutative; two
    all-masked partials give (0, -inf) without NaN."""
    rng = np.random.default_rng(8)
    T, H, D = 6, 2, 3
    o, l = _rand(rng, T, H, D), _rand(rng, H, T)
    z, zl = np.zeros((T, H, D)), np.full((H, T), -np.inf)
    a, b = S.lse_merge(o, l, z, zl)
    assert np.array_equal(a, o) and np.array_equal(b, l)
    a, b = S.lse_merge(z, zl, o, l)
    assert np.allclose(a, o, atol=1e-15) and np.array_equal(b, l)
    o2, l2 = _rand(rng, T, H, D), _rand(rng, H, T)
    a1, b1 = S.lse_merge(o, l, o2, l2)
    a2, b2 = S.lse_merge(o2, l2, o, l)
    assert np.allclose(a1, a2, atol=1e-14) and np.allclose(b1, b2, atol=1e-14)
    a, b = S.lse_merge(z, zl, z, zl)
    assert np.all(a == 0) and np.all(b == -np.inf)
    # weights: merging a partial with itself doubles the mass but keeps O
    a, b = S.lse_merge(o, l, o, l)
    assert np.allclose(a, o, atol=1e-14) and np.allclose(b, l + np.log(2), atol=1e-14)


def pin_ulysses_equals_no_sp(A, S):
    """Dummy-Head Ulysses over all ranks equals attention without SP, for MHA
    with hs % sp != 0 and for GQA (the paper's forward-exactness check)."""
    rng = np.random.default_rng(9)
    for L, hs, hkv, sp, D in ((16, 7, 7, 2, 4), (24, 7, 1, 4, 3), (16, 6, 2, 4, 4), (8, 3, 3, 4, 2)):
        q, k, v = _rand(rng, L, hs, D), _rand(rng, L, hkv, D), _rand(rng, L, hkv, D)
        cu = np.array([0, L // 2 + 1, L])
        pos = np.concatenate([np.arange(L // 2 + 1), np.arange(L - L // 2 - 1)])
        o, lses = S.ulysses_simulate(q, k, v, sp, scale=0.5, cu=cu, pos=pos, gqa_group=hs // hkv)
        ref, _ = A.attn_forward(q, k, v, cu_q=cu, cu_k=cu, pos_q=pos, pos_k=pos, H_loc=hs,
                                head_offset=0, num_real_heads=hs, gqa_group=hs // hkv,
                                kv_head_offset=0, scale=0.5)
        assert o.shape == (L, hs, D)
        assert np.allclose(o, ref, atol=1e-13)
        hs_new = padded_heads(hs, sp)
        hloc = hs_new // sp
        for j in range(sp):  # dummy slots carry LSE = -inf
            for h in range(hloc):
                if j * hloc + h >= hs:
                    assert np.all(lses[j][h] == -np.inf)


def pin_pack_unpack(S):
    """unpack(pack(x)) = x bit for bit; pack(x)[j] holds heads j*H.. with
    zero dummies (closed form of the sequential split + head slicing)."""
    rng = np.random.default_rng(10)
    for T, hs, sp, D in ((12, 7, 2, 4), (8, 28, 8, 2), (6, 40, 16, 3)):
        bits = rng.integers(0, 65536, size=(T, hs, D), dtype=np.uint16)
        hs_new = padded_heads(hs, sp)
        hloc = hs_new // sp
        hm = np.array([h if h < hs else -1 for h in range(hs_new)])
        packed = S.ulysses_pack(bits, sp, hloc, hm)
        assert packed.shape == (sp, T, hloc, D)
        padded = S.pad_heads(bits[None], sp)[0]
        for j in range(sp):
            assert np.array_equal(packed[j], padded[:, j * hloc:(j + 1) * hloc])
        back = S.ulysses_unpack(packed, np.where(hm >= 0, hm, -1), hs)
        assert back.dtype == bits.dtype and np.array_equal(back, bits)


def pin_unpack_add_adjoint(S):
    """The summing unpack is the adjoint of the pack (the pack replicates a
    head into every slot that names it): <pack(x), y> = <x, unpack_add(y)>
    for the GQA K/V maps and the MHA map with dummies; with a one-to-one map
    it is the plain unpack."""
    rng = np.random.default_rng(12)
    cases = [(28, 4, 8), (40, 8, 16), (7, 1, 4), (6, 2, 4), (7, 7, 2)]
    for hs, hkv, sp in cases:
        hm = ulysses_kv_head_map(hs, hkv, sp) if hkv != hs else ulysses_q_head_map(hs, sp)
        H = len(hm) // sp
        T, D = 5, 3
        x = _rand(rng, T, hkv, D)
        y = _rand(rng, sp, T, H, D)
        lhs = float(np.sum(S.ulysses_pack(x, sp, H, hm) * y))
        rhs = float(np.sum(x * S.ulysses_unpack_add(y, hm, hkv)))
        assert abs(lhs - rhs) <= 1e-12 * (1.0 + abs(lhs)), (hs, hkv, sp, lhs, rhs)
    hm = ulysses_q_head_map(7, 2)
    y = _rand(rng, 2, 4, 4, 3)
    assert np.array_equal(S.ulysses_unpack_add(y, hm, 7), S.ulysses_unpack(y, hm, 7))


def pin_unpack_add_bf16(S):
    """bfloat16 summing unpack: float32 sum of the copies, one rounding to
    bfloat16, nearest-even.  Closed-form cases (bit patterns): 1 + 2^-9 -> 1
    (under half an ulp), 1 + 2^-8 -> 1 (tie, even), 1 + 2^-8 + 2^-8 -> 1 + 2^-7
    (exact), (1 + 2^-7) + 2^-8 -> 1 + 2^-6 (tie, odd rounds up); random data
    within half an ulp (plus float32 error) of the float64 sum."""
    one, e9, e8, one7 = 0x3F80, 0x3B00, 0x3B80, 0x3F81
    src = np.array([[one, one, one, one7], [e9, e8, e8, e8], [0, 0, e8, 0]],
                   dtype=np.uint16).reshape(3, 1, 1, 4)
    got = S.ulysses_unpack_add_bf16(src, np.array([0, 0, 0]), 1)
    assert got.dtype == np.uint16
    assert got.reshape(-1).tolist() == [0x3F80, 0x3F80, 0x3F81, 0x3F82], got
    rng = np.random.default_rng(13)
    hm = ulysses_kv_head_map(28, 4, 8)
    bits = rng.integers(0x3C00, 0x4100, size=(8, 6, len(hm) // 8, 4)).astype(np.uint16)
    bits |= (rng.integers(0, 2, size=bits.shape) << 15).astype(np.uint16)  # random signs
    got = (S.ulysses_unpack_add_bf16(bits, hm, 4).astype(np.uint32) << 16).view(np.float32)
    vals = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ref = S.ulysses_unpack_add(vals, hm, 4)
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-6)


def pin_ulysses_backward_equals_no_sp(A, S):
    """DHU backward over all ranks (dO through the same pad + all-to-all, dQ
    back through the reverse all-to-all and unpad, replicated GQA K/V
    gradients summed by the unpack) equals the backward without SP."""
    rng = np.random.default_rng(14)
    for L, hs, hkv, sp, D in ((16, 7, 7, 2, 4), (24, 7, 1, 4, 3), (16, 6, 2, 4, 4),
                              (16, 28, 4, 8, 2)):
        q, k, v = _rand(rng, L, hs, D), _rand(rng, L, hkv, D), _rand(rng, L, hkv, D)
        do = _rand(rng, L, hs, D)
        cu = np.array([0, L // 2 + 1, L])
        pos = np.concatenate([np.arange(L // 2 + 1), np.arange(L - L // 2 - 1)])
        g = hs // hkv
        dq, dk, dv = S.ulysses_simulate_backward(q, k, v, do, sp, scale=0.5, cu=cu, pos=pos,
                                                 gqa_group=g)
        rq, rk, rv = A.attn_backward(q, k, v, do, cu_q=cu, cu_k=cu, pos_q=pos, pos_k=pos,
                                     H_loc=hs, head_offset=0, num_real_heads=hs, gqa_group=g,
                                     kv_head_offset=0, scale=0.5)
        for a, b in ((dq, rq), (dk, rk), (dv, rv)):
            assert a.shape == b.shape and np.allclose(a, b, atol=1e-12), (L, hs, hkv, sp)


def pin_usp_equals_no_sp(A, S):
    """USP over every rank of an sp_hp x sp_cp mesh (Ulysses inside ring
    groups, zigzag ring across them, Table 1) equals attention without SP,
    forward and backward: MHA with dummy heads, GQA with replicated KV heads
    and a one-KV-head-per-rank GQA layout."""
    rng = np.random.default_rng(15)
    for L, hs, hkv, hp, cp, D in ((24, 7, 7, 2, 2, 3), (36, 6, 2, 2, 3, 4), (32, 8, 4, 4, 2, 2)):
        q, k, v = _rand(rng, L, hs, D), _rand(rng, L, hkv, D), _rand(rng, L, hkv, D)
        do = _rand(rng, L, hs, D)
        g = hs // hkv
        O, dQ, dK, dV, per = S.usp_simulate(q, k, v, do, hp, cp, scale=0.45, gqa_group=g)
        full = dict(cu_q=np.array([0, L]), cu_k=np.array([0, L]), pos_q=np.arange(L),
                    pos_k=np.arange(L), H_loc=hs, head_offset=0, num_real_heads=hs,
                    gqa_group=g, kv_head_offset=0, scale=0.45)
        Om, _ = A.attn_forward(q, k, v, **full)
        rq, rk, rv = A.attn_backward(q, k, v, do, **full)
        for a, b in ((O, Om), (dQ, rq), (dK, rk), (dV, rv)):
            assert np.allclose(a, b, atol=1e-12), (L, hs, hkv, hp, cp)
        assert len(per) == hp * cp


# ------------------------------------------------------------------ loss
def pin_token_logprobs_torch(Lo):
    """Token log-probabilities against torch's float64 cross entropy (minus
    it), with ignored labels; closed forms: a constant row gives
    lse = c + log V and logp = -log V."""
    rng = np.random.default_rng(16)
    T, V = 9, 37
    x = rng.standard_normal((T, V)) * 3
    lab = rng.integers(0, V, T)
    lab[[2, 5]] = -100
    logp, lse = Lo.token_logprobs(x, lab)
    ce = torch.nn.functional.cross_entropy(torch.from_numpy(x), torch.from_numpy(lab),
                                           ignore_index=-100, reduction="none").numpy()
    assert np.allclose(logp, -ce, atol=1e-12) and np.all(logp[[2, 5]] == 0.0)
    assert np.allclose(lse, torch.logsumexp(torch.from_numpy(x), 1).numpy(), atol=1e-12)
    c = np.full((2, V), 1.75)
    lp, ls = Lo.token_logprobs(c, np.array([0, V - 1]))
    assert np.allclose(ls, 1.75 + np.log(V), atol=1e-13) and np.allclose(lp, -np.log(V), atol=1e-13)
    assert np.allclose(Lo.sequence_sums(logp, [0, 4, 9]), [logp[:4].sum(), logp[4:].sum()])


def pin_token_grad_fd(Lo):
    """dlogits of sum_s g_s * (sum of logp over sequence s): central finite
    differences; each token's row sums to zero; ignored tokens and tokens
    past the last sequence get zero."""
    rng = np.random.default_rng(17)
    T, V = 7, 5
    x = rng.standard_normal((T, V))
    lab = rng.integers(0, V, T)
    lab[3] = -100
    cu = np.array([0, 2, 6])  # token 6 is padding
    g = np.array([0.7, -1.3])

    def f(xx):
        return float(np.dot(g, Lo.sequence_sums(Lo.token_logprobs(xx, lab)[0], cu)))

    d = Lo.token_logprob_grad(x, lab, g, cu)
    h = 1e-6
    fd = np.zeros_like(x)
    for t in range(T):
        for v in range(V):
            e = np.zeros_like(x)
            e[t, v] = h
            fd[t, v] = (f(x + e) - f(x - e)) / (2 * h)
    assert np.allclose(d, fd, atol=1e-8)
    assert np.allclose(d.sum(axis=1), 0.0, atol=1e-14)
    assert np.all(d[3] == 0) and np.all(d[6] == 0)


def pin_listing2_worked_example(Lo):
    """The paper's Listing 2 numbers (golden fixture): w0 gradients 8 / 12
    with the gradient-carrying all-reduce, 4 / 6 without, 10 locally."""
    with open(os.path.join(os.path.dirname(__file__), "golden", "listing2_allreduce_grads.json")) as fh:
        gold = json.load(fh)
    x = gold["x_per_rank"]
    assert Lo.listing2_w0_grads(x, autograd=True).tolist() == gold["w0_grad_nn_all_reduce"]
    assert Lo.listing2_w0_grads(x, autograd=False).tolist() == gold["w0_grad_plain_all_reduce"]
    assert Lo.listing2_w0_grads([gold["x_local"]], autograd=True).tolist() == [gold["w0_grad_local"]]
    assert np.mean(Lo.listing2_w0_grads(x, autograd=True)) == gold["w0_grad_local"]


def _linear_head_grads(Lo, h, W, lab, cu, sp, kind, autograd, ref_sums=None, beta=0.1, scale=1.0):
    """Weight gradient of a shared linear head (logits = h W) averaged over
    sp ranks that each hold a sequential slice of every sequence's tokens."""
    L = h.shape[0]
    Tl = L // sp
    parts = []
    for r in range(sp):
        rows = np.arange(r * Tl, (r + 1) * Tl)
        lp, _ = Lo.token_logprobs(h[rows] @ W, lab[rows])
        # sequence boundaries inside the slice
        cu_r = np.clip(np.asarray(cu) - r * Tl, 0, Tl)
        parts.append((rows, cu_r, Lo.sequence_sums(lp, cu_r)))
    ps = np.stack([p[2] for p in parts])
    if kind == "sft":
        loss, up = Lo.sft_loss(ps, scale=scale, autograd=autograd)
    else:
        loss, up = Lo.dpo_loss(ps, ref_sums, beta, autograd=autograd)
    dW = np.zeros_like(W)
    for r, (rows, cu_r, _) in enumerate(parts):
        dW += h[rows].T @ Lo.token_logprob_grad(h[rows] @ W, lab[rows], up[r], cu_r)
    return loss, dW / sp


def pin_sp_loss_equals_no_sp(Lo):
    """SFT and DPO with the all-reduced sums: with the gradient-carrying
    all-reduce, the rank-averaged gradient of a shared linear head equals
    the gradient without SP (and the loss is the same); with a plain
    all-reduce it is 1/sp of it -- Listing 2's finding, for the losses of
    Section 3.3.  DPO against torch float64 autograd of -logsigmoid."""
    rng = np.random.default_rng(18)
    L, d, V, sp = 24, 6, 11, 3
    h = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V)) * 0.5
    lab = rng.integers(0, V, L)
    lab[[0, 13]] = -100
    cu = np.array([0, 10, 24])  # DPO: sequence 0 chosen, sequence 1 rejected
    ref = rng.standard_normal((1, 2)) * 3
    for kind in ("sft", "dpo"):
        kw = dict(ref_sums=ref, beta=0.3, scale=1.0 / 22)
        loss1, g1 = _linear_head_grads(Lo, h, W, lab, cu, 1, kind, True, **kw)
        lossn, gn = _linear_head_grads(Lo, h, W, lab, cu, sp, kind, True,
                                       **dict(kw, ref_sums=np.vstack([ref] + [np.zeros((1, 2))] * (sp - 1))))
        lossp, gp = _linear_head_grads(Lo, h, W, lab, cu, sp, kind, False,
                                       **dict(kw, ref_sums=np.vstack([ref] + [np.zeros((1, 2))] * (sp - 1))))
        assert abs(loss1 - lossn) <= 1e-12 and np.allclose(g1, gn, atol=1e-12), kind
        assert np.allclose(gp * sp, g1, atol=1e-12), kind
    # DPO loss and gradient against torch autograd on the reduced sums
    ps = torch.tensor(rng.standard_normal((sp, 4)), dtype=torch.float64, requires_grad=True)
    rs = rng.standard_normal((sp, 4))
    tot, rtot = ps.sum(0), torch.from_numpy(rs.sum(0))
    z = 0.3 * ((tot[0::2] - rtot[0::2]) - (tot[1::2] - rtot[1::2]))
    lt = -torch.nn.functional.logsigmoid(z).mean()
    lt.backward()
    lo, up = Lo.dpo_loss(ps.detach().numpy(), rs, 0.3, autograd=False)
    assert abs(lo - float(lt.detach())) <= 1e-12 and np.allclose(up, ps.grad.numpy(), atol=1e-12)


ATTN_PINS = [pin_single_visible_key, pin_zero_query_uniform, pin_torch_sdpa,
             pin_finite_differences, pin_gradient_sums, pin_packed_equals_separate,
             pin_sampled_checkers, pin_bf16_decode]
SP_PINS = [pin_merge_identity, pin_pack_unpack, pin_unpack_add_adjoint, pin_unpack_add_bf16]
LOSS_PINS = [pin_token_logprobs_torch, pin_token_grad_fd, pin_listing2_worked_example,
             pin_sp_loss_equals_no_sp]
BOTH_PINS = [pin_ring_fold, pin_zigzag_fold, pin_ulysses_equals_no_sp,
             pin_ulysses_backward_equals_no_sp, pin_usp_equals_no_sp]
