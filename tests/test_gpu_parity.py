"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded bf16 inputs.  Sizes span several tiles and ragged tails.

Bars: pack/unpack bit-exact; attention O, dQ, dK, dV max-abs <= 2e-2 and
rel-L2 <= 5e-3 over real heads; LSE max-abs <= 1e-3; dummy slots bit-zero;
the float32 merge within 1e-5 max-abs / 1e-6 rel-L2."""
import numpy as np
import pytest

import oracle
from tests.helpers import (assert_close, bits_from_dev, from_dev, lib_desc, make_shard,
                           oracle_kw, scaled_max_abs, to_dev, LSE_MAX_ABS)
from workloads import (bf16_bits_from_f32, padded_heads, randn_bf16_bits, shard_inputs,
                       ulysses_kv_head_map, ulysses_q_head_map, usp_shard, workload,
                       WORKLOADS)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _dec(bits):
    return oracle.bf16_bits_to_f64(bits)


# ------------------------------------------------------------ pack/unpack
@pytest.mark.parametrize("T,hs,sp_size,D", [(512, 7, 2, 64), (4096, 28, 8, 128), (1000, 40, 16, 128),
                                            (3, 5, 4, 64)])
def test_pack_unpack_bit_exact(sp, T, hs, sp_size, D):
    print(f"pack T={T} hs={hs} sp={sp_size} D={D}", flush=True)
    bits = randn_bf16_bits((T, hs, D), seed=T + hs)
    hm = ulysses_q_head_map(hs, sp_size)
    hloc = padded_heads(hs, sp_size) // sp_size
    x = to_dev(bits)
    packed = sp.sp_ulysses_pack(x, sp_size, hloc, hm)
    ref = oracle.ulysses_pack(bits, sp_size, hloc, hm)
    got = bits_from_dev(packed)
    assert np.array_equal(got, ref)
    back = sp.sp_ulysses_unpack(packed, hm, hs)
    assert np.array_equal(bits_from_dev(back), bits)
    assert np.array_equal(bits_from_dev(back), oracle.ulysses_unpack(ref, hm, hs))


def test_pack_gqa_kv_map_bit_exact(sp):
    bits = randn_bf16_bits((256, 4, 128), seed=5)
    hm = ulysses_kv_head_map(28, 4, 8)
    w = len(hm) // 8
    got = bits_from_dev(sp.sp_ulysses_pack(to_dev(bits), 8, w, hm))
    assert np.array_equal(got, oracle.ulysses_pack(bits, 8, w, hm))


@pytest.mark.parametrize("T,hs,hkv,sp_size,D", [(4096, 28, 4, 8, 128), (1000, 40, 8, 16, 128),
                                                (333, 7, 1, 4, 64), (3, 6, 2, 4, 128),
                                                (77, 7, 7, 2, 64)])
def test_unpack_add_bit_exact(sp, T, hs, hkv, sp_size, D):
    """Summing unpack of replicated K/V gradients: bit-exact against the
    oracle's float32 ordered sum + one RNE rounding (GQA maps, where KV heads
    appear in up to three slots, and the one-copy MHA map)."""
    print(f"unpack_add T={T} hs={hs} hkv={hkv} sp={sp_size} D={D}", flush=True)
    hm = (ulysses_kv_head_map(hs, hkv, sp_size) if hkv != hs else ulysses_q_head_map(hs, sp_size))
    w = len(hm) // sp_size
    rng = np.random.default_rng(T + hs + D)
    bits = randn_bf16_bits((sp_size, T, w, D), seed=T + 7 * hs)
    got = bits_from_dev(sp.sp_ulysses_unpack_add(to_dev(bits), hm, hkv))
    ref = oracle.ulysses_unpack_add_bf16(bits, hm, hkv)
    assert got.shape == ref.shape and np.array_equal(got, ref)
    if hkv == hs:  # one copy per head: the plain unpack
        assert np.array_equal(got, oracle.ulysses_unpack(bits, hm, hkv))
    # a head no slot names comes out +0; cancelling copies give +0 too
    hm2 = np.array([0, -1, 0, 2], dtype=np.int32)
    b2 = rng.integers(0x0080, 0x7F00, size=(2, T, 2, D)).astype(np.uint16)  # normal
    b2[1, :, 0] = b2[0, :, 0] ^ 0x8000  # x + (-x)
    got2 = bits_from_dev(sp.sp_ulysses_unpack_add(to_dev(b2), hm2, 3))
    assert np.array_equal(got2, oracle.ulysses_unpack_add_bf16(b2, hm2, 3))
    assert np.all(got2[:, 1] == 0) and np.all(got2[:, 0] == 0)


# ------------------------------------------------------------------ merge
@pytest.mark.parametrize("part_bf16", [False, True])
def test_lse_merge(sp, part_bf16):
    import torch
    rng = np.random.default_rng(3)
    T, H, D = 777, 3, 128
    oa = rng.standard_normal((T, H, D)).astype(np.float32)
    la = rng.standard_normal((H, T)).astype(np.float32) * 3
    ob_bits = randn_bf16_bits((T, H, D), seed=9)
    ob = _dec(ob_bits).astype(np.float32) if part_bf16 else rng.standard_normal((T, H, D)).astype(np.float32)
    lb = rng.standard_normal((H, T)).astype(np.float32) * 3
    la[0, :50] = -np.inf
    lb[0, 25:75] = -np.inf
    lb[1, :10] = -np.inf
    la[1, :10] = -np.inf
    d_oa = torch.from_numpy(oa).cuda()
    d_la = torch.from_numpy(la).cuda()
    d_ob = to_dev(ob_bits) if part_bf16 else torch.from_numpy(ob).cuda()
    d_lb = torch.from_numpy(lb).cuda()
    out = torch.empty((T, H, D), dtype=torch.bfloat16, device="cuda")
    sp.sp_lse_merge(d_oa, d_la, d_ob, d_lb, o_out=out)
    ro, rl = oracle.lse_merge(oa.astype(np.float64), la.astype(np.float64), ob.astype(np.float64),
                              lb.astype(np.float64))
    go, gl = d_oa.cpu().numpy().astype(np.float64), d_la.cpu().numpy().astype(np.float64)
    assert np.array_equal(np.isneginf(gl), np.isneginf(rl))
    fin = np.isfinite(rl)
    assert np.abs(gl[fin] - rl[fin]).max() < 1e-5
    assert_close(go, ro, "merged O", max_abs=1e-5, rel_l2=1e-6)
    assert np.all(go[:10, 1] == 0)  # both -inf rows -> 0
    assert_close(from_dev(out), ro, "bf16 finalize", max_abs=2e-2, rel_l2=5e-3)


# -------------------------------------------------------- attention parity
CASES = [
    # name, T_q, T_k, D, H_loc, head_off, real, padded, gqa, Hkv, kv_off, seg_q, seg_k, extra
    ("gqa4_T333_d128", 333, 333, 128, 4, 0, 4, 4, 4, 1, 0, [333], None, {}),
    ("varlen_gqa5_dummy2_d128", 439, 439, 128, 4, 8, 10, 12, 5, 1, 1, [5, 130, 0, 200, 64], None, {}),
    ("mha_dummy_d64", 300, 300, 64, 4, 4, 7, 8, 1, 4, 4, [300], None, {}),
    ("ring_offsets_d128", 200, 300, 128, 2, 0, 2, 2, 1, 2, 0, [200], [300],
     dict(pos_q=1000 + np.arange(200), pos_k=900 + np.arange(300))),
    ("noncausal_varlen_d64", 300, 280, 64, 3, 0, 3, 3, 3, 1, 0, [100, 200], [180, 100],
     dict(causal=False)),
    ("gqa2_partial_d128", 257, 257, 128, 4, 0, 4, 4, 2, 2, 0, [129, 128], None, {}),
    # pieces of one sequence (SP_DESC_SINGLE_SEQUENCE), uneven, with gaps
    ("pieces_uneven_d128", 300, 330, 128, 2, 0, 2, 2, 1, 2, 0, [40, 200, 60], [100, 30, 200],
     dict(pos_q=np.r_[10 + np.arange(40), 150 + np.arange(200), 600 + np.arange(60)],
          pos_k=np.r_[np.arange(100), 140 + np.arange(30), 400 + np.arange(200)],
          single_sequence=True)),
]


def _case(c, seed):
    name, Tq, Tk, D, H, ho, nr, npd, g, Hkv, ko, sq, sk, extra = c
    return make_shard(name, Tq, Tk, D, H, ho, nr, npd, g, Hkv, ko, sq, sk, seed_base=seed, **extra)


def _run_fwd_bwd(sp, sh, q, k, v, do):
    import torch
    d = lib_desc(sh)
    dq_, dk_, dv_ = (to_dev(x) for x in (q, k, v))
    o, lse = sp.sp_attn_fwd(d, dq_, dk_, dv_)
    gq, gk, gv = sp.sp_attn_bwd(d, dq_, dk_, dv_, o, lse, to_dev(do))
    torch.cuda.synchronize()
    return o, lse, gq, gk, gv


@pytest.mark.parametrize("c", CASES, ids=lambda c: c[0])
def test_attention_fwd_bwd_parity(sp, c):
    sh = _case(c, seed=1000 + len(c[0]))
    print(f"case {sh.name}", flush=True)
    q, k, v, do = shard_inputs(sh)
    o, lse, gq, gk, gv = _run_fwd_bwd(sp, sh, q, k, v, do)
    Q, K, V, dO = (_dec(x) for x in (q, k, v, do))
    kw = oracle_kw(sh)
    RO, RL = oracle.attn_forward(Q, K, V, **kw)
    RdQ, RdK, RdV = oracle.attn_backward(Q, K, V, dO, **kw)
    nr = sh.n_real_loc
    GO, GL = from_dev(o), lse.cpu().numpy().astype(np.float64)
    assert_close(GO[:, :nr], RO[:, :nr], "O")
    fin = np.isfinite(RL[:nr])
    assert np.array_equal(np.isfinite(GL[:nr]), fin)
    assert np.abs(GL[:nr][fin] - RL[:nr][fin]).max() <= LSE_MAX_ABS
    assert_close(from_dev(gq)[:, :nr], RdQ[:, :nr], "dQ")
    assert_close(from_dev(gk), RdK, "dK")
    assert_close(from_dev(gv), RdV, "dV")
    # dummy slots: bit-zero outputs, LSE -inf
    if nr < sh.H_loc:
        assert np.all(bits_from_dev(o)[:, nr:] == 0)
        assert np.all(bits_from_dev(gq)[:, nr:] == 0)
        assert np.all(np.isneginf(GL[nr:]))
    # rows with no keys: exact zero
    none = ~np.isfinite(RL[0]) if nr else np.zeros(sh.T_q, bool)
    if nr and none.any():
        assert np.all(bits_from_dev(o)[none][:, :nr] == 0)


def test_c0_workload_and_dummy_kv(sp):
    """The tiny Ulysses shard: MHA 7 heads padded to 8 for SP 2, rank 1 (head
    7 and KV head 7 are dummies), D = 64, L = 1024."""
    sh = workload(WORKLOADS[0])
    q, k, v, do = shard_inputs(sh)
    o, lse, gq, gk, gv = _run_fwd_bwd(sp, sh, q, k, v, do)
    Q, K, V, dO = (_dec(x) for x in (q, k, v, do))
    kw = oracle_kw(sh)
    RO, RL = oracle.attn_forward(Q, K, V, **kw)
    RdQ, RdK, RdV = oracle.attn_backward(Q, K, V, dO, **kw)
    assert_close(from_dev(o)[:, :3], RO[:, :3], "O")
    assert_close(from_dev(gq)[:, :3], RdQ[:, :3], "dQ")
    assert_close(from_dev(gk)[:, :3], RdK[:, :3], "dK")
    assert_close(from_dev(gv)[:, :3], RdV[:, :3], "dV")
    for t in (o, gq, gk, gv):
        assert np.all(bits_from_dev(t)[:, 3] == 0)
    assert np.all(np.isneginf(lse.cpu().numpy()[3]))


def test_peaky_inputs_exercise_rescale(sp):
    """Q scaled by 3 makes the running max jump often (online rescale path)."""
    sh = _case(CASES[0], seed=77)
    q, k, v, do = shard_inputs(sh, peaky=3.0)
    o, lse, gq, gk, gv = _run_fwd_bwd(sp, sh, q, k, v, do)
    Q, K, V, dO = (_dec(x) for x in (q, k, v, do))
    kw = oracle_kw(sh)
    RO, RL = oracle.attn_forward(Q, K, V, **kw)
    RdQ, RdK, RdV = oracle.attn_backward(Q, K, V, dO, **kw)
    # Q x 3 scales dK up to |10|, where one bf16 ulp is 0.0625: the absolute
    # bar becomes two bf16 ulps of the largest reference value (never below
    # 2e-2); rel-L2 keeps the 5e-3 bar.
    for g, r, what in ((from_dev(o), RO, "O"), (from_dev(gq), RdQ, "dQ"),
                       (from_dev(gk), RdK, "dK"), (from_dev(gv), RdV, "dV")):
        assert_close(g, r, what, max_abs=scaled_max_abs(r))
    assert np.abs(lse.cpu().numpy() - RL).max() <= LSE_MAX_ABS


@pytest.mark.parametrize("causal", [True, False])
def test_rising_scores_raise_the_max_every_tile(sp, causal):
    """Scores that climb along the keys (a ramp in one dimension of K, met by
    a constant in Q: about 1.6 per key before scaling, against the raise
    threshold 8 / (scale log2 e) ~ 63 per 64-key tile) raise the forward's
    running max in most tiles of every row, so the carried threshold, the
    scaled max and the O / row-sum rescale run tile after tile; T = 333
    leaves a ragged last tile.  Checked: O, LSE, dV, dK, and dQ except its
    ramp column: with |K| up to ~133 there, dQ[:, :, 0] is
    scale * sum_j dS_j K_j with sum_j dS_j = 0 per row, a small difference
    of large terms in which the bf16 rounding of dS (as in any bf16
    backward) is magnified ~100-fold.  The other 127 columns multiply
    N(0, 1) keys and dK has no such cancellation, so both take the usual
    bars."""
    T, H, D = 333, 2, 128
    sh = make_shard("ramp", T, T, D, H, 0, H, H, 1, H, 0, [T], [T], causal=causal)
    q = randn_bf16_bits((T, H, D), 81)
    k = randn_bf16_bits((T, H, D), 82)
    v = randn_bf16_bits((T, H, D), 83)
    do = randn_bf16_bits((T, H, D), 84)
    q[:, :, 0] = bf16_bits_from_f32(np.full((T, H), 4.0, np.float32))
    k[:, :, 0] = bf16_bits_from_f32(np.repeat((0.4 * np.arange(T, dtype=np.float32))[:, None], H, 1))
    o, lse, gq, gk, gv = _run_fwd_bwd(sp, sh, q, k, v, do)
    Q, K, V, dO = (_dec(x) for x in (q, k, v, do))
    kw = oracle_kw(sh)
    RO, RL = oracle.attn_forward(Q, K, V, **kw)
    RdQ, RdK, RdV = oracle.attn_backward(Q, K, V, dO, **kw)
    assert_close(from_dev(o), RO, "O")
    gq_, gk_ = from_dev(gq), from_dev(gk)
    assert_close(gq_[:, :, 1:], RdQ[:, :, 1:], "dQ (columns 1..)",
                 max_abs=scaled_max_abs(RdQ[:, :, 1:]))
    assert_close(gk_, RdK, "dK", max_abs=scaled_max_abs(RdK))
    assert np.abs(lse.cpu().numpy() - RL).max() <= LSE_MAX_ABS
    # without the causal mask every row's weight piles onto the top keys,
    # whose dV sums all 333 rows of dO (|dV| past 16, where one bf16 ulp is
    # 0.125): two bf16 ulps of the largest reference value, rel-L2 unchanged
    assert_close(from_dev(gv), RdV, "dV", max_abs=scaled_max_abs(RdV))


def test_deterministic(sp):
    sh = _case(CASES[1], seed=5)
    q, k, v, do = shard_inputs(sh)
    a = _run_fwd_bwd(sp, sh, q, k, v, do)
    b = _run_fwd_bwd(sp, sh, q, k, v, do)
    for x, y in zip(a, b):
        if x.dtype.is_floating_point and x.dtype != __import__("torch").float32:
            assert np.array_equal(bits_from_dev(x), bits_from_dev(y))
        else:
            assert np.array_equal(x.cpu().numpy(), y.cpu().numpy())


# -------------------------------------------------------------------- ring
def test_ring_rank_fwd_bwd(sp):
    """Rank r = 2 of a contiguous ring: Q chunk against KV chunks 0..2 with
    the fused LSE merge; backward per chunk with the final O/LSE and an fp32
    dQ accumulator.  Oracle: ring fold and per-chunk backward."""
    import torch
    C, r, H, Hkv, D = 160, 2, 4, 2, 128
    base = make_shard("ring", C, C, D, H, 0, H, H, 2, Hkv, 0, [C], [C])
    q = randn_bf16_bits((C, H, D), 11)
    do = randn_bf16_bits((C, H, D), 12)
    ks = [randn_bf16_bits((C, Hkv, D), 20 + c) for c in range(r + 1)]
    vs = [randn_bf16_bits((C, Hkv, D), 40 + c) for c in range(r + 1)]
    pos_q = r * C + np.arange(C)
    dq = to_dev(q)
    o_acc = torch.empty((C, H, D), dtype=torch.float32, device="cuda")
    lse_acc = torch.empty((H, C), dtype=torch.float32, device="cuda")
    o_bf = torch.empty((C, H, D), dtype=torch.bfloat16, device="cuda")
    for c in range(r + 1):
        d = lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C))
        sp.sp_ring_step(d, dq, to_dev(ks[c]), to_dev(vs[c]), o_acc, lse_acc, init=(c == 0),
                        o_out=o_bf if c == r else None)
    common = dict(H_loc=H, head_offset=0, num_real_heads=H, gqa_group=2, kv_head_offset=0,
                  scale=base.scale)
    chunks = [(_dec(ks[c]), _dec(vs[c])) for c in range(r + 1)]
    kvpos = [c * C + np.arange(C) for c in range(r + 1)]
    RO, RL = oracle.ring_forward(_dec(q), chunks, q_pos=pos_q, kv_pos=kvpos, **common)
    assert_close(o_acc.cpu().numpy().astype(np.float64), RO, "ring O acc")
    assert_close(from_dev(o_bf), RO, "ring O bf16")
    assert np.abs(lse_acc.cpu().numpy() - RL).max() <= LSE_MAX_ABS
    # backward
    dq_acc = torch.zeros((C, H, D), dtype=torch.float32, device="cuda")
    dks, dvs = [], []
    for c in range(r + 1):
        d = lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C))
        _, gk, gv = sp.sp_attn_bwd(d, dq, to_dev(ks[c]), to_dev(vs[c]), o_bf, lse_acc, to_dev(do),
                                   dq_acc=dq_acc)
        dks.append(from_dev(gk))
        dvs.append(from_dev(gv))
    RdQ, RdKs, RdVs = oracle.ring_backward(_dec(q), chunks, _dec(do), RO, RL, q_pos=pos_q,
                                           kv_pos=kvpos, **common)
    assert_close(dq_acc.cpu().numpy().astype(np.float64), RdQ, "ring dQ")
    gq_bf = sp.sp_f32_to_bf16(dq_acc)
    assert_close(from_dev(gq_bf), RdQ, "ring dQ bf16")
    for c in range(r + 1):
        assert_close(dks[c], RdKs[c], f"ring dK chunk {c}")
        assert_close(dvs[c], RdVs[c], f"ring dV chunk {c}")
    # the row statistics formed once (chunk 0) and reused by the other
    # chunks' calls on one workspace: the same bits
    ws = torch.empty(sp.sp_attn_workspace_size(lib_desc(base, pos_q=pos_q, pos_k=np.arange(C)),
                                               sp.SP_OP_BWD), dtype=torch.uint8, device="cuda")
    dq_acc2 = torch.zeros((C, H, D), dtype=torch.float32, device="cuda")
    for c in range(r + 1):
        d = lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C), rowstats_ready=c > 0)
        _, gk, gv = sp.sp_attn_bwd(d, dq, to_dev(ks[c]), to_dev(vs[c]), o_bf, lse_acc, to_dev(do),
                                   dq_acc=dq_acc2, workspace=ws)
        assert np.array_equal(from_dev(gk), dks[c]) and np.array_equal(from_dev(gv), dvs[c])
    assert np.array_equal(dq_acc2.cpu().numpy(), dq_acc.cpu().numpy())
    # the accumulator started by the first chunk (SP_DESC_DQ_ACC_INIT: its
    # NaN start is never read) and finished by the last, which writes bf16
    # dQ directly and leaves the accumulator at the other chunks' sum: the
    # same values as the cleared accumulator and the separate cast
    dq_acc3 = torch.full((C, H, D), float("nan"), dtype=torch.float32, device="cuda")
    dq_bf3 = torch.empty((C, H, D), dtype=torch.bfloat16, device="cuda")
    for c in range(r + 1):
        d = lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C), rowstats_ready=c > 0,
                     dq_acc_init=c == 0)
        sp.sp_attn_bwd(d, dq, to_dev(ks[c]), to_dev(vs[c]), o_bf, lse_acc, to_dev(do),
                       dq=dq_bf3 if c == r else None, dq_acc=dq_acc3, workspace=ws)
    assert np.array_equal(from_dev(dq_bf3), from_dev(gq_bf))
    partial = torch.zeros((C, H, D), dtype=torch.float32, device="cuda")
    for c in range(r):
        sp.sp_attn_bwd(lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C)), dq,
                       to_dev(ks[c]), to_dev(vs[c]), o_bf, lse_acc, to_dev(do), dq_acc=partial)
    assert np.array_equal(dq_acc3.cpu().numpy(), partial.cpu().numpy())


def test_ring_steps_with_dummy_slots(sp):
    """Ring steps on a rank with dummy query slots (7 real heads padded to 8
    for SP 2, rank 1: slot 3 is a dummy), the accumulators holding garbage
    before the first chunk: after init the dummy slot is the merge identity
    (O_acc = +0, LSE = -inf), later chunks leave it so, the bf16 copy of the
    last chunk is +0 there, and the real slots match the oracle's ring fold.
    The dummy fills are work items of the ring-step launch itself."""
    import torch
    C, r, H, D = 300, 1, 4, 64
    base = make_shard("ring_dummy", C, C, D, H, 4, 7, 8, 7, 1, 0, [C], [C])
    nr = base.n_real_loc
    q = randn_bf16_bits((C, H, D), 61)
    q[:, nr:] = 0
    ks = [randn_bf16_bits((C, 1, D), 62 + c) for c in range(r + 1)]
    vs = [randn_bf16_bits((C, 1, D), 64 + c) for c in range(r + 1)]
    pos_q = r * C + np.arange(C)
    o_acc = torch.full((C, H, D), float("nan"), dtype=torch.float32, device="cuda")
    lse_acc = torch.full((H, C), 3.0, dtype=torch.float32, device="cuda")
    o_bf = torch.full((C, H, D), 5.0, dtype=torch.bfloat16, device="cuda")
    for c in range(r + 1):
        d = lib_desc(base, pos_q=pos_q, pos_k=c * C + np.arange(C))
        sp.sp_ring_step(d, to_dev(q), to_dev(ks[c]), to_dev(vs[c]), o_acc, lse_acc, init=(c == 0),
                        o_out=o_bf if c == r else None)
        if c == 0:
            torch.cuda.synchronize()
            assert torch.all(o_acc[:, nr:] == 0) and bool(torch.all(torch.isneginf(lse_acc[nr:])))
    torch.cuda.synchronize()
    assert np.all(o_acc[:, nr:].cpu().numpy().view(np.int32) == 0)
    assert bool(torch.all(torch.isneginf(lse_acc[nr:])))
    assert np.all(bits_from_dev(o_bf)[:, nr:] == 0)
    common = dict(H_loc=H, head_offset=4, num_real_heads=7, gqa_group=7, kv_head_offset=0,
                  scale=base.scale)
    chunks = [(_dec(ks[c]), _dec(vs[c])) for c in range(r + 1)]
    kvpos = [c * C + np.arange(C) for c in range(r + 1)]
    RO, RL = oracle.ring_forward(_dec(q), chunks, q_pos=pos_q, kv_pos=kvpos, **common)
    assert_close(o_acc[:, :nr].cpu().numpy().astype(np.float64), RO[:, :nr], "ring O acc")
    assert_close(from_dev(o_bf)[:, :nr], RO[:, :nr], "ring O bf16")
    assert np.abs(lse_acc[:nr].cpu().numpy() - RL[:nr]).max() <= LSE_MAX_ABS


@pytest.mark.parametrize("D,Hkv", [(128, 2), (64, 4)])
def test_zigzag_rank_fwd_bwd(sp, D, Hkv):
    """Zigzag ring (Section 3.2) with sp = 3 and 2*sp chunks of C tokens:
    rank 1 holds chunks 1 and 4 and meets, step by step, the chunks of ranks
    1, 0, 2 -- every step is one sp_ring_step / sp_attn_bwd over pieces of one
    sequence (SP_DESC_SINGLE_SEQUENCE) whose positions jump between pieces.
    Oracle: ring fold and per-step backward over the same pieces."""
    import torch
    spn, C, r, H = 3, 72, 1, 4
    base = make_shard("zigzag", 2 * C, 2 * C, D, H, 0, H, H, H // Hkv, Hkv, 0, [C, C], [C, C],
                      single_sequence=True)
    pos_q = np.r_[r * C + np.arange(C), (2 * spn - 1 - r) * C + np.arange(C)]
    q = randn_bf16_bits((2 * C, H, D), 61)
    do = randn_bf16_bits((2 * C, H, D), 62)
    steps = [(r - s) % spn for s in range(spn)]
    kvpos = [np.r_[j * C + np.arange(C), (2 * spn - 1 - j) * C + np.arange(C)] for j in steps]
    ks = [randn_bf16_bits((2 * C, Hkv, D), 70 + s) for s in range(spn)]
    vs = [randn_bf16_bits((2 * C, Hkv, D), 80 + s) for s in range(spn)]
    dq = to_dev(q)
    o_acc = torch.empty((2 * C, H, D), dtype=torch.float32, device="cuda")
    lse_acc = torch.empty((H, 2 * C), dtype=torch.float32, device="cuda")
    o_bf = torch.empty((2 * C, H, D), dtype=torch.bfloat16, device="cuda")
    for s in range(spn):
        d = lib_desc(base, pos_q=pos_q, pos_k=kvpos[s])
        sp.sp_ring_step(d, dq, to_dev(ks[s]), to_dev(vs[s]), o_acc, lse_acc, init=(s == 0),
                        o_out=o_bf if s == spn - 1 else None)
    common = dict(H_loc=H, head_offset=0, num_real_heads=H, gqa_group=H // Hkv, kv_head_offset=0,
                  scale=base.scale)
    chunks = [(_dec(ks[s]), _dec(vs[s])) for s in range(spn)]
    RO, RL = oracle.ring_forward(_dec(q), chunks, q_pos=pos_q, kv_pos=kvpos, **common)
    assert_close(o_acc.cpu().numpy().astype(np.float64), RO, "zigzag O acc")
    assert_close(from_dev(o_bf), RO, "zigzag O bf16")
    assert np.abs(lse_acc.cpu().numpy() - RL).max() <= LSE_MAX_ABS
    dq_acc = torch.zeros((2 * C, H, D), dtype=torch.float32, device="cuda")
    dks, dvs = [], []
    for s in range(spn):
        d = lib_desc(base, pos_q=pos_q, pos_k=kvpos[s])
        _, gk, gv = sp.sp_attn_bwd(d, dq, to_dev(ks[s]), to_dev(vs[s]), o_bf, lse_acc, to_dev(do),
                                   dq_acc=dq_acc)
        dks.append(from_dev(gk))
        dvs.append(from_dev(gv))
    RdQ, RdKs, RdVs = oracle.ring_backward(_dec(q), chunks, _dec(do), RO, RL, q_pos=pos_q,
                                           kv_pos=kvpos, **common)
    assert_close(dq_acc.cpu().numpy().astype(np.float64), RdQ, "zigzag dQ")
    for s in range(spn):
        assert_close(dks[s], RdKs[s], f"zigzag dK step {s}")
        assert_close(dvs[s], RdVs[s], f"zigzag dV step {s}")


@pytest.mark.parametrize("hs,hkv,D", [(6, 2, 128), (7, 7, 64)])
def test_usp_ring_groups(sp, hs, hkv, D):
    """USP (Ulysses inside zigzag-ring groups, Table 1) on a 2 x 2 mesh: every
    rank's share is assembled on the GPU by the Ulysses pack of each source
    rank's token slice (the all-to-all as slicing), the zigzag ring steps and
    their backward run through the C ABI, and the reverse unpack returns the
    layer's O and dQ.  Oracle: the all-rank USP simulation (its rank results,
    and the layer output, which equals attention without SP)."""
    import math
    import torch
    hp, cp, C = 2, 2, 96
    L = 2 * cp * C
    print(f"usp hs={hs} hkv={hkv} D={D} L={L}", flush=True)
    qb, kb, vb, db = (randn_bf16_bits((L, h, D), 91 + i)
                      for i, h in enumerate((hs, hkv, hkv, hs)))
    O, dQ, _, _, per = oracle.usp_simulate(_dec(qb), _dec(kb), _dec(vb), _dec(db), hp, cp,
                                           scale=1 / math.sqrt(D), gqa_group=hs // hkv)
    qmap = ulysses_q_head_map(hs, hp)
    kmap = qmap if hkv == hs else ulysses_kv_head_map(hs, hkv, hp)
    hloc, kvw, Tl = len(qmap) // hp, len(kmap) // hp, 2 * C // hp
    share = [np.r_[r * C + np.arange(C), (2 * cp - 1 - r) * C + np.arange(C)] for r in range(cp)]

    def exchange(bits, width, hmap, r):
        packs = [sp.sp_ulysses_pack(to_dev(bits[share[r][i * Tl:(i + 1) * Tl]]), hp, width, hmap)
                 for i in range(hp)]
        return [torch.cat([packs[i][j] for i in range(hp)]).contiguous() for j in range(hp)]

    Q, K, V, DO = ([exchange(b, w, m, r) for r in range(cp)]
                   for b, w, m in ((qb, hloc, qmap), (kb, kvw, kmap), (vb, kvw, kmap), (db, hloc, qmap)))
    for r in range(cp):
        outs, dqs = [], []
        for j in range(hp):
            sh = usp_shard("usp_test", L, hp, cp, r, j, D, hs, hkv, 0)
            assert sh.Hkv_loc == kvw and np.array_equal(sh.pos_q, share[r])
            nr, ref = sh.n_real_loc, per[(r, j)]
            steps = [(r - s) % cp for s in range(cp)]
            o_acc = torch.empty((2 * C, hloc, D), dtype=torch.float32, device="cuda")
            lse_acc = torch.empty((hloc, 2 * C), dtype=torch.float32, device="cuda")
            o_bf = torch.empty((2 * C, hloc, D), dtype=torch.bfloat16, device="cuda")
            for s, r2 in enumerate(steps):
                sp.sp_ring_step(lib_desc(sh, pos_k=share[r2]), Q[r][j], K[r2][j], V[r2][j], o_acc,
                                lse_acc, init=(s == 0), o_out=o_bf if s == cp - 1 else None)
            assert_close(from_dev(o_bf)[:, :nr], ref["o"][:, :nr], f"USP rank ({r},{j}) O")
            assert np.abs(lse_acc.cpu().numpy()[:nr] - ref["lse"][:nr]).max() <= LSE_MAX_ABS
            dq_acc = torch.zeros((2 * C, hloc, D), dtype=torch.float32, device="cuda")
            for s, r2 in enumerate(steps):
                _, gk, gv = sp.sp_attn_bwd(lib_desc(sh, pos_k=share[r2]), Q[r][j], K[r2][j],
                                           V[r2][j], o_bf, lse_acc, DO[r][j], dq_acc=dq_acc)
                # three query heads sum into a KV head: |dV| reaches 4-8
                assert_close(from_dev(gk), ref["dk"][s], f"USP rank ({r},{j}) dK step {s}",
                             max_abs=scaled_max_abs(ref["dk"][s]))
                assert_close(from_dev(gv), ref["dv"][s], f"USP rank ({r},{j}) dV step {s}",
                             max_abs=scaled_max_abs(ref["dv"][s]))
            assert_close(dq_acc.cpu().numpy().astype(np.float64)[:, :nr], ref["dq"][:, :nr],
                         f"USP rank ({r},{j}) dQ")
            dq_bf = torch.empty_like(o_bf)
            sp.sp_f32_to_bf16(dq_acc, dq_bf)
            outs.append(o_bf)
            dqs.append(dq_bf)
        for i in range(hp):  # reverse exchange: Ulysses rank i gets chunk i of every rank j
            rows = share[r][i * Tl:(i + 1) * Tl]
            for got, want, what in ((outs, O, "O"), (dqs, dQ, "dQ")):
                recv = torch.stack([got[j][i * Tl:(i + 1) * Tl] for j in range(hp)]).contiguous()
                assert_close(from_dev(sp.sp_ulysses_unpack(recv, qmap, hs)), want[rows],
                             f"USP layer {what} group {r} slice {i}")


def test_all_dummy_rank(sp):
    """A rank whose slots are all dummies (ranks 14-15 of 40 heads padded to
    48 for SP 16): nothing is computed, O / dQ are +0, LSE is -inf, the KV
    slot gets dK = dV = +0."""
    import torch
    sh = make_shard("all_dummy", 700, 700, 128, 3, 42, 40, 48, 5, 1, 0, [400, 300], seed_base=3)
    assert sh.n_real_loc == 0
    q, k, v, do = shard_inputs(sh)
    o, lse, gq, gk, gv = _run_fwd_bwd(sp, sh, q, k, v, do)
    for t in (o, gq, gk, gv):
        assert torch.all(t.view(torch.int16) == 0)
    assert bool(torch.all(torch.isneginf(lse)))


def test_empty_inputs(sp):
    """Zero query rows: a no-op forward and dK = dV = +0; zero keys: every row
    gets O = +0 and LSE = -inf, dQ = +0, and a first ring step leaves the
    accumulators at (0, -inf)."""
    import torch
    D, H = 128, 2
    e = lambda *shape: torch.empty(shape, dtype=torch.bfloat16, device="cuda")  # noqa: E731
    # no rows, 100 keys
    sh = make_shard("no_rows", 0, 100, D, H, 0, H, H, 1, H, 0, [0], [100])
    d = lib_desc(sh)
    k, v = to_dev(randn_bf16_bits((100, H, D), 1)), to_dev(randn_bf16_bits((100, H, D), 2))
    o, lse = sp.sp_attn_fwd(d, e(0, H, D), k, v)
    assert o.numel() == 0 and lse.numel() == 0
    dk, dv = torch.full_like(k, 1.0), torch.full_like(v, 1.0)
    sp.sp_attn_bwd(d, e(0, H, D), k, v, o, lse, e(0, H, D), dq=e(0, H, D), dk=dk, dv=dv)
    torch.cuda.synchronize()
    assert torch.all(dk.view(torch.int16) == 0) and torch.all(dv.view(torch.int16) == 0)
    # 50 rows, no keys
    sh = make_shard("no_keys", 50, 0, D, H, 0, H, H, 1, H, 0, [50], [0])
    d = lib_desc(sh)
    q, do = to_dev(randn_bf16_bits((50, H, D), 3)), to_dev(randn_bf16_bits((50, H, D), 4))
    o, lse = sp.sp_attn_fwd(d, q, e(0, H, D), e(0, H, D))
    torch.cuda.synchronize()
    assert torch.all(o.view(torch.int16) == 0) and bool(torch.all(torch.isneginf(lse)))
    dq, _, _ = sp.sp_attn_bwd(d, q, e(0, H, D), e(0, H, D), o, lse, do)
    torch.cuda.synchronize()
    assert torch.all(dq.view(torch.int16) == 0)
    o_acc = torch.full((50, H, D), 7.0, dtype=torch.float32, device="cuda")
    lse_acc = torch.full((H, 50), 7.0, dtype=torch.float32, device="cuda")
    sp.sp_ring_step(d, q, e(0, H, D), e(0, H, D), o_acc, lse_acc, init=True)
    torch.cuda.synchronize()
    assert torch.all(o_acc == 0) and bool(torch.all(torch.isneginf(lse_acc)))
