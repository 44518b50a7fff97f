"""GPU parity at the benchmark's full shard sizes, in the launch configuration
bench.py times (same entry points, same tile schedule).

The oracle evaluates sampled outputs one by one: O and LSE for sampled query
rows, dQ for sampled rows, dK/dV for sampled keys near segment ends (only
rows after them see those keys) and for "deep" keys that ~15-16K rows see
(the dK/dV kernel's longest accumulation: hundreds of query chunks summed in
float32, each chunk's P exchanged as fp16).  For a deep key the oracle
needs the full softmax row of every row that sees it, so it runs on the
exact sub-problem that holds the key -- its segment (segments are
independent), or one KV head's group of query heads (GQA groups are).  Over
the whole arrays, properties that hold at any size are checked: per segment
and KV head sum_j dK_j = 0 and sum_j dV_j = sum over the group's rows of
dO_i (rows of P sum to one), and dummy slots are bit-zero."""
import numpy as np
import pytest

import oracle
from tests.helpers import (LSE_MAX_ABS, assert_close, bits_from_dev, from_dev, lib_desc, oracle_kw,
                           to_dev)
from workloads import (ring_chunk_positions, shard_inputs, workload, WORKLOADS, zigzag_inputs,
                       zigzag_step_positions)

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(420)]


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _sample_rows(sh, n_rand=24, seed=0):
    rng = np.random.default_rng(seed)
    rows = set()
    for s in range(len(sh.cu_q) - 1):
        a, b = int(sh.cu_q[s]), int(sh.cu_q[s + 1])
        if b > a:
            rows.update([a, min(a + 1, b - 1), (a + b) // 2, b - 1])
    rows.update(rng.integers(0, sh.T_q, size=n_rand).tolist())
    return np.array(sorted(rows))


def _tail_keys(sh, per_seg=4):
    keys = []
    for s in range(len(sh.cu_k) - 1):
        a, b = int(sh.cu_k[s]), int(sh.cu_k[s + 1])
        if b - a >= 8:
            keys += [b - 1, b - 3, b - 40 if b - 40 >= a else a, b - 130 if b - 130 >= a else a][:per_seg]
    return np.array(sorted(set(keys)))


def _deep_keys_check(sh, kw, qf, kf, vf, dof, gk, gv, nr, keys, seg):
    """dK / dV of `keys` (all in segment `seg`, seen by many rows) against
    the oracle on that segment alone (its rows, keys and positions)."""
    import time
    qa, qb = int(sh.cu_q[seg]), int(sh.cu_q[seg + 1])
    ka, kb = int(sh.cu_k[seg]), int(sh.cu_k[seg + 1])
    sub = dict(kw, cu_q=np.array([0, qb - qa]), cu_k=np.array([0, kb - ka]),
               pos_q=np.asarray(kw["pos_q"])[qa:qb], pos_k=np.asarray(kw["pos_k"])[ka:kb])
    t0 = time.perf_counter()
    RdK, RdV = oracle.attn_dkdv_keys(qf[qa:qb], kf[ka:kb], vf[ka:kb], dof[qa:qb], keys - ka, **sub)
    seen = [int(((np.asarray(kw["pos_k"])[k] <= sub["pos_q"]) if kw["causal"] else
                 np.ones(qb - qa, bool)).sum()) for k in keys]
    print(f"deep keys {keys.tolist()} seen by {seen} rows; oracle {time.perf_counter() - t0:.1f} s",
          flush=True)
    used = sorted({sh.kv_of(h) for h in range(nr)})
    assert_close(from_dev(gk[keys])[:, used], RdK[:, used], "dK deep keys")
    assert_close(from_dev(gv[keys])[:, used], RdV[:, used], "dV deep keys")


def _deep_keys(sh):
    """Two keys of the longest segment, at a quarter and half of it (causal:
    the rows after them, ~3/4 and ~1/2 of the segment, see them), and the
    segment's index."""
    lens = np.diff(sh.cu_k)
    seg = int(np.argmax(lens))
    a, n = int(sh.cu_k[seg]), int(lens[seg])
    return np.array([a + n // 4 + 3, a + n // 2 + 1]), seg


def _grad_sums(sh, dk, dv, do, nr):
    """Whole-array gradient identities per segment and KV head."""
    for s in range(len(sh.cu_k) - 1):
        a, b = int(sh.cu_k[s]), int(sh.cu_k[s + 1])
        qa, qb = int(sh.cu_q[s]), int(sh.cu_q[s + 1])
        if b <= a or qb <= qa:
            continue
        for kv in range(sh.Hkv_loc):
            heads = [h for h in range(nr) if sh.kv_of(h) == kv]
            if not heads:
                continue
            sk = dk[a:b, kv].sum(axis=0)
            nk = np.sqrt((dk[a:b, kv] ** 2).sum())
            assert np.abs(sk).max() <= 2e-2 * max(nk, 1e-6), ("sum dK", s, kv)
            want = do[qa:qb][:, heads].sum(axis=(0, 1))
            got = dv[a:b, kv].sum(axis=0)
            assert np.abs(got - want).max() <= 1e-2 * max(1.0, np.abs(want).max()), ("sum dV", s, kv)


@pytest.mark.parametrize("name", [w for w in WORKLOADS if not w.startswith(("ring", "zigzag", "usp"))])
def test_fullsize_shard(sp, name):
    import torch
    sh = workload(name)
    print(f"full-size {name}: T={sh.T_q} H_loc={sh.H_loc} real={sh.n_real_loc}", flush=True)
    q, k, v, do = shard_inputs(sh)
    d = lib_desc(sh)
    Q, K, V, dO = (to_dev(x) for x in (q, k, v, do))
    o, lse = sp.sp_attn_fwd(d, Q, K, V)
    gq, gk, gv = sp.sp_attn_bwd(d, Q, K, V, o, lse, dO)
    torch.cuda.synchronize()
    nr = sh.n_real_loc
    qf, kf, vf, dof = (oracle.bf16_bits_to_f64(x) for x in (q, k, v, do))
    kw = oracle_kw(sh)
    rows = _sample_rows(sh)
    RO, RL = oracle.attn_forward(qf, kf, vf, rows=rows, **kw)
    GO = from_dev(o[torch.from_numpy(rows).cuda()])
    assert_close(GO[:, :nr], RO[:, :nr], "O rows")
    GL = lse.cpu().numpy()[:, rows].astype(np.float64)
    assert np.abs(GL[:nr] - RL[:nr]).max() <= LSE_MAX_ABS
    rq = rows[::2]
    RdQ, _, _ = oracle.attn_dq_rows(qf, kf, vf, dof, rq, **kw)
    assert_close(from_dev(gq[torch.from_numpy(rq).cuda()])[:, :nr], RdQ[:, :nr], "dQ rows")
    keys = _tail_keys(sh)
    RdK, RdV = oracle.attn_dkdv_keys(qf, kf, vf, dof, keys, **kw)
    kidx = torch.from_numpy(keys).cuda()
    used = sorted({sh.kv_of(h) for h in range(nr)})
    assert_close(from_dev(gk[kidx])[:, used], RdK[:, used], "dK keys")
    assert_close(from_dev(gv[kidx])[:, used], RdV[:, used], "dV keys")
    if sh.T_q >= 16384:
        dkeys, seg = _deep_keys(sh)
        _deep_keys_check(sh, kw, qf, kf, vf, dof, gk, gv, nr, dkeys, seg)
    _grad_sums(sh, from_dev(gk), from_dev(gv), dof, nr)
    if nr < sh.H_loc:
        assert torch.all(o[:, nr:].view(torch.int16) == 0)
        assert torch.all(gq[:, nr:].view(torch.int16) == 0)
        assert bool(torch.all(torch.isneginf(lse[nr:])))


def test_fullsize_ring_rank(sp):
    """Ring rank 4 of 8 (Q chunk of 16384 against KV chunks 0..4, 28 query /
    4 KV heads): fused ring steps, then per-chunk backward into an fp32 dQ
    accumulator.  The oracle is monolithic attention over the concatenated
    chunks (the ring fold equals it exactly)."""
    import torch
    sh = [workload(w) for w in WORKLOADS if w.startswith("ring")][0]
    n, C, H, D = sh.ring_chunks, sh.chunk, sh.H_loc, sh.D
    q, _, _, do = shard_inputs(sh, chunk=0)
    ks, vs = [], []
    for c in range(n):
        _, k, v, _ = shard_inputs(sh, chunk=c)
        ks.append(k)
        vs.append(v)
    Q, dO = to_dev(q), to_dev(do)
    Ks, Vs = [to_dev(x) for x in ks], [to_dev(x) for x in vs]
    o_acc = torch.empty((C, H, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((H, C), dtype=torch.float32, device="cuda")
    o = torch.empty((C, H, D), dtype=torch.bfloat16, device="cuda")
    descs = [lib_desc(sh, pos_k=ring_chunk_positions(sh, c)) for c in range(n)]
    for c in range(n):
        sp.sp_ring_step(descs[c], Q, Ks[c], Vs[c], o_acc, lse, init=(c == 0),
                        o_out=o if c == n - 1 else None)
    # the benchmark's flow: one workspace (the row statistics formed by chunk
    # 0's call are reused), the dQ accumulator started by chunk 0 (its NaN
    # start never read) and turned into bf16 dQ by the last chunk
    dq_acc = torch.full((C, H, D), float("nan"), dtype=torch.float32, device="cuda")
    dq = torch.empty((C, H, D), dtype=torch.bfloat16, device="cuda")
    dks, dvs = [], []
    descs_b = [lib_desc(sh, pos_k=ring_chunk_positions(sh, c), rowstats_ready=c > 0,
                        dq_acc_init=c == 0) for c in range(n)]
    ws = torch.empty(max(sp.sp_attn_workspace_size(d, sp.SP_OP_BWD) for d in descs_b),
                     dtype=torch.uint8, device="cuda")
    for c in range(n):
        _, gk, gv = sp.sp_attn_bwd(descs_b[c], Q, Ks[c], Vs[c], o, lse, dO,
                                   dq=dq if c == n - 1 else None, dq_acc=dq_acc, workspace=ws)
        dks.append(gk)
        dvs.append(gv)
    torch.cuda.synchronize()
    # monolithic oracle over the concatenated keys
    kcat = oracle.bf16_bits_to_f64(np.concatenate(ks))
    vcat = oracle.bf16_bits_to_f64(np.concatenate(vs))
    qf, dof = oracle.bf16_bits_to_f64(q), oracle.bf16_bits_to_f64(do)
    kw = dict(cu_q=np.array([0, C]), cu_k=np.array([0, n * C]), pos_q=sh.pos_q,
              pos_k=np.arange(n * C), H_loc=H, head_offset=0, num_real_heads=H,
              gqa_group=sh.gqa_group, kv_head_offset=0, scale=sh.scale, causal=True)
    rows = np.array(sorted({0, 1, C // 2, C - 1} | set(np.random.default_rng(1).integers(0, C, 12).tolist())))
    RO, RL = oracle.attn_forward(qf, kcat, vcat, rows=rows, **kw)
    ridx = torch.from_numpy(rows).cuda()
    assert_close(from_dev(o[ridx]), RO, "ring O rows")
    assert_close(o_acc[ridx].cpu().numpy().astype(np.float64), RO, "ring O acc rows")
    assert np.abs(lse[:, ridx].cpu().numpy() - RL).max() <= LSE_MAX_ABS
    RdQ, _, _ = oracle.attn_dq_rows(qf, kcat, vcat, dof, rows[::2], **kw)
    assert_close(from_dev(dq[torch.from_numpy(rows[::2]).cuda()]), RdQ, "ring dQ rows")
    # keys near the end of the diagonal chunk: few rows see them
    keys = np.array([n * C - 1, n * C - 5, n * C - 70])
    RdK, RdV = oracle.attn_dkdv_keys(qf, kcat, vcat, dof, keys, **kw)
    kl = torch.from_numpy(keys - (n - 1) * C).cuda()
    assert_close(from_dev(dks[-1][kl]), RdK, "ring dK keys")
    assert_close(from_dev(dvs[-1][kl]), RdV, "ring dV keys")
    # deep keys: two keys of KV chunk 0, which all 16384 rows see (every row
    # accumulates the whole chunk); the oracle on KV head 0's group of query
    # heads (GQA groups are independent)
    import time
    g = sh.gqa_group
    grp = dict(kw, H_loc=g, num_real_heads=g)
    deep = np.array([100, C // 2 + 7])
    t0 = time.perf_counter()
    RdK0, RdV0 = oracle.attn_dkdv_keys(qf[:, :g], kcat[:, :1], vcat[:, :1], dof[:, :g], deep, **grp)
    print(f"ring deep keys {deep.tolist()} (KV head 0, heads 0-{g - 1}, all {C} rows); "
          f"oracle {time.perf_counter() - t0:.1f} s", flush=True)
    kd = torch.from_numpy(deep).cuda()
    assert_close(from_dev(dks[0][kd])[:, :1], RdK0, "ring dK deep keys")
    assert_close(from_dev(dvs[0][kd])[:, :1], RdV0, "ring dV deep keys")
    # whole-array identities over all chunks
    dk_all = np.concatenate([from_dev(x) for x in dks])
    dv_all = np.concatenate([from_dev(x) for x in dvs])
    for kv in range(sh.Hkv_loc):
        heads = [h for h in range(H) if sh.kv_of(h) == kv]
        assert np.abs(dk_all[:, kv].sum(axis=0)).max() <= 2e-2 * np.sqrt((dk_all[:, kv] ** 2).sum())
        want = dof[:, heads].sum(axis=(0, 1))
        assert np.abs(dv_all[:, kv].sum(axis=0) - want).max() <= 1e-2 * max(1.0, np.abs(want).max())


@pytest.mark.parametrize("name", [w for w in WORKLOADS if w.startswith(("zigzag", "usp"))])
def test_fullsize_zigzag_rank(sp, name):
    """Zigzag ring rank 4 of 8 (Section 3.2; chunks 4 and 11 of 16, 8192
    tokens each, 28 query / 4 KV heads), and the USP rank (ring rank 1 of 2,
    Ulysses rank 2 of 4: chunks 1 and 2 of 4, 32768 tokens each, query heads
    14-20 on KV head 2): ring steps over pieces of one sequence with the
    fused merge, then per-step backward into an fp32 dQ accumulator.
    Oracle: monolithic attention over the keys of all steps (positions decide
    visibility), on sampled rows and keys; whole-array gradient identities
    over all steps."""
    import torch
    sh = workload(name)
    print(f"full-size {name}: T={sh.T_q} H_loc={sh.H_loc} steps={sh.ring_chunks}", flush=True)
    n, T, H, D = sh.ring_chunks, sh.T_q, sh.H_loc, sh.D
    q, do = zigzag_inputs(sh)
    kvs = [zigzag_inputs(sh, s) for s in range(n)]
    pks = [zigzag_step_positions(sh, s) for s in range(n)]
    Q, dO = to_dev(q), to_dev(do)
    Ks, Vs = [to_dev(k) for k, _ in kvs], [to_dev(v) for _, v in kvs]
    o_acc = torch.empty((T, H, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((H, T), dtype=torch.float32, device="cuda")
    o = torch.empty((T, H, D), dtype=torch.bfloat16, device="cuda")
    descs = [lib_desc(sh, pos_k=pks[s]) for s in range(n)]
    for s in range(n):
        sp.sp_ring_step(descs[s], Q, Ks[s], Vs[s], o_acc, lse, init=(s == 0),
                        o_out=o if s == n - 1 else None)
    dq_acc = torch.full((T, H, D), float("nan"), dtype=torch.float32, device="cuda")
    dq = torch.empty((T, H, D), dtype=torch.bfloat16, device="cuda")
    dks, dvs = [], []
    descs_b = [lib_desc(sh, pos_k=pks[s], rowstats_ready=s > 0, dq_acc_init=s == 0)
               for s in range(n)]
    ws = torch.empty(max(sp.sp_attn_workspace_size(d, sp.SP_OP_BWD) for d in descs_b),
                     dtype=torch.uint8, device="cuda")
    for s in range(n):
        _, gk, gv = sp.sp_attn_bwd(descs_b[s], Q, Ks[s], Vs[s], o, lse, dO,
                                   dq=dq if s == n - 1 else None, dq_acc=dq_acc, workspace=ws)
        dks.append(gk)
        dvs.append(gv)
    torch.cuda.synchronize()
    kcat = oracle.bf16_bits_to_f64(np.concatenate([k for k, _ in kvs]))
    vcat = oracle.bf16_bits_to_f64(np.concatenate([v for _, v in kvs]))
    pcat = np.concatenate(pks)
    qf, dof = oracle.bf16_bits_to_f64(q), oracle.bf16_bits_to_f64(do)
    kw = dict(cu_q=np.array([0, T]), cu_k=np.array([0, n * T]), pos_q=sh.pos_q, pos_k=pcat,
              H_loc=H, head_offset=sh.head_offset, num_real_heads=sh.num_real_heads,
              gqa_group=sh.gqa_group, kv_head_offset=sh.kv_head_offset, scale=sh.scale,
              causal=True)
    C = sh.chunk
    rows = np.array(sorted({0, 1, C - 1, C, C + 1, T - 1} |
                           set(np.random.default_rng(2).integers(0, T, 10).tolist())))
    RO, RL = oracle.attn_forward(qf, kcat, vcat, rows=rows, **kw)
    ridx = torch.from_numpy(rows).cuda()
    assert_close(from_dev(o[ridx]), RO, "zigzag O rows")
    assert np.abs(lse[:, ridx].cpu().numpy() - RL).max() <= LSE_MAX_ABS
    RdQ, _, _ = oracle.attn_dq_rows(qf, kcat, vcat, dof, rows[::2], **kw)
    assert_close(from_dev(dq[torch.from_numpy(rows[::2]).cuda()]), RdQ, "zigzag dQ rows")
    # keys at the end of the rank's own second chunk (step 0): only the last
    # rows see them, so the oracle evaluates few rows
    loc = np.array([2 * C - 1, 2 * C - 3, 2 * C - 40])
    RdK, RdV = oracle.attn_dkdv_keys(qf, kcat, vcat, dof, loc, **kw)
    kl = torch.from_numpy(loc).cuda()
    assert_close(from_dev(dks[0][kl]), RdK, "zigzag dK keys")
    assert_close(from_dev(dvs[0][kl]), RdV, "zigzag dV keys")
    dk_all = np.concatenate([from_dev(x) for x in dks])
    dv_all = np.concatenate([from_dev(x) for x in dvs])
    for kv in range(sh.Hkv_loc):
        heads = [h for h in range(H) if sh.kv_of(h) == kv]
        assert np.abs(dk_all[:, kv].sum(axis=0)).max() <= 2e-2 * np.sqrt((dk_all[:, kv] ** 2).sum())
        want = dof[:, heads].sum(axis=(0, 1))
        assert np.abs(dv_all[:, kv].sum(axis=0) - want).max() <= 1e-2 * max(1.0, np.abs(want).max())
