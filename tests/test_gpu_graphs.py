"""HIP graph capture through the C ABI.

The entry points that pass their host arrays by value in the kernel
arguments (Ulysses pack / unpack / summing unpack, the LSE merge, the
fp32 -> bf16 finalize and the loss path) are recorded into one graph and
replayed several times.  Between replays the program's own eager work
overwrites every output and resets the merge accumulators; each replay must
match the eager run bit for bit.  The attention entry points copy host-built
work lists on every call, so on a capturing stream they return
SP_ERR_UNSUPPORTED and enqueue nothing."""
import numpy as np
import pytest

from tests.helpers import lib_desc, make_shard
from workloads import randn_bf16_bits, shard_inputs, ulysses_kv_head_map, ulysses_q_head_map

pytestmark = pytest.mark.gpu

T_L, V_L = 64, 704          # loss path: tokens per rank, vocabulary
CU = np.array([2, 30, 61], dtype=np.int32)
T_M, H_M, D_M = 96, 3, 128  # merge


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _inputs():
    import torch
    rng = np.random.default_rng(4)
    lab = rng.integers(0, V_L, (2, T_L)).astype(np.int32)
    lab[:, ::3] = -100
    f32 = lambda shape: torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).cuda()
    return dict(
        xq=_bf16(randn_bf16_bits((96, 7, 64), 1)),
        recv=_bf16(randn_bf16_bits((8, 40, 2, 64), 2)),
        o_acc0=f32((T_M, H_M, D_M)), lse_acc0=f32((H_M, T_M)),
        o_part=_bf16(randn_bf16_bits((T_M, H_M, D_M), 3)), lse_part=f32((H_M, T_M)),
        f32src=f32((1000,)),
        logits=[_bf16(randn_bf16_bits((T_L, V_L), 10 + r, scale=2.0)) for r in range(2)],
        rlogits=[_bf16(randn_bf16_bits((T_L, V_L), 20 + r, scale=2.0)) for r in range(2)],
        labels=[torch.from_numpy(lab[r].copy()).cuda() for r in range(2)],
    )


def _outputs():
    import torch
    bf, f = torch.bfloat16, torch.float32
    e = lambda shape, dt: torch.empty(shape, dtype=dt, device="cuda")
    return dict(packed=e((2, 96, 4, 64), bf), unpacked=e((96, 7, 64), bf),
                ua=e((40, 4, 64), bf), o_acc=e((T_M, H_M, D_M), f), lse_acc=e((H_M, T_M), f),
                o_fin=e((T_M, H_M, D_M), bf), cvt=e((1000,), bf),
                logp=e((2, T_L), f), lse=e((2, T_L), f), rlogp=e((2, T_L), f),
                rlse=e((2, T_L), f), parts=e((2, 2), f), rparts=e((2, 2), f),
                loss=e((1,), f), grad=e((2, 2), f), dl=e((T_L, V_L), bf))


def _reset(x, out):
    """Eager: garbage into every output, the merge accumulators restored."""
    for k, t in out.items():
        t.fill_(7.0 if t.is_floating_point() else 7)
    out["o_acc"].copy_(x["o_acc0"])
    out["lse_acc"].copy_(x["lse_acc0"])


def _steps(sp, x, out):
    """Every by-value entry point, writing into the preallocated outputs."""
    hm = ulysses_q_head_map(7, 2)
    sp.sp_ulysses_pack(x["xq"], 2, 4, hm, dst=out["packed"])
    sp.sp_ulysses_unpack(out["packed"], hm, 7, dst=out["unpacked"])
    sp.sp_ulysses_unpack_add(x["recv"], ulysses_kv_head_map(28, 4, 8), 4, dst=out["ua"])
    sp.sp_lse_merge(out["o_acc"], out["lse_acc"], x["o_part"], x["lse_part"], o_out=out["o_fin"])
    sp.sp_f32_to_bf16(x["f32src"], dst=out["cvt"])
    for r in range(2):
        sp.sp_token_logprob(x["logits"][r], x["labels"][r], CU, logp=out["logp"][r],
                            lse=out["lse"][r], seq_sum=out["parts"][r])
        sp.sp_token_logprob(x["rlogits"][r], x["labels"][r], CU, logp=out["rlogp"][r],
                            lse=out["rlse"][r], seq_sum=out["rparts"][r])
    sp.sp_loss_reduce(out["parts"], sp.SP_LOSS_DPO, 0.1, ref_partial_sums=out["rparts"],
                      loss=out["loss"], grad=out["grad"])
    sp.sp_token_logprob_bwd(x["logits"][0], x["labels"][0], out["lse"][0], CU, out["grad"][0],
                            dlogits=out["dl"])


def _bits(t):
    import torch
    t = t.detach().contiguous().cpu()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def test_by_value_entry_points_replay_in_a_graph(sp):
    import torch
    x, out = _inputs(), _outputs()
    _reset(x, out)
    _steps(sp, x, out)
    torch.cuda.synchronize()
    ref = {k: _bits(t) for k, t in out.items()}

    g = torch.cuda.CUDAGraph()
    _reset(x, out)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        _steps(sp, x, out)
    torch.cuda.synchronize()
    for rep in range(3):
        _reset(x, out)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, r in ref.items():
            assert np.array_equal(_bits(out[k]), r), f"replay {rep}: {k} differs from eager"


def test_attention_refuses_a_capturing_stream(sp):
    import torch
    sh = make_shard("graph_refusal", 200, 200, 64, 2, 0, 2, 2, 1, 2, 0, [200], seed_base=3)
    q, k, v, do = (_bf16(a) for a in shard_inputs(sh))
    d = lib_desc(sh)
    o = torch.full((200, 2, 64), 3.0, dtype=torch.bfloat16, device="cuda")
    lse = torch.full((2, 200), 3.0, dtype=torch.float32, device="cuda")
    o_acc = torch.full((200, 2, 64), 3.0, dtype=torch.float32, device="cuda")
    dk = torch.full((200, 2, 64), 3.0, dtype=torch.bfloat16, device="cuda")
    dv, dq = dk.clone(), o.clone()
    ws = torch.empty(max(sp.sp_attn_workspace_size(d, op) for op in
                         (sp.SP_OP_FWD, sp.SP_OP_BWD, sp.SP_OP_RING_STEP)),
                     dtype=torch.uint8, device="cuda")
    marker = torch.zeros(1, device="cuda")
    torch.cuda.synchronize()
    statuses = []
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        marker.add_(1.0)
        calls = [
            lambda: sp.sp_attn_fwd(d, q, k, v, o=o, lse=lse, workspace=ws),
            lambda: sp.sp_ring_step(d, q, k, v, o_acc, lse, init=True, workspace=ws),
            lambda: sp.sp_attn_bwd(d, q, k, v, o, lse, do, dq=dq, dk=dk, dv=dv, workspace=ws),
        ]
        for call in calls:
            try:
                call()
                statuses.append(sp.SP_OK)
            except sp.SpError as e:
                statuses.append(e.status)
    assert statuses == [sp.SP_ERR_UNSUPPORTED] * 3
    g.replay()
    torch.cuda.synchronize()
    assert float(marker.cpu()[0]) == 1.0
    for t in (o, lse, o_acc, dq, dk, dv):
        assert bool((t.float() == 3.0).all()), "a refused call wrote an output"
    # the same calls outside capture run normally
    sp.sp_attn_fwd(d, q, k, v, o=o, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    assert not bool((o.float() == 3.0).all())
