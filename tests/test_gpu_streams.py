"""Every entry point runs on the stream it is given.

The whole hot path (Ulysses pack / unpack / summing unpack, attention
forward and backward, a ring step with the LSE merge and the fp32 -> bf16
finalize, the loss path) is run twice: on the default stream, and on a side
stream whose queue starts with a long spin, after which the inputs are
written on that stream.  A kernel or copy issued anywhere else would run
before the writes and read the zeros the inputs held; since every kernel is
deterministic, the two runs must agree bit for bit."""
import numpy as np
import pytest

from tests.helpers import lib_desc, make_shard
from workloads import randn_bf16_bits, shard_inputs, ulysses_kv_head_map, ulysses_q_head_map

pytestmark = pytest.mark.gpu


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


def _sources():
    """Device input tensors of one small instance of every step."""
    import torch
    sh = make_shard("streams_varlen_gqa", 300, 300, 128, 4, 0, 4, 4, 2, 2, 0, [120, 0, 150],
                    seed_base=5)
    q, k, v, do = shard_inputs(sh)
    rng = np.random.default_rng(9)
    T, V = 64, 704  # V: a multiple of 8
    lab = rng.integers(0, V, T).astype(np.int32)
    lab[::4] = -100
    src = dict(q=_bf16(q), k=_bf16(k), v=_bf16(v), do=_bf16(do),
               xq=_bf16(randn_bf16_bits((96, 7, 64), 1)),
               recv=_bf16(randn_bf16_bits((8, 40, 2, 64), 2)),
               ck=_bf16(randn_bf16_bits((300, 2, 128), 3)),
               cv=_bf16(randn_bf16_bits((300, 2, 128), 4)),
               logits=_bf16(randn_bf16_bits((T, V), 6, scale=2.0)),
               labels=torch.from_numpy(lab).cuda())
    return sh, src


def _path(sp, sh, x):
    """Run every step on the current stream; returns the outputs."""
    import torch
    out = {}
    hm = ulysses_q_head_map(7, 2)
    packed = sp.sp_ulysses_pack(x["xq"], 2, 4, hm)
    out["pack"] = packed
    out["unpack"] = sp.sp_ulysses_unpack(packed, hm, 7)
    out["unpack_add"] = sp.sp_ulysses_unpack_add(x["recv"], ulysses_kv_head_map(28, 4, 8), 4)
    d = lib_desc(sh)
    o, lse = sp.sp_attn_fwd(d, x["q"], x["k"], x["v"])
    gq, gk, gv = sp.sp_attn_bwd(d, x["q"], x["k"], x["v"], o, lse, x["do"])
    out.update(o=o, lse=lse, gq=gq, gk=gk, gv=gv)
    # a second KV chunk as a ring step onto (O, LSE), then merge a copy back
    o_acc = o.float()
    lse_acc = lse.clone()
    sp.sp_ring_step(d, x["q"], x["ck"], x["cv"], o_acc, lse_acc, init=False)
    o_fin = sp.sp_f32_to_bf16(o_acc)
    o_m, l_m = o_acc.clone(), lse_acc.clone()
    sp.sp_lse_merge(o_m, l_m, o, lse)
    out.update(o_acc=o_acc, lse_acc=lse_acc, o_fin=o_fin, o_m=o_m, l_m=l_m)
    cu = np.array([3, 30, 60], dtype=np.int32)
    logp, lse_t, ssum = sp.sp_token_logprob(x["logits"], x["labels"], cu)
    loss, grad = sp.sp_loss_reduce(torch.stack([ssum, ssum * 0.5]), sp.SP_LOSS_DPO, 0.1,
                                   ref_partial_sums=torch.stack([ssum * 0.9, ssum * 0.4]))
    dl = sp.sp_token_logprob_bwd(x["logits"], x["labels"], lse_t, cu, grad[0].contiguous())
    out.update(logp=logp, lse_t=lse_t, ssum=ssum, loss=loss, grad=grad, dl=dl)
    return out


def _bits(t):
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy()
    if t.dtype == torch.float32:
        return t.view(torch.int32).numpy()
    return t.numpy()


def test_side_stream_runs_after_its_own_queue(sp):
    import torch
    sh, src = _sources()
    ref = {k: _bits(v) for k, v in _path(sp, sh, src).items()}
    torch.cuda.synchronize()
    work = {k: torch.zeros_like(v) for k, v in src.items()}
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        torch.cuda._sleep(50_000_000)  # tens of milliseconds of spinning on s
        for k, v in src.items():
            work[k].copy_(v)
        got = _path(sp, sh, work)
    s.synchronize()
    torch.cuda.synchronize()
    for k, r in ref.items():
        g = _bits(got[k])
        assert g.shape == r.shape and np.array_equal(g, r), f"{k} differs on the side stream"


def test_concurrent_host_threads(sp):
    """Two host threads run the whole path at once, each on its own stream
    (the library holds no shared mutable state: schedules and uploads are
    per call, the optional kernel timers per thread).  Each thread's outputs
    match the single-threaded run bit for bit."""
    import threading
    import torch
    sh, src = _sources()
    ref = {k: _bits(v) for k, v in _path(sp, sh, src).items()}
    torch.cuda.synchronize()
    results, errors = [None, None], []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                outs = [_path(sp, sh, src) for _ in range(3)]
            s.synchronize()
            results[i] = [{k: _bits(v) for k, v in o.items()} for o in outs]
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    for i in range(2):
        assert results[i] is not None, f"thread {i} did not finish"
        for o in results[i]:
            for k, r in ref.items():
                assert np.array_equal(o[k], r), f"{k} differs in thread {i}"


def test_explicit_stream_argument_keeps_its_buffers(sp):
    """stream= given while the current stream is the default one: the
    wrapper's own outputs and workspaces belong to the launch stream, so
    memory the default stream allocates and overwrites while the launch
    stream is still queued behind a spin is never theirs.  The results
    match the default-stream run bit for bit."""
    import torch
    sh, src = _sources()
    d = lib_desc(sh)
    o_r, lse_r = sp.sp_attn_fwd(d, src["q"], src["k"], src["v"])
    g_r = sp.sp_attn_bwd(d, src["q"], src["k"], src["v"], o_r, lse_r, src["do"])
    ref = [_bits(t) for t in (o_r, lse_r, *g_r)]
    torch.cuda.synchronize()
    sizes = [sp.sp_attn_workspace_size(d, sp.SP_OP_FWD), sp.sp_attn_workspace_size(d, sp.SP_OP_BWD),
             o_r.numel() * 2, lse_r.numel() * 4]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        torch.cuda._sleep(50_000_000)  # the launch stream waits tens of milliseconds
    o, lse = sp.sp_attn_fwd(d, src["q"], src["k"], src["v"], stream=s)
    g = sp.sp_attn_bwd(d, src["q"], src["k"], src["v"], o, lse, src["do"], stream=s)
    # meanwhile the default stream allocates blocks of the same sizes and
    # overwrites them
    junk = [torch.full((n,), 255, dtype=torch.uint8, device="cuda") for n in sizes for _ in range(2)]
    s.synchronize()
    torch.cuda.synchronize()
    del junk
    for name, a, r in zip(("o", "lse", "dq", "dk", "dv"), (o, lse, *g), ref):
        assert np.array_equal(_bits(a), r), f"{name} differs with stream= given"
