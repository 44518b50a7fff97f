"""GPU parity of the SP-aware loss path (Sections 3.3 and 5.1): token
log-probabilities, per-sequence sums, the SFT / DPO reduction over ranks and
the backward to the logits, through the C ABI, against the float64 oracle on
the same bf16 logits.

Bars (derived from the float32 arithmetic): lse and logp within 1e-4
absolute (a float32 log-sum-exp over up to 152064 terms); sequence sums
within 1e-3 + 1e-6 relative; the reduction's loss and gradients within 1e-5
relative; bf16 dlogits within rel-L2 5e-3 and two bf16 ulps of the largest
reference entry; rows that carry no gradient bit-zero."""
import math

import numpy as np
import pytest

import oracle
from tests.helpers import assert_close, bits_from_dev
from workloads import LOSS_WORKLOAD, bf16_bits_from_f32, loss_inputs, randn_bf16_bits

pytestmark = pytest.mark.gpu
LP_ABS = 1e-4


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _dev_bits(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _dec(bits):
    return oracle.bf16_bits_to_f64(bits)


@pytest.mark.parametrize("T,V", [(333, 1000), (40, 152064)])
def test_token_logprob_fwd_bwd(sp, T, V):
    import torch
    print(f"token logprob T={T} V={V}", flush=True)
    bits = randn_bf16_bits((T, V), 31 + V, scale=2.0)
    rng = np.random.default_rng(T)
    lab = rng.integers(0, V, T).astype(np.int32)
    lab[::7] = -100                 # prompt tokens
    lab[3] = V + 5                  # outside the vocabulary: not scored
    cu = np.array([5, T // 3, T - 4], dtype=np.int32)  # rows 0-4 and the last 4 outside
    X = _dev_bits(bits)
    L = torch.from_numpy(lab).cuda()
    logp, lse, ssum = sp.sp_token_logprob(X, L, cu)
    x = _dec(bits)
    lab_o = np.where((lab >= 0) & (lab < V), lab, -100)
    inside = np.zeros(T, bool)
    inside[cu[0]:cu[-1]] = True
    lab_o = np.where(inside, lab_o, -100)
    rlp, rlse = oracle.loss.token_logprobs(x, lab_o)
    assert np.abs(lse.cpu().numpy() - rlse).max() <= LP_ABS
    assert np.abs(logp.cpu().numpy() - rlp).max() <= LP_ABS
    assert np.all(logp.cpu().numpy()[lab_o == -100] == 0.0)
    rs = np.array([rlp[cu[s]:cu[s + 1]].sum() for s in range(len(cu) - 1)])
    assert np.allclose(ssum.cpu().numpy(), rs, atol=1e-3, rtol=1e-6)
    g = np.array([0.7, -1.3], dtype=np.float32)
    dl = sp.sp_token_logprob_bwd(X, L, lse, cu, torch.from_numpy(g).cuda())
    ref = oracle.loss.token_logprob_grad(x, lab_o, g.astype(np.float64), cu)
    got = dl.float().cpu().numpy().astype(np.float64)
    assert_close(got, ref, "dlogits", max_abs=2.0 ** -7 * np.abs(ref).max() + 1e-7)
    zero_rows = np.nonzero(lab_o == -100)[0]
    assert np.all(bits_from_dev(dl)[zero_rows] == 0)


@pytest.mark.parametrize("kind", ["sft", "dpo"])
def test_loss_reduce(sp, kind):
    import torch
    rng = np.random.default_rng(5)
    spn, n = 4, 6
    ps = (rng.standard_normal((spn, n)) * 40 - 300).astype(np.float32)
    rs = (rng.standard_normal((spn, n)) * 40 - 300).astype(np.float32)
    if kind == "sft":
        coef = 1.0 / 1234
        loss, grad = sp.sp_loss_reduce(torch.from_numpy(ps).cuda(), sp.SP_LOSS_SFT, coef)
        rl, rg = oracle.loss.sft_loss(ps.astype(np.float64), scale=coef, autograd=True)
    else:
        coef = 0.1
        loss, grad = sp.sp_loss_reduce(torch.from_numpy(ps).cuda(), sp.SP_LOSS_DPO, coef,
                                       ref_partial_sums=torch.from_numpy(rs).cuda())
        rl, rg = oracle.loss.dpo_loss(ps.astype(np.float64), rs.astype(np.float64), coef,
                                      autograd=True)
    assert abs(float(loss.cpu()[0]) - rl) <= 1e-5 * max(1.0, abs(rl))
    assert np.allclose(grad.cpu().numpy(), rg, rtol=1e-5, atol=1e-7)


def test_sp_loss_on_one_gpu(sp):
    """A DPO pair over sp = 4 simulated ranks on one GPU (sequential token
    slices): every rank's log-probs and sums, the reduction with the
    gradient-carrying all-reduce, every rank's backward.  With a shared
    linear head (logits = h W), the rank-averaged gradient of W equals the
    gradient without SP (Listing 2's finding), and the loss is the same."""
    import torch
    spn, Lr, d, V = 4, 96, 16, 512
    L = spn * Lr
    rng = np.random.default_rng(8)
    h = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V)) * 0.4
    bits = bf16_bits_from_f32((h @ W).astype(np.float32))
    rbits = bf16_bits_from_f32((h @ (W + 0.05 * rng.standard_normal((d, V)))).astype(np.float32))
    lab = rng.integers(0, V, L).astype(np.int32)
    lab[:20] = -100
    lab[L // 2:L // 2 + 20] = -100
    cu = np.array([0, L // 2, L], dtype=np.int32)
    beta = 0.2
    parts, refs, saved = [], [], []
    for r in range(spn):
        rows = slice(r * Lr, (r + 1) * Lr)
        cu_r = np.clip(cu - r * Lr, 0, Lr).astype(np.int32)
        X, R = _dev_bits(bits[rows]), _dev_bits(rbits[rows])
        Lb = torch.from_numpy(lab[rows].copy()).cuda()
        _, lse, s = sp.sp_token_logprob(X, Lb, cu_r)
        _, _, rs = sp.sp_token_logprob(R, Lb, cu_r)
        parts.append(s)
        refs.append(rs)
        saved.append((X, Lb, lse, cu_r, rows))
    loss, grad = sp.sp_loss_reduce(torch.stack(parts), sp.SP_LOSS_DPO, beta,
                                   ref_partial_sums=torch.stack(refs))
    dW = np.zeros_like(W)
    for r, (X, Lb, lse, cu_r, rows) in enumerate(saved):
        dl = sp.sp_token_logprob_bwd(X, Lb, lse, cu_r, grad[r].contiguous())
        dW += h[rows].T @ dl.float().cpu().numpy().astype(np.float64)
    dW /= spn
    # no SP: the oracle on the whole sequence, one rank
    x, xr = _dec(bits), _dec(rbits)
    lp, _ = oracle.loss.token_logprobs(x, lab)
    rlp, _ = oracle.loss.token_logprobs(xr, lab)
    rl, up = oracle.loss.dpo_loss(oracle.loss.sequence_sums(lp, cu)[None],
                                  oracle.loss.sequence_sums(rlp, cu)[None], beta)
    ref_dW = h.T @ oracle.loss.token_logprob_grad(x, lab, up[0], cu)
    assert abs(float(loss.cpu()[0]) - rl) <= 1e-4 * max(1.0, abs(rl))
    assert_close(dW, ref_dW, "dW (rank average)", max_abs=2.0 ** -6 * np.abs(ref_dW).max())


def test_loss_fullsize(sp):
    """The loss workload's shape (4096 tokens of the 7B-like rank, 152064
    vocabulary, a DPO pair): sampled rows against the oracle, the sums
    against the kernel's own per-token values."""
    import torch
    w = LOSS_WORKLOAD
    print(f"loss full size T={w['T']} V={w['V']}", flush=True)
    bits, lab, cu = loss_inputs(w["T"], w["V"], w["n_seqs"], w["seed"])
    X = _dev_bits(bits)
    L = torch.from_numpy(lab).cuda()
    logp, lse, ssum = sp.sp_token_logprob(X, L, cu)
    g = torch.tensor([-1.0 / 4096, 1.0 / 4096], dtype=torch.float32, device="cuda")
    dl = sp.sp_token_logprob_bwd(X, L, lse, cu, g)
    torch.cuda.synchronize()
    rows = np.array(sorted({0, 511, 512, 1500, 2047, 2048, 2600, 3000, 4095} |
                           set(np.random.default_rng(3).integers(0, w["T"], 6).tolist())))
    x = _dec(bits[rows])
    rlp, rlse = oracle.loss.token_logprobs(x, lab[rows])
    assert np.abs(lse.cpu().numpy()[rows] - rlse).max() <= LP_ABS
    assert np.abs(logp.cpu().numpy()[rows] - rlp).max() <= LP_ABS
    lp_all = logp.cpu().numpy().astype(np.float64)
    want = np.array([lp_all[cu[s]:cu[s + 1]].sum() for s in range(len(cu) - 1)])
    assert np.allclose(ssum.cpu().numpy(), want, rtol=1e-5)
    gs = g.cpu().numpy().astype(np.float64)
    seq = np.searchsorted(cu, rows, side="right") - 1
    ref = oracle.loss.token_logprob_grad(x, lab[rows], gs[seq], np.arange(len(rows) + 1))
    got = dl[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
    assert_close(got, ref, "dlogits rows", max_abs=2.0 ** -7 * np.abs(ref).max() + 1e-9)
