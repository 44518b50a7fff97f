"""SP-aware loss reduction (CPU oracle, float64).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this.

Section 3.3 (Correct Loss Calculation) and Section 5.1 (Distributed
Communication Problem, Listing 2):

  * each rank holds a slice of the sequence, so it can only form the
    log-probabilities of its own tokens: log p(x_i) = logit[label] -
    logsumexp(logits), summed per sequence;
  * SFT (Eq. 1): the loss is minus the sum over all tokens, i.e. the sum of
    the ranks' partial sums (an all-reduce);
  * DPO (Eq. 2): the sigmoid is not linear, so the four sequence
    log-probabilities (policy / reference, chosen / rejected) are all-reduced
    first and the loss is formed from the totals.  The printed equation drops
    the log on the rejected ratio; the reading here is the standard form
    beta * [(log pi(y_w) - log ref(y_w)) - (log pi(y_l) - log ref(y_l))];
  * the all-reduce must carry gradients (torch.distributed.nn.all_reduce):
    its backward all-reduces the upstream gradient, so every rank's partial
    receives the sum over ranks of the (identical) upstream gradient, sp
    times the local value.  A plain all-reduce leaves the local upstream,
    and gradients come out sp times too small once averaged over the ranks.
"""
from __future__ import annotations

import numpy as np


def token_logprobs(logits, labels, ignore_index=-100):
    """logits [T, V] (float), labels [T] -> (logp [T], lse [T]).  logp is
    logit[label] - logsumexp over the vocabulary; tokens whose label is
    ignore_index get logp = 0 (they are not part of the loss)."""
    x = np.asarray(logits, dtype=np.float64)
    m = x.max(axis=1)
    lse = m + np.log(np.exp(x - m[:, None]).sum(axis=1))
    lab = np.asarray(labels, dtype=np.int64)
    ok = lab != ignore_index
    logp = np.zeros(x.shape[0])
    idx = np.nonzero(ok)[0]
    logp[idx] = x[idx, lab[idx]] - lse[idx]
    return logp, lse


def sequence_sums(logp, cu_seqlens):
    """Sum of the token log-probabilities of each sequence [cu[s], cu[s+1])."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    return np.array([logp[cu[s]:cu[s + 1]].sum() for s in range(len(cu) - 1)])


def token_logprob_grad(logits, labels, grad_seq, cu_seqlens, ignore_index=-100):
    """Gradient of sum_s grad_seq[s] * (sum of logp over sequence s) w.r.t.
    the logits: for a token t of sequence s with a label,
    g * (onehot(label) - softmax(logits[t])), with g = grad_seq[s]; tokens
    without a label or outside every sequence get 0."""
    x = np.asarray(logits, dtype=np.float64)
    T = x.shape[0]
    m = x.max(axis=1)
    p = np.exp(x - m[:, None])
    p /= p.sum(axis=1, keepdims=True)
    g = np.zeros(T)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    for s in range(len(cu) - 1):
        g[cu[s]:cu[s + 1]] = grad_seq[s]
    lab = np.asarray(labels, dtype=np.int64)
    g[lab == ignore_index] = 0.0
    onehot = np.zeros_like(x)
    idx = np.nonzero(lab != ignore_index)[0]
    onehot[idx, lab[idx]] = 1.0
    return g[:, None] * (onehot - p)


def allreduce_backward(upstream_per_rank, autograd=True):
    """Gradient each rank's partial receives from an all-reduce (sum) whose
    result every rank uses: with autograd (dist.nn.all_reduce) the sum over
    ranks of their upstream gradients; without it, the rank's own upstream."""
    u = np.asarray(upstream_per_rank, dtype=np.float64)
    return np.broadcast_to(u.sum(axis=0), u.shape).copy() if autograd else u.copy()


def sft_loss(partial_sums, scale=1.0, autograd=True):
    """SFT (Eq. 1) over sp ranks: partial_sums [sp, n] are the ranks' per-
    sequence log-probability sums.  loss = -scale * total; returns (loss,
    upstream gradient of every rank's partials [sp, n])."""
    ps = np.asarray(partial_sums, dtype=np.float64)
    loss = -scale * ps.sum()
    local = np.full(ps.shape, -scale)  # d loss / d (all-reduced sum), on every rank
    return loss, allreduce_backward(local, autograd)


def dpo_loss(partial_sums, ref_partial_sums, beta, autograd=True):
    """DPO (Eq. 2) over sp ranks.  Sequences come in pairs: 2p chosen, 2p+1
    rejected.  The policy and reference partial sums [sp, 2P] are all-reduced
    first; z_p = beta * ((pi_w - ref_w) - (pi_l - ref_l)); loss = mean over
    pairs of -log sigmoid(z_p).  Returns (loss, upstream gradient of the
    policy partials [sp, 2P]) -- the reference sums carry no gradient."""
    pi = np.asarray(partial_sums, dtype=np.float64).sum(axis=0)
    ref = np.asarray(ref_partial_sums, dtype=np.float64).sum(axis=0)
    P = pi.shape[0] // 2
    z = beta * ((pi[0::2] - ref[0::2]) - (pi[1::2] - ref[1::2]))
    loss = float(np.mean(np.logaddexp(0.0, -z)))
    sig_neg = 1.0 / (1.0 + np.exp(z))  # sigmoid(-z) = d softplus(-z) / d(-z)
    d = np.zeros(2 * P)
    d[0::2] = -beta * sig_neg / P
    d[1::2] = beta * sig_neg / P
    sp = np.asarray(partial_sums).shape[0]
    local = np.broadcast_to(d, (sp, 2 * P))
    return loss, allreduce_backward(local, autograd)


def listing2_w0_grads(x_per_rank, autograd=True):
    """The worked example of Listing 2: w0 = 1, rank r computes y_r = w0 x_r,
    y = all-reduce(y_r), loss = 2 y - 1 on every rank.  Returns the gradient
    of w0 on every rank (d loss / d y = 2 on each rank, passed back through
    the all-reduce, times d y_r / d w0 = x_r)."""
    x = np.asarray(x_per_rank, dtype=np.float64)
    upstream = np.full(x.shape, 2.0)
    return allreduce_backward(upstream, autograd) * x
