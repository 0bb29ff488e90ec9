"""fp64 reference for token log-probabilities through the LM head and the
training objectives built on them.

TEST INFRASTRUCTURE ONLY: the HIP library's LM-head calls are checked
against this module.  Only tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP path.

What it computes (DiRL, arXiv 2512.22234):

* Section 2.1, Eq. 3: the blockwise NELBO is a w(t)-weighted cross-entropy
  between the model's distribution at each masked position and the clean
  token there.  Per position: loss = -w log p(target).
* Section 2.2, Eq. 4-5 (GRPO) and Section 3.2, Eq. 6-7 (DiPO): the clipped
  surrogate min(r A, clip(r, 1 - eps, 1 + eps) A) of the ratio
  r = pi_theta / pi_old of each decoded token's probability, weighted by one
  over the total trajectory length, minus beta times a KL penalty towards a
  reference policy.  With online updates (Eq. 7) pi_old is the detached
  current policy, so r = 1 in value.

Readings taken where the paper is silent: the per-token probability is the
softmax over the vocabulary of the LM head's logits h . w_v (no temperature,
no bias); the KL penalty is estimated per token as
exp(ref - logp) - (ref - logp) - 1 (the non-negative estimator GRPO uses);
a target outside [0, V) marks a position that is not scored.

Everything is the plain definition in float64: dense logits, a max-shifted
log-sum-exp, the softmax, and the textbook gradient of log-softmax.
"""
from __future__ import annotations

import numpy as np


def _as64(x):
    return np.asarray(x, dtype=np.float64)


def lm_head_logprobs(H, W, targets):
    """(logp [N], lse [N]): log p(targets[n]) under softmax(H W^T) per row
    (Eq. 3 and Eq. 6 take their per-token probabilities from it); rows whose
    target is outside [0, V) get logp 0."""
    H, W = _as64(H), _as64(W)
    t = np.asarray(targets, dtype=np.int64)
    logits = H @ W.T
    m = logits.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(logits - m).sum(axis=1, keepdims=True)))[:, 0]
    V = W.shape[0]
    valid = (t >= 0) & (t < V)
    logp = np.zeros(H.shape[0])
    idx = np.nonzero(valid)[0]
    logp[idx] = logits[idx, t[idx]] - lse[idx]
    return logp, lse


def lm_head_backward(H, W, targets, dlogp):
    """(dH, dW) of sum_n dlogp[n] logp[n]: with p the row softmax,
    dlogits = dlogp[n] (onehot(t_n) - p), dH = dlogits W, dW = dlogits^T H."""
    H, W = _as64(H), _as64(W)
    t = np.asarray(targets, dtype=np.int64)
    c = _as64(dlogp).copy()
    V = W.shape[0]
    valid = (t >= 0) & (t < V)
    c[~valid] = 0.0
    logits = H @ W.T
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    g = -p
    idx = np.nonzero(valid)[0]
    g[idx, t[idx]] += 1.0
    g *= c[:, None]
    return g @ W, g.T @ H


def masked_ce_objective(logp, weight):
    """Eq. 3 per position: (loss, dloss/dlogp) = (-w logp, -w); w carries the
    masked-position indicator and w(t)."""
    logp, w = _as64(logp), _as64(weight)
    return -w * logp, -w


def dipo_objective(logp, logp_old, logp_ref, adv, weight, eps, beta):
    """Eq. 6-7 per position, as a loss to minimise: with r = exp(logp - logp_old),
    s = min(r A, clip(r, 1 - eps, 1 + eps) A) and kl = exp(ref - logp) - (ref - logp) - 1,
    loss = -w (s - beta kl).  Returns (loss, dloss/dlogp); the derivative of s
    is r A where the unclipped term is the minimum and 0 where the clipped
    term is (r outside the clip range); dkl/dlogp = 1 - exp(ref - logp)."""
    logp, old, A, w = _as64(logp), _as64(logp_old), _as64(adv), _as64(weight)
    r = np.exp(logp - old)
    un = r * A
    cl = np.clip(r, 1.0 - eps, 1.0 + eps) * A
    use_un = un <= cl
    s = np.where(use_un, un, cl)
    ds = np.where(use_un, un, 0.0)
    if beta != 0.0:
        d = _as64(logp_ref) - logp
        kl = np.exp(d) - d - 1.0
        dkl = 1.0 - np.exp(d)
    else:
        kl = np.zeros_like(logp)
        dkl = np.zeros_like(logp)
    return -w * (s - beta * kl), -w * (ds - beta * dkl)


def lm_head_sampled(H, W, targets, dlogp, rows, vocab_rows, chunk=16384):
    """The same quantities at a few positions, for shapes whose full logits do
    not fit in memory: (logp[rows], lse[rows], dH[rows], dW[vocab_rows]).
    dW[vocab_rows] is exact when dlogp vanishes outside `rows` (it sums over
    those positions only).  The logits of the chosen rows are computed in
    vocabulary chunks of `chunk` rows of W (float64), which changes only the
    memory bound, not the arithmetic of any entry."""
    rows = np.asarray(rows, dtype=np.int64)
    vocab_rows = np.asarray(vocab_rows, dtype=np.int64)
    Hr = _as64(np.asarray(H)[rows])
    V = W.shape[0]
    logits = np.empty((len(rows), V))
    for v0 in range(0, V, chunk):
        logits[:, v0:v0 + chunk] = Hr @ _as64(np.asarray(W[v0:v0 + chunk])).T
    m = logits.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(logits - m).sum(axis=1, keepdims=True)))[:, 0]
    t = np.asarray(targets, dtype=np.int64)[rows]
    valid = (t >= 0) & (t < V)
    logp = np.where(valid, logits[np.arange(len(rows)), np.where(valid, t, 0)] - lse, 0.0)
    c = np.where(valid, _as64(np.asarray(dlogp)[rows]), 0.0)
    g = -np.exp(logits - lse[:, None])
    g[np.nonzero(valid)[0], t[valid]] += 1.0
    g *= c[:, None]
    dH = np.zeros((len(rows), W.shape[1]))
    for v0 in range(0, V, chunk):
        dH += g[:, v0:v0 + chunk] @ _as64(np.asarray(W[v0:v0 + chunk]))
    dW = g[:, vocab_rows].T @ Hr
    return logp, lse, dH, dW
