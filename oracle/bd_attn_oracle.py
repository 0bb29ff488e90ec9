"""fp64 reference for block-diffusion masked attention over a packed [x_t | x_0] sequence.

TEST INFRASTRUCTURE ONLY: this module is the oracle that the HIP library is
checked against.  Only tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP path and imports nothing from it.

What it computes (DiRL, arXiv 2512.22234):

* Section 2.1, Eq. 1: a sequence of L tokens is cut into K blocks of S tokens
  and modelled autoregressively across blocks, so the clean copy x_0 attends
  block-causally: clean block k sees clean blocks 0..k.
* Section 2.1, Eq. 2: the noisy state of block k is denoised in parallel from
  its own noisy tokens (bidirectionally) and the clean history b^{<k}: a noisy
  token of block k sees the noisy tokens of block k and the clean tokens of
  blocks 0..k-1.  A clean token never sees a noisy one.
* Section 4.1 (and the caption of Fig. 4): DiRL repeats the whole sequence
  (prompt and output alike) and trains with one regular mask, so attention
  runs over the 2L tokens [x_t | x_0] (noisy copy first) with the mask above
  and no prompt/output distinction.

Readings taken where the paper is silent: positions p < L are noisy, block
index b(p) = (p mod L) div S (a shorter last block when S does not divide L),
softmax scale defaults to 1/sqrt(D), LSE is the natural-log log-sum-exp of the
scaled scores over visible keys, query head h uses KV head h div (Hq/Hkv).

Everything is the plain definition written out in float64: the explicit
2L x 2L mask, dense scores, softmax, and the textbook softmax-attention
vector-Jacobian product.  Rows are processed in chunks only to bound memory;
the arithmetic per row is unchanged.
"""
from __future__ import annotations

import math

import numpy as np


def block_index(L: int, S: int) -> np.ndarray:
    """b(p) = (p mod L) div S for every packed position p in [0, 2L) (Section 2.1)."""
    p = np.arange(2 * L)
    return (p % L) // S


def visibility_mask(L: int, S: int) -> np.ndarray:
    """Boolean [2L, 2L] mask, M[q, k] true iff query q may attend to key k.

    Noisy query (q < L): noisy key of the same block (Eq. 2, bidirectional
    within the block) or clean key of an earlier block (Eq. 2's b^{<k}).
    Clean query: clean key of the same or an earlier block (Eq. 1).
    Clean query, noisy key: never.
    """
    if L < 1 or S < 1:
        raise ValueError("L and S must be >= 1")
    p = np.arange(2 * L)
    noisy = p < L
    b = (p % L) // S
    nq, nk = noisy[:, None], noisy[None, :]
    bq, bk = b[:, None], b[None, :]
    M = (nq & nk & (bq == bk)) | (nq & ~nk & (bk < bq)) | (~nq & ~nk & (bk <= bq))
    # every row sees at least its own position
    assert M.any(axis=1).all()
    return M


def allowed_count(L: int, S: int) -> int:
    """Number of visible (query, key) pairs for one (batch, head)."""
    return int(visibility_mask(L, S).sum())


def _as64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def _check_shapes(Q, K, V, L):
    if Q.ndim != 4 or K.ndim != 4 or V.shape != K.shape:
        raise ValueError("Q [B,Hq,2L,D], K/V [B,Hkv,2L,D] expected")
    B, Hq, N, D = Q.shape
    if N != 2 * L or K.shape[0] != B or K.shape[2] != N or K.shape[3] != D:
        raise ValueError("inconsistent shapes")
    Hkv = K.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    return B, Hq, Hkv, D


def _rows(N: int, chunk: int):
    for r0 in range(0, N, chunk):
        yield r0, min(N, r0 + chunk)


def _softmax_rows(Zc: np.ndarray, Mc: np.ndarray):
    """Masked row softmax of a chunk of scores: returns P, row max, row sum."""
    Z = np.where(Mc, Zc, -np.inf)
    m = Z.max(axis=1, keepdims=True)
    E = np.exp(Z - m)
    l = E.sum(axis=1, keepdims=True)
    return E / l, m, l


def forward(Q, K, V, L: int, S: int, scale: float | None = None,
            heads=None, row_chunk: int = 1024):
    """O = softmax(scale * Q K^T masked) V and LSE = log sum exp of the masked scores.

    heads: optional iterable of (b, hq) pairs to compute; other heads are NaN.
    Returns (O [B,Hq,2L,D], LSE [B,Hq,2L]) in float64.
    """
    Q, K, V = _as64(Q), _as64(K), _as64(V)
    B, Hq, Hkv, D = _check_shapes(Q, K, V, L)
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = visibility_mask(L, S)
    N = 2 * L
    O = np.full(Q.shape, np.nan)
    LSE = np.full(Q.shape[:3], np.nan)
    todo = [(b, h) for b in range(B) for h in range(Hq)] if heads is None else list(heads)
    for b, h in todo:
        g = h // G
        for r0, r1 in _rows(N, row_chunk):
            Zc = scale * (Q[b, h, r0:r1] @ K[b, g].T)
            P, m, l = _softmax_rows(Zc, M[r0:r1])
            O[b, h, r0:r1] = P @ V[b, g]
            LSE[b, h, r0:r1] = (m + np.log(l))[:, 0]
    return O, LSE


def probabilities(Q, K, L: int, S: int, scale: float | None = None) -> np.ndarray:
    """Dense attention probabilities P [B,Hq,2L,2L] (small shapes only)."""
    Q, K = _as64(Q), _as64(K)
    B, Hq, Hkv, D = _check_shapes(Q, K, K, L)
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = visibility_mask(L, S)
    P = np.empty((B, Hq, 2 * L, 2 * L))
    for b in range(B):
        for h in range(Hq):
            P[b, h] = _softmax_rows(scale * (Q[b, h] @ K[b, h // G].T), M)[0]
    return P


def backward(dO, Q, K, V, L: int, S: int, scale: float | None = None,
             groups=None, row_chunk: int = 1024):
    """Gradients of <dO, O> with respect to Q, K and V.

    The textbook vector-Jacobian product of softmax attention:
        dV = P^T dO,  dP = dO V^T,  Delta = rowsum(dO * O),
        dS = P * (dP - Delta),  dQ = scale dS K,  dK = scale dS^T Q,
    with P the masked softmax of the forward pass, and dK/dV of a KV head
    summed over the query heads that share it.

    groups: optional iterable of (b, hkv) pairs; only those KV heads and their
    query heads are computed, everything else is NaN.
    Returns (dQ, dK, dV) in float64.
    """
    dO, Q, K, V = _as64(dO), _as64(Q), _as64(K), _as64(V)
    B, Hq, Hkv, D = _check_shapes(Q, K, V, L)
    if dO.shape != Q.shape:
        raise ValueError("dO must have Q's shape")
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = visibility_mask(L, S)
    N = 2 * L
    dQ = np.full(Q.shape, np.nan)
    dK = np.full(K.shape, np.nan)
    dV = np.full(V.shape, np.nan)
    todo = [(b, g) for b in range(B) for g in range(Hkv)] if groups is None else list(groups)
    for b, g in todo:
        dK[b, g] = 0.0
        dV[b, g] = 0.0
        for h in range(g * G, (g + 1) * G):
            for r0, r1 in _rows(N, row_chunk):
                Zc = scale * (Q[b, h, r0:r1] @ K[b, g].T)
                P, _, _ = _softmax_rows(Zc, M[r0:r1])
                dOc = dO[b, h, r0:r1]
                Oc = P @ V[b, g]
                dP = dOc @ V[b, g].T
                delta = (dOc * Oc).sum(axis=1, keepdims=True)
                dS = P * (dP - delta)
                dQ[b, h, r0:r1] = scale * (dS @ K[b, g])
                dK[b, g] += scale * (dS.T @ Q[b, h, r0:r1])
                dV[b, g] += P.T @ dOc
    return dQ, dK, dV


def sampled(dO, Q, K, V, L: int, S: int, b: int, hkv: int, query_rows, key_rows,
            scale: float | None = None, row_chunk: int = 1024):
    """Selected outputs of one KV group (batch b, KV head hkv), for shapes too
    large to evaluate whole.

    For every query head h of the group: O, LSE and dQ at `query_rows`.
    For the KV head: dK and dV at `key_rows`, summed over the group's query
    heads and over every query that sees those keys (queries that see none of
    them contribute exactly zero, since P vanishes there).  Each needed query
    row is evaluated in full with the same definitions as forward/backward.
    Returns dict with O [G,nq,D], LSE [G,nq], dQ [G,nq,D], dK [nk,D], dV [nk,D].
    """
    Qb, Kb, Vb, dOb = _as64(Q[b]), _as64(K[b, hkv]), _as64(V[b, hkv]), _as64(dO[b])
    Hq, N, D = Qb.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = visibility_mask(L, S)
    qr = np.asarray(list(query_rows), dtype=np.int64)
    kr = np.asarray(list(key_rows), dtype=np.int64)
    seers = np.nonzero(M[:, kr].any(axis=1))[0] if len(kr) else np.zeros(0, np.int64)
    out = {"O": np.zeros((G, len(qr), D)), "LSE": np.zeros((G, len(qr))),
           "dQ": np.zeros((G, len(qr), D)), "dK": np.zeros((len(kr), D)), "dV": np.zeros((len(kr), D))}
    for gi in range(G):
        h = hkv * G + gi
        for rows, is_query in ((qr, True), (seers, False)):
            for r0, r1 in _rows(len(rows), row_chunk):
                idx = rows[r0:r1]
                Zc = scale * (Qb[h, idx] @ Kb.T)
                P, m, l = _softmax_rows(Zc, M[idx])
                Oc = P @ Vb
                dOc = dOb[h, idx]
                dP = dOc @ Vb.T
                delta = (dOc * Oc).sum(axis=1, keepdims=True)
                dS = P * (dP - delta)
                if is_query:
                    out["O"][gi, r0:r1] = Oc
                    out["LSE"][gi, r0:r1] = (m + np.log(l))[:, 0]
                    out["dQ"][gi, r0:r1] = scale * (dS @ Kb)
                else:
                    out["dK"] += scale * (dS[:, kr].T @ Qb[h, idx])
                    out["dV"] += P[:, kr].T @ dOc
    return out


# ---------------------------------------------------------------------------
# Several sequences packed into one buffer (the dynamic packing that
# Section 5.2 names as the next speed-up of blockwise training).
#
# Sequence i of length L_i (tokens per copy) occupies packed rows
# [2 c_i, 2 c_{i+1}) of every head, c = cumulative lengths (c_0 = 0): its noisy
# copy x_t first, then its clean copy x_0, exactly the single-sequence layout
# of Section 4.1.  A query sees a key iff both lie in the same sequence and
# that sequence's mask (Eq. 1 / Eq. 2 at their local positions) allows the
# pair.  Sequences never see each other; a sequence of length 0 has no rows.

def varlen_visibility_mask(lengths, S: int) -> np.ndarray:
    """Boolean [2T, 2T] mask of the packed layout, T = sum(lengths), built
    from the per-pair rule: same sequence, then noisy query -> noisy key of
    the same block or clean key of an earlier block; clean query -> clean key
    of the same or an earlier block; clean query -> noisy key never."""
    lengths = [int(x) for x in lengths]
    if S < 1 or any(x < 0 for x in lengths):
        raise ValueError("S >= 1 and lengths >= 0 required")
    seq, local, Ls = [], [], []
    for i, Li in enumerate(lengths):
        seq += [i] * (2 * Li)
        local += list(range(2 * Li))
        Ls += [Li] * (2 * Li)
    seq, local, Ls = np.array(seq, dtype=np.int64), np.array(local, dtype=np.int64), np.array(Ls, dtype=np.int64)
    if seq.size == 0:
        return np.zeros((0, 0), dtype=bool)
    noisy = local < Ls
    b = np.where(Ls > 0, (local % np.maximum(Ls, 1)) // S, 0)
    same = seq[:, None] == seq[None, :]
    nq, nk = noisy[:, None], noisy[None, :]
    bq, bk = b[:, None], b[None, :]
    M = same & ((nq & nk & (bq == bk)) | (nq & ~nk & (bk < bq)) | (~nq & ~nk & (bk <= bq)))
    assert M.any(axis=1).all()
    return M


def _check_varlen(Q, K, V, lengths):
    if Q.ndim != 3 or K.ndim != 3 or V.shape != K.shape:
        raise ValueError("Q [Hq,2T,D], K/V [Hkv,2T,D] expected")
    Hq, N, D = Q.shape
    Hkv = K.shape[0]
    if N != 2 * sum(lengths) or K.shape[1] != N or K.shape[2] != D or Hq % Hkv:
        raise ValueError("inconsistent shapes")
    return Hq, Hkv, D


def varlen_forward(Q, K, V, lengths, S: int, scale: float | None = None):
    """O [Hq,2T,D] and LSE [Hq,2T] of the packed sequences: dense masked
    softmax attention over all 2T packed rows with varlen_visibility_mask."""
    Q, K, V = _as64(Q), _as64(K), _as64(V)
    Hq, Hkv, D = _check_varlen(Q, K, V, lengths)
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = varlen_visibility_mask(lengths, S)
    O = np.zeros(Q.shape)
    LSE = np.zeros(Q.shape[:2])
    for h in range(Hq):
        P, m, l = _softmax_rows(scale * (Q[h] @ K[h // G].T), M)
        O[h] = P @ V[h // G]
        LSE[h] = (m + np.log(l))[:, 0]
    return O, LSE


def varlen_backward(dO, Q, K, V, lengths, S: int, scale: float | None = None):
    """dQ, dK, dV of <dO, O> for the packed sequences (the same textbook
    vector-Jacobian product as backward, over the packed mask)."""
    dO, Q, K, V = _as64(dO), _as64(Q), _as64(K), _as64(V)
    Hq, Hkv, D = _check_varlen(Q, K, V, lengths)
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    M = varlen_visibility_mask(lengths, S)
    dQ = np.zeros(Q.shape)
    dK = np.zeros(K.shape)
    dV = np.zeros(V.shape)
    for h in range(Hq):
        g = h // G
        P, _, _ = _softmax_rows(scale * (Q[h] @ K[g].T), M)
        O = P @ V[g]
        dP = dO[h] @ V[g].T
        delta = (dO[h] * O).sum(axis=1, keepdims=True)
        dS = P * (dP - delta)
        dQ[h] = scale * (dS @ K[g])
        dK[g] += scale * (dS.T @ Q[h])
        dV[g] += P.T @ dO[h]
    return dQ, dK, dV


# ---------------------------------------------------------------------------
# Decoding (rollouts): the KV-cache reading of Section 2.1.  While block k is
# denoised, its S noisy tokens attend to the clean tokens of the blocks
# before it, held in a KV cache, and to each other in both directions (Eq. 2);
# nothing else exists yet.  So the noisy rows of block k see every cached key
# and every key of their own block, with no further mask.

def decode_forward(Q, Kc, Vc, Kn, Vn, cache_lens, scale: float | None = None):
    """O [B,Hq,S,D] and LSE [B,Hq,S] of one block's noisy queries Q [B,Hq,S,D]
    over the clean cache Kc/Vc [B,Hkv,C,D] (the first cache_lens[b] rows of
    sequence b are valid) and the block's own noisy keys Kn/Vn [B,Hkv,S,D]:
    dense softmax attention over the concatenation [cache ; block]."""
    Q, Kc, Vc, Kn, Vn = _as64(Q), _as64(Kc), _as64(Vc), _as64(Kn), _as64(Vn)
    B, Hq, S, D = Q.shape
    Hkv = Kc.shape[1]
    if Hq % Hkv or Kn.shape != (B, Hkv, S, D) or Vn.shape != Kn.shape or Vc.shape != Kc.shape:
        raise ValueError("inconsistent shapes")
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None or scale <= 0 else float(scale)
    O = np.zeros(Q.shape)
    LSE = np.zeros(Q.shape[:3])
    for b in range(B):
        n = int(cache_lens[b])
        if not 0 <= n <= Kc.shape[2]:
            raise ValueError("cache length out of range")
        for h in range(Hq):
            g = h // G
            Kall = np.concatenate([Kc[b, g, :n], Kn[b, g]], axis=0)
            Vall = np.concatenate([Vc[b, g, :n], Vn[b, g]], axis=0)
            P, m, l = _softmax_rows(scale * (Q[b, h] @ Kall.T), np.ones((S, n + S), dtype=bool))
            O[b, h] = P @ Vall
            LSE[b, h] = (m + np.log(l))[:, 0]
    return O, LSE
