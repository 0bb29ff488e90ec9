"""Pins for the fp64 oracle: each test checks it against something other than itself.

* hand-written masks for the Fig. 4 shape (L=8, S=2) and a ragged case;
* the mask rebuilt block by block from the roles in Eq. 1 / Eq. 2;
* closed-form visible-pair counts;
* a closed form of the forward pass (uniform attention when K = 0);
* the S=1 and S=L special cases against torch's own scaled-dot-product
  attention (causal / unmasked) in fp64;
* the per-block KV-cache view (Section 2.1) against torch SDPA, forward, LSE
  and torch-autograd gradients;
* finite differences of <dO, O>;
* invariants: clean-half independence, GQA = repeated-KV MHA, equivariance
  under permutations inside a noisy block, softmax rows summing to one;
* packed sequences (varlen): the packed mask against plain pair-by-pair loops,
  one sequence against the single-sequence mask, equal lengths against the
  batched oracle, each sequence against its own batched call, independence of
  the sequences, and finite differences;
* decoding: the noisy rows of block k of the training forward pass (the
  KV-cache view of Section 2.1), torch SDPA over the concatenated keys, and
  cache rows past the length having no effect.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_mask(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([c == "1" for c in line])
    return np.array(rows, dtype=bool)


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------- mask pins

@pytest.mark.parametrize("name,L,S", [("mask_L8_S2.txt", 8, 2), ("mask_L5_S2.txt", 5, 2)])
def test_mask_matches_hand_written_golden(name, L, S):
    np.testing.assert_array_equal(oracle.visibility_mask(L, S), _read_mask(name))


def _mask_by_blocks(L, S):
    """Rebuild the mask from the block roles: for each block k, its noisy
    tokens get their own noisy block plus the clean history b^{<k} (Eq. 2),
    its clean tokens get clean blocks 0..k (Eq. 1)."""
    N = 2 * L
    M = np.zeros((N, N), dtype=bool)
    starts = list(range(0, L, S))
    for k, a in enumerate(starts):
        e = min(L, a + S)
        noisy_rows = range(a, e)
        clean_rows = range(L + a, L + e)
        for r in noisy_rows:
            for c in range(a, e):
                M[r, c] = True
            for c in range(L, L + a):
                M[r, c] = True
        for r in clean_rows:
            for c in range(L, L + e):
                M[r, c] = True
    return M


def test_mask_brute_force_all_small_shapes():
    for L in range(1, 17):
        for S in range(1, L + 2):
            np.testing.assert_array_equal(oracle.visibility_mask(L, S), _mask_by_blocks(L, S),
                                          err_msg=f"L={L} S={S}")


def test_mask_counts_closed_form():
    for L in range(1, 33):
        for S in range(1, L + 1):
            sizes = [min(S, L - a) for a in range(0, L, S)]
            prefix = np.cumsum([0] + sizes[:-1])
            want = sum(2 * s * (p + s) for s, p in zip(sizes, prefix))
            assert oracle.allowed_count(L, S) == want
            if L % S == 0:
                assert want == L * (L + S)
    # the configurations' per-head counts
    assert oracle.allowed_count(2048, 4) == 4_202_496
    assert oracle.allowed_count(1024, 4) == 1_052_672
    assert oracle.allowed_count(64, 4) == 4_352


def test_block_index_examples():
    np.testing.assert_array_equal(oracle.block_index(5, 2), [0, 0, 1, 1, 2, 0, 0, 1, 1, 2])


def test_s_greater_than_l_equals_s_equal_l():
    for L in (1, 3, 7):
        np.testing.assert_array_equal(oracle.visibility_mask(L, L), oracle.visibility_mask(L, 5 * L))


# ---------------------------------------------------------- forward closed form

def _visible_keys(L, S, p):
    """Visible key positions of packed query p, from Eq. 1 / Eq. 2 directly."""
    if p < L:
        a = (p // S) * S
        return list(range(a, min(L, a + S))) + list(range(L, L + a))
    i = p - L
    e = min(L, (i // S + 1) * S)
    return list(range(L, L + e))


@pytest.mark.parametrize("L,S", [(8, 2), (12, 5), (16, 1), (9, 9)])
def test_uniform_attention_closed_form(L, S):
    """K = 0 gives equal weight on every visible key: O is the mean of the
    visible V rows and LSE = log(number of visible keys)."""
    D = 6
    Q = _rand((1, 1, 2 * L, D), 1)
    K = np.zeros((1, 1, 2 * L, D))
    V = _rand((1, 1, 2 * L, D), 2)
    O, LSE = oracle.forward(Q, K, V, L, S)
    for p in range(2 * L):
        keys = _visible_keys(L, S, p)
        np.testing.assert_allclose(O[0, 0, p], V[0, 0, keys].mean(axis=0), rtol=0, atol=1e-13)
        assert abs(LSE[0, 0, p] - math.log(len(keys))) < 1e-13


# ------------------------------------------------------ special cases via torch

def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x))


def test_s1_clean_half_is_causal_attention():
    L, D = 24, 8
    Q, K, V = _rand((2, 3, 2 * L, D), 3), _rand((2, 3, 2 * L, D), 4), _rand((2, 3, 2 * L, D), 5)
    O, LSE = oracle.forward(Q, K, V, L, 1)
    c = slice(L, 2 * L)
    ref = F.scaled_dot_product_attention(_t(Q[:, :, c]), _t(K[:, :, c]), _t(V[:, :, c]), is_causal=True)
    np.testing.assert_allclose(O[:, :, c], ref.numpy(), rtol=0, atol=1e-12)
    # noisy row i (S=1): its own noisy token plus clean tokens < i
    for i in range(L):
        keys = [i] + list(range(L, L + i))
        ref_i = F.scaled_dot_product_attention(_t(Q[:, :, i:i + 1]), _t(K[:, :, keys]), _t(V[:, :, keys]))
        np.testing.assert_allclose(O[:, :, i:i + 1], ref_i.numpy(), rtol=0, atol=1e-12)


def test_s_equal_l_halves_are_unmasked_attention():
    L, D = 20, 8
    Q, K, V = _rand((1, 2, 2 * L, D), 6), _rand((1, 2, 2 * L, D), 7), _rand((1, 2, 2 * L, D), 8)
    O, _ = oracle.forward(Q, K, V, L, L)
    for half in (slice(0, L), slice(L, 2 * L)):
        ref = F.scaled_dot_product_attention(_t(Q[:, :, half]), _t(K[:, :, half]), _t(V[:, :, half]))
        np.testing.assert_allclose(O[:, :, half], ref.numpy(), rtol=0, atol=1e-12)


def _decomposed_torch(q, k, v, L, S, scale):
    """Block-by-block evaluation (the KV-cache view of Section 2.1): noisy
    block j attends, without a mask, to [clean blocks < j ; noisy block j];
    clean block j attends to clean blocks <= j.  Returns O and LSE for one
    (batch, head); q, k, v are [2L, D] torch fp64 tensors."""
    out = [None] * (2 * L)
    lse = [None] * (2 * L)
    for a in range(0, L, S):
        e = min(L, a + S)
        groups = [(list(range(a, e)), list(range(L, L + a)) + list(range(a, e))),
                  (list(range(L + a, L + e)), list(range(L, L + e)))]
        for rows, keys in groups:
            qs, ks, vs = q[rows], k[keys], v[keys]
            o = F.scaled_dot_product_attention(qs[None], ks[None], vs[None], scale=scale)[0]
            ls = torch.logsumexp(scale * qs @ ks.T, dim=1)
            for t, r in enumerate(rows):
                out[r] = o[t]
                lse[r] = ls[t]
    return torch.stack(out), torch.stack(lse)


@pytest.mark.parametrize("L,S,Hq,Hkv", [(16, 4, 2, 1), (13, 3, 4, 2), (10, 10, 1, 1), (7, 1, 3, 3)])
def test_forward_matches_per_block_decomposition(L, S, Hq, Hkv):
    D = 8
    B = 2
    Q, K, V = _rand((B, Hq, 2 * L, D), 9), _rand((B, Hkv, 2 * L, D), 10), _rand((B, Hkv, 2 * L, D), 11)
    scale = 0.3
    O, LSE = oracle.forward(Q, K, V, L, S, scale=scale)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            o, ls = _decomposed_torch(_t(Q[b, h]), _t(K[b, h // G]), _t(V[b, h // G]), L, S, scale)
            np.testing.assert_allclose(O[b, h], o.numpy(), rtol=0, atol=1e-12)
            np.testing.assert_allclose(LSE[b, h], ls.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("L,S,Hq,Hkv", [(12, 4, 2, 1), (9, 2, 2, 2), (8, 8, 3, 1), (6, 1, 2, 1)])
def test_backward_matches_torch_autograd_of_decomposition(L, S, Hq, Hkv):
    D = 8
    B = 1
    G = Hq // Hkv
    Q, K, V = _rand((B, Hq, 2 * L, D), 12), _rand((B, Hkv, 2 * L, D), 13), _rand((B, Hkv, 2 * L, D), 14)
    dO = _rand((B, Hq, 2 * L, D), 15)
    dQ, dK, dV = oracle.backward(dO, Q, K, V, L, S)
    scale = 1.0 / math.sqrt(D)
    q, k, v = (_t(x).clone().requires_grad_(True) for x in (Q, K, V))
    loss = 0
    for h in range(Hq):
        o, _ = _decomposed_torch(q[0, h], k[0, h // G], v[0, h // G], L, S, scale)
        loss = loss + (o * _t(dO[0, h])).sum()
    loss.backward()
    np.testing.assert_allclose(dQ, q.grad.numpy(), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dK, k.grad.numpy(), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dV, v.grad.numpy(), rtol=0, atol=1e-11)


@pytest.mark.parametrize("L,S", [(4, 1), (6, 2), (7, 3), (5, 5)])
def test_backward_finite_differences(L, S):
    D, Hq, Hkv = 4, 2, 1
    Q, K, V = _rand((1, Hq, 2 * L, D), 16), _rand((1, Hkv, 2 * L, D), 17), _rand((1, Hkv, 2 * L, D), 18)
    dO = _rand((1, Hq, 2 * L, D), 19)
    grads = oracle.backward(dO, Q, K, V, L, S)
    h = 1e-6

    def loss(Qx, Kx, Vx):
        return float((oracle.forward(Qx, Kx, Vx, L, S)[0] * dO).sum())

    rng = np.random.default_rng(20)
    for which, X in enumerate((Q, K, V)):
        for _ in range(12):
            idx = tuple(rng.integers(0, s) for s in X.shape)
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h
            Xm[idx] -= h
            args_p = [Q, K, V]
            args_m = [Q, K, V]
            args_p[which], args_m[which] = Xp, Xm
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            an = grads[which][idx]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (which, idx, fd, an)


# ---------------------------------------------------------------- invariants

def test_clean_half_independent_of_noisy_inputs():
    L, S, D = 16, 4, 8
    Q, K, V = _rand((1, 2, 2 * L, D), 21), _rand((1, 1, 2 * L, D), 22), _rand((1, 1, 2 * L, D), 23)
    O1, L1 = oracle.forward(Q, K, V, L, S)
    Q2, K2, V2 = Q.copy(), K.copy(), V.copy()
    Q2[:, :, :L] += 5 * _rand((1, 2, L, D), 24)
    K2[:, :, :L] += 5 * _rand((1, 1, L, D), 25)
    V2[:, :, :L] += 5 * _rand((1, 1, L, D), 26)
    O2, L2 = oracle.forward(Q2, K2, V2, L, S)
    np.testing.assert_array_equal(O1[:, :, L:], O2[:, :, L:])
    np.testing.assert_array_equal(L1[:, :, L:], L2[:, :, L:])
    # a loss on clean rows only has exactly zero gradient on noisy K/V
    dO = _rand((1, 2, 2 * L, D), 27)
    dO[:, :, :L] = 0
    _, dK, dV = oracle.backward(dO, Q, K, V, L, S)
    assert np.all(dK[:, :, :L] == 0) and np.all(dV[:, :, :L] == 0)


def test_gqa_equals_repeated_kv():
    L, S, D, Hq, Hkv = 10, 3, 8, 4, 2
    G = Hq // Hkv
    Q, K, V = _rand((2, Hq, 2 * L, D), 28), _rand((2, Hkv, 2 * L, D), 29), _rand((2, Hkv, 2 * L, D), 30)
    dO = _rand((2, Hq, 2 * L, D), 31)
    Kr, Vr = np.repeat(K, G, axis=1), np.repeat(V, G, axis=1)
    O, LSE = oracle.forward(Q, K, V, L, S)
    Or, LSEr = oracle.forward(Q, Kr, Vr, L, S)
    np.testing.assert_allclose(O, Or, atol=1e-14, rtol=0)
    np.testing.assert_allclose(LSE, LSEr, atol=1e-14, rtol=0)
    dQ, dK, dV = oracle.backward(dO, Q, K, V, L, S)
    dQr, dKr, dVr = oracle.backward(dO, Q, Kr, Vr, L, S)
    np.testing.assert_allclose(dQ, dQr, atol=1e-13, rtol=0)
    np.testing.assert_allclose(dK, dKr.reshape(2, Hkv, G, 2 * L, D).sum(axis=2), atol=1e-12, rtol=0)
    np.testing.assert_allclose(dV, dVr.reshape(2, Hkv, G, 2 * L, D).sum(axis=2), atol=1e-12, rtol=0)


def test_permutation_inside_noisy_block_is_equivariant():
    L, S, D = 12, 4, 8
    Q, K, V = _rand((1, 1, 2 * L, D), 32), _rand((1, 1, 2 * L, D), 33), _rand((1, 1, 2 * L, D), 34)
    O, LSE = oracle.forward(Q, K, V, L, S)
    perm = np.arange(2 * L)
    perm[4:8] = [6, 4, 7, 5]          # shuffle noisy block 1 (tokens 4..7)
    Op, LSEp = oracle.forward(Q[:, :, perm], K[:, :, perm], V[:, :, perm], L, S)
    np.testing.assert_allclose(Op, O[:, :, perm], atol=1e-13, rtol=0)
    np.testing.assert_allclose(LSEp, LSE[:, :, perm], atol=1e-13, rtol=0)


def test_probabilities_rows_sum_to_one_and_vanish_off_mask():
    L, S, D = 11, 3, 8
    Q, K = _rand((1, 2, 2 * L, D), 35), _rand((1, 1, 2 * L, D), 36)
    P = oracle.probabilities(Q, K, L, S)
    np.testing.assert_allclose(P.sum(axis=-1), 1.0, atol=1e-12, rtol=0)
    M = oracle.visibility_mask(L, S)
    assert np.all(P[..., ~M] == 0)
    V = _rand((1, 1, 2 * L, D), 37)
    O, _ = oracle.forward(Q, K, V, L, S)
    np.testing.assert_allclose(O, P @ V, atol=1e-13, rtol=0)


def test_row_chunking_and_subsets_do_not_change_results():
    L, S, D = 20, 4, 8
    Q, K, V = _rand((2, 4, 2 * L, D), 38), _rand((2, 2, 2 * L, D), 39), _rand((2, 2, 2 * L, D), 40)
    dO = _rand((2, 4, 2 * L, D), 41)
    O, LSE = oracle.forward(Q, K, V, L, S)
    Oc, LSEc = oracle.forward(Q, K, V, L, S, row_chunk=7)
    np.testing.assert_allclose(O, Oc, atol=1e-14, rtol=0)
    np.testing.assert_allclose(LSE, LSEc, atol=1e-14, rtol=0)
    Os, _ = oracle.forward(Q, K, V, L, S, heads=[(1, 3)])
    np.testing.assert_array_equal(Os[1, 3], O[1, 3])
    assert np.isnan(Os[0, 0]).all()
    g = oracle.backward(dO, Q, K, V, L, S)
    gc = oracle.backward(dO, Q, K, V, L, S, row_chunk=6)
    gs = oracle.backward(dO, Q, K, V, L, S, groups=[(1, 1)])
    for a, b, s in zip(g, gc, gs):
        np.testing.assert_allclose(a, b, atol=1e-13, rtol=0)
    np.testing.assert_allclose(gs[0][1, 2:4], g[0][1, 2:4], atol=0, rtol=0)
    np.testing.assert_allclose(gs[1][1, 1], g[1][1, 1], atol=0, rtol=0)


def test_sampled_matches_full_evaluation():
    L, S, D, Hq, Hkv = 18, 4, 8, 4, 2
    Q, K, V = _rand((2, Hq, 2 * L, D), 42), _rand((2, Hkv, 2 * L, D), 43), _rand((2, Hkv, 2 * L, D), 44)
    dO = _rand((2, Hq, 2 * L, D), 45)
    O, LSE = oracle.forward(Q, K, V, L, S)
    dQ, dK, dV = oracle.backward(dO, Q, K, V, L, S)
    qr, kr = [0, 5, 17, 18, 30, 35], [1, 4, 16, 20, 27, 35]
    s = oracle.sampled(dO, Q, K, V, L, S, b=1, hkv=1, query_rows=qr, key_rows=kr, row_chunk=5)
    np.testing.assert_allclose(s["O"], O[1, 2:4][:, qr], atol=1e-13, rtol=0)
    np.testing.assert_allclose(s["LSE"], LSE[1, 2:4][:, qr], atol=1e-13, rtol=0)
    np.testing.assert_allclose(s["dQ"], dQ[1, 2:4][:, qr], atol=1e-12, rtol=0)
    np.testing.assert_allclose(s["dK"], dK[1, 1, kr], atol=1e-12, rtol=0)
    np.testing.assert_allclose(s["dV"], dV[1, 1, kr], atol=1e-12, rtol=0)


# ------------------------------------------------- packed sequences (varlen)

def _varlen_mask_by_loops(lengths, S):
    """The packed mask pair by pair with plain loops: locate each row's
    sequence and local position by walking the lengths, then apply the
    single-sequence rule of Eq. 1 / Eq. 2 when both rows share a sequence."""
    rows = []
    for i, Li in enumerate(lengths):
        for local in range(2 * Li):
            rows.append((i, local, Li))
    N = len(rows)
    M = np.zeros((N, N), dtype=bool)
    for q, (iq, pq, Lq) in enumerate(rows):
        for k, (ik, pk, Lk) in enumerate(rows):
            if iq != ik:
                continue
            q_noisy, k_noisy = pq < Lq, pk < Lk
            bq, bk = (pq % Lq) // S, (pk % Lk) // S
            if q_noisy and k_noisy:
                M[q, k] = bq == bk
            elif q_noisy:
                M[q, k] = bk < bq
            elif not k_noisy:
                M[q, k] = bk <= bq
    return M


@pytest.mark.parametrize("lengths", [[1], [3], [2, 3], [4, 0, 1], [5, 2, 3], [0, 7, 0], [6, 6]])
def test_varlen_mask_brute_force(lengths):
    for S in range(1, 8):
        np.testing.assert_array_equal(oracle.varlen_visibility_mask(lengths, S), _varlen_mask_by_loops(lengths, S),
                                      err_msg=f"S={S}")


def test_varlen_mask_one_sequence_is_the_single_mask():
    for L in (1, 5, 8, 13):
        for S in (1, 2, 3, 8, 20):
            np.testing.assert_array_equal(oracle.varlen_visibility_mask([L], S), oracle.visibility_mask(L, S))


def _pack(x):
    """[B, H, 2L, D] -> [H, 2BL, D]: sequence b at packed rows [2bL, 2(b+1)L)."""
    B, H, N, D = x.shape
    return np.transpose(x, (1, 0, 2, 3)).reshape(H, B * N, D)


def test_varlen_equal_lengths_match_batched_forward_backward():
    B, Hq, Hkv, L, S, D = 3, 4, 2, 9, 2, 8
    Q, K, V, dO = (_rand(s, i) for i, s in enumerate([(B, Hq, 2 * L, D), (B, Hkv, 2 * L, D),
                                                      (B, Hkv, 2 * L, D), (B, Hq, 2 * L, D)]))
    O, LSE = oracle.forward(Q, K, V, L, S)
    dQ, dK, dV = oracle.backward(dO, Q, K, V, L, S)
    Ov, LSEv = oracle.varlen_forward(_pack(Q), _pack(K), _pack(V), [L] * B, S)
    dQv, dKv, dVv = oracle.varlen_backward(_pack(dO), _pack(Q), _pack(K), _pack(V), [L] * B, S)
    np.testing.assert_allclose(Ov, _pack(O), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(LSEv, np.transpose(LSE, (1, 0, 2)).reshape(Hq, -1), rtol=1e-12, atol=1e-12)
    for a, b in ((dQv, dQ), (dKv, dK), (dVv, dV)):
        np.testing.assert_allclose(a, _pack(b), rtol=1e-10, atol=1e-12)


def test_varlen_each_sequence_matches_its_own_batched_call():
    lengths, S, Hq, Hkv, D = [5, 0, 11, 1, 7], 3, 4, 1, 8
    T = sum(lengths)
    Q, K, V, dO = (_rand(s, 10 + i) for i, s in enumerate([(Hq, 2 * T, D), (Hkv, 2 * T, D),
                                                           (Hkv, 2 * T, D), (Hq, 2 * T, D)]))
    O, LSE = oracle.varlen_forward(Q, K, V, lengths, S)
    dQ, dK, dV = oracle.varlen_backward(dO, Q, K, V, lengths, S)
    c = 0
    for Li in lengths:
        if Li:
            r = slice(2 * c, 2 * (c + Li))
            Oi, LSEi = oracle.forward(Q[None, :, r], K[None, :, r], V[None, :, r], Li, S)
            dQi, dKi, dVi = oracle.backward(dO[None, :, r], Q[None, :, r], K[None, :, r], V[None, :, r], Li, S)
            np.testing.assert_allclose(O[:, r], Oi[0], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(LSE[:, r], LSEi[0], rtol=1e-12, atol=1e-12)
            for a, b in ((dQ[:, r], dQi[0]), (dK[:, r], dKi[0]), (dV[:, r], dVi[0])):
                np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
        c += Li


def test_varlen_sequences_do_not_see_each_other():
    lengths, S, D = [6, 4], 2, 4
    T = sum(lengths)
    Q, K, V = (_rand((2, 2 * T, D), 30 + i) for i in range(3))
    O, _ = oracle.varlen_forward(Q, K, V, lengths, S)
    K2, V2 = K.copy(), V.copy()
    K2[:, 12:] += 3.0  # the second sequence's rows
    V2[:, 12:] -= 2.0
    O2, _ = oracle.varlen_forward(Q, K2, V2, lengths, S)
    np.testing.assert_array_equal(O[:, :12], O2[:, :12])
    assert not np.allclose(O[:, 12:], O2[:, 12:])


def test_varlen_backward_finite_differences():
    lengths, S, D = [3, 2], 2, 3
    T = sum(lengths)
    Q, K, V, dO = _rand((2, 2 * T, D), 40), _rand((1, 2 * T, D), 41), _rand((1, 2 * T, D), 42), _rand((2, 2 * T, D), 43)
    dQ, dK, dV = oracle.varlen_backward(dO, Q, K, V, lengths, S)
    f = lambda q, k, v: float((dO * oracle.varlen_forward(q, k, v, lengths, S)[0]).sum())
    h = 1e-6
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        for idx in [(0, 0, 0), (0, 3, 2), (0, 7, 1), (0, 9, 0)]:
            if X.shape[0] <= idx[0]:
                continue
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h
            Xm[idx] -= h
            args_p = [Xp if Y is X else Y for Y in (Q, K, V)]
            args_m = [Xm if Y is X else Y for Y in (Q, K, V)]
            fd = (f(*args_p) - f(*args_m)) / (2 * h)
            assert abs(fd - G[idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, G[idx])


# ------------------------------------------------------------- decoding

def test_decode_equals_noisy_rows_of_the_training_mask():
    """The KV-cache view of Section 2.1: with the cache holding the clean K/V
    of blocks 0..k-1, decoding block k gives exactly the noisy rows of block k
    of the training forward pass (whose mask sees the same keys)."""
    S, D, Hq, Hkv = 4, 8, 4, 2
    for L, k in ((16, 0), (16, 2), (16, 3), (14, 3)):   # L=14: a shorter last block
        Q, K, V = _rand((1, Hq, 2 * L, D), 50 + k), _rand((1, Hkv, 2 * L, D), 60 + k), _rand((1, Hkv, 2 * L, D), 70 + k)
        O, LSE = oracle.forward(Q, K, V, L, S)
        a, e = k * S, min(L, (k + 1) * S)
        C = L
        Kc = np.zeros((1, Hkv, C, D)); Vc = np.zeros((1, Hkv, C, D))
        Kc[:, :, :a] = K[:, :, L:L + a]
        Vc[:, :, :a] = V[:, :, L:L + a]
        Od, LSEd = oracle.decode_forward(Q[:, :, a:e], Kc, Vc, K[:, :, a:e], V[:, :, a:e], [a])
        np.testing.assert_allclose(Od, O[:, :, a:e], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(LSEd, LSE[:, :, a:e], rtol=1e-12, atol=1e-12)


def test_decode_matches_torch_sdpa_over_the_concatenation():
    B, Hq, Hkv, S, D, C = 3, 4, 1, 5, 16, 12
    Q, Kc, Vc = _rand((B, Hq, S, D), 80), _rand((B, Hkv, C, D), 81), _rand((B, Hkv, C, D), 82)
    Kn, Vn = _rand((B, Hkv, S, D), 83), _rand((B, Hkv, S, D), 84)
    lens = [0, 7, 12]
    O, LSE = oracle.decode_forward(Q, Kc, Vc, Kn, Vn, lens)
    for b, n in enumerate(lens):
        kk = torch.from_numpy(np.concatenate([Kc[b, :, :n], Kn[b]], axis=1)).repeat_interleave(Hq // Hkv, 0)
        vv = torch.from_numpy(np.concatenate([Vc[b, :, :n], Vn[b]], axis=1)).repeat_interleave(Hq // Hkv, 0)
        ref = F.scaled_dot_product_attention(torch.from_numpy(Q[b])[None], kk[None], vv[None])[0].numpy()
        np.testing.assert_allclose(O[b], ref, rtol=1e-10, atol=1e-12)
        z = (Q[b] @ np.swapaxes(np.concatenate([Kc[b, :, :n], Kn[b]], axis=1), 1, 2).repeat(Hq // Hkv, 0)) / math.sqrt(D)
        np.testing.assert_allclose(LSE[b], np.log(np.exp(z).sum(-1)), rtol=1e-12, atol=1e-12)


def test_decode_ignores_cache_rows_past_the_length():
    B, Hq, Hkv, S, D, C = 1, 2, 1, 3, 8, 10
    Q, Kc, Vc = _rand((B, Hq, S, D), 90), _rand((B, Hkv, C, D), 91), _rand((B, Hkv, C, D), 92)
    Kn, Vn = _rand((B, Hkv, S, D), 93), _rand((B, Hkv, S, D), 94)
    O1, _ = oracle.decode_forward(Q, Kc, Vc, Kn, Vn, [6])
    Kc[:, :, 6:] = 1e3
    Vc[:, :, 6:] = -1e3
    O2, _ = oracle.decode_forward(Q, Kc, Vc, Kn, Vn, [6])
    np.testing.assert_array_equal(O1, O2)
