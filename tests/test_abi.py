"""CPU checks of the C-ABI library: it loads, exports what include/bd_attn.h
declares, its host tile classifier and tile walks agree with the oracle's
explicit mask, and argument validation rejects bad calls before touching the
device (these calls return before any HIP call, so no GPU is needed)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2512_22234_amd as bd
from paper_2512_22234_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bd_attn.h")


def test_library_exports_every_declared_symbol():
    text = open(HEADER).read()
    names = sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(bd_attn_\w+)\s*\(", text, re.M)))
    assert len(names) >= 7, names
    L = _lib.lib()
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings():
    assert bd.bd_attn_version() == 100
    seen = set()
    for st in range(6):
        s = bd.bd_attn_status_string(st)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 6
    assert bd.bd_attn_status_string(99) == "unknown status"


def _brute_classes(L, S, BM, BN):
    M = oracle.visibility_mask(L, S)
    nqt, nkt = -(-L // BM), -(-L // BN)
    out = np.zeros((2 * nqt, 2 * nkt), dtype=np.int8)
    for a in range(2 * nqt):
        qh, i = divmod(a, nqt)
        q0, q1 = qh * L + i * BM, qh * L + min(L, (i + 1) * BM)
        for c in range(2 * nkt):
            kh, j = divmod(c, nkt)
            k0, k1 = kh * L + j * BN, kh * L + min(L, (j + 1) * BN)
            blk = M[q0:q1, k0:k1]
            full_size = (q1 - q0) == BM and (k1 - k0) == BN
            if not blk.any():
                out[a, c] = 0
            elif blk.all() and full_size:
                out[a, c] = 1
            else:
                out[a, c] = 2
    return out


CASES = [(L, S, BM, BN) for L in (1, 2, 5, 16, 33, 64, 100, 130, 257)
         for S in (1, 2, 3, 4, 7, 16, 64, 1000)
         for BM, BN in ((128, 64), (64, 128), (16, 16), (8, 32))]


@pytest.mark.parametrize("L,S,BM,BN", CASES[::3] + [(2048, 4, 128, 64), (2048, 64, 64, 128), (300, 5, 128, 64)])
def test_classifier_matches_explicit_mask(L, S, BM, BN):
    got = bd.bd_attn_classify_tiles_host(L, S, BM, BN)
    want = _brute_classes(L, S, BM, BN)
    # soundness first (a wrong FULL/EMPTY would corrupt results), then exactness
    assert not np.any((got == 1) & (want != 1)), "FULL claimed where a pair is hidden or tile ragged"
    assert not np.any((got == 0) & (want != 0)), "EMPTY claimed where a pair is visible"
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("L,S,BM,BN", CASES[1::3] + [(2048, 4, 128, 64), (2048, 4, 64, 128), (8192, 4, 128, 64),
                                                    (2048, 4, 32, 128), (2048, 64, 32, 128), (300, 5, 32, 128),
                                                    (33, 40, 32, 128), (1, 1, 32, 128)])
def test_tile_walks_visit_each_nonempty_pair_once(L, S, BM, BN):
    cls = bd.bd_attn_classify_tiles_host(L, S, BM, BN)
    visits = bd.bd_attn_visit_lists_host(L, S, BM, BN, False)
    np.testing.assert_array_equal(visits, (cls != 0).astype(np.int8), err_msg="by query tile")
    # the dK/dV walks, with each clean key tile's walk in 2 or 4 parts
    for nsplit in (2, 4):
        visits = bd.bd_attn_visit_lists_host(L, S, BM, BN, True, nsplit)
        np.testing.assert_array_equal(visits, (cls != 0).astype(np.int8), err_msg=f"by key tile, {nsplit} parts")


def test_walk_split_count_is_validated():
    with pytest.raises(bd.BdAttnError):
        bd.bd_attn_visit_lists_host(64, 4, 32, 128, True, 3)


def test_forward_full_prefix_holds_only_full_tiles():
    """The forward and dQ kernels run the leading key tiles of a query tile's
    walk in a loop with no visibility test; the host twin marks a pair of
    that prefix that is not FULL (and any other walk error) with 64.  Swept
    over the kernels' own tiles (128 query rows, 64 keys)."""
    for L in list(range(1, 70)) + [100, 127, 128, 129, 200, 255, 256, 257, 300, 513, 1000, 2048]:
        for S in sorted({1, 2, 3, 4, 5, 7, 8, 16, 31, 32, 33, 64, 100, 128, 129, L, L + 1}):
            visits = bd.bd_attn_visit_lists_host(L, S, 128, 64, False)
            cls = bd.bd_attn_classify_tiles_host(L, S, 128, 64)
            np.testing.assert_array_equal(visits, (cls != 0).astype(np.int8), err_msg=f"L={L} S={S}")


@pytest.mark.parametrize("by_key", [False, True])
def test_kernel_mask_windows_match_oracle_mask(by_key):
    for L in (1, 2, 3, 5, 8, 13, 16, 31, 64):
        for S in range(1, L + 2):
            got = bd.bd_attn_mask_windows_host(L, S, by_key).astype(bool)
            np.testing.assert_array_equal(got, oracle.visibility_mask(L, S), err_msg=f"L={L} S={S}")


@pytest.mark.parametrize("by_key", [False, True])
def test_run_windows_are_the_union_of_row_masks(by_key):
    """The per-wave windows the kernels skip 32-wide blocks with: for every run
    of `group` consecutive rows of a half, exactly the keys (queries) that
    some row of the run sees (is seen by) in the oracle's mask."""
    for L in (1, 3, 8, 13, 31, 64, 100):
        for S in sorted({1, 2, 3, 4, 5, 8, 32, L, L + 1}):
            M = oracle.visibility_mask(L, S)
            if by_key:
                M = M.T  # rows: keys, columns: the queries that see them
            for group in (1, 4, 32):
                want = np.zeros_like(M)
                for h in (0, 1):
                    for r0 in range(0, L, group):
                        rows = slice(h * L + r0, h * L + min(L, r0 + group))
                        want[rows] = M[rows].any(axis=0)
                got = bd.bd_attn_group_windows_host(L, S, by_key, group).astype(bool)
                if by_key:
                    got = got.T
                np.testing.assert_array_equal(got, want, err_msg=f"L={L} S={S} group={group}")


def test_clean_key_groups_are_seen_by_nested_query_sets():
    """The dK/dV kernel skips the blocks of a 32-key group that no query sees;
    its consumer waves, which take two adjacent groups, rely on every query
    that sees a clean key group also seeing the group before it (checked on
    the oracle's mask, run by run)."""
    for L in (1, 3, 8, 31, 33, 64, 100, 200):
        for S in sorted({1, 2, 3, 4, 5, 8, 16, 32, 33, 64, L, L + 1}):
            M = oracle.visibility_mask(L, S).T  # rows: keys, columns: queries that see them
            for r0 in range(0, L - 32, 32):
                first = M[L + r0:L + r0 + 32].any(axis=0)
                second = M[L + r0 + 32:L + min(L, r0 + 64)].any(axis=0)
                assert not (second & ~first).any(), f"L={L} S={S} r0={r0}"


def test_classifier_tile_counts_8b_shape():
    # L=2048, S=4 with 128x128 tiles: per (b, h) 1024 pairs; 240 FULL, 48 PARTIAL, 736 EMPTY
    c = bd.bd_attn_classify_tiles_host(2048, 4, 128, 128)
    assert c.size == 1024
    assert (c == 1).sum() == 240 and (c == 2).sum() == 48 and (c == 0).sum() == 736


def test_workspace_bytes():
    f = bd.bd_attn_workspace_bytes
    assert f(2, 2048, 4, 32, 8, 128, 0, 0) == 0      # bf16 forward needs no workspace
    assert f(2, 2048, 4, 32, 8, 128, 0, 1) > 0
    assert f(1, 64, 4, 1, 1, 64, 1, 0) > 0
    assert f(1, 64, 4, 1, 1, 64, 1, 1) > f(1, 64, 4, 1, 1, 64, 0, 1)
    assert f(2, 2048, 4, 32, 7, 128, 0, 0) == 0      # Hq % Hkv
    assert f(2, 2048, 4, 32, 8, 96, 0, 0) == 0       # D unsupported
    assert f(2, 0, 4, 32, 8, 128, 0, 0) == 0         # L < 1
    assert f(2, 2048, 4, 32, 8, 128, 7, 0) == 0      # dtype


def test_workspace_bytes_follow_the_dkdv_split():
    """bf16 backward workspace = (lse2, delta) per query row + float32 sums of
    nsplit - 1 parts of the clean key tiles' walks (dK and dV of the 128 keys
    of every clean key tile and sequence x KV head, a ragged last tile padded)
    + 32 pairing ints per (clean key tile, sequence x KV head) (each piece
    rounded up to 256 bytes).  Few KV heads x length (the small configuration)
    split each walk in four parts, the 8B one in two."""
    f = bd.bd_attn_workspace_bytes

    def want(B, L, Hq, Hkv, D, nsplit):
        r256 = lambda x: -(-x // 256) * 256
        nkt = -(-L // 128)
        return (r256(B * Hq * 2 * L * 8) + r256((nsplit - 1) * 2 * B * Hkv * nkt * 128 * D * 4)
                + r256(32 * B * Hkv * nkt * 4))

    assert f(4, 1024, 4, 16, 4, 64, 0, 1) == want(4, 1024, 16, 4, 64, 4) == 26_230_784
    assert f(2, 2048, 4, 32, 8, 128, 0, 1) == want(2, 2048, 32, 8, 128, 2) == 35_684_352
    assert f(1, 8192, 4, 32, 8, 128, 0, 1) == want(1, 8192, 32, 8, 128, 2)
    assert f(2, 300, 4, 8, 2, 64, 0, 1) == want(2, 300, 8, 2, 64, 4)       # ragged last key tile


def test_varlen_workspace_bytes_follow_the_dkdv_split():
    """bf16 packed backward workspace = (lse2, delta) per query row + float32 sums
    of nsplit - 1 parts of the clean key tiles' walks (a bound on the key
    tiles of all sequences, T/128 + n, at most n * cdiv(max_L, 128), times
    Hkv; 2 x 128 x D floats each) + the pairing counters (n x Hkv x
    cdiv(max_L, 128) key tiles, 32 ints each)."""
    f = bd.bd_attn_varlen_workspace_bytes
    r256 = lambda x: -(-x // 256) * 256

    def want(n, T, maxL, Hq, Hkv, D, nsplit):
        nkt = -(-maxL // 128)
        slots = min(T // 128 + n, n * nkt) * Hkv
        return r256(Hq * 2 * T * 8) + r256((nsplit - 1) * slots * 2 * 128 * D * 4) + r256(32 * n * Hkv * nkt * 4)

    # the measured packed workload (6 sequences, 4096 tokens, longest 1701): two parts
    assert f(6, 4096, 1701, 4, 32, 8, 128, 0, 1) == want(6, 4096, 1701, 32, 8, 128, 2)
    # few KV heads x tokens: four parts
    assert f(3, 600, 300, 4, 8, 2, 64, 0, 1) == want(3, 600, 300, 8, 2, 64, 4)


# Fake, never-dereferenced device addresses: every call below fails validation
# and returns before any HIP call (the defaults use the float32 path so that
# the workspace is non-empty and the workspace checks are exercised).
A = 1 << 40
SZ = 1 << 32


def _fwd(**kw):
    a = dict(Q=A, K=A + SZ, V=A + 2 * SZ, B=1, L=64, S=4, Hq=2, Hkv=1, D=64, scale=0.0, dtype=1,
             O=A + 3 * SZ, LSE=A + 4 * SZ, ws=A + 5 * SZ, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    L = _lib.lib()
    vp = ctypes.c_void_p
    return L.bd_attn_fwd(vp(a["Q"]), vp(a["K"]), vp(a["V"]), a["B"], a["L"], a["S"], a["Hq"], a["Hkv"],
                         a["D"], a["scale"], a["dtype"], vp(a["O"]), vp(a["LSE"]), vp(a["ws"]),
                         a["ws_bytes"], vp(a["stream"]))


def _bwd(**kw):
    a = dict(dO=A, Q=A + SZ, K=A + 2 * SZ, V=A + 3 * SZ, O=A + 4 * SZ, LSE=A + 5 * SZ, B=1, L=64, S=4,
             Hq=2, Hkv=1, D=64, scale=0.0, dtype=1, dQ=A + 6 * SZ, dK=A + 7 * SZ, dV=A + 8 * SZ,
             ws=A + 9 * SZ, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    L = _lib.lib()
    vp = ctypes.c_void_p
    return L.bd_attn_bwd(vp(a["dO"]), vp(a["Q"]), vp(a["K"]), vp(a["V"]), vp(a["O"]), vp(a["LSE"]),
                         a["B"], a["L"], a["S"], a["Hq"], a["Hkv"], a["D"], a["scale"], a["dtype"],
                         vp(a["dQ"]), vp(a["dK"]), vp(a["dV"]), vp(a["ws"]), a["ws_bytes"], vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(D=96), 2), (dict(D=256), 2), (dict(dtype=3), 2),
    (dict(Hq=3, Hkv=2), 1), (dict(B=0), 1), (dict(L=0), 1), (dict(S=0), 1),
    (dict(L=(1 << 22) + 1), 1),            # beyond 32-bit buffer offsets of one head
    (dict(Q=0), 1), (dict(O=0), 1), (dict(LSE=0), 1), (dict(ws=0), 1),
    (dict(Q=A + 8), 1), (dict(O=A + 3 * SZ + 2), 1), (dict(LSE=A + 4 * SZ + 2), 1),
    (dict(O=A + 16), 1),                   # output overlaps Q
    (dict(LSE=A + 3 * SZ + 64), 1),        # LSE overlaps O
    (dict(ws=A + 2 * SZ + 32), 1),         # workspace overlaps V
    (dict(ws_bytes=16), 3),
    (dict(ws_bytes=16, ws=A + 16), 3),     # too small is reported before overlap
    (dict(scale=float("nan")), 1),
    (dict(dtype=0, ws=0, Q=0), 1),         # bf16: no workspace needed, other checks still apply
])
def test_fwd_validation(kw, status):
    assert _fwd(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(D=32), 2), (dict(Hq=4, Hkv=3), 1), (dict(dO=0), 1), (dict(dV=0), 1), (dict(L=(1 << 22) + 1), 1),
    (dict(dQ=A + SZ + 16), 1),             # dQ overlaps Q
    (dict(dK=A + 6 * SZ + 64), 1),         # dK overlaps dQ
    (dict(dV=A + 5 * SZ), 1),              # dV overlaps LSE
    (dict(dK=A + 7 * SZ + 4), 1),          # misaligned
    (dict(ws_bytes=1000), 3),
])
def test_bwd_validation(kw, status):
    assert _bwd(**kw) == status


def test_decode_workspace_bytes():
    f = bd.bd_attn_decode_workspace_bytes
    # B=64, Hkv=8, one 32-row query tile each (G*S = 16): 512 items, a 16-byte
    # descriptor each, then partial slots for up to 1024 + 512 (wave, item) runs
    items = 64 * 8
    assert f(64, 4, 32, 8, 128, 8192, 0) == items * 16 + (1024 + items) * 32 * (128 + 4) * 4
    assert f(2, 4, 4, 2, 64, 0, 0) > 0                       # no cache: the block alone
    for bad in [dict(dtype=1), dict(D=96), dict(Hq=31), dict(C=-1), dict(C=(1 << 22) + 1), dict(S=0), dict(B=0)]:
        a = dict(B=2, S=4, Hq=4, Hkv=2, D=64, C=100, dtype=0)
        a.update(bad)
        assert f(a["B"], a["S"], a["Hq"], a["Hkv"], a["D"], a["C"], a["dtype"]) == 0, bad
    # the kernels count key tiles in int32
    assert f(1 << 16, 4, 64, 64, 128, 1 << 22, 0) == 0


def _dec(**kw):
    a = dict(Q=A, Kc=A + SZ, Vc=A + 2 * SZ, Kn=A + 3 * SZ, Vn=A + 4 * SZ, lens=A + 5 * SZ, B=1, S=4, Hq=2,
             Hkv=1, D=64, C=64, scale=0.0, dtype=0, O=A + 6 * SZ, LSE=A + 7 * SZ,
             ws=A + 8 * SZ, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    vp = ctypes.c_void_p
    return _lib.lib().bd_attn_decode_fwd(
        vp(a["Q"]), vp(a["Kc"]), vp(a["Vc"]), vp(a["Kn"]), vp(a["Vn"]), vp(a["lens"]), a["B"], a["S"], a["Hq"],
        a["Hkv"], a["D"], a["C"], a["scale"], a["dtype"], vp(a["O"]), vp(a["LSE"]),
        vp(a["ws"]), a["ws_bytes"], vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(D=96), 2), (dict(dtype=1), 2),
    (dict(Hq=3, Hkv=2), 1), (dict(B=0), 1), (dict(S=0), 1), (dict(C=(1 << 22) + 1), 1), (dict(C=-1), 1),
    (dict(scale=float("inf")), 1),
    (dict(Q=0), 1), (dict(Kn=0), 1), (dict(lens=0), 1), (dict(O=0), 1), (dict(Kc=0), 1), (dict(ws=0), 1),
    (dict(Q=A + 8), 1), (dict(lens=A + 5 * SZ + 2), 1), (dict(LSE=A + 7 * SZ + 2), 1),
    (dict(O=A + 64), 1),                   # output overlaps Q
    (dict(LSE=A + 5 * SZ), 1),             # LSE overlaps cache_lens
    (dict(ws=A + 6 * SZ + 256), 1),        # workspace overlaps O
    (dict(ws_bytes=64), 3),
])
def test_decode_validation(kw, status):
    assert _dec(**kw) == status


def test_lce_workspace_bytes():
    f = bd.bd_lce_workspace_bytes
    # forward: a (max, sum) pair per position and vocabulary tile of 256
    assert f(4096, 151936, 4096, 0) == 4096 * 594 * 8
    # backward: g as bf16 [N][V rounded up to 256]
    assert f(4096, 151936, 4096, 1) == 4096 * 594 * 256 * 2
    for bad in [dict(N=0), dict(V=0), dict(Dm=128), dict(Dm=300), dict(dtype=1), dict(N=(1 << 22) + 1),
                dict(V=(1 << 22) + 1), dict(Dm=1 << 17)]:
        a = dict(N=8, V=300, Dm=256, dtype=0)
        a.update(bad)
        assert f(a["N"], a["V"], a["Dm"], 0, a["dtype"]) == 0, bad


def _lce_fwd(**kw):
    a = dict(H=A, W=A + SZ, t=A + 2 * SZ, N=8, V=300, Dm=256, dtype=0, lse=A + 3 * SZ, logp=A + 4 * SZ,
             ws=A + 5 * SZ, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    vp = ctypes.c_void_p
    return _lib.lib().bd_lce_fwd(vp(a["H"]), vp(a["W"]), vp(a["t"]), a["N"], a["V"], a["Dm"], a["dtype"],
                                 vp(a["lse"]), vp(a["logp"]), vp(a.get("logits", 0)), vp(a["ws"]), a["ws_bytes"],
                                 vp(a["stream"]))


def _lce_bwd(**kw):
    a = dict(H=A, W=A + SZ, t=A + 2 * SZ, lse=A + 3 * SZ, dl=A + 4 * SZ, N=8, V=300, Dm=256, dtype=0,
             dH=A + 5 * SZ, dW=A + 6 * SZ, ws=A + 7 * SZ, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    vp = ctypes.c_void_p
    return _lib.lib().bd_lce_bwd(vp(a["H"]), vp(a["W"]), vp(a["t"]), vp(a["lse"]), vp(a["dl"]), vp(a.get("logits", 0)),
                                 a["N"], a["V"],
                                 a["Dm"], a["dtype"], vp(a["dH"]), vp(a["dW"]), vp(a["ws"]), a["ws_bytes"],
                                 vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=1), 2), (dict(N=0), 1), (dict(Dm=384), 1), (dict(H=0), 1), (dict(t=0), 1), (dict(ws=0), 1),
    (dict(H=A + 8), 1), (dict(lse=A + 3 * SZ + 2), 1),
    (dict(logp=A + 16), 1),                # output overlaps H
    (dict(ws=A + 3 * SZ + 16), 1),         # workspace overlaps LSE
    (dict(ws_bytes=64), 3),
    (dict(logits=A + 8 * SZ + 4), 1),      # misaligned kept logits
    (dict(logits=A + 16), 1),              # kept logits overlap H
    (dict(logits=A + 5 * SZ), 1),          # kept logits overlap the workspace
])
def test_lce_fwd_validation(kw, status):
    assert _lce_fwd(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=1), 2), (dict(V=0), 1), (dict(dl=0), 1), (dict(dW=0), 1), (dict(dH=A + 5 * SZ + 4), 1),
    (dict(dW=A + SZ + 64), 1),             # dW overlaps W
    (dict(dH=A + 6 * SZ), 1),              # dH overlaps dW
    (dict(ws_bytes=1000), 3),
    (dict(logits=A + 8 * SZ, dW=A + 8 * SZ + 256), 1),   # dW overlaps the kept logits
])
def test_lce_bwd_validation(kw, status):
    assert _lce_bwd(**kw) == status


@pytest.mark.parametrize("kind,eps,beta,old,adv,ref,status", [
    (2, 0.2, 0.0, 1, 1, 1, 1),             # unknown objective
    (1, 0.2, 0.0, 0, 1, 0, 1),             # DiPO without logp_old
    (1, 0.2, 0.1, 1, 1, 0, 1),             # KL without the reference
    (1, -0.1, 0.0, 1, 1, 0, 1),            # negative clip range
    (1, 0.2, float("nan"), 1, 1, 1, 1),
])
def test_lce_objective_validation(kind, eps, beta, old, adv, ref, status):
    vp = ctypes.c_void_p
    p = lambda i, on=1: vp(A + i * SZ if on else 0)  # noqa: E731
    st = _lib.lib().bd_lce_objective(p(0), p(1, old), p(2, ref), p(3, adv), p(4), 8, kind, eps, beta, p(5), p(6),
                                     vp(None))
    assert st == status


def _bwd_noalloc(**kw):
    a = dict(dO=A, Q=A + SZ, K=A + 2 * SZ, V=A + 3 * SZ, O=A + 4 * SZ, LSE=A + 5 * SZ, B=1, L=64, S=4,
             Hq=2, Hkv=1, D=64, scale=0.0, dtype=0, dQ=A + 6 * SZ, dK=A + 7 * SZ, dV=A + 8 * SZ, stream=None)
    a.update(kw)
    vp = ctypes.c_void_p
    return _lib.lib().bd_attn_bwd_noalloc(vp(a["dO"]), vp(a["Q"]), vp(a["K"]), vp(a["V"]), vp(a["O"]),
                                          vp(a["LSE"]), a["B"], a["L"], a["S"], a["Hq"], a["Hkv"], a["D"],
                                          a["scale"], a["dtype"], vp(a["dQ"]), vp(a["dK"]), vp(a["dV"]),
                                          vp(a["stream"]))


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define BD_ATTN_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == bd.BD_ATTN_NOALLOC_SCRATCH_BYTES
    # the long workload's bf16 backward fits, its float32 variant does not
    assert bd.bd_attn_workspace_bytes(1, 8192, 4, 32, 8, 128, 0, 1) <= bd.BD_ATTN_NOALLOC_SCRATCH_BYTES
    assert bd.bd_attn_workspace_bytes(1, 8192, 4, 32, 8, 128, 1, 1) > bd.BD_ATTN_NOALLOC_SCRATCH_BYTES


@pytest.mark.parametrize("kw,status", [
    (dict(D=96), 2), (dict(dtype=3), 2), (dict(Hq=3, Hkv=2), 1), (dict(B=0), 1), (dict(L=0), 1),
    (dict(L=(1 << 22) + 1), 1),
    # workspace beyond the scratch array: rejected before any HIP call
    (dict(B=4, L=8192, Hq=32, Hkv=8, D=128), 5), (dict(B=1, L=8192, Hq=32, Hkv=8, D=128, dtype=1), 5),
    (dict(dO=0), 1), (dict(dV=0), 1), (dict(LSE=A + 5 * SZ + 2), 1), (dict(dK=A + 7 * SZ + 4), 1),
])
def test_bwd_noalloc_validation(kw, status):
    assert _bwd_noalloc(**kw) == status
