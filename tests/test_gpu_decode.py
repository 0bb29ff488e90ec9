"""GPU parity of block decoding over a KV cache against the fp64 oracle.

The oracle (oracle.decode_forward) computes dense softmax attention of each
block's noisy queries over [cache rows 0..len) ; block keys] on the same bf16
values.  Tolerances are those of the training forward pass, whose arithmetic
this path repeats (bf16 operands and probabilities, float32 accumulation):
O max-abs <= 2e-2 and rel-L2 <= 5e-3, LSE max-abs <= 1e-3.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22234_amd import (BD_ATTN_BF16, BD_ATTN_FP32, BdAttnError, bd_attn_decode_fwd,
                                  bd_attn_decode_workspace_bytes, lib)
from paper_2512_22234_amd.workloads import DECODE_WORKLOADS, decode_cache_lens, make_decode_inputs

pytestmark = pytest.mark.gpu

O_MAX, O_REL, LSE_MAX = 2e-2, 5e-3, 1e-3
DEV = torch.device("cuda:0")


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(a, ref):
    return float(np.linalg.norm(a - ref) / max(np.linalg.norm(ref), 1e-30))


def _check(O, LSE, Or, LSEr, tag):
    errs = dict(o_max=float(np.abs(O - Or).max()), o_rel=_rel(O, Or), lse_max=float(np.abs(LSE - LSEr).max()))
    print(f"[decode] {tag} errors {errs}", flush=True)
    assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
    assert errs["lse_max"] <= LSE_MAX, errs


# The key tiles of all items are shared out over 1024 waves: with fewer
# tiles than waves every wave holds at most one tile (every item of more than
# one tile is merged from partial results, waves without tiles in between);
# with more, runs start and end inside items and cross item boundaries.
DECODE_CASES = [
    # B, Hq, Hkv, D, S, capacity, cache lengths
    (3, 4, 2, 64, 4, 200, [0, 37, 200]),                 # empty cache, ragged tile, full cache
    (4, 32, 8, 128, 4, 1100, [1, 100, 513, 1100]),       # the 8B heads; 16 of 32 query rows used
    (2, 16, 1, 128, 4, 300, [299, 64]),                  # G*S = 64: two query tiles per KV head
    (2, 8, 2, 128, 40, 300, [250, 0]),                   # S = 40: two block tiles, three query tiles
    (2, 2, 2, 64, 1, 70, [70, 33]),                      # one-token blocks
    (1, 4, 1, 128, 32, 0, [0]),                          # no cache at all
    (16, 4, 4, 128, 4, 12000, [12000, 3] * 8),           # 12k tiles: runs cross several items
    (300, 4, 2, 64, 2, 64, list(range(0, 600, 2))[:300]),  # more sequences than threads in the scan
]


@pytest.mark.parametrize("B,Hq,Hkv,D,S,C,lens", DECODE_CASES)
def test_decode_matches_oracle(B, Hq, Hkv, D, S, C, lens):
    lens = [min(x, C) for x in lens]
    print(f"[decode] B{B} H{Hq}/{Hkv} D{D} S{S} C{C} lens={lens[:8]}", flush=True)
    q, kc, vc, kn, vn, cl = make_decode_inputs(B, Hq, Hkv, D, S, C, lens, seed=300 + B * S + C)
    o, lse = bd_attn_decode_fwd(*(t.to(DEV) for t in (q, kc, vc, kn, vn, cl)))
    torch.cuda.synchronize()
    Or, LSEr = oracle.decode_forward(*(t.double().numpy() for t in (q, kc, vc, kn, vn)), lens)
    _check(_np(o), _np(lse), Or, LSEr, f"B{B} S{S} C{C}")


def test_decode_cache_lengths_are_clamped():
    """Lengths beyond the capacity act as the capacity, negative ones as 0."""
    B, Hq, Hkv, D, S, C = 2, 4, 2, 64, 4, 96
    q, kc, vc, kn, vn, _ = make_decode_inputs(B, Hq, Hkv, D, S, C, [0, 0], seed=41)
    cl = torch.tensor([C + 50, -7], dtype=torch.int32, device=DEV)
    o, lse = bd_attn_decode_fwd(*(t.to(DEV) for t in (q, kc, vc, kn, vn)), cl)
    torch.cuda.synchronize()
    Or, LSEr = oracle.decode_forward(*(t.double().numpy() for t in (q, kc, vc, kn, vn)), [C, 0])
    _check(_np(o), _np(lse), Or, LSEr, "clamped")


def test_decode_ignores_cache_rows_past_the_length():
    B, Hq, Hkv, D, S, C = 2, 8, 2, 128, 4, 160
    q, kc, vc, kn, vn, cl = (t.to(DEV) for t in make_decode_inputs(B, Hq, Hkv, D, S, C, [70, 131], seed=42))
    o1, l1 = bd_attn_decode_fwd(q, kc, vc, kn, vn, cl)
    kc2, vc2 = kc.clone(), vc.clone()
    kc2[0, :, 70:] = 1e4
    vc2[0, :, 70:] = float("nan")
    kc2[1, :, 131:] = -1e4
    vc2[1, :, 131:] = float("inf")
    o2, l2 = bd_attn_decode_fwd(q, kc2, vc2, kn, vn, cl)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_decode_deterministic_and_partition_invariant():
    """Bitwise reproducible; and a sequence's result depends on the others
    only through where the runs of waves cut its keys (float32 rounding)."""
    B, Hq, Hkv, D, S, C = 4, 32, 8, 128, 4, 2048
    lens = [2048, 1500, 33, 700]
    q, kc, vc, kn, vn, cl = (t.to(DEV) for t in make_decode_inputs(B, Hq, Hkv, D, S, C, lens, seed=43))
    o1, l1 = bd_attn_decode_fwd(q, kc, vc, kn, vn, cl)
    o2, l2 = bd_attn_decode_fwd(q, kc, vc, kn, vn, cl)
    # sequence 0 alone: the same keys, cut into different runs
    o3, l3 = bd_attn_decode_fwd(q[:1].contiguous(), kc[:1].contiguous(), vc[:1].contiguous(), kn[:1].contiguous(),
                                vn[:1].contiguous(), cl[:1].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert float((o3.float() - o1[:1].float()).abs().max()) <= 1e-2
    assert float((l3 - l1[:1]).abs().max()) <= 1e-4


def test_decode_full_workload_sampled_rows():
    """The measured rollout workload at full size (64 sequences, caches of
    512..8192 tokens), in the launch configuration the benchmark times;
    sampled (sequence, head) pairs against the oracle."""
    w = DECODE_WORKLOADS["8b_decode"]
    lens = decode_cache_lens(w["B"], w["seed"], w["lo"], w["hi"])
    q, kc, vc, kn, vn, cl = make_decode_inputs(w["B"], w["Hq"], w["Hkv"], w["D"], w["S"], w["capacity"], lens,
                                               seed=w["seed"], device="cuda")
    o, lse = bd_attn_decode_fwd(q, kc, vc, kn, vn, cl)
    torch.cuda.synchronize()
    G = w["Hq"] // w["Hkv"]
    longest = int(np.argmax(lens))
    picks = [(longest, 0), (longest, w["Hq"] - 1), (int(np.argmin(lens)), 5), (7, 13), (31, 22), (63, 31)]
    for b, h in picks:
        n, g = lens[b], h // G
        sl = lambda t, rows: t[b:b + 1, g:g + 1, :rows].double().cpu().numpy()  # noqa: E731
        Or, LSEr = oracle.decode_forward(q[b:b + 1, h:h + 1].double().cpu().numpy(), sl(kc, n), sl(vc, n),
                                         sl(kn, w["S"]), sl(vn, w["S"]), [n])
        _check(_np(o[b:b + 1, h:h + 1]), _np(lse[b:b + 1, h:h + 1]), Or, LSEr, f"full b{b} h{h} len{n}")


def test_decode_invalid_arguments():
    B, Hq, Hkv, D, S, C = 1, 4, 2, 64, 4, 64
    q, kc, vc, kn, vn, cl = (t.to(DEV) for t in make_decode_inputs(B, Hq, Hkv, D, S, C, [10], seed=44))
    assert bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, C, BD_ATTN_FP32) == 0
    assert bd_attn_decode_workspace_bytes(B, S, 3, Hkv, D, C, BD_ATTN_BF16) == 0
    # a workspace below the size needed is refused before any launch
    need = bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, C, BD_ATTN_BF16)
    assert need > 0
    ws = torch.empty(need - 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(BdAttnError) as e:
        bd_attn_decode_fwd(q, kc, vc, kn, vn, cl, workspace=ws)
    assert e.value.status == 3
    # float32 inputs are not a decode dtype (status 2 from the library)
    import ctypes
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, S), dtype=torch.float32, device=DEV)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    st = lib().bd_attn_decode_fwd(*(ctypes.c_void_p(t.data_ptr()) for t in (q, kc, vc, kn, vn, cl)), B, S, Hq,
                                  Hkv, D, C, 0.0, BD_ATTN_FP32, ctypes.c_void_p(o.data_ptr()),
                                  ctypes.c_void_p(lse.data_ptr()), ctypes.c_void_p(ws.data_ptr()), need, None)
    assert st == 2
