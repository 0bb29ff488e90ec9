"""GPU check of bd_attn_bwd_noalloc, the backward whose workspace is the
library's own scratch array: two calls in a row (the second on a smaller
problem, so it runs on what the first left in the array), each compared
bitwise with bd_attn_bwd on a workspace of its own and with the fp64 oracle
within the parity tolerances (dQ/dK/dV rel-L2 <= 1e-2)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22234_amd import bd_attn_bwd, bd_attn_bwd_noalloc, bd_attn_fwd
from paper_2512_22234_amd.workloads import make_random_case

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
G_REL = 1e-2


def _rel(a, ref):
    a = a.detach().double().cpu().numpy()
    return float(np.linalg.norm(a - ref) / max(np.linalg.norm(ref), 1e-30))


CASES = [
    # B, Hq, Hkv, D, L, S, seed: the second is smaller than the first
    (2, 8, 2, 128, 640, 4, 41),
    (1, 4, 1, 64, 150, 3, 42),
]


def test_noalloc_matches_workspace_backward_twice():
    for B, Hq, Hkv, D, L, S, seed in CASES:
        print(f"[noalloc] B{B} H{Hq}/{Hkv} D{D} L{L} S{S} seed {seed}", flush=True)
        q, k, v, do = make_random_case(B, Hq, Hkv, D, L, S, seed=seed)
        qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
        o, lse = bd_attn_fwd(qd, kd, vd, L, S)
        ref = bd_attn_bwd(dod, qd, kd, vd, o, lse, L, S)
        # outputs filled with NaN first: everything must be written by the call
        out = [torch.full_like(t, float("nan")) for t in ref]
        torch.cuda.synchronize()
        got = bd_attn_bwd_noalloc(dod, qd, kd, vd, o, lse, L, S, *out)
        torch.cuda.synchronize()
        for a, b in zip(got, ref):
            assert torch.equal(a, b)
        Q, K, V, dO = (t.double().numpy() for t in (q, k, v, do))
        dQr, dKr, dVr = oracle.backward(dO, Q, K, V, L, S)
        errs = (_rel(got[0], dQr), _rel(got[1], dKr), _rel(got[2], dVr))
        print(f"[noalloc] rel-L2 dQ/dK/dV {errs}", flush=True)
        assert max(errs) <= G_REL, errs
