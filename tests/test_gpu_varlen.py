"""GPU parity of the packed-sequence (varlen) calls against the fp64 oracle.

Several [x_t | x_0] sequences of different lengths share one buffer
(cu_seqlens on the device); the oracle builds the explicit packed mask and
computes dense masked attention and its vector-Jacobian product on the same
bf16 values.  Tolerances are those of the single-sequence calls: O max-abs
<= 2e-2 and rel-L2 <= 5e-3, LSE max-abs <= 1e-3, dQ/dK/dV rel-L2 <= 1e-2.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22234_amd import (BdAttnError, bd_attn_bwd, bd_attn_fwd, bd_attn_varlen, bd_attn_varlen_bwd,
                                  bd_attn_varlen_fwd)
from paper_2512_22234_amd.workloads import make_random_case, make_varlen_inputs

pytestmark = pytest.mark.gpu

O_MAX, O_REL, LSE_MAX, G_REL = 2e-2, 5e-3, 1e-3, 1e-2
DEV = torch.device("cuda:0")


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(a, ref):
    return float(np.linalg.norm(a - ref) / max(np.linalg.norm(ref), 1e-30))


def run_varlen(q, k, v, do, cu, max_L, S):
    qd, kd, vd, dod, cud = (t.to(DEV) for t in (q, k, v, do, cu))
    o, lse = bd_attn_varlen_fwd(qd, kd, vd, cud, max_L, S)
    dq, dk, dv = bd_attn_varlen_bwd(dod, qd, kd, vd, o, lse, cud, max_L, S)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


VARLEN_CASES = [
    # lengths, Hq, Hkv, D, S, extra on max_L
    ([37, 0, 130, 5, 256, 1], 4, 2, 64, 4, 0),      # empty and one-token sequences, ragged tiles
    ([300, 129, 64], 2, 1, 128, 8, 0),               # several tiles per sequence, GQA 2
    ([1], 1, 1, 64, 1, 0),                            # a single token
    ([65, 64, 63], 4, 4, 128, 64, 0),                 # S at, above and below the lengths
    ([200, 3, 17], 6, 2, 128, 3, 100),                # GQA 3, S not dividing, max_L above every length
    ([513, 250], 8, 2, 128, 4, 0),                    # several full key tiles, split walks
]


@pytest.mark.parametrize("lengths,Hq,Hkv,D,S,extra", VARLEN_CASES)
def test_varlen_matches_oracle(lengths, Hq, Hkv, D, S, extra):
    print(f"[varlen] lengths={lengths} H{Hq}/{Hkv} D{D} S{S} max_L+{extra}", flush=True)
    q, k, v, do, cu = make_varlen_inputs(lengths, Hq, Hkv, D, seed=200 + sum(lengths))
    o, lse, dq, dk, dv = run_varlen(q, k, v, do, cu, max(lengths) + extra, S)
    Q, K, V, dO = (t.double().numpy() for t in (q, k, v, do))
    Or, LSEr = oracle.varlen_forward(Q, K, V, lengths, S)
    dQr, dKr, dVr = oracle.varlen_backward(dO, Q, K, V, lengths, S)
    O, LSE = _np(o), _np(lse)
    errs = dict(o_max=float(np.abs(O - Or).max()), o_rel=_rel(O, Or), lse_max=float(np.abs(LSE - LSEr).max()),
                dq_rel=_rel(_np(dq), dQr), dk_rel=_rel(_np(dk), dKr), dv_rel=_rel(_np(dv), dVr))
    print(f"[varlen] errors {errs}", flush=True)
    assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
    assert errs["lse_max"] <= LSE_MAX, errs
    assert max(errs["dq_rel"], errs["dk_rel"], errs["dv_rel"]) <= G_REL, errs


def _pack(x):
    """[B, H, 2L, D] -> [H, 2BL, D]: sequence b at packed rows [2bL, 2(b+1)L)."""
    B, H, N, D = x.shape
    return x.permute(1, 0, 2, 3).reshape(H, B * N, D).contiguous()


def test_varlen_equal_lengths_bitwise_equal_to_batched():
    B, Hq, Hkv, D, L, S = 3, 4, 2, 128, 200, 4
    q, k, v, do = (t.to(DEV) for t in make_random_case(B, Hq, Hkv, D, L, S, seed=21))
    o, lse = bd_attn_fwd(q, k, v, L, S)
    dq, dk, dv = bd_attn_bwd(do, q, k, v, o, lse, L, S)
    cu = torch.arange(0, (B + 1) * L, L, dtype=torch.int32, device=DEV)
    ov, lsev = bd_attn_varlen_fwd(_pack(q), _pack(k), _pack(v), cu, L, S)
    dqv, dkv, dvv = bd_attn_varlen_bwd(_pack(do), _pack(q), _pack(k), _pack(v), ov, lsev, cu, L, S)
    torch.cuda.synchronize()
    assert torch.equal(ov, _pack(o))
    assert torch.equal(lsev, lse.permute(1, 0, 2).reshape(Hq, -1))
    for a, b in ((dqv, dq), (dkv, dk), (dvv, dv)):
        assert torch.equal(a, _pack(b))


def test_varlen_deterministic_and_autograd():
    lengths = [130, 40, 300]
    q, k, v, do, cu = (t.to(DEV) for t in make_varlen_inputs(lengths, 4, 1, 64, seed=22))
    r1 = run_varlen(q, k, v, do, cu, 300, 4)
    r2 = run_varlen(q, k, v, do, cu, 300, 4)
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    out = bd_attn_varlen(qa, ka, va, cu, 300, 4)
    out.backward(do)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), r1[0])
    assert torch.equal(qa.grad, r1[2]) and torch.equal(ka.grad, r1[3]) and torch.equal(va.grad, r1[4])


def test_varlen_no_tokens_is_a_no_op():
    q = torch.empty((2, 0, 64), dtype=torch.bfloat16, device=DEV)
    k = torch.empty((1, 0, 64), dtype=torch.bfloat16, device=DEV)
    cu = torch.zeros(3, dtype=torch.int32, device=DEV)
    o, lse = bd_attn_varlen_fwd(q, k, k, cu, 8, 4)
    dq, dk, dv = bd_attn_varlen_bwd(q, q, k, k, o, lse, cu, 8, 4)
    torch.cuda.synchronize()
    assert o.numel() == 0 and dq.numel() == 0 and dk.numel() == 0


def test_varlen_invalid_arguments_raise():
    q, k, v, do, cu = (t.to(DEV) for t in make_varlen_inputs([10, 20], 2, 1, 64, seed=23))
    with pytest.raises(BdAttnError) as e:
        bd_attn_varlen_fwd(q, k, v, cu, 0, 4)       # max_L < 1
    assert e.value.status == 1
    with pytest.raises(BdAttnError) as e:
        bd_attn_varlen_fwd(q, k, v, cu, 20, 0)      # S < 1
    assert e.value.status == 1


def test_varlen_measured_packed_workload():
    """The packed workload the benchmark measures (the 8B heads, 4096 tokens per
    copy split into six sequences of 130..1701 tokens), every output compared:
    each sequence of each GQA group against the single-sequence oracle on that
    sequence's rows (the packed oracle equals it sequence by sequence)."""
    from paper_2512_22234_amd.workloads import VARLEN_WORKLOADS, varlen_lengths
    c = VARLEN_WORKLOADS["8b_packed"]
    lengths = varlen_lengths(c["total"], c["seed"], c["lo"], c["hi"])
    Hq, Hkv, D, S = c["Hq"], c["Hkv"], c["D"], c["S"]
    print(f"[varlen] 8b_packed lengths={lengths} H{Hq}/{Hkv} D{D} S{S}", flush=True)
    q, k, v, do, cu = make_varlen_inputs(lengths, Hq, Hkv, D, c["seed"])
    res = run_varlen(q, k, v, do, cu, max(lengths), S)
    # bitwise reproducible: the parts of each split key-tile walk are added in
    # part order whichever finishes first
    for a, b in zip(res, run_varlen(q, k, v, do, cu, max(lengths), S)):
        assert torch.equal(a, b)
    o, lse, dq, dk, dv = (_np(t) for t in res)
    Q, K, V, dO = (t.double().numpy() for t in (q, k, v, do))
    for i, Li in enumerate(lengths):
        r0, r1 = 2 * int(cu[i]), 2 * int(cu[i + 1])
        one = lambda x: x[None, :, r0:r1]  # [1, H, 2 Li, D]: the sequence as a batch of one
        Or, LSEr = oracle.forward(one(Q), one(K), one(V), Li, S)
        dQr, dKr, dVr = oracle.backward(one(dO), one(Q), one(K), one(V), Li, S)
        errs = dict(o_max=float(np.abs(one(o) - Or).max()), o_rel=_rel(one(o), Or),
                    lse_max=float(np.abs(lse[None, :, r0:r1] - LSEr).max()),
                    dq_rel=max(_rel(one(dq)[:, h], dQr[:, h]) for h in range(Hq)),
                    dk_rel=max(_rel(one(dk)[:, g], dKr[:, g]) for g in range(Hkv)),
                    dv_rel=max(_rel(one(dv)[:, g], dVr[:, g]) for g in range(Hkv)))
        print(f"[varlen] 8b_packed sequence {i} (L={Li}) errors {errs}", flush=True)
        assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
        assert errs["lse_max"] <= LSE_MAX, errs
        assert max(errs["dq_rel"], errs["dk_rel"], errs["dv_rel"]) <= G_REL, errs
