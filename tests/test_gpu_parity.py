"""GPU parity: the HIP library (through its C-ABI binding) against the fp64 oracle
on identical seeded inputs.

Tolerances (bf16 inputs, fp32 accumulation): forward O max-abs <= 2e-2 and
rel-L2 <= 5e-3, LSE max-abs <= 1e-3, dQ/dK/dV rel-L2 <= 1e-2 each.  The
oracle sees the exact bf16 values the kernels see (float32 inputs are
rounded to bf16 first, as the library does).

Small and medium shapes are compared element by element in full; the 8B
shape on every GQA group (all of its outputs); the block-size-sweep shapes on
two whole GQA groups each; the long shape on sampled query rows and key rows,
each evaluated exactly by the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_22234_amd import bd_attn, bd_attn_bwd, bd_attn_fwd
from paper_2512_22234_amd.workloads import WORKLOADS, make_inputs, make_random_case

pytestmark = pytest.mark.gpu

O_MAX, O_REL, LSE_MAX, G_REL = 2e-2, 5e-3, 1e-3, 1e-2
DEV = torch.device("cuda:0")


def _say(msg):
    print(msg, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(a, ref):
    return float(np.linalg.norm(a - ref) / max(np.linalg.norm(ref), 1e-30))


def _oracle_inputs(q, k, v, do):
    # the values the kernels compute on: bf16 (float32 inputs are rounded)
    return [t.to(torch.bfloat16).double().numpy() for t in (q, k, v, do)]


def run_gpu(q, k, v, do, L, S, scale=None):
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o, lse = bd_attn_fwd(qd, kd, vd, L, S, scale)
    dq, dk, dv = bd_attn_bwd(dod, qd, kd, vd, o, lse, L, S, scale)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


def check_full(q, k, v, do, L, S, scale=None, label=""):
    _say(f"[parity] {label} shape q={tuple(q.shape)} k={tuple(k.shape)} L={L} S={S} dtype={q.dtype}")
    o, lse, dq, dk, dv = run_gpu(q, k, v, do, L, S, scale)
    Q, K, V, dO = _oracle_inputs(q, k, v, do)
    Or, LSEr = oracle.forward(Q, K, V, L, S, scale)
    dQr, dKr, dVr = oracle.backward(dO, Q, K, V, L, S, scale)
    O, LSE = _np(o), _np(lse)
    errs = dict(o_max=float(np.abs(O - Or).max()), o_rel=_rel(O, Or), lse_max=float(np.abs(LSE - LSEr).max()),
                dq_rel=_rel(_np(dq), dQr), dk_rel=_rel(_np(dk), dKr), dv_rel=_rel(_np(dv), dVr))
    _say(f"[parity] {label} errors {errs}")
    assert np.isfinite(O).all() and np.isfinite(LSE).all()
    assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
    assert errs["lse_max"] <= LSE_MAX, errs
    assert errs["dq_rel"] <= G_REL and errs["dk_rel"] <= G_REL and errs["dv_rel"] <= G_REL, errs
    return errs


def check_groups(w, groups, label):
    q, k, v, do = make_inputs(w)
    _say(f"[parity] {label} {w.describe()} groups={groups}")
    o, lse, dq, dk, dv = run_gpu(q, k, v, do, w.L, w.S)
    O, LSE, dQ, dK, dV = (_np(t) for t in (o, lse, dq, dk, dv))
    Q, K, V, dO = _oracle_inputs(q, k, v, do)
    G = w.Hq // w.Hkv
    heads = [(b, h) for b, g in groups for h in range(g * G, (g + 1) * G)]
    Or, LSEr = oracle.forward(Q, K, V, w.L, w.S, heads=heads)
    dQr, dKr, dVr = oracle.backward(dO, Q, K, V, w.L, w.S, groups=groups)
    for b, g in groups:
        hs = slice(g * G, (g + 1) * G)
        errs = dict(o_max=float(np.abs(O[b, hs] - Or[b, hs]).max()), o_rel=_rel(O[b, hs], Or[b, hs]),
                    lse_max=float(np.abs(LSE[b, hs] - LSEr[b, hs]).max()),
                    dq_rel=_rel(dQ[b, hs], dQr[b, hs]), dk_rel=_rel(dK[b, g], dKr[b, g]),
                    dv_rel=_rel(dV[b, g], dVr[b, g]))
        _say(f"[parity] {label} group (b={b}, hkv={g}) errors {errs}")
        assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
        assert errs["lse_max"] <= LSE_MAX, errs
        assert max(errs["dq_rel"], errs["dk_rel"], errs["dv_rel"]) <= G_REL, errs
    # every other output must at least be finite
    assert all(np.isfinite(t).all() for t in (O, LSE, dQ, dK, dV))


# ------------------------------------------------------------------ configs

def test_tiny_fp32_config():
    w = WORKLOADS["tiny"]
    q, k, v, do = make_inputs(w)
    check_full(q, k, v, do, w.L, w.S, label="tiny")
    # information only: error against the unrounded float32 inputs (input
    # rounding alone exceeds the LSE bound, so parity binds on rounded values)
    o, lse, *_ = run_gpu(q, k, v, do, w.L, w.S)
    O32, LSE32 = oracle.forward(q.double().numpy(), k.double().numpy(), v.double().numpy(), w.L, w.S)
    _say(f"[parity] tiny vs unrounded fp32 inputs: o_rel={_rel(_np(o), O32):.2e} "
         f"lse_max={np.abs(_np(lse) - LSE32).max():.2e}")


def test_small_config_full():
    w = WORKLOADS["small"]
    q, k, v, do = make_inputs(w)
    check_full(q, k, v, do, w.L, w.S, label="small")


@pytest.mark.parametrize("b", [0, 1])
def test_8b_config_all_groups(b):
    """Every (batch, KV head) group of the 8B workload, element by element:
    one batch entry (8 groups, 32 query heads) per test."""
    w = WORKLOADS["8b"]
    check_groups(w, [(b, g) for g in range(w.Hkv)], "8b")


@pytest.mark.parametrize("name", ["8b_s8", "8b_s16", "8b_s32", "8b_s64"])
def test_block_size_sweep_groups(name):
    # the first and the last group of the batch (XCD remap and both batch entries)
    check_groups(WORKLOADS[name], [(0, 0), (1, 7)], name)


def test_long_config_sampled():
    w = WORKLOADS["long"]
    q, k, v, do = make_inputs(w)
    _say(f"[parity] long {w.describe()} sampled rows")
    o, lse, dq, dk, dv = run_gpu(q, k, v, do, w.L, w.S)
    Q, K, V, dO = _oracle_inputs(q, k, v, do)
    L, S, G = w.L, w.S, w.Hq // w.Hkv
    rng = np.random.default_rng(7)
    b, g = 0, 5
    qrows = np.unique(np.concatenate([rng.integers(0, 2 * L, 96), [0, L - 1, L, 2 * L - 1]]))
    # keys whose seers are few enough to evaluate: noisy keys (seen by their own
    # block) and clean keys of the last blocks, plus one clean block mid-way
    krows = np.unique(np.concatenate([rng.integers(0, L, 48), np.arange(2 * L - 24, 2 * L),
                                      np.arange(L + 6000, L + 6008)]))
    ref = oracle.sampled(dO, Q, K, V, L, S, b, g, qrows, krows)
    hs = slice(g * G, (g + 1) * G)
    O, LSE, dQ = _np(o)[b, hs][:, qrows], _np(lse)[b, hs][:, qrows], _np(dq)[b, hs][:, qrows]
    dK, dV = _np(dk)[b, g, krows], _np(dv)[b, g, krows]
    errs = dict(o_max=float(np.abs(O - ref["O"]).max()), o_rel=_rel(O, ref["O"]),
                lse_max=float(np.abs(LSE - ref["LSE"]).max()), dq_rel=_rel(dQ, ref["dQ"]),
                dk_rel=_rel(dK, ref["dK"]), dv_rel=_rel(dV, ref["dV"]))
    _say(f"[parity] long errors {errs}")
    assert errs["o_max"] <= O_MAX and errs["o_rel"] <= O_REL, errs
    assert errs["lse_max"] <= LSE_MAX, errs
    assert max(errs["dq_rel"], errs["dk_rel"], errs["dv_rel"]) <= G_REL, errs
    for t in (o, lse, dq, dk, dv):
        assert torch.isfinite(t).all()


def test_long_config_scalar_outliers_sampled():
    """The weaker reading of the outlier recipe: +8 on 1% of individual K entries."""
    w = WORKLOADS["long"]
    q, k, v, do = make_inputs(w, outlier_mode="scalars")
    _say(f"[parity] long (scalar outliers) {w.describe()}")
    o, lse, dq, dk, dv = run_gpu(q, k, v, do, w.L, w.S)
    Q, K, V, dO = _oracle_inputs(q, k, v, do)
    qrows = np.arange(w.L - 40, w.L + 40)
    krows = np.arange(2 * w.L - 16, 2 * w.L)
    ref = oracle.sampled(dO, Q, K, V, w.L, w.S, 0, 2, qrows, krows)
    G = w.Hq // w.Hkv
    O = _np(o)[0, 2 * G:3 * G][:, qrows]
    LSE = _np(lse)[0, 2 * G:3 * G][:, qrows]
    assert np.abs(O - ref["O"]).max() <= O_MAX and _rel(O, ref["O"]) <= O_REL
    assert np.abs(LSE - ref["LSE"]).max() <= LSE_MAX
    assert _rel(_np(dq)[0, 2 * G:3 * G][:, qrows], ref["dQ"]) <= G_REL
    assert _rel(_np(dk)[0, 2, krows], ref["dK"]) <= G_REL
    assert _rel(_np(dv)[0, 2, krows], ref["dV"]) <= G_REL


# ------------------------------------------------------------- edge cases

EDGE = [
    # B, Hq, Hkv, D, L, S
    (1, 1, 1, 64, 1, 1),        # single token per half
    (1, 2, 1, 64, 3, 2),        # S does not divide L, tiny
    (1, 1, 1, 128, 17, 4),      # ragged everything
    (2, 4, 2, 64, 100, 7),      # S does not divide L, GQA 2
    (1, 4, 1, 128, 129, 4),     # one row past a 128 tile
    (1, 2, 2, 128, 130, 130),   # S = L: halves unmasked
    (1, 2, 1, 64, 64, 1000),    # S > L behaves as S = L
    (1, 4, 4, 128, 200, 1),     # S = 1
    (2, 8, 2, 128, 256, 16),    # several full tiles, GQA 4
    (1, 4, 1, 64, 300, 64),     # ragged, large blocks
    (1, 2, 1, 128, 513, 3),     # several tiles + ragged tail
    (1, 3, 1, 64, 100, 4),      # odd GQA ratio (the split walk halves are uneven)
    (1, 6, 2, 128, 384, 8),     # GQA 3, several key tiles
]


@pytest.mark.parametrize("B,Hq,Hkv,D,L,S", EDGE)
def test_edge_shapes(B, Hq, Hkv, D, L, S):
    q, k, v, do = make_random_case(B, Hq, Hkv, D, L, S, seed=100 + L)
    check_full(q, k, v, do, L, S, label=f"edge B{B} H{Hq}/{Hkv} D{D} L{L} S{S}")


def test_custom_scale():
    q, k, v, do = make_random_case(1, 2, 1, 64, 96, 4, seed=11)
    check_full(q, k, v, do, 96, 4, scale=0.2, label="scale=0.2")


def test_fp32_path_matches_bf16_path():
    q, k, v, do = make_random_case(1, 4, 2, 64, 160, 4, seed=12, dtype="fp32", amp=1.0)
    r32 = run_gpu(q, k, v, do, 160, 4)
    r16 = run_gpu(*(t.to(torch.bfloat16) for t in (q, k, v, do)), 160, 4)
    for a, b in zip(r32, r16):
        assert a.dtype == torch.float32
        np.testing.assert_array_equal(_np(a), _np(b))


# --------------------------------------------------------------- robustness

def test_deterministic_bitwise():
    q, k, v, do = make_random_case(2, 8, 2, 128, 384, 4, seed=13)
    r1 = run_gpu(q, k, v, do, 384, 4)
    r2 = run_gpu(q, k, v, do, 384, 4)
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)


def test_guard_bands_untouched():
    """Outputs live inside larger NaN-filled buffers; nothing outside them changes."""
    B, Hq, Hkv, D, L, S = 1, 4, 2, 128, 150, 4
    q, k, v, do = (t.to(DEV) for t in make_random_case(B, Hq, Hkv, D, L, S, seed=14))
    pad = 4096

    def band(shape, dtype):
        n = int(np.prod(shape))
        buf = torch.full((n + 2 * pad,), float("nan"), dtype=dtype, device=DEV)
        return buf, buf[pad:pad + n].view(shape)

    ob, o = band(q.shape, torch.bfloat16)
    lb, lse = band((B, Hq, 2 * L), torch.float32)
    o, lse = bd_attn_fwd(q, k, v, L, S, out=o, lse=lse)
    qb, dq = band(q.shape, torch.bfloat16)
    kb, dk = band(k.shape, torch.bfloat16)
    vb, dv = band(v.shape, torch.bfloat16)
    bd_attn_bwd(do, q, k, v, o, lse, L, S, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    for buf in (ob, lb, qb, kb, vb):
        assert torch.isnan(buf[:pad].float()).all() and torch.isnan(buf[-pad:].float()).all()
        assert torch.isfinite(buf[pad:-pad].float()).all()


def test_non_default_stream():
    q, k, v, do = make_random_case(1, 4, 1, 64, 128, 4, seed=15)
    ref = run_gpu(q, k, v, do, 128, 4)
    s = torch.cuda.Stream(device=DEV)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        o, lse = bd_attn_fwd(qd, kd, vd, 128, 4)
        dq, dk, dv = bd_attn_bwd(dod, qd, kd, vd, o, lse, 128, 4)
    s.synchronize()
    for a, b in zip(ref, (o, lse, dq, dk, dv)):
        assert torch.equal(a, b)


def test_autograd_function():
    q, k, v, do = (t.to(DEV) for t in make_random_case(1, 4, 2, 64, 64, 4, seed=16))
    qa, ka, va = (t.clone().requires_grad_(True) for t in (q, k, v))
    out = bd_attn(qa, ka, va, 64, 4)
    out.backward(do)
    o, lse = bd_attn_fwd(q, k, v, 64, 4)
    dq, dk, dv = bd_attn_bwd(do, q, k, v, o, lse, 64, 4)
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), o)
    assert torch.equal(qa.grad, dq) and torch.equal(ka.grad, dk) and torch.equal(va.grad, dv)


def test_workspace_too_small_raises_on_device():
    from paper_2512_22234_amd import BdAttnError
    q, k, v, do = (t.to(DEV) for t in make_random_case(1, 2, 1, 64, 64, 4, seed=17))
    o, lse = bd_attn_fwd(q, k, v, 64, 4)
    ws = torch.empty(64, dtype=torch.uint8, device=DEV)
    with pytest.raises(BdAttnError) as e:
        bd_attn_bwd(do, q, k, v, o, lse, 64, 4, workspace=ws)
    assert e.value.status == 3
    with pytest.raises(BdAttnError) as e:
        bd_attn_fwd(q.float(), k.float(), v.float(), 64, 4, workspace=ws)
    assert e.value.status == 3
