"""GPU parity of the LM-head log-probability calls (bd_lce_fwd / bd_lce_bwd /
bd_lce_objective) against the fp64 oracle (oracle/lce_oracle.py) on the same
bf16 inputs.

Tolerances follow the arithmetic: logits are exact bf16 products summed in
float32 (relative error ~1e-6 of the logit scale), so LSE and logp are held
to 1e-3 absolute like the attention LSE; g = dlogp (onehot - p) is rounded
to bf16 before the two gradient products and dH, dW are written in bf16, so
they are held to 1e-2 relative L2 like the attention gradients.  The
objective kernel is float32 elementwise arithmetic: 1e-5 relative.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22234_amd import (BD_ATTN_FP32, BD_LCE_CE, BD_LCE_DIPO, BdAttnError, bd_lce_bwd, bd_lce_fwd,
                                  bd_lce_objective, bd_lce_workspace_bytes, lib, lm_head_logprobs)
from paper_2512_22234_amd.workloads import LCE_WORKLOADS, make_lce_inputs

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
LP_MAX, G_REL = 1e-3, 1e-2


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(a, ref):
    return float(np.linalg.norm(a - ref) / max(np.linalg.norm(ref), 1e-30))


LCE_CASES = [
    # N, V, Dm
    (1, 256, 256),        # one position, one vocabulary tile
    (100, 1000, 256),     # ragged tiles on both sides
    (300, 4133, 512),     # several vocabulary tiles, ragged last one
    (513, 2048, 768),     # ragged position tile
    (64, 300, 256),       # a vocabulary tile with 44 of 256 rows
]


@pytest.mark.parametrize("N,V,Dm", LCE_CASES)
def test_lce_matches_oracle(N, V, Dm):
    print(f"[lce] N{N} V{V} Dm{Dm}", flush=True)
    h, w, t = make_lce_inputs(N, V, Dm, seed=400 + N + V)
    if N > 1:
        t[::7] = -1  # some positions are not scored
    c = torch.randn(N, generator=torch.Generator().manual_seed(N), dtype=torch.float32)
    hd, wd, td, cd = h.to(DEV), w.to(DEV), t.to(DEV), c.to(DEV)
    lse, logp = bd_lce_fwd(hd, wd, td)
    dh, dw = bd_lce_bwd(hd, wd, td, lse, cd)
    torch.cuda.synchronize()
    H, W, T = h.double().numpy(), w.double().numpy(), t.numpy()
    lp_r, lse_r = oracle.lm_head_logprobs(H, W, T)
    dH_r, dW_r = oracle.lm_head_backward(H, W, T, c.double().numpy())
    errs = dict(lse=float(np.abs(_np(lse) - lse_r).max()), logp=float(np.abs(_np(logp) - lp_r).max()),
                dh=_rel(_np(dh), dH_r), dw=_rel(_np(dw), dW_r))
    print(f"[lce] errors {errs}", flush=True)
    assert errs["lse"] <= LP_MAX and errs["logp"] <= LP_MAX, errs
    assert errs["dh"] <= G_REL and errs["dw"] <= G_REL, errs
    unscored = T < 0
    assert np.all(_np(logp)[unscored] == 0) and np.all(_np(dh)[unscored] == 0)


@pytest.mark.parametrize("N,V,Dm", [(100, 1000, 256), (513, 2048, 768)])
def test_lce_kept_logits_match_recompute(N, V, Dm):
    """The backward from kept logits agrees with the recomputing one and with
    the oracle; the kept logits themselves are the oracle's logits."""
    from paper_2512_22234_amd import bd_lce_logits_bytes
    h, w, t = make_lce_inputs(N, V, Dm, seed=500 + N)
    t[::5] = -1
    c = torch.randn(N, generator=torch.Generator().manual_seed(7), dtype=torch.float32)
    hd, wd, td, cd = h.to(DEV), w.to(DEV), t.to(DEV), c.to(DEV)
    keep = torch.empty(bd_lce_logits_bytes(N, V, Dm) // 4, dtype=torch.float32, device=DEV)
    lse, logp = bd_lce_fwd(hd, wd, td, logits=keep)
    lse2, logp2 = bd_lce_fwd(hd, wd, td)
    dh_k, dw_k = bd_lce_bwd(hd, wd, td, lse, cd, logits=keep)
    dh_r, dw_r = bd_lce_bwd(hd, wd, td, lse, cd)
    torch.cuda.synchronize()
    assert torch.equal(lse, lse2) and torch.equal(logp, logp2)  # keeping the logits changes nothing else
    H, W = h.double().numpy(), w.double().numpy()
    Vp = keep.numel() // N
    kept = keep.view(N, Vp)[:, :V].double().cpu().numpy()
    assert np.abs(kept - H @ W.T).max() <= 1e-4 * max(1.0, np.abs(H @ W.T).max())
    dH_o, dW_o = oracle.lm_head_backward(H, W, t.numpy(), c.double().numpy())
    for got, want in ((dh_k, dH_o), (dw_k, dW_o), (dh_r, dH_o), (dw_r, dW_o)):
        assert _rel(_np(got), want) <= G_REL
    assert _rel(_np(dh_k), _np(dh_r)) <= 2e-3 and _rel(_np(dw_k), _np(dw_r)) <= 2e-3


def test_lce_deterministic():
    h, w, t = (x.to(DEV) for x in make_lce_inputs(700, 3000, 512, seed=41))
    c = torch.randn(700, device=DEV)
    r1 = bd_lce_fwd(h, w, t)
    g1 = bd_lce_bwd(h, w, t, r1[0], c)
    r2 = bd_lce_fwd(h, w, t)
    g2 = bd_lce_bwd(h, w, t, r2[0], c)
    torch.cuda.synchronize()
    for a, b in zip(r1 + g1, r2 + g2):
        assert torch.equal(a, b)


def test_lce_autograd_matches_oracle():
    N, V, Dm = 200, 1500, 256
    h, w, t = make_lce_inputs(N, V, Dm, seed=42)
    c = torch.randn(N, generator=torch.Generator().manual_seed(3), dtype=torch.float32)
    hd = h.to(DEV).requires_grad_()
    wd = w.to(DEV).requires_grad_()
    logp = lm_head_logprobs(hd, wd, t.to(DEV))
    (logp * c.to(DEV)).sum().backward()
    torch.cuda.synchronize()
    dH_r, dW_r = oracle.lm_head_backward(h.double().numpy(), w.double().numpy(), t.numpy(), c.double().numpy())
    assert _rel(_np(hd.grad), dH_r) <= G_REL and _rel(_np(wd.grad), dW_r) <= G_REL


def test_lce_objectives_match_oracle():
    N = 1000
    g = torch.Generator().manual_seed(4)
    logp = -torch.rand(N, generator=g) * 6
    old = logp + torch.randn(N, generator=g) * 0.3  # ratios on both sides of the clip range
    ref = logp + torch.randn(N, generator=g) * 0.5
    adv = torch.randn(N, generator=g)
    wgt = torch.rand(N, generator=g) * (torch.arange(N) % 4 != 0)
    d = {k: v.to(DEV) for k, v in dict(logp=logp, old=old, ref=ref, adv=adv, w=wgt).items()}
    l0, dl0 = bd_lce_objective(d["logp"], d["w"], BD_LCE_CE)
    l1, dl1 = bd_lce_objective(d["logp"], d["w"], BD_LCE_DIPO, logp_old=d["old"], logp_ref=d["ref"], adv=d["adv"],
                               eps=0.2, beta=0.04)
    l2, dl2 = bd_lce_objective(d["logp"], d["w"], BD_LCE_DIPO, logp_old=d["logp"], adv=d["adv"], eps=0.2, beta=0.0)
    torch.cuda.synchronize()
    n = {k: v.double().numpy() for k, v in dict(logp=logp, old=old, ref=ref, adv=adv, w=wgt).items()}
    r0 = oracle.masked_ce_objective(n["logp"], n["w"])
    r1 = oracle.dipo_objective(n["logp"], n["old"], n["ref"], n["adv"], n["w"], 0.2, 0.04)
    r2 = oracle.dipo_objective(n["logp"], n["logp"], None, n["adv"], n["w"], 0.2, 0.0)
    for got, want in ((l0, r0[0]), (dl0, r0[1]), (l1, r1[0]), (dl1, r1[1]), (l2, r2[0]), (dl2, r2[1])):
        np.testing.assert_allclose(_np(got), want, rtol=1e-5, atol=1e-6)


def test_lce_full_size_sampled():
    """The 8B LM head at full size (4096 positions, 151,936 vocabulary rows,
    hidden 4096), in the launch configuration the benchmark times; logp and
    LSE of sampled positions, and the gradients of a loss on those positions
    only (dH entirely, dW on sampled vocabulary rows and in its column sums)."""
    c = LCE_WORKLOADS["8b_lm_head"]
    N, V, Dm = c["N"], c["V"], c["Dm"]
    h, w, t = make_lce_inputs(N, V, Dm, seed=c["seed"], device="cuda")
    rows = [0, 1, 777, 2048, 4000, N - 1]
    dl = torch.zeros(N, device=DEV)
    dl[rows] = torch.tensor([1.0, -0.5, 2.0, 0.25, -1.5, 0.75], device=DEV)
    lse, logp = bd_lce_fwd(h, w, t)
    dh, dw = bd_lce_bwd(h, w, t, lse, dl)
    torch.cuda.synchronize()
    T = t.cpu().numpy()
    vocab_rows = sorted(set(T[rows].tolist()) | {0, 1, 5000, 75000, 151935})
    Hn = h.float().cpu().numpy()
    Wn = w.float().cpu().numpy()
    lp_r, lse_r, dH_r, dW_r = oracle.lm_head_sampled(Hn, Wn, T, dl.cpu().numpy(), rows, vocab_rows)
    assert np.abs(_np(lse[rows]) - lse_r).max() <= LP_MAX
    assert np.abs(_np(logp[rows]) - lp_r).max() <= LP_MAX
    dh_np = _np(dh)
    assert _rel(dh_np[rows], dH_r) <= G_REL
    others = np.setdiff1d(np.arange(N), rows)
    assert np.all(dh_np[others] == 0)
    assert _rel(_np(dw[vocab_rows]), dW_r) <= G_REL
    # every row of g sums to zero over the vocabulary, so dW's column sums vanish
    # up to bf16 rounding of g and dW
    col = _np(dw.float().sum(0))
    assert np.abs(col).max() <= 1e-2 * np.abs(_np(dw)).sum(0).max()


def test_lce_full_size_kept_logits_match_recompute():
    """The kept-logits variants at the full 8B LM-head shape (the forward that
    also stores the float32 logits, and the backward that forms g from them):
    LSE and logp are bitwise those of the plain forward, the kept logits of
    sampled positions are H W^T, and the gradients agree with the recomputing
    backward to the bf16 rounding of g."""
    from paper_2512_22234_amd import bd_lce_logits_bytes
    c = LCE_WORKLOADS["8b_lm_head"]
    N, V, Dm = c["N"], c["V"], c["Dm"]
    h, w, t = make_lce_inputs(N, V, Dm, seed=c["seed"], device="cuda")
    dl = torch.randn(N, generator=torch.Generator(device="cuda").manual_seed(3), device=DEV) / N
    keep = torch.empty(bd_lce_logits_bytes(N, V, Dm) // 4, dtype=torch.float32, device=DEV)
    lse_k, logp_k = bd_lce_fwd(h, w, t, logits=keep)
    lse, logp = bd_lce_fwd(h, w, t)
    dh_k, dw_k = bd_lce_bwd(h, w, t, lse_k, dl, logits=keep)
    dh, dw = bd_lce_bwd(h, w, t, lse, dl)
    torch.cuda.synchronize()
    assert torch.equal(lse_k, lse) and torch.equal(logp_k, logp)
    rows = [0, 1, 2047, N - 1]
    Vp = keep.numel() // N
    kept = keep.view(N, Vp)[rows, :V].double().cpu().numpy()
    want = h[rows].double().cpu().numpy() @ w.double().cpu().numpy().T
    assert np.abs(kept - want).max() <= 1e-4 * max(1.0, np.abs(want).max())
    assert np.all(keep.view(N, Vp)[rows, V:].cpu().numpy() == 0)  # the zero rows' logits
    def rel(x, y):  # relative L2 on the device (the full gradients are large)
        x, y = x.float(), y.float()
        return float(torch.linalg.vector_norm(x - y) / torch.linalg.vector_norm(y))
    assert rel(dh_k, dh) <= 2e-3 and rel(dw_k, dw) <= 2e-3


def test_lce_invalid_arguments():
    h, w, t = (x.to(DEV) for x in make_lce_inputs(8, 300, 256, seed=5))
    assert bd_lce_workspace_bytes(8, 300, 200, 0) == 0           # Dm not a multiple of 256
    assert bd_lce_workspace_bytes(0, 300, 256, 0) == 0
    assert bd_lce_workspace_bytes(8, 300, 256, 0, BD_ATTN_FP32) == 0
    need = bd_lce_workspace_bytes(8, 300, 256, 0)
    ws = torch.empty(need - 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(BdAttnError) as e:
        bd_lce_fwd(h, w, t, workspace=ws)
    assert e.value.status == 3
    lse = torch.empty(8, device=DEV)
    logp = torch.empty(8, device=DEV)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    st = lib().bd_lce_fwd(ctypes.c_void_p(h.data_ptr()), ctypes.c_void_p(w.data_ptr()), ctypes.c_void_p(t.data_ptr()),
                          8, 300, 256, BD_ATTN_FP32, ctypes.c_void_p(lse.data_ptr()),
                          ctypes.c_void_p(logp.data_ptr()), None, ctypes.c_void_p(ws.data_ptr()), need, None)
    assert st == 2
    with pytest.raises(BdAttnError) as e:
        bd_lce_objective(lse, lse, BD_LCE_DIPO)  # DiPO needs logp_old and adv
    assert e.value.status == 1
