"""Seeded synthetic workloads for block-diffusion attention.

This module only describes shapes and draws random numbers; it holds none of
the attention arithmetic, so both the HIP library's tests and the CPU oracle
can take their inputs from it.

The shapes stand in for the paper's training workload (SDAR-8B on math data
with up to 8k-token sequences, Sections 3.1-3.2 and 4.3), whose data and
weights are not available: Q/K/V are N(0,1) draws (times 0.5 for the bf16
shapes), dO is N(0,1), drawn on the host in the fixed order Q, K, V, dO from a
torch CPU generator, then rounded to nearest-even bf16.
"""
from __future__ import annotations

import dataclasses

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    L: int
    S: int
    seed: int
    dtype: str = "bf16"          # storage type of Q/K/V/dO handed to the library
    amp: float = 0.5             # Q/K/V ~ N(0,1) * amp
    k_outlier: float = 0.0       # added to every channel of a fraction of K rows
    outlier_frac: float = 0.0

    @property
    def N(self) -> int:          # packed length 2L
        return 2 * self.L

    def describe(self) -> str:
        return (f"{self.name}: B={self.B} Hq={self.Hq} Hkv={self.Hkv} D={self.D} "
                f"L={self.L} S={self.S} {self.dtype}")


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 1, 64, 64, 4, seed=0, dtype="fp32", amp=1.0),
    "small": Workload("small", 4, 16, 4, 64, 1024, 4, seed=1),
    "8b": Workload("8b", 2, 32, 8, 128, 2048, 4, seed=2),
    "8b_s8": Workload("8b_s8", 2, 32, 8, 128, 2048, 8, seed=3),
    "8b_s16": Workload("8b_s16", 2, 32, 8, 128, 2048, 16, seed=4),
    "8b_s32": Workload("8b_s32", 2, 32, 8, 128, 2048, 32, seed=5),
    "8b_s64": Workload("8b_s64", 2, 32, 8, 128, 2048, 64, seed=6),
    "long": Workload("long", 1, 32, 8, 128, 8192, 4, seed=7,
                     k_outlier=8.0, outlier_frac=0.01),
}


def torch_dtype(name: str) -> torch.dtype:
    return {"bf16": torch.bfloat16, "fp32": torch.float32}[name]


def make_inputs(w: Workload, seed: int | None = None, outlier_mode: str = "rows"):
    """Return CPU tensors q, k, v, do in the workload's storage dtype.

    outlier_mode: "rows" adds k_outlier to every channel of
    ceil(outlier_frac * B*Hkv*2L) randomly chosen K rows (both halves);
    "scalars" adds it to that fraction of individual K entries instead.
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(w.seed if seed is None else seed)
    N = w.N
    q = torch.randn((w.B, w.Hq, N, w.D), generator=g) * w.amp
    k = torch.randn((w.B, w.Hkv, N, w.D), generator=g) * w.amp
    v = torch.randn((w.B, w.Hkv, N, w.D), generator=g) * w.amp
    do = torch.randn((w.B, w.Hq, N, w.D), generator=g)
    if w.k_outlier and w.outlier_frac > 0:
        if outlier_mode == "rows":
            rows = k.shape[0] * k.shape[1] * N
            n = -(-int(round(w.outlier_frac * rows * 1e6)) // 1_000_000)
            idx = torch.randperm(rows, generator=g)[:n]
            flat = k.view(rows, w.D)
            flat[idx] += w.k_outlier
        elif outlier_mode == "scalars":
            total = k.numel()
            n = -(-int(round(w.outlier_frac * total * 1e6)) // 1_000_000)
            idx = torch.randperm(total, generator=g)[:n]
            k.view(-1)[idx] += w.k_outlier
        else:
            raise ValueError(outlier_mode)
    dt = torch_dtype(w.dtype)
    return q.to(dt), k.to(dt), v.to(dt), do.to(dt)


def make_random_case(B, Hq, Hkv, D, L, S, seed, dtype="bf16", amp=0.5):
    """Inputs for an arbitrary shape (parity sweeps and edge cases)."""
    w = Workload("case", B, Hq, Hkv, D, L, S, seed=seed, dtype=dtype, amp=amp)
    return make_inputs(w)


# ---------------------------------------------------------------------------
# Packed sequences (several [x_t | x_0] pairs of different lengths in one
# buffer, the dynamic packing of Section 5.2).

def varlen_lengths(total: int, seed: int, lo: int = 64, hi: int = 2048) -> list:
    """Sequence lengths (tokens per copy) summing to `total`: log-uniform draws
    in [lo, hi] from a seeded generator, the last one cut to fit.  RL rollouts
    of different lengths packed into one training buffer look like this."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    out, left = [], total
    while left > 0:
        u = float(torch.rand((), generator=g))
        n = int(round(lo * (hi / lo) ** u))
        n = max(1, min(n, left))
        out.append(n)
        left -= n
    return out


def make_varlen_inputs(lengths, Hq: int, Hkv: int, D: int, seed: int, dtype: str = "bf16", amp: float = 0.5):
    """CPU tensors q [Hq, 2T, D], k, v [Hkv, 2T, D], do [Hq, 2T, D] and
    cu_seqlens (int32, len(lengths) + 1): N(0,1)*amp inputs and N(0,1) dO
    drawn in the order q, k, v, dO from a seeded generator, then rounded."""
    T = int(sum(lengths))
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    q = torch.randn((Hq, 2 * T, D), generator=g) * amp
    k = torch.randn((Hkv, 2 * T, D), generator=g) * amp
    v = torch.randn((Hkv, 2 * T, D), generator=g) * amp
    do = torch.randn((Hq, 2 * T, D), generator=g)
    cu = torch.zeros(len(lengths) + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(torch.tensor(lengths, dtype=torch.int64), 0).to(torch.int32)
    dt = torch_dtype(dtype)
    return q.to(dt), k.to(dt), v.to(dt), do.to(dt), cu


# The packed workload measured beside the 8B batch: the same heads, head size
# and block size, 4096 tokens per copy in all (as many as the 8B batch of two
# 2048-token sequences) split into sequences of 64..2048 tokens.
VARLEN_WORKLOADS = {
    "8b_packed": dict(total=4096, Hq=32, Hkv=8, D=128, S=4, seed=8, lo=64, hi=2048),
}


# ---------------------------------------------------------------------------
# Block decoding over a KV cache (rollouts, Section 2.1): a batch of sequences
# at different points of their generation, each denoising one block of S
# tokens against the cached K/V of everything before it.

def decode_cache_lens(B: int, seed: int, lo: int, hi: int) -> list:
    """B cache lengths, log-uniform in [lo, hi] from a seeded generator: a
    rollout batch whose prompts and generated prefixes differ in length."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    u = torch.rand((B,), generator=g, dtype=torch.float64)
    return [int(round(lo * (hi / lo) ** float(x))) for x in u]


def make_decode_inputs(B: int, Hq: int, Hkv: int, D: int, S: int, capacity: int, cache_lens, seed: int,
                       amp: float = 0.5, device: str = "cpu"):
    """bf16 tensors q [B,Hq,S,D], k_cache, v_cache [B,Hkv,capacity,D], k_new,
    v_new [B,Hkv,S,D] (N(0,1)*amp, drawn in that order from a generator seeded
    with `seed` on `device`) and cache_lens (int32 [B], on `device`).  Cache
    rows past a sequence's length hold draws too: nothing may read them."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)

    def draw(*shape):
        return (torch.randn(shape, generator=g, device=device) * amp).to(torch.bfloat16)

    q = draw(B, Hq, S, D)
    kc = draw(B, Hkv, capacity, D)
    vc = draw(B, Hkv, capacity, D)
    kn = draw(B, Hkv, S, D)
    vn = draw(B, Hkv, S, D)
    lens = torch.tensor([int(x) for x in cache_lens], dtype=torch.int32, device=device)
    return q, kc, vc, kn, vn, lens


# The decode workload measured beside the training step: 64 rollouts of the
# 8B shape (32 query heads, 8 KV heads, D = 128, blocks of 4 tokens) with
# caches of 512..8192 tokens (log-uniform), cache capacity 8192.
DECODE_WORKLOADS = {
    "8b_decode": dict(B=64, Hq=32, Hkv=8, D=128, S=4, capacity=8192, lo=512, hi=8192, seed=9),
}


# ---------------------------------------------------------------------------
# Token log-probabilities through the LM head: the positions scored by the
# objectives of Eq. 3 and Eq. 6-7 (the noisy positions of a training batch).

def make_lce_inputs(N: int, V: int, Dm: int, seed: int, logit_std: float = 3.0, device: str = "cpu"):
    """bf16 H [N, Dm] ~ N(0, 1) (normalised final hidden states) and W [V, Dm] ~
    N(0, logit_std^2 / Dm) (so the logits have standard deviation logit_std),
    drawn in that order from a generator seeded with `seed` on `device`, and
    int32 targets uniform in [0, V) from a CPU generator with the same seed."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    h = torch.randn((N, Dm), generator=g, device=device).to(torch.bfloat16)
    w = (torch.randn((V, Dm), generator=g, device=device) * (logit_std / Dm ** 0.5)).to(torch.bfloat16)
    gc = torch.Generator(device="cpu")
    gc.manual_seed(seed)
    t = torch.randint(0, V, (N,), generator=gc, dtype=torch.int64).to(torch.int32).to(device)
    return h, w, t


# The LM head of the 8B model (hidden 4096; a Qwen3-family vocabulary of
# 151,936 entries, the base of SDAR-8B) over the 4096 noisy positions of the
# 8B training batch (two sequences of 2048 tokens).
LCE_WORKLOADS = {
    "8b_lm_head": dict(N=4096, V=151936, Dm=4096, seed=10),
}
