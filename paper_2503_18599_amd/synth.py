"""Seeded synthetic workloads: K/V activations, queries, calibration sets, paged block tables.

This module only draws random inputs.  It holds none of the quantizer's or the
attention's arithmetic, so both the HIP path and the CPU oracle can be fed from it.

The distributions stand in for real model KV caches, which the paper profiles on
Wikitext2/PIQA/Hellaswag (Sec. 4.1) and which are not available here:
  * per-layer ranges differ by model (Obs. 1) and are input-independent (Obs. 2):
    a per-(KV head, channel) scale is drawn once from the "model" seed and shared by
    the calibration set and every later token;
  * large values concentrate in a few channels, with exceptions (Obs. 3): heavy-tailed
    Student-t(3) values under LogNormal channel scales, or a few outlier channels x20.

Seeds per workload c: model = 100c+1, calibration = 100c+2, data = 100c+3,
query = 100c+4, block table / lengths = 100c+5.
"""
from __future__ import annotations

import dataclasses
import math

import torch

PAGE = 16  # tokens per page


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    n_seqs: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ctx: int                 # context length (fixed) or upper bound (variable lengths)
    ctx_min: int             # lower bound for variable lengths (== ctx when fixed)
    k_dist: str
    v_dist: str
    n_calib_tokens: int
    decode_steps: int = 1
    prefill: bool = False    # cache built by one prefill-time quantization call

    @property
    def calib_runs(self) -> int:
        return max(1, self.n_calib_tokens // 512)

    @property
    def calib_tokens_per_run(self) -> int:
        return min(512, self.n_calib_tokens)

    def seed(self, what: str) -> int:
        return 100 * self.cid + {"model": 1, "calib": 2, "data": 3, "query": 4, "table": 5}[what]


WORKLOADS = {
    1: Workload(1, "tiny", 2, 4, 4, 64, 128, 128, "gauss_spiky", "gauss_spiky", 512),
    2: Workload(2, "llama2-7b-layer", 64, 32, 32, 128, 1024, 1024, "t3_lognormal", "t3_lognormal", 4096),
    3: Workload(3, "llama2-13b-layer", 256, 40, 40, 128, 2048, 2048, "t3_lognormal", "t3_lognormal", 4096),
    4: Workload(4, "mistral-7b-gqa", 256, 32, 8, 128, 8192, 512, "gauss_outlier_ch", "gauss", 4096),
    5: Workload(5, "llama3-8b-32k", 16, 32, 8, 128, 32768, 32768, "t3_lognormal", "t3_lognormal", 4096,
                decode_steps=64, prefill=True),
}


def scaled(w: Workload, n_seqs: int | None = None, ctx: int | None = None,
           ctx_min: int | None = None) -> Workload:
    """Same distributions and head shapes, fewer sequences / shorter context (parity sizes)."""
    c = ctx if ctx is not None else w.ctx
    cm = ctx_min if ctx_min is not None else (c if w.ctx_min == w.ctx else min(w.ctx_min, c))
    return dataclasses.replace(w, n_seqs=n_seqs or w.n_seqs, ctx=c, ctx_min=cm)


# --------------------------------------------------------------------------- #
def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def model_params(w: Workload, which: str):
    """Per-(KV head, channel) structure fixed by the model seed (CPU tensors)."""
    g = _gen(w.seed("model") * 10 + (0 if which == "k" else 1), "cpu")
    H, d = w.n_kv_heads, w.head_dim
    dist = w.k_dist if which == "k" else w.v_dist
    if dist == "t3_lognormal":
        return {"scale": torch.exp(0.5 * torch.randn(H, d, generator=g))}
    if dist == "gauss_outlier_ch":
        n_out = max(1, round(0.03 * d))
        mult = torch.ones(H, d)
        for h in range(H):
            idx = torch.randperm(d, generator=g)[:n_out]
            mult[h, idx] = 20.0
        return {"scale": mult}
    return {"scale": torch.ones(H, d)}


def kv_values(w: Workload, which: str, n_tokens: int, seed: int, device="cpu") -> torch.Tensor:
    """fp16 [n_tokens][H_kv][d] activations for K (which='k') or V ('v')."""
    H, d = w.n_kv_heads, w.head_dim
    dist = w.k_dist if which == "k" else w.v_dist
    g = _gen(seed * 2 + (0 if which == "k" else 1), device)
    scale = model_params(w, which)["scale"].to(device)
    shape = (n_tokens, H, d)
    if dist == "gauss_spiky":
        x = torch.randn(shape, generator=g, device=device)
        spike = torch.rand(shape, generator=g, device=device) < 0.01
        x = torch.where(spike, x * 10.0, x)
    elif dist == "t3_lognormal":
        z = torch.randn(shape, generator=g, device=device)
        c = torch.randn((3,) + shape, generator=g, device=device).square_().sum(0)
        x = z / torch.sqrt(c / 3.0) * scale          # Student-t(3) x channel scale
    elif dist == "gauss_outlier_ch":
        x = torch.randn(shape, generator=g, device=device) * scale
    else:
        x = torch.randn(shape, generator=g, device=device)
    return x.clamp_(-60000.0, 60000.0).to(torch.float16)


def calibration_set(w: Workload, which: str, device="cpu") -> torch.Tensor:
    """fp16 [R][T][H][d]: held-out tokens from the same model, grouped in runs of 512."""
    R, T = w.calib_runs, w.calib_tokens_per_run
    x = kv_values(w, which, R * T, w.seed("calib"), device)
    return x.reshape(R, T, w.n_kv_heads, w.head_dim).contiguous()


def queries(w: Workload, step: int = 0, device="cpu") -> torch.Tensor:
    g = _gen(w.seed("query") * 1000 + step, device)
    return torch.randn(w.n_seqs, w.n_q_heads, w.head_dim, generator=g, device=device).to(torch.float16)


def seq_lengths(w: Workload) -> torch.Tensor:
    """int32 [n_seqs] context lengths (uniform integers in [ctx_min, ctx] when they vary)."""
    if w.ctx_min == w.ctx:
        return torch.full((w.n_seqs,), w.ctx, dtype=torch.int32)
    g = _gen(w.seed("table"), "cpu")
    return torch.randint(w.ctx_min, w.ctx + 1, (w.n_seqs,), generator=g, dtype=torch.int32)


def block_table(w: Workload, lens: torch.Tensor, extra_tokens: int = 0):
    """Shuffled physical pages: returns (int32 [n_seqs][max_blocks], num_blocks)."""
    nb = [math.ceil((int(L) + extra_tokens) / PAGE) for L in lens]
    max_blocks = max(nb)
    total = sum(nb)
    g = _gen(w.seed("table") + 7, "cpu")
    perm = torch.randperm(total, generator=g).to(torch.int32)
    bt = torch.zeros(len(nb), max_blocks, dtype=torch.int32)
    off = 0
    for s, n in enumerate(nb):
        bt[s, :n] = perm[off: off + n]
        off += n
    return bt, total


def kv_values_seq(w: Workload, which: str, seq: int, n_tokens: int, device="cpu") -> torch.Tensor:
    """fp16 [n_tokens][H_kv][d] for one sequence, reproducible on its own (seeded by the
    data seed and the sequence index), so large caches can be built in chunks and any
    sampled sequence regenerated later."""
    return kv_values(w, which, n_tokens, w.seed("data") * 100003 + seq, device)


def new_token_values(w: Workload, which: str, step: int, device="cpu") -> torch.Tensor:
    """fp16 [n_seqs][H_kv][d]: the K or V row each sequence appends at decode step `step`."""
    return kv_values(w, which, w.n_seqs, w.seed("data") * 7919 + 1000 + step, device)
