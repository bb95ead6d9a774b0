"""One decoder layer's decode step around the Oaken KV cache.

The layer is Llama-shaped: RMSNorm, a fused QKV projection, Oaken's online quantization
of the new key and value (quantize_kv), decode attention over the quantized cache with
in-register dequantization (decode_attention), the output projection and residual, then
RMSNorm, a SwiGLU MLP and residual.  Projections and norms are plain torch bf16 ops
(library GEMMs); the KV path is the HIP library through its C ABI.  Positional rotation
is left out: it does not touch the cache format.

`step` runs the phases in order on the current stream and can record per-phase HIP events
(the quantization and attention shares of a layer step: the latency breakdown of
Sec. 6.2).
`step_overlapped` splits the batch into micro-batches on separate streams, so that one
micro-batch's memory-bound attention can run beside another's compute-bound GEMMs: the
GPU form of overlapping KV quantization and dequantization with other requests' work
(token-level batch scheduling, Sec. 5.3).
"""
from __future__ import annotations

import math

import torch

from . import binding as B

PHASES = ("pre", "quantize", "attention", "post")


class DecoderLayer:
    def __init__(self, d_model: int, n_heads: int, n_kv_heads: int, head_dim: int, d_ff: int,
                 cache: B.Cache, seed: int = 0, device: str = "cuda"):
        if n_heads % n_kv_heads or cache.n_kv_heads != n_kv_heads or cache.head_dim != head_dim:
            raise ValueError("head configuration does not match the cache")
        self.d_model, self.n_heads, self.n_kv_heads, self.head_dim, self.d_ff = d_model, n_heads, n_kv_heads, head_dim, d_ff
        self.cache = cache
        g = torch.Generator(device="cpu").manual_seed(seed)

        def w(i, o):
            return (torch.randn(i, o, generator=g) / math.sqrt(i)).to(torch.bfloat16).to(device)

        qkv_out = (n_heads + 2 * n_kv_heads) * head_dim
        self.w_qkv = w(d_model, qkv_out)
        self.w_o = w(n_heads * head_dim, d_model)
        self.w_gate = w(d_model, d_ff)
        self.w_up = w(d_model, d_ff)
        self.w_down = w(d_ff, d_model)
        self.norm1 = torch.ones(d_model, dtype=torch.bfloat16, device=device)
        self.norm2 = torch.ones(d_model, dtype=torch.bfloat16, device=device)
        self.scale = float(1.0 / math.sqrt(head_dim))
        self.keep_attention = False   # keep the last step's attention output (for checks)
        self.last_attention = None

    @staticmethod
    def _rms(x: torch.Tensor, weight: torch.Tensor) -> torch.Tensor:
        xf = x.float()
        return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + 1e-5)).to(torch.bfloat16) * weight

    def project(self, x: torch.Tensor):
        """bf16 hidden [n][d_model] -> fp16 q [n][Hq][d], k, v [n][H][d]."""
        n = x.shape[0]
        qkv = self._rms(x, self.norm1) @ self.w_qkv
        hq, hk, d = self.n_heads, self.n_kv_heads, self.head_dim
        q = qkv[:, :hq * d].reshape(n, hq, d).to(torch.float16)
        k = qkv[:, hq * d:(hq + hk) * d].reshape(n, hk, d).to(torch.float16).contiguous()
        v = qkv[:, (hq + hk) * d:].reshape(n, hk, d).to(torch.float16).contiguous()
        return q.contiguous(), k, v

    def finish(self, x: torch.Tensor, attn: torch.Tensor) -> torch.Tensor:
        """Output projection, residual, MLP, residual."""
        n = x.shape[0]
        h = x + attn.reshape(n, -1).to(torch.bfloat16) @ self.w_o
        y = self._rms(h, self.norm2)
        return h + (torch.nn.functional.silu(y @ self.w_gate) * (y @ self.w_up)) @ self.w_down

    def step(self, x: torch.Tensor, block_table: torch.Tensor, seq_lens: torch.Tensor, max_seq_len: int,
             events: dict | None = None, workspace: torch.Tensor | None = None) -> torch.Tensor:
        """One decode step for n sequences: x bf16 [n][d_model]; seq_lens count the new token,
        which is written at position seq_lens - 1.  events: optional {phase: (start, end)}."""
        n = x.shape[0]

        def mark(phase, i):
            if events is not None:
                events[phase][i].record()

        mark("pre", 0)
        q, k, v = self.project(x)
        mark("pre", 1)
        mark("quantize", 0)
        B.quantize_kv(self.cache, k, v, block_table, (seq_lens - 1).to(torch.int32),
                      torch.arange(n + 1, dtype=torch.int32, device=x.device), 1)
        mark("quantize", 1)
        mark("attention", 0)
        attn = B.decode_attention(self.cache, q, block_table, seq_lens, max_seq_len, self.scale, workspace=workspace)
        mark("attention", 1)
        if self.keep_attention:
            self.last_attention = attn
        mark("post", 0)
        out = self.finish(x, attn)
        mark("post", 1)
        return out

    def step_overlapped(self, x: torch.Tensor, block_table: torch.Tensor, seq_lens: torch.Tensor,
                        max_seq_len: int, streams: list, workspaces: list | None = None) -> torch.Tensor:
        """The same step with the batch split into len(streams) micro-batches, each running
        its phases on its own stream after the current stream's prior work."""
        n = x.shape[0]
        m = len(streams)
        bounds = [n * i // m for i in range(m + 1)]
        cur = torch.cuda.current_stream()
        start = torch.cuda.Event()
        start.record(cur)
        outs = []
        for i, s in enumerate(streams):
            lo, hi = bounds[i], bounds[i + 1]
            s.wait_event(start)
            with torch.cuda.stream(s):
                ws = workspaces[i] if workspaces else None
                outs.append(self.step(x[lo:hi], block_table[lo:hi], seq_lens[lo:hi], max_seq_len, workspace=ws))
        for s in streams:
            cur.wait_stream(s)
        for o in outs:
            o.record_stream(cur)
        return torch.cat(outs)
