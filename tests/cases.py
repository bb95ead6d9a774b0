"""Shared builders for parity tests: seeded inputs from ``synth`` feed both the oracle
(host numpy) and the HIP library (device tensors); expected values come only from the
oracle."""
from __future__ import annotations

import math

import numpy as np
import torch

from paper_2503_18599_amd import synth

P = 16


def np16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().numpy()


class Case:
    """A workload at a chosen size: thresholds (oracle), prefill K/V, block table."""

    def __init__(self, w: synth.Workload, lens=None, thresholds=None):
        self.w = w
        self.H, self.Hq, self.d = w.n_kv_heads, w.n_q_heads, w.head_dim
        self.lens = (torch.as_tensor(lens, dtype=torch.int32) if lens is not None
                     else synth.seq_lengths(w))
        self.n_seqs = int(self.lens.numel())
        self.bt, self.num_blocks = synth.block_table(w, self.lens, extra_tokens=8)
        self.max_blocks = self.bt.shape[1]
        self.k = synth.kv_values(w, "k", int(self.lens.sum()), w.seed("data"))
        self.v = synth.kv_values(w, "v", int(self.lens.sum()), w.seed("data"))
        self.cu = torch.zeros(self.n_seqs + 1, dtype=torch.int32)
        self.cu[1:] = torch.cumsum(self.lens, 0)
        self.thr = thresholds

    def calibrate_oracle(self, ref):
        kc = synth.calibration_set(self.w, "k")
        vc = synth.calibration_set(self.w, "v")
        self.thr = ref.calibrate(np16(kc), np16(vc), 0.04, 0.06)
        return self.thr

    def oracle_pool(self, ref, start=None):
        lay = ref.layout(P, self.d)
        pool = np.zeros(self.num_blocks * self.H * 2 * lay["stride"], np.uint8)
        sp = np.zeros(self.n_seqs, np.int32) if start is None else start
        ref.quantize_kv(pool, self.num_blocks, P, self.H, self.d, self.thr, np16(self.k),
                        np16(self.v), self.bt.numpy(), sp, self.cu.numpy())
        return pool

    def used_regions(self, ref, pool: np.ndarray):
        """Yield (block, head, which, bytes) over the used prefix of every record."""
        lay = ref.layout(P, self.d)
        st = lay["stride"]
        for b in range(self.num_blocks):
            for h in range(self.H):
                for w in (0, 1):
                    off = ((b * self.H + h) * 2 + w) * st
                    used = lay["sparse"] + int(pool[off:off + lay["meta"]].sum())
                    yield b, h, w, off, used


def compare_pools(ref, case: Case, got: np.ndarray, want: np.ndarray):
    """Bit-exact comparison of every record's used prefix; returns the number of records."""
    n = 0
    lay = ref.layout(P, case.d)
    for b, h, w, off, used in case.used_regions(ref, want):
        g = got[off:off + used]
        e = want[off:off + used]
        if not np.array_equal(g, e):
            bad = np.nonzero(g != e)[0]
            field = ("counts" if bad[0] < lay["meta"] else "meta" if bad[0] < lay["dense"]
                     else "dense" if bad[0] < lay["sparse"] else "sparse")
            raise AssertionError(f"record (block {b}, head {h}, {'KV'[w]}) differs at byte {bad[0]} "
                                 f"({field}): got {g[bad[0]]} want {e[bad[0]]}; {bad.size} bytes differ")
        n += 1
    return n


def attention_tolerance(got: np.ndarray, want: np.ndarray, atol=2e-3, rtol=1e-2):
    err = np.abs(got.astype(np.float64) - want.astype(np.float64))
    lim = atol + rtol * np.abs(want.astype(np.float64))
    ok = err <= lim
    return bool(ok.all()), float(err.max()), float((err / np.maximum(np.abs(want), 1e-30)).max())
