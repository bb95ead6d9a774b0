"""Randomized GPU parity for decode attention over the shapes the C ABI accepts: KV heads,
query heads per KV head (1..8, so every split of a KV head's query heads over
workgroups), head_dim 64 or 128, ragged lengths, sliding windows and, at head_dim 128,
on-demand sparse pages.  Each case is drawn from a seed, quantized by the library and by
the oracle (pools compared bit for bit), and attended by both; outputs must agree within
|gpu - ref| <= 2e-3 + 1e-2 |ref|.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import Case, attention_tolerance, compare_pools, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
P = 16
N_CASES = 16


def _draw(seed: int):
    g = np.random.default_rng(1000 + seed)
    d = int(g.choice([64, 128]))
    H = int(g.choice([1, 2, 3, 4, 8]))
    G = int(g.integers(1, 9))
    n = int(g.integers(1, 6))
    lens = [int(x) for x in g.integers(1, 600, size=n)]
    window = int(g.choice([0, 0, int(g.integers(1, 700))]))
    paged = d == 128 and bool(g.integers(0, 2))
    base = 4 if d == 128 else 1   # Mistral-shaped distributions at 128, the tiny workload's at 64
    return d, H, G, lens, window, paged, base


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_shape_attention(B, ref, seed):
    d, H, G, lens, window, paged, base = _draw(seed)
    w = dataclasses.replace(synth.scaled(synth.WORKLOADS[base], n_seqs=len(lens), ctx=max(lens), ctx_min=1),
                            n_q_heads=H * G, n_kv_heads=H, head_dim=d)
    case = Case(w, lens=lens)
    case.calibrate_oracle(ref)
    pool_ref = case.oracle_pool(ref)
    thr = torch.from_numpy(case.thr).to(DEV)
    sparse = 2 * case.num_blocks * H * 2 + 16 if paged else 0
    cache = B.Cache(case.num_blocks, H, d, thr, sparse_pages=sparse)
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt, torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV),
                  case.cu.to(DEV), int(case.lens.max()))
    if not paged:
        compare_pools(ref, case, cache.pool.cpu().numpy(), pool_ref)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, P, H, d, case.thr, np16(q), case.bt.numpy(),
                                case.lens.numpy(), scale, window=window)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale, window=window)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"seed {seed}: d={d} H={H} G={G} lens={lens} window={window} paged={paged}: "
          f"max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)
