"""GPU parity for every head shape the C ABI accepts.

The attention entry points take head_dim 64 or 128 and 1..8 query heads per KV head
(G).  head_dim 128 runs the matrix-core kernel, which takes 1, 2 or 4 query heads per
workgroup (G = 3 as three workgroups of one head, G = 8 as two of four); head_dim 64 runs
the vector-unit kernel.  The workload tests cover G = 1 and 4; this module adds G = 2
(fixed records and on-demand sparse pages), 3 and 8 at head_dim 128 and G = 2, 4 and 8
at head_dim 64: decode attention over ragged
lengths (one token, page multiples, ragged tails, several page ranges per sequence so the
split combine runs), sliding windows, and chunked prefill, each against the oracle
within |gpu - ref| <= 2e-3 + 1e-2 |ref|.
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
LENS = [1, 16, 17, 31, 200, 700]

# (query heads, KV heads, head_dim, base workload): the head_dim 128 shapes use the
# Mistral-shaped distributions (outlier channels in K), the head_dim 64 shapes the tiny
# workload's (1 % spikes)
SHAPES = {
    "g2-d128": (16, 8, 128, 4),
    "g3-d128": (24, 8, 128, 4),
    "g8-d128": (64, 8, 128, 4),
    "g2-d64": (8, 4, 64, 1),
    "g4-d64": (16, 4, 64, 1),
    "g8-d64": (32, 4, 64, 1),
}


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _case(ref, shape, lens=LENS):
    hq, h, d, base = SHAPES[shape]
    w = dataclasses.replace(synth.scaled(synth.WORKLOADS[base], n_seqs=len(lens), ctx=max(lens), ctx_min=1),
                            n_q_heads=hq, n_kv_heads=h, head_dim=d)
    c = Case(w, lens=lens)
    c.calibrate_oracle(ref)
    return c


def _cache(B, case, sparse_pages=0):
    thr = torch.from_numpy(case.thr).to(DEV)
    cache = B.Cache(case.num_blocks, case.H, case.d, thr, sparse_pages=sparse_pages)
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt, torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV),
                  case.cu.to(DEV), int(case.lens.max()))
    return cache, bt


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("window", [0, 17, 300])
def test_decode_attention_head_shapes(B, ref, shape, window):
    case = _case(ref, shape)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _cache(B, case)
    if window == 0:
        compare_pools(ref, case, cache.pool.cpu().numpy(), pool_ref)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, P, case.H, case.d, case.thr, np16(q), case.bt.numpy(),
                                case.lens.numpy(), scale, window=window)
    # max_seq_len beyond every length, so the split plan has empty trailing ranges
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), case.max_blocks * P, scale, window=window)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"{shape} window {window}: max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)


@pytest.mark.parametrize("shape", ["g2-d128", "g3-d128", "g8-d128"])
@pytest.mark.parametrize("window", [0, 100])
def test_decode_attention_sparse_pages_head_shapes(B, ref, shape, window):
    """G = 2, 3 and 8 on the matrix cores (one, three and two workgroups per KV head) with
    on-demand sparse pages."""
    case = _case(ref, shape)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _cache(B, case, sparse_pages=2 * case.num_blocks * case.H * 2 + 16)
    assert not cache.sparse_status()[1]
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, P, case.H, case.d, case.thr, np16(q), case.bt.numpy(),
                                case.lens.numpy(), scale, window=window)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale, window=window)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    assert ok, (max_abs, max_rel)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_prefill_attention_head_shapes(B, ref, shape):
    """Chunked prefill (the last 24 tokens of each sequence, whole prompts for the short
    ones) against the oracle's decode attention evaluated per query token."""
    case = _case(ref, shape, lens=[1, 20, 90, 333])
    n, H, Hq, d = case.n_seqs, case.H, case.Hq, case.d
    lens = case.lens
    clen = torch.clamp(lens, max=24).to(torch.int32)
    start = (lens - clen).to(torch.int32)
    cache, bt = _cache(B, case)
    cu = torch.zeros(n + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(clen, 0)
    n_tok = int(cu[-1])
    q = torch.randn(n_tok, Hq, d, generator=torch.Generator().manual_seed(11)).to(torch.float16)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    got = B.prefill_attention(cache, q.to(DEV), bt, start.to(DEV), cu.to(DEV), int(lens.max()), scale).cpu().numpy()
    pool = case.oracle_pool(ref)
    seq = np.concatenate([np.full(int(clen[s]), s) for s in range(n)])
    pos = np.concatenate([np.arange(int(start[s]), int(lens[s])) for s in range(n)])
    want = ref.decode_attention(pool, case.num_blocks, P, H, d, case.thr, np16(q), case.bt.numpy()[seq],
                                (pos + 1).astype(np.int32), scale)
    ok, max_abs, max_rel = attention_tolerance(got, want)
    print(f"{shape} prefill: {n_tok} query tokens, max_abs={max_abs:.3e}")
    assert ok, (max_abs, max_rel)


def test_more_than_eight_query_heads_rejected(B, ref):
    case = _case(ref, "g8-d64", lens=[5])
    cache, bt = _cache(B, case)
    q = torch.zeros(1, 9 * case.H, case.d, dtype=torch.float16, device=DEV)
    with pytest.raises(B.OakenError) as e:
        B.decode_attention(cache, q, bt, case.lens.to(DEV), 16, 0.1)
    assert e.value.status == 2
