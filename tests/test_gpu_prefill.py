"""Chunked-prefill attention over the quantized cache: every query token of a chunk
attends causally over its sequence's keys up to its own position.  The reference is the
oracle's decode attention evaluated once per query token (its sequence's block table,
length = position + 1), over the oracle's bit-identical cache."""
import dataclasses
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import Case, attention_tolerance, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
P = 16


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _run(B, ref, case, chunk, window=0, paged=False, seed=5):
    """Cache all tokens (prefix, then the chunk), then prefill attention for the chunk's
    queries; returns (got, want)."""
    n, H, Hq, d = case.n_seqs, case.H, case.Hq, case.d
    lens = case.lens
    clen = torch.minimum(torch.as_tensor(chunk, dtype=torch.int32).expand(n), lens)   # chunk tokens per sequence
    start = (lens - clen).to(torch.int32)
    thr = torch.from_numpy(case.thr).to(DEV)
    cache = B.Cache(case.num_blocks, H, d, thr, sparse_pages=4 * case.num_blocks * H * 2 if paged else 0)
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt, torch.zeros(n, dtype=torch.int32, device=DEV),
                  case.cu.to(DEV), int(lens.max()))
    cu = torch.zeros(n + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(clen, 0)
    n_tok = int(cu[-1])
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(n_tok, Hq, d, generator=g).to(torch.float16)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    got = B.prefill_attention(cache, q.to(DEV), bt, start.to(DEV), cu.to(DEV), int(lens.max()), scale,
                              window=window).cpu().numpy()
    # oracle: one decode-attention row per query token
    pool = case.oracle_pool(ref)
    seq = np.concatenate([np.full(int(clen[s]), s) for s in range(n)])
    pos = np.concatenate([np.arange(int(start[s]), int(lens[s])) for s in range(n)])
    want = ref.decode_attention(pool, case.num_blocks, P, H, d, case.thr, np16(q), case.bt.numpy()[seq],
                                (pos + 1).astype(np.int32), scale, window=window)
    return got, want


@pytest.mark.parametrize("cid,kw,chunk,window,paged", [
    (3, dict(n_seqs=3, ctx=600), 37, 0, False),           # MHA, ragged chunk (64-row blocks)
    (3, dict(n_seqs=3, ctx=600), 24, 0, False),           # MHA, 32-row blocks
    (4, dict(n_seqs=4, ctx=300, ctx_min=40), 8, 0, False),   # GQA, 8-token chunks: 32-row blocks
    (4, dict(n_seqs=4, ctx=700, ctx_min=40), 64, 0, False),  # GQA, chunk = whole prompt for short ones (128-row blocks)
    (4, dict(n_seqs=4, ctx=700, ctx_min=40), 50, 100, False),  # GQA with a sliding window (128-row blocks)
    (2, dict(n_seqs=3, ctx=203), 203, 0, False),          # whole prompts from position 0 (128-row blocks)
    (2, dict(n_seqs=2, ctx=700), 300, 0, False),          # MHA chunks of 300 tokens: three 128-row blocks each
    (1, dict(), 16, 0, False)])                           # head_dim 64, 16-row blocks
def test_prefill_attention_matches_oracle(B, ref, cid, kw, chunk, window, paged):
    case = Case(synth.scaled(synth.WORKLOADS[cid], **kw))
    case.calibrate_oracle(ref)
    got, want = _run(B, ref, case, chunk, window, paged)
    ok, max_abs, max_rel = attention_tolerance(got, want)
    print(f"{case.w.name} chunk {chunk} window {window}: {got.shape[0]} query tokens, max_abs={max_abs:.3e}")
    assert ok, (max_abs, max_rel)


@pytest.mark.parametrize("hq,hkv,chunk", [
    (16, 8, 40),    # two query heads per KV head: 80 rows per chunk, 128-row blocks
    (32, 4, 10),    # eight: 80 rows, 128-row blocks of 16 tokens
    (32, 4, 3),     # eight: 24 rows, 32-row blocks of 4 tokens
    (12, 4, 5)])    # three: 15 rows, 16-row blocks of 5 tokens
def test_prefill_other_head_ratios(B, ref, hq, hkv, chunk):
    """Head ratios the benchmark workloads do not have, through every block width."""
    w = dataclasses.replace(synth.scaled(synth.WORKLOADS[4], n_seqs=3, ctx=300, ctx_min=40),
                            n_q_heads=hq, n_kv_heads=hkv)
    case = Case(w)
    case.calibrate_oracle(ref)
    got, want = _run(B, ref, case, chunk)
    ok, max_abs, max_rel = attention_tolerance(got, want)
    print(f"{hq}/{hkv} heads chunk {chunk}: {got.shape[0]} query tokens, max_abs={max_abs:.3e}")
    assert ok, (max_abs, max_rel)


def test_prefill_short_mean_long_chunks(B, ref):
    """Blocks are sized to the mean chunk: chunks of 20, 3, 2 and 20 tokens average 12 rows,
    so the blocks hold 16 rows and each 20-token chunk takes two of them."""
    case = Case(synth.scaled(synth.WORKLOADS[3], n_seqs=4, ctx=64, ctx_min=1), lens=[64, 3, 2, 50])
    case.calibrate_oracle(ref)
    got, want = _run(B, ref, case, 20)
    ok, max_abs, max_rel = attention_tolerance(got, want)
    assert ok, (max_abs, max_rel)


@pytest.mark.parametrize("cid,chunk", [(3, 48), (4, 40)])
def test_prefill_attention_paged(B, ref, cid, chunk):
    """On-demand sparse pages: 48-token MHA chunks (64-row blocks) and 40-token chunks of
    four query heads per KV head (160 rows: the 128-row blocks on fp16 matrix cores)."""
    case = Case(synth.scaled(synth.WORKLOADS[cid], n_seqs=3, ctx=600))
    case.calibrate_oracle(ref)
    got, want = _run(B, ref, case, chunk, paged=True)
    ok, max_abs, max_rel = attention_tolerance(got, want)
    assert ok, (max_abs, max_rel)


def test_prefill_last_token_is_decode(B, ref):
    """The last query of a chunk sees the whole sequence: its output is decode attention's
    (the two kernels compute differently -- fp32 matrix cores over dequantized tiles here,
    integer limbs and COO corrections there -- so they agree within the attention
    tolerance)."""
    case = Case(synth.scaled(synth.WORKLOADS[4], n_seqs=4, ctx=300, ctx_min=20))
    case.calibrate_oracle(ref)
    n, Hq, d = case.n_seqs, case.Hq, case.d
    thr = torch.from_numpy(case.thr).to(DEV)
    cache = B.Cache(case.num_blocks, case.H, d, thr)
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt, torch.zeros(n, dtype=torch.int32, device=DEV),
                  case.cu.to(DEV), int(case.lens.max()))
    q = synth.queries(case.w).to(DEV)
    dec = B.decode_attention(cache, q, bt, case.lens.to(DEV), int(case.lens.max()), 0.09)
    pre = B.prefill_attention(cache, q, bt, (case.lens - 1).to(torch.int32).to(DEV),
                              torch.arange(n + 1, dtype=torch.int32).to(DEV), int(case.lens.max()), 0.09)
    ok, max_abs, max_rel = attention_tolerance(pre.cpu().numpy(), dec.cpu().numpy())
    assert ok, (max_abs, max_rel)
