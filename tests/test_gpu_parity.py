"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bit-exact: calibrated thresholds, and the used prefix of every page record (counts,
fp16 scales, dense nibbles, COO bytes).  Attention: |gpu - ref| <= 2e-3 + 1e-2 |ref|
elementwise against the oracle's fp64 attention over its own (bit-identical) cache.
Sizes keep the oracle within seconds while spanning many pages, ragged last pages,
split ranges and every workload's head shape.
"""
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import P, Case, attention_tolerance, compare_pools, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _gpu_cache(B, case: Case, prefill=True):
    thr = torch.from_numpy(case.thr).to(DEV)
    cache = B.Cache(case.num_blocks, case.H, case.d, thr)
    bt = case.bt.to(DEV)
    if prefill:
        B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt,
                      torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), case.cu.to(DEV),
                      int(case.lens.max()))
    return cache, bt


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_calibration_bit_exact(B, ref, cid):
    w = synth.WORKLOADS[cid]
    kc = synth.calibration_set(w, "k")
    vc = synth.calibration_set(w, "v")
    want = ref.calibrate(np16(kc), np16(vc), 0.04, 0.06)
    got = B.calibrate_thresholds(kc.to(DEV), vc.to(DEV), 0.04, 0.06).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (got, want)


@pytest.mark.parametrize("ratios", [(0.0, 0.0), (0.10, 0.30), (0.5, 0.0)])
def test_calibration_other_ratios(B, ref, ratios):
    w = synth.WORKLOADS[2]
    kc = synth.calibration_set(w, "k")[:2]
    vc = synth.calibration_set(w, "v")[:2]
    want = ref.calibrate(np16(kc), np16(vc), *ratios)
    got = B.calibrate_thresholds(kc.contiguous().to(DEV), vc.contiguous().to(DEV), *ratios).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


CASES = {
    "tiny": (1, dict()),
    "llama2-7b": (2, dict(n_seqs=6, ctx=203)),
    "llama2-13b": (3, dict(n_seqs=3, ctx=2048)),
    "mistral-gqa": (4, dict(n_seqs=5, ctx=1500, ctx_min=1)),
    "llama3-32k": (5, dict(n_seqs=2, ctx=3000)),
    # many (sequence, head) units: one page range per unit, no split combine
    "llama2-13b-wide": (3, dict(n_seqs=103, ctx=37)),
}


def _case(ref, name):
    cid, kw = CASES[name]
    w = synth.scaled(synth.WORKLOADS[cid], **kw)
    c = Case(w)
    c.calibrate_oracle(ref)
    return c


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_quantize_bit_exact(B, ref, name):
    case = _case(ref, name)
    want = case.oracle_pool(ref)
    cache, _ = _gpu_cache(B, case)
    got = cache.pool.cpu().numpy()
    n = compare_pools(ref, case, got, want)
    assert n > 0
    # a second run writes identical bytes (no races in the compaction / scans)
    cache2, _ = _gpu_cache(B, case)
    assert torch.equal(cache.pool, cache2.pool)


@pytest.mark.parametrize("name", ["tiny", "llama2-7b", "mistral-gqa"])
def test_decode_append_bit_exact(B, ref, name):
    """Prefill all but the last few tokens, then append one token per sequence per call."""
    case = _case(ref, name)
    n_dec = 5
    lens = case.lens.clone()
    pre = torch.clamp(lens - n_dec, min=0)
    cache, bt = _gpu_cache(B, case, prefill=False)
    # prefill rows: first pre[s] rows of each sequence
    rows = torch.cat([torch.arange(int(case.cu[s]), int(case.cu[s]) + int(pre[s])) for s in range(case.n_seqs)])
    cu_pre = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
    cu_pre[1:] = torch.cumsum(pre, 0)
    B.quantize_kv(cache, case.k[rows].to(DEV), case.v[rows].to(DEV), bt,
                  torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), cu_pre.to(DEV), int(pre.max()))
    for step in range(n_dec):
        pos = pre + step
        act = (pos < lens)
        r = (case.cu[:-1] + pos).clamp(max=int(case.cu[-1]) - 1)
        cnt = act.to(torch.int32)
        cu = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
        cu[1:] = torch.cumsum(cnt, 0)
        sel = r[act]
        B.quantize_kv(cache, case.k[sel].to(DEV), case.v[sel].to(DEV), bt, pos.to(torch.int32).to(DEV),
                      cu.to(DEV), 1)
    want = case.oracle_pool(ref)
    compare_pools(ref, case, cache.pool.cpu().numpy(), want)


@pytest.mark.parametrize("mode", ["segment", "token"])
def test_quantize_rows_beyond_the_launch_bound(B, ref, mode):
    """A sequence with more new rows than max_new_per_seq (a caller error the library cannot
    see): the other sequence's record is exact, and no byte outside the two sequences' own
    pages is written.  The segment kernel still writes the overrunning sequence's first page;
    the decode-step kernel skips that sequence."""
    lens, bound = ([60, 10], 20) if mode == "segment" else ([2, 1], 1)
    w = synth.scaled(synth.WORKLOADS[2], n_seqs=2, ctx=max(lens))
    case = Case(w, lens=lens)
    case.calibrate_oracle(ref)
    want = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case, prefill=False)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt,
                  torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), case.cu.to(DEV), bound)
    got = cache.pool.cpu().numpy()
    lay = ref.layout(P, case.d)
    st = lay["stride"]
    pages = [(int(lens[s]) + P - 1) // P for s in range(2)]
    own0 = {int(b) for b in case.bt[0, :pages[0]]}
    exact = {int(case.bt[1, 0])} | ({int(case.bt[0, 0])} if mode == "segment" else set())
    for b in range(case.num_blocks):
        for h in range(case.H):
            for wv in (0, 1):
                off = ((b * case.H + h) * 2 + wv) * st
                g, e = got[off:off + st], want[off:off + st]
                if b in exact:
                    used = lay["sparse"] + int(e[:lay["meta"]].sum())
                    assert np.array_equal(g[:used], e[:used]), (mode, b, h, wv)
                elif b not in own0:
                    assert not g.any(), (mode, b, h, wv)
    if mode == "token":
        b0 = int(case.bt[0, 0])
        assert not got[b0 * case.H * 2 * st:(b0 + 1) * case.H * 2 * st].any()


def test_quantize_edge_thresholds(B, ref):
    """All-inner thresholds (every value an outlier: full COO capacity), collapsed inner
    interval, and constant / zero vectors."""
    w = synth.scaled(synth.WORKLOADS[2], n_seqs=2, ctx=40)
    case = Case(w)
    H = case.H
    thr = np.zeros((H, 2, 4), np.float32)
    thr[:, :, 0], thr[:, :, 1], thr[:, :, 2], thr[:, :, 3] = -np.inf, -np.inf, np.inf, np.inf
    thr[1::2] = np.array([-1.0, 0.0, 0.0, 1.0], np.float32)
    case.thr = thr
    case.k[3] = 0.0
    case.v[5] = 1.5
    case.k[7, :, :64] = -2.0
    want = case.oracle_pool(ref)
    cache, _ = _gpu_cache(B, case)
    compare_pools(ref, case, cache.pool.cpu().numpy(), want)


@pytest.mark.parametrize("cid", [2, 1])
def test_quantize_edge_thresholds_token_by_token(B, ref, cid):
    """The decode-step path (one new token per sequence per call) under the same edge
    thresholds: every value an outlier (each record's COO stream fills its capacity one
    slot at a time), a collapsed inner interval, constant and zero vectors; head_dim 128
    and 64, even and odd slots."""
    w = synth.scaled(synth.WORKLOADS[cid], n_seqs=3, ctx=37)
    case = Case(w)
    H = case.H
    thr = np.zeros((H, 2, 4), np.float32)
    thr[:, :, 0], thr[:, :, 1], thr[:, :, 2], thr[:, :, 3] = -np.inf, -np.inf, np.inf, np.inf
    thr[1::2] = np.array([-1.0, 0.0, 0.0, 1.0], np.float32)
    case.thr = thr
    case.k[3] = 0.0
    case.v[5] = 1.5
    case.k[7, :, : case.d // 2] = -2.0
    want = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case, prefill=False)
    lens = case.lens
    for step in range(int(lens.max())):
        act = step < lens
        cnt = act.to(torch.int32)
        cu = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
        cu[1:] = torch.cumsum(cnt, 0)
        sel = (case.cu[:-1] + step)[act]
        B.quantize_kv(cache, case.k[sel].to(DEV), case.v[sel].to(DEV), bt,
                      torch.full((case.n_seqs,), step, dtype=torch.int32, device=DEV), cu.to(DEV), 1)
    compare_pools(ref, case, cache.pool.cpu().numpy(), want)


@pytest.mark.parametrize("mode", ["prefill", "token"])
@pytest.mark.parametrize("cid", [2, 1])
def test_quantize_signed_zeros_and_threshold_ties(B, ref, cid, mode):
    """Values exactly on the thresholds and zeros of both signs, in both quantize kernels
    (a prefill call, and one token per call): thresholds (-1, -0, +0, 1), where zeros of
    either sign are inner (side set: x >= 0 holds for -0) and every other value is a middle
    or outer one, and (-0.5, -0.25, 0.25, 0.5) with a quarter of the inputs planted on
    +-0, +-0.25, +-0.5 and +-1 (a value on a threshold stays in the narrower group)."""
    w = synth.scaled(synth.WORKLOADS[cid], n_seqs=3, ctx=37)
    case = Case(w)
    thr = np.zeros((case.H, 2, 4), np.float32)
    thr[0::2] = np.array([-1.0, -0.0, 0.0, 1.0], np.float32)
    thr[1::2] = np.array([-0.5, -0.25, 0.25, 0.5], np.float32)
    case.thr = thr
    g = torch.Generator().manual_seed(11)
    planted = torch.tensor([-0.0, 0.0, -0.25, 0.25, -0.5, 0.5, -1.0, 1.0], dtype=case.k.dtype)
    for x in (case.k, case.v):
        flat = x.view(-1)
        n = flat.numel() // 4
        flat[torch.randint(0, flat.numel(), (n,), generator=g)] = planted[torch.randint(0, 8, (n,), generator=g)]
    want = case.oracle_pool(ref)
    if mode == "prefill":
        cache, _ = _gpu_cache(B, case)
    else:
        cache, bt = _gpu_cache(B, case, prefill=False)
        lens = case.lens
        for step in range(int(lens.max())):
            act = step < lens
            cu = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
            cu[1:] = torch.cumsum(act.to(torch.int32), 0)
            sel = (case.cu[:-1] + step)[act]
            B.quantize_kv(cache, case.k[sel].to(DEV), case.v[sel].to(DEV), bt,
                          torch.full((case.n_seqs,), step, dtype=torch.int32, device=DEV), cu.to(DEV), 1)
    compare_pools(ref, case, cache.pool.cpu().numpy(), want)


@pytest.mark.parametrize("name", list(CASES))
def test_attention_matches_oracle(B, ref, name):
    case = _case(ref, name)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case)
    compare_pools(ref, case, cache.pool.cpu().numpy(), pool_ref)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, 16, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), scale)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"{name}: max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)


def test_attention_single_token_and_ragged(B, ref):
    """Lengths 1 (softmax over one token), exact page multiples and ragged tails in one
    batch; max_seq_len larger than every length."""
    w = synth.scaled(synth.WORKLOADS[4], n_seqs=6)
    case = Case(w, lens=[1, 16, 17, 31, 64, 250])
    case.calibrate_oracle(ref)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case)
    q = synth.queries(case.w)
    scale = 0.088
    want = ref.decode_attention(pool_ref, case.num_blocks, 16, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), scale)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), case.max_blocks * 16, scale)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    assert ok, (max_abs, max_rel)


@pytest.mark.parametrize("name,window", [("tiny", 1), ("tiny", 5), ("llama2-7b", 17), ("llama2-13b", 1000),
                                         ("mistral-gqa", 16), ("mistral-gqa", 513), ("llama3-32k", 2049),
                                         ("llama2-13b-wide", 20)])
def test_attention_sliding_window(B, ref, name, window):
    """Sliding-window attention (keys L-W .. L-1) against the oracle: windows shorter than
    a page, straddling page boundaries, and longer than some of the sequences."""
    case = _case(ref, name)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, 16, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), scale, window=window)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale, window=window)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"{name} window {window}: max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)


def test_attention_sliding_window_ragged(B, ref):
    """Windows of 1, 15, 16, 17 and L tokens over lengths that are page multiples and
    ragged; max_seq_len larger than every length."""
    w = synth.scaled(synth.WORKLOADS[4], n_seqs=6)
    case = Case(w, lens=[1, 16, 17, 31, 64, 250])
    case.calibrate_oracle(ref)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case)
    q = synth.queries(case.w)
    for window in (1, 15, 16, 17, 250):
        want = ref.decode_attention(pool_ref, case.num_blocks, 16, case.H, case.d, case.thr, np16(q),
                                    case.bt.numpy(), case.lens.numpy(), 0.088, window=window)
        got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), case.max_blocks * 16, 0.088,
                                 window=window)
        ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
        assert ok, (window, max_abs, max_rel)


@pytest.mark.parametrize("mode", ["all-outliers", "no-inner", "mixed"])
def test_attention_edge_thresholds(B, ref, mode):
    """Attention over extreme COO loads: every value an outlier (the largest page groups,
    read from HBM instead of staged), no inner group, and heads alternating between the
    two; with collapsed intervals, zero and constant vectors."""
    w = synth.scaled(synth.WORKLOADS[3], n_seqs=3, ctx=300)
    case = Case(w)
    H = case.H
    thr = np.zeros((H, 2, 4), np.float32)
    if mode in ("all-outliers", "mixed"):
        thr[:, :, 0], thr[:, :, 1], thr[:, :, 2], thr[:, :, 3] = -np.inf, -np.inf, np.inf, np.inf
    if mode in ("no-inner", "mixed"):
        sel = slice(None) if mode == "no-inner" else slice(1, None, 2)
        thr[sel] = np.array([-1.0, 0.0, 0.0, 1.0], np.float32)
    case.thr = thr
    case.k[3] = 0.0
    case.v[5] = 1.5
    case.k[7, :, :64] = -2.0
    pool_ref = case.oracle_pool(ref)
    cache, bt = _gpu_cache(B, case)
    compare_pools(ref, case, cache.pool.cpu().numpy(), pool_ref)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, 16, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), scale)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"{mode}: max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)


def test_abi_rejects_bad_arguments_on_gpu(B):
    thr = torch.zeros(2, 2, 4, device=DEV)
    cache = B.Cache(4, 2, 128, thr)
    q = torch.zeros(1, 4, 128, dtype=torch.float16, device=DEV)
    bt = torch.zeros(1, 4, dtype=torch.int32, device=DEV)
    lens = torch.ones(1, dtype=torch.int32, device=DEV)
    with pytest.raises(B.OakenError) as e:
        B.decode_attention(cache, torch.zeros(1, 3, 128, dtype=torch.float16, device=DEV), bt, lens, 16, 0.1)
    assert e.value.status == 1
    with pytest.raises(B.OakenError):
        B.decode_attention(cache, q, bt, lens, 4096, 0.1)   # block table too narrow
