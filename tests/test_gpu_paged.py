"""GPU parity with on-demand sparse pages (the dense and sparse management tables of
Sec. 5.2): COO bytes live in a separate pool of 256-byte pages taken as each record's
stream grows.

Every record is reassembled into the fixed layout (counts, meta and nibbles from the
record, then its COO stream gathered through its sparse page table) and compared bit for
bit with the oracle's record.  Page ownership is checked too: held pages are in range
and distinct, and the free list counts exactly the pages nobody holds.  Attention over
the paged cache is compared with the oracle within the stated tolerance.
"""
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import Case, attention_tolerance, compare_pools, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
P = 16
SPB = 256


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _case(ref, cid, **kw):
    c = Case(synth.scaled(synth.WORKLOADS[cid], **kw))
    c.calibrate_oracle(ref)
    return c


def _paged_cache(B, case, pages=None, prefill=True):
    nrec = case.num_blocks * case.H * 2
    cache = B.Cache(case.num_blocks, case.H, case.d, torch.from_numpy(case.thr).to(DEV),
                    sparse_pages=pages or 2 * nrec + 16)
    bt = case.bt.to(DEV)
    if prefill:
        B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt,
                      torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), case.cu.to(DEV),
                      int(case.lens.max()))
    return cache, bt


def _assemble(ref, case, cache):
    """Fixed-layout image of every record, plus each record's page table and page need."""
    lay = ref.layout(P, case.d)
    nrec = case.num_blocks * case.H * 2
    nt = P * case.d // SPB
    recs = cache.pool.cpu().numpy().reshape(nrec, cache.stride)
    spool = cache.sparse_pool.cpu().numpy().reshape(-1, SPB)
    tab = np.ascontiguousarray(recs[:, lay["sparse"]:lay["sparse"] + 4 * nt]).view(np.int32)
    used = recs[:, :lay["meta"]].astype(np.int64).sum(1)
    need = (used + SPB - 1) // SPB
    out = np.zeros((nrec, lay["stride"]), np.uint8)
    out[:, :lay["sparse"]] = recs[:, :lay["sparse"]]
    for i in range(nt):
        rows = np.nonzero(need > i)[0]
        ids = tab[rows, i] - 1
        assert ((ids >= 0) & (ids < cache.sparse_pages)).all(), "a needed page is missing or out of range"
        out[rows, lay["sparse"] + SPB * i: lay["sparse"] + SPB * (i + 1)] = spool[ids]
    return out.reshape(-1), tab, need


def _check_ownership(B, cache, tab):
    held = tab[tab > 0] - 1
    assert held.min(initial=0) >= 0 and held.max(initial=-1) < cache.sparse_pages
    assert np.unique(held).size == held.size, "a sparse page is held by two records"
    free, overflow = cache.sparse_status()
    assert not overflow
    assert free == cache.sparse_pages - held.size, (free, cache.sparse_pages, held.size)
    return held.size


@pytest.mark.parametrize("cid,kw", [(2, dict(n_seqs=6, ctx=203)), (3, dict(n_seqs=3, ctx=2048)),
                                    (4, dict(n_seqs=5, ctx=1500, ctx_min=1)), (3, dict(n_seqs=103, ctx=37)),
                                    (1, dict())])
def test_paged_prefill_bit_exact(B, ref, cid, kw):
    case = _case(ref, cid, **kw)
    want = case.oracle_pool(ref)
    cache, _ = _paged_cache(B, case)
    got, tab, need = _assemble(ref, case, cache)
    assert compare_pools(ref, case, got, want) > 0
    held = _check_ownership(B, cache, tab)
    assert held == int(need.sum())   # pages are taken only as the streams need them
    # the fixed records would reserve P*d COO bytes each
    print(f"workload {case.w.name}: {held} sparse pages for {need.size} records "
          f"({held * SPB / max(1, need.size):.0f} B/record vs {P * case.d} reserved)")


def test_paged_decode_append_and_rewrite(B, ref):
    """Token-by-token appends take pages as streams cross 256-byte boundaries; writing the
    same position again reuses the pages the record holds."""
    case = _case(ref, 4, n_seqs=5, ctx=300, ctx_min=1)
    n_dec = 40
    lens = case.lens.clone()
    pre = torch.clamp(lens - n_dec, min=0)
    cache, bt = _paged_cache(B, case, prefill=False)
    rows = torch.cat([torch.arange(int(case.cu[s]), int(case.cu[s]) + int(pre[s])) for s in range(case.n_seqs)])
    cu_pre = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
    cu_pre[1:] = torch.cumsum(pre, 0)
    B.quantize_kv(cache, case.k[rows].to(DEV), case.v[rows].to(DEV), bt,
                  torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), cu_pre.to(DEV), int(pre.max()))

    def step(pos):
        act = pos < lens
        r = (case.cu[:-1] + pos).clamp(max=int(case.cu[-1]) - 1)
        cu = torch.zeros(case.n_seqs + 1, dtype=torch.int32)
        cu[1:] = torch.cumsum(act.to(torch.int32), 0)
        sel = r[act]
        B.quantize_kv(cache, case.k[sel].to(DEV), case.v[sel].to(DEV), bt, pos.to(torch.int32).to(DEV),
                      cu.to(DEV), 1)

    for i in range(n_dec):
        step(pre + i)
    free_before, _ = cache.sparse_status()
    step(lens - 1)            # the last position again: same bytes, same pages
    step(lens - 1)
    free_after, _ = cache.sparse_status()
    assert free_after == free_before
    want = case.oracle_pool(ref)
    got, tab, _ = _assemble(ref, case, cache)
    compare_pools(ref, case, got, want)
    _check_ownership(B, cache, tab)


def test_paged_release_and_reuse(B, ref):
    """Releasing blocks returns exactly their pages and empties their records; refilling
    reproduces the same records."""
    case = _case(ref, 2, n_seqs=6, ctx=203)
    want = case.oracle_pool(ref)
    cache, bt = _paged_cache(B, case)
    _, tab, _ = _assemble(ref, case, cache)
    held0 = _check_ownership(B, cache, tab)
    # sequence 0's blocks
    nb0 = math.ceil(int(case.lens[0]) / P)
    blocks = case.bt[0, :nb0].clone()
    lay = ref.layout(P, case.d)
    recs = cache.pool.cpu().numpy().reshape(case.num_blocks, case.H, 2, cache.stride)
    t0 = np.ascontiguousarray(recs[blocks.numpy(), :, :, lay["sparse"]:lay["sparse"] + 4 * (P * case.d // SPB)])
    n_rel = int((t0.view(np.int32) > 0).sum())
    cache.release(blocks.to(torch.int32).to(DEV))
    free, overflow = cache.sparse_status()
    assert not overflow and free == cache.sparse_pages - held0 + n_rel
    recs = cache.pool.cpu().numpy().reshape(case.num_blocks, case.H, 2, cache.stride)
    assert not recs[blocks.numpy(), :, :, :lay["meta"]].any(), "released records keep counts"
    # release everything, then prefill again: same records, same page count
    cache.release(torch.arange(case.num_blocks, dtype=torch.int32, device=DEV))
    assert cache.sparse_status() == (cache.sparse_pages, False)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt,
                  torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV), case.cu.to(DEV), int(case.lens.max()))
    got, tab, _ = _assemble(ref, case, cache)
    compare_pools(ref, case, got, want)
    assert _check_ownership(B, cache, tab) == held0


def test_paged_overflow_sets_flag(B, ref):
    """A pool too small for the cache sets the overflow flag; attention still runs, reading
    only inside the pools; a reset clears the flag."""
    case = _case(ref, 2, n_seqs=6, ctx=203)
    cache, bt = _paged_cache(B, case, pages=8)
    free, overflow = cache.sparse_status()
    assert overflow and 0 <= free <= 8
    q = synth.queries(case.w)
    out = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), 0.088)
    torch.cuda.synchronize()
    assert out.shape == (case.n_seqs, case.Hq, case.d)
    cache.sparse_reset()
    assert cache.sparse_status() == (8, False)


def test_paged_exact_pool_never_overflows(B, ref):
    """A pool holding exactly the pages the records need: every concurrent reservation
    succeeds (a reservation only takes pages while enough are free), the list ends empty
    and the records are bit-exact."""
    case = _case(ref, 4, n_seqs=5, ctx=1500, ctx_min=1)
    want = case.oracle_pool(ref)
    big, _ = _paged_cache(B, case)
    _, tab, need = _assemble(ref, case, big)
    n_need = int(need.sum())
    del big
    for _ in range(3):
        cache, _ = _paged_cache(B, case, pages=n_need)
        free, overflow = cache.sparse_status()
        assert not overflow and free == 0, (free, overflow)
        got, tab, _ = _assemble(ref, case, cache)
        compare_pools(ref, case, got, want)
        held = tab[tab > 0] - 1
        assert np.unique(held).size == held.size == n_need


def _free_list(cache):
    fl = cache.sparse_free.cpu().numpy()
    return int(fl[0]), fl[2:2 + int(fl[0])]


def test_paged_overflow_then_release_restores_the_list(B, ref):
    """An undersized pool overflows; after every block is released the free list holds
    each page exactly once (no page handed to two records, none lost)."""
    case = _case(ref, 4, n_seqs=5, ctx=1500, ctx_min=1)
    pages = 200
    cache, bt = _paged_cache(B, case, pages=pages)
    free, overflow = cache.sparse_status()
    assert overflow
    tab = _tables(B, case, cache)
    held = tab[tab > 0] - 1
    assert np.unique(held).size == held.size, "a sparse page is held by two records"
    assert free == pages - held.size
    cache.release(torch.arange(case.num_blocks, dtype=torch.int32, device=DEV))
    n, ids = _free_list(cache)
    assert n == pages and np.array_equal(np.sort(ids), np.arange(pages))


def _tables(B, case, cache):
    """Every record's sparse page table (int32 [records][entries])."""
    nt = P * case.d // SPB
    recs = cache.pool.cpu().numpy().reshape(case.num_blocks * case.H * 2, cache.stride)
    off = B.record_layout(case.d)["sparse"]
    return np.ascontiguousarray(recs[:, off:off + 4 * nt]).view(np.int32)


@pytest.mark.parametrize("cid,kw,window", [(2, dict(n_seqs=6, ctx=203), 0), (3, dict(n_seqs=3, ctx=2048), 0),
                                           (4, dict(n_seqs=5, ctx=1500, ctx_min=1), 0),
                                           (4, dict(n_seqs=5, ctx=1500, ctx_min=1), 513),
                                           (5, dict(n_seqs=2, ctx=3000), 0), (3, dict(n_seqs=103, ctx=37), 0)])
def test_paged_attention_matches_oracle(B, ref, cid, kw, window):
    case = _case(ref, cid, **kw)
    pool_ref = case.oracle_pool(ref)
    cache, bt = _paged_cache(B, case)
    q = synth.queries(case.w)
    scale = float(np.float32(1.0 / math.sqrt(case.d)))
    want = ref.decode_attention(pool_ref, case.num_blocks, P, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), scale, window=window)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), scale, window=window)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    print(f"{case.w.name} window {window}: max_abs={max_abs:.3e}")
    assert ok, (max_abs, max_rel)


def test_paged_attention_all_outliers(B, ref):
    """Every value an outlier: 2 KiB COO streams over eight sparse pages per record, read
    from HBM through the page table (larger than a staging slot)."""
    w = synth.scaled(synth.WORKLOADS[2], n_seqs=2, ctx=40)
    case = Case(w)
    thr = np.zeros((case.H, 2, 4), np.float32)
    thr[:, :, 0], thr[:, :, 1], thr[:, :, 2], thr[:, :, 3] = -np.inf, -np.inf, np.inf, np.inf
    case.thr = thr
    pool_ref = case.oracle_pool(ref)
    cache, bt = _paged_cache(B, case, pages=case.num_blocks * case.H * 2 * (P * case.d // SPB))
    assert not cache.sparse_status()[1]
    got_pool, tab, need = _assemble(ref, case, cache)
    compare_pools(ref, case, got_pool, pool_ref)
    assert need.max() == P * case.d // SPB
    q = synth.queries(case.w)
    want = ref.decode_attention(pool_ref, case.num_blocks, P, case.H, case.d, case.thr, np16(q),
                                case.bt.numpy(), case.lens.numpy(), 0.088)
    got = B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), 0.088)
    ok, max_abs, max_rel = attention_tolerance(got.cpu().numpy(), want)
    assert ok, (max_abs, max_rel)


def test_paged_attention_rejects_unsupported_shape(B, ref):
    """Paged attention needs head_dim 128 (the matrix-core kernel)."""
    case = _case(ref, 1)
    cache, bt = _paged_cache(B, case)
    q = synth.queries(case.w)
    with pytest.raises(B.OakenError) as e:
        B.decode_attention(cache, q.to(DEV), bt, case.lens.to(DEV), int(case.lens.max()), 0.125)
    assert e.value.status == 2
