"""The allocation-free decode attention (split partials in the library's static scratch)
against the entry point with a caller workspace: same kernels, so the outputs must be
identical, over two calls in a row on one device, the second smaller than the first; and
sizes beyond the scratch are rejected before anything runs."""
import ctypes
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import Case

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _setup(B, ref, cid, **kw):
    case = Case(synth.scaled(synth.WORKLOADS[cid], **kw))
    case.calibrate_oracle(ref)
    cache = B.Cache(case.num_blocks, case.H, case.d, torch.from_numpy(case.thr).to(DEV))
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k.to(DEV), case.v.to(DEV), bt, torch.zeros(case.n_seqs, dtype=torch.int32, device=DEV),
                  case.cu.to(DEV), int(case.lens.max()))
    return case, cache, bt


def test_noalloc_matches_workspace_entry_point(ref):
    from paper_2503_18599_amd import binding as B
    runs = [(3, dict(n_seqs=8, ctx=2048), 0), (4, dict(n_seqs=5, ctx=700, ctx_min=1), 300)]
    for cid, kw, window in runs:   # the second call is smaller than the first
        case, cache, bt = _setup(B, ref, cid, **kw)
        q = synth.queries(case.w).to(DEV)
        scale = float(np.float32(1.0 / math.sqrt(case.d)))
        max_len = int(case.lens.max())
        assert B.attention_workspace_bytes(case.n_seqs, case.Hq, case.H, case.d, max_len, window) > 0
        want = B.decode_attention(cache, q, bt, case.lens.to(DEV), max_len, scale, window=window)
        out = torch.full_like(want, float("nan"))
        got = B.decode_attention_noalloc(cache, q, bt, case.lens.to(DEV), max_len, scale, out, window=window)
        torch.cuda.synchronize()
        assert torch.equal(got, want), float((got - want).abs().max())


def test_noalloc_rejects_partials_beyond_the_scratch(ref):
    from paper_2503_18599_amd import binding as B
    case, cache, bt = _setup(B, ref, 2, n_seqs=2, ctx=64)
    L = B.lib()
    # 4096 sequences of 32768 tokens: far more split partials than the scratch holds
    n, hq = 4096, case.Hq
    need = L.oaken_attention_workspace_bytes(n, hq, case.H, case.d, 32768)
    assert need > (32 << 20)
    q = torch.zeros(n, hq, case.d, dtype=torch.float16, device=DEV)
    out = torch.zeros(n, hq, case.d, dtype=torch.float32, device=DEV)
    lens = torch.ones(n, dtype=torch.int32, device=DEV)
    bt_wide = torch.zeros(n, 2048, dtype=torch.int32, device=DEV)
    st = L.oaken_decode_attention_noalloc(cache.struct, q.data_ptr(), hq, bt_wide.data_ptr(), 2048, lens.data_ptr(),
                                          n, 32768, 0, ctypes.c_float(0.1), out.data_ptr(), None)
    assert st == 3 and b"scratch" in L.oaken_last_error()
