"""The benchmark's roofline numerator: the algorithmic bytes of one attention launch, counted
from the records' COO counts by bench.py, against a position-by-position count over a cache
the oracle wrote (CPU; no GPU)."""
import types

import numpy as np
import torch

import bench
from paper_2503_18599_amd import synth
from tests.cases import P, Case


def test_attention_bytes_match_a_count_per_position(ref):
    w = synth.scaled(synth.WORKLOADS[2], n_seqs=3, ctx=203)
    case = Case(w, lens=[203, 17, 64])
    case.calibrate_oracle(ref)
    pool = case.oracle_pool(ref)
    lay = ref.layout(P, case.d)
    st, nc = lay["stride"], case.d // 64
    cache = types.SimpleNamespace(head_dim=case.d, n_kv_heads=case.H, num_blocks=case.num_blocks,
                                  pool=torch.from_numpy(pool), stride=st)
    prefix = bench.outlier_prefix(cache, case.bt, case.n_seqs, int(case.lens.max()))
    for window in (0, 50):
        kv, total, n_out, n_vec, pages = bench.attention_bytes(cache, prefix, case.lens, window, case.Hq,
                                                               case.n_seqs)
        want_out = want_vec = want_pages = 0
        for s in range(case.n_seqs):
            L = int(case.lens[s])
            lo = max(0, L - window) if window else 0
            want_pages += (L + P - 1) // P - lo // P
            for pos in range(lo, L):
                blk, slot = int(case.bt[s, pos // P]), pos % P
                for h in range(case.H):
                    for wv in (0, 1):
                        off = ((blk * case.H + h) * 2 + wv) * st + lay["counts"] + slot * nc
                        want_out += int(pool[off:off + nc].astype(np.int64).sum())
                        want_vec += 1
        assert (n_out, n_vec, pages) == (want_out, want_vec, want_pages), window
        # per vector: d/2 nibbles, d/64 count bytes, 12 metadata bytes; then its COO bytes
        assert kv == want_vec * (case.d // 2 + nc + 12) + want_out
        # plus queries (fp16 in, fp32 out), block-table entries and lengths
        assert total == kv + case.n_seqs * case.Hq * case.d * 6 + want_pages * 4 + case.n_seqs * 4
        assert 0 < want_out < want_vec * case.d
