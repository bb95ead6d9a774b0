"""Parity at the full workload sizes the benchmark runs.

The whole cache is built on the GPU through the C ABI, the same way the benchmark builds
it: prefill quantization of all but the last token of every sequence, then one appended
token per sequence.  Decode attention then runs over every sequence.

A sample of sequences is checked against the oracle:
- their page records (counts, scales, nibbles, COO bytes) bit for bit;
- their attention outputs within |gpu - ref| <= 2e-3 + 1e-2 |ref|.

The sample includes the shortest and the longest sequence when lengths vary.  The
Mistral-shaped workload is also checked under Mistral-7B's 4096-token sliding window.
"""
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import attention_tolerance, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
P = 16


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _sample(lens: torch.Tensor, n: int):
    order = torch.argsort(lens, stable=True).tolist()
    picks = {order[0], order[-1]}
    step = max(1, len(order) // n)
    for i in range(0, len(order), step):
        if len(picks) >= n:
            break
        picks.add(order[i])
    return sorted(picks)


@pytest.mark.parametrize("cid,n_sample,window", [(3, 6, 0), (4, 6, 4096), (5, 2, 0)])
def test_full_size_sampled_parity(B, ref, cid, n_sample, window):
    w = synth.WORKLOADS[cid]
    H, Hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    n = w.n_seqs

    # thresholds on the GPU; they must equal the oracle's bit for bit
    kc = synth.calibration_set(w, "k", DEV)
    vc = synth.calibration_set(w, "v", DEV)
    thr = B.calibrate_thresholds(kc, vc, 0.04, 0.06)
    thr_np = thr.cpu().numpy()
    want_thr = ref.calibrate(np16(kc), np16(vc), 0.04, 0.06)
    assert np.array_equal(thr_np.view(np.uint32), want_thr.view(np.uint32))
    del kc, vc

    # full cache: prefill all but the last token of each sequence, then append it
    lens = synth.seq_lengths(w)
    bt_cpu, nblk = synth.block_table(w, lens)
    bt = bt_cpu.to(DEV)
    cache = B.Cache(nblk, H, d, thr)
    for s0 in range(0, n, 16):
        ss = list(range(s0, min(n, s0 + 16)))
        pre = [int(lens[s]) - 1 for s in ss]
        k = torch.cat([synth.kv_values_seq(w, "k", s, p, DEV) for s, p in zip(ss, pre)])
        v = torch.cat([synth.kv_values_seq(w, "v", s, p, DEV) for s, p in zip(ss, pre)])
        cu = torch.zeros(len(ss) + 1, dtype=torch.int32)
        cu[1:] = torch.cumsum(torch.tensor(pre, dtype=torch.int32), 0)
        B.quantize_kv(cache, k, v, bt[s0:s0 + len(ss)].contiguous(),
                      torch.zeros(len(ss), dtype=torch.int32, device=DEV), cu.to(DEV), max(pre))
        del k, v
    k_new = synth.new_token_values(w, "k", 0, DEV)
    v_new = synth.new_token_values(w, "v", 0, DEV)
    B.quantize_kv(cache, k_new, v_new, bt, (lens - 1).to(torch.int32).to(DEV),
                  torch.arange(n + 1, dtype=torch.int32, device=DEV), 1)
    q = synth.queries(w, 0, DEV)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    out = B.decode_attention(cache, q, bt, lens.to(DEV), int(lens.max()), scale).cpu().numpy()

    # oracle on the sample, with its own compact block table
    sample = _sample(lens, n_sample)
    S = len(sample)
    lay = ref.layout(P, d)
    nb_s = [(int(lens[s]) + P - 1) // P for s in sample]
    bt_s = np.zeros((S, max(nb_s)), np.int32)
    off = 0
    for i, nb in enumerate(nb_s):
        bt_s[i, :nb] = np.arange(off, off + nb)
        off += nb
    pool_s = np.zeros(off * H * 2 * lay["stride"], np.uint8)
    pre = np.array([int(lens[s]) - 1 for s in sample], np.int32)
    kk = torch.cat([synth.kv_values_seq(w, "k", s, int(p), DEV) for s, p in zip(sample, pre)]).cpu().numpy()
    vv = torch.cat([synth.kv_values_seq(w, "v", s, int(p), DEV) for s, p in zip(sample, pre)]).cpu().numpy()
    cu = np.concatenate([[0], np.cumsum(pre)]).astype(np.int32)
    ref.quantize_kv(pool_s, off, P, H, d, thr_np, kk, vv, bt_s, np.zeros(S, np.int32), cu)
    del kk, vv
    ref.quantize_kv(pool_s, off, P, H, d, thr_np, k_new.cpu().numpy()[sample], v_new.cpu().numpy()[sample],
                    bt_s, pre, np.arange(S + 1, dtype=np.int32))

    # the sampled sequences' records, bit for bit (used prefix of each record)
    st = lay["stride"]
    rec_gpu = cache.pool.view(nblk, H, 2, st)
    want_recs = pool_s.reshape(off, H, 2, st)
    n_checked = 0
    for i, s in enumerate(sample):
        blocks = bt_cpu[s, :nb_s[i]].long().to(DEV)
        got = rec_gpu.index_select(0, blocks).cpu().numpy()
        want = want_recs[bt_s[i, :nb_s[i]]]
        for pg in range(nb_s[i]):
            for h in range(H):
                for wh in (0, 1):
                    e = want[pg, h, wh]
                    used = lay["sparse"] + int(e[:lay["meta"]].sum())
                    if not np.array_equal(got[pg, h, wh, :used], e[:used]):
                        bad = int(np.nonzero(got[pg, h, wh, :used] != e[:used])[0][0])
                        raise AssertionError(f"seq {s} page {pg} head {h} {'KV'[wh]}: byte {bad} differs")
                    n_checked += 1
    assert n_checked == sum(nb_s) * H * 2

    lens_s = np.array([int(lens[s]) for s in sample], np.int32)
    want_out = ref.decode_attention(pool_s, off, P, H, d, thr_np, np16(q)[sample], bt_s, lens_s, scale)
    ok, max_abs, max_rel = attention_tolerance(out[sample], want_out)
    print(f"workload {w.name}: {S} sequences, {n_checked} records bit-exact, "
          f"attention max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
    assert ok, (max_abs, max_rel)

    if window:
        # the same cache under the model's sliding window
        out_w = B.decode_attention(cache, q, bt, lens.to(DEV), int(lens.max()), scale, window=window)
        want_w = ref.decode_attention(pool_s, off, P, H, d, thr_np, np16(q)[sample], bt_s, lens_s, scale,
                                      window=window)
        ok, max_abs, max_rel = attention_tolerance(out_w.cpu().numpy()[sample], want_w)
        print(f"  window {window}: attention max_abs={max_abs:.3e} max_rel={max_rel:.3e}")
        assert ok, (max_abs, max_rel)
