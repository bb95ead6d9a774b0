"""Pins for the oracle's paged record writer/reader and its decode attention (Sec. 2.1,
Sec. 5.2 MMU / dequantization engine) against closed forms and invariants."""
import math

import numpy as np
import pytest

P = 16


def _build(ref, rng, n_seqs, H, d, lens, thr=None, k=None, v=None, shuffle=True):
    lay = ref.layout(P, d)
    nb = [math.ceil(L / P) for L in lens]
    total = sum(nb)
    perm = rng.permutation(total) if shuffle else np.arange(total)
    bt = np.zeros((n_seqs, max(nb)), np.int32)
    off = 0
    for s, n in enumerate(nb):
        bt[s, :n] = perm[off:off + n]
        off += n
    if thr is None:
        thr = np.tile(np.array([-2.5, -0.1, 0.1, 2.5], np.float32), (H, 2, 1))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ntok = int(cu[-1])
    if k is None:
        k = (rng.standard_t(3, (ntok, H, d))).astype(np.float16)
    if v is None:
        v = (rng.standard_t(3, (ntok, H, d))).astype(np.float16)
    pool = np.zeros(total * H * 2 * lay["stride"], np.uint8)
    ref.quantize_kv(pool, total, P, H, d, thr, k, v, bt, np.zeros(n_seqs, np.int32), cu)
    return pool, total, bt, thr, k, v, cu


def _dq(ref, pool, H, d, thr, bt, s, t, h, which):
    return ref.dequantize_slot(pool, P, H, d, thr, int(bt[s, t // P]), h, which, t % P)


def test_incremental_append_equals_bulk(ref):
    """Appending tokens one call at a time (decode) gives the same records as one bulk
    call (prefill): later slots find their sparse bytes after the earlier slots'."""
    rng = np.random.default_rng(31)
    H, d, lens = 2, 128, [37, 16, 5]
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 3, H, d, lens)
    pool2 = np.zeros_like(pool)
    for step in range(max(lens)):
        act = [s for s in range(3) if step < lens[s]]
        rows = np.array([cu[s] + step for s in act])
        sub_bt = bt[act]
        ref.quantize_kv(pool2, total, P, H, d, thr, k[rows], v[rows], sub_bt,
                        np.full(len(act), step, np.int32), np.arange(len(act) + 1, dtype=np.int32))
    lay = ref.layout(P, d)
    for blk in range(total):
        for h in range(H):
            for which in (0, 1):
                a = ref.record(pool, P, H, d, blk, h, which)
                b = ref.record(pool2, P, H, d, blk, h, which)
                used = lay["sparse"] + int(a[:lay["meta"]].sum())
                assert np.array_equal(a[:used], b[:used])


def test_sparse_offsets_are_prefix_sums(ref):
    rng = np.random.default_rng(32)
    H, d = 1, 128
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 1, H, d, [16])
    lay = ref.layout(P, d)
    rec = ref.record(pool, P, H, d, int(bt[0, 0]), 0, 0)
    counts = rec[:P * 2].reshape(P, 2).astype(int)
    start = 0
    for t in range(P):
        r = ref.quantize_vector(k[t, 0], thr[0, 0])
        n = len(r["coo"])
        assert counts[t].tolist() == r["counts"].tolist()
        assert rec[lay["sparse"] + start: lay["sparse"] + start + n].tolist() == r["coo"].tolist()
        start += n


def test_single_token_returns_its_value(ref):
    """L = 1: softmax over one token is 1, so out = dequantized v_0 for every query head."""
    rng = np.random.default_rng(33)
    H, d, Hq = 2, 64, 6
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 2, H, d, [1, 1])
    q = rng.standard_normal((2, Hq, d)).astype(np.float16)
    out = ref.decode_attention(pool, total, P, H, d, thr, q, bt, [1, 1], 0.125)
    for s in range(2):
        for hq in range(Hq):
            want = _dq(ref, pool, H, d, thr, bt, s, 0, hq // (Hq // H), 1)
            assert np.allclose(out[s, hq], want, rtol=1e-6, atol=1e-6)


def test_gqa_head_mapping(ref):
    """Query head h reads KV head h // (Hq/H): with L = 1 each query head must return the
    value vector of exactly that KV head (all KV heads differ)."""
    rng = np.random.default_rng(34)
    H, d, Hq = 4, 64, 16
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 1, H, d, [1])
    q = rng.standard_normal((1, Hq, d)).astype(np.float16)
    out = ref.decode_attention(pool, total, P, H, d, thr, q, bt, [1], 0.125)
    vals = [_dq(ref, pool, H, d, thr, bt, 0, 0, h, 1) for h in range(H)]
    for hq in range(Hq):
        match = [h for h in range(H) if np.allclose(out[0, hq], vals[h], atol=1e-6)]
        assert match == [hq // 4]


def test_equal_keys_give_mean_of_values(ref):
    """All keys equal (or q = 0) -> uniform softmax -> out = mean of dequantized values."""
    rng = np.random.default_rng(35)
    H, d, L = 1, 128, 40
    kconst = np.tile(rng.standard_normal(d).astype(np.float16), (L, H, 1))
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 1, H, d, [L], k=kconst)
    q = rng.standard_normal((1, 1, d)).astype(np.float16)
    vals = np.stack([_dq(ref, pool, H, d, thr, bt, 0, t, 0, 1) for t in range(L)])
    out = ref.decode_attention(pool, total, P, H, d, thr, q, bt, [L], 0.1)
    assert np.allclose(out[0, 0], vals.mean(0), rtol=1e-6, atol=1e-6)
    pool2, total2, bt2, thr2, k2, v2, _ = _build(ref, rng, 1, H, d, [L])
    vals2 = np.stack([_dq(ref, pool2, H, d, thr2, bt2, 0, t, 0, 1) for t in range(L)])
    out0 = ref.decode_attention(pool2, total2, P, H, d, thr2, np.zeros((1, 1, d), np.float16),
                                bt2, [L], 0.1)
    assert np.allclose(out0[0, 0], vals2.mean(0), rtol=1e-6, atol=1e-6)


def test_two_token_closed_form(ref):
    """L = 2: out = v0 + (v1 - v0) * sigmoid(s1 - s0) with s_t = scale * q . k_t, for every
    query head of a GQA layout (query head h uses its own q row and KV head h // G)."""
    rng = np.random.default_rng(36)
    H, d, Hq = 2, 64, 6
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 2, H, d, [2, 2])
    q = rng.standard_normal((2, Hq, d)).astype(np.float16)
    out = ref.decode_attention(pool, total, P, H, d, thr, q, bt, [2, 2], 0.125)
    for s in range(2):
        for hq in range(Hq):
            h = hq // (Hq // H)
            k0, k1 = (_dq(ref, pool, H, d, thr, bt, s, t, h, 0) for t in (0, 1))
            v0, v1 = (_dq(ref, pool, H, d, thr, bt, s, t, h, 1) for t in (0, 1))
            qd = q[s, hq].astype(np.float64)
            z = 0.125 * (qd @ k1 - qd @ k0)
            want = v0 + (v1 - v0) / (1.0 + math.exp(-z))
            assert np.allclose(out[s, hq], want, rtol=1e-6, atol=1e-6)


def test_output_is_convex_combination_and_page_order_invariant(ref):
    rng = np.random.default_rng(37)
    H, d, lens = 2, 128, [70, 33, 16]
    k = rng.standard_t(3, (sum(lens), H, d)).astype(np.float16)
    v = rng.standard_t(3, (sum(lens), H, d)).astype(np.float16)
    q = rng.standard_normal((3, 4, d)).astype(np.float16)
    outs = []
    for shuffle_seed in (1, 2):
        r2 = np.random.default_rng(shuffle_seed)
        pool, total, bt, thr, _, _, _ = _build(ref, r2, 3, H, d, lens, k=k, v=v)
        outs.append(ref.decode_attention(pool, total, P, H, d, thr, q, bt, lens, 0.09))
        for s, L in enumerate(lens):
            for hq in range(4):
                vals = np.stack([_dq(ref, pool, H, d, thr, bt, s, t, hq // 2, 1) for t in range(L)])
                o = outs[-1][s, hq].astype(np.float64)
                assert np.all(o >= vals.min(0) - 1e-5) and np.all(o <= vals.max(0) + 1e-5)
    assert np.array_equal(outs[0], outs[1])


def test_record_field_layout(ref):
    """Documented record layout: counts [P][d/64]; meta fp16 [P][6] little-endian
    (Min, Delta) x (inner, middle, outer); dense nibbles with K token-major (byte
    t*d/2 + j/2, low nibble = even j) and V channel-major (byte j*P/2 + t/2, low nibble =
    even t); the stride is a multiple of 128 bytes."""
    rng = np.random.default_rng(38)
    for d in (64, 128):
        H = 1
        pool, total, bt, thr, k, v, cu = _build(ref, rng, 1, H, d, [16])
        lay = ref.layout(P, d)
        assert lay["stride"] % 128 == 0 and lay["meta"] % 16 == 0 and lay["dense"] % 16 == 0
        for which, src in ((0, k), (1, v)):
            rec = ref.record(pool, P, H, d, int(bt[0, 0]), 0, which)
            for t in range(P):
                r = ref.quantize_vector(src[t, 0], thr[0, which])
                meta = rec[lay["meta"] + 12 * t: lay["meta"] + 12 * t + 12].view(np.uint16)
                assert meta.tolist() == r["meta"].tolist()
                assert rec[t * (d // 64):(t + 1) * (d // 64)].tolist() == r["counts"].tolist()
                for j in range(d):
                    if which == 0:
                        byte, high = t * d // 2 + j // 2, j & 1
                    else:
                        byte, high = j * P // 2 + t // 2, t & 1
                    b = int(rec[lay["dense"] + byte])
                    assert ((b >> 4) if high else (b & 15)) == (int(r["code"][j]) & 15)


def test_sliding_window_pins(ref):
    """Sliding window W (the Mistral/Mixtral models of Sec. 6.1): the query at position L-1
    sees keys L-W .. L-1.  Pinned three ways:
    - W >= L is the full attention;
    - W = 1 returns the last token's dequantized value;
    - quantization is per token, so windowed attention over L tokens equals plain
      attention over a fresh cache holding only the last W tokens (relocation)."""
    rng = np.random.default_rng(41)
    H, d, Hq = 2, 64, 4
    lens = [53, 40, 7]
    pool, total, bt, thr, k, v, cu = _build(ref, rng, 3, H, d, lens)
    q = rng.standard_normal((3, Hq, d)).astype(np.float16)
    full = ref.decode_attention(pool, total, P, H, d, thr, q, bt, lens, 0.125)
    assert np.array_equal(ref.decode_attention(pool, total, P, H, d, thr, q, bt, lens, 0.125, window=64), full)
    last = ref.decode_attention(pool, total, P, H, d, thr, q, bt, lens, 0.125, window=1)
    for s in range(3):
        for hq in range(Hq):
            want = _dq(ref, pool, H, d, thr, bt, s, lens[s] - 1, hq // (Hq // H), 1)
            assert np.array_equal(last[s, hq], want.astype(np.float32))
    for W in (5, 16, 17, 33):
        win = ref.decode_attention(pool, total, P, H, d, thr, q, bt, lens, 0.125, window=W)
        keep = [min(W, L) for L in lens]
        rows = np.concatenate([np.arange(cu[s + 1] - keep[s], cu[s + 1]) for s in range(3)])
        pool2, total2, bt2, _, _, _, _ = _build(ref, rng, 3, H, d, keep, thr=thr, k=k[rows], v=v[rows])
        want = ref.decode_attention(pool2, total2, P, H, d, thr, q, bt2, keep, 0.125)
        assert np.allclose(win, want, rtol=1e-6, atol=1e-7), W
        if W < min(lens):
            assert not np.allclose(win, full, atol=1e-4)
