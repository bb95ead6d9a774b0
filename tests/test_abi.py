"""Host-only tests of the C ABI (no GPU needed): the library loads, exports every
function declared in include/oaken.h, agrees with the oracle on the record layout, and
rejects bad arguments with the documented status codes before launching anything."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2503_18599_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("liboaken.so not built (run __graft_entry__.build())")
    return binding.lib()


def _declared():
    src = open(os.path.join(ROOT, "include", "oaken.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(oaken_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert len(names) >= 9
    for n in names:
        assert hasattr(L, n), n


def test_layout_matches_oracle(L, ref):
    from paper_2503_18599_amd import binding
    for d in (64, 128):
        assert binding.record_layout(d) == ref.layout(16, d)
        assert binding.record_bytes(d) == ref.layout(16, d)["stride"]
    assert L.oaken_record_bytes(16, 96) == -1
    assert L.oaken_record_bytes(8, 128) == -1


def test_status_strings(L):
    for s in range(5):
        assert L.oaken_status_string(s)
    assert L.oaken_status_string(99) == b"unknown status"


def _cache(**kw):
    from paper_2503_18599_amd.binding import _CacheStruct
    f = dict(num_blocks=4, block_size=16, n_kv_heads=2, head_dim=128, record_stride=3328,
             pool=0x1000, thresholds=0x2000)
    f.update(kw)
    return _CacheStruct(**f)


def test_quantize_validation(L):
    c = _cache()
    P = ctypes.byref
    assert L.oaken_quantize_kv(None, 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == 1
    assert L.oaken_quantize_kv(P(_cache(block_size=8)), 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == 2
    assert L.oaken_quantize_kv(P(_cache(head_dim=96)), 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == 2
    assert L.oaken_quantize_kv(P(_cache(record_stride=100)), 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == 1
    assert b"record_stride" in L.oaken_last_error()
    assert L.oaken_quantize_kv(P(_cache(pool=None)), 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == 1
    assert L.oaken_quantize_kv(P(c), None, 1, 1, 1, 1, 1, 1, 1, 1, None) == 1
    assert L.oaken_quantize_kv(P(c), 1, 1, 1, 0, 1, 1, 1, 1, 1, None) == 1
    assert L.oaken_quantize_kv(P(c), 1, 1, 1, 1, 1, 1, -1, 1, 1, None) == 1
    # nothing to write: succeeds without launching
    assert L.oaken_quantize_kv(P(c), 1, 1, 1, 1, 1, 1, 1, 0, 1, None) == 0
    assert L.oaken_last_error() == b""


def test_attention_validation(L):
    P = ctypes.byref
    c = _cache()
    args = lambda **kw: [kw.get("cache", P(c)), kw.get("q", 1), kw.get("hq", 4), 1, kw.get("mb", 128),
                         1, kw.get("ns", 1), kw.get("ml", 2048), kw.get("scale", 0.1), kw.get("out", 1),
                         None, 0, None]
    assert L.oaken_decode_attention(*args(hq=3)) == 1            # Hq not a multiple of H
    assert L.oaken_decode_attention(*args(hq=18)) == 2           # G > 8
    assert L.oaken_decode_attention(*args(q=None)) == 1
    assert L.oaken_decode_attention(*args(out=None)) == 1
    assert L.oaken_decode_attention(*args(mb=4)) == 1            # table narrower than max_seq_len
    assert L.oaken_decode_attention(*args(ns=0)) == 1
    assert L.oaken_decode_attention(*args(scale=float("inf"))) == 1
    # a long sequence on few units needs split partials: missing workspace is rejected
    need = L.oaken_attention_workspace_bytes(1, 4, 2, 128, 2048)
    assert need > 0
    assert L.oaken_decode_attention(*args()) == 3
    assert b"workspace" in L.oaken_last_error()
    # a workspace that is large enough but not 16-byte aligned is rejected before any launch
    a = args()
    a[10], a[11] = 0x1008, need
    assert L.oaken_decode_attention(*a) == 1
    assert b"aligned" in L.oaken_last_error()


def test_calibrate_validation(L):
    f = L.oaken_calibrate_thresholds
    assert f(None, 1, 1, 8, 1, 64, 0.04, 0.06, 1, 1, 1 << 20, None) == 1
    assert f(1, 1, 0, 8, 1, 64, 0.04, 0.06, 1, 1, 1 << 20, None) == 1
    assert f(1, 1, 1, 8, 1, 64, 1.0, 0.0, 1, 1, 1 << 20, None) == 1
    assert f(1, 1, 1, 8, 1, 64, 0.5, 0.6, 1, 1, 1 << 20, None) == 1
    assert f(1, 1, 1, 8, 1, 64, float("nan"), 0.0, 1, 1, 1 << 20, None) == 1
    assert f(1, 1, 2, 8, 1, 64, 0.04, 0.06, 1, 1, 4, None) == 3
    assert L.oaken_calibrate_workspace_bytes(2, 1) == 2 * 1 * 2 * 3 * 4


def test_probe_validation(L):
    f = L.oaken_probe_read
    assert f(None, 16, 16, 1, 0x1000, None) == 1
    assert f(0x1000, 16, 16, 1, None, None) == 1
    assert f(0x1000, 24, 32, 1, 0x2000, None) == 1        # not a multiple of 16
    assert f(0x1000, 8192, 8192, 1, 0x2000, None) == 1    # more than 4 KiB per record
    assert f(0x1000, 32, 16, 1, 0x2000, None) == 1        # stride shorter than the record
    assert f(0x1000, 16, 16, 0, 0x2000, None) == 1
    assert f(0x1008, 16, 16, 1, 0x2000, None) == 1        # base not 16-byte aligned
    assert b"aligned" in L.oaken_last_error()


def test_probe_chunk_limit(L):
    # 2^31 chunks of 16 bytes are beyond one call
    assert L.oaken_probe_read(0x1000, 4096, 4096, 1 << 23, 0x2000, None) == 1


def test_probe_record_division_rule():
    """The probe finds a chunk's record as (j * magic) >> (31 + l), l = ceil(log2 c),
    magic = ceil(2^(31 + l) / c): equal to j // c for every 31-bit j (checked at the ends
    of the range and on random values) and for every record length c of 1..256 chunks."""
    import random
    rng = random.Random(7)
    for c in range(1, 257):
        l = (c - 1).bit_length()
        s = 31 + l
        m = ((1 << s) + c - 1) // c
        assert m < (1 << 32)
        for j in [0, 1, c - 1, c, c + 1, (1 << 31) - 1, (1 << 31) - 2] + [rng.randrange(1 << 31) for _ in range(300)]:
            assert (j * m) >> s == j // c, (c, j)
