"""CPU oracle for Oaken's KV quantizer and decode attention (ctypes over numpy).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP library in ``paper_2503_18599_amd``.

Every function takes and returns numpy arrays; fp16 data travels as its uint16
bit pattern.  Section/equation references are to the Oaken paper (ISCA 2025).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oaken_ref.c")
_LIB_PATH = os.path.join(_HERE, "liboaken_ref.so")
_lib = None

INNER, MIDDLE, OUTER = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C11, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    lib.oaken_ref_half_to_float.argtypes = [ctypes.c_uint16]
    lib.oaken_ref_half_to_float.restype = f32
    lib.oaken_ref_float_to_half.argtypes = [f32]
    lib.oaken_ref_float_to_half.restype = ctypes.c_uint16
    lib.oaken_ref_layout.argtypes = [i32, i32, P]
    lib.oaken_ref_layout.restype = None
    lib.oaken_ref_quantize_vector.argtypes = [P, i32, P, P, P, P, P, P, P]
    lib.oaken_ref_quantize_vector.restype = None
    lib.oaken_ref_quantize_kv.argtypes = [P, i32, i32, i32, i32, i64, P, P, P, P, i32, P, P, i32]
    lib.oaken_ref_quantize_kv.restype = i32
    lib.oaken_ref_dequantize_slot.argtypes = [P, i32, i32, i32, i32, P, P, P]
    lib.oaken_ref_dequantize_slot.restype = None
    lib.oaken_ref_decode_attention.argtypes = [P, i32, i32, i32, i32, i64, P, P, i32, P, i32, P,
                                               i32, i32, f32, P]
    lib.oaken_ref_decode_attention.restype = i32
    lib.oaken_ref_calibrate.argtypes = [P, P, i32, i32, i32, i32, f32, f32, P]
    lib.oaken_ref_calibrate.restype = i32
    lib.oaken_ref_set_threads.argtypes = [i32]
    lib.oaken_ref_set_threads.restype = None
    lib.oaken_ref_max_threads.argtypes = []
    lib.oaken_ref_max_threads.restype = i32
    lib.oaken_ref_variant_info.argtypes = [i32, P]
    lib.oaken_ref_variant_info.restype = i32
    lib.oaken_ref_variant_quantize_vector.argtypes = [i32, P, i32, P, P, P, P, P, P]
    lib.oaken_ref_variant_quantize_vector.restype = i32
    lib.oaken_ref_variant_dequantize_vector.argtypes = [i32, P, P, P, P, i32, P, P]
    lib.oaken_ref_variant_dequantize_vector.restype = i32
    lib.oaken_ref_variant_quantize.argtypes = [i32, P, i32, i32, i32, P, P, P, P, P, P]
    lib.oaken_ref_variant_quantize.restype = i32
    lib.oaken_ref_variant_dequantize.argtypes = [i32, P, P, P, P, i32, i32, i32, P, P]
    lib.oaken_ref_variant_dequantize.restype = i32
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _bits16(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    assert a.dtype == np.uint16
    return np.ascontiguousarray(a)


# --------------------------------------------------------------------------- #
def half_to_float(bits: int) -> float:
    return float(_load().oaken_ref_half_to_float(int(bits)))


def float_to_half(x: float) -> int:
    return int(_load().oaken_ref_float_to_half(float(x)))


def layout(P: int, d: int) -> dict:
    """Byte offsets of the record fields and the record stride."""
    out = np.zeros(5, dtype=np.int64)
    _load().oaken_ref_layout(P, d, _ptr(out))
    return dict(counts=int(out[0]), meta=int(out[1]), dense=int(out[2]), sparse=int(out[3]),
                stride=int(out[4]))


def max_threads() -> int:
    return int(_load().oaken_ref_max_threads())


def set_threads(n: int) -> None:
    """Thread count of the oracle's parallel loops (for timing at 1 and at all cores)."""
    _load().oaken_ref_set_threads(int(n))


def quantize_vector(x, thr):
    """Eq. 1-4 + fused encoding for one vector.  Returns a dict of numpy arrays."""
    x = _bits16(x).reshape(-1)
    d = x.size
    assert d % 64 == 0
    thr = np.ascontiguousarray(np.asarray(thr, dtype=np.float32).reshape(4))
    code = np.zeros(d, np.uint8)
    group = np.zeros(d, np.uint8)
    meta = np.zeros(6, np.uint16)
    counts = np.zeros(d // 64, np.uint8)
    coo = np.zeros(d, np.uint8)
    n = ctypes.c_int(0)
    _load().oaken_ref_quantize_vector(_ptr(x), d, _ptr(thr), _ptr(code), _ptr(group), _ptr(meta),
                                      _ptr(counts), _ptr(coo), ctypes.byref(n))
    return dict(code=code, group=group, meta=meta, counts=counts, coo=coo[: n.value].copy())


def quantize_kv(pool: np.ndarray, num_blocks, P, H, d, thresholds, k_new, v_new, block_table,
                start_pos, cu_tokens):
    """Encode new K/V rows into the (host) page pool in place."""
    lay = layout(P, d)
    assert pool.dtype == np.uint8 and pool.size >= num_blocks * H * 2 * lay["stride"]
    thr = np.ascontiguousarray(np.asarray(thresholds, np.float32))
    k = _bits16(k_new)
    v = _bits16(v_new)
    bt = np.ascontiguousarray(np.asarray(block_table, np.int32))
    sp = np.ascontiguousarray(np.asarray(start_pos, np.int32))
    cu = np.ascontiguousarray(np.asarray(cu_tokens, np.int32))
    rc = _load().oaken_ref_quantize_kv(_ptr(pool), num_blocks, P, H, d, lay["stride"], _ptr(thr),
                                       _ptr(k), _ptr(v), _ptr(bt), bt.shape[1], _ptr(sp), _ptr(cu),
                                       sp.size)
    if rc != 0:
        raise ValueError("oracle quantize_kv: invalid block table or position")


def record(pool: np.ndarray, P, H, d, blk, h, which) -> np.ndarray:
    st = layout(P, d)["stride"]
    off = ((blk * H + h) * 2 + which) * st
    return pool[off: off + st]


def dequantize_slot(pool, P, H, d, thresholds, blk, h, which, slot, return_groups=False):
    rec = np.ascontiguousarray(record(pool, P, H, d, blk, h, which))
    thr = np.ascontiguousarray(np.asarray(thresholds, np.float32)[h, which])
    out = np.zeros(d, np.float64)
    grp = np.zeros(d, np.uint8)
    _load().oaken_ref_dequantize_slot(_ptr(rec), which, P, d, slot, _ptr(thr), _ptr(out), _ptr(grp))
    return (out, grp) if return_groups else out


def decode_attention(pool, num_blocks, P, H, d, thresholds, q, block_table, seq_lens, scale, window=0):
    """fp64 softmax(q K^T scale) V over the dequantized cache; returns fp32 [n_seqs, Hq, d].

    window > 0 restricts sequence s to its last `window` keys (sliding-window attention)."""
    lay = layout(P, d)
    thr = np.ascontiguousarray(np.asarray(thresholds, np.float32))
    qb = _bits16(q)
    n_seqs, Hq = qb.shape[0], qb.shape[1]
    bt = np.ascontiguousarray(np.asarray(block_table, np.int32))
    sl = np.ascontiguousarray(np.asarray(seq_lens, np.int32))
    out = np.zeros((n_seqs, Hq, d), np.float32)
    rc = _load().oaken_ref_decode_attention(_ptr(pool), num_blocks, P, H, d, lay["stride"],
                                            _ptr(thr), _ptr(qb), Hq, _ptr(bt), bt.shape[1],
                                            _ptr(sl), n_seqs, int(window), float(scale), _ptr(out))
    if rc != 0:
        raise ValueError("oracle decode_attention: invalid arguments")
    return out


def calibrate(k_calib, v_calib, outer_ratio=0.04, inner_ratio=0.06):
    """Offline thresholds [H][2][4] = (lo_o, lo_i, hi_i, hi_o) from fp16 [R][T][H][d] sets."""
    k = _bits16(k_calib)
    v = _bits16(v_calib)
    assert k.shape == v.shape and k.ndim == 4
    R, T, H, d = k.shape
    out = np.zeros((H, 2, 4), np.float32)
    rc = _load().oaken_ref_calibrate(_ptr(k), _ptr(v), R, T, H, d, float(outer_ratio),
                                     float(inner_ratio), _ptr(out))
    if rc != 0:
        raise ValueError("oracle calibrate: invalid ratios or shapes")
    return out


# --------------------------------------------------------------------------- #
# Group-count variants (Sec. 6.2, number-of-groups study).
VARIANTS = {"g3": 0, "g2": 1, "g4": 2, "g5": 3, "g4-o4": 4, "g5-o4": 5}


def variant_info(variant: int) -> dict:
    """Outer levels, inner levels, outlier magnitude bits, COO bits and bytes, groups."""
    out = np.zeros(6, np.int32)
    if _load().oaken_ref_variant_info(int(variant), _ptr(out)) != 0:
        raise ValueError("unknown variant")
    return dict(n_out=int(out[0]), n_in=int(out[1]), out_bits=int(out[2]), coo_bits=int(out[3]),
                coo_bytes=int(out[4]), groups=int(out[5]))


def variant_thresholds(variant: int, thr_a, thr_b=None) -> np.ndarray:
    """The eight boundaries [..][8] = lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob from
    calibrations at the variant's full shares (thr_a) and at its innermost/outermost level
    shares (thr_b), each [..][4] = lo_o, lo_i, hi_i, hi_o.  Unused boundaries repeat a used one."""
    info = variant_info(variant)
    a = np.asarray(thr_a, np.float32)
    b = a if thr_b is None else np.asarray(thr_b, np.float32)
    lo_oa, lo_ia, hi_ia, hi_oa = a[..., 0], a[..., 1], a[..., 2], a[..., 3]
    lo_ob, hi_ob = (b[..., 0], b[..., 3]) if info["n_out"] == 2 else (lo_oa, hi_oa)
    lo_ib, hi_ib = (b[..., 1], b[..., 2]) if info["n_in"] == 2 else (lo_ia, hi_ia)
    return np.ascontiguousarray(np.stack([lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob], -1))


def variant_quantize_vector(variant: int, x, thr8) -> dict:
    x = _bits16(x).reshape(-1)
    d = x.size
    info = variant_info(variant)
    thr8 = np.ascontiguousarray(np.asarray(thr8, np.float32).reshape(8))
    nib = np.zeros(d // 2, np.uint8)
    coo = np.zeros(d * info["coo_bytes"], np.uint8)
    counts = np.zeros(d // 64, np.uint8)
    meta = np.zeros(2 * info["groups"], np.uint16)
    n = ctypes.c_int(0)
    if _load().oaken_ref_variant_quantize_vector(int(variant), _ptr(x), d, _ptr(thr8), _ptr(nib), _ptr(coo),
                                                 _ptr(counts), _ptr(meta), ctypes.byref(n)) != 0:
        raise ValueError("oracle variant quantize: invalid arguments")
    return dict(nib=nib, coo=coo[: n.value * info["coo_bytes"]].copy(), counts=counts, meta=meta, n_coo=n.value)


def variant_dequantize_vector(variant: int, enc: dict, thr8) -> np.ndarray:
    info = variant_info(variant)
    nib = np.ascontiguousarray(enc["nib"], dtype=np.uint8)
    d = nib.size * 2
    coo = np.zeros(d * info["coo_bytes"], np.uint8)
    coo[: enc["coo"].size] = enc["coo"]
    counts = np.ascontiguousarray(enc["counts"], dtype=np.uint8)
    meta = np.ascontiguousarray(enc["meta"], dtype=np.uint16)
    thr8 = np.ascontiguousarray(np.asarray(thr8, np.float32).reshape(8))
    out = np.zeros(d, np.float64)
    if _load().oaken_ref_variant_dequantize_vector(int(variant), _ptr(nib), _ptr(coo), _ptr(counts), _ptr(meta), d,
                                                   _ptr(thr8), _ptr(out)) != 0:
        raise ValueError("oracle variant dequantize: invalid encoding")
    return out


def variant_quantize(variant: int, x, thr8) -> dict:
    """Batch encode fp16 [n][H][d] with per-head boundaries thr8 [H][8]."""
    x = _bits16(x)
    n, H, d = x.shape
    info = variant_info(variant)
    thr8 = np.ascontiguousarray(np.asarray(thr8, np.float32).reshape(H, 8))
    out = dict(nib=np.zeros((n, H, d // 2), np.uint8), coo=np.zeros((n, H, d * info["coo_bytes"]), np.uint8),
               counts=np.zeros((n, H, d // 64), np.uint8), meta=np.zeros((n, H, 2 * info["groups"]), np.uint16),
               n_coo=np.zeros((n, H), np.int32))
    if _load().oaken_ref_variant_quantize(int(variant), _ptr(x), n, H, d, _ptr(thr8), _ptr(out["nib"]),
                                          _ptr(out["coo"]), _ptr(out["counts"]), _ptr(out["meta"]),
                                          _ptr(out["n_coo"])) != 0:
        raise ValueError("oracle variant quantize: invalid arguments")
    return out


def variant_dequantize(variant: int, enc: dict, thr8) -> np.ndarray:
    """fp64 [n][H][d] from a batch encoding."""
    n, H, half = enc["nib"].shape
    d = 2 * half
    thr8 = np.ascontiguousarray(np.asarray(thr8, np.float32).reshape(H, 8))
    out = np.zeros((n, H, d), np.float64)
    a = {k: np.ascontiguousarray(enc[k]) for k in ("nib", "coo", "counts", "meta")}
    if _load().oaken_ref_variant_dequantize(int(variant), _ptr(a["nib"]), _ptr(a["coo"]), _ptr(a["counts"]),
                                            _ptr(a["meta"]), n, H, d, _ptr(thr8), _ptr(out)) != 0:
        raise ValueError("oracle variant dequantize: invalid encoding")
    return out
