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
    lib.oaken_ref_max_threads.argtypes = []
    lib.oaken_ref_max_threads.restype = i32
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
