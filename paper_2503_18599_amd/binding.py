"""ctypes binding of liboaken.so (include/oaken.h) for torch tensors.

Argument marshalling only: tensors are checked for device, dtype and contiguity and
passed by data pointer together with torch's current HIP stream.  Every step of the
computation runs in the library's HIP kernels; there is no fallback path, and a
missing library raises at first use.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboaken.so")
PAGE = 16

_lib = None


class OakenError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"oaken status {status}: {detail}")
        self.status = status


class _CacheStruct(ctypes.Structure):
    _fields_ = [
        ("num_blocks", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("record_stride", ctypes.c_int64),
        ("pool", ctypes.c_void_p),
        ("thresholds", ctypes.c_void_p),
        ("sparse_pool", ctypes.c_void_p),
        ("sparse_free", ctypes.c_void_p),
        ("sparse_pages", ctypes.c_int32),
    ]


def lib():
    """Load liboaken.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    L.oaken_record_bytes.argtypes = [i32, i32]
    L.oaken_record_bytes.restype = i64
    L.oaken_record_bytes_paged.argtypes = [i32, i32]
    L.oaken_record_bytes_paged.restype = i64
    L.oaken_sparse_free_list_bytes.argtypes = [i32]
    L.oaken_sparse_free_list_bytes.restype = sz
    L.oaken_sparse_reset.argtypes = [ctypes.POINTER(_CacheStruct), P]
    L.oaken_sparse_reset.restype = ctypes.c_int
    L.oaken_sparse_release.argtypes = [ctypes.POINTER(_CacheStruct), P, i32, P]
    L.oaken_sparse_release.restype = ctypes.c_int
    L.oaken_sparse_status.argtypes = [ctypes.POINTER(_CacheStruct), ctypes.POINTER(i32), ctypes.POINTER(i32), P]
    L.oaken_sparse_status.restype = ctypes.c_int
    L.oaken_prefill_attention_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    L.oaken_prefill_attention_workspace_bytes.restype = sz
    L.oaken_prefill_attention.argtypes = [ctypes.POINTER(_CacheStruct), P, i32, P, i32, P, P, i32, i32, i32, i32,
                                          f32, P, P, sz, P]
    L.oaken_prefill_attention.restype = ctypes.c_int
    L.oaken_record_layout.argtypes = [i32, i32, P]
    L.oaken_record_layout.restype = ctypes.c_int
    L.oaken_calibrate_workspace_bytes.argtypes = [i32, i32]
    L.oaken_calibrate_workspace_bytes.restype = sz
    L.oaken_attention_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    L.oaken_attention_workspace_bytes.restype = sz
    L.oaken_calibrate_thresholds.argtypes = [P, P, i32, i32, i32, i32, f32, f32, P, P, sz, P]
    L.oaken_calibrate_thresholds.restype = ctypes.c_int
    L.oaken_quantize_kv.argtypes = [ctypes.POINTER(_CacheStruct), P, P, P, i32, P, P, i32, i32, i32, P]
    L.oaken_quantize_kv.restype = ctypes.c_int
    L.oaken_decode_attention.argtypes = [ctypes.POINTER(_CacheStruct), P, i32, P, i32, P, i32, i32,
                                         f32, P, P, sz, P]
    L.oaken_decode_attention.restype = ctypes.c_int
    L.oaken_attention_workspace_bytes_window.argtypes = [i32, i32, i32, i32, i32, i32]
    L.oaken_attention_workspace_bytes_window.restype = sz
    L.oaken_decode_attention_window.argtypes = [ctypes.POINTER(_CacheStruct), P, i32, P, i32, P, i32, i32,
                                                i32, f32, P, P, sz, P]
    L.oaken_decode_attention_window.restype = ctypes.c_int
    L.oaken_variant_info.argtypes = [i32, P]
    L.oaken_variant_info.restype = ctypes.c_int
    L.oaken_variant_quantize.argtypes = [i32, P, i32, i32, i32, P, P, P, P, P, P, P]
    L.oaken_variant_quantize.restype = ctypes.c_int
    L.oaken_variant_dequantize.argtypes = [i32, P, P, P, P, i32, i32, i32, P, P, P]
    L.oaken_variant_dequantize.restype = ctypes.c_int
    L.oaken_decode_attention_noalloc.argtypes = [ctypes.POINTER(_CacheStruct), P, i32, P, i32, P, i32, i32, i32,
                                                 f32, P, P]
    L.oaken_decode_attention_noalloc.restype = ctypes.c_int
    L.oaken_probe_read.argtypes = [P, i64, i64, i64, P, P]
    L.oaken_probe_read.restype = ctypes.c_int
    L.oaken_status_string.argtypes = [ctypes.c_int]
    L.oaken_status_string.restype = ctypes.c_char_p
    L.oaken_last_error.argtypes = []
    L.oaken_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise OakenError(status, lib().oaken_last_error().decode())


def _dev(t: torch.Tensor, dtype, name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def record_bytes(head_dim: int, block_size: int = PAGE) -> int:
    return int(lib().oaken_record_bytes(block_size, head_dim))


def record_bytes_paged(head_dim: int, block_size: int = PAGE) -> int:
    return int(lib().oaken_record_bytes_paged(block_size, head_dim))


SPARSE_PAGE_BYTES = 256


def record_layout(head_dim: int, block_size: int = PAGE) -> dict:
    out = (ctypes.c_int64 * 5)()
    _check(lib().oaken_record_layout(block_size, head_dim, out))
    return dict(counts=out[0], meta=out[1], dense=out[2], sparse=out[3], stride=out[4])


class Cache:
    """One layer's quantized KV cache: a uint8 page pool plus fp32 thresholds [H][2][4].

    sparse_pages > 0 keeps the COO bytes in a separate pool of that many 256-byte sparse
    pages, taken on demand (the records then hold a sparse page table instead of their
    worst-case COO capacity)."""

    def __init__(self, num_blocks: int, n_kv_heads: int, head_dim: int, thresholds: torch.Tensor,
                 pool: torch.Tensor | None = None, sparse_pages: int = 0):
        self.sparse_pages = int(sparse_pages)
        stride = record_bytes_paged(head_dim) if self.sparse_pages > 0 else record_bytes(head_dim)
        if stride < 0:
            raise OakenError(2, f"head_dim {head_dim} unsupported")
        nbytes = num_blocks * n_kv_heads * 2 * stride
        if pool is None:
            pool = torch.zeros(nbytes, dtype=torch.uint8, device=thresholds.device)
        if pool.numel() < nbytes:
            raise ValueError("pool too small")
        if tuple(thresholds.shape) != (n_kv_heads, 2, 4):
            raise ValueError("thresholds must be [n_kv_heads][2][4]")
        self.pool = pool
        self.thresholds = thresholds.contiguous()
        self.num_blocks, self.n_kv_heads, self.head_dim, self.stride = num_blocks, n_kv_heads, head_dim, stride
        self.sparse_pool = self.sparse_free = None
        sp = sf = None
        if self.sparse_pages > 0:
            dev = thresholds.device
            self.sparse_pool = torch.zeros(self.sparse_pages * SPARSE_PAGE_BYTES, dtype=torch.uint8, device=dev)
            nfree = int(lib().oaken_sparse_free_list_bytes(self.sparse_pages)) // 4
            self.sparse_free = torch.zeros(nfree, dtype=torch.int32, device=dev)
            sp = _dev(self.sparse_pool, torch.uint8, "sparse_pool")
            sf = _dev(self.sparse_free, torch.int32, "sparse_free")
        self._s = _CacheStruct(num_blocks, PAGE, n_kv_heads, head_dim, stride,
                               _dev(self.pool, torch.uint8, "pool"),
                               _dev(self.thresholds, torch.float32, "thresholds"), sp, sf, self.sparse_pages)
        if self.sparse_pages > 0:
            self.sparse_reset()

    def sparse_reset(self):
        """Every sparse page free, every record empty."""
        _check(lib().oaken_sparse_reset(self.struct, _stream()))

    def release(self, block_ids: torch.Tensor):
        """Retire blocks: their records give their sparse pages back and become empty."""
        _check(lib().oaken_sparse_release(self.struct, _dev(block_ids, torch.int32, "block_ids"),
                                          block_ids.numel(), _stream()))

    def sparse_status(self) -> tuple[int, bool]:
        """(free sparse pages, overflow flag); synchronizes the current stream."""
        fp, ov = ctypes.c_int32(0), ctypes.c_int32(0)
        _check(lib().oaken_sparse_status(self.struct, ctypes.byref(fp), ctypes.byref(ov), _stream()))
        return int(fp.value), bool(ov.value)

    @property
    def struct(self):
        return ctypes.byref(self._s)


def calibrate_thresholds(k_calib: torch.Tensor, v_calib: torch.Tensor, outer_ratio: float = 0.04,
                         inner_ratio: float = 0.06) -> torch.Tensor:
    """fp16 [R][T][H][d] calibration sets -> fp32 thresholds [H][2][4] (device)."""
    if k_calib.shape != v_calib.shape or k_calib.dim() != 4:
        raise ValueError("calibration sets must both be [R][T][H][d]")
    R, T, H, d = k_calib.shape
    out = torch.empty(H, 2, 4, dtype=torch.float32, device=k_calib.device)
    ws_bytes = int(lib().oaken_calibrate_workspace_bytes(R, H))
    ws = torch.empty(max(ws_bytes, 4), dtype=torch.uint8, device=k_calib.device)
    _check(lib().oaken_calibrate_thresholds(
        _dev(k_calib, torch.float16, "k_calib"), _dev(v_calib, torch.float16, "v_calib"),
        R, T, H, d, float(outer_ratio), float(inner_ratio), out.data_ptr(), ws.data_ptr(), ws_bytes,
        _stream()))
    return out


def quantize_kv(cache: Cache, k_new: torch.Tensor, v_new: torch.Tensor, block_table: torch.Tensor,
                start_pos: torch.Tensor, cu_tokens: torch.Tensor, max_new_per_seq: int):
    """Quantize fp16 rows [n_tokens][H][d] into the cache at positions start_pos[s] + i."""
    n_tokens = k_new.shape[0]
    if tuple(k_new.shape) != (n_tokens, cache.n_kv_heads, cache.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [n_tokens][n_kv_heads][head_dim]")
    n_seqs = start_pos.numel()
    if cu_tokens.numel() != n_seqs + 1 or block_table.dim() != 2 or block_table.shape[0] != n_seqs:
        raise ValueError("cu_tokens must have n_seqs+1 entries and block_table n_seqs rows")
    _check(lib().oaken_quantize_kv(
        cache.struct, _dev(k_new, torch.float16, "k_new"), _dev(v_new, torch.float16, "v_new"),
        _dev(block_table, torch.int32, "block_table"), block_table.shape[1],
        _dev(start_pos, torch.int32, "start_pos"), _dev(cu_tokens, torch.int32, "cu_tokens"),
        n_seqs, n_tokens, int(max_new_per_seq), _stream()))


def attention_workspace_bytes(n_seqs, n_q_heads, n_kv_heads, head_dim, max_seq_len, window: int = 0) -> int:
    if window:
        return int(lib().oaken_attention_workspace_bytes_window(n_seqs, n_q_heads, n_kv_heads, head_dim,
                                                                max_seq_len, int(window)))
    return int(lib().oaken_attention_workspace_bytes(n_seqs, n_q_heads, n_kv_heads, head_dim, max_seq_len))


def decode_attention(cache: Cache, q: torch.Tensor, block_table: torch.Tensor, seq_lens: torch.Tensor,
                     max_seq_len: int, scale: float, out: torch.Tensor | None = None,
                     workspace: torch.Tensor | None = None, window: int = 0) -> torch.Tensor:
    """fp16 q [n_seqs][Hq][d] -> fp32 out [n_seqs][Hq][d].  window > 0: sliding-window
    attention over each sequence's last `window` keys."""
    n_seqs, Hq, d = q.shape
    if d != cache.head_dim or seq_lens.numel() != n_seqs or block_table.shape[0] != n_seqs:
        raise ValueError("q / seq_lens / block_table shapes disagree")
    if out is None:
        out = torch.empty(n_seqs, Hq, d, dtype=torch.float32, device=q.device)
    ws_bytes = attention_workspace_bytes(n_seqs, Hq, cache.n_kv_heads, d, max_seq_len, window)
    if ws_bytes and (workspace is None or workspace.numel() < ws_bytes):
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    ws_ptr = workspace.data_ptr() if (ws_bytes and workspace is not None) else None
    if window:
        _check(lib().oaken_decode_attention_window(
            cache.struct, _dev(q, torch.float16, "q"), Hq, _dev(block_table, torch.int32, "block_table"),
            block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), n_seqs, int(max_seq_len),
            int(window), float(scale), _dev(out, torch.float32, "out"), ws_ptr, ws_bytes, _stream()))
    else:
        _check(lib().oaken_decode_attention(
            cache.struct, _dev(q, torch.float16, "q"), Hq, _dev(block_table, torch.int32, "block_table"),
            block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), n_seqs, int(max_seq_len),
            float(scale), _dev(out, torch.float32, "out"), ws_ptr, ws_bytes, _stream()))
    return out


def decode_attention_noalloc(cache: Cache, q: torch.Tensor, block_table: torch.Tensor, seq_lens: torch.Tensor,
                             max_seq_len: int, scale: float, out: torch.Tensor, window: int = 0) -> torch.Tensor:
    """decode_attention with the split partials in the library's static scratch: the call
    allocates nothing (the caller passes `out`)."""
    n_seqs, Hq, d = q.shape
    if d != cache.head_dim or seq_lens.numel() != n_seqs or block_table.shape[0] != n_seqs:
        raise ValueError("q / seq_lens / block_table shapes disagree")
    if tuple(out.shape) != (n_seqs, Hq, d):
        raise ValueError("out must be [n_seqs][n_q_heads][head_dim]")
    _check(lib().oaken_decode_attention_noalloc(
        cache.struct, _dev(q, torch.float16, "q"), Hq, _dev(block_table, torch.int32, "block_table"),
        block_table.shape[1], _dev(seq_lens, torch.int32, "seq_lens"), n_seqs, int(max_seq_len), int(window),
        float(scale), _dev(out, torch.float32, "out"), _stream()))
    return out


def prefill_attention(cache: Cache, q: torch.Tensor, block_table: torch.Tensor, start_pos: torch.Tensor,
                      cu_tokens: torch.Tensor, max_seq_len: int, scale: float, window: int = 0,
                      out: torch.Tensor | None = None, workspace: torch.Tensor | None = None) -> torch.Tensor:
    """Chunked-prefill attention: fp16 q [n_tokens][Hq][d] of new tokens (already quantized
    into the cache) -> fp32 out [n_tokens][Hq][d]; each query attends causally over its
    sequence's keys up to its own position."""
    n_tokens, Hq, d = q.shape
    n_seqs = start_pos.numel()
    if d != cache.head_dim or cu_tokens.numel() != n_seqs + 1 or block_table.shape[0] != n_seqs:
        raise ValueError("q / start_pos / cu_tokens / block_table shapes disagree")
    if out is None:
        out = torch.empty(n_tokens, Hq, d, dtype=torch.float32, device=q.device)
    ws_bytes = int(lib().oaken_prefill_attention_workspace_bytes(n_tokens, Hq, cache.n_kv_heads, d,
                                                                 int(max_seq_len), int(window)))
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    _check(lib().oaken_prefill_attention(
        cache.struct, _dev(q, torch.float16, "q"), Hq, _dev(block_table, torch.int32, "block_table"),
        block_table.shape[1], _dev(start_pos, torch.int32, "start_pos"), _dev(cu_tokens, torch.int32, "cu_tokens"),
        n_seqs, n_tokens, int(max_seq_len), int(window), float(scale), _dev(out, torch.float32, "out"),
        workspace.data_ptr(), ws_bytes, _stream()))
    return out


def probe_read(buf: torch.Tensor, bytes_per_record: int, record_stride: int, n_records: int,
               checksum: torch.Tensor | None = None) -> torch.Tensor:
    """Streaming-read probe over a uint8 device buffer: XOR of every 32-bit word of the
    first bytes_per_record bytes of each record (int32 device scalar)."""
    if buf.dtype != torch.uint8 or buf.device.type != "cuda":
        raise TypeError("buf must be a uint8 GPU tensor")
    if (n_records - 1) * record_stride + bytes_per_record > buf.numel():
        raise ValueError("records extend past the buffer")
    if checksum is None:
        checksum = torch.zeros(1, dtype=torch.int32, device=buf.device)
    _check(lib().oaken_probe_read(buf.data_ptr(), int(bytes_per_record), int(record_stride), int(n_records),
                                  _dev(checksum, torch.int32, "checksum"), _stream()))
    return checksum


# --------------------------------------------------------------------------- #
# Group-count variants (Sec. 6.2, number-of-groups study)
VARIANTS = {"g3": 0, "g2": 1, "g4": 2, "g5": 3, "g4-o4": 4, "g5-o4": 5}


def variant_info(variant: int) -> dict:
    out = (ctypes.c_int32 * 6)()
    _check(lib().oaken_variant_info(int(variant), out))
    return dict(n_out=out[0], n_in=out[1], out_bits=out[2], coo_bits=out[3], coo_bytes=out[4], groups=out[5])


def variant_boundaries(variant: int, thr_full: torch.Tensor, thr_level: torch.Tensor | None = None) -> torch.Tensor:
    """[..][8] = lo_ob, lo_oa, lo_ia, lo_ib, hi_ib, hi_ia, hi_oa, hi_ob from thresholds [..][4]
    (lo_o, lo_i, hi_i, hi_o) calibrated at the variant's full outer/inner shares and, for the
    extra levels, at the outermost and innermost level shares."""
    info = variant_info(variant)
    a = thr_full
    b = thr_level if thr_level is not None else thr_full
    ob = (b[..., 0], b[..., 3]) if info["n_out"] == 2 else (a[..., 0], a[..., 3])
    ib = (b[..., 1], b[..., 2]) if info["n_in"] == 2 else (a[..., 1], a[..., 2])
    return torch.stack([ob[0], a[..., 0], a[..., 1], ib[0], ib[1], a[..., 2], a[..., 3], ob[1]], -1).contiguous()


def variant_quantize(variant: int, x: torch.Tensor, thr8: torch.Tensor) -> dict:
    """Encode fp16 [n][H][d] (d 64 or 128) with boundaries [H][8]; returns the buffers."""
    n, H, d = x.shape
    info = variant_info(variant)
    dev = x.device
    enc = dict(nib=torch.empty(n, H, d // 2, dtype=torch.uint8, device=dev),
               coo=torch.zeros(n, H, d * info["coo_bytes"], dtype=torch.uint8, device=dev),
               counts=torch.empty(n, H, d // 64, dtype=torch.uint8, device=dev),
               meta=torch.empty(n, H, 2 * info["groups"], dtype=torch.int16, device=dev),
               n_coo=torch.empty(n, H, dtype=torch.int32, device=dev))
    if tuple(thr8.shape) != (H, 8):
        raise ValueError("boundaries must be [n_kv_heads][8]")
    _check(lib().oaken_variant_quantize(
        int(variant), _dev(x, torch.float16, "x"), n, H, d, _dev(thr8, torch.float32, "thr8"),
        enc["nib"].data_ptr(), enc["coo"].data_ptr(), enc["counts"].data_ptr(), enc["meta"].data_ptr(),
        enc["n_coo"].data_ptr(), _stream()))
    return enc


def variant_dequantize(variant: int, enc: dict, thr8: torch.Tensor) -> torch.Tensor:
    n, H, half = enc["nib"].shape
    d = 2 * half
    out = torch.empty(n, H, d, dtype=torch.float32, device=enc["nib"].device)
    _check(lib().oaken_variant_dequantize(
        int(variant), _dev(enc["nib"], torch.uint8, "nib"), _dev(enc["coo"], torch.uint8, "coo"),
        _dev(enc["counts"], torch.uint8, "counts"), _dev(enc["meta"], torch.int16, "meta"), n, H, d,
        _dev(thr8, torch.float32, "thr8"), out.data_ptr(), _stream()))
    return out
