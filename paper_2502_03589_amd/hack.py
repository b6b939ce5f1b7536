"""Python binding of libhack.so (ctypes).

Argument marshalling only: every step of the method runs in the HIP kernels
behind the C ABI declared in include/hack.h.  PyTorch supplies device memory
and the stream.  There is no fallback: if the library is missing, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

# the in-tree build only (paper_2502_03589_amd.build writes it here)
_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhack.so")
_lib = None

HACK_OK = 0
ROUND_NEAREST_EVEN = 0
ROUND_STOCHASTIC = 1
TAIL_FP16 = 0
TAIL_REQUANT = 1
TAIL_DEQUANT = 2
K_CODES, K_META, K_SUMS, V_CODES, V_META, V_SUMS, V_TAIL = range(7)
SECTIONS = ("k_codes", "k_meta", "k_sums", "v_codes", "v_meta", "v_sums", "v_tail")


class HackError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {hack_status_string(status)} (status {status})")
        self.status = status


class hack_kv_layout(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("kv_bits", ctypes.c_int32), ("partition", ctypes.c_int32),
                ("page_tokens", ctypes.c_int32), ("qp_bits", ctypes.c_int32),
                ("rounding", ctypes.c_int32), ("sum_bytes", ctypes.c_int32),
                ("seed", ctypes.c_uint64)]


class hack_kv_cache(ctypes.Structure):
    _fields_ = [("k_codes", ctypes.c_void_p), ("k_meta", ctypes.c_void_p), ("k_sums", ctypes.c_void_p),
                ("v_codes", ctypes.c_void_p), ("v_meta", ctypes.c_void_p), ("v_sums", ctypes.c_void_p),
                ("v_tail", ctypes.c_void_p), ("block_table_dev", ctypes.c_void_p),
                ("max_blocks_per_seq", ctypes.c_int32), ("reserved0", ctypes.c_int32),
                ("num_pages", ctypes.c_int64)]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_LAY = ctypes.POINTER(hack_kv_layout)
_CAC = ctypes.POINTER(hack_kv_cache)
_SIGS = {
    "hack_kv_layout_make": (_I32, [_LAY, _I32, _I32, _I32, _I32, _I32, _I32, _I32, ctypes.c_uint64]),
    "hack_kv_layout_set_sums": (_I32, [_LAY, _I32]),
    "hack_kv_bytes": (_I64, [_LAY, _I64, _I32]),
    "hack_quantize": (_I32, [_LAY, _CAC, _P, _P, _P, _I32, _I32, _P]),
    "hack_append": (_I32, [_LAY, _CAC, _P, _P, _P, _I32, _I32, _I32, _P]),
    "hack_decode_workspace_bytes": (_I64, [_LAY, _I32, _I32, _I32]),
    "hack_attend_decode": (_I32, [_LAY, _CAC, _P, _I32, _P, _I32, _I32, _I32, _P, _P, _I64, _P]),
    "hack_attend_decode_noalloc": (_I32, [_LAY, _CAC, _P, _I32, _P, _I32, _I32, _I32, _P, _P]),
    "hack_decode_step": (_I32, [_LAY, _CAC, _P, _P, _P, _I32, _P, _P, _I32, _I32, _I32, _P, _P, _I64, _P]),
    "hack_attend_prefill": (_I32, [_LAY, _CAC, _P, _I32, _I32, _I32, _I32, _P, _P]),
    "hack_project_qkv": (_I32, [_LAY, _CAC, _P, _P, _I32, _I32, _I32, _I32, _P, _P]),
    "hack_prefill_from_embeddings": (_I32, [_LAY, _CAC, _P, _P, _I32, _I32, _I32, _I32, _I32, _P, _P, _P]),
    "hack_status_string": (ctypes.c_char_p, [_I32]),
    "hack_debug_qk_products": (_I32, [_LAY, _CAC, _P, _I32, _P, _I32, _I32, _P, _P, _P, _P]),
    "hack_debug_pv_products": (_I32, [_LAY, _CAC, _P, _P, _I32, _P, _I32, _I32, _P, _P, _P]),
}
EXPORTS = tuple(_SIGS)


def library_path() -> str:
    return _LIB_PATH


def lib():
    """The loaded libhack.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with paper_2502_03589_amd.build.build()")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != HACK_OK:
        raise HackError(status, where)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev(t: torch.Tensor, dtype, name: str) -> int:
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA tensor")
    return t.data_ptr()


def hack_status_string(status: int) -> str:
    return lib().hack_status_string(status).decode()


def hack_kv_layout_make(head_dim: int, num_kv_heads: int, kv_bits: int, partition: int,
                        page_tokens: int, qp_bits: int = 8, rounding: int = ROUND_NEAREST_EVEN,
                        seed: int = 0, sums_cached: bool = True) -> hack_kv_layout:
    """A validated layout; sums_cached=False turns summation elimination off
    (hack_kv_layout_set_sums): no code sums are stored and decode rebuilds them."""
    out = hack_kv_layout()
    _check(lib().hack_kv_layout_make(ctypes.byref(out), head_dim, num_kv_heads, kv_bits, partition,
                                     page_tokens, qp_bits, rounding, seed), "hack_kv_layout_make")
    if not sums_cached:
        hack_kv_layout_set_sums(out, False)
    return out


def hack_kv_layout_set_sums(layout: hack_kv_layout, cached: bool) -> None:
    _check(lib().hack_kv_layout_set_sums(ctypes.byref(layout), 1 if cached else 0), "hack_kv_layout_set_sums")


def hack_kv_bytes(layout: hack_kv_layout, count: int, section: int) -> int:
    return int(lib().hack_kv_bytes(ctypes.byref(layout), count, section))


class KVCache:
    """Device buffers of one quantized cache (torch uint8 tensors) and the C struct
    pointing at them.  block_table: int32 [batch][max_blocks] CUDA tensor or None."""

    def __init__(self, layout: hack_kv_layout, num_pages: int, num_seqs: int,
                 block_table: Optional[torch.Tensor] = None, device="cuda", fill: int = 0):
        self.layout = layout
        self.num_pages = num_pages
        self.num_seqs = num_seqs
        self.buffers = {}
        for i, name in enumerate(SECTIONS):
            count = num_seqs if i == V_TAIL else num_pages
            n = hack_kv_bytes(layout, count, i)
            self.buffers[name] = torch.full((max(n, 1),), fill, dtype=torch.uint8, device=device)
        self.block_table = block_table
        c = hack_kv_cache()
        for name in SECTIONS:
            setattr(c, name, self.buffers[name].data_ptr())
        if block_table is not None:
            c.block_table_dev = _dev(block_table, torch.int32, "block_table")
            c.max_blocks_per_seq = block_table.shape[1]
        c.num_pages = num_pages
        self.struct = c

    @property
    def capacity(self) -> int:
        mb = self.block_table.shape[1] if self.block_table is not None else 1
        return mb * self.layout.page_tokens

    def nbytes(self) -> int:
        return sum(b.numel() for b in self.buffers.values())

    def sequences(self, first: int, count: int) -> "CacheSlice":
        """A view of sequences [first, first + count) of this cache, for calls that
        take a smaller batch (e.g. quantizing one long sequence at a time)."""
        return CacheSlice(self, first, count)


class CacheSlice:
    """Sequences [first, first + count) of a KVCache: the same buffers, with the
    per-sequence pointers (block-table rows, open-block rows, and for a contiguous
    cache the pages themselves) advanced to `first`."""

    def __init__(self, cache: KVCache, first: int, count: int):
        if first < 0 or count < 0 or first + count > cache.num_seqs:
            raise ValueError("sequence range outside the cache")
        lay, src = cache.layout, cache.struct
        c = hack_kv_cache()
        for name, _ in hack_kv_cache._fields_:
            setattr(c, name, getattr(src, name))
        if cache.block_table is None:
            for i, name in enumerate(SECTIONS):
                if i != V_TAIL:
                    setattr(c, name, getattr(src, name) + first * hack_kv_bytes(lay, 1, i))
            c.num_pages = count
        else:
            c.block_table_dev = src.block_table_dev + first * src.max_blocks_per_seq * 4
        c.v_tail = src.v_tail + first * hack_kv_bytes(lay, 1, V_TAIL)
        self.layout, self.struct, self.parent = lay, c, cache


def hack_quantize(layout, cache: KVCache, k: torch.Tensor, v: torch.Tensor, seq_lens: torch.Tensor,
                  max_len: Optional[int] = None, stream=None):
    batch = k.shape[0]
    max_len = k.shape[2] if max_len is None else max_len
    _check(lib().hack_quantize(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(k, torch.float16, "k"),
                               _dev(v, torch.float16, "v"), _dev(seq_lens, torch.int32, "seq_lens"),
                               batch, max_len, _stream(stream)), "hack_quantize")


def hack_append(layout, cache: KVCache, k_new: torch.Tensor, v_new: torch.Tensor, seq_lens: torch.Tensor,
                max_len: int, tail_mode: int = TAIL_FP16, stream=None):
    _check(lib().hack_append(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(k_new, torch.float16, "k_new"),
                             _dev(v_new, torch.float16, "v_new"), _dev(seq_lens, torch.int32, "seq_lens"),
                             k_new.shape[0], max_len, tail_mode, _stream(stream)), "hack_append")


def hack_decode_workspace_bytes(layout, batch: int, num_q_heads: int, max_len: int) -> int:
    return int(lib().hack_decode_workspace_bytes(ctypes.byref(layout), batch, num_q_heads, max_len))


def decode_workspace(layout, batch: int, num_q_heads: int, max_len: int, device="cuda") -> torch.Tensor:
    """Zero-filled workspace of the size hack_attend_decode needs."""
    n = hack_decode_workspace_bytes(layout, batch, num_q_heads, max_len)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def hack_attend_decode(layout, cache: KVCache, q: torch.Tensor, seq_lens: torch.Tensor, max_len: int,
                       tail_mode: int = TAIL_FP16, out: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    batch, hq, d = q.shape
    if out is None:
        out = torch.empty((batch, hq, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = decode_workspace(layout, batch, hq, max_len, q.device)
    _check(lib().hack_attend_decode(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(q, torch.float16, "q"),
                                    hq, _dev(seq_lens, torch.int32, "seq_lens"), batch, max_len, tail_mode,
                                    _dev(out, torch.float32, "out"), _dev(workspace, torch.uint8, "workspace"),
                                    workspace.numel(), _stream(stream)), "hack_attend_decode")
    return out


def hack_attend_decode_noalloc(layout, cache: KVCache, q: torch.Tensor, seq_lens: torch.Tensor, max_len: int,
                               tail_mode: int = TAIL_FP16, out: Optional[torch.Tensor] = None,
                               stream=None) -> torch.Tensor:
    """hack_attend_decode with the library's own static split-K scratch (no workspace)."""
    batch, hq, d = q.shape
    if out is None:
        out = torch.empty((batch, hq, d), dtype=torch.float32, device=q.device)
    _check(lib().hack_attend_decode_noalloc(ctypes.byref(layout), ctypes.byref(cache.struct),
                                            _dev(q, torch.float16, "q"), hq, _dev(seq_lens, torch.int32, "seq_lens"),
                                            batch, max_len, tail_mode, _dev(out, torch.float32, "out"),
                                            _stream(stream)), "hack_attend_decode_noalloc")
    return out


def hack_decode_step(layout, cache: KVCache, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor,
                     lens_in: torch.Tensor, lens_out: torch.Tensor, max_len: int, tail_mode: int = TAIL_FP16,
                     out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """Append one token per (sequence, kv head) and decode-attend over the longer
    cache in one launch; lens_out = lens_in + 1.  `max_len` bounds lens_in."""
    batch, hq, d = q.shape
    if out is None:
        out = torch.empty((batch, hq, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = decode_workspace(layout, batch, hq, max_len + 1, q.device)
    _check(lib().hack_decode_step(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(k_new, torch.float16, "k_new"),
                                  _dev(v_new, torch.float16, "v_new"), _dev(q, torch.float16, "q"), hq,
                                  _dev(lens_in, torch.int32, "lens_in"), _dev(lens_out, torch.int32, "lens_out"),
                                  batch, max_len, tail_mode, _dev(out, torch.float32, "out"),
                                  _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream)),
           "hack_decode_step")
    return out


def hack_attend_prefill(layout, cache: KVCache, q: torch.Tensor, causal: bool = True,
                        out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    batch, hq, length, d = q.shape
    if out is None:
        out = torch.empty((batch, hq, length, d), dtype=torch.float32, device=q.device)
    _check(lib().hack_attend_prefill(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(q, torch.float16, "q"),
                                     hq, batch, length, int(bool(causal)), _dev(out, torch.float32, "out"),
                                     _stream(stream)), "hack_attend_prefill")
    return out


def hack_project_qkv(layout, cache: KVCache, e: torch.Tensor, w: torch.Tensor, num_q_heads: int,
                     q_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """QKV generation fused with quantize-on-write: e fp16 [B][L][hidden], w fp16
    [(H_q + 2 H_kv) * 128][hidden].  Returns the fp16 query heads [B][H_q][L][128];
    the key and value heads go quantized into `cache`."""
    batch, length, hidden = e.shape
    if q_out is None:
        q_out = torch.empty((batch, num_q_heads, length, 128), dtype=torch.float16, device=e.device)
    _check(lib().hack_project_qkv(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(e, torch.float16, "e"),
                                  _dev(w, torch.float16, "w"), num_q_heads, hidden, batch, length,
                                  _dev(q_out, torch.float16, "q_out"), _stream(stream)), "hack_project_qkv")
    return q_out


def hack_prefill_from_embeddings(layout, cache: KVCache, e: torch.Tensor, w: torch.Tensor, num_q_heads: int,
                                 causal: bool = True, q_out: Optional[torch.Tensor] = None,
                                 out: Optional[torch.Tensor] = None, stream=None):
    """Projection + quantize-on-write + prefill attention; returns (out fp32, q fp16)."""
    batch, length, hidden = e.shape
    if q_out is None:
        q_out = torch.empty((batch, num_q_heads, length, 128), dtype=torch.float16, device=e.device)
    if out is None:
        out = torch.empty((batch, num_q_heads, length, 128), dtype=torch.float32, device=e.device)
    _check(lib().hack_prefill_from_embeddings(ctypes.byref(layout), ctypes.byref(cache.struct),
                                              _dev(e, torch.float16, "e"), _dev(w, torch.float16, "w"), num_q_heads,
                                              hidden, batch, length, int(bool(causal)),
                                              _dev(q_out, torch.float16, "q_out"), _dev(out, torch.float32, "out"),
                                              _stream(stream)), "hack_prefill_from_embeddings")
    return out, q_out


def hack_debug_qk_products(layout, cache: KVCache, q: torch.Tensor, seq_lens: torch.Tensor, max_len: int,
                           stream=None):
    batch, hq, d = q.shape
    P = d // layout.partition
    qc = torch.zeros((batch, hq, d), dtype=torch.uint8, device=q.device)
    qm = torch.zeros((batch, hq, P, 2), dtype=torch.float32, device=q.device)
    prod = torch.zeros((batch, hq, max(max_len, 1), P), dtype=torch.int32, device=q.device)
    _check(lib().hack_debug_qk_products(ctypes.byref(layout), ctypes.byref(cache.struct), _dev(q, torch.float16, "q"),
                                        hq, _dev(seq_lens, torch.int32, "seq_lens"), batch, max_len,
                                        qc.data_ptr(), qm.data_ptr(), prod.data_ptr(), _stream(stream)),
           "hack_debug_qk_products")
    return qc, qm, prod


def hack_debug_pv_products(layout, cache: KVCache, p_codes: torch.Tensor, p_meta: torch.Tensor,
                           seq_lens: torch.Tensor, max_len: int, stream=None):
    batch, hq, nb, pi = p_codes.shape
    d = layout.head_dim
    prod = torch.zeros((batch, hq, max(nb, 1), d), dtype=torch.int32, device=p_codes.device)
    out = torch.zeros((batch, hq, d), dtype=torch.float32, device=p_codes.device)
    _check(lib().hack_debug_pv_products(ctypes.byref(layout), ctypes.byref(cache.struct),
                                        _dev(p_codes, torch.uint8, "p_codes"), _dev(p_meta, torch.float32, "p_meta"),
                                        hq, _dev(seq_lens, torch.int32, "seq_lens"), batch, max_len,
                                        prod.data_ptr(), out.data_ptr(), _stream(stream)), "hack_debug_pv_products")
    return prod, out


class BoundCall:
    """A library call with its arguments marshalled once (for tight loops): calling
    it passes the prepared ctypes arguments and the current stream."""

    def __init__(self, fn_name: str, where: str, *args):
        self._fn = getattr(lib(), fn_name)
        self._args = args
        self._where = where

    def __call__(self, stream=None):
        _check(self._fn(*self._args, _stream(stream)), self._where)


def bind_append(layout, cache: KVCache, k_new, v_new, seq_lens, max_len: int, tail_mode: int = TAIL_FP16):
    return BoundCall("hack_append", "hack_append", ctypes.byref(layout), ctypes.byref(cache.struct),
                     _dev(k_new, torch.float16, "k_new"), _dev(v_new, torch.float16, "v_new"),
                     _dev(seq_lens, torch.int32, "seq_lens"), k_new.shape[0], max_len, tail_mode)


def bind_attend_decode(layout, cache: KVCache, q, seq_lens, max_len: int, tail_mode: int, out, workspace):
    batch, hq, _ = q.shape
    return BoundCall("hack_attend_decode", "hack_attend_decode", ctypes.byref(layout), ctypes.byref(cache.struct),
                     _dev(q, torch.float16, "q"), hq, _dev(seq_lens, torch.int32, "seq_lens"), batch, max_len,
                     tail_mode, _dev(out, torch.float32, "out"), _dev(workspace, torch.uint8, "workspace"),
                     workspace.numel())


def bind_decode_step(layout, cache: KVCache, k_new, v_new, q, lens_in, lens_out, max_len: int, tail_mode: int,
                     out, workspace):
    """Pre-marshalled hack_decode_step (see bind_append)."""
    batch, hq, _ = q.shape
    return BoundCall("hack_decode_step", "hack_decode_step", ctypes.byref(layout), ctypes.byref(cache.struct),
                     _dev(k_new, torch.float16, "k_new"), _dev(v_new, torch.float16, "v_new"),
                     _dev(q, torch.float16, "q"), hq, _dev(lens_in, torch.int32, "lens_in"),
                     _dev(lens_out, torch.int32, "lens_out"), batch, max_len, tail_mode,
                     _dev(out, torch.float32, "out"), _dev(workspace, torch.uint8, "workspace"), workspace.numel())
