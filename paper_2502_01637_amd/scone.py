"""Python binding of libscone.so (argument marshalling only).

Every function here checks dtypes, devices and shapes, then passes raw
pointers and sizes to the C ABI declared in ``include/scone.h``; all of the
lookup and gather work runs in the library's HIP kernels.  PyTorch supplies
device memory and the current stream.  When the library is missing or cannot
be loaded, every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libscone.so")

OK, EINVAL, ELEN, EID, EDUP, EFULL, ENOMEM, EHIP, ETOKEN, EROW, ESCRATCH = range(11)
SPLIT_STATIC_BYTES = 32 << 20   # scone_gather_split_static's scratch (SCONE_SPLIT_STATIC_BYTES)
PLACE_HBM, PLACE_HOST = 0, 1
MAX_FGRAM_LEN = 7
TOKEN_LIMIT = 65536

_lib = None
_lock = threading.Lock()


class SconeError(RuntimeError):
    def __init__(self, code: int, what: str):
        msg = lib().scone_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{what}: {msg} (status {code})")
        self.code = code


def _declare(L):
    P, I64, I32, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
    L.scone_build_fgram_table.argtypes = [P, P, P, I64, I32, ctypes.c_double, P,
                                          ctypes.POINTER(P)]
    L.scone_build_fgram_table.restype = I
    L.scone_lookup.argtypes = [P, P, I64, I64, I32, P, P, P]
    L.scone_lookup.restype = I
    L.scone_lookup_counted.argtypes = [P, P, I64, I64, I32, P, P, P, P]
    L.scone_lookup_counted.restype = I
    L.scone_gather.argtypes = [P, I64, P, I64, I64, P, I32, P]
    L.scone_gather.restype = I
    L.scone_embed.argtypes = [P, P, I64, I64, I32, P, I64, I64, I32, P, P, P, P]
    L.scone_embed.restype = I
    L.scone_embed_pipelined.argtypes = [P, P, I64, I64, I32, P, P, P, I64, P, I64, I64, I32, P,
                                        P]
    L.scone_embed_pipelined.restype = I
    L.scone_decode_step.argtypes = [P, P, P, I32, P, I64, I32, P, I64, I64, I32, P, P, P, P]
    L.scone_decode_step.restype = I
    L.scone_discover_fgrams.argtypes = [P, I64, I64, I32, I32, I64, P, P, P,
                                        ctypes.POINTER(I64), P, I64, P]
    L.scone_discover_workspace.argtypes = [I64, I64, I32]
    L.scone_discover_workspace.restype = I64
    L.scone_discover_fgrams.restype = I
    L.scone_tag.argtypes = [P, P, I64, I64, I32, P, P, P]
    L.scone_tag.restype = I
    L.scone_gather_split.argtypes = [P, I64, P, I64, P, I64, I64, P, P, I64, P, P]
    L.scone_gather_split.restype = I
    L.scone_gather_split_workspace.argtypes = [I64, I64]
    L.scone_gather_split_workspace.restype = I64
    L.scone_gather_split_static.argtypes = [P, I64, P, I64, P, I64, I64, P, P, P]
    L.scone_gather_split_static.restype = I
    L.scone_fgram_model_forward.argtypes = [P, P, P, I64, I32, P, I64, P, I32, I32, I32, I32,
                                            P, I64, P]
    L.scone_fgram_model_forward.restype = I
    L.scone_fgram_model_layout.argtypes = [I32, I32, I32, I32, I32, ctypes.POINTER(I64),
                                           ctypes.POINTER(I64), ctypes.POINTER(I64)]
    L.scone_fgram_model_layout.restype = I
    L.scone_host_alloc.argtypes = [I64, ctypes.POINTER(P), ctypes.POINTER(P)]
    L.scone_host_alloc.restype = I
    L.scone_host_free.argtypes = [P]
    L.scone_host_free.restype = I
    L.scone_check.argtypes = [P]
    L.scone_check.restype = I
    L.scone_table_destroy.argtypes = [P]
    L.scone_table_destroy.restype = None
    L.scone_table_info.argtypes = [P, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                   ctypes.POINTER(I32), ctypes.POINTER(I32),
                                   ctypes.POINTER(I64)]
    L.scone_table_info.restype = I
    L.scone_strerror.argtypes = [I]
    L.scone_strerror.restype = ctypes.c_char_p
    return L


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(
                    f"{LIB_PATH} is missing: build it with paper_2502_01637_amd._build.build()")
            _lib = _declare(ctypes.CDLL(LIB_PATH))
        return _lib


def _check(rc: int, what: str):
    if rc != OK:
        raise SconeError(rc, what)


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_i32(t: torch.Tensor, name: str, ndim: Optional[int] = None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != torch.int32:
        raise TypeError(f"{name} must be int32, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")
    return t


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None or t.numel() == 0 else t.data_ptr()


class Table:
    """A built f-gram dictionary (owns the library's table handle)."""

    def __init__(self, handle: ctypes.c_void_p, device: torch.device):
        self._h = handle
        self.device = device
        n, cap, ent = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        ml, sb = ctypes.c_int32(), ctypes.c_int32()
        _check(lib().scone_table_info(handle, ctypes.byref(n), ctypes.byref(cap),
                                      ctypes.byref(ml), ctypes.byref(sb), ctypes.byref(ent)),
               "scone_table_info")
        self.n, self.capacity, self.entries = n.value, cap.value, ent.value
        self.max_len, self.slot_bytes = ml.value, sb.value

    @property
    def handle(self) -> ctypes.c_void_p:
        if self._h is None:
            raise ValueError("table already destroyed")
        return self._h

    @property
    def nbytes(self) -> int:
        return self.capacity * self.slot_bytes

    def close(self):
        if self._h is not None:
            lib().scone_table_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def build_fgram_table(fgrams: torch.Tensor, lengths: torch.Tensor, ids: torch.Tensor,
                      max_load: float = 0.25, stream=None) -> Table:
    """scone_build_fgram_table: fgrams [n, K] int32, lengths [n], ids [n] (device)."""
    _dev_i32(fgrams, "fgrams", 2)
    _dev_i32(lengths, "lengths", 1)
    _dev_i32(ids, "ids", 1)
    n, K = fgrams.shape
    if lengths.numel() != n or ids.numel() != n:
        raise ValueError("fgrams, lengths and ids disagree on n")
    h = ctypes.c_void_p()
    with torch.cuda.device(fgrams.device):
        rc = lib().scone_build_fgram_table(_ptr(fgrams), _ptr(lengths), _ptr(ids), n, K,
                                           float(max_load), _stream(stream), ctypes.byref(h))
    _check(rc, "scone_build_fgram_table")
    return Table(h, fgrams.device)


def lookup(table: Table, token_ids: torch.Tensor, max_n: int,
           fgram_ids: Optional[torch.Tensor] = None, match_len: Optional[torch.Tensor] = None,
           want_len: bool = False, stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """scone_lookup on token_ids [B, T]; returns (fgram_ids [B, T], match_len or None)."""
    _dev_i32(token_ids, "token_ids", 2)
    B, T = token_ids.shape
    if fgram_ids is None:
        fgram_ids = torch.empty((B, T), dtype=torch.int32, device=token_ids.device)
    _dev_i32(fgram_ids, "fgram_ids")
    if fgram_ids.numel() != B * T:
        raise ValueError("fgram_ids has the wrong size")
    if match_len is None and want_len:
        match_len = torch.empty((B, T), dtype=torch.int8, device=token_ids.device)
    if match_len is not None and (match_len.dtype != torch.int8 or match_len.numel() != B * T
                                  or not match_len.is_contiguous()):
        raise ValueError("match_len must be a contiguous int8 tensor of B*T elements")
    with torch.cuda.device(token_ids.device):
        rc = lib().scone_lookup(table.handle, _ptr(token_ids), B, T, int(max_n),
                                _ptr(fgram_ids), _ptr(match_len), _stream(stream))
    _check(rc, "scone_lookup")
    return fgram_ids, match_len


def lookup_counted(table: Table, token_ids: torch.Tensor, max_n: int,
                   stream=None) -> Tuple[torch.Tensor, torch.Tensor, int]:
    """scone_lookup_counted on token_ids [B, T]: (fgram_ids, match_len, keys
    probed).  Synchronises the stream to read the count."""
    _dev_i32(token_ids, "token_ids", 2)
    B, T = token_ids.shape
    fgram_ids = torch.empty((B, T), dtype=torch.int32, device=token_ids.device)
    match_len = torch.empty((B, T), dtype=torch.int8, device=token_ids.device)
    probes = torch.zeros(1, dtype=torch.int64, device=token_ids.device)
    with torch.cuda.device(token_ids.device):
        rc = lib().scone_lookup_counted(table.handle, _ptr(token_ids), B, T, int(max_n),
                                        _ptr(fgram_ids), _ptr(match_len), _ptr(probes),
                                        _stream(stream))
    _check(rc, "scone_lookup_counted")
    return fgram_ids, match_len, int(probes.item())


def tag(table: Table, token_ids: torch.Tensor, max_n: int,
        match_len: Optional[torch.Tensor] = None, hist: Optional[torch.Tensor] = None,
        want_len: bool = True, stream=None):
    """scone_tag: match lengths [B, T] int8 and/or an accumulated histogram
    (int64 tensor of MAX_FGRAM_LEN + 1 counts, indexed by length)."""
    _dev_i32(token_ids, "token_ids", 2)
    B, T = token_ids.shape
    if match_len is None and want_len:
        match_len = torch.empty((B, T), dtype=torch.int8, device=token_ids.device)
    if match_len is not None and (match_len.dtype != torch.int8 or match_len.numel() != B * T
                                  or not match_len.is_contiguous()):
        raise ValueError("match_len must be a contiguous int8 tensor of B*T elements")
    if hist is not None and (hist.dtype != torch.int64 or hist.numel() != MAX_FGRAM_LEN + 1
                             or hist.device.type != "cuda" or not hist.is_contiguous()):
        raise ValueError("hist must be a contiguous CUDA int64 tensor of MAX_FGRAM_LEN+1")
    with torch.cuda.device(token_ids.device):
        rc = lib().scone_tag(table.handle, _ptr(token_ids), B, T, int(max_n), _ptr(match_len),
                             _ptr(hist), _stream(stream))
    _check(rc, "scone_tag")
    return match_len, hist


def discover_workspace_bytes(B: int, T: int, max_len: int) -> int:
    """Bytes of scratch scone_discover_fgrams needs (-1 for rejected sizes)."""
    return int(lib().scone_discover_workspace(int(B), int(T), int(max_len)))


def discover_fgrams(token_ids: torch.Tensor, max_len: int, S: int, min_count: int = 5,
                    workspace: Optional[torch.Tensor] = None, stream=None):
    """scone_discover_fgrams: the S most frequent n-grams (2 <= n <= max_len) of
    the [B, T] token matrix.  Returns (fgrams [n, max_len], lengths [n],
    counts [n]) as CUDA int32 tensors, n = min(S, candidates).  The scratch
    is `workspace` (a CUDA uint8 tensor of discover_workspace_bytes) or, when
    None, a tensor from torch's caching allocator, so that repeated calls
    allocate no device memory."""
    _dev_i32(token_ids, "token_ids", 2)
    B, T = token_ids.shape
    dev = token_ids.device
    need = discover_workspace_bytes(B, T, max_len)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None and (workspace.dtype != torch.uint8 or workspace.device != dev
                                  or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor on the tokens' device")
    fg = torch.empty((max(S, 1), max_len), dtype=torch.int32, device=dev)
    ln = torch.empty(max(S, 1), dtype=torch.int32, device=dev)
    ct = torch.empty(max(S, 1), dtype=torch.int32, device=dev)
    n = ctypes.c_int64()
    with torch.cuda.device(dev):
        rc = lib().scone_discover_fgrams(_ptr(token_ids), B, T, int(max_len), int(min_count),
                                         int(S), _ptr(fg), _ptr(ln), _ptr(ct), ctypes.byref(n),
                                         _ptr(workspace),
                                         0 if workspace is None else workspace.numel(),
                                         _stream(stream))
    _check(rc, "scone_discover_fgrams")
    k = n.value
    return fg[:k], ln[:k], ct[:k]


_LAYER_PARAMS = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ln2_g", "ln2_b",
                 "w_fc1", "b_fc1", "w_fc2", "b_fc2")


class FgramModel:
    """Parameters of an f-gram model packed into one bf16 device blob in the
    order scone_fgram_model_forward reads them.

    ``params`` maps names to tensors (or arrays) of bf16 values or raw bf16
    bits (int16/uint16): "pos", "l{i}.<name>" for every layer i and name in
    ln1_g ln1_b w_qkv b_qkv w_o b_o ln2_g ln2_b w_fc1 b_fc1 w_fc2 b_fc2, then
    "lnf_g", "lnf_b".  Linear weights are [out_features, in_features]."""

    def __init__(self, params, d: int, n_heads: int, d_ff: int, n_layers: int, max_len: int,
                 device=None):
        self.d, self.n_heads, self.d_ff = int(d), int(n_heads), int(d_ff)
        self.n_layers, self.max_len = int(n_layers), int(max_len)
        n_par, total = ctypes.c_int64(), ctypes.c_int64()
        rc = lib().scone_fgram_model_layout(self.d, self.n_heads, self.d_ff, self.n_layers,
                                            self.max_len, None, ctypes.byref(n_par),
                                            ctypes.byref(total))
        _check(rc, "scone_fgram_model_layout")
        offs = (ctypes.c_int64 * n_par.value)()
        lib().scone_fgram_model_layout(self.d, self.n_heads, self.d_ff, self.n_layers,
                                       self.max_len, offs, ctypes.byref(n_par),
                                       ctypes.byref(total))
        names = ["pos"] + [f"l{i}.{p}" for i in range(self.n_layers) for p in _LAYER_PARAMS] \
            + ["lnf_g", "lnf_b"]
        assert len(names) == n_par.value
        device = torch.device("cuda", torch.cuda.current_device()) if device is None \
            else torch.device(device)
        blob = torch.zeros(total.value, dtype=torch.int16, device=device)
        for k, name in enumerate(names):
            v = params[name]
            t = v if isinstance(v, torch.Tensor) else torch.from_numpy(v)
            if t.dtype == torch.bfloat16:
                t = t.view(torch.int16)
            elif t.dtype == torch.uint16:
                t = t.view(torch.int16)
            elif t.dtype != torch.int16:
                raise TypeError(f"{name}: expected bf16 values or bits, got {t.dtype}")
            flat = t.reshape(-1)
            blob[offs[k]:offs[k] + flat.numel()].copy_(flat)
        self.blob = blob
        self.device = device


def precompute_fgram_rows(model: FgramModel, fgrams: torch.Tensor, lengths: torch.Tensor,
                          row_ids: torch.Tensor, tok_rows: torch.Tensor, rows: torch.Tensor,
                          stream=None):
    """scone_fgram_model_forward: rows[row_ids[k]] = F(f-gram k) (bf16), the
    f-gram model's output at the last token.  tok_rows [vocab, d] bf16 is the
    token embedding layer; rows [n_rows, d] bf16 is written in place.
    Synchronous."""
    _dev_i32(fgrams, "fgrams", 2)
    _dev_i32(lengths, "lengths", 1)
    _dev_i32(row_ids, "row_ids", 1)
    for name, t in (("tok_rows", tok_rows), ("rows", rows)):
        if t.device.type != "cuda" or t.dtype != torch.bfloat16 or t.dim() != 2 \
                or not t.is_contiguous() or t.shape[1] != model.d:
            raise ValueError(f"{name} must be a contiguous [*, {model.d}] bf16 CUDA tensor")
    n, K = fgrams.shape
    if K != model.max_len or lengths.numel() != n or row_ids.numel() != n:
        raise ValueError("fgrams must be [n, max_len] with n lengths and n row ids")
    with torch.cuda.device(rows.device):
        rc = lib().scone_fgram_model_forward(
            _ptr(fgrams), _ptr(lengths), _ptr(row_ids), n, model.max_len, _ptr(tok_rows),
            tok_rows.shape[0], model.blob.data_ptr(), model.d, model.n_heads, model.d_ff,
            model.n_layers, _ptr(rows), rows.shape[0], _stream(stream))
    _check(rc, "scone_fgram_model_forward")
    return rows


class HostRows:
    """A row table in pinned host memory that kernels read over PCIe."""

    def __init__(self, n_rows: int, row_shape, dtype: torch.dtype):
        self.n_rows = int(n_rows)
        self.row_shape = tuple(row_shape)
        self.dtype = dtype
        elem = torch.empty((), dtype=dtype).element_size()
        per_row = elem
        for s in self.row_shape:
            per_row *= s
        self.row_bytes = per_row
        self.nbytes = self.n_rows * per_row
        hp, dp = ctypes.c_void_p(), ctypes.c_void_p()
        _check(lib().scone_host_alloc(max(self.nbytes, 1), ctypes.byref(hp), ctypes.byref(dp)),
               "scone_host_alloc")
        self.host_ptr, self.device_ptr = hp.value, dp.value
        self._closed = False

    def rows(self, start: int, stop: int) -> "HostRows":
        """A view of rows [start, stop) sharing this allocation (not owning it)."""
        if not 0 <= start <= stop <= self.n_rows:
            raise ValueError("row range out of bounds")
        v = HostRows.__new__(HostRows)
        v.n_rows, v.row_shape, v.dtype, v.row_bytes = stop - start, self.row_shape, self.dtype, \
            self.row_bytes
        v.nbytes = v.n_rows * v.row_bytes
        v.host_ptr = self.host_ptr + start * self.row_bytes
        v.device_ptr = self.device_ptr + start * self.row_bytes
        v._closed = True  # a view never frees
        v._owner = self
        return v

    def tensor(self) -> torch.Tensor:
        """A CPU tensor view of the pinned memory (for filling and checking)."""
        buf = (ctypes.c_uint8 * self.nbytes).from_address(self.host_ptr)
        t = torch.frombuffer(buf, dtype=torch.uint8)
        return t.view(self.dtype).view((self.n_rows,) + self.row_shape)

    def close(self):
        if not self._closed:
            lib().scone_host_free(self.host_ptr)
            self._closed = True

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def gather(fgram_ids: torch.Tensor, rows, out: Optional[torch.Tensor] = None,
           stream=None) -> torch.Tensor:
    """scone_gather: out[k] = rows[fgram_ids[k]]; rows is a CUDA tensor or HostRows."""
    _dev_i32(fgram_ids, "fgram_ids")
    n_tok = fgram_ids.numel()
    placement, base, n_rows, row_bytes, row_shape, dtype = _rows_arg(rows)
    if out is None:
        out = torch.empty(tuple(fgram_ids.shape) + row_shape, dtype=dtype,
                          device=fgram_ids.device)
    if not out.is_contiguous() or out.numel() * out.element_size() != n_tok * row_bytes:
        raise ValueError("out must be contiguous with n_tok * row_bytes bytes")
    with torch.cuda.device(fgram_ids.device):
        rc = lib().scone_gather(_ptr(fgram_ids), n_tok, base, n_rows, row_bytes, _ptr(out),
                                placement, _stream(stream))
    _check(rc, "scone_gather")
    return out


def _rows_arg(rows):
    """(placement, pointer, n_rows, row_bytes, row_shape, dtype) of a row table."""
    if isinstance(rows, HostRows):
        return PLACE_HOST, rows.device_ptr, rows.n_rows, rows.row_bytes, rows.row_shape, rows.dtype
    if not isinstance(rows, torch.Tensor) or rows.device.type != "cuda":
        raise TypeError("rows must be a CUDA tensor or HostRows")
    if not rows.is_contiguous() or rows.dim() < 1:
        raise ValueError("rows must be a contiguous [n_rows, ...] tensor")
    row_shape = tuple(rows.shape[1:])
    row_bytes = int(torch.Size(row_shape).numel()) * rows.element_size()
    return PLACE_HBM, _ptr(rows), rows.shape[0], row_bytes, row_shape, rows.dtype


def embed(table: Table, token_ids: torch.Tensor, max_n: int, rows, out=None,
          fgram_ids: Optional[torch.Tensor] = None, match_len: Optional[torch.Tensor] = None,
          stream=None) -> torch.Tensor:
    """scone_embed: fused lookup + gather; returns out [B, T, *row_shape]."""
    _dev_i32(token_ids, "token_ids", 2)
    B, T = token_ids.shape
    placement, base, n_rows, row_bytes, row_shape, dtype = _rows_arg(rows)
    if out is None:
        out = torch.empty((B, T) + row_shape, dtype=dtype, device=token_ids.device)
    if not out.is_contiguous() or out.numel() * out.element_size() != B * T * row_bytes:
        raise ValueError("out must be contiguous with B * T * row_bytes bytes")
    for name, t, dt in (("fgram_ids", fgram_ids, torch.int32), ("match_len", match_len, torch.int8)):
        if t is not None and (t.dtype != dt or t.numel() != B * T or not t.is_contiguous()
                              or t.device != token_ids.device):
            raise ValueError(f"{name} must be a contiguous {dt} device tensor of B*T elements")
    with torch.cuda.device(token_ids.device):
        rc = lib().scone_embed(table.handle, _ptr(token_ids), B, T, int(max_n), base, n_rows,
                               row_bytes, placement, _ptr(out), _ptr(fgram_ids), _ptr(match_len),
                               _stream(stream))
    _check(rc, "scone_embed")
    return out


def embed_pipelined(table: Table, next_tokens: Optional[torch.Tensor], max_n: int,
                    next_ids: Optional[torch.Tensor], cur_ids: Optional[torch.Tensor], rows,
                    out: Optional[torch.Tensor] = None, next_len: Optional[torch.Tensor] = None,
                    stream=None) -> Optional[torch.Tensor]:
    """scone_embed_pipelined: in one launch, look up next_tokens [B, T] into
    next_ids and gather the rows of cur_ids into out [*cur_ids.shape, *row_shape].
    Either half may be None (lookup only, or gather only).  Returns out."""
    placement, base, n_rows, row_bytes, row_shape, dtype = _rows_arg(rows)
    B = T = 0
    if next_tokens is not None:
        _dev_i32(next_tokens, "next_tokens", 2)
        B, T = next_tokens.shape
        if next_ids is None:
            raise ValueError("next_ids is required with next_tokens")
        _dev_i32(next_ids, "next_ids")
        if next_ids.numel() != B * T:
            raise ValueError("next_ids has the wrong size")
        if next_len is not None and (next_len.dtype != torch.int8 or next_len.numel() != B * T
                                     or not next_len.is_contiguous()):
            raise ValueError("next_len must be a contiguous int8 tensor of B*T elements")
    n_cur = 0
    if cur_ids is not None:
        _dev_i32(cur_ids, "cur_ids")
        n_cur = cur_ids.numel()
        if out is None:
            out = torch.empty(tuple(cur_ids.shape) + row_shape, dtype=dtype,
                              device=cur_ids.device)
        if not out.is_contiguous() or out.numel() * out.element_size() != n_cur * row_bytes:
            raise ValueError("out must be contiguous with n_cur * row_bytes bytes")
    device = next_tokens.device if next_tokens is not None else (
        cur_ids.device if cur_ids is not None else table.device)
    with torch.cuda.device(device):
        rc = lib().scone_embed_pipelined(
            table.handle, _ptr(next_tokens), B, T, int(max_n), _ptr(next_ids), _ptr(next_len),
            _ptr(cur_ids), n_cur, base, n_rows, row_bytes, placement, _ptr(out),
            _stream(stream))
    _check(rc, "scone_embed_pipelined")
    return out


def decode_step(table: Table, ctx: torch.Tensor, ctx_len: torch.Tensor, new_tok: torch.Tensor,
                max_n: int, rows, out: torch.Tensor, fgram_ids: Optional[torch.Tensor] = None,
                match_len: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """scone_decode_step: ctx [S, cap] and ctx_len [S] are updated in place."""
    _dev_i32(ctx, "ctx", 2)
    _dev_i32(ctx_len, "ctx_len", 1)
    _dev_i32(new_tok, "new_tok", 1)
    S, cap = ctx.shape
    if ctx_len.numel() != S or new_tok.numel() != S:
        raise ValueError("ctx, ctx_len and new_tok disagree on S")
    placement, base, n_rows, row_bytes, _, _ = _rows_arg(rows)
    if not out.is_contiguous() or out.numel() * out.element_size() != S * row_bytes:
        raise ValueError("out must be contiguous with S * row_bytes bytes")
    for name, t, dt in (("fgram_ids", fgram_ids, torch.int32), ("match_len", match_len, torch.int8)):
        if t is not None and (t.dtype != dt or t.numel() != S or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous {dt} tensor of S elements")
    with torch.cuda.device(ctx.device):
        rc = lib().scone_decode_step(table.handle, _ptr(ctx), _ptr(ctx_len), cap, _ptr(new_tok),
                                     S, int(max_n), base, n_rows, row_bytes, placement, _ptr(out),
                                     _ptr(fgram_ids), _ptr(match_len), _stream(stream))
    _check(rc, "scone_decode_step")
    return out


def split_workspace_bytes(n_tok: int, row_bytes: int) -> int:
    """scone_gather_split_workspace."""
    n = lib().scone_gather_split_workspace(int(n_tok), int(row_bytes))
    if n < 0:
        raise ValueError("invalid sizes")
    return n


def gather_split(fgram_ids: torch.Tensor, near_rows: torch.Tensor, far_rows: "HostRows",
                 workspace: torch.Tensor, out: Optional[torch.Tensor] = None,
                 n_unique: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """scone_gather_split: ids < len(near_rows) read near_rows (device), the rest
    read far_rows (pinned host), each distinct far row crossing PCIe once."""
    _dev_i32(fgram_ids, "fgram_ids")
    n_tok = fgram_ids.numel()
    pn, near_ptr, n_near, rb_n, shape_n, dt_n = _rows_arg(near_rows)
    pf, far_ptr, n_far, rb_f, shape_f, dt_f = _rows_arg(far_rows)
    if pn != PLACE_HBM or pf != PLACE_HOST:
        raise TypeError("near_rows must be a CUDA tensor and far_rows HostRows")
    if rb_n != rb_f or dt_n != dt_f:
        raise ValueError("near and far rows differ in width or dtype")
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    if out is None:
        out = torch.empty(tuple(fgram_ids.shape) + shape_n, dtype=dt_n, device=fgram_ids.device)
    if not out.is_contiguous() or out.numel() * out.element_size() != n_tok * rb_n:
        raise ValueError("out must be contiguous with n_tok * row_bytes bytes")
    if n_unique is not None and (n_unique.dtype != torch.int32 or n_unique.device.type != "cuda"):
        raise ValueError("n_unique must be a CUDA int32 tensor")
    with torch.cuda.device(fgram_ids.device):
        rc = lib().scone_gather_split(_ptr(fgram_ids), n_tok, near_ptr, n_near, far_ptr, n_far,
                                      rb_n, _ptr(out), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(),
                                      _ptr(n_unique), _stream(stream))
    _check(rc, "scone_gather_split")
    return out


def check(stream=None, device=None) -> int:
    """scone_check: wait for the stream and return (and clear) the device's error status."""
    dev = device if device is not None else torch.cuda.current_device()
    with torch.cuda.device(dev):
        return lib().scone_check(_stream(stream))


def check_ok(stream=None):
    _check(check(stream), "asynchronous call")
