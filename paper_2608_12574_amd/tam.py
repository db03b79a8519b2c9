"""Python binding of ``libtam.so`` (ctypes; argument marshalling only).

Every step of the path runs in the library: the host trie and vocabulary
tables in its C++ code, everything else in its HIP kernels.  PyTorch only
provides device memory (through the allocator callbacks) and the stream
(``torch.cuda.current_stream()``).  The library must have been built
(``python -m paper_2608_12574_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import functools
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
# TAM_LIBRARY names another build of the same library (e.g. the host-sanitized
# one of ``build.py --sanitize``); the default is the in-tree build.
LIB_PATH = os.environ.get("TAM_LIBRARY") or os.path.join(PKG, "libtam.so")

TAM_OK = 0
TAM_DEAD = -1
DTYPE_FP32, DTYPE_BF16 = 0, 1
FLAG_HOST_ONLY, FLAG_NO_TABLE, FLAG_TIMING, FLAG_TAIL_LISTS, FLAG_LAZY_ROWS = 1, 2, 4, 8, 16
PHASE_LISTS, PHASE_ZERO, PHASE_MARK, PHASE_COUNT = 1, 2, 4, 8
PHASE_TABLE = PHASE_ZERO | PHASE_MARK

STATUS = {0: "TAM_OK", -1: "TAM_E_INVAL", -2: "TAM_E_TERMINATOR", -3: "TAM_E_NOMEM",
          -4: "TAM_E_DEVICE", -5: "TAM_E_TOOLARGE", -6: "TAM_E_STATE"}

# the entry points declared in include/tam.h
ENTRY_POINTS = ("tam_compile", "tam_vocab_create", "tam_compile_vocab", "tam_compile_format", "tam_rebuild",
                "tam_info_get", "tam_layout_get",
                "tam_apply_mask", "tam_advance", "tam_export_rows", "tam_valid_counts", "tam_valid_pairs",
                "tam_timing_get",
                "tam_format_rows_noalloc", "tam_vocab_destroy", "tam_destroy", "tam_last_error")


class TamError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {msg}")
        self.status = status


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class Allocator(ctypes.Structure):
    _fields_ = [("alloc", ALLOC_FN), ("free", FREE_FN), ("ctx", ctypes.c_void_p)]


class Options(ctypes.Structure):
    _fields_ = [("terminator", ctypes.c_int), ("flags", ctypes.c_uint32), ("cache_rows", ctypes.c_int64)]


class Info(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("num_sets", ctypes.c_int64),
                ("num_strings", ctypes.c_int64), ("vocab_size", ctypes.c_int64),
                ("words_per_row", ctypes.c_int64), ("row_stride_words", ctypes.c_int64),
                ("max_token_len", ctypes.c_int64), ("device_bytes", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("terminator", ctypes.c_int32),
                ("roots", ctypes.POINTER(ctypes.c_int32)), ("parent", ctypes.POINTER(ctypes.c_int32)),
                ("depth", ctypes.POINTER(ctypes.c_int32)), ("edge_byte", ctypes.POINTER(ctypes.c_uint8)),
                ("is_final", ctypes.POINTER(ctypes.c_uint8)), ("table", ctypes.c_void_p),
                ("dense_rows", ctypes.c_int64), ("dense_row", ctypes.POINTER(ctypes.c_int32)),
                ("cache_rows", ctypes.c_int64), ("subtree_end", ctypes.POINTER(ctypes.c_int32)),
                ("list_capacity", ctypes.c_int64)]


class Layout(ctypes.Structure):
    _fields_ = [("blob_bytes", ctypes.c_int64), ("blob", ctypes.POINTER(ctypes.c_uint8)),
                ("node_at", ctypes.POINTER(ctypes.c_int32)), ("depth", ctypes.POINTER(ctypes.c_int32)),
                ("node_pos", ctypes.POINTER(ctypes.c_int32)), ("parent", ctypes.POINTER(ctypes.c_int32)),
                ("errors", ctypes.c_int64)]


class Timing(ctypes.Structure):
    _fields_ = [("host_trie_ms", ctypes.c_double), ("host_vocab_ms", ctypes.c_double),
                ("upload_ms", ctypes.c_double), ("dev_lists_ms", ctypes.c_float),
                ("dev_zero_ms", ctypes.c_float), ("dev_mark_ms", ctypes.c_float),
                ("dev_total_ms", ctypes.c_float)]

    def as_dict(self) -> dict:
        return {k: float(getattr(self, k)) for k, _ in self._fields_}


_lib = None


def lib() -> ctypes.CDLL:
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_12574_amd.build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        P, i64 = ctypes.c_void_p, ctypes.c_int64
        L.tam_compile.argtypes = [P, P, i64, P, P, i64, P, i64, ctypes.POINTER(Options),
                                  ctypes.POINTER(Allocator), P, ctypes.POINTER(P)]
        L.tam_vocab_create.argtypes = [P, P, i64, ctypes.c_uint32, ctypes.POINTER(Allocator), P,
                                       ctypes.POINTER(P)]
        L.tam_compile_vocab.argtypes = [P, P, i64, P, P, i64, ctypes.POINTER(Options),
                                        ctypes.POINTER(Allocator), P, ctypes.POINTER(P)]
        L.tam_compile_format.argtypes = [P, i64, P, ctypes.POINTER(Options), ctypes.POINTER(Allocator), P,
                                         ctypes.POINTER(P)]
        L.tam_format_rows_noalloc.argtypes = [P, i64, ctypes.c_int, P, P, i64, P, P]
        L.tam_vocab_destroy.argtypes = [P]
        L.tam_vocab_destroy.restype = None
        L.tam_rebuild.argtypes = [P, ctypes.c_uint, P]
        L.tam_info_get.argtypes = [P, ctypes.POINTER(Info)]
        L.tam_layout_get.argtypes = [P, ctypes.POINTER(Layout)]
        L.tam_apply_mask.argtypes = [P, P, i64, P, ctypes.c_int, i64, P]
        L.tam_advance.argtypes = [P, P, P, i64, P, P]
        L.tam_export_rows.argtypes = [P, P, i64, P, P]
        L.tam_valid_counts.argtypes = [P, P, i64, P, P]
        L.tam_valid_pairs.argtypes = [P, P, ctypes.POINTER(i64)]
        L.tam_timing_get.argtypes = [P, ctypes.POINTER(Timing)]
        L.tam_destroy.argtypes = [P]
        L.tam_destroy.restype = None
        L.tam_last_error.restype = ctypes.c_char_p
        for name in ENTRY_POINTS:
            if name not in ("tam_vocab_destroy", "tam_destroy", "tam_last_error"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != TAM_OK:
        raise TamError(rc, where, lib().tam_last_error().decode(errors="replace"))


def csr(items) -> tuple:
    """list[bytes] -> (uint8 blob, int64 offsets[len+1]) as numpy arrays.  A pair
    (blob, offsets) of arrays is taken as already packed."""
    if isinstance(items, tuple) and len(items) == 2 and isinstance(items[0], np.ndarray):
        blob = np.ascontiguousarray(items[0], dtype=np.uint8)
        off = np.ascontiguousarray(items[1], dtype=np.int64)
        return (blob if blob.size else np.zeros(1, dtype=np.uint8)), off
    if not isinstance(items, list):
        items = list(items)
    off = np.zeros(len(items) + 1, dtype=np.int64)
    if items:
        np.cumsum(np.fromiter(map(len, items), dtype=np.int64, count=len(items)), out=off[1:])
    blob = np.frombuffer(b"".join(items), dtype=np.uint8)
    if blob.size == 0:
        blob = np.zeros(1, dtype=np.uint8)
    return np.ascontiguousarray(blob), off


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


class _TorchAllocator:
    """Device memory for the library, taken from torch's caching allocator."""

    def __init__(self, device):
        import torch
        self.torch = torch
        self.device = device
        self.live = {}
        self.c_alloc = ALLOC_FN(self._alloc)
        self.c_free = FREE_FN(self._free)
        self.struct = Allocator(self.c_alloc, self.c_free, None)

    def _alloc(self, nbytes, ctx):
        try:
            t = self.torch.empty(int(nbytes), dtype=self.torch.uint8, device=self.device)
        except Exception:  # out of memory: the library reports TAM_E_NOMEM
            return None
        p = t.data_ptr()
        self.live[p] = t
        return p

    def _free(self, p, ctx):
        self.live.pop(p, None)


def _stream_ptr(stream, host_only=False):
    """The HIP stream for a call: ``stream``, else torch's current stream on the
    current device (read as a raw pointer: building a Stream object costs more
    than the call it serves)."""
    if host_only:
        return ctypes.c_void_p(None)
    import torch
    if stream is not None:
        return ctypes.c_void_p(stream.cuda_stream)
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    if raw is not None:
        return ctypes.c_void_p(raw(torch.cuda.current_device()))
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class Handle:
    """A compiled set (or forest of sets) with its per-node token masks."""

    def __init__(self, raw, allocator, device, host_only):
        self._raw = raw
        self._alloc = allocator
        self.device = device
        self.host_only = host_only
        info = Info()
        _check(lib().tam_info_get(raw, ctypes.byref(info)), "tam_info_get")
        self.num_nodes = int(info.num_nodes)
        self.num_sets = int(info.num_sets)
        self.num_strings = int(info.num_strings)
        self.vocab_size = int(info.vocab_size)
        self.words_per_row = int(info.words_per_row)
        self.row_stride_words = int(info.row_stride_words)
        self.max_token_len = int(info.max_token_len)
        self.device_bytes = int(info.device_bytes)
        self.flags = int(info.flags)
        self.terminator = int(info.terminator)
        self.dense_rows = int(info.dense_rows)
        self.cache_rows = int(info.cache_rows)
        self.list_capacity = int(info.list_capacity)
        self.roots = np.ctypeslib.as_array(info.roots, shape=(self.num_sets,)).copy()
        self.table_ptr = info.table
        self._info = info  # per-node host arrays are copied on first use

    def _host_array(self, name):
        if self._raw is None:
            raise TamError(-6, name, "handle is closed")
        ptr = getattr(self._info, name)
        return np.ctypeslib.as_array(ptr, shape=(self.num_nodes,)).copy()

    @functools.cached_property
    def parent(self):
        return self._host_array("parent")

    @functools.cached_property
    def depth(self):
        return self._host_array("depth")

    @functools.cached_property
    def edge_byte(self):
        return self._host_array("edge_byte")

    @functools.cached_property
    def is_final(self):
        return self._host_array("is_final")

    @functools.cached_property
    def dense_row(self):
        """Table row of each node (-1: kept as a list), or None when row = node id."""
        if not self._info.dense_row:
            return None
        return self._host_array("dense_row")

    @functools.cached_property
    def subtree_end(self):
        """One past the last node of each node's subtree (rows built on demand), or None."""
        if not self._info.subtree_end:
            return None
        return self._host_array("subtree_end")

    # -- lifetime ------------------------------------------------------------
    def close(self):
        if self._raw is not None:
            lib().tam_destroy(self._raw)
            self._raw = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- serving ---------------------------------------------------------------
    def apply_mask(self, node_ids, logits, stream=None):
        """In place: logits[b, v] = -inf where token v is not valid at node_ids[b]."""
        import torch
        assert node_ids.dtype == torch.int32 and node_ids.is_cuda and node_ids.is_contiguous()
        assert logits.is_cuda and logits.dim() == 2 and logits.stride(1) == 1
        assert logits.shape[0] == node_ids.numel() and logits.shape[1] >= self.vocab_size
        dtype = {torch.float32: DTYPE_FP32, torch.bfloat16: DTYPE_BF16}[logits.dtype]
        _check(lib().tam_apply_mask(self._raw, ctypes.c_void_p(node_ids.data_ptr()), node_ids.numel(),
                                    ctypes.c_void_p(logits.data_ptr()), dtype, logits.stride(0),
                                    _stream_ptr(stream, self.host_only)), "tam_apply_mask")
        return logits

    def advance(self, node_ids, token_ids, out=None, stream=None):
        """out[b] = node reached from node_ids[b] by the bytes of token_ids[b], or -1."""
        import torch
        assert node_ids.dtype == torch.int32 and token_ids.dtype == torch.int32
        assert node_ids.is_contiguous() and token_ids.is_contiguous()
        assert node_ids.numel() == token_ids.numel()
        if out is None:
            out = torch.empty_like(node_ids)
        assert out.dtype == torch.int32 and out.is_contiguous() and out.numel() == node_ids.numel()
        _check(lib().tam_advance(self._raw, ctypes.c_void_p(node_ids.data_ptr()),
                                 ctypes.c_void_p(token_ids.data_ptr()), node_ids.numel(),
                                 ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream, self.host_only)), "tam_advance")
        return out

    def export_rows(self, node_ids, stream=None):
        """Canonical rows: int64 tensor [n, W] holding the uint64 mask words."""
        import torch
        assert node_ids.dtype == torch.int32 and node_ids.is_contiguous()
        out = torch.empty((node_ids.numel(), self.words_per_row), dtype=torch.int64,
                          device=node_ids.device)
        _check(lib().tam_export_rows(self._raw, ctypes.c_void_p(node_ids.data_ptr()), node_ids.numel(),
                                     ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream, self.host_only)),
               "tam_export_rows")
        return out

    def valid_counts(self, node_ids, stream=None):
        """int32 tensor [n]: |valid[node_ids[r]]| (0 for a dead node)."""
        import torch
        assert node_ids.dtype == torch.int32 and node_ids.is_contiguous()
        out = torch.empty(node_ids.numel(), dtype=torch.int32, device=node_ids.device)
        _check(lib().tam_valid_counts(self._raw, ctypes.c_void_p(node_ids.data_ptr()), node_ids.numel(),
                                      ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream, self.host_only)),
               "tam_valid_counts")
        return out

    def rebuild(self, phases: int = 0, stream=None):
        """Rerun device phases (PHASE_* mask; 0 = the handle's default; with
        FLAG_LAZY_ROWS, 0 empties the row cache)."""
        _check(lib().tam_rebuild(self._raw, phases, _stream_ptr(stream, self.host_only)), "tam_rebuild")

    def valid_pairs(self, stream=None) -> int:
        m = ctypes.c_int64()
        _check(lib().tam_valid_pairs(self._raw, _stream_ptr(stream, self.host_only), ctypes.byref(m)),
               "tam_valid_pairs")
        return int(m.value)

    def layout(self) -> dict:
        """The device's trie layout computed on the host (host-only handles):
        blob, node_at, depth, node_pos, parent (numpy copies) and errors."""
        lay = Layout()
        _check(lib().tam_layout_get(self._raw, ctypes.byref(lay)), "tam_layout_get")
        BB, N = int(lay.blob_bytes), self.num_nodes
        arr = lambda p, n: np.ctypeslib.as_array(p, shape=(n,)).copy()  # noqa: E731
        return {"blob": arr(lay.blob, BB), "node_at": arr(lay.node_at, BB), "depth": arr(lay.depth, N),
                "node_pos": arr(lay.node_pos, N), "parent": arr(lay.parent, N), "errors": int(lay.errors)}

    def timing(self) -> dict:
        t = Timing()
        _check(lib().tam_timing_get(self._raw, ctypes.byref(t)), "tam_timing_get")
        return t.as_dict()


class Vocab:
    """A vocabulary's device tables, built once per tokenizer (tam_vocab_create)
    and shared by every compile against it."""

    def __init__(self, tokens, host_only: bool = False, device=None, stream=None):
        tb, to = csr(tokens)
        self.size = len(to) - 1
        self.host_only = host_only
        self._alloc = None
        raw = ctypes.c_void_p()
        if host_only:
            rc = lib().tam_vocab_create(_ptr(tb), _ptr(to), self.size, FLAG_HOST_ONLY, None, None,
                                        ctypes.byref(raw))
            self.device = None
        else:
            import torch
            dev = torch.device(device if device is not None else "cuda")
            if dev.index is None:
                dev = torch.device("cuda", torch.cuda.current_device())
            self.device = dev
            self._alloc = _TorchAllocator(dev)
            with torch.cuda.device(dev):
                rc = lib().tam_vocab_create(_ptr(tb), _ptr(to), self.size, 0, ctypes.byref(self._alloc.struct),
                                            _stream_ptr(stream), ctypes.byref(raw))
        _check(rc, "tam_vocab_create")
        self._raw = raw

    def close(self):
        if getattr(self, "_raw", None) is not None:
            lib().tam_vocab_destroy(self._raw)
            self._raw = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def compile(strings, vocab, sets=None, terminator: int = 0x22, flags: int = 0, device=None,
            stream=None, cache_rows: int = 0) -> Handle:
    """tam_compile over ``strings`` (list[bytes], or a packed pair (uint8 blob,
    int64 offsets[K+1])) and ``vocab`` (a ``Vocab``, or a list[bytes] or packed
    pair, token id = index).

    ``sets``: optional forest offsets (S+1 ints) splitting ``strings`` into S sets.
    With ``FLAG_HOST_ONLY`` no GPU is touched (host tables only).
    ``cache_rows``: rows of the row cache with ``FLAG_LAZY_ROWS`` (0 = the default).
    """
    sb, so = csr(strings)
    set_arr = None
    S = 0
    if sets is not None:
        set_arr = np.ascontiguousarray(np.asarray(sets, dtype=np.int64))
        S = set_arr.size - 1
    opt = Options(terminator, flags, cache_rows)
    raw = ctypes.c_void_p()
    host_only = bool(flags & FLAG_HOST_ONLY)
    allocator = None
    sets_p = _ptr(set_arr) if set_arr is not None else None
    keep = None
    if not host_only:
        import torch
        device = torch.device(device if device is not None else "cuda")
        if device.index is None:
            device = torch.device("cuda", torch.cuda.current_device())
        allocator = _TorchAllocator(device)
        with torch.cuda.device(device):
            stream_p = _stream_ptr(stream)
            if isinstance(vocab, Vocab):
                keep = vocab
                rc = lib().tam_compile_vocab(_ptr(sb), _ptr(so), len(so) - 1, vocab._raw, sets_p, S,
                                             ctypes.byref(opt), ctypes.byref(allocator.struct), stream_p,
                                             ctypes.byref(raw))
            else:
                tb, to = csr(vocab)
                rc = lib().tam_compile(_ptr(sb), _ptr(so), len(so) - 1, _ptr(tb), _ptr(to), len(to) - 1,
                                       sets_p, S, ctypes.byref(opt), ctypes.byref(allocator.struct), stream_p,
                                       ctypes.byref(raw))
    else:
        if isinstance(vocab, Vocab):
            keep = vocab
            rc = lib().tam_compile_vocab(_ptr(sb), _ptr(so), len(so) - 1, vocab._raw, sets_p, S,
                                         ctypes.byref(opt), None, None, ctypes.byref(raw))
        else:
            tb, to = csr(vocab)
            rc = lib().tam_compile(_ptr(sb), _ptr(so), len(so) - 1, _ptr(tb), _ptr(to), len(to) - 1, sets_p, S,
                                   ctypes.byref(opt), None, None, ctypes.byref(raw))
    _check(rc, "tam_compile")
    h = Handle(raw, allocator, device, host_only)
    h._vocab = keep  # the vocabulary's allocator must outlive the handle
    return h


def format_class_rows(classes) -> np.ndarray:
    """Per-position allowed bytes (a list of L byte strings) as the [L][32] bit
    rows of tam_compile_format: byte c of position p is bit c & 7 of row[p][c >> 3]."""
    rows = np.zeros((len(classes), 32), dtype=np.uint8)
    for p, allowed in enumerate(classes):
        b = np.frombuffer(bytes(allowed), dtype=np.uint8)
        np.bitwise_or.at(rows[p], b >> 3, (1 << (b & 7)).astype(np.uint8))
    return rows


def format_rows_noalloc(classes, vocab: "Vocab", out, pairs_out=None, terminator: int = 0x22, stream=None):
    """tam_format_rows_noalloc: the character-position rows of ``classes`` (a list
    of L byte strings) written into ``out`` (a device int64 tensor [L + 2, >= W])
    without allocating; the valid-pair count into ``pairs_out`` (device int64
    [1]) when given."""
    import torch
    rows = np.ascontiguousarray(format_class_rows(classes))
    assert out.dtype == torch.int64 and out.is_cuda and out.dim() == 2 and out.stride(1) == 1
    assert out.shape[0] == len(classes) + 2
    _check(lib().tam_format_rows_noalloc(_ptr(rows), len(classes), terminator, vocab._raw,
                                         ctypes.c_void_p(out.data_ptr()), out.stride(0),
                                         ctypes.c_void_p(pairs_out.data_ptr()) if pairs_out is not None else None,
                                         _stream_ptr(stream)), "tam_format_rows_noalloc")
    return out


def compile_format(classes, vocab, terminator: int = 0x22, flags: int = 0, device=None, stream=None) -> Handle:
    """tam_compile_format: character-position masks of a fixed-format value whose
    character p is any byte of ``classes[p]`` (a bytes object); node p = position
    p, node L+1 = after the terminator.  ``vocab`` is a ``Vocab`` or a list[bytes]."""
    rows = np.ascontiguousarray(format_class_rows(classes))
    host_only = bool(flags & FLAG_HOST_ONLY)
    if not isinstance(vocab, Vocab):
        vocab = Vocab(vocab, host_only=host_only, device=device, stream=stream)
    opt = Options(terminator, flags)
    raw = ctypes.c_void_p()
    allocator = None
    if not host_only:
        import torch
        device = torch.device(device if device is not None else "cuda")
        if device.index is None:
            device = torch.device("cuda", torch.cuda.current_device())
        allocator = _TorchAllocator(device)
        with torch.cuda.device(device):
            rc = lib().tam_compile_format(_ptr(rows), len(classes), vocab._raw, ctypes.byref(opt),
                                          ctypes.byref(allocator.struct), _stream_ptr(stream), ctypes.byref(raw))
    else:
        rc = lib().tam_compile_format(_ptr(rows), len(classes), vocab._raw, ctypes.byref(opt), None, None,
                                      ctypes.byref(raw))
    _check(rc, "tam_compile_format")
    h = Handle(raw, allocator, device, host_only)
    h._vocab = vocab
    return h
