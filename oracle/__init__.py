"""The oracle: TEST INFRASTRUCTURE ONLY.

A plain, slow, single-threaded CPU implementation of the trie-automaton mask
path (``oracle.c``, plain C built with gcc) plus a pure-Python brute force for
tiny inputs (``brute.py``).  It shares no code with the HIP library and the
product never imports it; only the tests, ``__graft_entry__.smoke()`` and the
bench's CPU-baseline leg do.

Parity of every function here is pinned by ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

DEAD = -1
DTYPE_FP32, DTYPE_BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc (single-threaded, -O2)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build(force=True)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        L.oracle_build.argtypes = [P, P, i64, P, i64, ctypes.c_int, ctypes.POINTER(P)]
        L.oracle_build.restype = ctypes.c_int
        L.oracle_free.argtypes = [P]
        L.oracle_num_nodes.argtypes = [P]
        L.oracle_num_nodes.restype = i64
        L.oracle_num_sets.argtypes = [P]
        L.oracle_num_sets.restype = i64
        L.oracle_roots.argtypes = [P, P]
        L.oracle_node_info.argtypes = [P, P, P, P, P]
        L.oracle_mask_rows.argtypes = [P, P, P, i64, P, i64, P]
        L.oracle_mask_rows.restype = ctypes.c_int
        L.oracle_advance.argtypes = [P, P, P, i64, P, P, i64, P]
        L.oracle_advance.restype = ctypes.c_int
        L.oracle_apply.argtypes = [P, P, P, i64, P, i64, P, i64, ctypes.c_int]
        L.oracle_apply.restype = ctypes.c_int
        L.oracle_format_rows.argtypes = [P, i64, ctypes.c_int, P, P, i64, P, i64, P]
        L.oracle_format_rows.restype = ctypes.c_int
        L.oracle_format_advance.argtypes = [P, i64, ctypes.c_int, P, P, i64, P, P, i64, P]
        L.oracle_format_advance.restype = ctypes.c_int
        L.oracle_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def csr(items) -> tuple:
    """list[bytes] -> (uint8 blob, int64 offsets[len+1])."""
    lens = np.fromiter((len(x) for x in items), dtype=np.int64, count=len(items))
    off = np.zeros(len(items) + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    blob = np.frombuffer(b"".join(items), dtype=np.uint8)
    if blob.size == 0:
        blob = np.zeros(1, dtype=np.uint8)
    return np.ascontiguousarray(blob), off


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"oracle error {code}: {msg}")
        self.code = code


class Oracle:
    """Trie of one set (or a forest of sets) plus a vocabulary, on the CPU."""

    def __init__(self, strings, vocab, set_offsets=None, terminator=0x22):
        L = lib()
        self._sb, self._so = csr(list(strings))
        self._tb, self._to = csr(list(vocab))
        self.V = len(vocab)
        self.W = (self.V + 63) // 64
        so = None
        S = 1
        if set_offsets is not None:
            so = np.asarray(set_offsets, dtype=np.int64)
            S = len(so) - 1
        self._set_off = so
        h = ctypes.c_void_p()
        rc = L.oracle_build(_p(self._sb), _p(self._so), len(strings),
                            _p(so) if so is not None else None, S, terminator, ctypes.byref(h))
        if rc != 0:
            raise OracleError(rc, L.oracle_last_error().decode())
        self._h = h
        self.N = int(L.oracle_num_nodes(h))
        self.S = int(L.oracle_num_sets(h))
        self.roots = np.zeros(self.S, dtype=np.int32)
        L.oracle_roots(h, _p(self.roots))
        self.parent = np.zeros(self.N, dtype=np.int32)
        self.depth = np.zeros(self.N, dtype=np.int32)
        self.edge = np.zeros(self.N, dtype=np.uint8)
        self.is_final = np.zeros(self.N, dtype=np.uint8)
        L.oracle_node_info(h, _p(self.parent), _p(self.depth), _p(self.edge), _p(self.is_final))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.oracle_free(h)
            self._h = None

    def mask_rows(self, nodes) -> np.ndarray:
        nodes = np.ascontiguousarray(nodes, dtype=np.int32)
        out = np.zeros((nodes.size, self.W), dtype=np.uint64)
        lib().oracle_mask_rows(self._h, _p(self._tb), _p(self._to), self.V, _p(nodes), nodes.size,
                               _p(out))
        return out

    def advance(self, nodes, tokens) -> np.ndarray:
        nodes = np.ascontiguousarray(nodes, dtype=np.int32)
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.zeros(nodes.size, dtype=np.int32)
        lib().oracle_advance(self._h, _p(self._tb), _p(self._to), self.V, _p(nodes), _p(tokens),
                             nodes.size, _p(out))
        return out

    def apply(self, nodes, logits_bits: np.ndarray, dtype: int) -> np.ndarray:
        """Masked copy of ``logits_bits`` (uint32 rows for fp32, uint16 for bf16)."""
        nodes = np.ascontiguousarray(nodes, dtype=np.int32)
        out = np.array(logits_bits, copy=True, order="C")
        assert out.ndim == 2 and out.shape[0] == nodes.size and out.shape[1] >= self.V
        lib().oracle_apply(self._h, _p(self._tb), _p(self._to), self.V, _p(nodes), nodes.size,
                           _p(out), out.shape[1], dtype)
        return out

    def valid_ids(self, node) -> np.ndarray:
        row = self.mask_rows([node])[0]
        bits = np.unpackbits(row.view(np.uint8), bitorder="little")[: self.V]
        return np.flatnonzero(bits)


def class_rows(classes) -> np.ndarray:
    """list of L byte strings (the allowed bytes of each position) -> [L, 32] uint8
    bit rows: byte c allowed at position p iff bit c & 7 of row[p][c >> 3]."""
    rows = np.zeros((max(len(classes), 1), 32), dtype=np.uint8)
    for p, allowed in enumerate(classes):
        for c in bytes(allowed):
            rows[p, c >> 3] |= np.uint8(1 << (c & 7))
    return rows


class Format:
    """Character-position masks of a fixed-format value (appendix "Constraint-Aware
    Dispatch Beyond Finite Sets"): positions 0..L, then L+1 after the terminator."""

    def __init__(self, classes, vocab, terminator=0x22):
        lib()
        self.L = len(classes)
        self.N = self.L + 2
        self.T = terminator
        self._cls = class_rows(classes)
        self._tb, self._to = csr(list(vocab))
        self.V = len(vocab)
        self.W = (self.V + 63) // 64

    def mask_rows(self, pos) -> np.ndarray:
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        out = np.zeros((pos.size, self.W), dtype=np.uint64)
        rc = lib().oracle_format_rows(_p(self._cls), self.L, self.T, _p(self._tb), _p(self._to), self.V,
                                      _p(pos), pos.size, _p(out))
        assert rc == 0
        return out

    def advance(self, pos, tokens) -> np.ndarray:
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.zeros(pos.size, dtype=np.int32)
        lib().oracle_format_advance(_p(self._cls), self.L, self.T, _p(self._tb), _p(self._to), self.V,
                                    _p(pos), _p(tokens), pos.size, _p(out))
        return out
