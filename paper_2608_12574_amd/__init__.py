"""Trie-automaton token masks for constrained decoding on MI355X (gfx950).

``compile`` builds the trie of a finite set of strings and the per-node
vocabulary bitmasks; ``Handle.apply_mask`` / ``Handle.advance`` are the
per-step serving operations.  All of them call ``libtam.so`` (C ABI in
``include/tam.h``).
"""
from .tam import (DTYPE_BF16, DTYPE_FP32, FLAG_HOST_ONLY, FLAG_LAZY_ROWS, FLAG_NO_TABLE, FLAG_TAIL_LISTS, FLAG_TIMING,
                  PHASE_COUNT, PHASE_LISTS, PHASE_MARK,
                  PHASE_TABLE, PHASE_ZERO,
                  TAM_DEAD,
                  Handle, TamError, Vocab, compile, compile_format, format_rows_noalloc, lib)

__all__ = ["compile", "compile_format", "format_rows_noalloc", "Vocab", "Handle", "TamError", "lib", "TAM_DEAD", "DTYPE_FP32", "DTYPE_BF16",
           "FLAG_HOST_ONLY", "FLAG_LAZY_ROWS", "FLAG_NO_TABLE", "FLAG_TAIL_LISTS", "FLAG_TIMING", "PHASE_LISTS", "PHASE_ZERO", "PHASE_MARK",
           "PHASE_TABLE", "PHASE_COUNT"]
