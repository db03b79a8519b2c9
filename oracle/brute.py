"""Pure-Python brute force of the trie-automaton masks: TEST INFRASTRUCTURE ONLY.

For tiny inputs only.  It is the plain definition, written without any trie:

* L = { s + T : s in the set }  (every value closed by the terminator byte T)
* the states are the distinct prefixes of the words of L (appendix "FSM
  Complexity Analysis": one state per distinct prefix, plus a dead state),
  numbered by their rank in bytewise lexicographic order (a proper prefix sorts
  before its extensions; Python's ``bytes`` ordering is exactly that);
* token t is valid at prefix p iff t is non-empty and p + t is a prefix of some
  word of L (appendix "Correctness", conditions (i) and (ii));
* advance(p, t) is the state of p + t, or -1 (dead) when t is not valid.
"""
from __future__ import annotations


def prefixes(strings, terminator: bytes = b'"') -> list:
    words = {bytes(s) + terminator for s in strings}
    return sorted({w[:i] for w in words for i in range(len(w) + 1)})


class Brute:
    def __init__(self, strings, vocab, terminator: bytes = b'"', base: int = 0):
        self.words = sorted({bytes(s) + terminator for s in strings})
        self.P = prefixes(strings, terminator)
        self.id = {p: base + i for i, p in enumerate(self.P)}
        self.base = base
        self.N = len(self.P)
        self.vocab = [bytes(t) for t in vocab]
        self.T = terminator

    def is_valid(self, node: int, v: int) -> bool:
        t = self.vocab[v]
        if not t or not (self.base <= node < self.base + self.N):
            return False
        p = self.P[node - self.base] + t
        return any(w.startswith(p) for w in self.words)

    def valid_set(self, node: int) -> set:
        return {v for v in range(len(self.vocab)) if self.is_valid(node, v)}

    def advance(self, node: int, v: int) -> int:
        if not (0 <= v < len(self.vocab)) or not self.is_valid(node, v):
            return -1
        return self.id[self.P[node - self.base] + self.vocab[v]]

    def is_final(self, node: int) -> bool:
        return self.P[node - self.base] in set(self.words)


def forest(sets, vocab, terminator: bytes = b'"') -> list:
    """One Brute per set, numbered one after another."""
    out, base = [], 0
    for strings in sets:
        b = Brute(strings, vocab, terminator, base)
        out.append(b)
        base += b.N
    return out
