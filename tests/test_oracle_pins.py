"""Pins of the oracle against what the paper and the mathematics fix.

* the paper's worked example and Figure 2 (golden files, cited there);
* closed forms (node count of disjoint strings, single chains, byte vocabularies);
* exhaustive and randomised comparison with the brute-force definition;
* masked logits against an independent library routine (``torch.where``),
  compared as raw bits.
"""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import DEAD, Oracle, OracleError
from oracle.brute import Brute, forest

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def rowset(row, V):
    bits = np.unpackbits(np.asarray(row, dtype=np.uint64).view(np.uint8), bitorder="little")
    assert not bits[V:].any(), "bits beyond V must be zero"
    return set(np.flatnonzero(bits[:V]).tolist())


def node_of(o: Oracle, prefix: bytes, root=0) -> int:
    """Find a node by walking single-byte steps of the oracle's own tables."""
    n = root
    for c in prefix:
        kids = np.flatnonzero((o.parent == n) & (o.edge == c))
        assert kids.size == 1
        n = int(kids[0])
    return n


# ------------------------------------------------------------ worked example --

def test_worked_example_printed_facts(oracle_mod):
    g = json.load(open(os.path.join(GOLD, "worked_example.json")))["printed"]
    strings = [s.encode() for s in g["strings"]]
    vocab = [t.encode() for t in g["vocab"]]
    o = Oracle(strings, vocab)
    assert sum(len(s) for s in strings) == g["n_chars"]
    # the paper counts nodes without end markers: drop the K terminator nodes
    assert o.N - int(o.is_final.sum()) == g["trie_nodes"]
    for name, prefix in g["named_nodes"].items():
        assert node_of(o, prefix.encode()) == int(name[2:])
    tid = {t: i for i, t in enumerate(g["vocab"])}
    for prefix, toks in g["valid"].items():
        n = node_of(o, prefix.encode())
        assert rowset(o.mask_rows([n])[0], o.V) == {tid[t] for t in toks}
    for tok, prefix in g["valid_somewhere_in_chain"].items():
        assert tid[tok] in rowset(o.mask_rows([node_of(o, prefix.encode())])[0], o.V)
    # below the branch node, every row has at most one valid token
    rows = o.mask_rows(np.arange(o.N))
    branch = node_of(o, b"medical_")
    for n in range(branch + 1, o.N):
        assert len(rowset(rows[n], o.V)) <= 1


def test_worked_example_full_table(oracle_mod):
    """Every node id, row and a few advances, derived by hand from the definition.

    Prefixes of {medical_billing", medical_coding", medical_records"} in
    lexicographic order: '' m me med medi medic medica medical (=7) medical_ (=8)
    medical_b .. medical_bill (=12) .. medical_billing (=15) medical_billing" (=16)
    medical_c .. medical_cod (=19) .. medical_coding (=22) medical_coding" (=23)
    medical_r .. medical_rec (=26) .. medical_records (=30) medical_records" (=31).
    """
    g = json.load(open(os.path.join(GOLD, "worked_example.json")))["printed"]
    vocab = [t.encode() for t in g["vocab"]] + [b'"']
    o = Oracle([s.encode() for s in g["strings"]], vocab)
    assert o.N == 32
    assert set(np.flatnonzero(o.is_final).tolist()) == {16, 23, 31}
    rows = o.mask_rows(np.arange(o.N))
    expect = {0: {0}, 7: {1, 2, 3}, 12: {4}, 19: {4}, 26: {5}, 15: {6}, 22: {6}, 30: {6}}
    for n in range(o.N):
        assert rowset(rows[n], o.V) == expect.get(n, set()), n
    nodes = [0, 7, 12, 0, 15, 16, 26, 31, -1, 40, 7]
    toks = [0, 1, 4, 1, 6, 6, 5, 6, 0, 0, 99]
    assert o.advance(nodes, toks).tolist() == [7, 12, 15, DEAD, 16, DEAD, 30, DEAD, DEAD, DEAD, DEAD]


def test_fig2_toy(oracle_mod):
    g = json.load(open(os.path.join(GOLD, "fig2.json")))["printed"]
    strings = [s.encode() for s in g["strings"]]
    vocab = [t.encode() for t in g["vocab"]]
    o = Oracle(strings, vocab)
    tid = {t: i for i, t in enumerate(g["vocab"])}
    for prefix, toks in g["valid_superset"].items():
        got = rowset(o.mask_rows([node_of(o, prefix.encode())])[0], o.V)
        assert {tid[t] for t in toks} <= got
        b = Brute(strings, vocab)
        assert got == b.valid_set(b.id[prefix.encode()])
    for prefix, toks in g["valid_exact"].items():
        assert rowset(o.mask_rows([node_of(o, prefix.encode())])[0], o.V) == {tid[t] for t in toks}


# ------------------------------------------------------------- closed forms --

def test_node_count_disjoint_strings(oracle_mod):
    # no two strings share a first byte: nothing merges, N = 1 + sum(|s| + 1)
    strings = [b"alpha", b"bravo!", b"c", b"", b"\x80\x90\xa0"]
    o = Oracle(strings, [b"x"])
    assert o.N == 1 + sum(len(s) + 1 for s in strings)


def test_single_chain_with_byte_vocab(oracle_mod):
    s = b"chain_of_bytes"
    vocab = [bytes([c]) for c in range(256)]
    o = Oracle([s], vocab)
    assert o.N == len(s) + 2
    rows = o.mask_rows(np.arange(o.N))
    word = s + b'"'
    for n in range(o.N):
        got = rowset(rows[n], 256)
        if n == o.N - 1:
            assert got == set() and o.is_final[n]
        else:
            assert got == {word[n]}, n       # preorder of a chain = depth order
    assert o.depth.tolist() == list(range(len(s) + 2))


def test_root_row_of_byte_vocab_is_first_bytes(oracle_mod):
    strings = [b"zeta", b"alpha", b"alps", b"", b"\xffend", b"beta"]
    o = Oracle(strings, [bytes([c]) for c in range(256)])
    assert rowset(o.mask_rows([0])[0], 256) == {(s + b'"')[0] for s in strings}


def test_node_count_is_distinct_prefix_count(oracle_mod):
    import workloads as W
    w = W.config(1)
    o = Oracle(w.strings, [b"a"])
    words = {s + b'"' for s in w.strings}
    assert o.N == len({x[:i] for x in words for i in range(len(x) + 1)})


def test_terminator_rejected_and_bad_args(oracle_mod):
    with pytest.raises(OracleError) as e:
        Oracle([b'ab"c'], [b"a"])
    assert e.value.code == 2
    with pytest.raises(OracleError):
        Oracle([], [b"a"])
    # a different terminator accepts '"' inside strings
    o = Oracle([b'ab"c'], [b'b"c'], terminator=ord("|"))
    assert rowset(o.mask_rows([node_of(o, b"a")])[0], 1) == {0}


# ------------------------------------------------------------ brute force --

ALPHA = [b"", b"a", b"b", b"aa", b"ab", b"ba", b"bb"]
TINY_VOCAB = [b""] + [bytes(p) for n in (1, 2, 3) for p in itertools.product(b'ab"', repeat=n)]


def compare_with_brute(strings, vocab, sets=None):
    if sets is None:
        o = Oracle(strings, vocab)
        bs = [Brute(strings, vocab)]
    else:
        flat = [s for grp in sets for s in grp]
        offs = np.cumsum([0] + [len(g) for g in sets])
        o = Oracle(flat, vocab, set_offsets=offs)
        bs = forest(sets, vocab)
    assert o.N == sum(b.N for b in bs)
    assert o.roots.tolist() == [b.base for b in bs]
    rows = o.mask_rows(np.arange(o.N))
    nodes, toks, expect = [], [], []
    for b in bs:
        for i, p in enumerate(b.P):
            n = b.base + i
            assert o.depth[n] == len(p)
            assert bool(o.is_final[n]) == b.is_final(n)
            assert rowset(rows[n], len(vocab)) == b.valid_set(n), (p, n)
            for v in range(len(vocab)):
                nodes.append(n)
                toks.append(v)
                expect.append(b.advance(n, v))
    assert o.advance(nodes, toks).tolist() == expect


def test_exhaustive_tiny_sets(oracle_mod):
    # every non-empty set of strings over {a, b} of length <= 2, against every
    # token over {a, b, '"'} of length <= 3 and the empty token
    for r in range(1, len(ALPHA) + 1):
        for combo in itertools.combinations(ALPHA, r):
            compare_with_brute(list(combo), TINY_VOCAB)


def test_tiny_forest(oracle_mod):
    compare_with_brute(None, TINY_VOCAB, sets=[[b"ab", b"a"], [b""], [b"ba", b"bb", b"b"]])


@settings(max_examples=150, deadline=None)
@given(
    strings=st.lists(st.binary(max_size=6).map(lambda x: x.replace(b'"', b"q")), min_size=1, max_size=6),
    vocab=st.lists(st.sampled_from([b"", b"a", b"b", b'"', b"ab", b"ba", b'a"', b'"x', b"abc", b"q",
                                    b"\x80", b"\x00", b"aq", b"qq"]) | st.binary(max_size=4),
                   min_size=1, max_size=40),
)
def test_random_vs_brute(oracle_mod, strings, vocab):
    compare_with_brute(strings, vocab)


@settings(max_examples=40, deadline=None)
@given(sets=st.lists(st.lists(st.binary(min_size=0, max_size=4, ).map(lambda x: x.replace(b'"', b"")),
                              min_size=1, max_size=4), min_size=1, max_size=4))
def test_random_forest_vs_brute(oracle_mod, sets):
    compare_with_brute(None, TINY_VOCAB, sets=sets)


def test_edge_suite_vs_brute(oracle_mod):
    import workloads as W
    for name, strings, vocab in W.edge_cases():
        compare_with_brute(strings, vocab)


# ----------------------------------------------------------------- apply --

def _special_values(rng, B, V, np_dtype):
    x = rng.standard_normal((B, V)).astype(np.float32)
    flat = x.reshape(-1)
    k = min(flat.size, 64)
    flat[:k] = np.array([np.nan, -0.0, 0.0, np.inf, -np.inf, 1e-40, -1e-40, 3.0e38] * 8,
                        dtype=np.float32)[:k]
    rng.shuffle(flat)
    return x


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_apply_matches_torch_where(oracle_mod, dtype):
    import torch
    import workloads as W
    w = W.config(1)
    o = Oracle(w.strings, w.vocab[:5000])
    rng = np.random.default_rng(7)
    B = 6
    x = torch.from_numpy(_special_values(rng, B, 5000 + 37, np.float32))
    x[0, 5:9] = torch.tensor([float("nan")] * 4).view(torch.int32).add(7).view(torch.float32)  # NaN payloads
    if dtype == "bf16":
        x = x.to(torch.bfloat16)
        bits = x.view(torch.int16).numpy().view(np.uint16)
        code = 1
    else:
        bits = x.view(torch.int32).numpy().view(np.uint32)
        code = 0
    nodes = np.array([0, 3, o.N - 1, -1, o.N + 5, 1], dtype=np.int32)
    got = o.apply(nodes, bits, code)
    rows = o.mask_rows(np.clip(nodes, 0, o.N - 1))
    for b, n in enumerate(nodes):
        valid = np.unpackbits(rows[b].view(np.uint8), bitorder="little")[: o.V].astype(bool)
        if not (0 <= n < o.N):
            valid[:] = False
        full = np.zeros(x.shape[1], dtype=bool)
        full[: o.V] = valid
        full[o.V:] = True  # columns beyond V are outside the vocabulary: untouched
        ref = torch.where(torch.from_numpy(full), x[b], torch.tensor(float("-inf"), dtype=x.dtype))
        ref_bits = ref.view(torch.int16 if dtype == "bf16" else torch.int32).numpy()
        assert np.array_equal(got[b].view(ref_bits.dtype), ref_bits)


# ------------------------------------------------------ fixed-format strings --
# Character-position masks (appendix "Constraint-Aware Dispatch Beyond Finite
# Sets").  A fixed format with small classes is also a finite set (every string
# the format admits), whose trie the set oracle builds on its own; every trie
# node at depth p has the same continuations, so its row must equal the format's
# row at position p, and its advance the format's advance.

def _format_set(classes):
    return [bytes(t) for t in itertools.product(*[list(c) for c in classes])]


TINY_FORMATS = [
    [b"ab"],
    [b"ab", b"01"],
    [b"a", b"-", b"01"],
    [b"ab", b"ab", b"ab"],
    [b"0123", b"ab", b"x"],
]


@pytest.mark.parametrize("classes", TINY_FORMATS, ids=["-".join(c.decode() for c in f) for f in TINY_FORMATS])
def test_format_equals_trie_of_enumerated_set(oracle_mod, classes):
    alphabet = sorted(set(b"".join(classes)) | {ord('"'), ord("z")})
    vocab = [b""] + [bytes(t) for n in (1, 2, 3) for t in itertools.product(alphabet, repeat=n)]
    f = oracle_mod.Format(classes, vocab)
    strings = _format_set(classes)
    o = Oracle(strings, vocab)
    b = Brute(strings, vocab)
    L = len(classes)
    assert f.N == L + 2
    frows = f.mask_rows(np.arange(L + 2))
    trows = o.mask_rows(np.arange(o.N))
    toks = np.arange(len(vocab), dtype=np.int32)
    for n in range(o.N):
        p = int(o.depth[n])
        assert np.array_equal(trows[n], frows[p]), (n, p)
        assert rowset(frows[p], len(vocab)) == b.valid_set(n)
        fa = f.advance(np.full(len(vocab), p), toks)
        ta = o.advance(np.full(len(vocab), n), toks)
        assert np.array_equal(fa < 0, ta < 0)
        assert np.array_equal(fa[fa >= 0], o.depth[ta[ta >= 0]])
    # outside 0..L+1: dead, empty rows
    assert not f.mask_rows([-1, L + 2, 10 ** 6]).any()
    assert (f.advance([-1, L + 2], [1, 1]) == -1).all()


def test_format_closed_form_digits(oracle_mod):
    """L digit positions and a vocabulary of digit strings, with and without a
    closing quote: at position p the valid tokens are the digit strings of length
    <= L - p and the digit strings + '"' of length exactly L + 1 - p."""
    L = 6
    digits = b"0123456789"
    rng = np.random.default_rng(3)
    vocab = []
    for _ in range(400):
        n = int(rng.integers(1, 9))
        s = bytes(rng.choice(list(digits), size=n).tolist())
        vocab.append(s + b'"' if rng.random() < 0.3 else s)
    vocab += [b"1a", b"a1", b'"', b'""', b""]
    f = oracle_mod.Format([digits] * L, vocab)
    rows = f.mask_rows(np.arange(L + 2))
    for p in range(L + 2):
        exp = set()
        for v, t in enumerate(vocab):
            body, closed = (t[:-1], True) if t.endswith(b'"') else (t, False)
            if not t or not all(c in digits for c in body) or b'"' in body:
                continue
            if (not closed and 1 <= len(t) <= L - p) or (closed and len(t) == L + 1 - p):
                exp.add(v)
        assert rowset(rows[p], len(vocab)) == exp, p
    assert not rowset(rows[L + 1], len(vocab))
