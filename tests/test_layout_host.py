"""The device's trie layout, checked on the CPU against the oracle.

On a device compile the GPU derives its position tables (node_at, depth,
first positions, parents) from the string blob and one record per string.
``tam_layout_get`` runs the very functions those kernels call over the same
records on the host, so the layout can be pinned here: every position of the
blob must hold the node the oracle's trie reaches there (Section 4.1: one node
per distinct prefix), every depth and parent must be the oracle's, and no
record may be inconsistent.  Sets of strings nested as prefixes of one
another, whose records chain far back, are the case the layout walk has to
get right.
"""
import numpy as np
import pytest

import workloads as W
from oracle import Oracle

T = 0x22


@pytest.fixture(scope="module")
def P():
    import paper_2608_12574_amd as P
    try:
        P.lib()
    except RuntimeError:
        from paper_2608_12574_amd import build
        build.build()
    return P


def expected_layout(strings, offs, o, term=T):
    """Blob, node_at and first positions from the oracle's trie: per set in
    order, its distinct strings in trie (s + T) order, each after a pad byte
    that stands for the set's root."""
    child = {}
    par, edge = o.parent, o.edge
    for n in np.flatnonzero(par >= 0):
        child[(int(par[n]), int(edge[n]))] = int(n)
    if offs is None:
        offs = [0, len(strings)]
    tb = bytes([term])
    blob = bytearray(32)
    node_at = [0] * 32
    for j in range(len(offs) - 1):
        root = int(o.roots[j])
        for s in sorted(set(strings[offs[j]:offs[j + 1]]), key=lambda x: x + tb):
            blob.append(0)
            node_at.append(root)
            n = root
            for c in s + tb:
                n = child[(n, c)]
                blob.append(c)
                node_at.append(n)
    blob += bytes(32)
    node_at += [0] * 32
    node_at = np.asarray(node_at, dtype=np.int32)
    node_pos = np.full(o.N, -1, dtype=np.int64)
    first = np.unique(node_at, return_index=True)
    node_pos[first[0]] = first[1]
    node_pos[o.depth == 0] = -1
    return np.frombuffer(bytes(blob), dtype=np.uint8), node_at, node_pos


def check_layout(P, strings, vocab=(b"x",), sets=None, term=T):
    o = Oracle(strings, list(vocab), set_offsets=sets, terminator=term)
    h = P.compile(strings, list(vocab), sets=sets, terminator=term, flags=P.FLAG_HOST_ONLY)
    lay = h.layout()
    blob, node_at, node_pos = expected_layout(strings, sets, o, term)
    assert lay["errors"] == 0
    assert np.array_equal(lay["blob"], blob)
    assert np.array_equal(lay["node_at"], node_at)
    assert np.array_equal(lay["depth"], o.depth)
    assert np.array_equal(lay["node_pos"], node_pos)
    assert np.array_equal(lay["parent"], o.parent)
    # the child lists the device builds from these: every non-root node under its
    # parent, with the byte at its first position as the edge byte
    nonroot = o.depth > 0
    assert np.array_equal(lay["blob"][node_pos[nonroot]], o.edge[nonroot])
    h.close()
    return lay


def nested_chain(depth: int, a: bytes, b: bytes) -> list:
    """Strings each a prefix of the next, with side branches at every level:
    a record's shared prefix is owned by a string many records back."""
    out, cur = [], b""
    for k in range(depth):
        cur += a if k % 3 else b
        out += [cur, cur + b, cur + a + a]
    return out


def test_layout_worked_example(P):
    lay = check_layout(P, [b"medical_billing", b"medical_coding", b"medical_records"])
    assert lay["node_at"][32] == 0 and lay["node_at"][33 + 7 - 1] == 7  # pad = root, 'medical' = n7


@pytest.mark.parametrize("name,strings,vocab", W.edge_cases(), ids=[e[0] for e in W.edge_cases()])
def test_layout_edge_suite(P, name, strings, vocab):
    check_layout(P, strings, vocab)


def test_layout_nested_chains(P):
    for depth in (3, 8, 25, 71):
        check_layout(P, nested_chain(depth, b"ab", b"b"))
        check_layout(P, nested_chain(depth, b"a", b"ba") + [b""])


def test_layout_random_sets(P):
    """2,000 random sets and forests over two or three byte values: short
    strings, many of them prefixes of one another, the empty string often."""
    rng = np.random.default_rng(2608)
    for trial in range(2000):
        alpha = [b"a", b"b", b"\x00", b"\xff"][: int(rng.integers(2, 5))]
        nsets = int(rng.integers(1, 4))
        strings, offs = [], [0]
        for _ in range(nsets):
            base = [b"".join(rng.choice(alpha, size=int(rng.integers(0, 9)))) for _ in range(int(rng.integers(1, 5)))]
            grown = []
            for s in base:  # prefixes and extensions of each drawn string
                cut = int(rng.integers(0, len(s) + 1))
                grown += [s, s[:cut], s + b"".join(rng.choice(alpha, size=int(rng.integers(0, 4))))]
            k = int(rng.integers(1, len(grown) + 1))
            strings += [grown[i] for i in rng.permutation(len(grown))[:k]]
            offs.append(len(strings))
        check_layout(P, strings, sets=offs if nsets > 1 else None)


def test_layout_large_sets_built_in_parts(P):
    """Sets large enough that the host build cuts them into parts by first
    byte (each part's records chain only within it)."""
    strings, vocab, offs = W.mixed_forest()
    check_layout(P, strings, sets=offs)
    rng = np.random.default_rng(7)
    words = [b"get", b"ge", b"g", b"set", b"se", b"list_", b"l"]
    big = list({b"_".join(rng.choice(words, size=int(rng.integers(1, 5)))) for _ in range(6000)})
    check_layout(P, big + [b""])


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_layout_configs(P, cid):
    w = W.config(cid)
    check_layout(P, w.strings)


def test_layout_forest_c5_sets(P):
    w = W.config(5)
    sets = w.set_offsets[:41]  # the first 40 per-query sets
    check_layout(P, w.strings[: sets[-1]], sets=sets)


def test_layout_other_terminator(P):
    check_layout(P, [b'say "hi"', b"say", b"s"], term=ord("|"))


def test_layout_needs_host_only_set_handle(P):
    h = P.compile_format([b"0123456789"], [b"1"], flags=P.FLAG_HOST_ONLY)
    with pytest.raises(P.TamError) as e:
        h.layout()
    assert e.value.status == -6
