"""The C ABI without a GPU: symbols, argument checks, and the host trie tables.

``TAM_FLAG_HOST_ONLY`` runs the library's host phase (dedupe, sort, preorder
trie, child tables, vocabulary hash) and no HIP call, so the trie it builds can
be compared with the oracle's on the CPU.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import Oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tam.h")


@pytest.fixture(scope="module")
def P():
    import paper_2608_12574_amd as P
    try:
        P.lib()
    except RuntimeError:
        from paper_2608_12574_amd import build
        build.build()
    return P


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tam_[a-z_]+)\s*\(", src)))


def test_header_symbols_exported(P):
    names = declared_functions()
    assert "tam_compile" in names and "tam_apply_mask" in names and "tam_advance" in names
    L = ctypes.CDLL(P.tam.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(P.tam.ENTRY_POINTS)


def host(P, strings, vocab, sets=None, terminator=0x22):
    return P.compile(strings, vocab, sets=sets, terminator=terminator, flags=P.FLAG_HOST_ONLY)


def same_trie(h, o):
    assert h.num_nodes == o.N
    assert np.array_equal(h.roots, o.roots)
    assert np.array_equal(h.parent, o.parent)
    assert np.array_equal(h.depth, o.depth)
    assert np.array_equal(h.edge_byte, o.edge)
    assert np.array_equal(h.is_final, o.is_final)


def test_host_trie_worked_example(P):
    strings = [b"medical_billing", b"medical_coding", b"medical_records"]
    vocab = [b"medical", b"_bill", b"_cod", b"_rec", b"ing", b"ords"]
    h = host(P, strings, vocab)
    same_trie(h, Oracle(strings, vocab))
    assert h.num_nodes == 32 and h.words_per_row == 1 and h.max_token_len == 7


@pytest.mark.parametrize("name,strings,vocab", W.edge_cases(), ids=[e[0] for e in W.edge_cases()])
def test_host_trie_edge_suite(P, name, strings, vocab):
    h = host(P, strings, vocab)
    o = Oracle(strings, vocab)
    same_trie(h, o)
    assert h.num_strings == len(set(strings))


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_host_trie_configs(P, cid):
    w = W.config(cid)
    h = host(P, w.strings, w.vocab)
    same_trie(h, Oracle(w.strings, [b"x"]))
    assert h.vocab_size == w.V and h.words_per_row == (w.V + 63) // 64


def test_host_trie_forest(P):
    w = W.config(5)
    sets = w.set_offsets[:33]  # the first 32 sets
    strings = w.strings[: sets[-1]]
    h = host(P, strings, [b"x"], sets=sets)
    same_trie(h, Oracle(strings, [b"x"], set_offsets=sets))
    assert h.num_sets == 32


def test_host_only_vocabulary_reuse(P):
    w = W.config(1)
    voc = P.Vocab(w.vocab, host_only=True)
    h1 = P.compile(w.strings, voc, flags=P.FLAG_HOST_ONLY)
    h2 = P.compile(w.strings[:40], voc, flags=P.FLAG_HOST_ONLY)
    voc.close()
    same_trie(h1, Oracle(w.strings, [b"x"]))
    same_trie(h2, Oracle(w.strings[:40], [b"x"]))
    assert h1.vocab_size == w.V and h1.max_token_len == max(len(t) for t in w.vocab)
    h1.close()
    h2.close()


def test_other_terminator(P):
    strings = [b'say "hi"', b"say"]
    h = host(P, strings, [b"a"], terminator=ord("|"))
    same_trie(h, Oracle(strings, [b"a"], terminator=ord("|")))


def raw_compile(P, sb, so, K, tb, to, V, set_off=None, S=0, terminator=0x22, flags=1):
    L = P.lib()
    opt = P.tam.Options(terminator, flags)
    out = ctypes.c_void_p()
    p = lambda a: None if a is None else ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    rc = L.tam_compile(p(sb), p(so), K, p(tb), p(to), V, p(set_off), S, ctypes.byref(opt), None, None,
                       ctypes.byref(out))
    if rc == 0:
        L.tam_destroy(out)
    return rc, L.tam_last_error().decode()


def test_error_paths(P):
    sb, so = P.tam.csr([b"ab", b"cd"])
    tb, to = P.tam.csr([b"a", b"b"])
    assert raw_compile(P, sb, so, 2, tb, to, 2)[0] == 0
    assert raw_compile(P, sb, so, 0, tb, to, 2)[0] == -1                      # K = 0
    assert raw_compile(P, sb, so, 2, tb, to, 0)[0] == -1                      # V = 0
    assert raw_compile(P, sb, None, 2, tb, to, 2)[0] == -1                    # null offsets
    bad = so.copy()
    bad[1] = 5
    bad[2] = 4
    assert raw_compile(P, sb, bad, 2, tb, to, 2)[0] == -1                     # decreasing offsets
    assert raw_compile(P, sb, so, 2, tb, to, 2, terminator=300)[0] == -1      # not a byte
    rc, msg = raw_compile(P, sb, so, 2, tb, to, 2, terminator=ord("c"))
    assert rc == -2 and "string 1" in msg                                     # terminator inside
    sets = np.array([0, 2, 2], dtype=np.int64)
    assert raw_compile(P, sb, so, 2, tb, to, 2, set_off=sets, S=2)[0] == -1   # empty set
    sets = np.array([0, 1], dtype=np.int64)
    assert raw_compile(P, sb, so, 2, tb, to, 2, set_off=sets, S=1)[0] == -1   # does not end at K


def test_vocab_error_paths(P):
    L = P.lib()
    out = ctypes.c_void_p()
    tb, to = P.tam.csr([b"a", b"b"])
    p = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    assert L.tam_vocab_create(p(tb), p(to), 0, 1, None, None, ctypes.byref(out)) == -1
    assert L.tam_vocab_create(p(tb), None, 2, 1, None, None, ctypes.byref(out)) == -1
    assert L.tam_vocab_create(p(tb), p(to), 2, 1, None, None, None) == -1
    assert L.tam_vocab_create(p(tb), p(to), 2, 1, None, None, ctypes.byref(out)) == 0
    sb, so = P.tam.csr([b"ab"])
    h = ctypes.c_void_p()
    # a device compile against a host-only vocabulary is refused before any HIP call
    opt = P.tam.Options(0x22, 0)
    assert L.tam_compile_vocab(p(sb), p(so), 1, out, None, 0, ctypes.byref(opt), None, None,
                               ctypes.byref(h)) == -6
    assert L.tam_compile_vocab(p(sb), p(so), 1, None, None, 0, ctypes.byref(opt), None, None,
                               ctypes.byref(h)) == -1
    L.tam_vocab_destroy(out)
    L.tam_vocab_destroy(None)


def test_host_only_handle_refuses_device_work(P):
    h = host(P, [b"ab"], [b"a"])
    with pytest.raises(P.TamError) as e:
        h.rebuild()
    assert e.value.status == -6
    L = P.lib()
    assert L.tam_rebuild(h._raw, 0, None) == -6
    assert L.tam_apply_mask(h._raw, None, 0, None, 0, 1, None) == -6
    assert L.tam_advance(h._raw, None, None, 0, None, None) == -6
    assert L.tam_export_rows(h._raw, None, 0, None, None) == -6
    h.close()
    h.close()


def test_missing_library_fails_loudly(P, monkeypatch):
    import paper_2608_12574_amd.tam as T
    monkeypatch.setattr(T, "_lib", None)
    monkeypatch.setattr(T, "LIB_PATH", "/nonexistent/libtam.so")
    with pytest.raises(RuntimeError, match="no fallback"):
        T.lib()


def _branching(o):
    cnt = o.is_final.astype(np.int64)
    for n in range(o.N - 1, 0, -1):
        if o.parent[n] >= 0:
            cnt[o.parent[n]] += cnt[n]
    return cnt >= 2


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_tail_split_host_only(P, oracle_mod, cid):
    """Tail compression keeps dense rows for exactly the nodes with two or more
    final nodes below them, numbered in id order (host tables, no GPU)."""
    w = W.config(cid)
    o = oracle_mod.Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY | P.FLAG_TAIL_LISTS)
    branch = _branching(o)
    assert h.dense_rows == int(branch.sum())
    assert np.array_equal(h.dense_row >= 0, branch)
    assert np.array_equal(h.dense_row[branch], np.arange(h.dense_rows))
    # a tail stores how many nodes lie below it on its path
    size = np.ones(o.N, dtype=np.int64)
    for n in range(o.N - 1, 0, -1):
        size[o.parent[n]] += size[n]
    assert np.array_equal(-1 - h.dense_row[~branch], size[~branch] - 1)
    full = P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY)
    assert full.dense_row is None and full.dense_rows == o.N
    # without a table the split is the same, the branching nodes keeping lists
    lists = P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY | P.FLAG_NO_TABLE | P.FLAG_TAIL_LISTS)
    assert lists.dense_rows == 0 and np.array_equal(lists.dense_row, h.dense_row)
    assert P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY | P.FLAG_NO_TABLE).dense_row is None


def test_tail_split_forest_host_only(P, oracle_mod):
    sets = [[b"ab", b"a"], [b""], [b"ba", b"bb", b"b"], [b"abc"]]
    flat = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    vocab = [b"a", b"b", b"c", b'"']
    o = oracle_mod.Oracle(flat, vocab, set_offsets=offs)
    h = P.compile(flat, vocab, sets=offs, flags=P.FLAG_HOST_ONLY | P.FLAG_TAIL_LISTS)
    assert np.array_equal(h.dense_row >= 0, _branching(o))


def test_host_trie_forest_with_large_set(P):
    """A large set (built in parts cut by first byte) among small ones."""
    strings, vocab, offs = W.mixed_forest()
    h = host(P, strings, vocab, sets=offs)
    same_trie(h, Oracle(strings, [b"x"], set_offsets=offs))
    assert h.num_strings == sum(len(set(strings[offs[j]:offs[j + 1]])) for j in range(len(offs) - 1))


def test_format_host_tables_and_errors(P):
    """tam_compile_format on the host: positions 0..L+1 as a chain, the final
    node last; classes admitting the terminator and empty formats are refused."""
    classes = W.formats()["YYYY-MM-DD"]
    h = P.compile_format(classes, [b"1", b"-", b'"'], flags=P.FLAG_HOST_ONLY)
    L = len(classes)
    assert h.num_nodes == L + 2 and h.num_sets == 1 and h.num_strings == 0
    assert np.array_equal(h.roots, [0])
    assert np.array_equal(h.parent, np.arange(-1, L + 1))
    assert np.array_equal(h.depth, np.arange(L + 2))
    assert np.array_equal(h.is_final, [0] * (L + 1) + [1])
    assert h.dense_rows == L + 2 and h.dense_row is None
    with pytest.raises(P.TamError) as e:
        P.compile_format([b"0", b'9"'], [b"1"], flags=P.FLAG_HOST_ONLY)
    assert e.value.status == -2
    with pytest.raises(P.TamError) as e:
        P.compile_format([], [b"1"], flags=P.FLAG_HOST_ONLY)
    assert e.value.status == -1
    h2 = P.compile_format([b"ab|"], [b"a"], terminator=ord('"'), flags=P.FLAG_HOST_ONLY)  # '|' is a plain byte here
    assert h2.num_nodes == 3
    with pytest.raises(P.TamError):
        P.compile_format([b"ab|"], [b"a"], terminator=ord("|"), flags=P.FLAG_HOST_ONLY)


def test_packed_strings_input(P):
    """compile() takes the strings as a packed (blob, offsets) pair as well."""
    from paper_2608_12574_amd.tam import csr
    w = W.config(2)
    h1 = host(P, w.strings, w.vocab)
    h2 = host(P, csr(w.strings), w.vocab)
    assert h1.num_nodes == h2.num_nodes
    assert np.array_equal(h1.parent, h2.parent) and np.array_equal(h1.edge_byte, h2.edge_byte)


def _subtree_sizes(o):
    size = np.ones(o.N, dtype=np.int64)
    for n in range(o.N - 1, 0, -1):
        if o.parent[n] >= 0:
            size[o.parent[n]] += size[n]
    return size


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_subtree_end_host_only(P, oracle_mod, cid):
    """Rows built on demand scan a node's subtree as the preorder id range
    [n, subtree_end[n]): it must equal n plus the subtree's size, counted from
    the oracle's parent links."""
    w = W.config(cid)
    o = oracle_mod.Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY | P.FLAG_LAZY_ROWS)
    assert np.array_equal(h.subtree_end, np.arange(o.N) + _subtree_sizes(o))
    assert h.cache_rows == min(4096, o.N) and h.dense_rows == 0
    assert P.compile(w.strings, w.vocab, flags=P.FLAG_HOST_ONLY).subtree_end is None


def test_subtree_end_forest_and_edges(P, oracle_mod):
    strings, vocab, offs = W.mixed_forest()
    o = oracle_mod.Oracle(strings, [b"x"], set_offsets=offs)
    h = P.compile(strings, vocab, sets=offs, flags=P.FLAG_HOST_ONLY | P.FLAG_LAZY_ROWS, cache_rows=7)
    assert np.array_equal(h.subtree_end, np.arange(o.N) + _subtree_sizes(o))
    assert h.cache_rows == 7
    for name, st, voc in W.edge_cases():
        o = oracle_mod.Oracle(st, voc)
        h = P.compile(st, voc, flags=P.FLAG_HOST_ONLY | P.FLAG_LAZY_ROWS, cache_rows=10 ** 9)
        assert np.array_equal(h.subtree_end, np.arange(o.N) + _subtree_sizes(o)), name
        assert h.cache_rows == o.N, name


def test_lazy_rows_option_errors(P):
    with pytest.raises(P.TamError) as e:
        P.compile([b"ab"], [b"a"], flags=P.FLAG_HOST_ONLY | P.FLAG_LAZY_ROWS, cache_rows=-1)
    assert e.value.status == -1
    h = P.compile([b"ab"], [b"a"], flags=P.FLAG_HOST_ONLY | P.FLAG_LAZY_ROWS)
    L = P.lib()
    assert L.tam_rebuild(h._raw, 0, None) == -6  # host only: no device state
    h.close()


def _trie_digest(h):
    return tuple(np.asarray(a).tobytes() for a in (h.roots, h.parent, h.depth, h.edge_byte, h.is_final))


def test_host_compiles_on_several_threads(P):
    """Host compiles from several host threads at once: one runs its parallel
    loops on the worker pool, the others on threads of their own; every trie
    equals the one built alone."""
    import threading
    w = W.config(3)
    ref = _trie_digest(host(P, w.strings, [b"x"]))
    out, errors = {}, []

    def run(k):
        try:
            for r in range(3):
                out[(k, r)] = _trie_digest(host(P, w.strings, [b"x"]))
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(e)

    ts = [threading.Thread(target=run, args=(k,)) for k in range(4)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=120)
    assert not errors and not any(t.is_alive() for t in ts)
    assert len(out) == 12 and all(v == ref for v in out.values())


def _child_compile(q):
    import paper_2608_12574_amd as P2
    w = W.config(3)
    q.put(_trie_digest(P2.compile(w.strings, [b"x"], flags=P2.FLAG_HOST_ONLY)))


def test_host_compile_in_forked_child(P):
    """A child forked after the parent's worker pool exists builds the same
    trie (it starts a pool of its own)."""
    import multiprocessing as mp
    w = W.config(3)  # large enough to be built in parts, on the pool
    ref = _trie_digest(host(P, w.strings, [b"x"]))
    ctx = mp.get_context("fork")
    q = ctx.Queue()
    p = ctx.Process(target=_child_compile, args=(q,))
    p.start()
    got = q.get(timeout=120)
    p.join(timeout=60)
    assert p.exitcode == 0 and got == ref


def test_argument_errors_before_state(P):
    """Argument errors of the serving calls are TAM_E_INVAL, reported before the
    handle's state (a host-only handle would be TAM_E_STATE): an unsupported
    dtype, a row stride below V, logits not aligned to their element, null
    pointers with rows to process, negative sizes, a misaligned export."""
    h = host(P, [b"ab", b"ac"], [b"a", b"b", b"c"])  # V = 3
    L = P.lib()
    fake = ctypes.c_void_p(0x10000)             # never dereferenced: the checks come first
    odd = ctypes.c_void_p(0x10001)
    assert L.tam_apply_mask(h._raw, fake, 4, fake, 2, 3, None) == -1      # dtype 2
    assert L.tam_apply_mask(h._raw, fake, 4, fake, -1, 3, None) == -1     # dtype -1
    assert L.tam_apply_mask(h._raw, fake, 4, fake, 1, 2, None) == -1      # row_stride < V
    assert L.tam_apply_mask(h._raw, fake, 4, odd, 1, 3, None) == -1       # bf16 at an odd address
    assert L.tam_apply_mask(h._raw, fake, 4, ctypes.c_void_p(0x10002), 0, 3, None) == -1  # fp32 at 2 mod 4
    assert L.tam_apply_mask(h._raw, None, 4, fake, 1, 3, None) == -1      # null ids
    assert L.tam_apply_mask(h._raw, fake, 4, None, 1, 3, None) == -1      # null logits
    assert L.tam_apply_mask(h._raw, fake, -1, fake, 1, 3, None) == -1     # B < 0
    assert L.tam_apply_mask(None, fake, 4, fake, 1, 3, None) == -1        # null handle
    assert L.tam_apply_mask(h._raw, fake, 4, fake, 1, 3, None) == -6      # valid arguments: the state
    assert L.tam_advance(h._raw, fake, None, 4, fake, None) == -1
    assert L.tam_advance(h._raw, fake, fake, -2, fake, None) == -1
    assert L.tam_advance(h._raw, fake, fake, 4, fake, None) == -6
    assert L.tam_export_rows(h._raw, fake, 4, odd, None) == -1            # out not 8-byte aligned
    assert L.tam_export_rows(h._raw, fake, -1, fake, None) == -1
    assert L.tam_export_rows(h._raw, None, 4, fake, None) == -1
    assert L.tam_export_rows(h._raw, fake, 4, fake, None) == -6
    L.tam_export_rows(h._raw, fake, 4, odd, None)
    assert "aligned" in L.tam_last_error().decode()
    h.close()


def test_token_too_long(P):
    """A token of 65,536 bytes is beyond the 16-bit length field of the
    vocabulary table: TAM_E_TOOLARGE, with no handle made; 65,535 bytes fit."""
    with pytest.raises(P.TamError) as e:
        P.Vocab([b"a", b"b" * 65536], host_only=True)
    assert e.value.status == -5 and "65535" in str(e.value)
    with pytest.raises(P.TamError) as e:
        host(P, [b"ab"], [b"a", b"c" * 70000])
    assert e.value.status == -5
    v = P.Vocab([b"a", b"b" * 65535], host_only=True)
    h = P.compile([b"ab"], v, flags=P.FLAG_HOST_ONLY)
    assert h.max_token_len == 65535
    h.close()
    v.close()


def test_duplicate_token_limit(P):
    """More than 65,535 ids sharing one byte string: TAM_E_TOOLARGE."""
    with pytest.raises(P.TamError) as e:
        P.Vocab([b"q"] * 65536 + [b"r"], host_only=True)
    assert e.value.status == -5
    v = P.Vocab([b"q"] * 65535 + [b"r"], host_only=True)
    v.close()


def test_format_rows_noalloc_argument_errors(P):
    """tam_format_rows_noalloc checks its arguments before touching a device:
    L beyond the static scratch (TAM_NOALLOC_MAX_POSITIONS = 1024) or below 1,
    a class admitting the terminator, a short output stride, a host-only
    vocabulary."""
    L = P.lib()
    voc = P.Vocab([b"1", b"12", b"-"], host_only=True)
    fake = ctypes.c_void_p(0x10000)

    def call(classes, n, term=0x22, stride=1, out=fake, pairs=None):
        rows = np.ascontiguousarray(P.tam.format_class_rows(classes)) if classes else np.zeros((1, 32), np.uint8)
        return L.tam_format_rows_noalloc(ctypes.c_void_p(rows.ctypes.data), n, term, voc._raw, out, stride,
                                         pairs, None)

    assert call([b"0"] * 1025, 1025) == -1
    assert "1024" in L.tam_last_error().decode()
    assert call([b"0"], 0) == -1
    assert call([b"0"], 1, term=256) == -1
    assert call([b"0"], 1, stride=0) == -1
    assert call([b"0"], 1, out=ctypes.c_void_p(0x10004)) == -1
    assert call([b"0"], 1, pairs=ctypes.c_void_p(0x10004)) == -1
    assert call([b'0"'], 1) == -2
    assert call([b"0"] * 1024, 1024) == -6  # valid arguments: a host-only vocabulary has no device tables
    voc.close()


def _list_bound(P, h, vocab, flags):
    """The list capacity by its per-node definition: node m can end at most one
    distinct token string of each length d <= min(depth(m), max_len), which
    lands in a list according to the representation (all lengths for plain
    lists; with tail compression, lengths above the window on tail ancestors
    (d <= tail_span) and, without a table, every length on branching
    ancestors (d > tail_span)); each length counts the largest number of ids
    sharing one string of that length."""
    L = max(len(t) for t in vocab)
    dup = np.zeros(L + 1, dtype=np.int64)
    counts = {}
    for t in vocab:
        if t:
            counts[t] = counts.get(t, 0) + 1
    for t, c in counts.items():
        dup[len(t)] = max(dup[len(t)], c)
    cum = np.cumsum(dup)  # cum[d]: sum over lengths <= d (dup[0] = 0)
    depth = h.depth.astype(np.int64)
    all_ = np.minimum(depth, L)
    if not flags & P.FLAG_TAIL_LISTS:
        return int(cum[all_].sum())
    row, parent = h.dense_row, h.parent
    span = np.zeros(h.num_nodes, dtype=np.int64)  # tail ancestors of each node
    for m in range(h.num_nodes):  # preorder: a parent precedes its children
        p = parent[m]
        if row[m] < 0 and p >= 0 and row[p] < 0:
            span[m] = span[p] + 1
    sc = np.minimum(span, L)
    win = cum[np.minimum(sc, 16)]
    if flags & P.FLAG_NO_TABLE:
        return int((cum[all_] - win).sum())
    return int((cum[sc] - win).sum())


@pytest.mark.parametrize("flags", [2, 2 | 8, 8], ids=["lists", "tail_lists", "tail_long"])  # NO_TABLE, TAIL_LISTS
def test_list_capacity_matches_per_node_bound(P, flags):
    """The list capacity (computed per string in closed form) equals the
    per-node bound, on one set, a forest, and a vocabulary with tokens longer
    than the probe window (so that tail compression with a table keeps lists)."""
    w1, w5 = W.config(1), W.config(5)
    rng = np.random.default_rng(5)
    longs = []
    for s in w1.strings[:60]:
        if len(s) >= 18:
            a = int(rng.integers(0, len(s) - 17))
            longs.append(s[a:a + int(rng.integers(17, min(len(s) - a, 30) + 1))])
    vocab = list(w1.vocab[:3000]) + longs + longs[:5]  # duplicates of long strings too
    assert max(len(t) for t in vocab) > 16
    offs = [int(x) for x in w5.set_offsets[:7]]
    cases = [(w1.strings, None), (w5.strings[:offs[-1]], offs)]
    for strings, sets in cases:
        h = P.compile(strings, vocab, sets=sets, flags=flags | P.FLAG_HOST_ONLY)
        assert h.list_capacity == _list_bound(P, h, vocab, flags), (flags, sets is not None)
        h.close()
    # no lists without long tokens under tail compression with a table
    h = P.compile(w1.strings, w1.vocab[:3000], flags=P.FLAG_TAIL_LISTS | P.FLAG_HOST_ONLY)
    assert h.list_capacity == 0
