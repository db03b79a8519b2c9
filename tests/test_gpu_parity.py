"""GPU parity: the HIP path against the oracle, bit for bit.

Masks, advanced states and masked logits are integers / raw bit patterns, so
every comparison here is exact.  Small cases compare every row and every
(node, token) advance; the full-size configurations compare sampled rows (the
root, every depth-1 node, random nodes, the last node), every row visited by
the decode loops, and whole-table properties that hold at any size.
"""
import numpy as np
import pytest

import workloads as W
from oracle import Oracle
from oracle.brute import Brute

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_12574_amd as P
    P.lib()  # fails loudly when the library is missing
    return P


def rows_np(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint64)


def gpu_rows(h, nodes):
    ids = torch.as_tensor(np.asarray(nodes, dtype=np.int32), device="cuda")
    return rows_np(h.export_rows(ids))


def gpu_advance(h, nodes, toks):
    n = torch.as_tensor(np.asarray(nodes, dtype=np.int32), device="cuda")
    t = torch.as_tensor(np.asarray(toks, dtype=np.int32), device="cuda")
    return h.advance(n, t).cpu().numpy()


def bits_of(x):
    return x.view(torch.int16 if x.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


def host_logits(B, cols, dtype, seed):
    rng = np.random.default_rng(seed)
    x = torch.from_numpy(rng.standard_normal((B, cols), dtype=np.float32))
    flat = x.view(-1)
    k = min(flat.numel(), 256)
    idx = torch.from_numpy(rng.choice(flat.numel(), size=k, replace=False))
    flat[idx] = torch.tensor([float("nan"), -0.0, 0.0, float("inf"), 1e-40, -1e-40, 3e38, -5.0] * 32)[:k]
    return x.to(torch.bfloat16) if dtype == "bf16" else x


def check_apply(P, h, o, nodes, dtype, cols=None, seed=0, stride=None):
    """GPU apply vs the oracle's apply on the same bits (optionally padded rows)."""
    B = len(nodes)
    cols = cols or o.V
    x = host_logits(B, cols, dtype, seed)
    if stride is not None and stride != cols:
        big = torch.zeros((B, stride), dtype=x.dtype)
        big[:, :cols] = x
        dev = big.cuda()[:, :cols]
    else:
        dev = x.cuda()
    ids = torch.as_tensor(np.asarray(nodes, dtype=np.int32), device="cuda")
    h.apply_mask(ids, dev)
    got = bits_of(dev)
    ref_bits = bits_of(x)
    exp = o.apply(np.asarray(nodes, dtype=np.int32),
                  ref_bits.view(np.uint16 if dtype == "bf16" else np.uint32), 1 if dtype == "bf16" else 0)
    assert np.array_equal(got.view(exp.dtype), exp)


# ----------------------------------------------------------- small / exact --

def full_check(P, strings, vocab, sets=None, flags=0, terminator=0x22):
    o = Oracle(strings, vocab, set_offsets=sets, terminator=terminator)
    h = P.compile(strings, vocab, sets=sets, flags=flags, terminator=terminator)
    assert h.num_nodes == o.N
    assert np.array_equal(h.roots, o.roots)
    nodes = np.arange(-2, o.N + 2)
    assert np.array_equal(gpu_rows(h, nodes), np.concatenate(
        [np.zeros((2, o.W), np.uint64), o.mask_rows(np.arange(o.N)), np.zeros((2, o.W), np.uint64)]))
    if not flags & LAZY:
        cnt = h.valid_counts(torch.as_tensor(nodes.astype(np.int32), device="cuda")).cpu().numpy()
        assert np.array_equal(cnt[2:-2], np.unpackbits(o.mask_rows(np.arange(o.N)).view(np.uint8), axis=1).sum(1))
        assert not cnt[:2].any() and not cnt[-2:].any()
    nn, tt = np.meshgrid(nodes, np.arange(-1, o.V + 1), indexing="ij")
    assert np.array_equal(gpu_advance(h, nn.ravel(), tt.ravel()), o.advance(nn.ravel(), tt.ravel()))
    for dtype in ("fp32", "bf16"):
        check_apply(P, h, o, nodes, dtype, seed=len(nodes))
    return h, o


# the representations: full dense table, lists only, tail compression (dense
# rows for the branching nodes), tail compression without a table (lists for
# the branching nodes), rows built on demand into a row cache
LAZY = 16
TAIL_LISTS = 2 | 8
FLAGS = [0, 2, 8, TAIL_LISTS, LAZY]
FLAG_IDS = ["dense", "no_table", "tail", "tail_lists", "lazy"]


def branching_nodes(o: Oracle) -> np.ndarray:
    """Nodes with two or more final nodes below them (independent of the library)."""
    cnt = o.is_final.astype(np.int64)
    par = o.parent
    for n in range(o.N - 1, 0, -1):
        if par[n] >= 0:
            cnt[par[n]] += cnt[n]
    return cnt >= 2


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_worked_example(P, flags):
    vocab = [b"medical", b"_bill", b"_cod", b"_rec", b"ing", b"ords", b'"']
    h, o = full_check(P, [b"medical_billing", b"medical_coding", b"medical_records"], vocab, flags=flags)
    if flags != LAZY:  # rows built on demand have no pass over all nodes to count
        assert h.valid_pairs() == 10  # rows 0,7,12,19,26 (1+3+1+1+1) + '"' at 15,22,30
    rows = gpu_rows(h, [0, 7, 12, 19, 26])
    assert [int(r[0]) for r in rows] == [1, 0b1110, 0b10000, 0b10000, 0b100000]


@pytest.mark.parametrize("name,strings,vocab", W.edge_cases(), ids=[e[0] for e in W.edge_cases()])
def test_edge_suite(P, name, strings, vocab):
    for flags in FLAGS:
        full_check(P, strings, vocab, flags=flags)


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_tiny_random_sets(P, flags):
    rng = np.random.default_rng(123)
    alphabet = np.frombuffer(b'ab"\x80', dtype=np.uint8)
    vocab = [b""] + [bytes(alphabet[rng.integers(0, 4, size=rng.integers(1, 5))]) for _ in range(150)]
    for trial in range(12):
        strings = [bytes(alphabet[rng.integers(0, 2, size=rng.integers(0, 7))]).replace(b'"', b"a")
                   for _ in range(rng.integers(1, 7))]
        h, o = full_check(P, strings, vocab, flags=flags)
        if flags & 8:
            assert np.array_equal(h.dense_row >= 0, branching_nodes(o))
        b = Brute(strings, vocab)
        for n in range(o.N):
            got = np.unpackbits(gpu_rows(h, [n])[0].view(np.uint8), bitorder="little")[: len(vocab)]
            assert set(np.flatnonzero(got).tolist()) == b.valid_set(n)


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_apply_batch_beyond_one_launch(P, flags):
    """A batch larger than one launch's row limit (65,535 row groups; three
    rows per block for dense-table rows here): every representation splits it
    into several launches, and the fp32 batch ends exactly on a launch
    boundary.  Dead and out-of-range rows are spread over it."""
    rng = np.random.default_rng(77)
    words = [b"get_", b"list_", b"item", b"user", b"s", b"_id"]
    strings = sorted({b"".join(words[i] for i in rng.integers(0, 6, size=rng.integers(1, 4))) for _ in range(40)})
    vocab = [bytes([c]) for c in range(256)] + words + [b"get", b"list", b"er", b'"']
    o = Oracle(strings, vocab)
    h = P.compile(strings, vocab, flags=flags)
    B = 3 * 65535 + 3
    nodes = rng.integers(0, o.N, size=B).astype(np.int32)
    nodes[::1009] = -1
    nodes[5::2003] = o.N
    check_apply(P, h, o, nodes, "bf16", seed=1)
    check_apply(P, h, o, nodes[: 65535 * 3], "fp32", seed=2)
    h.close()


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_random_medium_sets(P, seed):
    """Seeded random sets and vocabularies over a small alphabet: heavy prefix
    sharing, tokens of 1-20 bytes that may hold the terminator, duplicate and
    empty tokens.  Every row, every (node, token) advance and both apply
    dtypes, for every representation."""
    rng = np.random.default_rng(1000 + seed)
    alpha = np.frombuffer(b'abc_"', dtype=np.uint8)

    def rand_bytes(lo, hi, with_terminator):
        n = int(rng.integers(lo, hi + 1))
        return bytes(alpha[rng.integers(0, 5 if with_terminator else 4, size=n)])

    strings = [rand_bytes(0, 24, False) for _ in range(300)]
    vocab = [rand_bytes(1, 20, True) for _ in range(1500)] + [b"", b"a", b"a", b'"']
    for flags in FLAGS:
        full_check(P, strings, vocab, flags=flags)


def test_tiny_forest(P):
    sets = [[b"ab", b"a"], [b""], [b"ba", b"bb", b"b"], [b"abc"]]
    flat = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    vocab = [b"a", b"b", b"c", b'"', b"ab", b"b\"", b"abc\"", b""]
    for flags in FLAGS:
        full_check(P, flat, vocab, sets=offs, flags=flags)


def test_other_terminator_and_high_bytes(P):
    for flags in FLAGS:
        full_check(P, [b'x"y', b"x", b"\xff\x00"], [b"x", b'"', b'"y', b"|", b"y|", b"\xff", b"\x00|"],
                   terminator=ord("|"), flags=flags)


def test_advance_stops_at_a_terminator(P):
    """A token that runs through a string's terminator and on into the bytes
    stored after it in the string blob (the next string's leading 0x00 pad)
    must end dead: the node after the terminator has no children.  The
    terminator falls at every offset of the walk's compare windows."""
    strings = [b"a" * 80, b"b" * 3]
    vocab = [b"\x00", b'"\x00', b"a", b'"']
    for k in range(1, 81):
        vocab += [b"a" * k + b'"' + b"\x00", b"a" * k + b'"', b"a" * k + b'"' + b"\x00b"]
    for flags in FLAGS:
        full_check(P, strings, vocab, flags=flags)


def test_tail_single_string(P):
    """One string: the whole trie is one path, so no node branches (the table
    keeps one unused row) and every row comes from a list."""
    h, o = full_check(P, [b"medical_billing"], [b"med", b"ical", b"_", b"billing", b'"', b"g\"", b"x"], flags=8)
    assert h.dense_rows == 0 and np.array_equal(-1 - h.dense_row, o.N - 1 - np.arange(o.N))


# ------------------------------------------------------------ configurations --

def sample_nodes(o: Oracle, k: int, seed: int):
    rng = np.random.default_rng(seed)
    depth1 = np.flatnonzero(o.depth == 1)
    finals = np.flatnonzero(o.is_final)[:4]
    pick = np.concatenate([o.roots, depth1[:64], rng.integers(0, o.N, size=k), finals, [o.N - 1]])
    return np.unique(pick).astype(np.int32)


_oracles = {}


@pytest.fixture(scope="module", params=[(1, 0), (2, 0), (3, 0), (4, 0), (1, 8), (2, 8), (3, 8), (4, 8),
                                        (2, TAIL_LISTS), (4, TAIL_LISTS),
                                        (1, LAZY), (2, LAZY), (3, LAZY), (4, LAZY)],
                ids=["c1", "c2", "c3", "c4", "c1-tail", "c2-tail", "c3-tail", "c4-tail",
                     "c2-tail_lists", "c4-tail_lists",
                     "c1-lazy", "c2-lazy", "c3-lazy", "c4-lazy"])
def compiled(request, P):
    cid, flags = request.param
    w = W.config(cid)
    if cid not in _oracles:
        _oracles.clear()
        _oracles[cid] = Oracle(w.strings, w.vocab)
    o = _oracles[cid]
    h = P.compile(w.strings, w.vocab, flags=flags)
    yield w, o, h
    h.close()
    torch.cuda.empty_cache()


def test_config_rows(P, compiled):
    w, o, h = compiled
    assert h.num_nodes == o.N
    nodes = np.arange(o.N, dtype=np.int32) if w.config_id == 1 else sample_nodes(o, 96, w.config_id)
    for i in range(0, len(nodes), 512):
        assert np.array_equal(gpu_rows(h, nodes[i:i + 512]), o.mask_rows(nodes[i:i + 512]))


def test_config_table_properties(P, compiled):
    """Whole-table facts at full size: with all 256 byte tokens in the vocabulary,
    a row is empty exactly at final nodes, and padding words stay zero.  With
    tail compression the table holds exactly the branching nodes (none final),
    and the lists and the table together count the full table's pairs."""
    w, o, h = compiled
    if h.flags & (LAZY | 2):
        pytest.skip("no dense table (rows built on demand, or tail compression with lists)")
    R = h.dense_rows
    table = h._alloc.live[h.table_ptr].view(torch.int64)[: R * h.row_stride_words].view(R, h.row_stride_words)
    nonempty = torch.zeros(R, dtype=torch.bool, device="cuda")
    for i in range(0, R, 16384):
        blk = table[i:i + 16384]
        nonempty[i:i + 16384] = blk[:, : h.words_per_row].ne(0).any(dim=1)
        if h.row_stride_words > h.words_per_row:
            assert not blk[:, h.words_per_row:].ne(0).any().item()
    if h.dense_row is None:
        assert R == o.N
        assert np.array_equal(nonempty.cpu().numpy(), o.is_final == 0)
    else:
        branch = branching_nodes(o)
        assert R == int(branch.sum()) and np.array_equal(h.dense_row >= 0, branch)
        assert np.array_equal(h.dense_row[branch], np.arange(R))
        assert nonempty.all().item()
        if w.config_id >= 3:
            hf = P.compile(w.strings, w.vocab)
            assert h.valid_pairs() == hf.valid_pairs()
            hf.close()
    if w.config_id <= 2:
        # total number of valid pairs against the oracle's full table
        M = 0
        for i in range(0, o.N, 4096):
            rows = o.mask_rows(np.arange(i, min(o.N, i + 4096), dtype=np.int32))
            M += int(np.unpackbits(rows.view(np.uint8)).sum())
        assert h.valid_pairs() == M


def test_config_rows_vs_advance(P, compiled):
    """mask[n][v] <=> advance(n, v) != dead, on GPU outputs, for sampled nodes."""
    w, o, h = compiled
    nodes = sample_nodes(o, 6, 100 + w.config_id)[:12]
    rows = gpu_rows(h, nodes)
    for r, n in enumerate(nodes):
        adv = gpu_advance(h, np.full(o.V, n), np.arange(o.V))
        bits = np.unpackbits(rows[r].view(np.uint8), bitorder="little")[: o.V].astype(bool)
        assert np.array_equal(adv != -1, bits)
        assert np.array_equal(adv, o.advance(np.full(o.V, n, np.int32), np.arange(o.V, dtype=np.int32)))


def test_config_apply(P, compiled):
    w, o, h = compiled
    if w.node_mode == "uniform":
        nodes = W.uniform_nodes(w.config_id, o.N, w.batch)
    else:
        nodes = np.full(w.batch, 0, np.int32)
    check_apply(P, h, o, nodes, w.dtype, seed=w.config_id)


def test_config_decode(P, compiled):
    """The serving loop: apply the mask, pick a valid token (uniformly, from the
    oracle's row), advance on GPU and oracle; finished rows restart at the root."""
    w, o, h = compiled
    rng = np.random.default_rng([w.config_id, W.ROLE_CHOICE, 2])
    nodes = W.uniform_nodes(w.config_id, o.N, w.batch) if w.node_mode == "uniform" \
        else np.zeros(w.batch, np.int32)
    nodes = np.where(o.is_final[nodes] == 1, 0, nodes).astype(np.int32)
    steps = min(w.decode_steps, 32)
    for step in range(steps):
        rows = o.mask_rows(nodes)
        if step % 8 == 0:
            assert np.array_equal(gpu_rows(h, nodes), rows)
        toks = W.choose_valid_tokens(rng, rows, o.V)
        got = gpu_advance(h, nodes, toks)
        exp = o.advance(nodes, toks)
        assert np.array_equal(got, exp), step
        nodes = np.where(o.is_final[exp] == 1, 0, exp).astype(np.int32)


def test_config_rebuild_identical(P, compiled):
    """Rebuilding (all phases, or marking again without the zero fill) gives the
    same table; the sparse lists built on a dense handle count the same pairs."""
    w, o, h = compiled
    nodes = sample_nodes(o, 32, 7)
    before = gpu_rows(h, nodes)
    if h.flags & LAZY:  # phase 0 empties the row cache; the rows come back the same
        check_apply(P, h, o, nodes, "fp32", seed=8)
        h.rebuild()
        check_apply(P, h, o, nodes, "fp32", seed=9)
        assert np.array_equal(gpu_rows(h, nodes), before)
        for bad in (P.PHASE_MARK, P.PHASE_LISTS, P.PHASE_TABLE):
            with pytest.raises(P.TamError):
                h.rebuild(phases=bad)
        with pytest.raises(P.TamError):
            h.valid_pairs()
        return
    M = h.valid_pairs()
    h.rebuild()
    assert np.array_equal(gpu_rows(h, nodes), before)
    assert h.valid_pairs() == M
    if h.flags & 2:  # tail compression with lists: the lists are its only phase
        for bad in (P.PHASE_MARK, P.PHASE_TABLE):
            with pytest.raises(P.TamError):
                h.rebuild(phases=bad)
        h.rebuild(phases=P.PHASE_LISTS)
        assert np.array_equal(gpu_rows(h, nodes), before)
        assert h.valid_pairs() == M
        h.rebuild(phases=P.PHASE_COUNT)  # the probe pass alone leaves the lists as they are
        assert np.array_equal(gpu_rows(h, nodes), before)
        assert h.valid_pairs() == M
        return
    with pytest.raises(P.TamError):
        h.rebuild(phases=P.PHASE_COUNT)  # no lists (no token is longer than 16 bytes)
    h.rebuild(phases=P.PHASE_MARK)
    assert np.array_equal(gpu_rows(h, nodes), before)
    assert h.valid_pairs() == M
    if h.dense_row is None:
        with pytest.raises(P.TamError):
            h.rebuild(phases=P.PHASE_LISTS)  # lists are kept only without a full table
    else:
        h.rebuild(phases=P.PHASE_TABLE)
        assert np.array_equal(gpu_rows(h, nodes), before)
        assert h.valid_pairs() == M
        with pytest.raises(P.TamError):
            h.rebuild(phases=P.PHASE_LISTS)  # no token is longer than 16 bytes: tails need no lists


def test_host_tables_recycled_between_compiles(P):
    """Device compiles keep their large host tables in pinned blocks that are
    recycled when a handle is destroyed: compiles of other sizes and
    representations that reuse them still give the oracle's trie and rows."""
    w = W.config(3)
    voc = P.Vocab(w.vocab)
    for k, flags in ((10000, 0), (4000, 8), (10000, LAZY), (7000, 2), (9000, 8)):
        strings = w.strings[:k]
        o = Oracle(strings, w.vocab)
        h = P.compile(strings, voc, flags=flags)
        assert h.num_nodes == o.N
        assert np.array_equal(h.parent, o.parent) and np.array_equal(h.depth, o.depth)
        assert np.array_equal(h.edge_byte, o.edge) and np.array_equal(h.is_final, o.is_final)
        nodes = sample_nodes(o, 64, k)
        assert np.array_equal(gpu_rows(h, nodes), o.mask_rows(nodes))
        check_apply(P, h, o, W.uniform_nodes(3, o.N, 32, k), "bf16", seed=k)
        h.close()
    voc.close()


def test_shared_vocabulary(P):
    """One vocabulary, built once, serves several compiles (dense and sparse),
    and outlives its creator's reference through the handles."""
    w = W.config(2)
    voc = P.Vocab(w.vocab)
    o = Oracle(w.strings, w.vocab)
    h1 = P.compile(w.strings, voc, flags=P.FLAG_TAIL_LISTS)
    h2 = P.compile(w.strings[:300], voc, flags=P.FLAG_NO_TABLE)
    h3 = P.compile(w.strings, w.vocab)
    o2 = Oracle(w.strings[:300], w.vocab)
    voc.close()  # the handles keep the vocabulary alive
    nodes = sample_nodes(o, 48, 21)
    assert np.array_equal(gpu_rows(h1, nodes), o.mask_rows(nodes))
    assert np.array_equal(gpu_rows(h3, nodes), o.mask_rows(nodes))
    nodes2 = sample_nodes(o2, 48, 22)
    assert np.array_equal(gpu_rows(h2, nodes2), o2.mask_rows(nodes2))
    assert h1.valid_pairs() == h3.valid_pairs()
    check_apply(P, h2, o2, W.uniform_nodes(2, o2.N, 8), "fp32", seed=9)
    for h in (h1, h2, h3):
        h.close()


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_long_and_duplicate_tokens(P, flags):
    """Tokens longer than the 16-byte probe window and duplicate token strings,
    at scale: sampled rows, a decode loop and both apply dtypes."""
    w = W.stress_case()
    o = Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=flags)
    assert h.max_token_len >= 17
    nodes = sample_nodes(o, 400, 77)
    if flags == 8:  # rows of tails whose path is longer than the window
        tails = np.flatnonzero(h.dense_row <= -18)
        nodes = np.unique(np.concatenate([nodes, tails[:: max(1, len(tails) // 200)]])).astype(np.int32)
    for i in range(0, len(nodes), 256):
        assert np.array_equal(gpu_rows(h, nodes[i:i + 256]), o.mask_rows(nodes[i:i + 256]))
    rows = o.mask_rows(nodes)
    long_ids = np.arange(60000, 62000)
    bits = np.unpackbits(rows.view(np.uint8), axis=1, bitorder="little")[:, : o.V]
    assert bits[:, long_ids].any(), "sample should contain valid long tokens"
    assert bits[:, 62000:].any(), "sample should contain valid duplicate tokens"
    if flags in (0, 8):  # the dense marks (and the tails' lists) and the sparse lists count the same pairs
        hs = P.compile(w.strings, w.vocab, flags=P.FLAG_NO_TABLE)
        assert h.valid_pairs() == hs.valid_pairs()
        hs.close()
    if flags == 8:  # tokens longer than 16 bytes: the tails keep lists for them
        M = h.valid_pairs()
        before = gpu_rows(h, nodes[:256])
        for ph in (P.PHASE_LISTS, P.PHASE_TABLE, P.PHASE_LISTS | P.PHASE_TABLE):
            h.rebuild(phases=ph)
            assert np.array_equal(gpu_rows(h, nodes[:256]), before)
            assert h.valid_pairs() == M
    rng = np.random.default_rng(11)
    cur = W.uniform_nodes(7, o.N, 64)
    for step in range(12):
        r = o.mask_rows(cur)
        assert np.array_equal(gpu_rows(h, cur), r)
        toks = W.choose_valid_tokens(rng, r, o.V)
        exp = o.advance(cur, toks)
        assert np.array_equal(gpu_advance(h, cur, toks), exp)
        cur = np.where((exp < 0) | (o.is_final[np.maximum(exp, 0)] == 1), 0, exp).astype(np.int32)
    check_apply(P, h, o, W.uniform_nodes(7, o.N, 64, 3), "bf16", seed=71)
    check_apply(P, h, o, W.uniform_nodes(7, o.N, 16, 4), "fp32", seed=72)
    h.close()


@pytest.mark.parametrize("cid", [3, 4])
def test_config_every_row(P, cid):
    """Every row of the full table at c3 and c4 against the oracle (its rows
    computed on a pool of host threads, in chunks), and every row of the tail
    compression and rows-built-on-demand handles against the full table's on
    the device: all three representations equal the oracle row for row."""
    import concurrent.futures as cf
    w = W.config(cid)
    o = Oracle(w.strings, w.vocab)
    hf = P.compile(w.strings, w.vocab)
    ht = P.compile(w.strings, w.vocab, flags=8)
    hl = P.compile(w.strings, w.vocab, flags=TAIL_LISTS)
    hz = P.compile(w.strings, w.vocab, flags=LAZY)
    assert hf.num_nodes == o.N
    chunk = 1024
    starts = list(range(0, o.N, chunk))
    with cf.ThreadPoolExecutor(max_workers=16) as pool:  # the oracle's C call releases the GIL
        futs = [pool.submit(o.mask_rows, np.arange(a, min(o.N, a + chunk), dtype=np.int32)) for a in starts]
        for a, f in zip(starts, futs):
            ids = torch.arange(a, min(o.N, a + chunk), dtype=torch.int32, device="cuda")
            full = hf.export_rows(ids)
            assert torch.equal(ht.export_rows(ids), full), a
            assert torch.equal(hl.export_rows(ids), full), a
            assert torch.equal(hz.export_rows(ids), full), a
            exp = f.result()
            assert np.array_equal(rows_np(full), exp), a
            cnt = popcounts(exp)
            assert np.array_equal(hf.valid_counts(ids).cpu().numpy(), cnt), a
            assert np.array_equal(ht.valid_counts(ids).cpu().numpy(), cnt), a
            assert np.array_equal(hl.valid_counts(ids).cpu().numpy(), cnt), a
    assert hf.valid_pairs() == ht.valid_pairs() == hl.valid_pairs()
    for h in (hf, ht, hl, hz):
        h.close()
    torch.cuda.empty_cache()


def popcounts(rows: np.ndarray) -> np.ndarray:
    return np.unpackbits(rows.view(np.uint8), axis=1).sum(axis=1).astype(np.int32)


@pytest.mark.parametrize("cid", [1, 2])
@pytest.mark.parametrize("flags", [0, 2, 8, TAIL_LISTS], ids=["dense", "no_table", "tail", "tail_lists"])
def test_valid_counts_every_node(P, cid, flags):
    """|valid[n]| of every node (and of dead ids) counted on the device equals the
    popcount of the oracle's row; rows built on demand keep no counts."""
    w = W.config(cid)
    o = Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=flags)
    nodes = np.arange(-3, o.N + 3, dtype=np.int32)
    got = h.valid_counts(torch.as_tensor(nodes, device="cuda")).cpu().numpy()
    exp = np.zeros(nodes.size, np.int32)
    for a in range(0, o.N, 2048):
        exp[3 + a:3 + min(o.N, a + 2048)] = popcounts(o.mask_rows(np.arange(a, min(o.N, a + 2048), dtype=np.int32)))
    assert np.array_equal(got, exp)
    assert int(got.sum()) == h.valid_pairs()
    h.close()
    hz = P.compile(w.strings, w.vocab, flags=LAZY)
    with pytest.raises(P.TamError) as e:
        hz.valid_counts(torch.zeros(1, dtype=torch.int32, device="cuda"))
    assert e.value.status == -6
    hz.close()


# ---------------------------------------------------------- sparse / forest --

def test_no_table_matches_dense_c4(P):
    w = W.config(4)
    o = Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=P.FLAG_NO_TABLE)
    assert h.row_stride_words == 0
    nodes = sample_nodes(o, 64, 44)
    assert np.array_equal(gpu_rows(h, nodes), o.mask_rows(nodes))
    check_apply(P, h, o, W.uniform_nodes(4, o.N, 256), "bf16", seed=4)
    check_apply(P, h, o, W.uniform_nodes(4, o.N, 16, 1), "fp32", seed=5)


@pytest.mark.parametrize("flags", [2, 8, TAIL_LISTS, LAZY], ids=["no_table", "tail", "tail_lists", "lazy"])
def test_forest_c5(P, flags):
    """Config 5: 256 per-query sets of 500 strings as one forest (sparse rows,
    tail compression's dense rows for the branching nodes, or rows built on
    demand into a 1024-row cache: 256 new rows per step evict from the fifth
    step on).  The oracle runs on sampled rows and on every row the 16-step
    decode visits."""
    w = W.config(5)
    o = Oracle(w.strings, w.vocab, set_offsets=w.set_offsets)
    h = P.compile(w.strings, w.vocab, sets=w.set_offsets, flags=flags, cache_rows=1024)
    assert h.num_nodes == o.N and np.array_equal(h.roots, o.roots)
    nodes = sample_nodes(o, 64, 55)
    assert np.array_equal(gpu_rows(h, nodes), o.mask_rows(nodes))
    rng = np.random.default_rng([5, W.ROLE_CHOICE, 2])
    cur = o.roots.astype(np.int32).copy()
    for step in range(w.decode_steps):
        rows = o.mask_rows(cur)
        assert np.array_equal(gpu_rows(h, cur), rows)
        if step in (0, 7) or flags == LAZY:
            # roots: long lists (LDS bitmap); later steps: short lists (ballot);
            # both with many mixed chunks, written without a read
            check_apply(P, h, o, cur, "bf16", seed=50 + step)
            check_apply(P, h, o, cur[:32], "fp32", seed=60 + step)
        toks = W.choose_valid_tokens(rng, rows, o.V)
        exp = o.advance(cur, toks)
        assert np.array_equal(gpu_advance(h, cur, toks), exp)
        cur = np.where(o.is_final[exp] == 1, o.roots, exp).astype(np.int32)
    h.close()


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_forest_with_large_set(P, flags):
    """A large set (its host trie built in parts cut by first byte, with the
    empty string and strings that prefix others) among small sets: sampled
    rows, every root's row, and a decode loop in every set."""
    strings, vocab, offs = W.mixed_forest()
    o = Oracle(strings, vocab, set_offsets=offs)
    h = P.compile(strings, vocab, sets=offs, flags=flags)
    assert h.num_nodes == o.N and np.array_equal(h.roots, o.roots)
    nodes = np.unique(np.concatenate([sample_nodes(o, 300, 81), o.roots])).astype(np.int32)
    assert np.array_equal(gpu_rows(h, nodes), o.mask_rows(nodes))
    rng = np.random.default_rng(82)
    start = np.repeat(o.roots, 16).astype(np.int32)
    cur = start.copy()
    for step in range(10):
        rows = o.mask_rows(cur)
        assert np.array_equal(gpu_rows(h, cur), rows)
        toks = W.choose_valid_tokens(rng, rows, o.V)
        exp = o.advance(cur, toks)
        assert np.array_equal(gpu_advance(h, cur, toks), exp)
        cur = np.where((exp < 0) | (o.is_final[np.maximum(exp, 0)] == 1), start, exp).astype(np.int32)
    check_apply(P, h, o, cur, "bf16", seed=83)
    h.close()


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_forest_written_in_groups(P, flags):
    """A forest of 14 sets (8 or more: the host writes it in four groups of
    sets and each group is uploaded while the next is written): the mixed
    forest's sets (a large set cut by first byte, a one-string set) after ten
    of c5's per-query sets, over the c1 vocabulary.  Every root's row, sampled
    rows, the whole rows of the last set's nodes, and a decode in every set."""
    w5 = W.config(5)
    mixed, vocab, moffs = W.mixed_forest()
    sets = [w5.strings[int(w5.set_offsets[j]):int(w5.set_offsets[j + 1])] for j in range(10)]
    sets += [mixed[int(moffs[j]):int(moffs[j + 1])] for j in range(len(moffs) - 1)]
    strings = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    o = Oracle(strings, vocab, set_offsets=offs)
    h = P.compile(strings, vocab, sets=offs, flags=flags)
    assert h.num_nodes == o.N and np.array_equal(h.roots, o.roots)
    last = np.arange(o.roots[-1], o.N, dtype=np.int32)
    nodes = np.unique(np.concatenate([sample_nodes(o, 2000, 91), o.roots, last])).astype(np.int32)
    exp_rows = o.mask_rows(nodes)
    assert np.array_equal(gpu_rows(h, nodes), exp_rows)
    if flags & 2:  # the lists' capacity: summed per group (device) or over all strings (host only)
        hh = P.compile(strings, vocab, sets=offs, flags=flags | P.FLAG_HOST_ONLY)
        assert h.list_capacity == hh.list_capacity > 0
        hh.close()
    if not flags & LAZY:  # counts, and the device phases run again over the groups' grid
        cnt = popcounts(exp_rows)
        assert np.array_equal(h.valid_counts(torch.as_tensor(nodes, device="cuda")).cpu().numpy(), cnt)
        M = h.valid_pairs()
        h.rebuild()
        assert np.array_equal(gpu_rows(h, nodes), exp_rows)
        assert np.array_equal(h.valid_counts(torch.as_tensor(nodes, device="cuda")).cpu().numpy(), cnt)
        assert h.valid_pairs() == M
    rng = np.random.default_rng(92)
    start = np.repeat(o.roots, 8).astype(np.int32)
    cur = start.copy()
    for step in range(8):
        rows = o.mask_rows(cur)
        assert np.array_equal(gpu_rows(h, cur), rows)
        toks = W.choose_valid_tokens(rng, rows, o.V)
        exp = o.advance(cur, toks)
        assert np.array_equal(gpu_advance(h, cur, toks), exp)
        cur = np.where((exp < 0) | (o.is_final[np.maximum(exp, 0)] == 1), start, exp).astype(np.int32)
    check_apply(P, h, o, cur, "bf16", seed=93)
    check_apply(P, h, o, nodes[:500], "fp32", seed=94)
    h.close()


@pytest.mark.parametrize("flags", [2, TAIL_LISTS], ids=["no_table", "tail_lists"])
def test_lists_over_many_scan_blocks(P, flags):
    """Four copies of c5's 256 sets as one forest of 1,024 sets (21.9 M nodes:
    the lists' offsets are scanned over more block sums than one block adds
    up, so the scan's middle pass runs).  Copy k's nodes are copy 0's shifted
    by k * N0, so each holds the same rows and counts, and the valid pairs are
    four times the single copy's; copy 0's rows are the oracle's (sampled, the
    last nodes of every copy included)."""
    import torch
    w = W.config(5)
    K = len(w.strings)
    offs = np.asarray(w.set_offsets, dtype=np.int64)
    offs4 = np.concatenate([offs[:-1] + k * K for k in range(4)] + [np.array([4 * K])])
    h1 = P.compile(w.strings, w.vocab, sets=offs, flags=flags)
    h4 = P.compile(w.strings * 4, w.vocab, sets=offs4, flags=flags)
    N0 = h1.num_nodes
    assert h4.num_nodes == 4 * N0 and 4 * N0 > 4096 * 4096
    assert h4.valid_pairs() == 4 * h1.valid_pairs()
    assert h4.list_capacity == 4 * h1.list_capacity
    rng = np.random.default_rng(95)
    nodes = np.unique(np.concatenate([rng.integers(0, N0, 1500), np.arange(N0 - 300, N0)])).astype(np.int32)
    o = Oracle(w.strings, w.vocab, set_offsets=w.set_offsets)
    rows = o.mask_rows(nodes)
    cnt = popcounts(rows)
    for k in range(4):
        ids = (nodes + k * N0).astype(np.int32)
        assert np.array_equal(gpu_rows(h4, ids), rows), k
        assert np.array_equal(h4.valid_counts(torch.as_tensor(ids, device="cuda")).cpu().numpy(), cnt), k
    h1.close()
    h4.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("flags", [2, TAIL_LISTS], ids=["no_table", "tail_lists"])
def test_graph_capture_replays_forest_groups(P, flags):
    """A forest written in four groups (fourteen sets), captured in a HIP graph:
    rebuild (for tail compression without a table, the probe pass over the
    groups' table in one launch, the scan and the records' fill), apply and
    advance; every replay, with eager rebuilds between replays, gives the
    oracle's rows, masked logits and states."""
    import torch
    w5 = W.config(5)
    mixed, vocab, moffs = W.mixed_forest()
    sets = [w5.strings[int(w5.set_offsets[j]):int(w5.set_offsets[j + 1])] for j in range(10)]
    sets += [mixed[int(moffs[j]):int(moffs[j + 1])] for j in range(len(moffs) - 1)]
    strings = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    o = Oracle(strings, vocab, set_offsets=offs)
    h = P.compile(strings, vocab, sets=offs, flags=flags)
    B, V = 96, len(vocab)
    nodes = np.unique(np.concatenate([o.roots, sample_nodes(o, 200, 96)])).astype(np.int32)[:B]
    B = len(nodes)
    ids = torch.as_tensor(nodes, device="cuda")
    src = torch.as_tensor(host_logits(B, V, "fp32", seed=97).numpy(), device="cuda")
    toks_np = W.choose_valid_tokens(np.random.default_rng(98), o.mask_rows(nodes), V)
    toks = torch.as_tensor(toks_np, device="cuda")
    x = src.clone()
    out = torch.empty_like(ids)
    exp_x = o.apply(nodes, bits_of(src.cpu()).view(np.uint32), 0)
    exp_out = o.advance(nodes, toks_np)
    M = h.valid_pairs()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        h.rebuild()
        h.apply_mask(ids, x)
        h.advance(ids, toks, out=out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        h.rebuild()
        h.apply_mask(ids, x)
        h.advance(ids, toks, out=out)
    for r in range(4):
        x.copy_(src)
        out.fill_(-7)
        if r % 2:
            h.rebuild()  # eager work on the same handle between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits_of(x).view(np.uint32), exp_x), r
        assert np.array_equal(out.cpu().numpy(), exp_out), r
        assert np.array_equal(gpu_rows(h, nodes[:48]), o.mask_rows(nodes[:48])), r
    assert h.valid_pairs() == M
    del graph
    torch.cuda.synchronize()
    h.close()


def nested_chain(depth: int, a: bytes, b: bytes) -> list:
    """a, aa, ..., a^depth, then a^i b and a^i b b for every i < depth: in trie
    order the a^i b strings come deepest first, so each one shares a shorter
    prefix with the string before it than that string did with its own
    predecessor, and the prefix nodes it reuses lie several strings back."""
    out = [a * i for i in range(1, depth + 1)]
    out += [a * i + b for i in range(depth)] + [a * i + b + b for i in range(0, depth, 3)]
    return out


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_nested_prefix_chains(P, flags):
    """Strings nested as prefixes of each other, one set of depth 48 and a
    forest of nine chains of depths 1-70 (written in groups of sets), every
    row, every advance and apply against the oracle.  Each string's prefix
    nodes are found by walking back over earlier strings that share ever
    shorter prefixes with it."""
    vocab = [b"a", b"b", b"c", b'"', b"aa", b"aaa", b"a" * 8, b"ab", b"bb", b'b"', b'a"', b"ba", b"c" * 5]
    h, _ = full_check(P, nested_chain(48, b"a", b"b"), vocab, flags=flags)
    h.close()
    sets = [nested_chain(d, a, b) for d, a, b in
            [(1, b"a", b"b"), (70, b"a", b"b"), (17, b"b", b"a"), (5, b"c", b"a"), (33, b"a", b"c"),
             (2, b"b", b"b"), (64, b"c", b"b"), (9, b"a", b"a"), (40, b"b", b"c")]]
    strings = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    h, _ = full_check(P, strings, vocab, sets=offs, flags=flags)
    h.close()


def long_token_case():
    """Strings of 60-200 bytes over {a, b, c}, some sharing their first 50+
    bytes with another, and tokens of 60-130 bytes cut from them (some ending
    in the terminator): token lengths of 64 and more, looked up in the
    per-length table rather than the 64-bit length mask."""
    rng = np.random.default_rng(64)
    abc = np.frombuffer(b"abc", dtype=np.uint8)
    base = [bytes(abc[rng.integers(0, 3, size=int(rng.integers(60, 201)))]) for _ in range(25)]
    strings = base + [b[:int(rng.integers(50, len(b)))] + bytes(abc[rng.integers(0, 3, size=int(rng.integers(1, 60)))])
                      for b in base[:15]]
    vocab = [b"a", b"b", b"c", b'"', b"ab", b"ca"]
    pool = [s for s in strings if len(s) >= 60]
    for k in range(200):
        src = pool[int(rng.integers(0, len(pool)))]
        n = int(rng.integers(60, min(130, len(src)) + 1))
        st = int(rng.integers(0, len(src) - n + 1))
        vocab.append(src[st:] + b'"' if k % 5 == 0 else src[st:st + n])
    vocab += [strings[0][:64], strings[1][3:68], strings[2][:63] + b'"']
    return strings, vocab


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_tokens_of_64_bytes_and_more(P, flags):
    """Every row, every advance and apply against the oracle when valid tokens
    are 64 to 200 bytes long and the trie branches below depth 64."""
    strings, vocab = long_token_case()
    h, o = full_check(P, strings, vocab, flags=flags)
    assert h.max_token_len >= 130
    h.close()


@pytest.mark.parametrize("seed", range(30))
def test_random_forests(P, seed):
    """Random forests (1-19 sets of 1-1,500 strings over 2-9 byte values,
    including 0x00, 0x80 and 0xff; sets that prefix, repeat and contain the
    empty string) and random vocabularies (empty, long and duplicate tokens, the
    terminator), in every representation: every row (or 20,000 sampled ones),
    5,000 random advances with out-of-range ids, and apply on 700 rows."""
    rng = np.random.default_rng(1000 + seed)
    alpha = np.frombuffer(b"abcde_\x00\xff\x80!", dtype=np.uint8)[: rng.integers(2, 10)]
    sets = []
    for _ in range(int(rng.integers(1, 20))):
        k = int(rng.integers(1, 300 if rng.random() < 0.8 else 1500))
        maxlen = int(rng.integers(1, 24))
        sets.append([bytes(alpha[rng.integers(0, len(alpha), size=rng.integers(0, maxlen + 1))]) for _ in range(k)])
    strings = [s for g in sets for s in g]
    offs = np.cumsum([0] + [len(g) for g in sets])
    vocab = [bytes(alpha[rng.integers(0, len(alpha), size=rng.integers(0, 20 if rng.random() < 0.9 else 40))])
             for _ in range(int(rng.integers(1, 2000)))]
    if rng.random() < 0.5:
        vocab += [b'"', bytes(alpha[:1]) + b'"']
    o = Oracle(strings, vocab, set_offsets=offs)
    if o.N <= 30000:
        nodes = np.arange(-1, o.N + 1, dtype=np.int32)
    else:
        nodes = np.unique(np.concatenate([o.roots, rng.integers(0, o.N, 20000)])).astype(np.int32)
    inside = (nodes >= 0) & (nodes < o.N)
    exp_rows = np.zeros((len(nodes), o.W), dtype=np.uint64)
    exp_rows[inside] = o.mask_rows(nodes[inside])
    nn = rng.integers(-1, o.N + 1, size=5000).astype(np.int32)
    tt = rng.integers(-1, o.V + 1, size=5000).astype(np.int32)
    exp_adv = o.advance(nn, tt)
    for flags in FLAGS:
        h = P.compile(strings, vocab, sets=offs, flags=flags, cache_rows=int(rng.integers(1, 200)))
        got = np.concatenate([gpu_rows(h, nodes[i:i + 1000]) for i in range(0, len(nodes), 1000)])
        assert np.array_equal(got, exp_rows), flags
        assert np.array_equal(gpu_advance(h, nn, tt), exp_adv), flags
        check_apply(P, h, o, nodes[:700], "bf16", seed=seed)
        h.close()


# ------------------------------------------------------ rows built on demand --

@pytest.mark.parametrize("cache", [1, 7, 64])
def test_lazy_cache_replacement(P, cache):
    """Rows built on demand with a cache smaller than the batch: groups of at
    most `cache` rows per assignment, evictions on every call, duplicate nodes
    inside a group, dead and out-of-range ids, and a decode loop whose every
    masked batch is checked against the oracle."""
    w = W.config(2)
    o = Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=LAZY, cache_rows=cache)
    assert h.cache_rows == cache and h.dense_rows == 0 and h.row_stride_words == 0
    rng = np.random.default_rng([cache, 17])
    start = W.uniform_nodes(2, o.N, 40, cache)
    start[:4] = 0
    start[4:8] = start[8:12]                      # the same nodes twice in one batch
    start = np.where(o.is_final[start] == 1, 0, start).astype(np.int32)
    cur = start.copy()
    for step in range(8):
        batch = cur.copy()
        batch[12], batch[13] = -1, o.N + 3         # dead rows are masked entirely
        check_apply(P, h, o, batch, "fp32" if step % 2 else "bf16", seed=step)
        rows = o.mask_rows(cur)
        toks = W.choose_valid_tokens(rng, rows, o.V)
        exp = o.advance(cur, toks)
        assert np.array_equal(gpu_advance(h, cur, toks), exp)
        cur = np.where((exp < 0) | (o.is_final[np.maximum(exp, 0)] == 1), start, exp).astype(np.int32)
    h.close()


def test_lazy_large_batch_hits_and_reset(P):
    """Batches larger than one group of 1024 rows; a second call on the same
    nodes finds every row in the cache; a reset empties it; two handles do not
    share cache state."""
    w = W.config(2)
    o = Oracle(w.strings, w.vocab)
    h = P.compile(w.strings, w.vocab, flags=LAZY)
    h2 = P.compile(w.strings, w.vocab, flags=LAZY, cache_rows=300)
    nodes = W.uniform_nodes(2, o.N, 2500, 9)
    nodes[::97] = 0
    check_apply(P, h, o, nodes, "bf16", seed=1)
    check_apply(P, h, o, nodes, "bf16", seed=2)
    check_apply(P, h2, o, nodes[:1500], "fp32", seed=3)
    check_apply(P, h, o, nodes[::-1].copy(), "fp32", seed=4)
    h.rebuild()
    check_apply(P, h, o, nodes[:100], "fp32", seed=5)
    check_apply(P, h2, o, nodes[1000:], "bf16", seed=6)
    assert np.array_equal(gpu_rows(h2, nodes[:700]), o.mask_rows(nodes[:700]))
    h.close()
    h2.close()


# ------------------------------------------------------ fixed-format strings --

@pytest.fixture(scope="module")
def c4_vocab(P):
    w = W.config(4)
    return w.vocab, P.Vocab(w.vocab)


@pytest.mark.parametrize("name", list(W.formats()))
def test_format_masks(P, c4_vocab, name):
    """Character-position masks over the 262,144-token vocabulary: every row,
    every (position, token) advance, apply and the pair count, against the
    oracle; rows again after a rebuild."""
    from oracle import Format
    classes = W.formats()[name]
    vocab, voc = c4_vocab
    f = Format(classes, vocab)
    h = P.compile_format(classes, voc)
    L = len(classes)
    assert h.num_nodes == L + 2 and h.dense_rows == L + 2
    pos = np.arange(-1, L + 3, dtype=np.int32)
    rows = f.mask_rows(pos)
    assert np.array_equal(gpu_rows(h, pos), rows)
    assert h.valid_pairs() == int(np.unpackbits(rows.view(np.uint8)).sum())
    V = len(vocab)
    for p in range(-1, L + 3):
        toks = np.arange(-1, V + 1, dtype=np.int32)
        assert np.array_equal(gpu_advance(h, np.full(toks.size, p), toks), f.advance(np.full(toks.size, p), toks)), p
    # apply: Eq. 1 on the oracle's rows, compared as raw bits
    rng = np.random.default_rng(91)
    ids = rng.integers(-1, L + 3, size=64).astype(np.int32)
    for dtype in ("bf16", "fp32"):
        x = host_logits(64, V, dtype, seed=92)
        dev = x.cuda()
        h.apply_mask(torch.as_tensor(ids, device="cuda"), dev)
        valid = np.unpackbits(f.mask_rows(ids).view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
        neg = np.uint16(0xFF80) if dtype == "bf16" else np.uint32(0xFF800000)
        ref = bits_of(x)
        ref = ref.view(np.uint16 if dtype == "bf16" else np.uint32)
        exp = np.where(valid, ref, neg)
        assert np.array_equal(bits_of(dev).view(exp.dtype), exp)
    for ph in (P.PHASE_MARK, P.PHASE_TABLE, P.PHASE_ZERO | P.PHASE_MARK):
        h.rebuild(phases=ph)
        assert np.array_equal(gpu_rows(h, pos), rows)
    with pytest.raises(P.TamError):
        h.rebuild(phases=P.PHASE_LISTS)
    h.close()


def test_format_decode_reaches_final(P, c4_vocab):
    """Decoding a date with uniformly random valid tokens always ends at the
    final position, having written L characters and the terminator."""
    from oracle import Format
    classes = W.formats()["YYYY-MM-DD"]
    vocab, voc = c4_vocab
    f = Format(classes, vocab)
    h = P.compile_format(classes, voc)
    rng = np.random.default_rng(93)
    cur = np.zeros(128, dtype=np.int32)
    text = [b""] * 128
    for step in range(len(classes) + 1):
        live = cur < len(classes) + 1
        rows = f.mask_rows(cur)
        toks = W.choose_valid_tokens(rng, rows, len(vocab))
        nxt = gpu_advance(h, cur, toks)
        assert np.array_equal(nxt, f.advance(cur, toks))
        for b in np.flatnonzero(live):
            text[b] += vocab[toks[b]]
        cur = np.where(live, nxt, cur).astype(np.int32)
    assert (cur == len(classes) + 1).all()
    for t in text:
        assert len(t) == len(classes) + 1 and t.endswith(b'"')
        assert all(c in cls for c, cls in zip(t, classes))
    h.close()


# ------------------------------------------------------------ layouts / edges --

@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_ragged_vocab_and_strides(P, flags):
    w = W.config(1)
    vocab = w.vocab[:1037]                      # V not a multiple of 8 or 64
    o = Oracle(w.strings, vocab)
    h = P.compile(w.strings, vocab, flags=flags)
    nodes = np.array([0, 1, 5, o.N - 1, -1, o.N, 2 ** 30], dtype=np.int32)
    for dtype in ("fp32", "bf16"):
        check_apply(P, h, o, nodes, dtype, seed=1)                  # contiguous rows
        check_apply(P, h, o, nodes, dtype, cols=1037, stride=1040, seed=2)   # aligned padded rows
        check_apply(P, h, o, nodes, dtype, cols=1037, stride=1045, seed=3)   # unaligned rows
    assert np.array_equal(gpu_rows(h, nodes), np.concatenate(
        [o.mask_rows(nodes[:4]), np.zeros((3, o.W), np.uint64)]))
    # zero-sized calls are no-ops
    empty = torch.empty(0, dtype=torch.int32, device="cuda")
    h.apply_mask(empty, torch.empty((0, 1037), device="cuda"))
    assert h.advance(empty, empty).numel() == 0


def test_many_rows_grid_split(P):
    """More than 65,535 batch rows in one call (the launcher splits the grid)."""
    strings = [b"ab", b"b"]
    vocab = [b"a", b"b", b"ab", b'"', b'b"'] + [b"z"] * 123
    o = Oracle(strings, vocab)
    B = 70000
    nodes = np.random.default_rng(0).integers(-1, o.N + 1, size=B).astype(np.int32)
    ids = torch.as_tensor(nodes, device="cuda")
    rows = o.mask_rows(np.arange(o.N, dtype=np.int32))
    valid = np.unpackbits(rows.view(np.uint8), axis=1, bitorder="little")[:, :128].astype(bool)
    exp = np.zeros((B, 128), dtype=bool)
    live = (nodes >= 0) & (nodes < o.N)
    exp[live] = valid[nodes[live]]
    for flags in FLAGS:
        h = P.compile(strings, vocab, flags=flags)
        x = torch.zeros((B, 128), dtype=torch.bfloat16, device="cuda")
        h.apply_mask(ids, x)
        assert np.array_equal(~torch.isinf(x).cpu().numpy(), exp)
        assert np.array_equal(gpu_rows(h, nodes[:66000]), np.where(
            live[:66000, None], rows[np.clip(nodes[:66000], 0, o.N - 1)], np.uint64(0)))
        h.close()


def test_c_abi_with_library_allocator(P):
    """The C ABI called directly: NULL allocator (the library's hipMalloc/hipFree)
    and the NULL stream, for a vocabulary, a compile against it, apply, advance,
    export and destroy, against the oracle."""
    import ctypes
    from paper_2608_12574_amd.tam import Options, csr
    L = P.lib()
    w = W.config(1)
    o = Oracle(w.strings, w.vocab)
    tb, to = csr(w.vocab)
    sb, so = csr(w.strings)
    voc = ctypes.c_void_p()
    assert L.tam_vocab_create(tb.ctypes.data, to.ctypes.data, len(w.vocab), 0, None, None, ctypes.byref(voc)) == 0
    for flags in FLAGS:
        h = ctypes.c_void_p()
        opt = Options(0x22, flags)
        assert L.tam_compile_vocab(sb.ctypes.data, so.ctypes.data, len(w.strings), voc, None, 0, ctypes.byref(opt),
                                   None, None, ctypes.byref(h)) == 0
        nodes = np.arange(-1, o.N + 1, dtype=np.int32)
        ids = torch.as_tensor(nodes, device="cuda")
        rows = torch.empty((nodes.size, o.W), dtype=torch.int64, device="cuda")
        assert L.tam_export_rows(h, ids.data_ptr(), nodes.size, rows.data_ptr(), None) == 0
        toks = torch.as_tensor(W.choose_valid_tokens(np.random.default_rng(5), o.mask_rows(nodes), o.V),
                               device="cuda")
        out = torch.empty_like(ids)
        assert L.tam_advance(h, ids.data_ptr(), toks.data_ptr(), nodes.size, out.data_ptr(), None) == 0
        x = host_logits(nodes.size, o.V, "bf16", seed=6)
        dev = x.cuda()
        assert L.tam_apply_mask(h, ids.data_ptr(), nodes.size, dev.data_ptr(), 1, o.V, None) == 0
        torch.cuda.synchronize()
        assert np.array_equal(rows.cpu().numpy().view(np.uint64), o.mask_rows(nodes))
        assert np.array_equal(out.cpu().numpy(), o.advance(nodes, toks.cpu().numpy()))
        exp = o.apply(nodes, bits_of(x).view(np.uint16), 1)
        assert np.array_equal(bits_of(dev).view(np.uint16), exp)
        L.tam_destroy(h)
    L.tam_vocab_destroy(voc)


@pytest.mark.parametrize("flags", FLAGS, ids=FLAG_IDS)
def test_graph_capture_replays(P, flags):
    """rebuild + apply + advance captured in a HIP graph: every replay, with eager
    work and synchronisation between replays, gives the eager results."""
    w = W.config(2)
    h = P.compile(w.strings, w.vocab, flags=flags)
    o = Oracle(w.strings, w.vocab)
    B, V = 64, len(w.vocab)
    nodes = W.uniform_nodes(2, o.N, B)
    ids = torch.as_tensor(nodes, device="cuda")
    src = torch.as_tensor(host_logits(B, V, "fp32", seed=12).numpy(), device="cuda")
    toks_np = W.choose_valid_tokens(np.random.default_rng(13), o.mask_rows(nodes), V)
    toks = torch.as_tensor(toks_np, device="cuda")
    x = src.clone()
    out = torch.empty_like(ids)
    exp_x = o.apply(nodes, bits_of(src.cpu()).view(np.uint32), 0)
    exp_out = o.advance(nodes, toks_np)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        h.rebuild()
        h.apply_mask(ids, x)
        h.advance(ids, toks, out=out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        h.rebuild()
        h.apply_mask(ids, x)
        h.advance(ids, toks, out=out)
    for r in range(5):
        x.copy_(src)
        out.fill_(-7)
        if r % 2:
            h.rebuild()  # eager work on the same handle between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits_of(x).view(np.uint32), exp_x), r
        assert np.array_equal(out.cpu().numpy(), exp_out), r
        assert np.array_equal(gpu_rows(h, nodes[:32]), o.mask_rows(nodes[:32])), r
    del graph
    torch.cuda.synchronize()
    h.close()
