"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws inputs (set strings, vocabularies, logits, batch node ids,
decode-token choices).  It holds none of the method's arithmetic: no trie, no
walk, no mask.  Both the oracle-based tests and the HIP path consume what it
returns, so neither side can influence the other's inputs.

The paper measures on real tokenizers (32K-262K vocabularies), on synthetic tool
names and on the ICD-10-CM code list (Sections 5 and the appendix on datasets).
None of those ship here; the five configurations below stand in for them:

  c1  K=100 word strings, V=32,000,    B=1   fp32
  c2  K=1,000 tool-name-like strings,  V=128,256, B=64  fp32
  c3  K=10,000 word strings,           V=151,936, B=256 bf16, 32 decode steps
  c4  K=10,000 code-like strings,      V=262,144, B=256 bf16, 32 decode steps
  c5  256 sets of K=500 drawn from a pool of 74,719 code-like strings,
      V=262,144, B=256 bf16, one set per batch row, 16 decode steps

Seeds: ``np.random.default_rng([config_id, role])`` with role 0 = lexicon,
1 = set strings, 2 = vocabulary corpus, 3 = vocabulary sampling, 4 = logits,
5 = node ids / decode-token choices, 6 = fragments (code-like vocabularies).
"""
from __future__ import annotations

import functools
from dataclasses import dataclass, field

import numpy as np

TERMINATOR = 0x22  # '"' closes every set string (the JSON string quote)

ROLE_LEXICON, ROLE_SET, ROLE_CORPUS, ROLE_VOCAB, ROLE_LOGITS, ROLE_CHOICE, ROLE_FRAG = range(7)

LOWER = b"abcdefghijklmnopqrstuvwxyz"
UPPER = b"ABCDEFGHIJKLMNOPQRSTUVWXYZ"
DIGITS = b"0123456789"
UPPER_DIGITS = DIGITS + UPPER


def rng_for(config_id: int, role: int) -> np.random.Generator:
    return np.random.default_rng([int(config_id), int(role)])


@dataclass
class Workload:
    """One configuration: the set strings, the vocabulary and the batch shape."""

    config_id: int
    name: str
    strings: list            # list[bytes]; for a forest, the concatenation of all sets
    vocab: list              # list[bytes], index = token id
    set_offsets: list | None  # forest: set j is strings[set_offsets[j]:set_offsets[j+1]]
    batch: int
    dtype: str               # "fp32" | "bf16"
    decode_steps: int
    node_mode: str           # "root" | "uniform" | "set_roots"
    description: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def K(self) -> int:
        return len(self.strings)

    @property
    def V(self) -> int:
        return len(self.vocab)

    @property
    def num_sets(self) -> int:
        return 1 if self.set_offsets is None else len(self.set_offsets) - 1


# ---------------------------------------------------------------------------
# building blocks
# ---------------------------------------------------------------------------

def make_lexicon(rng: np.random.Generator, L: int, lo: int = 3, hi: int = 8) -> list:
    """L distinct lowercase words, length uniform in [lo, hi]; rank = draw order."""
    seen = set()
    words = []
    letters = np.frombuffer(LOWER, dtype=np.uint8)
    while len(words) < L:
        n = int(rng.integers(lo, hi + 1))
        w = bytes(letters[rng.integers(0, 26, size=n)])
        if w not in seen:
            seen.add(w)
            words.append(w)
    return words


def zipf_probs(L: int, s: float = 1.1) -> np.ndarray:
    """Bounded Zipf over ranks 1..L: p_k proportional to k^-s."""
    p = np.arange(1, L + 1, dtype=np.float64) ** (-s)
    return p / p.sum()


def word_strings(rng, lexicon, probs, K, wmin, wmax, sep=b"_", prefixes=None, prefix_p=0.0):
    """K distinct strings of wmin..wmax i.i.d. Zipf words joined by ``sep``.

    With ``prefixes``, each string independently gets (with probability
    ``prefix_p``) a prefix drawn uniformly from that list.  Duplicates are
    redrawn until K distinct strings exist; order = first-draw order.
    """
    out, seen = [], set()
    L = len(lexicon)
    while len(out) < K:
        n = int(rng.integers(wmin, wmax + 1))
        idx = rng.choice(L, size=n, p=probs)
        s = sep.join(lexicon[i] for i in idx)
        if prefixes is not None and rng.random() < prefix_p:
            s = prefixes[int(rng.integers(0, len(prefixes)))] + s
        if s not in seen:
            seen.add(s)
            out.append(s)
    return out


def word_corpus(rng, lexicon, probs, nbytes, seps=(b"_", b" ")) -> bytes:
    """About ``nbytes`` of Zipf words, each followed by a separator drawn uniformly."""
    mean = sum(len(w) for w in lexicon) / len(lexicon) + 1.0
    n = int(nbytes / mean) + 16
    idx = rng.choice(len(lexicon), size=n, p=probs)
    sidx = rng.integers(0, len(seps), size=n)
    parts = []
    for i, j in zip(idx.tolist(), sidx.tolist()):
        parts.append(lexicon[i])
        parts.append(seps[j])
    return b"".join(parts)


def code_batch(rng, lexicon, probs, n, max_len=64):
    """A batch of ``n`` code-like strings: uppercase letter, two digits,
    optionally (probability 1/2) '.' plus 1-4 chars of [0-9A-Z], then ' - ' and
    3-8 Zipf words joined by spaces.  Trailing words are dropped to fit
    ``max_len`` bytes; a draw that would keep fewer than 3 words is None (the
    caller skips it).  All random draws of the batch are made up front."""
    lead = rng.integers(0, 26, size=n)
    dig = rng.integers(0, 10, size=(n, 2))
    dot = rng.random(n) < 0.5
    nfrag = rng.integers(1, 5, size=n)
    frag = rng.integers(0, 36, size=(n, 4))
    nw = rng.integers(3, 9, size=n)
    widx = rng.choice(len(lexicon), size=(n, 8), p=probs)
    out = []
    for i in range(n):
        head = bytes([UPPER[lead[i]], DIGITS[dig[i, 0]], DIGITS[dig[i, 1]]])
        if dot[i]:
            head += b"." + bytes(UPPER_DIGITS[j] for j in frag[i, :nfrag[i]])
        words = [lexicon[j] for j in widx[i, :nw[i]]]
        s = head + b" - " + b" ".join(words)
        while len(s) > max_len and len(words) > 3:
            words.pop()
            s = head + b" - " + b" ".join(words)
        out.append(s if len(s) <= max_len else None)
    return out


def code_strings(rng, lexicon, probs, K, distinct=True, max_len=64, batch=4096):
    """K code-like strings (distinct unless ``distinct`` is False), in draw order."""
    out, seen = [], set()
    while len(out) < K:
        for s in code_batch(rng, lexicon, probs, batch, max_len):
            if s is None:
                continue
            if distinct:
                if s in seen:
                    continue
                seen.add(s)
            out.append(s)
            if len(out) == K:
                break
    return out


def sample_substrings(rng, corpus: bytes, count: int, lo: int, hi: int, taken: set) -> list:
    """``count`` distinct substrings of ``corpus`` with length uniform in
    [lo, hi] and a uniform start, rejecting anything already in ``taken``
    (which is updated).  Returned in draw order."""
    out = []
    n = len(corpus)
    while len(out) < count:
        m = max(1024, (count - len(out)) * 2)
        lens = rng.integers(lo, hi + 1, size=m)
        starts = rng.integers(0, n - hi, size=m)
        for st, ln in zip(starts.tolist(), lens.tolist()):
            t = corpus[st:st + ln]
            if t in taken:
                continue
            taken.add(t)
            out.append(t)
            if len(out) == count:
                break
    return out


def byte_tokens() -> list:
    return [bytes([b]) for b in range(256)]


def random_fragments(rng, count, lo, hi, alphabet, taken: set) -> list:
    out = []
    alpha = np.frombuffer(alphabet, dtype=np.uint8)
    while len(out) < count:
        n = int(rng.integers(lo, hi + 1))
        t = bytes(alpha[rng.integers(0, len(alpha), size=n)])
        if t in taken:
            continue
        taken.add(t)
        out.append(t)
    return out


# ---------------------------------------------------------------------------
# the five configurations
# ---------------------------------------------------------------------------

CORPUS_BYTES = 8 << 20


def _word_vocab(cid, lexicon, probs, V, lo, hi):
    corpus = word_corpus(rng_for(cid, ROLE_CORPUS), lexicon, probs, CORPUS_BYTES)
    vocab = byte_tokens()
    taken = set(vocab)
    vocab += sample_substrings(rng_for(cid, ROLE_VOCAB), corpus, V - 256, lo, hi, taken)
    return vocab


def _code_vocab(cid, lexicon, probs, V):
    vocab = byte_tokens()
    taken = set(vocab)
    vocab += random_fragments(rng_for(cid, ROLE_FRAG), 16384, 2, 6, UPPER_DIGITS, taken)
    crng = rng_for(cid, ROLE_CORPUS)
    lines = []
    total = 0
    while total < CORPUS_BYTES:
        for s in code_batch(crng, lexicon, probs, 4096):
            if s is not None:
                lines.append(s)
                total += len(s) + 1
    corpus = b"\n".join(lines)
    vocab += sample_substrings(rng_for(cid, ROLE_VOCAB), corpus, V - len(vocab), 2, 16, taken)
    return vocab


@functools.lru_cache(maxsize=None)
def code_vocab_262k(cid: int) -> tuple:
    lex = make_lexicon(rng_for(cid, ROLE_LEXICON), 5000)
    probs = zipf_probs(5000)
    return tuple(_code_vocab(cid, lex, probs, 262144))


@functools.lru_cache(maxsize=None)
def config(cid: int) -> Workload:
    """The seeded workload of configuration ``cid`` (1..5)."""
    if cid == 1:
        lex = make_lexicon(rng_for(1, ROLE_LEXICON), 200)
        probs = zipf_probs(200)
        strings = word_strings(rng_for(1, ROLE_SET), lex, probs, 100, 2, 3)
        vocab = _word_vocab(1, lex, probs, 32000, 2, 12)
        return Workload(1, "c1", strings, vocab, None, 1, "fp32", 8, "root",
                        "K=100 word strings (2-3 Zipf words of a 200-word lexicon joined by '_'), "
                        "V=32,000 (256 bytes + corpus substrings of length 2-12), B=1 fp32")
    if cid == 2:
        lex = make_lexicon(rng_for(2, ROLE_LEXICON), 1000)
        probs = zipf_probs(1000)
        strings = word_strings(rng_for(2, ROLE_SET), lex, probs, 1000, 2, 4,
                               prefixes=[b"get_", b"list_", b"create_"], prefix_p=0.4)
        vocab = _word_vocab(2, lex, probs, 128256, 2, 16)
        return Workload(2, "c2", strings, vocab, None, 64, "fp32", 8, "uniform",
                        "K=1,000 tool-name-like strings (2-4 words, lexicon 1,000, 40% with a "
                        "get_/list_/create_ prefix), V=128,256 (lengths 2-16), B=64 fp32, "
                        "node ids uniform over the trie")
    if cid == 3:
        lex = make_lexicon(rng_for(3, ROLE_LEXICON), 5000)
        probs = zipf_probs(5000)
        strings = word_strings(rng_for(3, ROLE_SET), lex, probs, 10000, 2, 5)
        vocab = _word_vocab(3, lex, probs, 151936, 2, 16)
        return Workload(3, "c3", strings, vocab, None, 256, "bf16", 32, "root",
                        "K=10,000 word strings (2-5 words, lexicon 5,000), V=151,936 "
                        "(lengths 2-16), B=256 bf16 from the root, 32 decode steps")
    if cid == 4:
        lex = make_lexicon(rng_for(4, ROLE_LEXICON), 5000)
        probs = zipf_probs(5000)
        strings = code_strings(rng_for(4, ROLE_SET), lex, probs, 10000)
        vocab = list(code_vocab_262k(4))
        return Workload(4, "c4", strings, vocab, None, 256, "bf16", 32, "uniform",
                        "K=10,000 code-like strings (letter, 2 digits, optional '.'+1-4 "
                        "[0-9A-Z], ' - ', 3-8 Zipf words; <=64 B), V=262,144 (256 bytes, "
                        "16,384 [0-9A-Z] fragments of length 2-6, code-corpus substrings "
                        "of length 2-16), B=256 bf16, node ids uniform, 32 decode steps")
    if cid == 5:
        lex = make_lexicon(rng_for(5, ROLE_LEXICON), 5000)
        probs = zipf_probs(5000)
        pool = code_strings(rng_for(5, ROLE_SET), lex, probs, 74719)
        srng = rng_for(5, ROLE_CHOICE)
        strings, offs = [], [0]
        for _ in range(256):
            pick = srng.choice(len(pool), size=500, replace=False)
            strings += [pool[i] for i in pick.tolist()]
            offs.append(len(strings))
        vocab = list(code_vocab_262k(5))
        return Workload(5, "c5", strings, vocab, offs, 256, "bf16", 16, "set_roots",
                        "pool of 74,719 code-like strings; 256 sets of K=500 drawn without "
                        "replacement, compiled together as one forest; V=262,144 as c4; "
                        "B=256 bf16, row b decodes in set b from its root, 16 steps")
    raise ValueError(f"unknown configuration {cid}")


# ---------------------------------------------------------------------------
# serving-side inputs
# ---------------------------------------------------------------------------

def logits(cid: int, B: int, V: int, seed_extra: int = 0) -> np.ndarray:
    """N(0,1) float32 logits of shape [B, V] (cast to the target dtype by the caller)."""
    rng = np.random.default_rng([cid, ROLE_LOGITS, seed_extra])
    return rng.standard_normal(size=(B, V), dtype=np.float32)


def uniform_nodes(cid: int, num_nodes: int, B: int, seed_extra: int = 0) -> np.ndarray:
    rng = np.random.default_rng([cid, ROLE_CHOICE, 1, seed_extra])
    return rng.integers(0, num_nodes, size=B).astype(np.int32)


def choose_valid_tokens(rng: np.random.Generator, valid_rows: np.ndarray, V: int) -> np.ndarray:
    """For each packed row (uint64 words, token v = bit v&63 of word v>>6) pick a
    token uniformly among its set bits; rows with no set bit get -1."""
    out = np.full(valid_rows.shape[0], -1, dtype=np.int32)
    bits = np.unpackbits(valid_rows.view(np.uint8), axis=1, bitorder="little")[:, :V]
    for b in range(valid_rows.shape[0]):
        ids = np.flatnonzero(bits[b])
        if ids.size:
            out[b] = int(ids[int(rng.integers(0, ids.size))])
    return out


# ---------------------------------------------------------------------------
# edge suite: small hand-made sets and vocabularies covering degenerate cases
# ---------------------------------------------------------------------------

def edge_cases() -> list:
    """(name, strings, vocab) triples for the degenerate cases of the method."""
    q = b'"'
    base_vocab = byte_tokens() + [b"ab", b"abc", q, b'c"', b'",', b'"}', b'a"b', b"",
                                  b"ab", b"\x80\x81", b"\xff", b"get", b"get_", b"_user",
                                  b'user"', b'get"', b'"', b"\xc3\xa9", b"caf\xc3\xa9"]
    return [
        ("prefix_of_another", [b"get", b"get_user", b"get_users"], base_vocab),
        ("empty_string", [b"", b"a", b"ab"], base_vocab),
        ("duplicates", [b"abc", b"abc", b"ab", b"abc"], base_vocab),
        ("high_bytes", [b"\x80\x81\x82", b"\xff\xfe", b"caf\xc3\xa9", b"\xc3\xa9t\xc3\xa9"], base_vocab),
        ("single_char", [b"a"], base_vocab),
        ("no_shared_prefix", [b"xyz", b"abc", b"m"], base_vocab),
        ("only_empty", [b""], base_vocab),
        ("quote_tokens", [b"c", b"bc", b"abc"], [b'"', b'c"', b'bc"', b'abc"', b'",', b'"c', b"c", b""]),
        ("long_token", [b"a" * 40, b"a" * 20 + b"b"], byte_tokens() + [b"a" * k for k in range(2, 45)]),
        ("ragged_vocab", [b"hello", b"help", b"helm"], [b"h", b"he", b"hel", b"l", b"lo", b"p", b"m", b"o"]),
    ]


@functools.lru_cache(maxsize=None)
def stress_case() -> Workload:
    """3,000 code-like strings and a vocabulary that exercises the rare paths:
    60,000 tokens of the c4 vocabulary, 2,000 long tokens (17-48 bytes) cut from
    the set strings themselves (so they are valid somewhere), and 1,500 exact
    duplicates of earlier tokens (short and long)."""
    rng = rng_for(7, ROLE_SET)
    lex = make_lexicon(rng_for(7, ROLE_LEXICON), 5000)
    probs = zipf_probs(5000)
    strings = code_strings(rng, lex, probs, 3000)
    base = list(code_vocab_262k(4)[:60000])
    vrng = rng_for(7, ROLE_VOCAB)
    taken = set(base)
    longs = []
    while len(longs) < 2000:
        s = strings[int(vrng.integers(0, len(strings)))]
        if len(s) < 18:
            continue
        n = int(vrng.integers(17, min(48, len(s)) + 1))
        st = int(vrng.integers(0, len(s) - n + 1))
        t = s[st:st + n]
        if t not in taken:
            taken.add(t)
            longs.append(t)
    vocab = base + longs
    dups = [vocab[int(i)] for i in vrng.integers(0, len(vocab), size=1500)]
    vocab = vocab + dups
    return Workload(7, "stress", strings, vocab, None, 64, "bf16", 16, "uniform",
                    "3,000 code-like strings; 60,000 c4 tokens + 2,000 tokens of 17-48 bytes + 1,500 "
                    "duplicate tokens")


def mixed_forest():
    """A forest of one large set (over 1,024 strings, so the host cuts it by
    first byte), holding the empty string and strings that prefix others, and
    small sets, over the c1 vocabulary."""
    w = config(1)
    rng = rng_for(8, ROLE_SET)
    lex = make_lexicon(rng_for(8, ROLE_LEXICON), 300)
    big = word_strings(rng, lex, zipf_probs(len(lex)), 1500, 1, 3)
    big = [b""] + big + [s[:3] for s in big[:50]]
    small = [word_strings(rng, lex, zipf_probs(len(lex)), k, 1, 2) for k in (1, 7, 40)]
    sets = [small[0], big, small[1], small[2]]
    offs = np.cumsum([0] + [len(s) for s in sets])
    return [s for g in sets for s in g], w.vocab, offs


DIGITS = b"0123456789"
HEX = b"0123456789abcdef"


def formats() -> dict:
    """The fixed formats of the paper's character-position experiment, as byte
    classes per position: an ISO date, a date-time, a date-time with
    milliseconds, and a version-4 UUID (hex digits, the version digit 4, the
    variant digit 8/9/a/b)."""
    d = [DIGITS]
    date = d * 4 + [b"-"] + d * 2 + [b"-"] + d * 2
    dt = date + [b"T"] + d * 2 + [b":"] + d * 2 + [b":"] + d * 2
    dtms = dt + [b"."] + d * 3
    uuid = ([HEX] * 8 + [b"-"] + [HEX] * 4 + [b"-"] + [b"4"] + [HEX] * 3 + [b"-"] + [b"89ab"] + [HEX] * 3
            + [b"-"] + [HEX] * 12)
    return {"YYYY-MM-DD": date, "datetime": dt, "datetime.ms": dtms, "UUID v4": uuid}
