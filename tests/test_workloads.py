"""The seeded generators: shapes, determinism and the recipe's structure."""
import re

import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("cid,K,V,B,dtype", [(1, 100, 32000, 1, "fp32"), (2, 1000, 128256, 64, "fp32"),
                                            (3, 10000, 151936, 256, "bf16"),
                                            (4, 10000, 262144, 256, "bf16")])
def test_config_shapes(cid, K, V, B, dtype):
    w = W.config(cid)
    assert (w.K, w.V, w.batch, w.dtype) == (K, V, B, dtype)
    assert len(set(w.strings)) == K
    assert len(set(w.vocab)) == V
    assert w.vocab[:256] == [bytes([b]) for b in range(256)]
    assert all(b'"' not in s for s in w.strings)
    lens = np.array([len(t) for t in w.vocab[256:]])
    assert lens.min() >= 2 and lens.max() <= (12 if cid == 1 else 16)


def test_code_like_format():
    w = W.config(4)
    pat = re.compile(rb"^[A-Z][0-9]{2}(\.[0-9A-Z]{1,4})? - [a-z]+( [a-z]+){2,7}$")
    assert all(pat.match(s) and len(s) <= 64 for s in w.strings)
    frags = w.vocab[256:256 + 16384]
    assert all(re.fullmatch(rb"[0-9A-Z]{2,6}", t) for t in frags)


def test_forest_config():
    w = W.config(5)
    assert w.num_sets == 256 and w.K == 256 * 500
    for j in range(3):
        grp = w.strings[w.set_offsets[j]:w.set_offsets[j + 1]]
        assert len(set(grp)) == 500


def test_determinism():
    a = W.word_strings(W.rng_for(9, 1), [b"ab", b"cd", b"ef"], W.zipf_probs(3), 5, 1, 3)
    b = W.word_strings(W.rng_for(9, 1), [b"ab", b"cd", b"ef"], W.zipf_probs(3), 5, 1, 3)
    assert a == b
    assert np.array_equal(W.logits(1, 2, 10), W.logits(1, 2, 10))
    assert W.zipf_probs(200)[0] == pytest.approx(0.213, abs=2e-3)


def test_choose_valid_tokens():
    rows = np.zeros((3, 2), dtype=np.uint64)
    rows[0, 1] = np.uint64(1) << np.uint64(5)          # token 69
    rows[2, 0] = np.uint64(0b1010)                     # tokens 1, 3
    got = W.choose_valid_tokens(np.random.default_rng(0), rows, 100)
    assert got[0] == 69 and got[1] == -1 and got[2] in (1, 3)
