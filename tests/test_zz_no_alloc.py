"""tam_format_rows_noalloc, through the C ABI, against the rows and pair count
of tam_compile_format + tam_export_rows on the same formats and vocabularies.

Calls follow one another with smaller inputs after larger ones (the static
scratch keeps the last call's class bits), and reach the largest L the
scratch holds.
"""
import ctypes

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SENTINEL = 0x5A5A5A5A5A5A5A5A


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_12574_amd as P
    P.lib()
    return P


def noalloc_rows(P, classes, vocab, terminator=0x22, pad=3):
    """The raw C call into an output with `pad` extra words per row (left alone)."""
    L = len(classes)
    rows = np.ascontiguousarray(P.tam.format_class_rows(classes))
    W_ = (vocab.size + 63) // 64
    out = torch.full((L + 2, W_ + pad), SENTINEL, dtype=torch.int64, device="cuda")
    pairs = torch.full((1,), -7, dtype=torch.int64, device="cuda")
    rc = P.lib().tam_format_rows_noalloc(ctypes.c_void_p(rows.ctypes.data), L, terminator, vocab._raw,
                                         ctypes.c_void_p(out.data_ptr()), out.stride(0),
                                         ctypes.c_void_p(pairs.data_ptr()),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, P.lib().tam_last_error().decode()
    torch.cuda.synchronize()
    return out, pairs


def handle_rows(P, classes, vocab, terminator=0x22):
    h = P.compile_format(classes, vocab, terminator=terminator)
    rows = h.export_rows(torch.arange(len(classes) + 2, dtype=torch.int32, device="cuda"))
    pairs = h.valid_pairs()
    torch.cuda.synchronize()
    h.close()
    return rows, pairs


def check(P, classes, vocab, terminator=0x22):
    out, pairs = noalloc_rows(P, classes, vocab, terminator)
    exp, exp_pairs = handle_rows(P, classes, vocab, terminator)
    W_ = exp.shape[1]
    assert torch.equal(out[:, :W_], exp)
    assert bool((out[:, W_:] == SENTINEL).all())  # words past W are not written
    assert int(pairs.item()) == exp_pairs


def test_noalloc_format_rows_match_the_handle(P):
    big = P.Vocab(W.config(4).vocab)    # V = 262,144
    small = P.Vocab(W.config(1).vocab)  # V = 32,000
    fm = W.formats()
    check(P, fm["UUID v4"], big)               # L = 36
    check(P, fm["YYYY-MM-DD"], big)            # then a smaller L on the same GPU scratch
    check(P, fm["YYYY-MM-DD"], small)          # and a smaller vocabulary
    check(P, [b"0123456789"] * 3, small, terminator=ord("|"))
    big.close()
    small.close()


def test_noalloc_largest_format_then_smallest(P):
    voc = P.Vocab(W.config(1).vocab)
    L = 1024  # TAM_NOALLOC_MAX_POSITIONS
    digits = [b"0123456789", b"abcdefghijklmnopqrstuvwxyz", b"_ "]
    check(P, [digits[p % 3] for p in range(L)], voc)
    check(P, [b"a"], voc)
    rows = np.ascontiguousarray(P.tam.format_class_rows([b"0"] * (L + 1)))
    out = torch.zeros((L + 3, 512), dtype=torch.int64, device="cuda")
    rc = P.lib().tam_format_rows_noalloc(ctypes.c_void_p(rows.ctypes.data), L + 1, 0x22, voc._raw,
                                         ctypes.c_void_p(out.data_ptr()), 512, None, None)
    assert rc == -1 and "1024" in P.lib().tam_last_error().decode()
    voc.close()
