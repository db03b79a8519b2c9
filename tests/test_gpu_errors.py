"""Error paths of the C ABI on a device: a failing allocator, bad serving
arguments on a real handle, and the device error count of a good build.

These are the conditions a host can force; none makes a kernel fault.
"""
import ctypes

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def P():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_12574_amd as P
    P.lib()
    return P


class CountingAllocator:
    """Device memory from torch; the allocation numbered `fail_at` (0-based)
    returns NULL.  `live` holds what the library has not freed."""

    def __init__(self, P, fail_at=None):
        self.fail_at = fail_at
        self.calls = 0
        self.live = {}
        self.c_alloc = P.tam.ALLOC_FN(self._alloc)
        self.c_free = P.tam.FREE_FN(self._free)
        self.struct = P.tam.Allocator(self.c_alloc, self.c_free, None)

    def _alloc(self, nbytes, ctx):
        k = self.calls
        self.calls += 1
        if self.fail_at is not None and k >= self.fail_at:
            return None
        t = torch.empty(int(nbytes), dtype=torch.uint8, device="cuda")
        self.live[t.data_ptr()] = t
        return t.data_ptr()

    def _free(self, p, ctx):
        assert p in self.live, "freed a pointer the allocator never gave"
        del self.live[p]


def raw_compile(P, strings, vocab, flags, alloc, sets=None):
    sb, so = P.tam.csr(strings)
    tb, to = P.tam.csr(vocab)
    opt = P.tam.Options(0x22, flags, 64 if flags & P.FLAG_LAZY_ROWS else 0)
    out = ctypes.c_void_p()
    so_arr = None if sets is None else np.asarray(sets, dtype=np.int64)
    p = lambda a: None if a is None else ctypes.c_void_p(a.ctypes.data)  # noqa: E731
    L = P.lib()
    rc = L.tam_compile(p(sb), p(so), len(strings), p(tb), p(to), len(vocab), p(so_arr),
                       0 if sets is None else len(sets) - 1, ctypes.byref(opt), ctypes.byref(alloc.struct),
                       ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), ctypes.byref(out))
    return rc, out


@pytest.mark.parametrize("flags", [0, 2, 8, 16], ids=["dense", "no_table", "tail", "lazy"])
def test_allocator_failure_gives_nomem_and_frees_all(P, flags):
    """Every allocation of a compile failing in turn: TAM_E_NOMEM, no handle,
    and every block the library did get is handed back."""
    w = W.config(1)
    ok = CountingAllocator(P)
    rc, h = raw_compile(P, w.strings, w.vocab, flags, ok)
    assert rc == 0 and ok.calls >= 2
    P.lib().tam_destroy(h)
    torch.cuda.synchronize()
    assert not ok.live
    for k in range(ok.calls):
        a = CountingAllocator(P, fail_at=k)
        rc, h = raw_compile(P, w.strings, w.vocab, flags, a)
        assert rc == -3, (k, rc)
        assert not h.value
        assert "allocation failed" in P.lib().tam_last_error().decode()
        torch.cuda.synchronize()
        assert not a.live, (k, len(a.live))


@pytest.mark.parametrize("flags", [2, 2 | 8], ids=["no_table", "tail_lists"])
def test_allocator_failure_in_a_forest_written_in_groups(P, flags):
    """A forest of ten sets (written and uploaded in four groups; without a
    table under tail compression each group gets its own buffer of listed-hit
    records): every allocation failing in turn gives TAM_E_NOMEM, no handle,
    and every block back."""
    w = W.config(5)
    offs = [int(x) for x in w.set_offsets[:11]]
    strings = w.strings[:offs[-1]]
    ok = CountingAllocator(P)
    rc, h = raw_compile(P, strings, w.vocab, flags, ok, sets=offs)
    assert rc == 0 and ok.calls >= 3
    P.lib().tam_destroy(h)
    torch.cuda.synchronize()
    assert not ok.live
    for k in range(ok.calls):
        a = CountingAllocator(P, fail_at=k)
        rc, h = raw_compile(P, strings, w.vocab, flags, a, sets=offs)
        assert rc == -3, (k, rc)
        assert not h.value
        assert "allocation failed" in P.lib().tam_last_error().decode()
        torch.cuda.synchronize()
        assert not a.live, (k, len(a.live))


def test_allocator_failure_in_vocabulary_and_format(P):
    L = P.lib()
    tb, to = P.tam.csr([b"1", b"-", b'"', b"12"])
    a = CountingAllocator(P, fail_at=0)
    voc = ctypes.c_void_p()
    p = lambda x: ctypes.c_void_p(x.ctypes.data)  # noqa: E731
    assert L.tam_vocab_create(p(tb), p(to), 4, 0, ctypes.byref(a.struct), None, ctypes.byref(voc)) == -3
    assert not voc.value and not a.live
    good = CountingAllocator(P)
    assert L.tam_vocab_create(p(tb), p(to), 4, 0, ctypes.byref(good.struct), None, ctypes.byref(voc)) == 0
    classes = np.ascontiguousarray(P.tam.format_class_rows([b"0123456789"] * 3))
    for k in range(2):
        f = CountingAllocator(P, fail_at=k)
        h = ctypes.c_void_p()
        assert L.tam_compile_format(p(classes), 3, voc, None, ctypes.byref(f.struct), None, ctypes.byref(h)) == -3
        torch.cuda.synchronize()
        assert not h.value and not f.live
    L.tam_vocab_destroy(voc)
    torch.cuda.synchronize()
    assert not good.live


def test_serving_argument_errors_on_a_device_handle(P):
    w = W.config(1)
    h = P.compile(w.strings, w.vocab)
    L = P.lib()
    ids = torch.zeros(4, dtype=torch.int32, device="cuda")
    x = torch.zeros((4, w.V + 1), dtype=torch.bfloat16, device="cuda")
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert L.tam_apply_mask(h._raw, ptr(ids), 4, ptr(x), 7, x.stride(0), s) == -1          # dtype
    assert L.tam_apply_mask(h._raw, ptr(ids), 4, ptr(x), 1, w.V - 1, s) == -1             # stride < V
    assert L.tam_apply_mask(h._raw, ptr(ids), 4, ctypes.c_void_p(x.data_ptr() + 1), 1, x.stride(0), s) == -1
    xf = torch.zeros((4, w.V), dtype=torch.float32, device="cuda")
    assert L.tam_apply_mask(h._raw, ptr(ids), 4, ctypes.c_void_p(xf.data_ptr() + 2), 0, w.V, s) == -1
    assert L.tam_apply_mask(h._raw, ptr(ids), 4, ptr(x), 1, x.stride(0), s) == 0          # and it works
    assert L.tam_advance(h._raw, ptr(ids), None, 4, ptr(ids), s) == -1
    out = torch.zeros((4, h.words_per_row + 1), dtype=torch.int64, device="cuda")
    assert L.tam_export_rows(h._raw, ptr(ids), 4, ctypes.c_void_p(out.data_ptr() + 4), s) == -1
    torch.cuda.synchronize()
    # a good build met no inconsistent table entry on the device
    assert h.valid_pairs() > 0
    h.close()
