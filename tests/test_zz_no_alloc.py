"""The allocation-free LLPT entry point against lda_loglik, through the C ABI.

lda_loglik_noalloc keeps its scratch (per-region partial sums, the region
counter, the result) in a fixed device array shared by every call on a GPU;
lda_loglik keeps the same scratch in handle memory.  Both run the same kernels
in the same order, so the results must be equal bit for bit -- also when the
array still holds a larger input's partials from the call before.
"""
import ctypes

import numpy as np
import pytest

import lda_synth
import oracle
from gpu_common import SEED, corpus_kw, say

pytestmark = pytest.mark.gpu


class _CountingAllocator:
    """Device allocation hooks that count every allocation (torch tensors as backing store)."""

    def __init__(self):
        import torch
        import paper_2007_08725_amd as lda
        self.torch, self.live, self.calls = torch, {}, 0
        self.fa = lda.ALLOC_FN(self._alloc)
        self.ff = lda.FREE_FN(self._free)

    def _alloc(self, nbytes, ctx):
        self.calls += 1
        t = self.torch.empty(int(nbytes), dtype=self.torch.uint8, device="cuda")
        self.live[t.data_ptr()] = t
        return t.data_ptr()

    def _free(self, ptr, ctx):
        self.live.pop(ptr, None)


def _create(c, alloc, **opts):
    import paper_2007_08725_amd as lda
    lib = lda.load_library()
    o = lda.Options()
    o.dev_alloc, o.dev_free = alloc.fa, alloc.ff
    for k, v in opts.items():
        setattr(o, k, v)
    h = ctypes.c_void_p()
    w, d = np.ascontiguousarray(c.word, np.int32), np.ascontiguousarray(c.doc, np.int32)
    st = lib.lda_create(ctypes.c_void_p(w.ctypes.data), ctypes.c_void_p(d.ctypes.data), c.N, c.V, c.K, c.alpha,
                        c.beta, SEED, ctypes.byref(o), ctypes.byref(h))
    assert st == lda.LDA_OK, lib.lda_last_error(None)
    return lib, h


def _llpt(lib, h, name):
    out = ctypes.c_double()
    st = getattr(lib, name)(h, ctypes.byref(out))
    assert st == 0, lib.lda_last_error(h)
    return out.value


def test_noalloc_loglik_equals_loglik_on_two_calls_the_second_smaller():
    alloc = _CountingAllocator()
    big = lda_synth.make_corpus("c3", n_docs=12000)
    small = lda_synth.make_corpus("c1", n_docs=200)
    results = []
    for c, iters in ((big, 3), (small, 2)):
        say("noalloc LLPT N=%d" % c.N)
        lib, h = _create(c, alloc)
        try:
            assert lib.lda_iterate(h, iters, None) == 0
            ref = _llpt(lib, h, "lda_loglik")
            before = alloc.calls
            got = _llpt(lib, h, "lda_loglik_noalloc")
            assert alloc.calls == before  # the call allocated nothing through the hooks
            again = _llpt(lib, h, "lda_loglik_noalloc")
            assert got == ref and again == ref  # bit for bit
            results.append((c, h, got))
            # and the value is the oracle's LLPT of the GPU's own state
            cnt = _counts_z(lib, h, c.N)
            assert got == pytest.approx(oracle.llpt(c.word, c.doc, cnt, **corpus_kw(c)), rel=1e-12)
        finally:
            lib.lda_destroy(h)
    assert results[1][0].N < results[0][0].N


def _counts_z(lib, h, n):
    import paper_2007_08725_amd as lda
    c = lda.Counts()
    z = np.empty(n, np.int32)
    T = np.empty(1 << 16, np.int64)
    c.z, c.T = z.ctypes.data, T.ctypes.data
    assert lib.lda_get_counts(h, ctypes.byref(c)) == 0
    return z


def test_noalloc_loglik_rejects_layouts_beyond_its_array():
    """More regions than the fixed array holds partial sums for: LDA_E_RANGE before any launch."""
    import paper_2007_08725_amd as lda

    class C:
        pass

    c = C()
    n = lda.NOALLOC_MAX_REGIONS + 4096
    c.word = np.zeros(n, np.int32)  # one word, dense, cut into one-token regions
    c.doc = (np.arange(n) // 30000).astype(np.int32)
    c.N, c.V, c.K, c.alpha, c.beta = n, 1, 4, 0.5, 0.01
    alloc = _CountingAllocator()
    lib, h = _create(c, alloc, region_tokens=1)
    try:
        out = ctypes.c_double(123.0)
        st = lib.lda_loglik_noalloc(h, ctypes.byref(out))
        assert st == lda.LDA_E_RANGE and out.value == 123.0
        assert b"regions" in lib.lda_last_error(h)
        ll = _llpt(lib, h, "lda_loglik")  # the handle is still usable, and lda_loglik has no such limit
        assert np.isfinite(ll)
    finally:
        lib.lda_destroy(h)
