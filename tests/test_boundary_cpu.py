"""Boundary and host-layout tests that need no GPU.

* liblda.so loads and exports every symbol include/lda.h declares;
* argument validation of lda_create returns the documented status before
  touching a device;
* the host layout (lda_describe_layout): relabel by descending count, dense
  prefix iff count > K (Sec. 4.2), stable word order, regions that tile every
  word with at most R tokens (Sec. 5.1).
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2007_08725_amd as lda

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lda.LIB_PATH):
        from paper_2007_08725_amd import _build
        _build.build()
    return lda.load_library()


def test_exports_every_declared_symbol(lib):
    with open(os.path.join(ROOT, "include", "lda.h")) as f:
        header = f.read()
    declared = set(re.findall(r"\b(lda_[a-z_]+)\s*\(", header))
    assert declared == set(lda.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def _create(lib, word, doc, n, V, K, alpha, beta, opts=None):
    h = ctypes.c_void_p()
    st = lib.lda_create(word, doc, n, V, K, alpha, beta, 42, opts, ctypes.byref(h))
    return st, h


def test_create_argument_errors(lib):
    w = np.array([0, 1, 2], np.int32)
    d = np.array([0, 0, 1], np.int32)
    pw, pd = ctypes.c_void_p(w.ctypes.data), ctypes.c_void_p(d.ctypes.data)
    cases = [
        ((None, pd, 3, 3, 4, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, None, 3, 3, 4, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 0, 3, 4, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, -5, 3, 4, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 0, 4, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 1, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, lda.MAX_TOPICS + 1, 0.5, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 4, 0.0, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 4, -1.0, 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 4, float("nan"), 0.01), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 4, 0.5, float("inf")), lda.LDA_E_ARG),
        ((pw, pd, 3, 3, 4, 0.5, 0.0), lda.LDA_E_ARG),
        ((pw, pd, 3, 2, 4, 0.5, 0.01), lda.LDA_E_ARG),      # word id 2 >= V
    ]
    for args, want in cases:
        st, h = _create(lib, *args)
        assert st == want, args
        assert not h.value
        assert lib.lda_last_error(None)
    # negative doc id
    d2 = np.array([0, -1, 1], np.int32)
    st, h = _create(lib, pw, ctypes.c_void_p(d2.ctypes.data), 3, 3, 4, 0.5, 0.01)
    assert st == lda.LDA_E_ARG and not h.value
    # bad options
    for field, value in (("g", 4), ("g", -1), ("region_tokens", -2), ("sampler_block", 300),
                         ("sampler_block", 128), ("sampler_block", 2048), ("skip_marks", 3), ("skip_marks", -1),
                         ("always_skip_test", 2), ("always_skip_test", -1)):
        o = lda.Options()
        setattr(o, field, value)
        st, h = _create(lib, pw, pd, 3, 3, 4, 0.5, 0.01, ctypes.byref(o))
        assert st == lda.LDA_E_ARG, field
    # chunks: out of range, and the out-of-core mode needs input sorted by document
    for value in (-1, lda.MAX_CHUNKS + 1):
        o = lda.Options()
        o.chunks = value
        st, h = _create(lib, pw, pd, 3, 3, 4, 0.5, 0.01, ctypes.byref(o))
        assert st == lda.LDA_E_ARG and not h.value
    o = lda.Options()
    o.chunks = 2
    d_uns = np.array([1, 0, 1], np.int32)
    st, h = _create(lib, pw, ctypes.c_void_p(d_uns.ctypes.data), 3, 3, 4, 0.5, 0.01, ctypes.byref(o))
    assert st == lda.LDA_E_ARG and b"sorted by document" in lib.lda_last_error(None)
    o = lda.Options()
    o.dev_alloc = lda.ALLOC_FN(lambda n, c: None)
    st, h = _create(lib, pw, pd, 3, 3, 4, 0.5, 0.01, ctypes.byref(o))
    assert st == lda.LDA_E_ARG  # allocator without a matching free
    # NULL out pointer
    assert lib.lda_create(pw, pd, 3, 3, 4, 0.5, 0.01, 42, None, None) == lda.LDA_E_ARG


def test_layout_range_errors(lib):
    # a document with more than 65535 tokens does not fit the 16-bit counts
    # (lda_create reports the same after its device sort; see the GPU tests)
    n = lda.MAX_DOC_LEN + 1
    w = np.zeros(n, np.int32)
    d = np.zeros(n, np.int32)
    with pytest.raises(lda.LDAError) as ei:
        lda.describe_layout(w, d, 1, 4)
    assert ei.value.status == lda.LDA_E_RANGE
    assert b"65535" in lib.lda_last_error(None)
    # exactly 65535 is allowed
    L = lda.describe_layout(w[:-1], d[:-1], 1, 4)
    assert L["n_docs"] == 1


def test_handle_calls_reject_null(lib):
    assert lib.lda_iterate(None, 1, None) == lda.LDA_E_ARG
    assert lib.lda_loglik(None, None) == lda.LDA_E_ARG
    assert lib.lda_set_assignments(None, None, 0) == lda.LDA_E_ARG
    lib.lda_destroy(None)  # NULL-safe


def _layout_case(rng, n, V, M, K, shuffle):
    # Zipf-like word frequencies so that dense and sparse words both occur
    p = 1.0 / np.arange(1, V + 1) ** 1.1
    p /= p.sum()
    word = rng.permutation(V)[rng.choice(V, size=n, p=p)].astype(np.int32)
    doc = np.sort(rng.integers(0, M, n)).astype(np.int32)
    if shuffle:
        o = rng.permutation(n)
        word, doc = word[o], doc[o]
    return word, doc


@pytest.mark.parametrize("shuffle", [False, True])
@pytest.mark.parametrize("R", [7, 50, 10000])
def test_layout_properties(lib, shuffle, R):
    rng = np.random.default_rng(R + (1 if shuffle else 0))
    n, V, M, K = 5000, 300, 80, 16
    word, doc = _layout_case(rng, n, V, M, K, shuffle)
    L = lda.describe_layout(word, doc, V, K, R)
    cnt = np.bincount(word, minlength=V)
    rel = L["relabel"]
    assert sorted(rel.tolist()) == list(range(V))                       # a permutation
    order = np.argsort(rel)                                             # new id -> caller id
    assert np.all(np.diff(cnt[order]) <= 0)                             # descending counts
    ties = np.diff(cnt[order]) == 0
    assert np.all(np.diff(order)[ties] > 0)                             # ties by ascending id
    assert L["n_present"] == int((cnt > 0).sum())
    assert L["n_dense"] == int((cnt > K).sum())                         # dense iff count > K
    assert L["n_docs"] == int(doc.max()) + 1
    wo = L["word_off"].astype(np.int64)
    assert np.array_equal(np.diff(wo), cnt[order][:L["n_present"]])
    key = L["wt_key"].astype(np.int64)
    assert sorted(key.tolist()) == list(range(n))                       # word order is a permutation
    # word order: grouped by new word id, stable by (doc, input position) inside a word
    new_word = rel[word[key]]
    assert np.all(np.diff(new_word) >= 0)
    doc_pos = np.lexsort((np.arange(n), doc))                           # stable doc order
    rank = np.empty(n, np.int64)
    rank[doc_pos] = np.arange(n)
    same = np.diff(new_word) == 0
    assert np.all(np.diff(rank[key])[same] > 0)
    # regions tile every word exactly; only dense words are split; each region <= R
    reg_order = L["region"].astype(np.int64)
    reg = reg_order[np.argsort(reg_order[:, 1], kind="stable")]
    assert reg[0, 1] == 0 and reg[-1, 2] == n
    assert np.all(reg[1:, 1] == reg[:-1, 2])
    assert np.all(reg[:, 2] > reg[:, 1])
    # hand-out order: regions of split words by the middle of their span of
    # the word (ascending), then the unsplit words in word order
    cnt_new = np.diff(wo)
    split = np.array([cnt_new[w] > R and w < L["n_dense"] for w in reg_order[:, 0]])
    ns = int(split.sum())
    assert np.all(split[:ns]) and not np.any(split[ns:])
    mid = (reg_order[:ns, 1] + reg_order[:ns, 2] - 2 * wo[reg_order[:ns, 0]]) / (2.0 * cnt_new[reg_order[:ns, 0]])
    assert np.all(np.diff(mid) >= 0)
    assert np.all(np.diff(reg_order[ns:, 0]) > 0)
    for r in range(L["n_present"]):
        rows = reg[reg[:, 0] == r]
        assert rows[0, 1] == wo[r] and rows[-1, 2] == wo[r + 1]
        if r >= L["n_dense"]:
            assert rows.shape[0] == 1
        else:
            assert np.all(rows[:, 2] - rows[:, 1] <= R)
            assert rows.shape[0] == -(-(wo[r + 1] - wo[r]) // R)


@pytest.mark.parametrize("cutoff", [-1, 3, 40, 1 << 30])
def test_layout_dense_cutoff(lib, cutoff):
    """The hybrid-W cutoff: dense iff count > cutoff (0 = K, negative = every present word)."""
    rng = np.random.default_rng(5)
    n, V, M, K = 5000, 300, 80, 16
    word, doc = _layout_case(rng, n, V, M, K, False)
    L = lda.describe_layout(word, doc, V, K, 100, cutoff)
    cnt = np.bincount(word, minlength=V)
    want = int((cnt > 0).sum()) if cutoff < 0 else int((cnt > cutoff).sum())
    assert L["n_dense"] == want
    # regions: dense words split into <= R tokens, sparse words whole
    reg = L["region"].astype(np.int64)
    wo = L["word_off"].astype(np.int64)
    for r in range(L["n_present"]):
        rows = reg[reg[:, 0] == r]
        assert rows.shape[0] == (-(-(wo[r + 1] - wo[r]) // 100) if r < L["n_dense"] else 1)
    assert lda.describe_layout(word, doc, V, K, 100, 0)["n_dense"] == int((cnt > K).sum())


def test_layout_empty_documents_and_single_token(lib):
    word = np.array([3], np.int32)
    doc = np.array([5], np.int32)   # docs 0..4 are empty
    L = lda.describe_layout(word, doc, 4, 2)
    assert L["n_docs"] == 6 and L["n_present"] == 1 and L["n_dense"] == 0
    assert L["region"].tolist() == [[0, 0, 1]]
    assert L["relabel"][3] == 0
