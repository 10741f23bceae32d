"""Full-size parity in the launch configuration the benchmark times (default options).

At these sizes the oracle cannot run whole iterations in a test, so it draws a
random sample of tokens one by one from its own snapshot (its initial topics);
the GPU runs the whole first iteration.  The count tables are checked through
properties that hold at any size: T is the histogram of z, and the D rows of
sampled documents and W rows of sampled words are the histograms of their
tokens' topics.
"""
import os

import numpy as np
import pytest

import lda_synth
import oracle
from gpu_common import SEED, compare_draws, corpus_kw, make_lda, say

pytestmark = pytest.mark.gpu

SAMPLE = 20000


def _check_rows_sampled(c, cnt, rng):
    K = c.K
    z = cnt["z"]
    assert np.array_equal(cnt["T"], np.bincount(z, minlength=K))
    # documents (input is sorted by document)
    docs = np.sort(rng.choice(c.n_docs, 200, replace=False))
    lo = np.searchsorted(c.doc, docs)
    hi = np.searchsorted(c.doc, docs, side="right")
    for d, a, b in zip(docs, lo, hi):
        want = np.bincount(z[a:b], minlength=K)
        o0, o1 = cnt["D_off"][d], cnt["D_off"][d + 1]
        got = np.zeros(K, np.int64)
        got[cnt["D_topic"][o0:o1]] = cnt["D_count"][o0:o1]
        assert np.all(np.diff(cnt["D_topic"][o0:o1]) > 0)
        assert np.array_equal(got, want), d
    # words: the most frequent ones (dense rows, split into regions) and random ones
    freq = np.bincount(c.word, minlength=c.V)
    words = np.unique(np.concatenate([np.argsort(freq)[-5:], rng.choice(np.nonzero(freq)[0], 40, replace=False)]))
    pos = np.searchsorted(words, c.word)
    pos[pos == words.shape[0]] = 0
    mask = words[pos] == c.word
    hist = np.bincount(pos[mask].astype(np.int64) * K + z[mask], minlength=words.shape[0] * K).reshape(-1, K)
    for q, v in enumerate(words):
        o0, o1 = cnt["W_off"][v], cnt["W_off"][v + 1]
        got = np.zeros(K, np.int64)
        got[cnt["W_topic"][o0:o1]] = cnt["W_count"][o0:o1]
        assert np.array_equal(got, hist[q]), v


C5 = pytest.param("c5", marks=pytest.mark.skipif(
    not os.environ.get("LDA_FULLSIZE_C5"),
    reason="3.0e9-token corpus: about 7 minutes, mostly host-side generation and oracle counts; "
           "set LDA_FULLSIZE_C5=1 to run it"))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c6", C5])
def test_full_size_first_iteration(name):
    c = lda_synth.make_corpus(name)
    say("full-size %s N=%d V=%d K=%d" % (name, c.N, c.V, c.K))
    rng = np.random.default_rng(2024)
    idx = np.sort(rng.choice(c.N, SAMPLE, replace=False))
    z0 = oracle.init_topics(c.N, c.K, SEED)
    say("  oracle initial topics drawn")
    with make_lda(c) as m:
        say("  library created")
        cnt0 = m.counts()
        assert np.array_equal(cnt0["z"], z0)
        _check_rows_sampled(c, cnt0, rng)
        del cnt0
        say("  initial counts checked")
        st = m.iterate(1, stats=True)[0]
        say("  gpu iteration %.1f ms (sampler %.1f ms)" % (st["ms_iter"], st["ms_sampler"]))
        cnt1 = m.counts()
    assert st["skip_step3"] + st["sampled"] == c.N
    _check_rows_sampled(c, cnt1, rng)
    say("  new counts checked")
    say("  oracle on %d sampled tokens" % SAMPLE)
    zo, flags, ost = oracle.iterate(c.word, c.doc, z0, seed=SEED, t=0, idx=idx, **corpus_kw(c))
    n_bad = compare_draws(cnt1["z"][idx], zo, flags, c.N)
    say("  %d flagged mismatches; oracle skip3 %d of %d" % (n_bad, ost["skip3"], SAMPLE))


class _ManyDocs:
    """70M one-token documents: every D row takes its minimum of 32 slots, so D
    holds 2.24e9 slots and the rows of the last 2.2M documents start past 2^31
    (the 32-bit unsigned offsets that address them must never pass through a
    signed int)."""

    def __init__(self, n=70_000_000, V=1000, K=1000):
        rng = np.random.default_rng(31)
        self.word = ((rng.zipf(1.2, n) - 1) % V).astype(np.int32)
        self.doc = np.arange(n, dtype=np.int32)
        self.N, self.n_docs, self.V, self.K, self.alpha, self.beta = n, n, V, K, 0.05, 0.01


@pytest.mark.timeout(900)
def test_d_row_offsets_past_2_31():
    c = _ManyDocs()
    say("many one-token documents: N=M=%d, D slots %.3g" % (c.N, 32.0 * c.N))
    assert 32 * c.N > 2 ** 31
    rng = np.random.default_rng(7)
    # sampled tokens from the whole range and from the documents whose rows start past 2^31
    idx = np.unique(np.concatenate([rng.choice(c.N, 4000, replace=False),
                                    rng.choice(np.arange(c.N - 2_000_000, c.N), 4000, replace=False)]))
    z0 = oracle.init_topics(c.N, c.K, SEED)
    with make_lda(c) as m:
        say("  library created")
        st = m.iterate(1, stats=True)[0]
        say("  gpu iteration %.1f ms" % st["ms_iter"])
        cnt = m.counts()
    z = cnt["z"]
    assert st["skip_step3"] + st["sampled"] == c.N
    # a one-token document's row is its token's topic with count 1
    assert np.array_equal(cnt["D_off"], np.arange(c.N + 1))
    assert np.array_equal(cnt["D_topic"], z) and np.all(cnt["D_count"] == 1)
    assert np.array_equal(cnt["T"], np.bincount(z, minlength=c.K))
    W = np.bincount(c.word.astype(np.int64) * c.K + z, minlength=c.V * c.K)
    got = np.zeros(c.V * c.K, np.int64)
    rows = np.repeat(np.arange(c.V, dtype=np.int64), np.diff(cnt["W_off"]))
    got[rows * c.K + cnt["W_topic"]] = cnt["W_count"]
    assert np.array_equal(got, W)
    say("  counts checked; oracle on %d sampled tokens" % idx.size)
    zo, flags, _ = oracle.iterate(c.word, c.doc, z0, seed=SEED, t=0, idx=idx, **corpus_kw(c))
    n_bad = compare_draws(z[idx], zo, flags, c.N)
    say("  %d flagged mismatches" % n_bad)
