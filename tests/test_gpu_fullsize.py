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
