"""The out-of-core chunked corpus (lda_options.chunks) against the resident
path and the oracle, through the C ABI.

With C chunks the per-token arrays live in pinned host memory and stream
through two device slots each iteration; W and T are double-buffered, so every
chunk samples the same snapshot.  The draws must therefore be the resident
path's bit for bit, the counts the histograms of z, the LLPT the same up to the
summation order (partials per chunk), and a snapshot iteration the oracle's.
"""
import numpy as np
import pytest

import lda_synth
import oracle
from gpu_common import SEED, check_counts_are_histograms, compare_draws, corpus_kw, make_lda, oracle_step, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def c3r():
    return lda_synth.make_corpus("c3", n_docs=12000)


@pytest.fixture(scope="module")
def resident(c3r):
    with make_lda(c3r) as m:
        z0 = m.counts(D=False, W=False)["z"]
        st = m.iterate(10, stats=True)
        cnt = m.counts()
        ll = m.loglik()
    return z0, st, cnt, ll


@pytest.mark.parametrize("chunks", [2, 8, 13])
def test_chunked_iterations_equal_the_resident_path(c3r, resident, chunks):
    z0, st_r, cnt_r, ll_r = resident
    say("chunked %d: N=%d" % (chunks, c3r.N))
    with make_lda(c3r, chunks=chunks) as m:
        assert np.array_equal(m.counts(D=False, W=False)["z"], z0)  # the initial topics
        st = m.iterate(10, stats=True)
        cnt = m.counts()
        ll = m.loglik()
        ll_na = m.loglik_noalloc()
    assert np.array_equal(cnt["z"], cnt_r["z"])
    check_counts_are_histograms(c3r, cnt, c3r.K)
    for key in ("D_off", "D_topic", "D_count", "W_off", "W_topic", "W_count", "T"):
        assert np.array_equal(cnt[key], cnt_r[key]), key
    # the same decisions per iteration: skips, sampled tokens, draws in the max-topic branch (the
    # D-row entries read differ: a chunk's regions, and so the runs of one word in one document
    # whose later tokens draw from the first one's sums, split at other batch edges)
    for a, b in zip(st, st_r):
        assert (a["skip_step3"], a["sampled"], a["skip_after_s"], a["skip_test_ran"]) == \
               (b["skip_step3"], b["sampled"], b["skip_after_s"], b["skip_test_ran"])
        assert a["ms_iter"] > 0.0
    assert ll == pytest.approx(ll_r, rel=1e-12) and ll_na == ll
    say("  %d chunks: %.2f ms per iteration (resident %.2f)" % (
        chunks, np.mean([s["ms_iter"] for s in st[2:]]), np.mean([s["ms_iter"] for s in st_r[2:]])))


def test_chunked_snapshot_follows_the_oracle(c3r):
    """A snapshot set through lda_set_assignments, one iteration with steps 2-3 forced: the
    oracle's draws up to flagged near-boundary cases, counts the histograms of z."""
    z = oracle.init_topics(c3r.N, c3r.K, SEED)
    z, _, _ = oracle.iterate_threaded(c3r.word, c3r.doc, z, seed=SEED, t=0, **corpus_kw(c3r))
    zo, flags, ost = oracle.iterate_threaded(c3r.word, c3r.doc, z, seed=SEED, t=1, **corpus_kw(c3r))
    with make_lda(c3r, chunks=8, always_skip_test=True) as m:
        m.set_assignments(z, 1)
        st = m.iterate(1, stats=True)[0]
        cnt = m.counts()
    compare_draws(cnt["z"], zo, flags, c3r.N)
    check_counts_are_histograms(c3r, cnt, c3r.K)
    assert st["iteration"] == 1 and st["skip_test_ran"] == 1
    assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c3r.N)


def test_chunked_edge_shapes():
    """Empty documents at and between chunk edges, more chunks than non-empty documents would
    give equal shares, a word split into many regions, and the tiled sampler (K = 20,000)."""
    rng = np.random.default_rng(41)
    lens = rng.integers(0, 120, 400)
    lens[::7] = 0
    doc = np.repeat(np.arange(lens.shape[0], dtype=np.int32), lens)
    word = (rng.zipf(1.3, doc.shape[0]) % 300).astype(np.int32)

    class C:
        pass

    for K, chunks, R in ((64, 5, 0), (64, 40, 500), (20000, 3, 0)):
        c = C()
        c.word, c.doc, c.V, c.K, c.alpha, c.beta = word, doc, 300, K, 0.1, 0.01
        c.N, c.n_docs = word.shape[0], int(doc.max()) + 1
        say("chunk edges K=%d chunks=%d R=%d N=%d" % (K, chunks, R, c.N))
        outs = []
        for ch in (0, chunks):
            with make_lda(c, chunks=ch, region_tokens=R) as m:
                m.iterate(3)
                outs.append((m.counts(), m.loglik()))
        (a, lla), (b, llb) = outs
        for key in ("z", "D_off", "D_topic", "D_count", "W_off", "W_topic", "W_count", "T"):
            assert np.array_equal(a[key], b[key]), key
        check_counts_are_histograms(c, b, K)
        assert llb == pytest.approx(lla, rel=1e-12)
        z = a["z"]
        zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=3, **corpus_kw(c))
        with make_lda(c, chunks=chunks, region_tokens=R) as m:
            m.set_assignments(z, 3)
            m.iterate(1)
            compare_draws(m.counts(D=False, W=False)["z"], zo, flags, c.N)
