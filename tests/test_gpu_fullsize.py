"""Full-size parity in the launch configuration the benchmark times (default options).

The schedule on every workload: snapshots at t = 0 (the Philox initial topics),
t = 1 and t = 49.  The GPU runs whole iterations; at each checked t the oracle
takes the GPU's assignment z_t as its snapshot (t = 0: its own initial topics,
which must equal the GPU's) and draws a random sample of 20,000 tokens from it,
building only the count rows those tokens read.  The GPU's z_{t+1} must agree on
the sample up to flagged near-boundary draws.  After the t = 49 iteration the
GPU has run 50 iterations: its count tables are checked through properties that
hold at any size (T is the histogram of z; the D rows of sampled documents and W
rows of sampled words are the histograms of their tokens' topics), and its LLPT
is compared with the oracle's after its own 50 iterations (goldens written on
the CPU by tests/golden/make_llpt_goldens.py) within 1e-3 relative.
"""
import json
import os

import numpy as np
import pytest

import lda_synth
import oracle
from gpu_common import SEED, compare_draws, corpus_kw, make_lda, say

pytestmark = pytest.mark.gpu

SAMPLE = 20000
CHECKS = (0, 1, 49)
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
THREADS = min(16, oracle.default_threads())


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
    slot = np.full(c.V, -1, np.int32)
    slot[words] = np.arange(words.shape[0], dtype=np.int32)
    pos = slot[c.word]
    mask = pos >= 0
    hist = np.bincount(pos[mask].astype(np.int64) * K + z[mask], minlength=words.shape[0] * K).reshape(-1, K)
    del pos, mask
    for q, v in enumerate(words):
        o0, o1 = cnt["W_off"][v], cnt["W_off"][v + 1]
        got = np.zeros(K, np.int64)
        got[cnt["W_topic"][o0:o1]] = cnt["W_count"][o0:o1]
        assert np.array_equal(got, hist[q]), v


def _golden(case, c):
    path = os.path.join(GOLDEN, "llpt50_%s.json" % case)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        g = json.load(f)
    assert (g["N"], g["V"], g["K"], g["M"], g["seed"]) == (c.N, c.V, c.K, c.n_docs, SEED), path
    assert lda_synth.fingerprint(c) == g["corpus_fingerprint"], path
    return g


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5", "c6"])
def test_full_size_schedule(name):
    c = lda_synth.make_corpus(name, nthreads=THREADS)
    say("full-size %s N=%d V=%d K=%d" % (name, c.N, c.V, c.K))
    rng = np.random.default_rng(2024)
    idx = np.sort(rng.choice(c.N, SAMPLE, replace=False))
    kw = corpus_kw(c)
    z = oracle.init_topics(c.N, c.K, SEED, threads=THREADS)
    say("  oracle initial topics drawn")
    with make_lda(c) as m:
        say("  library created")
        assert np.array_equal(m.counts(D=False, W=False)["z"], z)
        t = 0
        for t_check in CHECKS:
            if t_check > t:
                m.iterate(t_check - t)
                t = t_check
                z = m.counts(D=False, W=False)["z"]  # the GPU's own state z_t is the snapshot
            st = m.iterate(1, stats=True)[0]
            assert st["iteration"] == t and st["skip_step3"] + st["sampled"] == c.N
            t += 1
            z_next = m.counts(D=False, W=False)["z"]
            zo, flags, ost = oracle.iterate(c.word, c.doc, z, seed=SEED, t=t_check, idx=idx, restricted=True, **kw)
            n_bad = compare_draws(z_next[idx], zo, flags, c.N)
            assert ost["sest_violations"] == 0 and ost["skip_not_k1"] == 0
            say("  t=%d: gpu %.1f ms (sampler %.1f), skipped %.4f; %d flagged mismatches of %d (oracle skip3 %d)"
                % (t_check, st["ms_iter"], st["ms_sampler"], st["skip_step3"] / c.N, n_bad, SAMPLE, ost["skip3"]))
            z = z_next
            del z_next
        del z
        assert t == 50
        cnt = m.counts()
        _check_rows_sampled(c, cnt, rng)
        del cnt
        say("  counts after 50 iterations checked")
        ll = m.loglik()
    g = _golden(name, c)
    if g is not None:
        say("  LLPT after 50 iterations: gpu %.6f, oracle %.6f" % (ll, g["llpt"]))
        assert ll == pytest.approx(g["llpt"], rel=1e-3)
    else:
        say("  LLPT after 50 iterations: gpu %.6f (no oracle golden at this size)" % ll)
    assert np.isfinite(ll)


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
    z0 = oracle.init_topics(c.N, c.K, SEED, threads=THREADS)
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
    zo, flags, _ = oracle.iterate(c.word, c.doc, z0, seed=SEED, t=0, idx=idx, restricted=True, **corpus_kw(c))
    n_bad = compare_draws(z[idx], zo, flags, c.N)
    say("  %d flagged mismatches" % n_bad)
