"""GPU parity: the HIP path (through the C ABI) against the oracle.

Bars (per draw): every GPU/oracle topic mismatch is a flagged near-boundary
draw and there are fewer than 1e-6*N of them; D, W and T are bit-exact given
the GPU's assignment; LLPT agrees with the oracle to 1e-12 relative on the same
assignment (1e-3 after trajectories diverge).
"""
import json
import os

import numpy as np
import pytest

import lda_synth
import oracle
from gpu_common import (SEED, check_counts_are_histograms, compare_draws, corpus_kw, make_lda, oracle_step,
                        say)

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module")
def c1():
    return lda_synth.make_corpus("c1")


@pytest.fixture(scope="module")
def c1_traj(c1):
    """Oracle trajectory of c1: initial topics, then 10 iterations with flags and stats."""
    z = oracle.init_topics(c1.N, c1.K, SEED)
    out = [(z, None, None)]
    for t in range(c1.spec.iters):
        zn, f, st = oracle_step(c1, z, t)
        out.append((zn, f, st))
        z = zn
    return out


def test_init_topics_match_oracle(c1, c1_traj):
    say("init c1 N=%d" % c1.N)
    with make_lda(c1) as m:
        cnt = m.counts()
    assert cnt["iteration"] == 0
    assert np.array_equal(cnt["z"], c1_traj[0][0])
    check_counts_are_histograms(c1, cnt, c1.K)


def test_c1_every_iteration_from_oracle_snapshot(c1, c1_traj):
    """At each t the GPU starts from the oracle's z_t and must reproduce z_{t+1}."""
    with make_lda(c1, always_skip_test=True) as m:
        for t in range(c1.spec.iters):
            say("c1 snapshot t=%d" % t)
            m.set_assignments(c1_traj[t][0], t)
            st = m.iterate(1, stats=True)[0]
            cnt = m.counts()
            zo, flags, ost = c1_traj[t + 1]
            compare_draws(cnt["z"], zo, flags, c1.N)
            check_counts_are_histograms(c1, cnt, c1.K)
            assert st["iteration"] == t and cnt["iteration"] == t + 1
            assert st["skip_step3"] + st["sampled"] == c1.N
            # the GPU's step-3 test is conservative (single precision with a margin):
            # it may skip a few tokens fewer than the oracle's fp64 test, never more
            assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c1.N)
            assert st["ms_sampler"] > 0.0


def test_c1_free_running_trajectory_and_llpt(c1, c1_traj):
    with make_lda(c1) as m:
        ll0 = m.loglik()
        m.iterate(c1.spec.iters)
        cnt = m.counts()
        ll = m.loglik()
    kw = corpus_kw(c1)
    zo = c1_traj[-1][0]
    lo0 = oracle.llpt(c1.word, c1.doc, c1_traj[0][0], **kw)
    assert ll0 == pytest.approx(lo0, rel=1e-12)
    lo = oracle.llpt(c1.word, c1.doc, zo, **kw)
    if np.array_equal(cnt["z"], zo):
        assert ll == pytest.approx(lo, rel=1e-12)
    else:
        assert ll == pytest.approx(lo, rel=1e-3)
    # the GPU's LLPT on its own state equals the oracle's LLPT on that same state
    assert ll == pytest.approx(oracle.llpt(c1.word, c1.doc, cnt["z"], **kw), rel=1e-12)
    assert ll > ll0


@pytest.mark.parametrize("opts", [dict(region_tokens=7), dict(region_tokens=100), dict(g=1), dict(g=3), dict(no_skip=True),
                                  dict(dense_cutoff=-1), dict(dense_cutoff=1 << 30), dict(dense_cutoff=3),
                                  dict(sampler_block=256), dict(sampler_block=512), dict(sampler_block=1024),
                                  dict(skip_marks=1), dict(skip_marks=2),
                                  dict(torch_allocator=False, torch_stream=False)])
def test_schedule_invariance(c1, opts):
    """Region size, S_est depth, the skip test, the hybrid-W cutoff (all dense, all sparse),
    the sampler's workgroup size, the skip bitmap, allocator and stream never change the draws."""
    say("invariance %s" % opts)
    with make_lda(c1) as a:
        a.iterate(3)
        za = a.counts(D=False, W=False)["z"]
    with make_lda(c1, **opts) as b:
        b.iterate(3)
        zb = b.counts(D=False, W=False)["z"]
    assert np.array_equal(za, zb)


def test_skip_bitmap_switch_follows_the_oracle():
    """The per-iteration choice between the two skip bitmaps, taken where it fires.  The corpus
    starts from a concentrated planted assignment, so iteration 0 skips well over a fifth of its
    tokens and carries its decisions in the word-ordered bitmap; iteration 1 then switches to the
    document-ordered bitmap.  Both iterations draw what the oracle draws from the same snapshot,
    and forcing either bitmap gives the same draws; shuffled input has no document-ordered bitmap
    and falls back to the word-ordered one."""
    c = lda_synth.concentrated()
    say("skip bitmap switch N=%d K=%d" % (c.N, c.K))
    runs = {}
    for marks in (0, 1, 2):
        with make_lda(c, skip_marks=marks) as m:
            m.set_assignments(c.topic, 0)
            z = c.topic
            rec = []
            for t in range(3):
                zo, flags, ost = oracle_step(c, z, t)
                st = m.iterate(1, stats=True)[0]
                zg = m.counts(D=False, W=False)["z"]
                compare_draws(zg, zo, flags, c.N)
                assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c.N)
                rec.append((st["skip_step3"] / c.N, st["skip_marks"], zg))
                z = zg  # the GPU's own state is the next snapshot
            runs[marks] = rec
    rates = [r[0] for r in runs[0]]
    say("  skip rates %s, bitmaps (auto) %s" % (["%.3f" % x for x in rates], [r[1] for r in runs[0]]))
    assert rates[0] > 0.2  # the threshold is crossed at once
    assert [r[1] for r in runs[0]] == [1, 2, 2]  # word order first (no previous count), then document order
    assert [r[1] for r in runs[1]] == [1, 1, 1] and [r[1] for r in runs[2]] == [2, 2, 2]
    for t in range(3):
        assert np.array_equal(runs[0][t][2], runs[1][t][2]) and np.array_equal(runs[0][t][2], runs[2][t][2])
        assert runs[0][t][0] == runs[1][t][0] == runs[2][t][0]
    cs = lda_synth.generate(lda_synth.SPECS["c1"], n_docs=300, shuffle=True)
    out = []
    for marks in (1, 2):
        with make_lda(cs, skip_marks=marks) as m:
            st = m.iterate(3, stats=True)
            assert all(s["skip_marks"] == 1 for s in st)
            out.append(m.counts(D=False, W=False)["z"])
    assert np.array_equal(out[0], out[1])


@pytest.fixture(scope="module")
def switch_snapshots(c1, c1_traj):
    """Snapshots every option is checked on, with the oracle's draws from each: c1 at t = 8, a
    reduced c3 at t = 0 and the concentrated corpus (most tokens skip) at t = 0 (iterations in
    which steps 2-3 run by default)."""
    c3 = lda_synth.make_corpus("c3", n_docs=12000)
    cc = lda_synth.concentrated()
    out = []
    for c, z, t in ((c1, c1_traj[8][0], 8), (c3, oracle.init_topics(c3.N, c3.K, SEED), 0), (cc, cc.topic, 0)):
        zo, flags, ost = oracle.iterate_threaded(c.word, c.doc, z, seed=SEED, t=t, **corpus_kw(c))
        out.append((c, z, t, zo, flags, ost))
    return out


@pytest.mark.parametrize("opts", [dict(no_skip=True), dict(dense_cutoff=-1), dict(dense_cutoff=1 << 30),
                                  dict(sampler_block=256), dict(sampler_block=512), dict(sampler_block=1024),
                                  dict(skip_marks=1), dict(skip_marks=2), dict(region_tokens=97), dict(g=1),
                                  dict(g=3), dict(always_skip_test=True)],
                         ids=lambda o: "-".join("%s=%s" % kv for kv in o.items()))
def test_every_option_follows_the_oracle(switch_snapshots, opts):
    """Each performance or ablation switch that must leave the draws unchanged, against the
    oracle (not only against the GPU's default): same snapshot, same draws up to flagged
    near-boundary cases, counts the histograms of z."""
    for c, z, t, zo, flags, ost in switch_snapshots:
        say("option %s on N=%d K=%d t=%d" % (opts, c.N, c.K, t))
        with make_lda(c, **opts) as m:
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            cnt = m.counts()
        compare_draws(cnt["z"], zo, flags, c.N)
        check_counts_are_histograms(c, cnt, c.K)
        if opts.get("no_skip"):
            assert st["skip_step3"] == 0 and st["sampled"] == c.N and st["skip_test_ran"] == 0
        else:
            assert st["skip_step3"] + st["sampled"] == c.N and st["skip_test_ran"] == 1
            if "g" in opts:  # the skip statistics at the same S_est depth (the draws do not depend on it)
                ost = oracle.iterate_threaded(c.word, c.doc, z, seed=SEED, t=t, g=opts["g"], **corpus_kw(c))[2]
            assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c.N)


def test_skip_test_runs_when_it_pays():
    """By default steps 2-3 run in every eighth iteration and after an iteration that skipped at
    least an eighth of the tokens; the draws are those of running them in every iteration."""
    for c, z0, want in ((lda_synth.make_corpus("c2", n_docs=2500), None, [1, 0, 0, 0, 0, 0, 0, 0, 1, 0]),
                        (lda_synth.concentrated(), "planted", [1] * 10)):
        zs, ran = [], []
        for always in (False, True):
            with make_lda(c, always_skip_test=always) as m:
                if z0 == "planted":
                    m.set_assignments(c.topic, 0)
                st = m.iterate(10, stats=True)
                zs.append(m.counts(D=False, W=False)["z"])
                ran.append([s["skip_test_ran"] for s in st])
                rates = [s["skip_step3"] / c.N for s in st]
        say("  N=%d skip rates %s ran %s" % (c.N, ["%.3f" % r for r in rates], ran[0]))
        assert ran[0] == want and ran[1] == [1] * 10
        assert np.array_equal(zs[0], zs[1])


@pytest.mark.parametrize("g", [1, 3])
def test_skip_counts_follow_the_oracle_for_every_depth(c1, c1_traj, g):
    """Step-3 skips at S_est depth g (Eq. 9) against the oracle's fp64 test on the same
    snapshots: the GPU's single-precision test with its margin skips a few tokens fewer,
    never more."""
    with make_lda(c1, g=g, always_skip_test=True) as m:
        for t in range(3):
            z = c1_traj[t][0]
            zo, flags, ost = oracle_step(c1, z, t, g=g)
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            compare_draws(m.counts(D=False, W=False)["z"], zo, flags, c1.N)
            assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c1.N)


def test_two_branch_mode_follows_the_oracle(c1, c1_traj):
    """The two-branch ablation (Sec. 2.2, draws over [S | Q]) against the oracle's two-branch
    form on c1 snapshots: same draws except flagged boundary cases, counts the histograms of z,
    and no token skipped."""
    with make_lda(c1, two_branch=True) as m:
        for t in range(3):
            z = c1_traj[t][0]
            zo, flags, ost = oracle_step(c1, z, t, branches=2)
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c1.N)
            check_counts_are_histograms(c1, cnt, c1.K)
            assert st["skip_step3"] == 0 and st["skip_after_s"] == 0 and st["sampled"] == c1.N
        z3 = m.counts(D=False, W=False)["z"]
    # a different canonical order: the same u gives other topics for some tokens
    assert not np.array_equal(z3, c1_traj[3][0])


def test_determinism_and_resume(c1):
    with make_lda(c1) as a:
        a.iterate(10)
        z10 = a.counts(D=False, W=False)["z"]
    with make_lda(c1) as b:
        b.iterate(5)
        z5 = b.counts(D=False, W=False)["z"]
    with make_lda(c1) as c:
        c.set_assignments(z5, 5)
        c.iterate(5)
        cnt = c.counts()
    assert cnt["iteration"] == 10
    assert np.array_equal(cnt["z"], z10)
    check_counts_are_histograms(c1, cnt, c1.K)


REDUCED = [
    # (name, overrides): corpus shapes of the five workloads at sizes the oracle finishes in seconds;
    # every one has words with more than 10,000 tokens (split into several regions)
    ("c2", dict(n_docs=2500)),
    ("c3", dict(n_docs=12000)),
    ("c4", dict(n_docs=1200, V=20000)),
    ("c5", dict(n_docs=3000, V=100000)),
]


@pytest.mark.parametrize("name,over", REDUCED, ids=[r[0] for r in REDUCED])
def test_reduced_config_snapshots(name, over):
    c = lda_synth.make_corpus(name, **over)
    say("reduced %s N=%d V=%d K=%d" % (name, c.N, c.V, c.K))
    z = oracle.init_topics(c.N, c.K, SEED)
    with make_lda(c) as m:
        assert np.array_equal(m.counts(D=False, W=False)["z"], z)
        for t in range(2):
            zo, flags, ost = oracle_step(c, z, t)
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c.N)
            check_counts_are_histograms(c, cnt, c.K)
            assert st["skip_step3"] + st["sampled"] == c.N
            assert st["regions"] > c.V // 50
            z = zo
        ll = m.loglik()
    assert ll == pytest.approx(oracle.llpt(c.word, c.doc, cnt["z"], **corpus_kw(c)), rel=1e-12)


@pytest.mark.parametrize("name,over", REDUCED[:2], ids=[r[0] for r in REDUCED[:2]])
def test_reduced_config_late_snapshot(name, over):
    """Iteration 49 from the GPU's own state after 49 iterations (higher skip rates than at the start)."""
    c = lda_synth.make_corpus(name, **over)
    say("late snapshot %s N=%d" % (name, c.N))
    with make_lda(c, always_skip_test=True) as m:
        m.iterate(49)
        z = m.counts(D=False, W=False)["z"]
        zo, flags, ost = oracle_step(c, z, 49)
        st = m.iterate(1, stats=True)[0]
        assert st["iteration"] == 49
        cnt = m.counts()
    compare_draws(cnt["z"], zo, flags, c.N)
    check_counts_are_histograms(c, cnt, c.K)
    assert st["skip_step3"] + st["sampled"] == c.N
    assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c.N)
    say("  skip3 gpu %d oracle %d of %d" % (st["skip_step3"], ost["skip3"], c.N))


def load_golden(case):
    with open(os.path.join(GOLDEN, "llpt50_%s.json" % case)) as f:
        return json.load(f)


@pytest.mark.parametrize("case", ["c2_reduced", "c3_reduced", "c4_reduced", "c5_reduced"])
def test_llpt_after_fifty_iterations_reduced(case):
    """Free-running GPU and oracle trajectories from the same initial topics diverge token by
    token, but after 50 iterations their per-token log-likelihoods agree within 1e-3 relative
    (the oracle's value: tests/golden, written on the CPU by make_llpt_goldens.py); the GPU's
    LLPT of its own state equals the oracle's LLPT of that state to 1e-12."""
    g = load_golden(case)
    c = lda_synth.make_corpus(g["workload"], **g["overrides"])
    assert lda_synth.fingerprint(c) == g["corpus_fingerprint"]
    kw = corpus_kw(c)
    say("LLPT-50 %s N=%d" % (case, c.N))
    with make_lda(c) as m:
        ll0 = m.loglik()
        m.iterate(50)
        lg = m.loglik()
        zg = m.counts(D=False, W=False)["z"]
    say("  LLPT gpu %.6f oracle %.6f" % (lg, g["llpt"]))
    assert ll0 == pytest.approx(g["llpt_trajectory"]["0"], rel=1e-12)  # the same initial state
    assert lg == pytest.approx(g["llpt"], rel=1e-3)
    assert lg == pytest.approx(oracle.llpt(c.word, c.doc, zg, **kw), rel=1e-12)
    assert lg > ll0


def test_shuffled_input_order():
    """Input not sorted by document: keys and z stay in the caller's order."""
    c = lda_synth.generate(lda_synth.SPECS["c1"], n_docs=300, shuffle=True)
    z = oracle.init_topics(c.N, c.K, SEED)
    zo, flags, _ = oracle_step(c, z, 0)
    with make_lda(c) as m:
        assert np.array_equal(m.counts(D=False, W=False)["z"], z)
        m.iterate(1)
        cnt = m.counts()
    compare_draws(cnt["z"], zo, flags, c.N)
    check_counts_are_histograms(c, cnt, c.K)


class _Tiny:
    def __init__(self, word, doc, V, K, alpha, beta=0.01):
        self.word = np.asarray(word, np.int32)
        self.doc = np.asarray(doc, np.int32)
        self.V, self.K, self.alpha, self.beta = V, K, alpha, beta
        self.n_docs = int(self.doc.max()) + 1
        self.N = self.word.shape[0]


def _edge_cases():
    rng = np.random.default_rng(77)
    yield "single_token", _Tiny([0], [0], 1, 2, 0.5)
    yield "empty_docs", _Tiny([1, 2, 2, 0], [3, 3, 9, 9], 5, 3, 0.3)
    yield "K2", _Tiny(rng.integers(0, 6, 400), np.sort(rng.integers(0, 20, 400)), 6, 2, 25.0)
    n = 30000
    yield "one_word_many_regions", _Tiny(np.zeros(n, np.int32), np.sort(rng.integers(0, 50, n)), 1, 8, 0.1)
    yield "longest_doc", _Tiny(rng.integers(0, 50, 65535), np.zeros(65535, np.int32), 50, 16, 0.2)
    yield "max_topics", _Tiny(rng.integers(0, 40, 3000), np.sort(rng.integers(0, 30, 3000)), 40, 16384, 0.01)
    yield "ragged_K", _Tiny(rng.integers(0, 300, 20000), np.sort(rng.integers(0, 200, 20000)), 300, 1013, 0.05)
    yield "max_topics_tiled", _Tiny(rng.integers(0, 40, 3000), np.sort(rng.integers(0, 30, 3000)), 40, 32768, 0.01)
    # document lengths on both sides of every chunk edge of the document-major kernels (64-token
    # chunks, 128 tokens and row slots loaded one document ahead, 32 documents per batch), with
    # empty documents in between, and rows of more than 128 entries
    lens = [0, 1, 63, 64, 65, 127, 128, 129, 191, 192, 193, 255, 256, 257, 383, 384, 385, 511, 512, 513]
    lens = [lens[(7 * i) % len(lens)] for i in range(85)]
    doc = np.repeat(np.arange(len(lens), dtype=np.int32), lens)
    word = rng.zipf(1.3, doc.shape[0]) % 400
    yield "chunk_edges", _Tiny(word, doc, 400, 301, 0.05)
    perm = rng.permutation(doc.shape[0])  # the same corpus in shuffled input order (keys are not positions)
    yield "chunk_edges_shuffled", _Tiny(word[perm], doc[perm], 400, 301, 0.05)
    # the largest K of the table-based per-word pass and W rebuild (whose LDS then passes 64 KB)
    r2 = np.random.default_rng(78)
    yield "K4095", _Tiny(r2.integers(0, 300, 20000), np.sort(r2.integers(0, 200, 20000)), 300, 4095, 0.05)


@pytest.mark.parametrize("name,c", list(_edge_cases()), ids=[e[0] for e in _edge_cases()])
def test_edge_cases(name, c):
    say("edge %s N=%d K=%d" % (name, c.N, c.K))
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    z = oracle.init_topics(c.N, c.K, SEED)
    with lda_make(c) as m:
        for t in range(3):
            zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=t, **kw)
            m.set_assignments(z, t)
            m.iterate(1)
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c.N)
            check_counts_are_histograms(c, cnt, c.K)
            z = zo
        ll = m.loglik()
    assert ll == pytest.approx(oracle.llpt(c.word, c.doc, cnt["z"], **kw), rel=1e-12, abs=1e-14)



def test_topic_list_running_out_follows_the_oracle():
    """From K = 4,096 on, a sparse word's top values come from its row and from the first topics
    outside the row in the list of the 512 topics of lowest T.  Here word 0 holds 4,094 of the
    4,096 topics, and the two it lacks carry the most tokens, so every listed topic is in its row
    and the per-word pass scans all topics instead; the draws are still the oracle's."""
    K = 4096
    rng = np.random.default_rng(31)
    n0, n1 = K - 2, 5000
    word = np.concatenate([np.zeros(n0, np.int32), np.ones(n1, np.int32), rng.integers(2, 60, 3000).astype(np.int32)])
    doc = rng.integers(0, 120, word.shape[0]).astype(np.int32)
    z = np.concatenate([rng.permutation(n0).astype(np.int32),           # word 0: topics 0..4093, once each
                        (K - 2 + np.arange(n1) % 2).astype(np.int32),   # word 1: the two topics word 0 lacks
                        rng.integers(0, K - 2, 3000).astype(np.int32)])
    order = np.argsort(doc, kind="stable")
    word, doc, z = word[order], doc[order], z[order]
    c = _Tiny(word, doc, 60, K, 0.05)
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    T = np.bincount(z, minlength=K)
    lowest = np.lexsort((np.arange(K), T))[:512]
    assert np.all(lowest < K - 2)  # every listed topic is one of word 0's
    say("topic list running out K=%d N=%d" % (K, c.N))
    with lda_make(c) as m:
        for t in range(2):
            zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=t, **kw)
            m.set_assignments(z, t)
            m.iterate(1)
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c.N)
            check_counts_are_histograms(c, cnt, c.K)
            z = zo


@pytest.mark.parametrize("K,marks,shuffle", [(64, 1, False), (64, 2, False), (1000, 0, False), (1000, 1, True),
                                              (20000, 0, False)])
def test_heavy_documents_follow_the_oracle(K, marks, shuffle):
    """Documents longer than 4,096 tokens get a whole workgroup in the doc pass and the D rebuild
    (the others one wave): with heavy documents of 4,097 to 30,000 tokens among light ones, both
    skip bitmaps, shuffled input and the tiled sampler, the draws are the oracle's and the counts
    the histograms of z.  The first snapshot gives every word one topic, so many tokens skip."""
    rng = np.random.default_rng(99)
    lens = np.concatenate([rng.integers(1, 300, 200), [4097, 8000, 30000, 4096, 12345]])
    rng.shuffle(lens)
    doc = np.repeat(np.arange(lens.shape[0], dtype=np.int32), lens)
    word = (rng.zipf(1.2, doc.shape[0]) % 500).astype(np.int32)
    if shuffle:
        perm = rng.permutation(doc.shape[0])
        word, doc = word[perm], doc[perm]
    c = _Tiny(word, doc, 500, K, 0.1)
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    z = ((c.word.astype(np.int64) * 7) % K).astype(np.int32)
    say("heavy documents K=%d marks=%d shuffle=%s N=%d" % (K, marks, shuffle, c.N))
    with lda_make(c, skip_marks=marks, always_skip_test=True) as m:
        for t in range(3):
            zo, flags, ost = oracle.iterate(c.word, c.doc, z, seed=SEED, t=t, **kw)
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c.N)
            check_counts_are_histograms(c, cnt, c.K)
            assert 0 <= ost["skip3"] - st["skip_step3"] <= max(2, 1e-3 * c.N)
            say("  t=%d skipped %d (oracle %d)" % (t, st["skip_step3"], ost["skip3"]))
            z = zo


@pytest.mark.parametrize("K", [16384, 5000])
@pytest.mark.parametrize("block", [0, 256, 512, 1024])
def test_sampler_block_sizes_at_large_K(K, block):
    """Every sampler workgroup size the LDS allows draws what the oracle draws at a
    large K (the W^ row of K fp64 values fills most of the LDS); the default picks
    one of them."""
    rng = np.random.default_rng(5)
    c = _Tiny(rng.integers(0, 60, 6000), np.sort(rng.integers(0, 40, 6000)), 60, K, 0.01)
    say("sampler block %d K=%d" % (block, K))
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    z = oracle.init_topics(c.N, c.K, SEED)
    zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=0, **kw)
    with lda_make(c, sampler_block=block) as m:
        st = m.iterate(1, stats=True)[0]
        cnt = m.counts()
    assert st["sampler_block"] == (block or st["sampler_block"]) and st["sampler_block"] in (256, 512, 1024)
    compare_draws(cnt["z"], zo, flags, c.N)
    check_counts_are_histograms(c, cnt, c.K)


def _large_k_corpus(K):
    """About 100K tokens over 40 words: the top word holds more than K tokens,
    so it is dense and split into regions; the rest are sparse."""
    rng = np.random.default_rng(11)
    n_docs, V = 1000, 40
    lens = rng.integers(60, 140, n_docs)
    p = 1.0 / np.arange(1, V + 1) ** 1.5
    word = rng.choice(V, size=int(lens.sum()), p=p / p.sum()).astype(np.int32)
    doc = np.repeat(np.arange(n_docs), lens).astype(np.int32)
    return _Tiny(word, doc, V, K, 0.05)


@pytest.mark.parametrize("K", [32768, 20000])
def test_large_k_tiled_sampler_follows_the_oracle(K):
    """K above what one workgroup's LDS holds as an fp64 row: the tiled sampler
    (two topic tiles, three passes per region) draws what the oracle draws, over
    three snapshots, with dense split words and sparse words; counts and LLPT too."""
    c = _large_k_corpus(K)
    cnt_w = np.bincount(c.word, minlength=c.V)
    assert (cnt_w > K).sum() >= 1  # a dense word, split into regions of 10,000
    say("large K=%d N=%d" % (K, c.N))
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    z = oracle.init_topics(c.N, c.K, SEED)
    with lda_make(c) as m:
        for t in range(3):
            zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=t, **kw)
            m.set_assignments(z, t)
            st = m.iterate(1, stats=True)[0]
            assert st["sampler_block"] == 1024 and st["sampled"] + st["skip_step3"] == c.N
            cnt = m.counts()
            compare_draws(cnt["z"], zo, flags, c.N)
            check_counts_are_histograms(c, cnt, c.K)
            z = zo
        ll = m.loglik()
    assert ll == pytest.approx(oracle.llpt(c.word, c.doc, cnt["z"], **kw), rel=1e-12, abs=1e-14)


def test_large_k_schedule_invariance():
    """The tiled sampler's draws do not depend on the region size."""
    c = _large_k_corpus(32768)
    with lda_make(c) as a:
        a.iterate(2)
        za = a.counts(D=False, W=False)["z"]
    with lda_make(c, region_tokens=777) as b:
        b.iterate(2)
        zb = b.counts(D=False, W=False)["z"]
    assert np.array_equal(za, zb)


def test_large_k_two_branch_follows_the_oracle():
    """The two-branch ablation through the tiled sampler and the large-K precompute
    (K = 32,768) against the oracle's two-branch form."""
    c = _large_k_corpus(32768)
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    z = oracle.init_topics(c.N, c.K, SEED)
    zo, flags, _ = oracle.iterate(c.word, c.doc, z, seed=SEED, t=0, branches=2, **kw)
    with lda_make(c, two_branch=True) as m:
        st = m.iterate(1, stats=True)[0]
        cnt = m.counts()
    compare_draws(cnt["z"], zo, flags, c.N)
    check_counts_are_histograms(c, cnt, c.K)
    assert st["skip_step3"] == 0 and st["skip_after_s"] == 0 and st["sampled"] == c.N


@pytest.mark.parametrize("opts", [dict(g=1), dict(g=3), dict(no_skip=True), dict(dense_cutoff=-1),
                                  dict(dense_cutoff=1 << 30)])
def test_large_k_options_leave_the_draws_unchanged(opts):
    """S_est depth, the skip test and the hybrid-W cutoff at K = 32,768 (tiled sampler,
    bitmap rebuilds, sparse-word precompute or its dense fallback)."""
    c = _large_k_corpus(32768)
    say("large K options %s" % opts)
    with lda_make(c) as a:
        a.iterate(2)
        za = a.counts(D=False, W=False)["z"]
        lla = a.loglik()
    with lda_make(c, **opts) as b:
        b.iterate(2)
        zb = b.counts(D=False, W=False)["z"]
        llb = b.loglik()
    assert np.array_equal(za, zb)
    assert llb == pytest.approx(lla, rel=1e-12)

def lda_make(c, **kw):
    import paper_2007_08725_amd as lda
    return lda.LDA(c.word, c.doc, c.V, c.K, c.alpha, c.beta, SEED, **kw)


def test_allocator_failure_reports_nomem(c1):
    import ctypes

    import paper_2007_08725_amd as lda
    lib = lda.load_library()
    calls = {"n": 0}

    def alloc(nbytes, ctx):
        calls["n"] += 1
        return None if calls["n"] == 4 else _pool.alloc(nbytes)

    def free(ptr, ctx):
        _pool.free(ptr)

    class Pool:
        def __init__(self):
            import torch
            self.torch = torch
            self.live = {}

        def alloc(self, n):
            t = self.torch.empty(int(n), dtype=self.torch.uint8, device="cuda")
            self.live[t.data_ptr()] = t
            return t.data_ptr()

        def free(self, p):
            self.live.pop(p)

    global _pool
    _pool = Pool()
    fa, ff = lda.ALLOC_FN(alloc), lda.FREE_FN(free)
    o = lda.Options()
    o.dev_alloc, o.dev_free = fa, ff
    h = ctypes.c_void_p()
    w = np.ascontiguousarray(c1.word)
    d = np.ascontiguousarray(c1.doc)
    st = lib.lda_create(ctypes.c_void_p(w.ctypes.data), ctypes.c_void_p(d.ctypes.data), c1.N, c1.V, c1.K, c1.alpha,
                        c1.beta, SEED, ctypes.byref(o), ctypes.byref(h))
    assert st == lda.LDA_E_NOMEM and not h.value
    assert not _pool.live  # everything allocated before the failure was released
    assert b"allocation" in lib.lda_last_error(None)


def test_set_assignments_rejects_bad_topics(c1):
    import paper_2007_08725_amd as lda
    with make_lda(c1) as m:
        z = np.zeros(c1.N, np.int32)
        z[5] = c1.K
        with pytest.raises(lda.LDAError) as ei:
            m.set_assignments(z, 0)
        assert ei.value.status == lda.LDA_E_ARG
        m.iterate(1)  # the handle is still usable


def test_create_rejects_too_long_document():
    import ctypes

    import paper_2007_08725_amd as lda
    lib = lda.load_library()
    n = lda.MAX_DOC_LEN + 1
    w = np.zeros(n, np.int32)
    d = np.zeros(n, np.int32)
    d[-1] = 0
    h = ctypes.c_void_p()
    st = lib.lda_create(ctypes.c_void_p(w.ctypes.data), ctypes.c_void_p(d.ctypes.data), n, 1, 4, 0.5, 0.01, SEED,
                        None, ctypes.byref(h))
    assert st == lda.LDA_E_RANGE and not h.value
    assert b"65535" in lib.lda_last_error(None)
