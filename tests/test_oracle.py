"""Pins for the oracle (CPU only).

Each test ties the oracle to something other than itself: the paper's worked
example (Sec. 2.2), rocRAND's Philox4x32-10, the closed-form conditional of
Eq. 1 (exact segment layout and a chi-square test), closed-form limits of the
LLPT, brute-force count tables, and the agreement of two independent forms
(dense brute force vs sparse decomposition).
"""
import json
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats as sps

import oracle as ora

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def _counts_np(word, doc, z, M, V, K):
    D = np.zeros((M, K), np.int64)
    W = np.zeros((V, K), np.int64)
    np.add.at(D, (np.asarray(doc), np.asarray(z)), 1)
    np.add.at(W, (np.asarray(word), np.asarray(z)), 1)
    return D, W, W.sum(axis=0)


def _eq1_layout(word, doc, z, M, V, K, alpha, beta, i, branches=3):
    """Canonical segments written from Eq. 1 with numpy: [K1 | S' asc | Q' asc] of Eq. 5, or the
    two-branch [S asc | Q asc] of Sec. 2.2."""
    D, W, T = _counts_np(word, doc, z, M, V, K)
    wh = (W[word[i]] + beta) / (T + V * beta)
    d = doc[i]
    if branches == 3:
        k1 = int(np.argmax(wh))  # first maximum = lowest topic id
        segs = [(k1, (D[d, k1] + alpha) * wh[k1])]
        segs += [(k, D[d, k] * wh[k]) for k in range(K) if k != k1 and D[d, k] > 0]
        segs += [(k, alpha * wh[k]) for k in range(K) if k != k1]
    else:
        segs = [(k, D[d, k] * wh[k]) for k in range(K) if D[d, k] > 0]
        segs += [(k, alpha * wh[k]) for k in range(K)]
    p = (D[d] + alpha) * wh  # Eq. 1 numerator
    return segs, p / p.sum()


def _tiny_case():
    """3 docs, 5 words, 4 topics (the closed-form brute-force case)."""
    word = np.array([0, 1, 2, 0, 3, 4, 1, 2, 0, 3, 3, 4], np.int32)
    doc = np.array([0, 0, 0, 0, 0, 1, 1, 1, 2, 2, 2, 2], np.int32)
    z = np.array([0, 1, 2, 3, 0, 1, 1, 2, 3, 3, 0, 2], np.int32)
    return word, doc, z, dict(M=3, V=5, K=4, alpha=0.5, beta=0.01)


def _random_corpus(rng, max_m=20, max_v=30, kmin=2, kmax=8, max_n=200):
    M = int(rng.integers(1, max_m + 1))
    V = int(rng.integers(1, max_v + 1))
    K = int(rng.integers(kmin, kmax + 1))
    n = int(rng.integers(1, max_n + 1))
    word = rng.integers(0, V, n).astype(np.int32)
    doc = rng.integers(0, M, n).astype(np.int32)
    return word, doc, M, V, K


# ---------------------------------------------------------------- worked example

@pytest.fixture(scope="module")
def wex():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        return json.load(f)


def _wex_args(w):
    return (np.array(w["word"], np.int32), np.array(w["doc"], np.int32), np.array(w["topic"], np.int32),
            dict(M=w["M"], V=w["V"], K=w["K"], alpha=w["alpha"], beta=w["beta"]))


def test_worked_example_counts(wex):
    word, doc, z, kw = _wex_args(wex)
    c = ora.build_counts(word, doc, z, kw["M"], kw["V"], kw["K"])
    assert c["T"].tolist() == wex["printed"]["T"]
    assert c["W"][0].tolist() == wex["printed"]["W0"]
    d2 = np.zeros(kw["K"], np.int64)
    sl = slice(c["doff"][2], c["doff"][3])
    d2[c["dtop"][sl]] = c["dcnt"][sl]
    assert d2.tolist() == wex["printed"]["D2"]
    assert c["len"].tolist() == [2, 2, 3]


def test_worked_example_what_and_two_branch(wex):
    """W^[0] o alpha, W^[0] o D[2], the Q prefix, the branch test and the new topic (Sec. 2.2)."""
    word, doc, z, kw = _wex_args(wex)
    pr = wex["printed"]
    wh = ora.what_row(word, doc, z, 0, M=kw["M"], V=kw["V"], K=kw["K"], beta=kw["beta"])
    np.testing.assert_allclose(kw["alpha"] * wh, pr["alpha_times_What0"], rtol=2e-3)
    np.testing.assert_allclose(wh * np.array(pr["D2"]), pr["What0_times_D2"], rtol=2e-3, atol=5e-5)
    q = np.cumsum(kw["alpha"] * wh)
    np.testing.assert_allclose(q, pr["Q_prefix"], rtol=2e-3)
    S = float(np.sum(wh * np.array(pr["D2"])))
    Q = float(q[-1])
    u = pr["u"]
    assert not (u <= S / (S + Q))           # the Q branch is taken
    x = (1 - u) * (S + Q)
    assert x == pytest.approx(pr["reflected_u_times_SQ"], rel=2e-3)
    assert int(np.argmax(q > x)) == pr["new_topic"]   # descending the Q tree
    # the oracle's canonical three-branch draw with the same u gives the same topic
    k, Z, flag = ora.draw_given_u(word, doc, z, wex["token_index"], u, **kw)
    assert k == pr["new_topic"]
    kd, Zd, flagd = ora.draw_given_u(word, doc, z, wex["token_index"], u, mode="dense", **kw)
    assert (kd, Zd, flagd) == (k, Z, flag)
    # the two-branch form, drawn forward over [S | Q]: x = u*(S+Q) lies past S and falls into
    # Q at the same topic, with the same total
    k2, Z2, _ = ora.draw_given_u(word, doc, z, wex["token_index"], u, branches=2, **kw)
    assert k2 == pr["new_topic"]
    assert Z2 == pytest.approx(S + Q, rel=1e-12) and Z2 == pytest.approx(Z, rel=1e-12)
    assert u * Z2 > S and u * Z2 - S < q[pr["new_topic"]] and u * Z2 - S >= q[pr["new_topic"] - 1]


def test_worked_example_three_branch(wex):
    """K1/K2, a1..a3, M, S', S_est, Q', Z of Eq. 5-9 on the example token."""
    word, doc, z, kw = _wex_args(wex)
    dv = wex["derived_three_branch_not_printed"]
    ws = ora.word_stats(word, doc, z, **kw)
    assert (ws["K1"][0], ws["K2"][0]) == (dv["K1"], dv["K2"])
    for key in ("a1", "a2", "a3"):
        assert ws[key][0] == pytest.approx(dv[key], rel=1e-4)
    assert ws["Qp"][0] == pytest.approx(dv["Q_prime"], rel=1e-5)
    _, Z, flag = ora.draw_given_u(word, doc, z, wex["token_index"], wex["printed"]["u"], **kw)
    assert Z == pytest.approx(dv["Z"], rel=1e-6)
    assert bool(flag & 2) == dv["skip3"]
    Mm = ws["a1"][0] * (0 + kw["alpha"])
    assert Mm == pytest.approx(dv["Mmax"], rel=1e-6)
    assert Z - Mm - ws["Qp"][0] == pytest.approx(dv["S_prime"], rel=1e-5)


# ------------------------------------------------------------------- Philox

def test_philox_matches_rocrand():
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = os.path.join(os.environ.get("TMPDIR", "/tmp"), "rocrand_philox_kat_%d" % os.getpid())
    subprocess.run([hipcc, "-O1", "-o", exe, os.path.join(HERE, "pins", "rocrand_philox_kat.cpp")], check=True,
                   capture_output=True)
    rng = np.random.default_rng(5)
    cases = [(42, 0, 0, 0, 0), (42, 5, 0, 3, 0), (2**64 - 1, 2**32 - 1, 2**30 - 1, 2**32 - 1, 2**32 - 1)]
    for _ in range(200):
        cases.append((int(rng.integers(0, 2**63)), int(rng.integers(0, 2**32)), int(rng.integers(0, 2**30)),
                      int(rng.integers(0, 2**32)), int(rng.integers(0, 2))))
    inp = "".join("%d %d %d %d %d\n" % c for c in cases)
    out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    os.unlink(exe)
    for c, line in zip(cases, out):
        want = [int(x) for x in line.split()]
        got = ora.philox(c[1:], [c[0] & 0xFFFFFFFF, c[0] >> 32]).tolist()
        assert got == want, c


def test_uniform_and_init_follow_the_stated_layout():
    """u and the initial topics as the boundary states them, from Philox words that rocRAND's
    engine computes (not the oracle's Philox): u = ((x0 << 32 | x1) >> 11) * 2^-53 at counter
    (i, 0, t, 0) and z0 = (x0 * K) >> 32 at counter (i, 0, 0, 1), key = seed.  A swapped
    word, a shift by another amount or a counter slot moved would change the bits."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = os.path.join(os.environ.get("TMPDIR", "/tmp"), "rocrand_philox_layout_%d" % os.getpid())
    subprocess.run([hipcc, "-O1", "-o", exe, os.path.join(HERE, "pins", "rocrand_philox_kat.cpp")], check=True,
                   capture_output=True)
    rng = np.random.default_rng(11)
    draws = [(int(rng.integers(0, 2**63)), int(rng.integers(0, 2**32)), int(rng.integers(0, 200))) for _ in range(100)]
    inits = [(int(rng.integers(0, 2**63)), int(rng.integers(0, 2**20)), int(rng.integers(1, 40000))) for _ in range(100)]
    inp = "".join("%d %d 0 %d 0\n" % (seed, i, t) for seed, i, t in draws)
    inp += "".join("%d %d 0 0 1\n" % (seed, i) for seed, i, _ in inits)
    out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    os.unlink(exe)
    words = [[int(x) for x in line.split()] for line in out[:len(draws) + len(inits)]]
    for (seed, i, t), x in zip(draws, words[:len(draws)]):
        want = float(((x[0] << 32) | x[1]) >> 11) * 2.0**-53
        assert ora.uniform(seed, t, i) == want, (seed, i, t)
    for (seed, i, K), x in zip(inits, words[len(draws):]):
        z = ora.init_topics(i + 1, K, seed)
        assert int(z[i]) == (x[0] * K) >> 32, (seed, i, K)


def test_uniform_and_init_are_uniform():
    n = 200_000
    z = ora.init_topics(n, 16, 42)
    obs = np.bincount(z, minlength=16)
    assert sps.chisquare(obs).pvalue > 1e-3
    u = np.array([ora.uniform(42, 3, i) for i in range(20_000)])
    assert u.min() >= 0.0 and u.max() < 1.0
    assert sps.kstest(u, "uniform").pvalue > 1e-3
    # the counter layout keys on (token, iteration): different t give different draws
    assert ora.uniform(42, 0, 7) != ora.uniform(42, 1, 7)
    assert ora.uniform(42, 0, 7) != ora.uniform(43, 0, 7)


# --------------------------------------------------------- closed form, Eq. 1

@pytest.mark.parametrize("branches", [3, 2])
@pytest.mark.parametrize("mode", ["sparse", "dense"])
def test_canonical_layout_from_eq1(mode, branches):
    """Every segment of [K1 | S' | Q'] (or the two-branch [S | Q]) built from Eq. 1 maps to its
    topic; edges are flagged."""
    cases = [_tiny_case()]
    rng = np.random.default_rng(17)
    for _ in range(6):
        word, doc, M, V, K = _random_corpus(rng, max_n=40)
        z = rng.integers(0, K, len(word)).astype(np.int32)
        cases.append((word, doc, z, dict(M=M, V=V, K=K, alpha=float(rng.uniform(0.05, 3)), beta=0.01)))
    for word, doc, z, kw in cases:
        for i in range(len(word)):
            segs, _ = _eq1_layout(word, doc, z, kw["M"], kw["V"], kw["K"], kw["alpha"], kw["beta"], i, branches)
            w = np.array([s[1] for s in segs])
            cum = np.concatenate([[0.0], np.cumsum(w)])
            Z = cum[-1]
            for j, (k, width) in enumerate(segs):
                if width <= 1e-6 * Z:
                    continue
                got, Zo, flag = ora.draw_given_u(word, doc, z, i, 0.5 * (cum[j] + cum[j + 1]) / Z, mode=mode,
                                                 branches=branches, **kw)
                assert got == k and not (flag & 1)
                assert Zo == pytest.approx(Z, rel=1e-12)
            # a draw exactly on an inner edge is flagged as near-boundary
            j = 1
            if cum[j] / Z < 1.0:
                _, _, flag = ora.draw_given_u(word, doc, z, i, cum[j] / Z, mode=mode, branches=branches, **kw)
                assert flag & 1


@pytest.mark.parametrize("branches", [3, 2])
def test_chi2_against_closed_form(branches):
    """10^6 Philox-driven draws on the 3-doc/5-word/4-topic case vs Eq. 1 (chi-square, p = 0.001)."""
    word, doc, z, kw = _tiny_case()
    n = len(word)
    iters = 1_000_000 // n + 1
    hist = np.zeros((n, kw["K"]), np.int64)
    for t in range(iters):
        zn, _, _ = ora.iterate(word, doc, z, seed=2024, t=t, branches=branches, **kw)
        hist[np.arange(n), zn] += 1
    total = 0.0
    for i in range(n):
        _, p = _eq1_layout(word, doc, z, kw["M"], kw["V"], kw["K"], kw["alpha"], kw["beta"], i)
        exp = p * iters
        chi = float(((hist[i] - exp) ** 2 / exp).sum())
        assert chi < sps.chi2.ppf(0.999, kw["K"] - 1), (i, hist[i], exp)
        total += chi
    assert total < sps.chi2.ppf(0.999, n * (kw["K"] - 1))


# ------------------------------------------------- dense == sparse, bit-exact

def test_dense_and_sparse_forms_bit_identical():
    rng = np.random.default_rng(123)
    for seed in range(20):
        word, doc, M, V, K = _random_corpus(rng)
        kw = dict(M=M, V=V, K=K, alpha=float(rng.choice([50.0 / K, 0.1, 1.0])), beta=0.01)
        z = ora.init_topics(len(word), K, seed)
        g = 1 + seed % 3
        br = 2 if seed % 4 == 3 else 3
        for t in range(20):
            zs, fs, ss, Zs = ora.iterate(word, doc, z, seed=seed, t=t, mode="sparse", g=g, want_Z=True, branches=br,
                                         **kw)
            zd, fd, sd, Zd = ora.iterate(word, doc, z, seed=seed, t=t, mode="dense", g=g, want_Z=True, branches=br,
                                         **kw)
            assert np.array_equal(zs, zd) and np.array_equal(fs, fd)
            assert np.array_equal(Zs.view(np.uint64), Zd.view(np.uint64))
            assert ss == sd
            assert ss["sest_violations"] == 0 and ss["skip_not_k1"] == 0
            z = zs


def test_subset_draws_equal_full_draws():
    rng = np.random.default_rng(9)
    word, doc, M, V, K = _random_corpus(rng, max_n=300)
    kw = dict(M=M, V=V, K=K, alpha=0.3, beta=0.01)
    z = ora.init_topics(len(word), K, 1)
    full, ff, _ = ora.iterate(word, doc, z, seed=1, t=4, **kw)
    idx = rng.choice(len(word), size=min(50, len(word)), replace=False)
    sub, fs, _ = ora.iterate(word, doc, z, seed=1, t=4, idx=idx, **kw)
    assert np.array_equal(full[idx], sub) and np.array_equal(ff[idx], fs)


# ------------------------------------------------------------ count tables

def test_count_tables_match_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(10):
        word, doc, M, V, K = _random_corpus(rng, max_n=500)
        z = rng.integers(0, K, len(word)).astype(np.int32)
        c = ora.build_counts(word, doc, z, M, V, K)
        D, W, T = _counts_np(word, doc, z, M, V, K)
        assert np.array_equal(c["W"], W) and np.array_equal(c["T"], T)
        for d in range(M):
            sl = slice(c["doff"][d], c["doff"][d + 1])
            tops = c["dtop"][sl]
            assert np.all(np.diff(tops) > 0)          # ascending, unique
            assert np.all(c["dcnt"][sl] > 0)
            row = np.zeros(K, np.int64)
            row[tops] = c["dcnt"][sl]
            assert np.array_equal(row, D[d])
        # invariants: sum_k D = len, sum_d D = sum_v W = T, sum T = N
        assert np.array_equal(D.sum(1), c["len"])
        assert np.array_equal(D.sum(0), T) and np.array_equal(W.sum(0), T)
        assert T.sum() == len(word)


# -------------------------------------------------------------- skip exactness

@pytest.fixture(scope="module")
def c1():
    import lda_synth
    return lda_synth.make_corpus("c1")


def test_skip_bound_and_exactness_on_c1(c1):
    """S' <= S_est on every token and 'skip => K1' on all 10 iterations of c1 (Eq. 8-9), for
    g = 1, 2, 3.  S_est(g+1) - S_est(g) = (a_{g+2} - a_{g+1}) * (the tokens outside K1..K_{g+1})
    <= 0, so every token that skips at depth g also skips at depth g+1."""
    kw = dict(M=c1.n_docs, V=c1.V, K=c1.K, alpha=c1.alpha, beta=c1.beta)
    z = ora.init_topics(c1.N, c1.K, 42)
    skips = []
    for t in range(10):
        runs = [ora.iterate(c1.word, c1.doc, z, seed=42, t=t, g=g, **kw) for g in (1, 2, 3)]
        for zg, fg, stg in runs:
            assert np.array_equal(zg, runs[1][0])  # g changes statistics, never draws
            assert stg["sest_violations"] == 0 and stg["skip_not_k1"] == 0
        for (_, fa, sa), (_, fb, sb) in zip(runs, runs[1:]):
            assert sb["skip3"] >= sa["skip3"]      # a tighter bound skips at least as often
            assert np.all((fb & 2) >= (fa & 2))    # token by token
        skips.append(runs[1][2]["skip3"])
        assert runs[1][2]["flagged"] < 1e-3 * c1.N
        z = runs[1][0]
    assert skips[-1] > skips[0]


def test_top_values_for_depth_three_by_hand():
    """K3 and a4 of Eq. 9 (g = 3) on a case worked by hand.  V = 2, K = 5, beta = 1/2 (so
    V*beta = 1); word 0 holds topics {0,0,0,2,3,3}, word 1 topics {0,1,1,2}; T = (4,2,2,2,0),
    den = T + 1 = (5,3,3,3,1).
      W^[0] = (3.5/5, 0.5/3, 1.5/3, 2.5/3, 0.5/1) = (0.7, 1/6, 0.5, 5/6, 0.5):
              K1 = 3, K2 = 0, K3 = 2 (0.5 at topics 2 and 4: the lower id), a3 = 0.5, a4 = 0.5;
      W^[1] = (1.5/5, 2.5/3, 1.5/3, 0.5/3, 0.5/1) = (0.3, 5/6, 0.5, 1/6, 0.5):
              K1 = 1, K2 = 2 (the tie again), K3 = 4, a3 = 0.5, a4 = 0.3."""
    word = np.array([0] * 6 + [1] * 4, np.int32)
    z = np.array([0, 0, 0, 2, 3, 3, 0, 1, 1, 2], np.int32)
    doc = np.zeros(10, np.int32)
    st = ora.word_stats(word, doc, z, M=1, V=2, K=5, alpha=0.3, beta=0.5)
    assert st["K1"].tolist() == [3, 1] and st["K2"].tolist() == [0, 2] and st["K3"].tolist() == [2, 4]
    assert st["a1"] == pytest.approx([2.5 / 3, 2.5 / 3], rel=1e-15)
    assert st["a2"] == pytest.approx([0.7, 0.5], rel=1e-15)
    assert st["a3"] == pytest.approx([0.5, 0.5], rel=1e-15)
    assert st["a4"] == pytest.approx([0.5, 0.3], rel=1e-15)
    # Q' = alpha * (sum of W^ over the topics other than K1)
    assert st["Qp"] == pytest.approx([0.3 * (0.7 + 0.5 / 3 + 0.5 + 0.5), 0.3 * (0.3 + 0.5 + 0.5 / 3 + 0.5)],
                                     rel=1e-14)


# ------------------------------------------------- snapshots for large corpora

def test_restricted_snapshot_draws_equal_the_full_snapshot():
    """Counts built only for the words and documents of a token sample give the sample's draws,
    normalisers, flags and statistics bit for bit as the full snapshot does, in every form."""
    rng = np.random.default_rng(21)
    for trial in range(12):
        word, doc, M, V, K = _random_corpus(rng, max_m=40, max_v=50, kmax=12, max_n=600)
        z = rng.integers(0, K, len(word)).astype(np.int32)
        idx = np.sort(rng.choice(len(word), max(1, len(word) // 5), replace=False))
        kw = dict(M=M, V=V, K=K, alpha=0.3, beta=0.02, seed=7, t=trial, idx=idx, want_Z=True)
        for mode in ("sparse", "dense"):
            for branches, g in ((3, 1), (3, 2), (3, 3), (2, 2)):
                full = ora.iterate(word, doc, z, mode=mode, branches=branches, g=g, **kw)
                sub = ora.iterate(word, doc, z, mode=mode, branches=branches, g=g, restricted=True, **kw)
                for a, b in zip(full, sub):
                    if isinstance(a, dict):
                        assert a == b
                    else:
                        assert np.array_equal(a, b)


def test_threaded_draws_equal_single_thread(c1):
    """Token ranges drawn from one snapshot by several host threads reproduce the single-threaded
    iteration exactly (each draw depends on (seed, t, i) and the snapshot only); the threaded
    LLPT differs from the sequential one by summation rounding only; threaded initial topics are
    the same topics."""
    kw = dict(M=c1.n_docs, V=c1.V, K=c1.K, alpha=c1.alpha, beta=c1.beta)
    z = ora.init_topics(c1.N, c1.K, 42)
    assert np.array_equal(z, ora.init_topics(c1.N, c1.K, 42, threads=4))
    big = ora.init_topics(3 << 20, 1000, 42)
    assert np.array_equal(big, ora.init_topics(3 << 20, 1000, 42, threads=5))
    for t in range(2):
        a = ora.iterate(c1.word, c1.doc, z, seed=42, t=t, **kw)
        b = ora.iterate_threaded(c1.word, c1.doc, z, seed=42, t=t, threads=3, **kw)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]
        z = a[0]
    assert ora.llpt_threaded(c1.word, c1.doc, z, threads=3, **kw) == pytest.approx(
        ora.llpt(c1.word, c1.doc, z, **kw), rel=1e-14)


# ---------------------------------------------------------------------- LLPT

def test_llpt_closed_form_limits():
    rng = np.random.default_rng(8)
    for _ in range(5):
        word, doc, M, V, K = _random_corpus(rng, max_n=300)
        z = rng.integers(0, K, len(word)).astype(np.int32)
        # one word: W^[0][k] = 1 for every k, and the doc mixture sums to 1 -> LLPT = 0
        w1 = np.zeros_like(word)
        for mode in ("sparse", "dense"):
            assert abs(ora.llpt(w1, doc, z, M=M, V=1, K=K, alpha=0.7, beta=0.01, mode=mode)) < 1e-12
        # beta -> infinity: W^ -> 1/V for every k -> LLPT = -log2 V
        for mode in ("sparse", "dense"):
            got = ora.llpt(word, doc, z, M=M, V=V, K=K, alpha=0.7, beta=1e13, mode=mode)
            assert got == pytest.approx(-math.log2(V), abs=1e-9)
        a = ora.llpt(word, doc, z, M=M, V=V, K=K, alpha=0.2, beta=0.01, mode="sparse")
        b = ora.llpt(word, doc, z, M=M, V=V, K=K, alpha=0.2, beta=0.01, mode="dense")
        assert a == pytest.approx(b, rel=1e-13)


def test_llpt_rises_on_c1(c1):
    """LLPT increases as sampling proceeds (Sec. 2.2, evaluation metric)."""
    kw = dict(M=c1.n_docs, V=c1.V, K=c1.K, alpha=c1.alpha, beta=c1.beta)
    traj = ora.run(c1.word, c1.doc, seed=42, iters=10, **kw)
    ll = [ora.llpt(c1.word, c1.doc, z, **kw) for z in traj]
    assert all(b > a for a, b in zip(ll, ll[1:]))
    assert ll[-1] > ll[0] + 0.03
