"""Helpers shared by the GPU parity tests (no sampler arithmetic here)."""
import sys

import numpy as np

import oracle
import paper_2007_08725_amd as lda

SEED = 42


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def corpus_kw(c, K=None, alpha=None):
    return dict(M=c.n_docs, V=c.V, K=c.K if K is None else K, alpha=c.alpha if alpha is None else alpha,
                beta=c.beta)


def histograms(word, doc, z, M, V, K):
    """D, W (dense, int64) and T as brute-force histograms of an assignment."""
    D = np.bincount(doc.astype(np.int64) * K + z, minlength=M * K).reshape(M, K)
    W = np.bincount(word.astype(np.int64) * K + z, minlength=V * K).reshape(V, K)
    return D, W, W.sum(axis=0)


def csr_to_dense(off, topic, count, rows, K):
    out = np.zeros((rows, K), np.int64)
    r = np.repeat(np.arange(rows), np.diff(off))
    out[r, topic] = count
    return out


def _csr_keys(off, topic, K):
    row_of = np.repeat(np.arange(off.shape[0] - 1, dtype=np.int64), np.diff(off))
    return row_of * K + topic


def check_counts_are_histograms(c, counts, K):
    """The GPU's D, W and T are exactly the histograms of the GPU's own z (bit-exact rebuild).

    Brute force by sorting: the unique (row, topic) keys of the tokens, with
    their multiplicities, are the CSR rows in ascending order.
    """
    z = counts["z"].astype(np.int64)
    assert z.min() >= 0 and z.max() < K
    assert np.array_equal(counts["T"], np.bincount(z, minlength=K))
    for ids, o, t, cnt in ((c.doc, counts["D_off"], counts["D_topic"], counts["D_count"]),
                           (c.word, counts["W_off"], counts["W_topic"], counts["W_count"])):
        keys, mult = np.unique(ids.astype(np.int64) * K + z, return_counts=True)
        assert np.array_equal(_csr_keys(o, t, K), keys)
        assert np.array_equal(cnt, mult)


def compare_draws(z_gpu, z_ora, flags, N):
    """Every mismatch must be a flagged near-boundary draw, and fewer than 1e-6 * N of them."""
    bad = np.nonzero(z_gpu != z_ora)[0]
    unflagged = bad[(flags[bad] & 1) == 0]
    assert unflagged.size == 0, "unflagged mismatches at tokens %s" % unflagged[:10].tolist()
    assert bad.size <= 1e-6 * N, "%d flagged mismatches" % bad.size
    return bad.size


def make_lda(c, K=None, alpha=None, **kw):
    return lda.LDA(c.word, c.doc, c.V, c.K if K is None else K, c.alpha if alpha is None else alpha, c.beta, SEED,
                   **kw)


def oracle_step(c, z, t, K=None, alpha=None, **kw):
    return oracle.iterate(c.word, c.doc, z, seed=SEED, t=t, **corpus_kw(c, K, alpha), **kw)
