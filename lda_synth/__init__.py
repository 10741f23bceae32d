"""Seeded planted-LDA corpora: the synthetic stand-ins for the paper's datasets.

The paper evaluates on NYTimes (~100M tokens), PubMed (738M tokens) and UMBC
(1.33B tokens) (Sec. 6, "Dataset").  None of them is available, so every
workload here is a planted LDA corpus with the same shape: document count,
length distribution, vocabulary size and a Zipf word-frequency base (the
power-law token distribution of Sec. 5.1, Fig. 8).

This module holds no sampler arithmetic.  It is the one input source shared by
the oracle's tests, the GPU parity tests and the benchmark.

``make_corpus(name, scale=1.0)`` returns a :class:`Corpus` with int32 ``word``
and ``doc`` arrays (doc-sorted unless ``shuffle=True``), the vocabulary size
``V`` and the fit parameters (``K``, ``alpha``, ``beta``, ``iters``).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "planted.c")
_LIB_PATH = os.path.join(_HERE, "_planted.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the generator with gcc (host code only)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-pthread", "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        lib.synth_perm.argtypes = [ctypes.c_int, ctypes.c_uint64, P]
        lib.synth_phi_alias.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_double,
                                        ctypes.c_uint64, ctypes.c_int, P, P, P]
        lib.synth_tokens.argtypes = [ctypes.c_int64, P, P, ctypes.c_int, ctypes.c_double, ctypes.c_int, P, P,
                                     ctypes.c_uint64, ctypes.c_int, P, P, P]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


@dataclasses.dataclass
class CorpusSpec:
    """Shape of one planted corpus and the LDA fit run on it."""
    name: str
    n_docs: int
    length: tuple          # ("poisson", mean) | ("lognormal", mean, sigma, cap)
    V: int
    zipf_s: float
    true_topics: int
    K: int
    alpha: float
    beta: float = 0.01
    iters: int = 50
    seed: int = 1001
    eta_scale: float = 0.05
    theta_conc: float = 0.1


# The five workloads, plus c6 for the largest topic count.  c4 and c6 reuse
# c2's corpus (same seed) with K = 10,000 and K = 32,768.
SPECS = {
    "c1": CorpusSpec("c1", 1_000, ("poisson", 50.0), 2_000, 1.0, 20, 16, 50.0 / 16, iters=10, seed=1001),
    "c2": CorpusSpec("c2", 300_000, ("poisson", 330.0), 102_000, 1.07, 200, 1000, 0.05, seed=1002),
    "c3": CorpusSpec("c3", 8_200_000, ("lognormal", 90.0, 0.8, None), 141_000, 1.1, 500, 1000, 0.05, seed=1003),
    "c4": CorpusSpec("c4", 300_000, ("poisson", 330.0), 102_000, 1.07, 200, 10_000, 0.1, seed=1002),
    "c5": CorpusSpec("c5", 20_000_000, ("lognormal", 150.0, 1.5, 50_000), 1_000_000, 1.2, 1000, 1000, 0.05,
                     seed=1005),
    "c6": CorpusSpec("c6", 300_000, ("poisson", 330.0), 102_000, 1.07, 200, 32_768, 0.05, seed=1002),
}

SAMPLER_SEED = 42


@dataclasses.dataclass
class Corpus:
    spec: CorpusSpec
    word: np.ndarray       # int32 [N]
    doc: np.ndarray        # int32 [N]
    V: int
    n_docs: int
    topic: np.ndarray | None = None   # planted topics (diagnostics only)

    @property
    def N(self) -> int:
        return int(self.word.shape[0])

    @property
    def K(self) -> int:
        return self.spec.K

    @property
    def alpha(self) -> float:
        return self.spec.alpha

    @property
    def beta(self) -> float:
        return self.spec.beta


def doc_lengths(spec: CorpusSpec, n_docs: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng([seed, 7])
    kind = spec.length[0]
    if kind == "poisson":
        L = rng.poisson(spec.length[1], size=n_docs)
    elif kind == "lognormal":
        mean, sigma, cap = spec.length[1], spec.length[2], spec.length[3]
        mu = math.log(mean) - 0.5 * sigma * sigma
        L = np.rint(rng.lognormal(mu, sigma, size=n_docs))
        if cap is not None:
            L = np.minimum(L, cap)
    else:
        raise ValueError(kind)
    return np.maximum(L, 1).astype(np.int32)


def generate(spec: CorpusSpec, *, n_docs: int | None = None, V: int | None = None, shuffle: bool = False,
             nthreads: int | None = None, keep_topics: bool = False) -> Corpus:
    lib = _load()
    n_docs = spec.n_docs if n_docs is None else int(n_docs)
    V = spec.V if V is None else int(V)
    if nthreads is None:
        nthreads = max(1, min(16, os.cpu_count() or 1))
    seed = spec.seed
    lens = doc_lengths(spec, n_docs, seed)
    start = np.zeros(n_docs + 1, dtype=np.int64)
    np.cumsum(lens, out=start[1:])
    N = int(start[-1])
    perm = np.empty(V, dtype=np.uint32)
    lib.synth_perm(V, seed, _ptr(perm))
    J = spec.true_topics
    prob = np.empty((J, V), dtype=np.float32)
    alias = np.empty((J, V), dtype=np.uint32)
    rc = lib.synth_phi_alias(V, spec.zipf_s, J, spec.eta_scale, seed, nthreads, _ptr(perm), _ptr(prob), _ptr(alias))
    if rc:
        raise RuntimeError("synth_phi_alias failed")
    word = np.empty(N, dtype=np.int32)
    doc = np.empty(N, dtype=np.int32)
    topic = np.empty(N, dtype=np.int32) if keep_topics else None
    rc = lib.synth_tokens(n_docs, _ptr(lens), _ptr(start), J, spec.theta_conc, V, _ptr(prob), _ptr(alias), seed,
                          nthreads, _ptr(word), _ptr(doc), _ptr(topic) if topic is not None else None)
    if rc:
        raise RuntimeError("synth_tokens failed")
    del prob, alias
    if shuffle:
        order = np.random.default_rng([seed, 11]).permutation(N)
        word, doc = word[order], doc[order]
        if topic is not None:
            topic = topic[order]
    return Corpus(spec, word, doc, V, n_docs, topic)


def make_corpus(name: str, *, n_docs: int | None = None, V: int | None = None, K: int | None = None,
                shuffle: bool = False, nthreads: int | None = None) -> Corpus:
    """Named workload, optionally reduced (fewer docs, smaller vocabulary) or refit with another K."""
    spec = SPECS[name]
    if K is not None:
        spec = dataclasses.replace(spec, K=int(K))
    return generate(spec, n_docs=n_docs, V=V, shuffle=shuffle, nthreads=nthreads)


def fingerprint(c: Corpus) -> str:
    """Hash of a corpus's shape and of a strided sample of its tokens (cheap at
    any size): stored next to values computed from a corpus, so that a changed
    generator shows up as such."""
    import hashlib
    h = hashlib.sha256()
    step = max(1, c.N // 4_000_000)
    for a in (np.array([c.N, c.V, c.n_docs, c.K], np.int64), c.word[::step], c.doc[::step],
              np.array([int(c.word.sum(dtype=np.int64)), int(c.doc.sum(dtype=np.int64))], np.int64)):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def concentrated(n_docs: int = 4000, K: int = 64, words_per_topic: int = 40, single_frac: float = 0.6,
                 mean_len: float = 60.0, alpha: float = 0.1, beta: float = 0.01, seed: int = 1009) -> Corpus:
    """A corpus whose planted assignment is already concentrated, for tests that
    need a high step-3 skip rate from the first iteration on.

    Topic j owns words [j*words_per_topic, (j+1)*words_per_topic).  A fraction
    ``single_frac`` of the documents draws every token from one topic (the
    planted topic of each of those tokens); the other documents mix three
    topics, and their tokens' planted topics are uniform over K.  Documents are
    sorted (doc ids ascend).  ``topic`` holds the planted assignment.
    """
    rng = np.random.default_rng([seed, 3])
    V = K * words_per_topic
    lens = np.maximum(rng.poisson(mean_len, n_docs), 1)
    doc = np.repeat(np.arange(n_docs, dtype=np.int32), lens)
    N = int(doc.shape[0])
    single = rng.random(n_docs) < single_frac
    main = rng.integers(0, K, n_docs)
    mix = rng.integers(0, K, (n_docs, 3))
    pick = rng.integers(0, 3, N)
    src = np.where(single[doc], main[doc], mix[doc, pick])          # topic each token's word comes from
    word = (src * words_per_topic + rng.integers(0, words_per_topic, N)).astype(np.int32)
    topic = np.where(single[doc], main[doc], rng.integers(0, K, N)).astype(np.int32)
    spec = CorpusSpec("concentrated", n_docs, ("poisson", mean_len), V, 0.0, K, K, alpha, beta=beta, iters=3,
                      seed=seed)
    return Corpus(spec, word, doc, V, n_docs, topic)
