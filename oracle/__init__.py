"""Python wrapper of the LDA oracle (plain single-threaded C, fp64).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the GPU library (``paper_2007_08725_amd``) and the library never calls it.

Every function follows the paper's definitions (arXiv 2007.08725):
  * ``iterate``  -- one synchronous ESCA iteration, Sec. 2.2 Eq. 1-2, drawn in
                    the three-branch canonical order of Sec. 3.2 Eq. 5;
                    ``mode="dense"`` is the brute-force form over all K topics,
                    ``mode="sparse"`` the decomposition over nz(D[d]).
  * ``llpt``     -- log-likelihood per token (log2), Sec. 2.2.
  * ``build_counts`` -- D (CSR), W (dense), T = column sums of W, Sec. 2.2.
  * ``philox``, ``uniform``, ``init_topics`` -- Philox4x32-10 draws
                    (Salmon et al., SC'11); the paper only says u ~ U[0,1].
  * ``Snapshot``   -- one counts snapshot drawn from in several calls: whole
                    token ranges from several host threads (``iterate_threaded``,
                    ``llpt_threaded``), or the words and documents of a token
                    sample only (``iterate(..., idx=..., restricted=True)``).
                    The C code stays single-threaded; threads only split the
                    tokens, and each draw depends on (seed, t, i) and the
                    snapshot alone.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lda_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_lda_oracle.so")
_lib = None

STAT_NAMES = ("flagged", "skip3", "sest_violations", "skip_not_k1", "fallback", "skip_after_s", "nnz_scanned")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc: -O2, IEEE fp64, no FMA contraction."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC", "-shared",
                        "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P, I64, I32, U64, U32, D = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                    ctypes.c_uint32, ctypes.c_double)
        lib.ora_philox4x32_10.argtypes = [P, P, P]
        lib.ora_uniform.argtypes = [U64, U32, U64]
        lib.ora_uniform.restype = D
        lib.ora_init_topic.argtypes = [U64, U64, I32]
        lib.ora_init_topic.restype = I32
        lib.ora_init.argtypes = [I64, I32, U64, P]
        lib.ora_build_counts.argtypes = [I64, P, P, P, I32, I32, I32, P, P, P, P, P, P]
        lib.ora_iterate.argtypes = [ctypes.c_int, ctypes.c_int, I64, P, P, I32, I32, I32, D, D, U64, U32, P, I64, P,
                                    P, P, P, P]
        lib.ora_llpt.argtypes = [ctypes.c_int, I64, P, P, P, I32, I32, I32, D, D]
        lib.ora_llpt.restype = D
        lib.ora_draw_given_u.argtypes = [ctypes.c_int, I64, P, P, P, I32, I32, I32, D, D, I64, D, P, P]
        lib.ora_draw_given_u.restype = I32
        lib.ora_what_row.argtypes = [I64, P, P, P, I32, I32, I32, D, I32, P]
        lib.ora_snapshot_new.argtypes = [I64, P, P, P, I32, I32, I32, D, D, ctypes.c_int, I64, P,
                                         ctypes.POINTER(P)]
        lib.ora_snapshot_draw.argtypes = [P, ctypes.c_int, ctypes.c_int, U64, U32, I64, I64, P, P, P, P, P]
        lib.ora_snapshot_llpt.argtypes = [P, I64, I64, ctypes.POINTER(D), ctypes.POINTER(D)]
        lib.ora_snapshot_free.argtypes = [P]
        lib.ora_snapshot_free.restype = None
        lib.ora_init_range.argtypes = [I64, I64, I32, U64, P]
        lib.ora_init_range.restype = None
        lib.ora_word_stats.argtypes = [I64, P, P, P, I32, I32, I32, D, D, P, P, P, P, P, P]
        lib.ora_word_top4.argtypes = [I64, P, P, P, I32, I32, I32, D, D, P, P]
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def philox(ctr, key) -> np.ndarray:
    """Philox4x32-10 of one 128-bit counter (4 x uint32) under a 64-bit key (2 x uint32)."""
    lib = _load()
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    lib.ora_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def uniform(seed: int, t: int, i: int) -> float:
    return float(_load().ora_uniform(seed, t, i))


def _ranges(n: int, parts: int):
    parts = max(1, min(parts, n))
    cuts = [n * q // parts for q in range(parts + 1)]
    return [(cuts[q], cuts[q + 1] - cuts[q]) for q in range(parts) if cuts[q + 1] > cuts[q]]


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def init_topics(n: int, K: int, seed: int, threads: int = 1) -> np.ndarray:
    """Initial topic of every token; ``threads`` host threads split the range."""
    z = np.empty(n, dtype=np.int32)
    lib = _load()
    if threads <= 1 or n < 1 << 20:
        lib.ora_init(n, K, seed, _p(z))
        return z
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda r: lib.ora_init_range(r[0], r[1], K, seed, ctypes.c_void_p(z.ctypes.data + 4 * r[0])),
                    _ranges(n, 4 * threads)))
    return z


def build_counts(word, doc, z, M: int, V: int, K: int) -> dict:
    lib = _load()
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    n = word.shape[0]
    out = dict(len=np.empty(M, np.int64), doff=np.empty(M + 1, np.int64), dtop=np.empty(max(n, 1), np.int32),
               dcnt=np.empty(max(n, 1), np.int32), W=np.empty((V, K), np.int32), T=np.empty(K, np.int64))
    rc = lib.ora_build_counts(n, _p(word), _p(doc), _p(z), M, V, K, _p(out["len"]), _p(out["doff"]),
                              _p(out["dtop"]), _p(out["dcnt"]), _p(out["W"]), _p(out["T"]))
    if rc:
        raise ValueError("ora_build_counts failed (%d)" % rc)
    nnz = int(out["doff"][M])
    out["dtop"] = out["dtop"][:nnz].copy()
    out["dcnt"] = out["dcnt"][:nnz].copy()
    return out


def _mode(mode: str, branches: int) -> int:
    if mode not in ("sparse", "dense") or branches not in (2, 3):
        raise ValueError("mode must be 'sparse' or 'dense', branches 2 or 3")
    return (1 if mode == "dense" else 0) | (2 if branches == 2 else 0)


def iterate(word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float, seed: int, t: int,
            mode: str = "sparse", g: int = 2, idx=None, want_Z: bool = False, branches: int = 3,
            restricted: bool = False):
    """One synchronous iteration from the snapshot built from ``z``.

    Returns ``(z_new, flags, stats[, Z])``; with ``idx`` only those tokens are
    drawn and the outputs are aligned with ``idx``.  flags bit0 = draw within
    1e-9*Z of a CDF edge, bit1 = step-3 skip test fired.  ``restricted`` (with
    ``idx``) builds only the W and D rows those tokens read: one pass over the
    corpus instead of every row and every word's top topics.
    """
    if restricted:
        if idx is None:
            raise ValueError("restricted needs idx")
        with Snapshot(word, doc, z, M=M, V=V, K=K, alpha=alpha, beta=beta, idx=idx,
                      with_words=(mode == "sparse")) as s:
            return s.draw(seed, t, idx=idx, mode=mode, g=g, want_Z=want_Z, branches=branches)
    lib = _load()
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    n = word.shape[0]
    if idx is not None:
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        m = idx.shape[0]
    else:
        m = n
    z_out = np.empty(m, np.int32)
    flags = np.empty(m, np.uint8)
    Z = np.empty(m, np.float64) if want_Z else None
    stats = np.zeros(8, np.int64)
    rc = lib.ora_iterate(_mode(mode, branches), g, n, _p(word), _p(doc), M, V, K, alpha, beta, seed, t, _p(z),
                         m if idx is not None else 0, _p(idx), _p(z_out), _p(flags), _p(Z), _p(stats))
    if rc:
        raise ValueError("ora_iterate failed (%d)" % rc)
    st = {name: int(stats[j]) for j, name in enumerate(STAT_NAMES)}
    if want_Z:
        return z_out, flags, st, Z
    return z_out, flags, st


def llpt(word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float, mode: str = "sparse") -> float:
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    return float(_load().ora_llpt(0 if mode == "sparse" else 1, word.shape[0], _p(word), _p(doc), _p(z), M, V, K,
                                  alpha, beta))


def word_stats(word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float) -> dict:
    lib = _load()
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    out = dict(K1=np.empty(V, np.int32), K2=np.empty(V, np.int32), a1=np.empty(V), a2=np.empty(V), a3=np.empty(V),
               Qp=np.empty(V))
    rc = lib.ora_word_stats(word.shape[0], _p(word), _p(doc), _p(z), M, V, K, alpha, beta, _p(out["K1"]),
                            _p(out["K2"]), _p(out["a1"]), _p(out["a2"]), _p(out["a3"]), _p(out["Qp"]))
    if rc:
        raise ValueError("ora_word_stats failed (%d)" % rc)
    out["K3"] = np.empty(V, np.int32)
    out["a4"] = np.empty(V)
    rc = lib.ora_word_top4(word.shape[0], _p(word), _p(doc), _p(z), M, V, K, alpha, beta, _p(out["K3"]),
                           _p(out["a4"]))
    if rc:
        raise ValueError("ora_word_top4 failed (%d)" % rc)
    return out


def run(word, doc, *, M: int, V: int, K: int, alpha: float, beta: float, seed: int, iters: int, t0: int = 0,
        z0=None, mode: str = "sparse"):
    """Initial topics (or ``z0``), then ``iters`` synchronous iterations.  Returns the list of z after each."""
    z = init_topics(len(word), K, seed) if z0 is None else _i32(z0)
    traj = [z]
    for t in range(t0, t0 + iters):
        z, _, _ = iterate(word, doc, z, M=M, V=V, K=K, alpha=alpha, beta=beta, seed=seed, t=t, mode=mode)
        traj.append(z)
    return traj


def draw_given_u(word, doc, z, i: int, u: float, *, M: int, V: int, K: int, alpha: float, beta: float,
                 mode: str = "sparse", branches: int = 3):
    """Draw token ``i`` of the snapshot built from ``z`` with the uniform ``u``.  Returns (topic, Z, flag)."""
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    Z = ctypes.c_double(0.0)
    f = ctypes.c_uint8(0)
    k = _load().ora_draw_given_u(_mode(mode, branches), word.shape[0], _p(word), _p(doc), _p(z), M, V, K,
                                 alpha, beta, i, u, ctypes.byref(Z), ctypes.byref(f))
    if k < 0:
        raise ValueError("ora_draw_given_u: bad argument")
    return int(k), float(Z.value), int(f.value)


def what_row(word, doc, z, v: int, *, M: int, V: int, K: int, beta: float) -> np.ndarray:
    """W^[v][k] = (W[v][k]+beta) / (T[k]+V*beta) for every topic k (Eq. 2)."""
    word, doc, z = _i32(word), _i32(doc), _i32(z)
    out = np.empty(K)
    if _load().ora_what_row(word.shape[0], _p(word), _p(doc), _p(z), M, V, K, beta, v, _p(out)):
        raise ValueError("ora_what_row failed")
    return out


class Snapshot:
    """Counts built once from ``z`` (all rows, or with ``idx`` only the rows of
    those tokens' words and documents), drawn from by several calls."""

    def __init__(self, word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float, idx=None,
                 with_words: bool = True):
        self._lib = _load()
        self.word, self.doc = _i32(word), _i32(doc)  # borrowed by the C snapshot: kept alive here
        self.n = int(self.word.shape[0])
        z = _i32(z)
        self._idx = None if idx is None else np.ascontiguousarray(idx, dtype=np.int64)
        self._h = ctypes.c_void_p()
        rc = self._lib.ora_snapshot_new(self.n, _p(self.word), _p(self.doc), _p(z), M, V, K, alpha, beta,
                                        1 if with_words else 0, 0 if self._idx is None else self._idx.shape[0],
                                        _p(self._idx), ctypes.byref(self._h))
        if rc:
            raise ValueError("ora_snapshot_new failed (%d)" % rc)

    def close(self):
        if self._h.value:
            self._lib.ora_snapshot_free(self._h)
            self._h = ctypes.c_void_p()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _draw_into(self, seed, t, first, cnt, idx_ptr, mode, g, branches, z_out, flags, Z, st, off):
        rc = self._lib.ora_snapshot_draw(self._h, _mode(mode, branches), g, seed, t, first, cnt, idx_ptr,
                                         ctypes.c_void_p(z_out.ctypes.data + 4 * off),
                                         ctypes.c_void_p(flags.ctypes.data + off),
                                         None if Z is None else ctypes.c_void_p(Z.ctypes.data + 8 * off), _p(st))
        if rc:
            raise ValueError("ora_snapshot_draw failed (%d)" % rc)

    def draw(self, seed: int, t: int, *, idx=None, mode: str = "sparse", g: int = 2, want_Z: bool = False,
             branches: int = 3, threads: int = 1):
        """Draw the tokens ``idx`` (default: every token), as ``iterate`` returns them."""
        if idx is not None:
            idx = np.ascontiguousarray(idx, dtype=np.int64)
        m = self.n if idx is None else int(idx.shape[0])
        z_out = np.empty(m, np.int32)
        flags = np.empty(m, np.uint8)
        Z = np.empty(m, np.float64) if want_Z else None
        parts = _ranges(m, 8 * threads) if m else []
        stats = np.zeros((max(len(parts), 1), 8), np.int64)

        def run(q):
            off, cnt = parts[q]
            if idx is None:
                self._draw_into(seed, t, off, cnt, None, mode, g, branches, z_out, flags, Z, stats[q], off)
            else:
                self._draw_into(seed, t, 0, cnt, ctypes.c_void_p(idx.ctypes.data + 8 * off), mode, g, branches,
                                z_out, flags, Z, stats[q], off)

        if threads <= 1:
            for q in range(len(parts)):
                run(q)
        else:
            with ThreadPoolExecutor(threads) as ex:
                list(ex.map(run, range(len(parts))))
        tot = stats.sum(axis=0)
        st = {name: int(tot[j]) for j, name in enumerate(STAT_NAMES)}
        if want_Z:
            return z_out, flags, st, Z
        return z_out, flags, st

    def llpt(self, threads: int = 1) -> float:
        """LLPT (sparse form) of the snapshot; partial compensated sums per token range, added in range order."""
        parts = _ranges(self.n, 8 * threads)
        out = [None] * len(parts)

        def run(q):
            s, c = ctypes.c_double(), ctypes.c_double()
            if self._lib.ora_snapshot_llpt(self._h, parts[q][0], parts[q][1], ctypes.byref(s), ctypes.byref(c)):
                raise ValueError("ora_snapshot_llpt failed")
            out[q] = (s.value, c.value)

        if threads <= 1:
            for q in range(len(parts)):
                run(q)
        else:
            with ThreadPoolExecutor(threads) as ex:
                list(ex.map(run, range(len(parts))))
        total, comp = 0.0, 0.0
        for s, c in out:
            comp += c
            t = total + s
            comp += ((total - t) + s) if abs(total) >= abs(s) else ((s - t) + total)
            total = t
        return (total + comp) / self.n


def iterate_threaded(word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float, seed: int, t: int,
                     threads: int | None = None, mode: str = "sparse", g: int = 2):
    """``iterate`` over every token, the tokens split over host threads (same result)."""
    threads = threads or default_threads()
    with Snapshot(word, doc, z, M=M, V=V, K=K, alpha=alpha, beta=beta, with_words=(mode == "sparse")) as s:
        return s.draw(seed, t, mode=mode, g=g, threads=threads)


def llpt_threaded(word, doc, z, *, M: int, V: int, K: int, alpha: float, beta: float,
                  threads: int | None = None) -> float:
    """``llpt`` (sparse form) with the tokens split over host threads (equal up to summation rounding)."""
    threads = threads or default_threads()
    with Snapshot(word, doc, z, M=M, V=V, K=K, alpha=alpha, beta=beta) as s:
        return s.llpt(threads=threads)
