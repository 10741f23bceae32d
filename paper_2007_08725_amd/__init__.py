"""MI355X-native synchronous LDA sampler (ezLDA, arXiv 2007.08725).

Thin ctypes binding over ``liblda.so`` (declared in ``include/lda.h``): it
marshals arguments and nothing else.  Every step of an iteration runs in the
library's HIP kernels.  PyTorch supplies only the stream and, optionally, the
caching device allocator.  If the library is not built, constructing an
:class:`LDA` raises :class:`ImportError`; there is no CPU fallback.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblda.so")
_lib = None

LDA_OK, LDA_E_ARG, LDA_E_RANGE, LDA_E_NOMEM, LDA_E_DEVICE, LDA_E_STATE = range(6)
STATUS_NAMES = {0: "LDA_OK", 1: "LDA_E_ARG", 2: "LDA_E_RANGE", 3: "LDA_E_NOMEM", 4: "LDA_E_DEVICE",
                5: "LDA_E_STATE"}
MAX_TOPICS = 32768
MAX_DOC_LEN = 65535
MAX_CHUNKS = 256

ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class Options(ctypes.Structure):
    _fields_ = [("stream", ctypes.c_void_p), ("dev_alloc", ALLOC_FN), ("dev_free", FREE_FN),
                ("alloc_ctx", ctypes.c_void_p), ("g", ctypes.c_int32), ("region_tokens", ctypes.c_int32),
                ("no_skip", ctypes.c_int32), ("dense_cutoff", ctypes.c_int32), ("two_branch", ctypes.c_int32),
                ("sampler_block", ctypes.c_int32), ("skip_marks", ctypes.c_int32),
                ("always_skip_test", ctypes.c_int32), ("chunks", ctypes.c_int32)]


class IterStats(ctypes.Structure):
    _fields_ = [("iteration", ctypes.c_int64), ("ms_iter", ctypes.c_double), ("ms_sampler", ctypes.c_double),
                ("ms_docpass", ctypes.c_double), ("ms_rebuild", ctypes.c_double), ("ms_precompute", ctypes.c_double),
                ("skip_step3", ctypes.c_int64), ("skip_after_s", ctypes.c_int64), ("sampled", ctypes.c_int64),
                ("nnz_scanned", ctypes.c_int64), ("regions", ctypes.c_int64), ("dense_regions", ctypes.c_int64),
                ("row_bytes", ctypes.c_int64), ("sampler_block", ctypes.c_int64), ("skip_marks", ctypes.c_int64),
                ("skip_test_ran", ctypes.c_int64)]


class Counts(ctypes.Structure):
    _fields_ = [("iteration", ctypes.c_int64), ("M", ctypes.c_int32), ("V", ctypes.c_int32), ("K", ctypes.c_int32),
                ("n_tokens", ctypes.c_int64), ("nnz_D", ctypes.c_int64), ("nnz_W", ctypes.c_int64),
                ("z", ctypes.c_void_p), ("T", ctypes.c_void_p), ("D_off", ctypes.c_void_p),
                ("D_topic", ctypes.c_void_p), ("D_count", ctypes.c_void_p), ("W_off", ctypes.c_void_p),
                ("W_topic", ctypes.c_void_p), ("W_count", ctypes.c_void_p)]


# Every symbol include/lda.h declares.
EXPORTS = ("lda_create", "lda_iterate", "lda_get_counts", "lda_loglik", "lda_set_assignments", "lda_destroy",
           "lda_last_error", "lda_describe_layout", "lda_loglik_noalloc")
NOALLOC_MAX_REGIONS = 1 << 21


class LDAError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, str(status)), msg))
        self.status = status


def load_library():
    """Load liblda.so; raises ImportError when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("liblda.so is not built (%s): run __graft_entry__.build() to compile the HIP library"
                          % LIB_PATH)
    # torch ships its own HIP runtime with the same soname; loading it first
    # makes liblda bind to that one runtime instead of a second copy
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
    lib.lda_create.argtypes = [P, P, I64, I32, I32, D, D, U64, P, ctypes.POINTER(P)]
    lib.lda_create.restype = ctypes.c_int
    lib.lda_iterate.argtypes = [P, I32, P]
    lib.lda_iterate.restype = ctypes.c_int
    lib.lda_get_counts.argtypes = [P, ctypes.POINTER(Counts)]
    lib.lda_get_counts.restype = ctypes.c_int
    lib.lda_loglik.argtypes = [P, ctypes.POINTER(D)]
    lib.lda_loglik.restype = ctypes.c_int
    lib.lda_loglik_noalloc.argtypes = [P, ctypes.POINTER(D)]
    lib.lda_loglik_noalloc.restype = ctypes.c_int
    lib.lda_set_assignments.argtypes = [P, P, I64]
    lib.lda_set_assignments.restype = ctypes.c_int
    lib.lda_destroy.argtypes = [P]
    lib.lda_destroy.restype = None
    lib.lda_last_error.argtypes = [P]
    lib.lda_last_error.restype = ctypes.c_char_p
    lib.lda_describe_layout.argtypes = [P, P, I64, I32, I32, I32, I32, P, P, P, P, P, P, P, P]
    lib.lda_describe_layout.restype = ctypes.c_int
    _lib = lib
    return lib


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _check(lib, handle, status):
    if status != LDA_OK:
        raise LDAError(status, lib.lda_last_error(handle).decode())


def describe_layout(word, doc, V: int, K: int, region_tokens: int = 0, dense_cutoff: int = 0) -> dict:
    """Host-only layout of a token list: relabel, dense prefix, word order and regions (no device)."""
    lib = load_library()
    word = np.ascontiguousarray(word, np.int32)
    doc = np.ascontiguousarray(doc, np.int32)
    n = word.shape[0]
    npres, nd, ndocs = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    nreg = ctypes.c_int64()
    st = lib.lda_describe_layout(_p(word), _p(doc), n, V, K, region_tokens, dense_cutoff, None, ctypes.byref(npres),
                                 ctypes.byref(nd), ctypes.byref(nreg), ctypes.byref(ndocs), None, None, None)
    _check(lib, None, st)
    relabel = np.empty(V, np.int32)
    word_off = np.empty(npres.value + 1, np.uint32)
    wt_key = np.empty(n, np.uint32)
    region = np.empty(3 * nreg.value, np.uint32)
    st = lib.lda_describe_layout(_p(word), _p(doc), n, V, K, region_tokens, dense_cutoff, _p(relabel), None, None,
                                 None, None, _p(word_off), _p(wt_key), _p(region))
    _check(lib, None, st)
    return dict(relabel=relabel, n_present=npres.value, n_dense=nd.value, n_docs=ndocs.value, word_off=word_off,
                wt_key=wt_key, region=region.reshape(-1, 3))


_LIVE = weakref.WeakSet()


@atexit.register
def _close_all():
    """Destroy the handles still open at exit, while torch's allocator can take their memory back."""
    for m in list(_LIVE):
        m.close()


class LDA:
    """One sampler on the current HIP device.

    ``word``/``doc``: int32 token list (any order); ``V`` vocabulary size, ``K``
    topics, ``alpha``/``beta`` priors of Eq. 1, ``seed`` the Philox key.
    ``g`` (1, 2 or 3), ``region_tokens``, ``no_skip`` and ``dense_cutoff`` are
    the options of ``lda_options``; none of them changes the draws.
    ``two_branch`` samples over [S | Q] (Sec. 2.2): same distribution, other
    canonical order.  ``sampler_block`` (256, 512, 1024; 0 = by occupancy)
    sets the sampler's workgroup size; ``skip_marks`` (0 auto, 1 word order,
    2 document order) how skip decisions reach the sampler; ``always_skip_test``
    runs steps 2-3 in every iteration instead of when they pay; ``chunks`` > 1
    keeps the per-token arrays in pinned host memory and streams them through
    the device in that many chunks of documents (input sorted by document).
    """

    def __init__(self, word, doc, V: int, K: int, alpha: float, beta: float = 0.01, seed: int = 42, *, g: int = 2,
                 region_tokens: int = 0, no_skip: bool = False, dense_cutoff: int = 0, two_branch: bool = False,
                 sampler_block: int = 0, skip_marks: int = 0, always_skip_test: bool = False, chunks: int = 0,
                 torch_stream: bool = True, torch_allocator: bool = True):
        self._lib = load_library()
        self._h = ctypes.c_void_p()
        word = np.ascontiguousarray(word, np.int32)
        doc = np.ascontiguousarray(doc, np.int32)
        self.N = int(word.shape[0])
        self.V, self.K, self.alpha, self.beta, self.seed = int(V), int(K), float(alpha), float(beta), int(seed)
        opts = Options()
        opts.g = g
        opts.region_tokens = region_tokens
        opts.no_skip = 1 if no_skip else 0
        opts.dense_cutoff = dense_cutoff
        opts.two_branch = 1 if two_branch else 0
        opts.sampler_block = sampler_block
        opts.skip_marks = skip_marks
        opts.always_skip_test = 1 if always_skip_test else 0
        opts.chunks = chunks
        self._keep = []
        if torch_stream or torch_allocator:
            import torch
            if not torch.cuda.is_available():
                raise RuntimeError("no HIP device visible to torch")
            dev = torch.cuda.current_device()
            stream = torch.cuda.current_stream(dev)
            if torch_stream:
                opts.stream = ctypes.c_void_p(stream.cuda_stream)
            if torch_allocator:
                def _alloc(nbytes, ctx, _dev=dev, _stream=stream):
                    try:
                        return torch.cuda.caching_allocator_alloc(int(nbytes), _dev, _stream)
                    except Exception:
                        return None

                def _free(ptr, ctx):
                    cuda = getattr(torch, "cuda", None)  # None while the interpreter shuts down
                    if cuda is not None:
                        cuda.caching_allocator_delete(ptr)

                fa, ff = ALLOC_FN(_alloc), FREE_FN(_free)
                self._keep += [fa, ff]
                opts.dev_alloc, opts.dev_free = fa, ff
        st = self._lib.lda_create(_p(word), _p(doc), self.N, self.V, self.K, self.alpha, self.beta, self.seed,
                                  ctypes.byref(opts), ctypes.byref(self._h))
        _check(self._lib, None, st)
        _LIVE.add(self)

    # -- lifetime ---------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.lda_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- calls ------------------------------------------------------------
    def iterate(self, n: int = 1, stats: bool = False):
        """Run ``n`` synchronous iterations; with ``stats`` return one dict per iteration."""
        buf = (IterStats * max(n, 1))() if stats else None
        st = self._lib.lda_iterate(self._h, n, ctypes.cast(buf, ctypes.c_void_p) if stats else None)
        _check(self._lib, self._h, st)
        if not stats:
            return None
        return [{f: getattr(buf[i], f) for f, _ in IterStats._fields_} for i in range(n)]

    def loglik(self) -> float:
        out = ctypes.c_double()
        _check(self._lib, self._h, self._lib.lda_loglik(self._h, ctypes.byref(out)))
        return out.value

    def loglik_noalloc(self) -> float:
        """``loglik`` through the entry point that allocates nothing (fixed device scratch)."""
        out = ctypes.c_double()
        _check(self._lib, self._h, self._lib.lda_loglik_noalloc(self._h, ctypes.byref(out)))
        return out.value

    def set_assignments(self, z, iteration: int):
        z = np.ascontiguousarray(z, np.int32)
        if z.shape[0] != self.N:
            raise ValueError("z must have one topic per token")
        _check(self._lib, self._h, self._lib.lda_set_assignments(self._h, _p(z), int(iteration)))

    def sizes(self) -> dict:
        c = Counts()
        _check(self._lib, self._h, self._lib.lda_get_counts(self._h, ctypes.byref(c)))
        return dict(iteration=c.iteration, M=c.M, V=c.V, K=c.K, n_tokens=c.n_tokens, nnz_D=c.nnz_D, nnz_W=c.nnz_W)

    def counts(self, z: bool = True, D: bool = True, W: bool = True) -> dict:
        """Assignment (input order) and count tables in the caller's ids (CSR, topics ascending)."""
        sz = self.sizes()
        c = Counts()
        out = dict(iteration=sz["iteration"], M=sz["M"])
        arrays = {}
        if z:
            arrays["z"] = np.empty(self.N, np.int32)
        arrays["T"] = np.empty(self.K, np.int64)
        if D:
            arrays["D_off"] = np.empty(sz["M"] + 1, np.int64)
            arrays["D_topic"] = np.empty(max(sz["nnz_D"], 1), np.int32)
            arrays["D_count"] = np.empty(max(sz["nnz_D"], 1), np.int32)
        if W:
            arrays["W_off"] = np.empty(self.V + 1, np.int64)
            arrays["W_topic"] = np.empty(max(sz["nnz_W"], 1), np.int32)
            arrays["W_count"] = np.empty(max(sz["nnz_W"], 1), np.int32)
        for name, arr in arrays.items():
            setattr(c, name, arr.ctypes.data)
        _check(self._lib, self._h, self._lib.lda_get_counts(self._h, ctypes.byref(c)))
        if D:
            arrays["D_topic"] = arrays["D_topic"][:sz["nnz_D"]]
            arrays["D_count"] = arrays["D_count"][:sz["nnz_D"]]
        if W:
            arrays["W_topic"] = arrays["W_topic"][:sz["nnz_W"]]
            arrays["W_count"] = arrays["W_count"][:sz["nnz_W"]]
        out.update(arrays)
        return out
