#!/usr/bin/env python3
"""Writes tests/golden/llpt50_<case>.json: the oracle's LLPT (Sec. 2.2,
evaluation metric; log2 per token) after 50 synchronous iterations from the
Philox initial topics, for the parity test that compares the GPU's LLPT after
its own 50 iterations within 1e-3 relative.

Calls only ``oracle`` (the draws, split over host threads by token range; the
result does not depend on the split) and ``lda_synth`` (the seeded inputs).
Each file also records a fingerprint of the corpus, so that a test can tell a
changed generator from a changed sampler, and the host, thread count and wall
time of the run.

    python tests/golden/make_llpt_goldens.py [case ...] [--threads N]
"""
import argparse
import json
import os
import platform
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import lda_synth  # noqa: E402
import oracle  # noqa: E402

SEED = 42
ITERS = 50

# case name -> (workload, reduced-size overrides); the reduced shapes are the
# ones the GPU parity tests use for the five workloads
CASES = {
    "c2_reduced": ("c2", dict(n_docs=2500)),
    "c3_reduced": ("c3", dict(n_docs=12000)),
    "c4_reduced": ("c4", dict(n_docs=1200, V=20000)),
    "c5_reduced": ("c5", dict(n_docs=3000, V=100000)),
    "c2": ("c2", {}),
    "c3": ("c3", {}),
    "c4": ("c4", {}),
}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def run_case(name, threads):
    workload, over = CASES[name]
    c = lda_synth.make_corpus(workload, **over)
    kw = dict(M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta)
    t0 = time.time()
    z = oracle.init_topics(c.N, c.K, SEED, threads=threads)
    ll0 = oracle.llpt_threaded(c.word, c.doc, z, threads=threads, **kw)
    traj = {0: ll0}
    for t in range(ITERS):
        z, _, st = oracle.iterate_threaded(c.word, c.doc, z, seed=SEED, t=t, threads=threads, **kw)
        assert st["sest_violations"] == 0 and st["skip_not_k1"] == 0
        print("%s t=%d skip3 %.4f  %.0f s" % (name, t, st["skip3"] / c.N, time.time() - t0), flush=True)
        if (t + 1) % 10 == 0:
            traj[t + 1] = oracle.llpt_threaded(c.word, c.doc, z, threads=threads, **kw)
            print("%s LLPT after %d iterations %.9f" % (name, t + 1, traj[t + 1]), flush=True)
    wall = time.time() - t0
    out = dict(case=name, workload=workload, overrides=over, N=c.N, V=c.V, K=c.K, M=c.n_docs, alpha=c.alpha,
               beta=c.beta, seed=SEED, iterations=ITERS, llpt=traj[ITERS],
               llpt_trajectory={str(k): v for k, v in sorted(traj.items())},
               corpus_fingerprint=lda_synth.fingerprint(c), threads=threads, cpu_model=cpu_model(),
               wall_s=round(wall, 1),
               source="oracle/lda_oracle.c sparse form, tokens split over host threads by range")
    path = os.path.join(HERE, "llpt50_%s.json" % name)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print("wrote %s (%.0f s)" % (path, wall), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("cases", nargs="*", default=list(CASES))
    ap.add_argument("--threads", type=int, default=oracle.default_threads())
    args = ap.parse_args()
    for name in args.cases:
        run_case(name, args.threads)


if __name__ == "__main__":
    main()
