"""Ablation runs of the synchronous iteration on one corpus (the trends of Sec. 6.2).

Each configuration switches one design choice off or changes one parameter,
with everything else at its default:

  default        three-branch sampling (Eq. 5), S_est depth g = 2, hybrid W
                 (dense iff count > K), large words split into regions of
                 10,000 tokens
  g1, g3         S_est depth 1 or 3 (Eq. 9): which tokens skip the S' scan
  no_skip        no step-3 test: every token scans its D row
  two_branch     sampling over [S | Q] (Sec. 2.2): no max-topic branch
  all_dense      every W row dense
  all_sparse     every W row sparse (except words above 65,535 tokens)
  no_split       large words are not split: one region per word (Sec. 5.1)
  word_marks     skip decisions always in the word-ordered bitmap
  doc_marks      skip decisions always in the document-ordered bitmap
  always_test    steps 2-3 in every iteration (by default they run when the
                 previous iteration skipped at least an eighth of the tokens,
                 and in every eighth iteration)

Only two_branch changes the draws (another canonical order of the same
distribution); the rest draw exactly the same topics.

    python -m paper_2007_08725_amd.ablation --workload c3 --warmup 1 --steps 20 --out ablation.jsonl
"""
import argparse
import json
import os
import sys
import time

CONFIGS = {
    "default": {},
    "g1": dict(g=1),
    "g3": dict(g=3),
    "no_skip": dict(no_skip=True),
    "two_branch": dict(two_branch=True),
    "all_dense": dict(dense_cutoff=-1),
    "all_sparse": dict(dense_cutoff=(1 << 31) - 1),
    "no_split": dict(region_tokens=(1 << 31) - 1),
    "word_marks": dict(skip_marks=1),
    "doc_marks": dict(skip_marks=2),
    "always_test": dict(always_skip_test=True),
}


def run(corpus, name, opts, warmup, steps):
    import numpy as np
    import torch

    import lda_synth

    from . import LDA

    t0 = time.perf_counter()
    m = LDA(corpus.word, corpus.doc, corpus.V, corpus.K, corpus.alpha, corpus.beta, lda_synth.SAMPLER_SEED, **opts)
    torch.cuda.synchronize()
    t_create = time.perf_counter() - t0
    if warmup:
        m.iterate(warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st = m.iterate(steps, stats=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ll = m.loglik()
    m.close()
    N = corpus.N
    mean = lambda k: float(np.mean([s[k] for s in st]))
    return {
        "config": name, "options": {k: int(v) for k, v in opts.items()},
        "iterations": "%d-%d" % (warmup, warmup + steps - 1),
        "ms_per_iteration": elapsed * 1e3 / steps, "tokens_per_s": N * steps / elapsed,
        "ms_sampler": mean("ms_sampler"), "ms_docpass": mean("ms_docpass"), "ms_rebuild": mean("ms_rebuild"),
        "skip_step3_frac": mean("skip_step3") / N, "nnz_per_sampled_token": mean("nnz_scanned") / max(1.0, mean("sampled")),
        "regions": int(st[0]["regions"]), "llpt_after": ll, "create_s": t_create,
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="c3", choices=["c1", "c2", "c3", "c4", "c5"])
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--configs", default=",".join(CONFIGS), help="comma-separated subset of " + ",".join(CONFIGS))
    ap.add_argument("--out", default=None, help="also write the JSON lines here")
    args = ap.parse_args(argv)
    import torch

    import lda_synth

    torch.cuda.set_device(0)
    corpus = lda_synth.make_corpus(args.workload)
    print("corpus %s: N=%d docs=%d V=%d K=%d" % (args.workload, corpus.N, corpus.n_docs, corpus.V, corpus.K),
          file=sys.stderr, flush=True)
    out = open(args.out, "w") if args.out else None
    for name in args.configs.split(","):
        rec = run(corpus, name, CONFIGS[name], args.warmup, args.steps)
        rec["workload"] = args.workload
        line = json.dumps(rec)
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()
    if out:
        out.close()


if __name__ == "__main__":
    main()
