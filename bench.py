#!/usr/bin/env python3
"""Benchmark of the synchronous LDA iteration on one MI355X.

Workload (default): the large planted corpus -- 8.2M documents with
lognormal lengths (mean 90, sigma 0.8), ~738M tokens, V = 141,000 with a
Zipf(1.1) vocabulary base, 500 planted topics -- fit with K = 1,000,
alpha = 0.05, beta = 0.01.  It stands in for PubMed (Sec. 6).  A step is one
full synchronous iteration: per-topic and per-word precompute, the
per-document C1/C2 + skip pass, the word-major sampler and the count rebuild.

Prints one JSON line: tokens/s over the timed steps, the sampler kernel's
algorithmic HBM bytes per launch divided by its HIP-event duration against the
8 TB/s peak (and against a plain device copy's measured rate), and the oracle
timed on two bounded samples of the same workload, one early and one from the
GPU's state after the timed iterations.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PCIE_PEAK_GBS = 64.0  # PCIe 5.0 x16, one direction
PMC_SUMMARY = os.path.join(ROOT, "profiles", "kernels_c3_counters.md")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2007_08725_amd", "csrc", "kernels.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def sampler_alg_bytes(st, N):
    """Bytes the sampler must move per launch: per token its skip bit (read)
    and its topic slot (written: the drawn topic, or K1 for a skipped token);
    per sampled token its key and D-row offset (8 B), row header (4 B) and
    the entries of its D row it reads (4 B each: the whole row, or one chunk
    for a later token of a long-row run of one word in one document); the W
    rows (4*K B per dense word, 4*nnz B per sparse word); the region and word
    records (12 + 48 B per region).  The skip bits are N/8 coalesced bytes in
    word order; with the document-ordered bitmap each token reads the 4-byte
    word that holds its bit at its document position instead."""
    skip = 4 * N if st.get("skip_marks") == 2 else N / 8
    return (skip + 2 * N + 12 * st["sampled"] + 4 * st["nnz_scanned"] + st["row_bytes"] + 60 * st["regions"])


def _profile_field(workload, first, last, field):
    """A per-launch k_sampler figure from the committed counter summary, if
    the summary covers this workload and the same iterations (first..last)
    and was taken on the current kernel source; else None."""
    if workload != "c3" or not os.path.exists(PMC_SUMMARY):
        return None
    txt = open(PMC_SUMMARY).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", txt)
    w = re.search(r"counter_window_iterations:\s*(\d+)-(\d+)", txt)
    b = re.search(field + r":\s*([0-9.eE+]+)", txt)
    if not m or not w or not b or (int(w.group(1)), int(w.group(2))) != (first, last):
        return None
    if hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest() != m.group(1):
        return None
    return float(b.group(1))


def traffic_from_profile(workload, first, last):
    """Bytes per sampler launch that the L2 requested from the memory fabric
    (reads by request size plus writes), from the committed counter summary
    (conditions of _profile_field); else None."""
    return _profile_field(workload, first, last, "k_sampler_fabric_bytes_per_launch")


def valu_from_profile(workload, first, last):
    """k_sampler's VALU wave instructions per launch from the committed
    counter summary (conditions of _profile_field); else None."""
    return _profile_field(workload, first, last, "k_sampler_valu_per_launch")


VALU_ISSUE_PER_S = 1024 * 2.4e9 / 4  # wave instructions per second: 1,024 SIMDs, 4 cycles each at 2.4 GHz


def copy_ceiling_gbs(torch, reps=10):
    """Bytes moved per second (read + write) by a plain 1 GiB device-to-device
    copy, timed with HIP events on torch's stream: the streaming rate this
    GPU sustains, stated beside the 8 TB/s peak."""
    a = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(2):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    e1.synchronize()
    gbs = 2.0 * a.numel() * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    return gbs


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


class _OneCore:
    """Runs the enclosed code on one core of this process's set (the calling
    thread's affinity), restoring the previous set afterwards."""

    def __enter__(self):
        self.old = os.sched_getaffinity(0)
        self.core = min(self.old)
        os.sched_setaffinity(0, {self.core})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.old)


def cpu_baseline(c, n_docs, z_late, t_late, n_docs_late):
    """The oracle as it stands, single thread pinned to one core.  Early sample:
    one synchronous iteration on the first n_docs documents from the Philox
    initial topics (counts, per-word precompute and every draw timed).  Late
    sample: the draws of the first n_docs_late documents' tokens at iteration
    t_late from the GPU's own state after its timed iterations (counts and
    per-word precompute built beforehand, untimed)."""
    import numpy as np
    import oracle

    m = int(np.searchsorted(c.doc, n_docs))
    w, d = c.word[:m], c.doc[:m]
    z = oracle.init_topics(m, c.K, lda_seed())
    with _OneCore() as pin:
        t0 = time.perf_counter()
        oracle.iterate(w, d, z, M=n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta, seed=lda_seed(), t=0)
        dt = time.perf_counter() - t0
    out = {"value": m / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle", "cpu_model": cpu_model(),
           "pinned_core": pin.core,
           "sample": "one synchronous iteration (counts rebuilt from the Philox initial topics, per-word "
                     "precompute over all %d words, every token drawn) on the first %d documents = %d tokens "
                     "of the same corpus, one thread pinned to one core, %.1f s" % (c.V, n_docs, m, dt)}
    if z_late is not None:
        ml = int(np.searchsorted(c.doc, n_docs_late))
        idx = np.arange(ml, dtype=np.int64)
        with oracle.Snapshot(c.word, c.doc, z_late, M=c.n_docs, V=c.V, K=c.K, alpha=c.alpha, beta=c.beta,
                             idx=idx) as s:
            with _OneCore():
                t0 = time.perf_counter()
                _, _, st = s.draw(lda_seed(), t_late, idx=idx)
                dl = time.perf_counter() - t0
        out["late"] = {"value": ml / dl, "unit": "tokens/s", "cores": 1,
                       "sample": "the draws of iteration %d for the first %d documents = %d tokens, from the GPU's "
                                 "assignments after its timed iterations (counts and per-word precompute over the "
                                 "whole corpus built untimed), one thread pinned to one core, %.1f s; %d of them "
                                 "skipped at step 3" % (t_late, n_docs_late, ml, dl, st.get("skip3", 0))}
    return out


def lda_seed():
    import lda_synth
    return lda_synth.SAMPLER_SEED


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c3", choices=["c1", "c2", "c3", "c4", "c5", "c6"])
    ap.add_argument("--cpu-docs", type=int, default=200000, help="documents in the oracle's timed sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dump-stats", default=None, help="write the per-iteration statistics (JSON lines) here")
    ap.add_argument("--always-skip-test", action="store_true", help="run steps 2-3 in every iteration")
    ap.add_argument("--chunks", type=int, default=0,
                    help="out-of-core mode: per-token arrays in pinned host memory, streamed in this many chunks")
    ap.add_argument("--cpu-docs-late", type=int, default=100000,
                    help="documents in the oracle's late-state sample")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the library runs on exactly one GPU; --gpus %d is not supported "
              "(sharding across GPUs is designed, not implemented)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import lda_synth
    import paper_2007_08725_amd as lda

    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    c = lda_synth.make_corpus(args.workload)
    log("generated %s: N=%d docs=%d V=%d K=%d in %.1f s" % (args.workload, c.N, c.n_docs, c.V, c.K,
                                                            time.perf_counter() - t0))
    t0 = time.perf_counter()
    m = lda.LDA(c.word, c.doc, c.V, c.K, c.alpha, c.beta, lda_synth.SAMPLER_SEED, chunks=args.chunks,
                always_skip_test=args.always_skip_test)
    torch.cuda.synchronize()
    t_create = time.perf_counter() - t0
    log("lda_create %.1f s" % t_create)

    copy_gbs = copy_ceiling_gbs(torch)
    log("plain 1 GiB device copy: %.0f GB/s (read + write)" % copy_gbs)

    if args.warmup:
        m.iterate(args.warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    st = m.iterate(args.steps, stats=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log("timed %d steps in %.3f s" % (args.steps, elapsed))
    if args.dump_stats:
        with open(args.dump_stats, "w") as f:
            for s in st:
                f.write(json.dumps(s) + "\n")
    llpt = m.loglik()
    z_late = None if args.no_cpu_baseline else m.counts(z=True, D=False, W=False)["z"]

    N = c.N
    value = N * args.steps / elapsed
    ms_sampler = np.array([s["ms_sampler"] for s in st])
    alg = np.array([sampler_alg_bytes(s, N) for s in st], dtype=np.float64)
    alg_per_launch = float(alg.mean())
    if args.chunks > 1:
        # out of core: the stream of per-token arrays over PCIe bounds the
        # iteration (6 B a token up: word-order slot and topic; 2 B down)
        h2d = 6.0 * N
        achieved = h2d * args.steps / elapsed / 1e9
        roofline = {"bound": "pcie", "achieved": achieved, "peak": PCIE_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / PCIE_PEAK_GBS, "traffic": None, "kernel": "host-to-device copies",
                    "h2d_bytes_per_iteration": h2d, "d2h_bytes_per_iteration": 2.0 * N, "chunks": args.chunks,
                    "hbm_copy_ceiling_gbs": copy_gbs}
    else:
        achieved = alg.sum() / (ms_sampler.sum() * 1e-3) / 1e9
        traffic = traffic_from_profile(args.workload, args.warmup, args.warmup + args.steps - 1)
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                    "traffic_kind": "fabric: bytes the L2 requested from memory per launch (reads by request "
                                    "size + writes, rocprofv3 TCC_EA0 counters over the same iterations); "
                                    "last-level-cache hits are inside it, so it bounds DRAM bytes from above",
                    "kernel": "k_sampler", "alg_bytes_per_launch": alg_per_launch,
                    "avg_launch_ms": float(ms_sampler.mean()),
                    "copy_ceiling_gbs": copy_gbs, "frac_of_copy": achieved / copy_gbs}
        if traffic is not None:
            roofline["traffic_gbs"] = traffic / (ms_sampler.mean() * 1e-3) / 1e9
        valu = valu_from_profile(args.workload, args.warmup, args.warmup + args.steps - 1)
        if valu is not None:
            # the limit the kernel actually meets: VALU instruction issue
            roofline["valu_issue_frac"] = valu / VALU_ISSUE_PER_S / (ms_sampler.mean() * 1e-3)
    stage_ms = {k: float(np.mean([s[k] for s in st])) for k in
                ("ms_precompute", "ms_docpass", "ms_sampler", "ms_rebuild", "ms_iter")}
    line = {
        "metric": "sampled tokens/sec per iteration + sampler HBM GB/s vs peak, K=1000",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic planted-LDA corpus (seeded), random initial topics",
        "config": {"workload": "%s: %d docs, %d tokens, V=%d, K=%d, alpha=%g, beta=%g, iterations %d-%d" % (
            args.workload, c.n_docs, N, c.V, c.K, c.alpha, c.beta, args.warmup, args.warmup + args.steps - 1),
            "parallelism": "single GPU" + (", out of core in %d chunks" % args.chunks if args.chunks > 1 else "")},
        "roofline": roofline,
        "breakdown_ms": stage_ms,
        "skip_step3_frac": float(np.mean([s["skip_step3"] for s in st]) / N),
        "llpt_after": llpt,
        "create_s": t_create,
    }
    m.close()
    if not args.no_cpu_baseline:
        log("timing the oracle on a sample ...")
        line["cpu_baseline"] = cpu_baseline(c, args.cpu_docs, z_late, args.warmup + args.steps,
                                            args.cpu_docs_late)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
