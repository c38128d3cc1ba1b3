#!/usr/bin/env python3
"""Throughput of the SPDP Gibbs sweep on one MI355X.

One step = one full sweep of the hot path (sampling kernel, count update,
repair, totals) over every token of a synthetic SPDP corpus resident in HBM.
Prints ONE JSON line: tokens resampled per second, the HBM roofline fraction
of the sampling kernel (algorithmic bytes per launch over its HIP-event
duration) and the fp64 oracle timed on the host cores over a bounded sample
of documents.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME|IDX]
                       [--assoc S [--assoc-eps E]] [--heldout S]

--assoc S runs the model with word associations instead (sparse
transformation matrices with S sources per word, from synth.associations)
and reports the same line for it.  --async runs the thesis's asynchronous
sweep (an ablation: live atomics, racy reads; --async-waves wavefronts, 0 for
the library's default) instead of the snapshot sweep.  --heldout S times the
held-out fold-in instead: the last 10 % of each group's documents are
held out, the rest trained for the warm-up sweeps, and the line reports test
tokens folded in per second of one fold-in sweep (with --assoc S, of the
model with word associations), taken as the difference
between an S-sweep and a 1-sweep held-out call (their uploads and host sums
cancel).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "tokens resampled/sec per Gibbs sweep (1 GPU) + % of HBM roofline"
HBM_PEAK_GBS = 8000.0  # MI355X datasheet HBM3E bandwidth
DEFAULT_WORKLOAD = "g20-d50000-k500"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def narrow_fraction(cp) -> float:
    """Share of tokens whose (group, word) pair occurs at most 255 times: the
    sampler reads those tokens' count rows as 16-bit cells (n | t << 8, half
    the bytes).  A pure function of the corpus."""
    import numpy as np

    q = np.repeat(cp.doc_group, np.diff(cp.doc_off)).astype(np.int64) * cp.vocab + cp.words
    c = np.bincount(q)
    return float(np.mean(c[q] <= 255)) if len(q) else 0.0


def sample_bytes_per_token(K: int, wide: bool, narrow: float = 0.0) -> float:
    """Bytes the sampling kernel must move per token in this library's layout:
    the K-cell count row of (group, word) (customers and tables packed in one
    int32 per cell, or in 16 bits for the share `narrow` of tokens whose pair
    occurs at most 255 times), the K-entry shadow-base row of the word (16-bit
    counts, or int32 once some count exceeds 65535), and the token stream
    (row index, state and narrow-row flag in, state out)."""
    return (4 - 2 * narrow) * K + (4 if wide else 2) * K + 13


def assoc_bytes_per_token(K: int, wide: bool, mean_sources: float, Sp: int,
                          narrow: float = 0.0) -> float:
    """Bytes the association sampler must move per token: the packed count
    row (16-bit cells for the share `narrow` of tokens, as in the plain
    sampler), one shadow-base row per source of the token's row (mean_sources
    on average), the token stream (row index, state and narrow-row flag in,
    state out) and the row's source record (Sp source words and Sp fp32 p)."""
    return (4 - 2 * narrow) * K + (4 if wide else 2) * K * mean_sources + 13 + 8 * Sp


def foldin_bytes_per_token(K: int) -> int:
    """Bytes one fold-in sweep must move per test token with P = I: the K-cell
    packed count row of (group, word), the word's K-entry int32 shadow-base
    row, and the token stream (row index and topic in, topic out)."""
    return 8 * K + 12


def async_bytes_per_token(K: int) -> int:
    """Bytes the asynchronous sweep's pass must move per token: the live
    packed count row, shadow-base row (int32) and document row of the token
    (the group's total rows stay in cache), the visiting order, row index,
    document and state of the token, and its state written back."""
    return 4 * K + 4 * K + 4 * K + 20


def dense_bytes_per_token(K: int) -> int:
    """The same for separate int32 rows n[g,w,:], t[g,w,:] and B[w,:]."""
    return 12 * K + 12


def shadow_base_wide(s) -> bool:
    """True when some shadow-base count exceeds 65535 (the samplers then read
    the 32-bit rows of B), from B copied on the device and reduced there."""
    import torch

    from paper_1510_06549_amd import spdp as sp

    B = torch.empty((s.V, s.K), dtype=torch.int32, device="cuda")
    sp.spdp_totals(s.h, None, None, B, None)
    return bool(B.max().item() > 0xFFFF)


def kernel_source_hash(kernel: str) -> str:
    """SHA-256 of what a sampling kernel is compiled from: its own file, the
    two headers that file includes, then the file's compiler flags."""
    import hashlib

    from paper_1510_06549_amd import build_lib

    csrc = os.path.join(ROOT, "paper_1510_06549_amd", "csrc")
    source = {"k_sample": "sample.hip", "k_sample_assoc": "sample_assoc.hip"}[kernel]
    h = hashlib.sha256()
    for name in (source, "sampler_common.hpp", "spdp_internal.hpp"):
        h.update(open(os.path.join(csrc, name), "rb").read())
    h.update(" ".join(build_lib.source_flags(source)).encode())
    return h.hexdigest()


def recorded_traffic(kernel: str, workload: str):
    """HBM bytes per launch of the sampling kernel measured with rocprofv3
    counters, if they were taken on the current source of that kernel
    (profiles/traffic_<kernel>_<workload>.txt holds the figure with
    kernel_source_hash() at the time), else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != kernel_source_hash(kernel) or "bytes_per_launch" not in kv:
        return None
    return float(kv["bytes_per_launch"])


def cpu_baseline(cp, wl, state, target_s: float, assoc=None, full_sweeps: int = 0,
                 seed: int = 0):
    """The oracle's whole sweep (sampling step, count rebuild, repair) timed on
    the host cores, from the library's state = (z, r) or (z, r, slot).

    full_sweeps = 0 (a bounded sample, about target_s + the rebuild): the
    sampling step over the first documents, sized to about target_s, against
    the sweep-start counts, and the count rebuild and repair of the whole
    corpus, timed once; the sweep's time is the sampling time scaled to all
    tokens plus the rebuild and repair time.  full_sweeps = S > 0: S whole
    sweeps of the oracle from the state, timed.  Both on all host threads and
    on one thread (one thread: whole sweeps only if they take at most two
    minutes, else the bounded sample)."""
    import numpy as np

    import oracle

    t0 = time.time()
    args = (cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab, wl.alpha, wl.a,
            wl.b, wl.gamma)
    m = oracle.Model(*args) if assoc is None else oracle.AssocModel(*args, *assoc)
    c = m.rebuild(*state)
    log(f"[bench] oracle model + dense counts ready in {time.time() - t0:.1f}s")
    threads = oracle.num_threads()
    N = m.N

    def rebuild_repair():
        st = [x.copy() for x in state]
        t = time.perf_counter()
        c2 = m.rebuild(*st, counts=c)
        m.repair(*st, c2)
        return time.perf_counter() - t

    def sampled(seconds, per_tok):
        """(tokens, seconds) of the sampling step over the first documents,
        sized to about `seconds`."""
        want = int(seconds / per_tok)
        d = max(1, min(int(np.searchsorted(m.doc_off, want)), m.D))
        t = time.perf_counter()
        m.sample_docs(c, *[x.copy() for x in state], 0, 1, 0, d)
        return int(m.doc_off[d]), time.perf_counter() - t, d

    def whole_sweeps(n):
        """Mean time of n whole sweeps: the sampling step of every document
        (in eight runs of documents, each logged), then rebuild and repair."""
        st = [x.copy() for x in state]
        cc = m.rebuild(*st)
        bounds = np.linspace(0, m.D, 9).astype(int)
        t = time.perf_counter()
        for k in range(n):
            for j in range(8):
                m.sample_docs(cc, *st, k, 1000 + seed, int(bounds[j]), int(bounds[j + 1]))
                if N > 10_000_000:
                    log(f"[bench] oracle sweep {k}: documents up to {bounds[j + 1]} sampled")
            cc = m.rebuild(*st, counts=cc)
            m.repair(*st, cc)
        return (time.perf_counter() - t) / n

    # calibration: a few documents
    d_cal = min(2048, m.D)
    t = time.perf_counter()
    m.sample_docs(c, *[x.copy() for x in state], 0, 1, 0, d_cal)
    per_tok = max(time.perf_counter() - t, 1e-6) / max(int(m.doc_off[d_cal]), 1)
    t_rr = rebuild_repair()  # serial: the same on one thread
    if full_sweeps > 0:
        t_sweep = whole_sweeps(full_sweeps)
        desc = (f"{full_sweeps} whole oracle sweep(s) (sampling step of all {N} tokens, count "
                f"rebuild, repair), fp64, OpenMP over documents: {t_sweep:.2f}s per sweep")
    else:
        toks, dt, d = sampled(target_s, per_tok)
        t_sweep = dt * N / max(toks, 1) + t_rr
        desc = (f"sampling step of the first {d} documents ({toks} tokens, {dt:.1f}s) against "
                f"the full sweep-start counts, scaled to all {N} tokens, plus the count rebuild "
                f"and repair of the whole corpus ({t_rr:.1f}s); fp64, OpenMP over documents")
    oracle.set_num_threads(1)
    try:
        t = time.perf_counter()
        m.sample_docs(c, *[x.copy() for x in state], 0, 1, 0, d_cal)
        per_tok1 = max(time.perf_counter() - t, 1e-6) / max(int(m.doc_off[d_cal]), 1)
        if full_sweeps > 0 and full_sweeps * (per_tok1 * N + t_rr) <= 120.0:
            t_sweep1 = whole_sweeps(full_sweeps)
            desc1 = f"{full_sweeps} whole oracle sweep(s) on one thread: {t_sweep1:.2f}s per sweep"
        else:
            toks1, dt1, d1 = sampled(target_s / 5, per_tok1)
            t_sweep1 = dt1 * N / max(toks1, 1) + t_rr
            desc1 = (f"sampling step of the first {d1} documents ({toks1} tokens, {dt1:.1f}s) on "
                     f"one thread, scaled to all tokens, plus the rebuild and repair "
                     f"({t_rr:.1f}s)")
    finally:
        oracle.set_num_threads(threads)
    return {
        "value": N / t_sweep,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": desc,
        "s_per_sweep": round(t_sweep, 4),
        "value_1thread": N / t_sweep1,
        "s_per_sweep_1thread": round(t_sweep1, 4),
        "sample_1thread": desc1,
        "host_cpu": host_cpu(),
    }


def read_probe(gib: int = 4, row_bytes: int = 2048, waves: int = 4096):
    """The device's read bandwidth, measured by the library's probe on a
    buffer of `gib` GiB: read whole, front to back (by 16 * `waves`
    wavefronts' worth of threads), and read as random rows of `row_bytes`,
    one row at a time per wavefront (`waves` of them, 16 per compute unit, as
    the sampler runs), each timed after one untimed run."""
    import torch

    from paper_1510_06549_amd import spdp as sp

    nbytes = gib << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    ptr = buf.data_ptr()
    st = torch.cuda.current_stream().cuda_stream
    out = {"buffer_GiB": gib, "row_bytes": row_bytes, "waves": waves}
    for key, rb in (("sequential_GBps", 0), ("random_rows_GBps", row_bytes)):
        rows = nbytes // max(rb, 1) if rb else 0
        w = 16 * waves if rb == 0 else waves
        sp.spdp_read_probe(ptr, nbytes, rb, rows, w, st)
        ms = sp.spdp_read_probe(ptr, nbytes, rb, rows, w, st)
        moved = nbytes if rb == 0 else -(-rows // waves) * waves * rb
        out[key] = round(moved / (ms * 1e-3) / 1e9, 1)
    del buf
    torch.cuda.synchronize()
    log(f"[bench] read probe {out}")
    return out


def copy_probe(mib: int):
    """A plain device copy of mib MiB: the known bytes that scale the HBM
    counters of the other kernels."""
    if mib <= 0:
        return
    import torch
    nbytes = mib << 20
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] copy probe: {nbytes} bytes read + {nbytes} bytes written")
    del src, dst


def heldout_bench(args, wl, cp):
    """--heldout S: fold-in sweeps of the test documents against the trained state."""
    import numpy as np
    import torch

    import synth
    from paper_1510_06549_amd import spdp as sp

    S = args.heldout
    tr, te = synth.split_heldout(cp, 0.1)
    log(f"[bench] held out: train {tr.n_tokens} tokens, test {te.n_tokens} tokens in "
        f"{te.n_docs} documents")
    assoc = (synth.associations(cp.n_groups, cp.vocab, args.assoc, args.assoc_eps, args.seed)
             if args.assoc > 0 else None)
    s = sp.Sampler(tr.words, tr.doc_off, tr.doc_group, tr.n_groups, wl.vocab, wl.K, wl.alpha,
                   wl.a, wl.b, wl.gamma, init_seed=args.seed,
                   hip_stream=torch.cuda.current_stream().cuda_stream, assoc=assoc)
    copy_probe(args.copy_probe_mib)
    seed = 1000 + args.seed
    for w in range(max(args.warmup, 1)):
        s.sweep(w, seed)
    s.heldout(te.words, te.doc_off, te.doc_group, 1, seed)
    torch.cuda.synchronize()
    log(f"[bench] {max(args.warmup, 1)} training sweep(s) and a warm-up fold-in done")
    t_one = t_many = 0.0
    ppl = None
    for k in range(args.steps):
        for n, acc in ((1, "one"), (S, "many")):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ppl, _, _ = s.heldout(te.words, te.doc_off, te.doc_group, n, seed + k)
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            if acc == "one":
                t_one += dt
            else:
                t_many += dt
        log(f"[bench] step {k}: held-out calls of 1 and {S} sweeps done, perplexity {ppl:.1f}")
    s.close()
    per_sweep = (t_many - t_one) / args.steps / (S - 1)
    T = te.n_tokens
    if assoc is None:
        bpt = foldin_bytes_per_token(wl.K)
    else:
        # the count row and one int32 shadow-base row per listed source of
        # each test token's row
        q = te.doc_group.astype(np.int64).repeat(np.diff(te.doc_off)) * cp.vocab + te.words
        mean_sources = float(np.diff(assoc[0])[q].mean())
        bpt = 4 * wl.K * (1.0 + mean_sources) + 12
    achieved = T * bpt / per_sweep / 1e9
    out = {
        "metric": "held-out test tokens folded in/sec per fold-in sweep (1 GPU) + % of HBM roofline",
        "value": round(T / per_sweep, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(per_sweep * 1000.0, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}-heldout",
            "train_tokens": tr.n_tokens,
            "test_tokens": T,
            "test_docs": te.n_docs,
            "foldin_sweeps": S,
            "topics": wl.K,
        },
        "perplexity": round(ppl, 2),
        "roofline": {
            "bound": "hbm",
            "kernel": "k_foldin",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "bytes_per_token": bpt,
            "ms_per_foldin_sweep": round(per_sweep * 1000.0, 3),
        },
        "cpu_baseline": None,
    }
    if assoc is not None:
        out["config"]["workload"] = f"{wl.name}-assoc{args.assoc}-heldout"
        out["config"]["sources_per_word"] = args.assoc
        out["config"]["assoc_eps"] = args.assoc_eps
        out["roofline"]["mean_sources_per_token"] = round(mean_sources, 4)
    print(json.dumps(out), flush=True)


def host_cpu() -> str:
    """The host CPU's model name and logical CPU count."""
    name = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                name = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return f"{name}, {os.cpu_count()} logical CPUs"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the measurement schedule of the largest workload: 20 timed sweeps after
    # 5 warm-up sweeps from the random initial state
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-read-probe", action="store_true",
                    help="skip the read-bandwidth probe reported beside the roofline")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cpu-sweeps", type=int, default=0,
                    help="time this many whole oracle sweeps instead of a bounded sample")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain device copy of this size (counter calibration)")
    ap.add_argument("--assoc", type=int, default=0,
                    help="sources per word of the word-association model (0: P = I)")
    ap.add_argument("--assoc-eps", type=float, default=0.3,
                    help="probability mass of the other sources of a word")
    ap.add_argument("--async", dest="async_sweep", action="store_true",
                    help="time the asynchronous (racy) sweep instead of the snapshot sweep")
    ap.add_argument("--async-waves", type=int, default=0,
                    help="wavefronts of the asynchronous sweep (0: library default)")
    ap.add_argument("--async-live-totals", action="store_true",
                    help="asynchronous sweep with the sums N, T, B_k updated live")
    ap.add_argument("--heldout", type=int, default=0,
                    help="time the held-out fold-in with this many sweeps instead")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the multi-GPU (group-sharded) sweep is not built; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.heldout and (args.heldout < 2 or args.async_sweep):
        print("bench.py: --heldout needs at least 2 fold-in sweeps and times the fold-in, "
              "not a sweep variant", file=sys.stderr)
        sys.exit(2)
    if args.async_sweep and args.assoc > 0:
        print("bench.py: the asynchronous sweep is built for P = I only", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_1510_06549_amd import spdp as sp

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = synth.workload(int(args.workload) if args.workload.isdigit() else args.workload)

    t0 = time.time()
    cp = synth.generate(wl, args.seed)
    log(f"[bench] workload {wl.name}: {cp.n_tokens} tokens, {cp.n_docs} docs, generated in "
        f"{time.time() - t0:.1f}s")

    if args.heldout:
        heldout_bench(args, wl, cp)
        return

    assoc = None
    if args.assoc > 0:
        t0 = time.time()
        assoc = synth.associations(cp.n_groups, cp.vocab, args.assoc, args.assoc_eps, args.seed)
        log(f"[bench] associations S={args.assoc} eps={args.assoc_eps}: {assoc[0][-1]} entries "
            f"in {time.time() - t0:.1f}s")

    stream = torch.cuda.current_stream()
    t0 = time.time()
    s = sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.vocab, wl.K, wl.alpha,
                   wl.a, wl.b, wl.gamma, init_seed=args.seed, hip_stream=stream.cuda_stream,
                   assoc=assoc)
    torch.cuda.synchronize()
    info = s.info
    log(f"[bench] state created in {time.time() - t0:.1f}s: {info}")

    copy_probe(args.copy_probe_mib)

    def one_sweep(k):
        if args.async_sweep:
            s.sweep_async(k, seed, args.async_waves, args.async_live_totals)
        else:
            s.sweep(k, seed)

    seed = 1000 + args.seed
    for w in range(args.warmup):
        one_sweep(w)
    torch.cuda.synchronize()
    log(f"[bench] {args.warmup} warm-up sweep(s) done")
    # width of the shadow-base rows the timed sweeps read (set by each rebuild)
    wide = shadow_base_wide(s)

    sp.spdp_kernel_timing(s.h, True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        one_sweep(args.warmup + k)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kt = sp.spdp_kernel_times(s.h)
    sp.spdp_kernel_timing(s.h, False)
    changed, repaired = s.stats()
    wide = wide or shadow_base_wide(s)
    log(f"[bench] {args.steps} timed sweeps in {elapsed:.3f}s; kernel ms {kt}; "
        f"last sweep changed={changed} repaired={repaired}")

    N = cp.n_tokens
    ms_step = 1000.0 * elapsed / args.steps
    value = N * args.steps / elapsed
    ms_sample, n_sample = kt["sample"]
    avg_sample_s = ms_sample / 1000.0 / max(n_sample, 1)
    if args.async_sweep:
        bpt = async_bytes_per_token(wl.K)
        traffic = None
    elif assoc is None:
        narrow = narrow_fraction(cp)
        bpt = sample_bytes_per_token(wl.K, wide, narrow)
        traffic = recorded_traffic("k_sample", wl.name)
    else:
        # mean length of the source list of each token's row
        lens = np.diff(assoc[0])
        q = np.repeat(cp.doc_group, np.diff(cp.doc_off)).astype(np.int64) * cp.vocab + cp.words
        mean_sources = float(lens[q].mean())
        Sp = 1 if s.S <= 1 else (2 if s.S <= 2 else (4 if s.S <= 4 else 8))
        narrow = narrow_fraction(cp)
        bpt = assoc_bytes_per_token(wl.K, wide, mean_sources, Sp, narrow)
        traffic = (recorded_traffic("k_sample_assoc", f"{wl.name}-assoc{args.assoc}")
                   if args.assoc_eps == 0.3 else None)
    alg = N * bpt
    achieved = alg / avg_sample_s / 1e9
    roofline = {
        "bound": "hbm",
        "kernel": ("k_sample_async" if args.async_sweep
                   else ("k_sample" if assoc is None else "k_sample_assoc")),
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": None if traffic is None else round(traffic / 1e9, 3),
        "traffic_unit": "GB per launch",
        "alg_bytes_per_launch_GB": round(alg / 1e9, 3),
        "bytes_per_token": round(bpt, 2),
        "shadow_base_bits": 32 if wide else 16,
        "avg_launch_ms": round(avg_sample_s * 1000.0, 3),
    }
    if args.async_sweep:
        pass
    elif assoc is None:
        roofline["narrow_row_token_share"] = round(narrow, 4)
        # context: the same launch time in the bytes of the layout without
        # narrow rows (32-bit count rows for every token)
        roofline["all_rows_32bit_equiv_GBps"] = round(
            N * sample_bytes_per_token(wl.K, wide, 0.0) / avg_sample_s / 1e9, 1)
        roofline["dense_int32_bytes_per_token"] = dense_bytes_per_token(wl.K)
        roofline["dense_int32_equiv_GBps"] = round(
            N * dense_bytes_per_token(wl.K) / avg_sample_s / 1e9, 1)
    else:
        roofline["narrow_row_token_share"] = round(narrow, 4)
        roofline["mean_sources_per_token"] = round(mean_sources, 4)

    if not args.no_read_probe:
        roofline["read_probe"] = read_probe()

    cpu = None
    if not args.no_cpu_baseline:
        state = s.assignments() + ((s.slots(),) if assoc is not None else ())
        s.close()
        cpu = cpu_baseline(cp, wl, state, args.cpu_seconds, assoc, args.cpu_sweeps, args.seed)
        log(f"[bench] cpu baseline {cpu}")
    else:
        s.close()

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "groups": wl.n_groups,
            "docs": cp.n_docs,
            "tokens": N,
            "vocab": wl.vocab,
            "topics": wl.K,
            "alpha": wl.alpha, "a": wl.a, "b": wl.b, "gamma": wl.gamma,
        },
        "kernels_ms_per_step": {k: round(v[0] / args.steps, 3) for k, v in kt.items()},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if args.async_sweep:
        out["config"]["workload"] = f"{wl.name}-async"
        out["config"]["async_waves"] = args.async_waves
        out["config"]["async_live_totals"] = bool(args.async_live_totals)
    if assoc is not None:
        out["config"]["workload"] = f"{wl.name}-assoc{args.assoc}"
        out["config"]["sources_per_word"] = args.assoc
        out["config"]["assoc_eps"] = args.assoc_eps
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
