"""Throughput of the clocked SSP/ESSP matrix-factorization SGD sweep on one MI355X.

One step = one clock of all P logical workers over one minibatch (sweep: residuals, dL
segment sums, dR accumulation; commit: the new version), i.e. every per-clock step of the
method.  The default workload is the Netflix-shaped 100M-rating matrix (480,189 users x
17,770 items, Zipf(1.1) user degrees capped at the item count, Zipf(0.9) item
popularity), rank K=128, P=64 workers, s=3, eta=0.002, lambda=0.05, one full shard per
clock; inputs are seeded synthetic data resident in HBM before timing starts.

Prints one JSON line: rating-updates/s, the dominant kernel's roofline position (HIP
events on the library's stream) and the CPU oracle timed on a bounded sample.

``--workload lda`` measures the second workload of the paper's Section 5 instead: LDA by
collapsed Gibbs sampling under SSP / ESSP, one step = one clock of all P workers over one
minibatch block of the tokens, on a seeded corpus drawn from the LDA generative process
(the "small" corpus: 20,000 documents of Poisson(200) tokens, 20,000 Zipf-shaped words,
K=100, P=64, s=3, ESSP, half of the tokens per clock; ``--corpus nyt``: the paper's shape,
100M tokens, 100,000 words, K=100, P=512); the line reports Gibbs-sampled tokens/s.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_VECTOR_TFLOPS = 157.3   # MI355X published fp32 vector peak (packed FMA)
PEAK_HBM_GBS = 8000.0             # MI355X HBM3E
POLICIES = {"lazy": 0, "worst": 1, "essp": 2, "ssp_row": 3, "essp_row": 4, "vap": 5}
LDA_POLICIES = {"lazy": 0, "worst": 1, "essp": 2}
STEPS = {"rowmean": 0, "sum": 1, "seq": 2}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30, help="timed clocks")
    ap.add_argument("--warmup", type=int, default=3, help="untimed clocks before timing")
    ap.add_argument("--config", default="full")
    ap.add_argument("--s", type=int, default=None, help="staleness (default: 3 for the full config)")
    ap.add_argument("--workload", default="mf", choices=("mf", "lda"),
                    help="mf: matrix-factorization SGD (default); lda: collapsed Gibbs sampling for LDA")
    ap.add_argument("--corpus", default="small", help="lda corpus")
    ap.add_argument("--workers", type=int, default=None, help="lda: P (default: the corpus's)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="lda: oracle clocks timed for about this long")
    ap.add_argument("--policy", default=None, choices=sorted(POLICIES),
                    help="default: lazy (mf), essp (lda: lazy, worst or essp)")
    ap.add_argument("--step", default="rowmean", choices=sorted(STEPS),
                    help="rowmean/sum: one fixed view per worker and clock; seq: every worker applies its "
                         "ratings one by one to its own rows")
    ap.add_argument("--strata", type=int, default=None, help="sub-epochs per clock of the seq step")
    ap.add_argument("--value-bound", type=float, default=None, help="v0 of the vap policy (v_t = v0 / sqrt(t))")
    ap.add_argument("--eta-decay", action="store_true", help="step eta / sqrt(c + 1) at clock c")
    ap.add_argument("--cpu-sample", type=int, default=10_000_000,
                    help="ratings in the oracle's timed sample (0 disables the CPU baseline)")
    ap.add_argument("--all-s", type=int, default=1,
                    help="1 (default): also time every other staleness bound of the configuration (one handle "
                         "each, same ratings) and report them under config.per_s; 0: only --s")
    ap.add_argument("--no-timing", action="store_true", help="do not record per-kernel events")
    ap.add_argument("--tile-bytes", type=int, default=None, help="bytes of user rows per L2 tile of the item-major sweep")
    ap.add_argument("--item-tile-bytes", type=int, default=None,
                    help="bytes of item rows per L2 tile of the user-major sweep (default 4 x --tile-bytes)")
    ap.add_argument("--unit-max", type=int, default=None, help="ratings per sweep work unit")
    ap.add_argument("--cells", type=int, default=None, help="1/0: LDS-staged cells for the dense part")
    ap.add_argument("--heavy-min", type=int, default=None, help="ratings from which a user goes to the cells")
    ap.add_argument("--two-streams", type=int, default=None, help="1/0: units on a second stream beside the cells")
    ap.add_argument("--sweep-graphs", type=int, default=None,
                    help="1/0: replay each clock's sweep launches from a captured HIP graph (default: 0)")
    ap.add_argument("--unit-commit", type=int, default=None,
                    help="1/0: a user's only work unit writes its new version (default: 1)")
    ap.add_argument("--hot-steps", type=int, default=None,
                    help="LDS sub-tiles of the most rated items whose light-user ratings go to cells (-1: auto)")
    ap.add_argument("--dense-min", type=int, default=None,
                    help="ratings from which a 64x64 tile is swept by the matrix-core cells (0: none, -1: auto)")
    ap.add_argument("--copy-calibration-bytes", type=int, default=0,
                    help="run one plain copy kernel (y = x * 2) of this many bytes before timing, for "
                         "calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE")
    ap.add_argument("--traffic-file", default=None,
                    help="measured HBM traffic of the sweep, used while the kernel source is unchanged (default: "
                         "profiles/sweep_full_traffic.json, or profiles/seq_full_traffic.json for --step seq)")
    return ap.parse_args()


def host_cpu():
    """The host CPU's model name (from /proc/cpuinfo) and the number of cores this process may use."""
    model = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        nproc = os.cpu_count() or 1
    return model, nproc


def pinned_to_one_core(fn):
    """Run fn with this process pinned to one of its allowed cores (as taskset -c would), then
    restore the affinity; returns (fn's result, the core)."""
    try:
        allowed = sorted(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        return fn(), None
    core = allowed[0]
    os.sched_setaffinity(0, {core})
    try:
        return fn(), core
    finally:
        os.sched_setaffinity(0, set(allowed))


def cpu_baseline(w, spec, K, s, policy, step, strata, value_bound, eta_decay, nsample, repeats=5):
    """The oracle, single-threaded and pinned to one core, on the ratings of a prefix of users:
    the median of `repeats` timed clocks (every clock sweeps the same ratings)."""
    import oracle

    order = np.argsort(w.user, kind="stable")
    take = order[:nsample]
    u, i, v = w.user[take], w.item[take], w.val[take]
    o = oracle.Oracle(spec.N, spec.M, K, spec.P, s, spec.eta, spec.lam, policy, step, spec.B, spec.seed,
                      strata=strata, value_bound=value_bound, eta_decay=eta_decay)
    o.load(u, i, v)
    o.set_factors(w.L0, w.R0)

    def timed():
        out = []
        for _ in range(repeats):
            t0 = time.perf_counter()
            o.clock(1)
            out.append(time.perf_counter() - t0)
        return out

    times, core = pinned_to_one_core(timed)
    o.close()
    dt = float(np.median(times))
    model, nproc = host_cpu()
    return {"value": len(take) / dt, "unit": "rating-updates/s", "cores": 1, "kind": "oracle",
            "sample": f"median of {repeats} clocks, each over the {len(take)} ratings of users {int(u.min())}.."
                      f"{int(u.max())} (users in id order) of the same workload: {dt:.2f} s per clock "
                      f"(all: {', '.join(f'{x:.2f}' for x in times)} s); 1 thread pinned to core {core} of "
                      f"{nproc} on {model}",
            "host": {"cpu": model, "nproc": nproc, "pinned_core": core}}


def measured_traffic(path, config, s, policy, step):
    """HBM bytes per clock of the sweep from committed rocprofv3 counter runs, or None when
    they are missing, were taken on another workload, or the kernel source has changed."""
    from paper_1410_8043_amd import rocprof_summary

    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != rocprof_summary.kernel_source_sha256():
        return None
    want = {"config": config, "s": s, "policy": policy}
    if step != "rowmean":
        want["step"] = step
    if t.get("workload") != want:
        return None
    return round(t["traffic_bytes_per_clock"])


def lda_cpu_baseline(corpus, spec, P, s, policy, seconds, max_tokens=8_000_000):
    """The oracle, single-threaded, running whole clocks for about `seconds`: on the same corpus,
    or on its first documents (tokens of a document are contiguous) when it holds more than
    max_tokens, so that one clock stays a few seconds."""
    import oracle

    n = corpus.ntok if corpus.ntok <= max_tokens else int(np.searchsorted(corpus.doc, corpus.doc[max_tokens]))
    D = spec.D if n == corpus.ntok else int(corpus.doc[n])
    o = oracle.LdaOracle(D, spec.V, spec.K, P, s, spec.alpha, spec.beta, policy, spec.B, spec.seed)
    o.load(corpus.doc[:n], corpus.word[:n], corpus.z0[:n])
    sizes = [o.export(oracle.LDA_BLOCK_ORDER, b).size for b in range(spec.B)]

    def timed():
        clocks, tokens = 0, 0
        t0 = time.perf_counter()
        while clocks == 0 or time.perf_counter() - t0 < seconds:
            o.clock(1)
            tokens += sizes[clocks % spec.B]
            clocks += 1
        return clocks, tokens, time.perf_counter() - t0

    (clocks, tokens, dt), core = pinned_to_one_core(timed)
    o.close()
    model, nproc = host_cpu()
    what = "the same corpus" if n == corpus.ntok else f"the first {D} documents ({n} tokens) of the same corpus"
    return {"value": tokens / dt, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"the first {clocks} clocks of {what} with the same settings ({tokens} token draws), "
                      f"{dt:.1f} s, 1 thread pinned to core {core} of {nproc} on {model}",
            "host": {"cpu": model, "nproc": nproc, "pinned_core": core}}


def lda_main(args):
    import torch

    from paper_1410_8043_amd import ps_lda, rocprof_summary
    from paper_1410_8043_amd.synth import lda_corpus as lc

    spec = lc.CORPORA[args.corpus]
    P = args.workers or spec.P
    s = args.s if args.s is not None else spec.s
    pname = args.policy or "essp"
    if pname not in LDA_POLICIES:
        raise SystemExit(f"--policy {pname} is not an LDA policy (lazy, worst, essp)")
    policy = LDA_POLICIES[pname]
    torch.cuda.set_device(0)
    t_gen = time.perf_counter()
    corpus = lc.generate(spec)
    print(f"[bench] generated lda {args.corpus}: {corpus.ntok} tokens in {time.perf_counter() - t_gen:.1f} s",
          file=sys.stderr, flush=True)
    g = ps_lda.PsLda(spec.D, spec.V, spec.K, P, s, spec.alpha, spec.beta, policy=policy, B=spec.B, seed=spec.seed,
                     timing=not args.no_timing, stream=torch.cuda.current_stream())
    t_load = time.perf_counter()
    g.load(corpus.doc, corpus.word, corpus.z0)
    print(f"[bench] layout + upload {time.perf_counter() - t_load:.1f} s", file=sys.stderr, flush=True)
    # tokens and (worker, document) runs of each block: a run reads and writes its doc-topic row
    tokens_b, runs_b = [], []
    for b in range(spec.B):
        d = corpus.doc[g.export(ps_lda.X_BLOCK_ORDER, b)]
        tokens_b.append(d.size)
        runs_b.append(int(d.size > 0) + int(np.count_nonzero(d[1:] != d[:-1])))
    ll0 = g.loglik()
    if args.copy_calibration_bytes > 0:
        src = torch.ones(args.copy_calibration_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 2.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    g.clock(args.warmup)
    torch.cuda.synchronize()
    base = g.kernel_time() if not args.no_timing else None
    t0 = time.perf_counter()
    g.clock(args.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(f"[bench] {args.steps} clocks in {dt * 1e3:.2f} ms", file=sys.stderr, flush=True)
    ll = g.loglik()
    timed = [(args.warmup + i) % spec.B for i in range(args.steps)]
    tokens = sum(tokens_b[b] for b in timed)
    K = spec.K
    roof, extra = None, {}
    if not args.no_timing:
        ms, n = g.kernel_time()
        launch_ms = (ms - base[0]) / (n - base[1])
        # per token: its 16-byte record, topic and row tag (4 + 4), the word's view row and own-
        # change row (2 x 4K); per (worker, document) run: the doc-topic row read and written
        bytes_launch = sum(tokens_b[b] * (8.0 * K + 24) + runs_b[b] * 8.0 * K for b in timed) / len(timed)
        achieved = bytes_launch / (launch_ms * 1e-3) / 1e9
        traffic = None
        try:
            with open(os.path.join(ROOT, "profiles", f"lda_{args.corpus}_traffic.json")) as f:
                t = json.load(f)
            src = os.path.join(ROOT, "paper_1410_8043_amd", "csrc", "ps_lda.hip")
            if (t.get("kernel_source_sha256") == rocprof_summary.kernel_source_sha256(src) and
                    t.get("workload") == {"config": args.corpus, "s": s, "policy": pname, "step": "lda"} and
                    P == spec.P):
                traffic = round(t["traffic_bytes_per_clock"])
        except (OSError, ValueError):
            pass
        roof = {"kernel": "k_lda_sweep (one launch per clock)", "bound": "hbm", "achieved": round(achieved, 2),
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 5), "traffic": traffic}
        extra = {"sweep_ms": round(launch_ms, 4), "token_latency_us": round(launch_ms * 1e3 * P / (tokens / len(timed)), 4)}
    g.close()
    cpu = None
    if args.cpu_sample > 0 and args.cpu_seconds > 0:
        print("[bench] timing the oracle", file=sys.stderr, flush=True)
        cpu = lda_cpu_baseline(corpus, spec, P, s, policy, args.cpu_seconds)
    line = {
        "metric": f"Gibbs-sampled tokens/sec, LDA K={K}, {corpus.ntok / 1e6:.1f}M tokens (1 GPU)",
        "value": round(tokens / dt, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic (seeded LDA generative process, Zipf-shaped topics)",
        "config": {"workload": f"lda {args.corpus}: {spec.D} documents, {spec.V} words, {corpus.ntok} tokens, K={K}, "
                               f"P={P}, s={s}, policy={pname}, B={spec.B}, alpha={spec.alpha}, beta={spec.beta}",
                   "global_batch": int(tokens / len(timed)), "parallelism": "1 GPU, P logical workers",
                   "loglik_before": ll0, "loglik_after": ll, **extra},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def measure_mf(args, spec, w, s, policy, step, stream, announce=True):
    """Build a handle for staleness s, run the warmup and the timed clocks, and return what
    the JSON line reports about them."""
    import torch

    from paper_1410_8043_amd import ps_mf

    seq = args.step == "seq"
    g = ps_mf.PsMf(spec.N, spec.M, spec.K, spec.P, s, spec.eta, spec.lam, policy=policy, step=step, strata=args.strata,
                   value_bound=args.value_bound, eta_decay=args.eta_decay, B=spec.B,
                   mb_seed=spec.seed, timing=not args.no_timing, stream=stream, tile_bytes=args.tile_bytes,
                   unit_max=args.unit_max, cells=args.cells, heavy_min=args.heavy_min, hot_steps=args.hot_steps,
                   two_streams=args.two_streams, dense_min=args.dense_min, item_tile_bytes=args.item_tile_bytes,
                   sweep_graphs=args.sweep_graphs, unit_commit=args.unit_commit)
    t_load = time.perf_counter()
    g.load_ratings(w.user, w.item, w.val)
    g.set_factors(w.L0, w.R0)
    t_load = time.perf_counter() - t_load
    print(f"[bench] s={s}: layout + upload {t_load:.1f} s", file=sys.stderr, flush=True)
    nnz_clock = w.nnz / spec.B  # mean ratings per clock (exact for B=1)
    split = sum(g.export_index(ps_mf.IDX_SPLIT, b) for b in range(spec.B))
    if announce and seq:
        print(f"[bench] sequential step: {int(split[0])} chains, {int(split[1])} user runs, {int(split[2])} ratings "
              f"over {spec.B} blocks", file=sys.stderr, flush=True)
    elif announce:
        print(f"[bench] ratings per direction in dense tiles / LDS cells / L2 units: {split[:3].tolist()} "
              f"(user-major), {split[3:6].tolist()} (item-major); partial rows {split[6:].tolist()}",
              file=sys.stderr, flush=True)

    if announce and args.copy_calibration_bytes > 0:
        src = torch.ones(args.copy_calibration_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 2.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    g.clock(args.warmup)
    torch.cuda.synchronize()
    if not args.no_timing:
        base_sweep = g.kernel_time(ps_mf.KERNEL_SWEEP)
        base_commit = g.kernel_time(ps_mf.KERNEL_COMMIT)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g.clock(args.steps)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(f"[bench] s={s}: {args.steps} clocks in {dt * 1e3:.2f} ms", file=sys.stderr, flush=True)
    loss = g.loss()
    # staleness profile of the clocks run (Fig. 1 left): share of parameter reads per clock
    # differential -(d+1)
    stale = g.export_index(ps_mf.IDX_STALENESS)
    profile = {str(-(d + 1)): round(float(x) / max(1, int(stale.sum())), 4) for d, x in enumerate(stale)}
    out = {"s": s, "dt": dt, "value": nnz_clock * args.steps / dt, "nnz_clock": nnz_clock, "split": split,
           "loss": loss, "profile": profile, "roof": None, "extra": {}}
    K = spec.K
    if not args.no_timing:
        ms_s, n_s = g.kernel_time(ps_mf.KERNEL_SWEEP)
        ms_c, n_c = g.kernel_time(ps_mf.KERNEL_COMMIT)
        sweep_ms = (ms_s - base_sweep[0]) / (n_s - base_sweep[1])
        commit_ms = (ms_c - base_commit[0]) / (n_c - base_commit[1])
        traffic = measured_traffic(args.traffic_file, args.config, s, args.policy, args.step)
        # compulsory HBM bytes of one clock: each rating once (int32 item + fp32 value),
        # the view version read, the base version read when s > 0, the new version written
        table = (spec.N + spec.M) * K * 4
        hbm_bytes = 8 * nnz_clock + table * (2 if s == 0 else 3)
        if seq:
            # the sequential step is HBM-bound: priced against the compulsory bytes of a clock
            # (the layout's own round trips of the workers' row copies are not algorithmic)
            achieved = hbm_bytes / (sweep_ms * 1e-3) / 1e9  # GB/s
            roof = {"kernel": "k_seq (one launch per sub-epoch)", "bound": "hbm", "achieved": round(achieved, 1),
                    "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 5),
                    "traffic": traffic}
            # what the layout moves: each rating reads and writes its item row in the worker's
            # copy (2 x 4K bytes) and reads its 16-byte record; each user run reads and writes
            # the user row
            runs_clock = float(split[1]) / spec.B
            moved = nnz_clock * (8.0 * K + 16) + runs_clock * 8.0 * K
            out["extra"]["layout_bytes_frac"] = round(moved / (sweep_ms * 1e-3) / (PEAK_HBM_GBS * 1e9), 4)
        else:
            flops = 6.0 * K * nnz_clock                  # 3K fp32 FMA per rating update
            achieved = flops / (sweep_ms * 1e-3) / 1e12  # TFLOP/s
            roof = {"kernel": "sweep (k_dense, k_cells and k_units, concurrent)", "bound": "alu",
                    "achieved": round(achieved, 3), "peak": PEAK_FP32_VECTOR_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_VECTOR_TFLOPS, 4), "traffic": traffic}
        out["roof"] = roof
        out["extra"].update({"sweep_ms": round(sweep_ms, 4), "commit_ms": round(commit_ms, 4),
                             "hbm_algorithmic_frac": round(hbm_bytes / (dt / args.steps) / (PEAK_HBM_GBS * 1e9), 4)})
    g.close()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU path is a design, not part of this build)", file=sys.stderr)
        sys.exit(2)
    if args.workload == "lda":
        return lda_main(args)
    if args.policy is None:
        args.policy = "lazy"
    if args.traffic_file is None:
        name = "seq_full_traffic.json" if args.step == "seq" else "sweep_full_traffic.json"
        args.traffic_file = os.path.join(ROOT, "profiles", name)
    import torch

    from paper_1410_8043_amd import synth

    spec = synth.CONFIGS[args.config]
    s = args.s if args.s is not None else (3 if 3 in spec.s_values else spec.s_values[0])
    policy = POLICIES[args.policy]
    step = STEPS[args.step]
    seq = args.step == "seq"
    torch.cuda.set_device(0)
    t_gen = time.perf_counter()
    w = synth.generate(spec)
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] generated {args.config}: {w.nnz} ratings in {t_gen:.1f} s", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    main_run = measure_mf(args, spec, w, s, policy, step, stream)
    # the other staleness bounds of the configuration, each on its own handle over the same
    # ratings, with the same warmup and timed clocks
    per_s = {}
    others = [x for x in spec.s_values if x != s] if args.all_s else []
    for x in others:
        r = measure_mf(args, spec, w, x, policy, step, stream, announce=False)
        per_s[str(x)] = {"value": round(r["value"], 1), "ms_per_step": round(r["dt"] / args.steps * 1e3, 4),
                         **({k: r["extra"][k] for k in ("sweep_ms", "commit_ms")} if r["extra"] else {}),
                         **({"frac": r["roof"]["frac"]} if r["roof"] else {}),
                         "loss_after": r["loss"] if np.isfinite(r["loss"]) else None}
    if per_s:
        r = main_run
        per_s[str(s)] = {"value": round(r["value"], 1), "ms_per_step": round(r["dt"] / args.steps * 1e3, 4),
                         **({k: r["extra"][k] for k in ("sweep_ms", "commit_ms")} if r["extra"] else {}),
                         **({"frac": r["roof"]["frac"]} if r["roof"] else {}),
                         "loss_after": r["loss"] if np.isfinite(r["loss"]) else None}
        per_s = {k: per_s[k] for k in sorted(per_s, key=int)}

    cpu = None
    if args.cpu_sample > 0:
        print("[bench] timing the oracle on a sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, spec, spec.K, s, policy, step, args.strata, args.value_bound, args.eta_decay,
                           min(args.cpu_sample, w.nnz))

    r = main_run
    loss, split = r["loss"], r["split"]
    line = {
        "metric": "rating-updates/sec at K=128, 100M ratings (1 GPU); % of HBM roofline",
        "value": round(r["value"], 1),
        "unit": "rating-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["dt"] / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded, Netflix-shaped)",
        "config": {"workload": f"{args.config}: {spec.N} users x {spec.M} items, {w.nnz} ratings, K={spec.K}, "
                               f"P={spec.P}, s={s}, policy={args.policy}, B={spec.B}, eta={spec.eta}, "
                               f"lambda={spec.lam}" + (f", step=seq, strata={args.strata or 256}" if seq else "") +
                               (f", v0={args.value_bound}" if args.policy == "vap" else "") +
                               (", eta/sqrt(t)" if args.eta_decay else ""),
                   "global_batch": int(r["nnz_clock"]), "parallelism": "1 GPU, P logical workers",
                   # null when the run diverged (strict JSON has no NaN)
                   "loss_after": loss if np.isfinite(loss) else None,
                   **({"chains_runs_ratings": [int(x) for x in split[:3]]} if seq else
                      {"dense_cells_units": [int(x) for x in split[:3]]}),
                   "staleness_profile": r["profile"], **r["extra"],
                   **({"per_s": per_s} if per_s else {})},
        "roofline": r["roof"],
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
