"""Throughput benchmark of the HogBatch epoch on one MI355X.

Workload (large-vocabulary throughput configuration): a seeded i.i.d.
Zipf(1.07) corpus of 10^9 word ids over V = 1,000,000 words (standing in for
the one-billion-word benchmark of the paper's Sec. 2), D = 300 fp32,
window 5, K = 5 shared negatives from unigram^0.75, subsampling t = 1e-4,
alpha 0.025 decaying linearly. One step = one w2v_train_epoch over the whole
corpus (every kernel of the path, inputs already resident in HBM).

Prints one JSON line: Mwords/s (raw corpus words per second, before
subsampling), the roofline of the epoch kernel from HIP events recorded on its
stream, and the CPU oracle's rate on a bounded sample of the same workload.
"""
import argparse
import dataclasses
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_1611_06172_amd import configs  # noqa: E402

LV = configs.LargeVocab()     # the throughput workload
KT = configs.KernelTest()     # the snapshot-batch workload

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, 8 TB/s
METRIC = "Mwords/sec at V=1M D=300 K=5 window=5 (1 GPU); achieved HBM GB/s"
KERNEL_SOURCES = ["device_common.h", "sgns_core.h", "kernel_args.h",
                  "sentence.h", "epoch_kernels.hip"]


WORKLOAD_NAME = {"hogbatch": "HogBatch",
                 "hogbatch_immediate": "HogBatch (no pending input rows)",
                 "pairwise": "Algorithm 1 (per-pair)"}


def kernel_hash():
    """Hash of the epoch kernel's sources with comments and blank space
    removed, so that editing a comment does not void a counter summary."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_1611_06172_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(path):
    """Counter figures per launch from a committed summary (HBM bytes from the
    per-request-size memory-side counters, L2 bytes), if it was taken on the
    current kernel sources (else None)."""
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_hash") != kernel_hash():
        return None
    return d


def on_one_core(fn):
    """Runs fn() with this process pinned to the first CPU it may use (its
    GPU work is done by then); returns (result, seconds, cpu, n_cpus)."""
    allowed = sorted(os.sched_getaffinity(0))
    os.sched_setaffinity(0, {allowed[0]})
    try:
        c0 = time.perf_counter()
        out = fn()
        return out, time.perf_counter() - c0, allowed[0], len(allowed)
    finally:
        os.sched_setaffinity(0, set(allowed))


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--tokens", type=float, default=float(LV.T))
    ap.add_argument("--vocab", type=int, default=LV.V)
    ap.add_argument("--dim", type=int, default=LV.D)
    ap.add_argument("--negative", type=int, default=LV.K)
    ap.add_argument("--window", type=int, default=LV.window)
    ap.add_argument("--sample", type=float, default=LV.sample)
    ap.add_argument("--max-inflight", type=int, default=0)
    ap.add_argument("--group", type=int, default=1,
                    help="consecutive targets sharing one draw of negatives "
                         "(1: HogBatch as in the paper)")
    ap.add_argument("--algorithm", choices=["hogbatch", "hogbatch_immediate", "pairwise"],
                    default="hogbatch",
                    help="hogbatch (Sec. 1.1, the measured path), hogbatch_immediate "
                         "(the same kernel applying every input-row update at the "
                         "end of its minibatch) or pairwise (Alg. 1, the paper's "
                         "baseline)")
    ap.add_argument("--hot-tol", type=float, default=0.5,
                    help="expected concurrent writers above which a row is "
                         "updated atomically (w2v_hot_rows)")
    ap.add_argument("--hot-rows", type=int, default=-1,
                    help="override the atomic-row threshold (-1: model)")
    ap.add_argument("--split-tol", type=float, default=128.0,
                    help="expected concurrent writers above which a row is "
                         "spread over per-XCD partial rows (w2v_hot_rows)")
    ap.add_argument("--split-rows", type=int, default=-1,
                    help="override the split-row threshold (-1: model)")
    ap.add_argument("--split-max", type=int, default=2,
                    help="cap on the model's split rows: every read of a split "
                         "row sums its 8 partial rows, which outweighs the "
                         "spread atomics beyond the first one or two words")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run a 1 GiB device copy first (counter calibration)")
    ap.add_argument("--cpu-sample-tokens", type=int, default=3_000_000,
                    help="oracle baseline sample: the first tokens of the corpus "
                         "(about 27 s of one core at 3e6)")
    ap.add_argument("--literal-steps", type=int, default=3,
                    help="timed epochs of the paper-literal write-back "
                         "(hogbatch_immediate) run after the headline, reported "
                         "beside it (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", choices=["large-vocab", "kernel-test", "vocab", "row-rmw"],
                    default="large-vocab",
                    help="large-vocab: the HogBatch epoch (the measured path); "
                         "kernel-test: one snapshot batch of 65,536 minibatches "
                         "(w2v_step_batch); vocab: the vocabulary pipeline "
                         "(w2v_build_vocab) over --tokens raw ids; row-rmw: the memory "
                         "system's rate for the epoch's row accesses (measurement kernel)")
    ap.add_argument("--step-mode", choices=["sorted", "atomic"], default="sorted",
                    help="kernel-test: w2v_step_batch_sorted or w2v_step_batch")
    ap.add_argument("--traffic-json",
                    default=os.path.join(ROOT, "profiles", "k_epoch_traffic.json"))
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(sharding is a design, not code); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.workload == "kernel-test":
        kernel_test(args)
        return
    if args.workload == "vocab":
        vocab_bench(args)
        return
    if args.workload == "row-rmw":
        row_rmw_bench(args)
        return

    import numpy as np
    import torch

    from paper_1611_06172_amd import inputs, w2v

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    V, D, K, W = args.vocab, args.dim, args.negative, args.window
    T = int(args.tokens)
    L = LV.sentence
    cfg = dataclasses.replace(LV, T=T, V=V, D=D, K=K, window=W, sample=args.sample)

    t0 = time.time()
    corpus = inputs.zipf_corpus_hashed(T, V, LV.zipf_s, LV.corpus_seed, dev)
    counts = torch.bincount(corpus, minlength=V).cpu().numpy().astype(np.int64)
    table_h, thr_h = w2v.build_tables(counts, 0.75, args.sample, LV.table_size)
    table = torch.from_numpy(table_h).to(dev)
    thr = torch.from_numpy(thr_h.view(np.int32)).to(dev)
    M_in0 = inputs.init_matrix(V, D, "uniform", LV.init_seed)
    # rows padded to whole 128-byte lines (ld = 320 floats at D = 300)
    M_in = w2v.alloc_matrix(V, D, dev, torch.from_numpy(M_in0))
    M_out = w2v.alloc_matrix(V, D, dev)
    stats = torch.zeros(5, dtype=torch.int64, device=dev)
    inflight = args.max_inflight or w2v.default_inflight(D, W, K, V=V, group=args.group)
    hot = (args.hot_rows if args.hot_rows >= 0 else
           w2v.hot_rows(counts, sample_t=args.sample, window=W, K=K,
                        inflight=inflight, tol=args.hot_tol))
    split = (args.split_rows if args.split_rows >= 0 else
             min(args.split_max,
                 w2v.hot_rows(counts, sample_t=args.sample, window=W, K=K,
                              inflight=inflight, tol=args.split_tol)))
    if args.algorithm == "pairwise":
        split = 0  # partial rows serve the HogBatch kernel only
    pend_slots = (w2v.pending_slots(D, W, K)
                   if args.algorithm == "hogbatch" and args.group == 1 else 0)
    ld = M_in.stride(0)
    ws_bytes = w2v.train_epoch_workspace_bytes(split, ld)
    workspace = (torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
                 if ws_bytes else None)
    if args.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        src.fill_(1.0)
        dst = src.clone()
        del src, dst
    torch.cuda.synchronize()
    print(f"[bench] setup {time.time() - t0:.1f}s: T={T} V={V} D={D} K={K} w={W}",
          file=sys.stderr, flush=True)

    literal = (args.literal_steps if args.algorithm == "hogbatch" and args.group == 1
               else 0)
    n_epochs = args.warmup + args.steps + (1 + literal if literal else 0)

    def step(i, algorithm=args.algorithm):
        w2v.train_epoch(corpus, M_in, M_out, table, thr, window=W, K=K,
                        alpha0=LV.alpha0, min_alpha_frac=1e-4, epoch=i,
                        n_epochs=n_epochs, seed=LV.sampling_seed, sentence_len=L,
                        stats=stats, max_inflight=args.max_inflight,
                        hot_rows=hot, split_rows=split, workspace=workspace,
                        algorithm=algorithm, group=args.group)

    for i in range(args.warmup):
        step(i)
        torch.cuda.synchronize()
        print(f"[bench] warmup {i} done", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    stats.zero_()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        evs[i][0].record(stream)
        step(args.warmup + i)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    kern_ms = [a.elapsed_time(b) for a, b in evs]
    # a throughput of a diverged run is no measurement of the method
    if not (bool(torch.isfinite(M_in).all()) and bool(torch.isfinite(M_out).all())):
        raise RuntimeError("the timed epochs left non-finite values in the matrices "
                           "(Hogwild divergence at this concurrency and learning rate); "
                           "no throughput is reported")
    st = stats.cpu().numpy().astype(np.float64) / args.steps
    print(f"[bench] timed {args.steps} steps in {wall:.2f}s; per launch "
          f"{[round(x, 1) for x in kern_ms]} ms", file=sys.stderr, flush=True)

    ms_per_step = wall * 1e3 / args.steps
    words_per_s = T / (wall / args.steps)
    # Algorithmic bytes per launch: every HogBatch minibatch gathers and writes
    # back its N + K + 1 rows (8 D bytes per row) and reads K table entries;
    # Algorithm 1 moves, per input word, its own row and K + 1 output rows and
    # reads K table entries; every raw word reads its id and keep threshold.
    n_mb, sum_n, raw, rows = st[0], st[1], st[2], st[4]
    if args.algorithm == "pairwise":
        alg_bytes = 8.0 * D * sum_n * (K + 2) + 4.0 * K * sum_n + 8.0 * raw
    elif args.group > 1:
        # A group reads and writes each of its distinct rows once (stats[4]);
        # every retained target still draws its K table entries.
        alg_bytes = 8.0 * D * rows + 4.0 * K * n_mb + 8.0 * raw
    else:
        alg_bytes = 8.0 * D * (sum_n + n_mb * (K + 1)) + 4.0 * K * n_mb + 8.0 * raw
    avg_kern_s = float(np.mean(kern_ms)) / 1e3
    achieved = alg_bytes / avg_kern_s / 1e9
    counters = (measured_traffic(args.traffic_json)
                if args.algorithm == "hogbatch" and args.group == 1
                and T == 10**9 and (V, D, K, W) == (10**6, 300, 5, 5) else None)
    traffic = counters["hbm_bytes_per_launch"] if counters else None

    result = {
        "metric": METRIC,
        "value": round(words_per_s / 1e6, 3),
        "unit": "Mwords/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"large-vocab {WORKLOAD_NAME[args.algorithm]} "
                         f"epoch: i.i.d. Zipf(1.07) corpus, "
                         f"T={T}, V={V}, D={D}, K={K}, window={W}, sample={args.sample}, "
                         f"sentence {L}, alpha 0.025 linear"),
            "V": V, "T": T, "D": D, "ld": ld, "K": K, "window": W, "sample": args.sample,
            "group": args.group,
            "inflight_sentences": int(inflight), "atomic_rows": int(hot),
            "pending_slots": int(pend_slots),
            "split_rows": int(split),
            "minibatches_per_step": int(n_mb), "mean_inputs_per_minibatch":
                round(sum_n / max(n_mb, 1), 4), "retained_fraction": round(n_mb / raw, 4),
            "workload_config": json.loads(configs.to_json(cfg)),
            "steps_are": (f"epochs {args.warmup}..{args.warmup + args.steps - 1} of a "
                          f"{n_epochs}-epoch schedule (alpha decays over the schedule; each "
                          f"epoch continues from the previous one's matrices), after "
                          f"{args.warmup} untimed"),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("k_epoch_pairwise" if args.algorithm == "pairwise" else
                       "k_epoch_grouped" if args.group > 1 else "k_epoch"),
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": alg_bytes,
            "achieved_is": "algorithmic bytes (every row of every minibatch read "
                           "and written once) / launch time",
            "kernel_ms": round(avg_kern_s * 1e3, 3),
        },
    }
    if counters:
        # Measured at the memory side and in L2 (committed counter run on the
        # same kernel sources), divided by this run's launch time.
        hbm_gbs = traffic / avg_kern_s / 1e9
        result["roofline"]["hbm_measured_GBs"] = round(hbm_gbs, 1)
        result["roofline"]["hbm_measured_frac"] = round(hbm_gbs / HBM_PEAK_GBS, 4)
        if counters.get("l2_bytes_per_launch"):
            result["roofline"]["l2_GBs"] = round(
                counters["l2_bytes_per_launch"] / avg_kern_s / 1e9, 1)
        result["roofline"]["counters"] = os.path.relpath(args.traffic_json, ROOT)

    if literal:
        # The paper's write-back (Sec. 1.1: every update reaches the matrices
        # at the end of its minibatch) on the same kernel, continuing the
        # schedule: one untimed epoch, then `literal` timed ones.
        e0 = args.warmup + args.steps
        step(e0, "hogbatch_immediate")
        torch.cuda.synchronize()
        lev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(literal)]
        stats.zero_()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for i in range(literal):
            lev[i][0].record(stream)
            step(e0 + 1 + i, "hogbatch_immediate")
            lev[i][1].record(stream)
        torch.cuda.synchronize()
        lwall = time.perf_counter() - t1
        lms = float(np.mean([a.elapsed_time(b) for a, b in lev]))
        lst = stats.cpu().numpy().astype(np.float64) / literal
        lbytes = 8.0 * D * (lst[1] + lst[0] * (K + 1)) + 4.0 * K * lst[0] + 8.0 * lst[2]
        result["paper_literal_writeback"] = {
            "algorithm": "hogbatch_immediate",
            "value": round(T / (lwall / literal) / 1e6, 3), "unit": "Mwords/s",
            "steps": literal, "ms_per_step": round(lwall * 1e3 / literal, 3),
            "roofline_frac": round(lbytes / (lms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "note": "every input-row update written back at the end of its "
                    "minibatch (no pending LDS slots); epochs continue the "
                    "headline run's schedule",
        }
        print(f"[bench] paper-literal write-back: {literal} epochs, "
              f"{lms:.1f} ms per launch", file=sys.stderr, flush=True)

    if not args.no_cpu_baseline:
        import oracle
        n_s = min(args.cpu_sample_tokens, T)
        sample_corpus = corpus[:n_s].cpu().numpy()
        o_in = M_in0.copy()
        o_out = np.zeros((V, D), dtype=np.float32)
        s = oracle.Sampling(sample_corpus, table_h, thr_h, window=W, K=K,
                            sentence_len=L, seed=LV.sampling_seed, n_epochs=1)
        if args.algorithm == "pairwise":
            run = lambda: oracle.pairwise_train_epoch(s, o_in, o_out)  # noqa: E731
        elif args.group > 1:
            run = lambda: oracle.grouped_train_epoch(s, args.group, o_in, o_out)  # noqa: E731
        else:
            run = lambda: oracle.train_epoch(s, o_in, o_out)  # noqa: E731
        (n_o, _), c_dt, cpu, n_cpu = on_one_core(run)
        result["cpu_baseline"] = {
            "value": round(n_s / c_dt / 1e6, 5),
            "unit": "Mwords/s",
            "cores": 1,
            "kind": "oracle",
            "sample": (f"first {n_s} tokens of the same corpus as a 1-epoch run "
                       f"({n_o} minibatches, same tables and initial M_in), "
                       f"single-threaded fp64 oracle pinned to CPU {cpu}, "
                       f"{c_dt:.1f}s; CPU {cpu_model()}, {n_cpu} CPUs "
                       f"available to the process"),
        }
    print(json.dumps(result), flush=True)


def kernel_test(args):
    """One snapshot batch per step on the kernel-test configuration: B =
    65,536 minibatches of 1 target, N = 10 inputs and K = 5 negatives, i.i.d.
    Zipf(1.0) ids over V = 100,000, D = 300 (rows padded to 320), M ~ N(0,
    0.1^2), alpha 0.025."""
    import numpy as np
    import torch

    from paper_1611_06172_amd import inputs, w2v

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, N, K, V, D = KT.B, KT.N, KT.K, KT.V, KT.D
    t, c, n = inputs.kernel_batch(B, N, K, V, KT.zipf_s, KT.ids_seed)
    Mi0 = inputs.init_matrix(V, D, "normal", KT.init_seed)
    Mo0 = inputs.init_matrix(V, D, "normal", KT.init_seed + 100)
    M_in = w2v.alloc_matrix(V, D, dev, torch.from_numpy(Mi0))
    M_out = w2v.alloc_matrix(V, D, dev, torch.from_numpy(Mo0))
    T, C, Ng = (torch.from_numpy(x).to(dev) for x in (t, c, n))
    srt = args.step_mode == "sorted"
    if args.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        src.fill_(1.0)
        dst = src.clone()
        del src, dst
    ws = w2v.step_batch(T, C, Ng, M_in, M_out, KT.alpha, D=D, sorted=srt)  # allocates
    for _ in range(max(args.warmup, 0)):
        w2v.step_batch(T, C, Ng, M_in, M_out, KT.alpha, D=D, workspace=ws, sorted=srt)
    steps = max(args.steps, 1) * 20   # a batch takes about a millisecond
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(steps):
        evs[i][0].record(stream)
        w2v.step_batch(T, C, Ng, M_in, M_out, KT.alpha, D=D, workspace=ws, sorted=srt)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    call_ms = [a.elapsed_time(b) for a, b in evs]
    print(f"[bench] timed {steps} batches in {wall:.3f}s; median call "
          f"{float(np.median(call_ms)):.3f} ms", file=sys.stderr, flush=True)
    # Algorithmic bytes: every minibatch gathers and writes back its N + K + 1
    # rows (8 D bytes per row).
    alg_bytes = 8.0 * D * B * (N + K + 1)
    call_s = float(np.mean(call_ms)) / 1e3
    achieved = alg_bytes / call_s / 1e9
    entry = "w2v_step_batch_sorted" if srt else "w2v_step_batch"
    result = {
        "metric": "Mminibatches/sec, snapshot batch (kernel test)",
        "value": round(B / (wall / steps) / 1e6, 3),
        "unit": "Mminibatches/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"kernel-test snapshot batch ({entry}): B={B}, N={N}, "
                               f"K={K}, i.i.d. Zipf(1.0) ids over V={V}, D={D}, "
                               f"alpha 0.025",
                   "B": B, "N": N, "K": K, "V": V, "D": D, "ld": M_in.stride(0),
                   "workspace_bytes": int(ws.numel())},
        "roofline": {"bound": "hbm", "kernel": entry + " (all launches of one call)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None, "alg_bytes_per_launch": alg_bytes,
                     "kernel_ms": round(call_s * 1e3, 4),
                     "median_call_ms": round(float(np.median(call_ms)), 4)},
        "snapshot": ("no copy of the matrices: every minibatch reads the unchanged "
                     "matrices and its updates go to " +
                     ("staging rows summed in a fixed order" if srt else
                      "fp64 delta buffers") + ", applied after all minibatches"),
    }
    if not args.no_cpu_baseline:
        import oracle
        bs = B
        _, c_dt, cpu, n_cpu = on_one_core(lambda: oracle.step_batch(
            t[:bs], c[:bs], n[:bs], Mi0, Mo0, KT.alpha, D=D, with_scale=False))
        result["cpu_baseline"] = {
            "value": round(bs / c_dt / 1e6, 5), "unit": "Mminibatches/s",
            "cores": 1, "kind": "oracle",
            "sample": (f"the whole batch ({bs} minibatches), single-threaded fp64 "
                       f"oracle snapshot batch pinned to CPU {cpu}, {c_dt:.1f}s; "
                       f"CPU {cpu_model()}, {n_cpu} CPUs available to the process"),
        }
    print(json.dumps(result), flush=True)


def vocab_bench(args):
    """The vocabulary pipeline on --tokens raw ids: i.i.d. Zipf(1.07) over
    2,000,000 raw words whose ids are shuffled (so raw order is not frequency
    order); count, rank (ties by raw id), cut at min_count 5, rewrite the
    corpus in ranked ids."""
    import numpy as np
    import torch

    from paper_1611_06172_amd import inputs, w2v

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T, V_raw, min_count = int(args.tokens), 2_000_000, 5
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    perm = torch.randperm(V_raw, generator=g, device=dev).to(torch.int32)
    raw = perm[inputs.zipf_corpus_device(T, V_raw, 1.07, 6, dev).long()]
    del perm
    L = w2v.lib()
    ranked = torch.empty(V_raw, dtype=torch.int64, device=dev)
    rank_of = torch.empty(V_raw, dtype=torch.int32, device=dev)
    v_kept = torch.empty(1, dtype=torch.int32, device=dev)
    corpus = torch.empty(T, dtype=torch.int32, device=dev)
    ws = torch.empty(int(L.w2v_build_vocab_workspace_bytes(V_raw, T)), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream()

    def call():
        rc = L.w2v_build_vocab(w2v._ptr(raw), T, V_raw, min_count, w2v._ptr(ranked),
                               w2v._ptr(rank_of), w2v._ptr(v_kept), w2v._ptr(corpus),
                               w2v._ptr(ws), ws.numel(), w2v._stream(stream))
        w2v._check(rc)

    for _ in range(max(args.warmup, 0)):
        call()
    steps = max(args.steps, 1)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(steps):
        evs[i][0].record(stream)
        call()
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    call_ms = [a.elapsed_time(b) for a, b in evs]
    V = int(v_kept.item())
    print(f"[bench] timed {steps} calls in {wall:.3f}s; per call "
          f"{[round(x, 2) for x in call_ms]} ms; V = {V}", file=sys.stderr, flush=True)
    # Algorithmic bytes: the raw ids are read twice (count, rewrite) and the
    # rewritten corpus written once; the per-word arrays are negligible.
    alg_bytes = 12.0 * T
    call_s = float(np.mean(call_ms)) / 1e3
    achieved = alg_bytes / call_s / 1e9
    result = {
        "metric": "Mtokens/sec, vocabulary pipeline (count, rank, cut, rewrite)",
        "value": round(T / (wall / steps) / 1e6, 1), "unit": "Mtokens/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / steps, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int32/int64",
        "data": "synthetic",
        "config": {"workload": f"vocabulary of {T} i.i.d. Zipf(1.07) raw ids over "
                               f"{V_raw} shuffled raw words, min_count {min_count}",
                   "T": T, "V_raw": V_raw, "min_count": min_count, "V_kept": V},
        "roofline": {"bound": "hbm", "kernel": "w2v_build_vocab (all launches of one call)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "alg_bytes_per_launch": alg_bytes, "kernel_ms": round(call_s * 1e3, 3)},
    }
    if not args.no_cpu_baseline:
        import oracle
        n_s = min(T, 100_000_000)
        sample = raw[:n_s].cpu().numpy()
        _, c_dt, cpu, n_cpu = on_one_core(lambda: oracle.build_vocab(sample, V_raw,
                                                                     min_count))
        result["cpu_baseline"] = {
            "value": round(n_s / c_dt / 1e6, 2), "unit": "Mtokens/s", "cores": 1,
            "kind": "oracle",
            "sample": (f"first {n_s} raw ids, numpy bincount + stable argsort oracle "
                       f"pinned to CPU {cpu}, {c_dt:.1f}s; CPU {cpu_model()}, "
                       f"{n_cpu} CPUs available to the process"),
        }
    print(json.dumps(result), flush=True)


def row_rmw_bench(args):
    """The memory system's rate for the epoch's row accesses, without the
    method: the rows of the first 2e7 tokens' minibatches (the throughput
    workload's sampling, exported by w2v_debug_minibatches: input rows, the
    target and the negatives, in minibatch order), taken 12 per step by 2048
    wavefronts as the epoch's 2048 sentences in flight take them, each row
    read and written back in place (coherent load, write-through store) or,
    for the last `atomic_rows` of a step, added with fp32 atomics. Rows of
    D = 300 floats at ld = 320 in a 1e6-row matrix. Also uniform random ids.
    Bytes are counted as the epoch's algorithmic bytes: every row read and
    written once (2 x 1200 B). Then the snapshot batch's rows (kernel-test
    shape) with every update an fp32 atomic, against uniform ids."""
    import ctypes
    import numpy as np
    import torch

    from paper_1611_06172_amd import inputs, w2v

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    V, D, W, K, T = 1_000_000, 300, 5, 5, 20_000_000
    corpus = inputs.zipf_corpus_hashed(T, V, 1.07, 6, dev)
    counts = torch.bincount(corpus, minlength=V).cpu().numpy().astype(np.int64)
    table_h, thr_h = w2v.build_tables(counts, 0.75, 1e-4, 10**8)
    table = torch.from_numpy(table_h).to(dev)
    thr = torch.from_numpy(thr_h.view(np.int32)).to(dev)
    mb = w2v.debug_minibatches(corpus, table, thr, V=V, window=W, K=K, seed=1234)
    keep = mb["targets"] >= 0
    R = torch.cat([mb["ctx"][keep], mb["targets"][keep][:, None], mb["negs"][keep]], 1)
    R = R.reshape(-1)
    R = R[R >= 0]
    rows = 12
    n_steps = R.numel() // rows
    epoch_ids = R[: n_steps * rows].contiguous()
    g = torch.Generator(device=dev)
    g.manual_seed(12)
    uniform_ids = torch.randint(0, V, (n_steps * rows,), generator=g, device=dev,
                                dtype=torch.int32)
    del corpus, mb, R
    M = w2v.alloc_matrix(V, D, dev)
    ld = M.stride(0)
    L = ctypes.CDLL(os.path.join(ROOT, "paper_1611_06172_amd", "libw2v_measure.so"))
    L.w2v_measure_row_rmw.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_void_p]
    stream = torch.cuda.current_stream()
    grid = args.max_inflight or 2048
    results = {}
    for label, ids, n_atomic in (("epoch rows, 3 of 12 atomic", epoch_ids, 3),
                                 ("epoch rows, no atomics", epoch_ids, 0),
                                 ("uniform rows, no atomics", uniform_ids, 0)):
        def call():
            rc = L.w2v_measure_row_rmw(M.data_ptr(), V, D, ld, ids.data_ptr(), n_steps,
                                       rows, n_atomic, grid, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"w2v_measure_row_rmw failed ({rc})")
        for _ in range(max(args.warmup, 1)):
            call()
        steps = max(args.steps, 1)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(steps)]
        torch.cuda.synchronize()
        for i in range(steps):
            evs[i][0].record(stream)
            call()
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
        gbs = 2.0 * 4 * D * n_steps * rows / (ms * 1e-3) / 1e9
        results[label] = {"ms": round(ms, 3), "GBs": round(gbs, 1)}
        print(f"[bench] row-rmw {label}: {ms:.2f} ms, {gbs:.0f} GB/s", file=sys.stderr,
              flush=True)
    # The snapshot batch's shape with every update atomic: the 16 rows of each
    # of 65,536 kernel-test minibatches (Zipf(1.0) ids over 1e5 words, as
    # w2v_step_batch adds them) against the same number of uniform ids, one
    # minibatch per wavefront; the rate of the memory side's atomics with and
    # without the head rows' contention.
    Vk, Bk, Rk = 100_000, 65536, 16
    t, c, n = inputs.kernel_batch(Bk, 10, 5, Vk, 1.0, 3)
    kt_ids = torch.from_numpy(np.ascontiguousarray(
        np.concatenate([c, t[:, None], n], 1).astype(np.int32).reshape(-1))).to(dev)
    kt_uniform = torch.randint(0, Vk, (Bk * Rk,), generator=g, device=dev, dtype=torch.int32)
    Mk = w2v.alloc_matrix(Vk, D, dev)
    per_row = (4 * D + 63) // 64     # 64-byte requests of one row's fp32 atomics
    for label, ids in (("kernel-test rows, all atomic", kt_ids),
                       ("uniform rows (V 1e5), all atomic", kt_uniform)):
        def call():
            rc = L.w2v_measure_row_rmw(Mk.data_ptr(), Vk, D, Mk.stride(0), ids.data_ptr(),
                                       Bk, Rk, Rk, Bk, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"w2v_measure_row_rmw failed ({rc})")
        call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(max(args.steps, 1)):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / max(args.steps, 1)
        rate = Bk * Rk * per_row / (ms * 1e-3)
        results[label] = {"ms": round(ms, 3), "atomic_requests_per_s": float(f"{rate:.4g}")}
        print(f"[bench] row-rmw {label}: {ms:.3f} ms, {rate / 1e9:.2f} G requests/s",
              file=sys.stderr, flush=True)
    head = results["epoch rows, 3 of 12 atomic"]
    result = {
        "metric": "GB/s, random row read-modify-write (the epoch's row accesses without "
                  "the method)",
        "value": head["GBs"], "unit": "GB/s", "n_gpus": 1, "steps": max(args.steps, 1),
        "warmup": max(args.warmup, 1), "ms_per_step": head["ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"rows of the throughput workload's first {T} tokens' "
                               f"minibatches, {rows} per step, {grid} wavefronts, D={D}, "
                               f"ld={ld}, V={V}",
                   "steps_per_call": n_steps, "rows_per_step": rows, "variants": results},
        "roofline": {"bound": "hbm", "kernel": "k_row_rmw", "achieved": head["GBs"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(head["GBs"] / HBM_PEAK_GBS, 4), "traffic": None},
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
