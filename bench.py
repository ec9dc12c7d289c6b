"""Throughput of the ALTR token-reduction path on one MI355X.

A step is one whole reduction (score -> select -> gather, every kernel of the
path) of one batch: 64 LLaVA-1.5-style images of 576 tokens x 4096 bf16
channels (plus their pre-/post-MLP states) reduced to 64 tokens each.  Inputs
are seeded synthetic tensors resident in HBM before the timed region.

Prints one JSON line with images/s, the roofline of the dominant kernel (the
fused scoring pass, HBM-bound) and the fp64 CPU oracle timed on the host.  The
default run also times the other benchmark workloads the same way (the
single-image fp32 case as microseconds per call over 64 rotated copies of its
buffers, so that no call finds its inputs in the 256 MB last-level cache) and
reports them under "workloads".
"""
from __future__ import annotations

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
METRIC = "images/s reducing 576x4096 bf16 to 64 tokens; achieved HBM GB/s vs peak"
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "score_kernel_traffic_llava_b64_576x4096_bf16.md")


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llava", choices=["llava", "llava_fp32", "llava_next",
                                                              "qwen_ragged", "video"],
                    help="llava (the headline: 64 x 576 x 4096 bf16) or another benchmark "
                         "workload of the synth module at its full size")
    ap.add_argument("--K", type=int, default=64, choices=[64, 128, 192],
                    help="kept tokens per image of the llava workload")
    ap.add_argument("--images", type=int, default=64, help="images of the llava workload")
    ap.add_argument("--lam", type=float, default=None,
                    help="balance factor lambda (default 1/3, the paper's setting); 1 and 0 are "
                         "the ablations without the diversity / importance stage, which skip "
                         "the score they do not use")
    ap.add_argument("--stride-real", action="store_true",
                    help="real-interval variant of the diversity stride")
    ap.add_argument("--shannon", action="store_true",
                    help="Shannon-entropy variant of the Stage I score")
    ap.add_argument("--mlp-fused", action="store_true",
                    help="the step before the path: X_post from the encoder MLP's second layer "
                         "(Dc = 1024, hidden 4096) with Eq. 6 fused into its epilogue, then the "
                         "module on the given key; timed against the library GEMM + tr_reduce")
    ap.add_argument("--project", type=int, default=0, metavar="NOUT",
                    help="the step after the path: project the kept tokens by a [NOUT, D] weight "
                         "inside the module (gather fused into the GEMM); timed against "
                         "tr_reduce + the library GEMM")
    ap.add_argument("--gemm", default="", metavar="M,N,K",
                    help="the matrix-core GEMM core alone: C[M,N] = A[M,K] . B[N,K]^T in bf16, timed "
                         "against the library GEMM (torch.matmul) on the same operands")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-workloads", action="store_true",
                    help="time the headline workload only (no 'workloads' object)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the oracle sample")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the measurement, run 3 plain device copies of this many MiB "
                         "(the reference dispatch for scaling PMC byte counters)")
    return ap.parse_args()


def score_source_sha() -> str:
    """sha256 of the scoring kernel's sources: the kernel, its interface header
    and the wavefront helpers it uses."""
    h = hashlib.sha256()
    for f in ("tr_score.hip", "tr_score.h", "tr_wave.h"):
        with open(os.path.join(ROOT, "paper_2607_13500_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic():
    """(HBM bytes per score launch or None, its source) from the committed PMC
    summary: the figure is used only while the scoring kernel's sources still
    hash to the ones the counters were taken on."""
    src = {"profile": os.path.relpath(TRAFFIC_PROFILE, ROOT), "sources_sha256": score_source_sha(),
           "what": "FETCH_SIZE + WRITE_SIZE per score_kernel dispatch (two rocprofv3 --pmc runs), "
                   "scaled by the same counters on 512 MiB device copies"}
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        src["status"] = "missing"
        return None, src
    sha = re.search(r"source_sha256:\s*([0-9a-f]{64})", text)
    byt = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not byt:
        src["status"] = "unreadable"
        return None, src
    src["profiled_sha256"] = sha.group(1)
    if sha.group(1) != src["sources_sha256"]:
        src["status"] = "stale: the scoring kernel changed since the counters were taken"
        return None, src
    src["status"] = "current"
    return float(byt.group(1)), src


def describe(w) -> str:
    n = sorted(set(w.N))
    ns = str(n[0]) if len(n) == 1 else "%d..%d" % (n[0], n[-1])
    k = sorted(set(w.K))
    ks = str(k[0]) if len(k) == 1 else ("%.0f %%" % (100 * w.keep_ratio) if w.keep_ratio else "ragged")
    kind = {"llava": "llava-1.5 visual tokens", "llava_fp32": "llava-1.5 vision-encoder tokens",
            "llava_next": "llava-next 5-tile tokens", "qwen_ragged": "dynamic-resolution tokens",
            "video": "video clips (32 frames)"}[w.name]
    dt = "bf16" if str(w.dtype).endswith("bfloat16") else "fp32"
    return "%s, %d x %s tokens x %d %s -> %s kept" % (kind, w.B, ns, w.D, dt, ks)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(w, seconds: float, entropy: int = 2, stride_mode: int = 0, threads: int = 1):
    """The fp64 C oracle, unchanged, on a bounded sample of the workload: the
    first images up to ~40k tokens, repeated to ~`seconds` in three trials.  With threads > 1
    the sample's images are split among that many threads (the oracle runs in
    C outside Python's lock)."""
    import concurrent.futures
    import oracle
    nb, rows = 0, 0
    while nb < w.B and (nb == 0 or rows + w.N[nb] <= 40000):
        rows += w.N[nb]
        nb += 1
    X, P, Q = w.X[:rows].cpu(), w.Xpre[:rows].cpu(), w.Xpost[:rows].cpu()
    # image subsets for the threads: contiguous runs of images, about equal rows
    threads = max(1, min(threads, nb))
    offs = [0]
    for n in w.N[:nb]:
        offs.append(offs[-1] + n)
    cuts = [0]
    for t in range(1, threads):
        target = rows * t / threads
        b = cuts[-1] + 1
        while b < nb and offs[b] < target:
            b += 1
        cuts.append(min(b, nb))
    cuts.append(nb)
    parts = [(cuts[t], cuts[t + 1]) for t in range(threads) if cuts[t] < cuts[t + 1]]

    def run(part):
        b0, b1 = part
        oracle.reduce(X[offs[b0]:offs[b1]], P[offs[b0]:offs[b1]], Q[offs[b0]:offs[b1]], w.N[b0:b1],
                      w.K[b0:b1], w.lam, want_out=True, want_scores=False, entropy=entropy,
                      stride_mode=stride_mode)

    # three timed trials of about seconds / 3 each; the value is their median
    rates, reps, total = [], 0, 0.0
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(parts)) as ex:
        for _ in range(3):
            runs = 0
            t0 = time.perf_counter()
            while True:
                list(ex.map(run, parts))
                runs += 1
                el = time.perf_counter() - t0
                if el >= seconds / 3 or runs >= 500:
                    break
            rates.append(runs * nb / el)
            reps += runs
            total += el
    return {"value": sorted(rates)[1], "unit": "images/s", "cores": len(parts), "kind": "oracle",
            "trials_images_per_s": [round(r, 1) for r in rates],
            "sample": "median of 3 trials, %d repetitions in all of the first %d of %d images (%d tokens; "
                      "fp64 C oracle, %d thread%s, %.1f s; host: %s, %d logical CPUs)"
                      % (reps, nb, w.B, rows, len(parts), "" if len(parts) == 1 else "s", total,
                         cpu_model(), os.cpu_count() or 0)}


def time_steps(torch, f, steps, warmup):
    for _ in range(warmup):
        f()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        f()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def time_events(torch, f, steps, stream):
    for _ in range(3):
        f()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(steps):
        f()
    ev1.record(stream)
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / steps * 1e-3


def needs_scores(tr, w):
    """Which scores the plan needs (the library decides the same way): H2
    unless lambda = 0, s unless lambda = 1."""
    plan = tr.plan(w.N, w.K, w.lam)
    need_x = any(0 < k1 < n for n, k1 in zip(w.N, plan[1]))
    need_s = any(0 < k2 < n - k1 for n, k1, k2 in zip(w.N, plan[1], plan[2]))
    return need_x, need_s


def time_workload(torch, tr, w, steps, warmup, copies=1, stride_real=False, shannon=False):
    """Whole steps of one workload (score -> select -> gather), timed like the
    headline: `warmup` untimed steps, then `steps` steps between two
    synchronizations.  With copies > 1 the steps rotate over that many copies
    of the input and output buffers, so that no step finds its inputs in the
    last-level cache; the per-call latency is then also taken with HIP events
    around single calls."""
    dev = w.X.device
    need_x, need_s = needs_scores(tr, w)
    r = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=w.B, max_tokens=sum(w.N),
                   max_N=max(w.N), stride_real=stride_real, shannon=shannon)
    sk = sum(w.K)
    sets = []
    for c in range(copies):
        X = w.X if c == 0 else w.X.clone()
        P = (w.Xpre if c == 0 else w.Xpre.clone()) if need_s else None
        Q = (w.Xpost if c == 0 else w.Xpost.clone()) if need_s else None
        sets.append((X, P, Q, torch.empty(sk, w.D, dtype=w.dtype, device=dev),
                     torch.empty(sk, dtype=torch.int32, device=dev), torch.empty(sk, dtype=torch.uint8, device=dev)))
    state = [0]

    def step():
        X, P, Q, out, idx, src = sets[state[0] % copies]
        state[0] += 1
        r.reduce(X, P, Q, w.N, w.K, out=out, out_idx=idx, out_src=src)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    res = {"ms_per_step": elapsed / steps * 1e3, "images_per_s": w.B * steps / elapsed,
           "tokens_per_s": sum(w.N) * steps / elapsed,
           "path_bytes": w.algorithmic_bytes(score_x=need_x, score_states=need_s), "r": r,
           "need_x": need_x, "need_s": need_s, "step": step}
    if copies == 1:
        # the gather's yardstick: a plain device copy (torch) of as many
        # contiguous rows as the step keeps, between the same two buffers
        dst, src = sets[0][3], w.X[:sk]
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        reps = 20
        t1 = time.perf_counter()
        for _ in range(reps):
            dst.copy_(src)
        torch.cuda.synchronize()
        cs = (time.perf_counter() - t1) / reps
        nb = 2 * dst.numel() * dst.element_size()
        res["plain_copy"] = {"bytes": nb, "us": round(cs * 1e6, 2), "GBs": round(nb / cs / 1e9, 1),
                             "what": "torch copy_ of the kept rows' byte count (contiguous rows), read + write"}
    if copies > 1:
        # latency of one call: events around each call, buffers rotating
        stream = torch.cuda.current_stream(dev)
        n = max(4 * copies, steps)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        torch.cuda.synchronize()
        for e0, e1 in evs:
            e0.record(stream)
            step()
            e1.record(stream)
        torch.cuda.synchronize()
        us = sorted(1e3 * e0.elapsed_time(e1) for e0, e1 in evs)
        # the same with the queue primed: a fixed spin kernel (torch's
        # cycle-count sleep, ~0.1 ms) before each call keeps the device busy
        # while the host enqueues the first event, the call's launches and the
        # second event, so the events time the device side of the call alone
        for e0, e1 in evs:
            torch.cuda._sleep(200000)
            e0.record(stream)
            step()
            e1.record(stream)
            torch.cuda.synchronize()
        ud = sorted(1e3 * e0.elapsed_time(e1) for e0, e1 in evs)
        res["us_per_call"] = {"median": round(us[len(us) // 2], 2), "p10": round(us[len(us) // 10], 2),
                              "p90": round(us[(9 * len(us)) // 10], 2), "calls": n, "buffer_copies": copies,
                              "how": "HIP events around each call on the library's stream; inputs and outputs "
                                     "rotate over %d copies (%.0f MB, above the 256 MB last-level cache)"
                                     % (copies, copies * sum(t.numel() * t.element_size()
                                                             for t in sets[0][:3] if t is not None) / 1e6),
                              "device": {"median": round(ud[len(ud) // 2], 2), "p10": round(ud[len(ud) // 10], 2),
                                         "p90": round(ud[(9 * len(ud)) // 10], 2),
                                         "how": "the same events with the queue primed by a ~0.1 ms spin "
                                                "kernel before each call: host-side time is not counted"}}
    return res


# Other benchmark workloads of the default run: (key, synth recipe, keyword
# arguments, buffer copies, description of the configuration).
OTHER_WORKLOADS = [
    ("llava_k128", "llava", dict(B=64, N=576, D=4096, K=128), 1, "64 x 576 x 4096 bf16 -> 128 kept"),
    ("llava_k192", "llava", dict(B=64, N=576, D=4096, K=192), 1, "64 x 576 x 4096 bf16 -> 192 kept"),
    ("llava_fp32", "llava_fp32", {}, 64, "1 x 576 x 1024 fp32 -> 64 kept (latency)"),
    # the one module timing the paper reports (Table II): one 576-token image at
    # the encoder width 1024, K = 192 (64 by entropy + 128 by stride)
    ("llava_fp32_k192", "llava_fp32", dict(K=192), 64, "1 x 576 x 1024 fp32 -> 192 kept (latency)"),
    ("llava_next", "llava_next", {}, 1, "16 x 2880 (5 tiles x 576) x 4096 bf16 -> 320 kept"),
    ("qwen_ragged", "qwen_ragged", {}, 1, "32 ragged images, N in [256, 16384], 3584 bf16 -> 11 % kept"),
    ("video", "video", {}, 1, "4 clips x 32 frames x 576 x 4096 bf16 -> 1152 kept"),
]


def other_workloads(torch, synth, tr, dev, steps, warmup, headline_w):
    """The other benchmark configurations, timed like the headline."""
    out = {}
    for key, recipe, kw, copies, what in OTHER_WORKLOADS:
        if recipe == "llava" and headline_w is not None:   # same tokens, another K
            w = synth.Workload(headline_w.name, headline_w.X, headline_w.Xpre, headline_w.Xpost,
                               list(headline_w.N), [kw["K"]] * headline_w.B, headline_w.lam)
        else:
            w = synth.make(recipe, device=dev, **kw)
        t = time_workload(torch, tr, w, steps, warmup, copies=copies)
        ms = t["ms_per_step"]
        e = {"config": what, "images": w.B, "tokens": sum(w.N), "kept": sum(w.K),
             "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
             "images_per_s": round(t["images_per_s"], 1), "tokens_per_s": round(t["tokens_per_s"], 1),
             "ms_per_step": round(ms, 5), "path_bytes": t["path_bytes"],
             "path_frac_of_8TBs": round(t["path_bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        if "us_per_call" in t:
            e["us_per_call"] = t["us_per_call"]
        if "plain_copy" in t:
            e["plain_copy"] = t["plain_copy"]
        out[key] = e
        t["r"].close()
        del t, w
        torch.cuda.empty_cache()
    return out


def bench_gemm(args, torch, tr, dev):
    """The hand-written GEMM core on its own, against the library GEMM."""
    M, N, K = (int(v) for v in args.gemm.split(","))
    g = torch.Generator(device=dev).manual_seed(11)
    A = torch.randn(M, K, device=dev, generator=g).to(torch.bfloat16)
    B = (torch.randn(N, K, device=dev, generator=g) / K ** 0.5).to(torch.bfloat16)
    C = torch.empty(M, N, device=dev, dtype=torch.bfloat16)
    r = tr.Reducer(K, K, torch.bfloat16, max_images=1, max_tokens=1, max_N=1)
    stream = torch.cuda.current_stream(dev)
    t_ours = time_events(torch, lambda: r.gemm(A, B, out=C), args.steps, stream)
    t_lib = time_events(torch, lambda: torch.matmul(A, B.t(), out=C), args.steps, stream)
    flops = 2.0 * M * N * K
    line = {"metric": "TFLOP/s of the bf16 GEMM core, %d x %d x %d" % (M, N, K),
            "value": round(flops / t_ours / 1e12, 1), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(t_ours * 1e3, 5), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "bf16 GEMM C = A . B^T", "M": M, "N": N, "K": K},
            "roofline": {"kernel": "gemm (tr_gemm_bf16)", "bound": "mfma", "achieved": round(flops / t_ours / 1e12, 1),
                         "peak": 2500.0, "unit": "TFLOP/s", "frac": round(flops / t_ours / 1e12 / 2500.0, 4),
                         "traffic": None, "avg_launch_ms": round(t_ours * 1e3, 5)},
            "library_gemm": {"ms": round(t_lib * 1e3, 5), "tflops": round(flops / t_lib / 1e12, 1),
                             "ratio_ours_to_library": round(t_lib / t_ours, 4)}}
    r.close()
    print(json.dumps(line), flush=True)


def bench_fused(args, torch, synth, tr, dev):
    """The two fusions around the path, each against its unfused form."""
    w = synth.llava(device=dev, B=args.images, N=576, D=4096, K=args.K)
    rows = sum(w.N)
    g = torch.Generator(device=dev).manual_seed(7)
    stream = torch.cuda.current_stream(dev)
    line = {"n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic"}
    if args.mlp_fused:
        Dc, Hd = 1024, 4096
        Xpre = torch.randn(rows, Dc, device=dev, generator=g).to(torch.bfloat16)
        H = torch.relu(torch.randn(rows, Hd, device=dev, generator=g) + 0.3).to(torch.bfloat16)
        W2 = (torch.randn(Dc, Hd, device=dev, generator=g) / Hd ** 0.5).to(torch.bfloat16)
        r = tr.Reducer(w.D, Dc, w.dtype, lam=w.lam, max_images=w.B, max_tokens=rows, max_N=576)
        Xpost = torch.empty(rows, Dc, dtype=torch.bfloat16, device=dev)
        sk = sum(w.K)
        out = torch.empty(sk, w.D, dtype=w.dtype, device=dev)
        idx = torch.empty(sk, dtype=torch.int32, device=dev)
        src = torch.empty(sk, dtype=torch.uint8, device=dev)

        def fused():
            _, s = r.mlp_out_cos(H, W2, Xpre, out=Xpost)
            r.reduce_given_s(w.X, s, w.N, w.K, out=out, out_idx=idx, out_src=src)

        def unfused():
            torch.matmul(H, W2.t(), out=Xpost)
            r.reduce(w.X, Xpre, Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src)

        t_f = time_steps(torch, fused, args.steps, args.warmup)
        t_u = time_steps(torch, unfused, args.steps, args.warmup)
        t_gemm = time_events(torch, lambda: r.mlp_out_cos(H, W2, Xpre, out=Xpost), args.steps, stream)
        t_lib = time_events(torch, lambda: torch.matmul(H, W2.t(), out=Xpost), args.steps, stream)
        flops = 2.0 * rows * Dc * Hd
        line.update({
            "metric": "images/s: encoder MLP second layer with Eq. 6 fused + the module "
                      "(64 x 576 tokens, Dc 1024, hidden 4096, X 4096 bf16 -> 64 kept)",
            "value": round(w.B / t_f, 1), "unit": "images/s", "ms_per_step": round(t_f * 1e3, 5),
            "config": {"workload": "llava-1.5 tokens with their CLIP-L last-MLP states, 64 x 576, "
                                   "Dc 1024, hidden 4096, D 4096 bf16 -> 64 kept",
                       "images": w.B, "tokens": rows, "D": w.D, "Dc": Dc, "hidden": Hd},
            "unfused": {"ms_per_step": round(t_u * 1e3, 5), "value": round(w.B / t_u, 1),
                        "what": "library GEMM (torch.matmul) + tr_reduce reading X_pre and X_post"},
            "roofline": {"kernel": "gemm_wide_kernel<cos epilogue> + cos_finish", "bound": "mfma",
                         "achieved": round(flops / t_gemm / 1e12, 1), "avg_launch_ms": round(t_gemm * 1e3, 5),
                         "peak": 2500.0, "unit": "TFLOP/s", "frac": round(flops / t_gemm / 1e12 / 2500.0, 4),
                         "traffic": None, "algorithmic_flops_per_launch": flops,
                         "library_gemm_ms": round(t_lib * 1e3, 5),
                         "library_gemm_tflops": round(flops / t_lib / 1e12, 1)},
        })
        r.close()
    else:
        nout = args.project
        r = tr.Reducer(w.D, w.Dc, w.dtype, lam=w.lam, max_images=w.B, max_tokens=rows, max_N=576)
        W = (torch.randn(nout, w.D, device=dev, generator=g) / w.D ** 0.5).to(torch.bfloat16)
        sk = sum(w.K)
        out = torch.empty(sk, w.D, dtype=w.dtype, device=dev)
        proj = torch.empty(sk, nout, dtype=torch.bfloat16, device=dev)
        idx = torch.empty(sk, dtype=torch.int32, device=dev)
        src = torch.empty(sk, dtype=torch.uint8, device=dev)

        def fused():
            r.reduce_project(w.X, w.Xpre, w.Xpost, w.N, w.K, W, out=proj, out_idx=idx, out_src=src)

        def unfused():
            r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src)
            torch.matmul(out, W.t(), out=proj)

        t_f = time_steps(torch, fused, args.steps, args.warmup)
        t_u = time_steps(torch, unfused, args.steps, args.warmup)
        r.reduce(w.X, w.Xpre, w.Xpost, w.N, w.K, out=out, out_idx=idx, out_src=src)
        torch.cuda.synchronize()
        t_gemm = time_events(torch, lambda: r.gemm(out, W, out=proj), args.steps, stream)
        t_lib = time_events(torch, lambda: torch.matmul(out, W.t(), out=proj), args.steps, stream)
        flops = 2.0 * sk * nout * w.D
        line.update({
            "metric": "images/s: the module with the projection of the kept tokens fused into its "
                      "gather (64 x 576 x 4096 bf16 -> 64 kept, projected to %d)" % nout,
            "value": round(w.B / t_f, 1), "unit": "images/s", "ms_per_step": round(t_f * 1e3, 5),
            "config": {"workload": "llava-1.5 visual tokens, 64 x 576 x 4096 bf16 -> 64 kept -> "
                                   "projected to %d" % nout,
                       "images": w.B, "tokens": rows, "D": w.D, "kept": sk, "Nout": nout},
            "unfused": {"ms_per_step": round(t_u * 1e3, 5), "value": round(w.B / t_u, 1),
                        "what": "tr_reduce (gathered copy) + library GEMM (torch.matmul)"},
            "roofline": {"kernel": "gemm_wide_kernel<row gather>", "bound": "mfma",
                         "achieved": round(flops / t_gemm / 1e12, 1), "avg_launch_ms": round(t_gemm * 1e3, 5),
                         "peak": 2500.0, "unit": "TFLOP/s", "frac": round(flops / t_gemm / 1e12 / 2500.0, 4),
                         "traffic": None, "algorithmic_flops_per_launch": flops,
                         "library_gemm_ms": round(t_lib * 1e3, 5),
                         "library_gemm_tflops": round(flops / t_lib / 1e12, 1)},
        })
        r.close()
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the path has no multi-GPU mode "
              "(images are independent; see the sharding notes). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_2607_13500_amd as tr

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device (an MI355X); none is visible", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.gemm:
        bench_gemm(args, torch, tr, dev)
        return
    if args.mlp_fused or args.project:
        bench_fused(args, torch, synth, tr, dev)
        return
    if args.workload == "llava":
        w = synth.llava(device=dev, B=args.images, N=576, D=4096, K=args.K)
    else:
        w = synth.make(args.workload, device=dev)
    if args.lam is not None:
        w.lam = float(args.lam)
    headline = (args.workload == "llava" and args.images == 64 and args.K == 64
                and w.lam == synth.LAMBDA and not args.stride_real and not args.shannon)
    torch.cuda.synchronize()
    # Timed region: K whole steps (score -> select -> gather), nothing else.
    # The single-image fp32 workload rotates over 64 copies of its 7 MB of
    # buffers (its step is latency-bound and would otherwise run from cache).
    copies = 64 if args.workload == "llava_fp32" else 1
    t = time_workload(torch, tr, w, args.steps, args.warmup, copies=copies, stride_real=args.stride_real,
                      shannon=args.shannon)
    r, need_x, need_s, step = t["r"], t["need_x"], t["need_s"], t["step"]
    states = (w.Xpre, w.Xpost) if need_s else (None, None)
    xs = w.X if need_x else None
    elapsed = t["ms_per_step"] * 1e-3 * args.steps

    # Roofline of the dominant kernel: K launches of the scoring kernel (the
    # same kernel, launch configuration and inputs as inside a step) between
    # two HIP events recorded on the stream the library launches on.
    key_imp = torch.empty(sum(w.N), dtype=torch.float32, device=dev) if need_x else None
    key_s = torch.empty(sum(w.N), dtype=torch.float32, device=dev) if need_s else None
    stream = torch.cuda.current_stream(dev)
    for _ in range(3):
        r.score(xs, *states, out=(key_imp, key_s))
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        r.score(xs, *states, out=(key_imp, key_s))
    ev1.record(stream)
    torch.cuda.synchronize()
    score_ms = ev0.elapsed_time(ev1) / args.steps

    # Streaming-read ceiling: the same three tensors read once by a kernel that
    # does nothing else (16-byte non-temporal loads), timed like the roofline.
    read_bufs = [t for t in (xs, *states) if t is not None]
    read_s = time_events(torch, lambda: tr.read_bandwidth(read_bufs), args.steps, stream)
    read_bytes = sum(t.numel() * t.element_size() for t in read_bufs)

    # Diagnostic: the distribution of single-step times, HIP events around each
    # step (the events add a little to each step).
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(min(args.steps, 100))]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    step_ev = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    pick = lambda q: step_ev[min(len(step_ev) - 1, int(q * len(step_ev)))]

    # Diagnostic: per-stage time with HIP events around each kernel of a step
    # (the events themselves add a few microseconds per stage).
    r.timing(True)
    for _ in range(min(args.steps, 100)):
        step()
    torch.cuda.synchronize()
    stage_ms, calls = r.timing_read()
    r.timing(False)

    # Serving form: one step captured in a HIP graph (tr_reduce allocates and
    # copies nothing, so it captures), replayed K times: the same kernels on
    # the same inputs, one graph launch per step from the host.
    side = torch.cuda.Stream(dev)
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        step()
    stream.wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        step()
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    g_elapsed = time.perf_counter() - t0
    del graph

    ms_step = 1e3 * elapsed / args.steps
    images_s = w.B * args.steps / elapsed
    rows = sum(w.N)
    e = w.X.element_size()
    # read X (if scored), X' and X'' (if s is scored); write one key per score
    score_bytes = rows * (need_x * (w.D * e + 4) + need_s * (2 * w.Dc * e + 4))
    achieved = score_bytes / (score_ms * 1e-3) / 1e9
    path_bytes = w.algorithmic_bytes(score_x=need_x, score_states=need_s)
    traffic, traffic_source = measured_traffic() if headline else (None, None)

    line = {
        "metric": METRIC if headline else "images/s (%s workload%s%s%s)" % (
            args.workload, "" if w.lam == synth.LAMBDA else ", lambda=%g" % w.lam,
            ", real-interval stride" if args.stride_real else "",
            ", Shannon entropy" if args.shannon else ""),
        "value": round(images_s, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "data": "synthetic",
        "config": {"workload": describe(w),
                   "images": w.B, "tokens": rows, "D": w.D, "Dc": w.Dc, "kept": sum(w.K),
                   "lambda": round(w.lam, 6),
                   "stride": "real-interval" if args.stride_real else "algorithm-1",
                   "entropy": "shannon" if args.shannon else "renyi-2",
                   "scores": "+".join(n for n, f in (("H2", need_x), ("s", need_s)) if f)},
        "tokens_per_s": round(rows * args.steps / elapsed, 1),
        "path_hbm": {"algorithmic_bytes": path_bytes,
                     "achieved_GBs": round(path_bytes / (ms_step * 1e-3) / 1e9, 1),
                     "frac": round(path_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "step_ms_events": {"median": round(pick(0.5), 5), "p10": round(pick(0.1), 5),
                           "p90": round(pick(0.9), 5), "steps": len(step_ev)},
        "graph_replay": {"ms_per_step": round(1e3 * g_elapsed / args.steps, 5),
                         "images_per_s": round(w.B * args.steps / g_elapsed, 1)},
        "stage_ms_with_events": {"score": round(stage_ms[0] / max(calls, 1), 5),
                                 "select": round(stage_ms[1] / max(calls, 1), 5),
                                 "gather": round(stage_ms[2] / max(calls, 1), 5)},
        "roofline": {"kernel": "score_kernel", "bound": "hbm", "achieved": round(achieved, 1),
                     "avg_launch_ms": round(score_ms, 5),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes_per_launch": score_bytes,
                     "read_ceiling_GBs": round(read_bytes / read_s / 1e9, 1),
                     "frac_of_read_ceiling": round(achieved / (read_bytes / read_s / 1e9), 4)},
    }
    if traffic_source is not None:
        line["roofline"]["traffic_source"] = traffic_source
    if "us_per_call" in t:
        line["us_per_call"] = t["us_per_call"]
    if "plain_copy" in t:
        line["plain_copy"] = t["plain_copy"]
    r.close()
    if headline and not args.no_workloads:
        line["workloads"] = other_workloads(torch, synth, tr, dev, args.steps, args.warmup, w)
    if not args.no_cpu_baseline:
        ent, sm = (1 if args.shannon else 2), (1 if args.stride_real else 0)
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, ent, sm)
        line["cpu_baseline_all_cores"] = cpu_baseline(w, args.cpu_seconds / 2, ent, sm,
                                                      threads=min(os.cpu_count() or 1, 16))
    print(json.dumps(line), flush=True)
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print("calibration: 3 device copies of %d bytes" % n, file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
