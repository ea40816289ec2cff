#!/usr/bin/env python3
"""Benchmark of the SparOA hot path on one MI355X: the FC/GEMM sparsity sweep.

Workload (one "step"): 24 FC operators y = x w^T, x [m, 4096], w [4096, 4096]
bf16 ~ N(0, 1/4096), m in {1, 8, 64}, activation sparsity rho in
{0, 0.5, 0.8, 0.95}, zeros placed i.i.d. or as 16 x 16 blocks, nonzeros
|N(0, 1)|.  Every operator has its own weight matrix (24 x 32 MiB, more than
the 256 MB Infinity Cache holds), so weights stream from HBM.  Per operator
the step runs the whole path: intensity from the shape (host), sparsity
measurement (GPU), routing, and the routed FC kernel.  Default (--mode graph):
the 24 operators are issued by one native executor call (sparoa_fc_ops_run),
captured once in a HIP graph; each FC kernel measures its own input and takes
the route decision itself, so a step is one graph launch of 24 kernels.
--mode eager issues the same executor call every step; --mode host reads the
counts back and routes on the host, one Python call per kernel.  Inputs are
resident in HBM before timing starts.

value = dense-equivalent TFLOP/s of the step: sum over operators of
2 m k n divided by the step time (skipped work counts as done).

Prints one JSON line on stdout.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("dense-equiv TFLOP/s & HBM GB/s vs activation sparsity; per-model latency @1 GPU")
HBM_PEAK_GBS = 8000.0
M_LIST = (1, 8, 64)
RHO_LIST = (0.0, 0.5, 0.8, 0.95)
PATTERNS = ("iid", "block")
K = N = 4096
INTENSITY_THR = 315.0   # bf16 ridge point of MI355X: 2.5 PFLOP/s / 8 TB/s (datasheet)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--cpu-seconds", type=float, default=20.0,
                   help="bound on the oracle CPU-baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--sparsity-thr", type=float, default=None,
                   help="routing threshold; default: calibrated from forced-path timings")
    p.add_argument("--cases-out", default=None, help="write the per-case table (JSON) here")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only run 5 plain device-to-device copies of MIB MiB and exit (the "
                        "reference kernel that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the forced-path and per-operator timings (needs --sparsity-thr): "
                        "only the step kernels run, e.g. under a profiler")
    p.add_argument("--mode", choices=("graph", "eager", "host"), default="graph",
                   help="graph: the executor call captured in a HIP graph, one replay per step; "
                        "eager: the executor call every step; host: counts read back, "
                        "sparoa_route on the host, then the fixed-path call")
    return p.parse_args()


def case_list():
    out = []
    for m in M_LIST:
        for rho in RHO_LIST:
            for pat in PATTERNS:
                out.append((m, rho, pat))
    return out


def source_digest():
    h = hashlib.sha256()
    for f in ("fc_bw.hip", "measure.hip"):
        with open(os.path.join(ROOT, "paper_2511_19457_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(digest):
    """HBM traffic per FC launch measured by rocprofv3 counters, if taken on
    the current kernel source (profiles/fc_bw_kernel_fc_sweep_traffic.json)."""
    path = os.path.join(ROOT, "profiles", "fc_bw_kernel_fc_sweep_traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != digest:
        return None
    return t.get("bytes_per_launch")


class Case:
    pass


def build_cases(abi, torch, synth, dev):
    from concurrent.futures import ThreadPoolExecutor
    specs = list(enumerate(case_list()))

    def draw(spec):     # host-side seeded draws (numpy releases the GIL)
        idx, (m, rho, pat) = spec
        return (synth.sparse_matrix(m, K, rho, pat, "bf16", synth.seed_for(2, idx)),
                synth.normal((N, K), "bf16", synth.seed_for(2, 50 + idx), std=1.0 / 64.0))

    with ThreadPoolExecutor(max_workers=8) as pool:
        drawn = list(pool.map(draw, specs))
    cases = []
    for (idx, (m, rho, pat)), (x_cpu, w_cpu) in zip(specs, drawn):
        c = Case()
        c.idx, c.m, c.rho, c.pattern = idx, m, rho, pat
        c.seed_x = synth.seed_for(2, idx)
        c.seed_w = synth.seed_for(2, 50 + idx)
        c.x_cpu = x_cpu
        c.desc = abi.fc_desc(m, K, N, abi.BF16)
        c.x = c.x_cpu.to(dev)
        w = w_cpu.to(dev)
        del w_cpu
        c.wp = torch.empty(abi.sparoa_fc_packed_bytes(c.desc) // 2, dtype=torch.bfloat16,
                           device=dev)
        abi.sparoa_fc_pack_weights(c.desc, w, c.wp)
        c.w = w                      # [n][k] for the MFMA paths
        c.inten = abi.sparoa_op_intensity_fc(c.desc)
        fam_skip = abi.PATH_SKIP_BW if c.inten["intensity"] < INTENSITY_THR else abi.PATH_SKIP_MFMA
        c.br, c.bc = abi.sparoa_fc_skip_block(c.desc, fam_skip)
        c.counts = torch.zeros(4, dtype=torch.int64, device=dev)
        c.mask = torch.zeros(abi.sparoa_mask_words(m, K, c.br, c.bc), dtype=torch.int32,
                             device=dev)
        ws = max(abi.sparoa_fc_workspace_size(c.desc, p) for p in range(4))
        c.ws = torch.zeros(max(16, ws), dtype=torch.uint8, device=dev)
        c.y = torch.empty(m, N, dtype=torch.bfloat16, device=dev)
        c.path_dev = torch.zeros(1, dtype=torch.int32, device=dev)
        cases.append(c)
    torch.cuda.synchronize()
    return cases


def run_case(abi, c, s_thr, ev=None):
    """One operator through the whole path; returns the routed path."""
    counts = abi.sparoa_measure_sparsity_sync(c.x, c.m, K, c.br, c.bc, 0, c.counts, c.mask)
    path = abi.sparoa_route(counts, c.inten, 0, s_thr, INTENSITY_THR)
    w = c.wp if path & 2 else c.w
    if ev is not None:
        ev[0].record()
    abi.sparoa_fc(c.desc, path, c.x, w, None, None, abi.ACT_NONE, c.mask if path & 1 else None,
                  c.y, c.ws)
    if ev is not None:
        ev[1].record()
    c.counts_host = counts
    return path


def forced_times(abi, torch, c, paths, reps=20, rounds=3):
    """Duration (us) of the FC kernel on each forced path: `reps` back-to-back
    launches between one pair of HIP events, best of `rounds` (the weights
    stay cache-resident here, so these read low next to the cold step)."""
    out = {}
    abi.sparoa_measure_sparsity_sync(c.x, c.m, K, c.br, c.bc, 0, c.counts, c.mask)
    for p in paths:
        w = c.wp if abi.sparoa_fc_uses_packed(c.desc, p) else c.w
        if w is None:
            continue
        best = None
        for _ in range(rounds):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                abi.sparoa_fc(c.desc, p, c.x, w, None, None, abi.ACT_NONE,
                              c.mask if p & 1 else None, c.y, c.ws)
            e1.record()
            e1.synchronize()
            t = e0.elapsed_time(e1) * 1e3 / reps
            best = t if best is None else min(best, t)
        out[p] = best
    return out


def path_time(abi, torch, c, s_thr, reps=20):
    """Duration (us) of one operator's whole path (sparoa_fc_measured:
    measure, route and FC), `reps` calls back to back between one pair of
    HIP events."""
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        abi.sparoa_fc_measured(c.desc, s_thr, INTENSITY_THR, abi.ROUTE_BLOCK, c.x, c.w, c.wp,
                               None, None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws, c.path_dev)
    e1.record()
    e1.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def alg_bytes(c, path, nonzero_cols):
    """Algorithmic HBM bytes of one FC launch: x, y and the weight rows the
    path must read (all of them, or only the nonzero input columns')."""
    rows = nonzero_cols if path & 1 else K
    return 2 * (c.m * K + c.m * N) + 2 * rows * N


def cpu_baseline_timed(cases, budget_s):
    """The oracle (C, double precision, OpenMP) on a bounded sample of the
    same sweep: measure + route + FC per operator, in case order, until the
    time budget is spent (weight generation excluded); returns the
    dense-equivalent flops done and the time taken."""
    import oracle
    import synth
    flops, elapsed, done = 0, 0.0, []
    for c in cases:
        w_cpu = synth.normal((N, K), "bf16", c.seed_w, std=1.0 / 64.0)   # not timed
        t1 = time.perf_counter()
        st = oracle.measure(c.x_cpu, c.m, K, c.m, 1)
        path = oracle.route(st["zeros"], st["numel"], st["zero_blocks"], st["num_blocks"],
                            c.inten["intensity"], 0, 0.5, INTENSITY_THR)
        oracle.fc(c.x_cpu, w_cpu, c.m, K, N,
                  skip_mask=st["mask"] if path & 1 else None, skip_rows=c.m, skip_cols=1)
        elapsed += time.perf_counter() - t1
        flops += 2 * c.m * K * N
        done.append(f"m{c.m}/rho{c.rho}/{c.pattern}")
        if elapsed > budget_s:
            break
    return flops, elapsed, done


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} is not supported "
              "(the hot path shards by batch with no exchange; see the design notes)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps(dict(copy_probe_bytes=n, copies=5)), flush=True)
        return
    import synth
    from paper_2511_19457_amd import abi
    print("bench: building 24 FC operators (packing weights)", file=sys.stderr, flush=True)
    cases = build_cases(abi, torch, synth, dev)

    # Forced-path timings per case (untimed phase): the sparsity sweep of the
    # metric, and the data the routing threshold is calibrated from.
    if args.no_sweep and args.sparsity_thr is None:
        print("bench.py: --no-sweep needs --sparsity-thr", file=sys.stderr)
        sys.exit(2)
    if not args.no_sweep:
        print("bench: forced-path sweep", file=sys.stderr, flush=True)
    for c in cases:
        c.forced = {} if args.no_sweep else forced_times(
            abi, torch, c, (abi.PATH_DENSE_BW, abi.PATH_SKIP_BW, abi.PATH_DENSE_MFMA))
    if args.sparsity_thr is None:
        # smallest block sparsity above which the skip path wins in every case
        pts = []
        for c in cases:     # forced_times left the counts at the skip block in c.counts
            st = c.counts.cpu().tolist()
            pts.append((st[2] / st[3], c.forced[abi.PATH_SKIP_BW] < c.forced[abi.PATH_DENSE_BW]))
        pts.sort()
        s_thr = 1.0
        for rb, wins in reversed(pts):
            if not wins:
                break
            s_thr = rb
        s_thr = max(s_thr, 1e-9)
    else:
        s_thr = args.sparsity_thr

    print(f"bench: warmup {args.warmup} steps, sparsity threshold {s_thr:.4g}", file=sys.stderr,
          flush=True)
    # the executor's batch: one sparoa_fc_measured per operator
    op_array = abi.fc_op_array([
        abi.fc_op(c.desc, c.x, c.w, c.wp, None, None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws,
                  c.path_dev) for c in cases])

    def executor_step():
        abi.sparoa_fc_ops_run(op_array, s_thr, INTENSITY_THR)

    # eager reference outputs: the graph replays must reproduce them
    executor_step()
    torch.cuda.synchronize()
    y_ref = [c.y.clone() for c in cases]
    graph = None
    if args.mode == "graph":
        cap = torch.cuda.Stream()                   # default priority
        cap.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(cap):
            with torch.cuda.graph(graph):
                executor_step()
        torch.cuda.synchronize()

    def step():
        if args.mode == "graph":
            graph.replay()
        elif args.mode == "eager":
            executor_step()
        else:
            for c in cases:
                run_case(abi, c, s_thr)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # one pair of HIP events brackets every step on the stream it runs on
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        ev[s][0].record()
        step()
        ev[s][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    paths = [int(c.path_dev.item()) for c in cases] if args.mode != "host" else \
        [run_case(abi, c, s_thr) for c in cases]
    torch.cuda.synchronize()
    for i, c in enumerate(cases):
        c.counts_host = dict(zip(("zeros", "numel", "zero_blocks", "num_blocks"),
                                 c.counts.cpu().tolist()))
        # the device decision must be the host rule's on the same counts
        assert paths[i] == abi.sparoa_route(c.counts_host, c.inten, 0, s_thr, INTENSITY_THR)
        assert torch.equal(c.y, y_ref[i]), f"operator {i}: step output differs from eager run"
    step_s = (t1 - t0) / args.steps
    print(f"bench: timed {args.steps} steps, {step_s * 1e3:.3f} ms/step", file=sys.stderr,
          flush=True)

    flops_step = sum(2 * c.m * K * N for c in cases)
    value = flops_step / step_s / 1e12
    # GPU time of a step from its events: 24 kernel launches back to back
    step_gpu_us = sum(a.elapsed_time(b) for a, b in ev) * 1e3 / args.steps
    for c in cases:   # per-operator view: the whole path of one operator, back to back
        c.path_us = None if args.no_sweep else path_time(abi, torch, c, s_thr)
    table = []
    tot_bytes = 0
    for i, c in enumerate(cases):
        ch = c.counts_host
        nz_cols = ch["num_blocks"] - ch["zero_blocks"]
        b = alg_bytes(c, paths[i], nz_cols)
        tot_bytes += b
        row = dict(m=c.m, rho=c.rho, pattern=c.pattern, rho_e=round(ch["zeros"] / ch["numel"], 4),
                   rho_b=round(ch["zero_blocks"] / ch["num_blocks"], 4),
                   path=abi.PATH_NAMES[paths[i]], alg_bytes=b)
        if c.path_us is not None:
            row.update(us=round(c.path_us, 2), gbps=round(b / c.path_us / 1e3, 1),
                       dense_equiv_tflops=round(2 * c.m * K * N / c.path_us / 1e6, 2))
        for p, name in ((abi.PATH_DENSE_BW, "dense_bw_us"), (abi.PATH_SKIP_BW, "skip_bw_us"),
                        (abi.PATH_DENSE_MFMA, "dense_mfma_us")):
            if p in c.forced:
                row[name] = round(c.forced[p], 2)
        table.append(row)
    launches = len(cases)
    achieved = tot_bytes / (step_gpu_us * 1e-6) / 1e9
    digest = source_digest()
    traffic = load_traffic(digest)
    roofline = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 4), traffic=traffic,
                    kernel="fc_bw_kernel (self-measuring)",
                    alg_bytes_per_launch=int(tot_bytes / launches),
                    avg_launch_us=round(step_gpu_us / launches, 3),
                    timing="HIP events around every timed step (24 launches, gaps between "
                           "launches included)",
                    source_digest=digest)

    line = dict(
        metric=METRIC, value=round(value, 3), unit="TFLOP/s", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(step_s * 1e3, 4), higher_is_better=True,
        scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload="fc_sweep: 24 FC operators, x [m,4096] (m in 1,8,64; sparsity "
                             "0/0.5/0.8/0.95 i.i.d. or 16x16 blocks) x w [4096,4096] bf16, "
                             "one weight matrix per operator; measure+route+execute each",
                    global_batch=sum(M_LIST) * len(RHO_LIST) * len(PATTERNS),
                    sparsity_thr=s_thr, intensity_thr=INTENSITY_THR, route_mode="block",
                    issue=args.mode),
        hbm_gbps_step=round(tot_bytes / step_s / 1e9, 1),
        step_gpu_us=round(step_gpu_us, 2),
        roofline=roofline,
        sweep=table,
    )
    if not args.no_cpu_baseline:
        print("bench: oracle CPU baseline", file=sys.stderr, flush=True)
        flops, elapsed, done = cpu_baseline_timed(cases, args.cpu_seconds)
        cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        line["cpu_baseline"] = dict(
            value=round(flops / elapsed / 1e12, 6), unit="TFLOP/s", cores=cores, kind="oracle",
            sample=f"first {len(done)} of 24 sweep operators in case order "
                   f"({done[0]} .. {done[-1]}): oracle measure + route + FC in double, "
                   f"{elapsed:.1f} s")
    else:
        line["cpu_baseline"] = None
    if args.cases_out:
        with open(args.cases_out, "w") as f:
            json.dump(table, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
