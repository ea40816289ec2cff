#!/usr/bin/env python3
"""Benchmark of the SparOA hot path on one MI355X: the FC/GEMM sparsity sweep.

Workload (one "step"): 24 FC operators y = x w^T, x [m, 4096], w [4096, 4096]
bf16 ~ N(0, 1/4096), m in {1, 8, 64}, activation sparsity rho in
{0, 0.5, 0.8, 0.95}, zeros placed i.i.d. or as 16 x 16 blocks, nonzeros
|N(0, 1)|.  Every operator has its own weight matrix (24 x 32 MiB, more than
the 256 MB Infinity Cache holds), so weights stream from HBM.  Per operator
the step runs the whole path: intensity from the shape (host), sparsity
measurement (GPU), routing, and the routed FC kernel.  Default (--mode eager):
the 24 operators are issued by one native executor call (sparoa_fc_ops_run)
per step.  The weight-streaming FCs measure their own input and take the
route decision themselves, in grouped launches (one per row-tile count);
the implicit-GEMM FCs run a grouped measurement, one GEMM each (device-side
route) and a grouped split-K reduction.  --mode graph replays the same call
captured once in a HIP graph (on this stack a replay leaves the GPU idle for
about 18 us between steps, where back-to-back executor calls leave none);
--mode host reads the counts back and routes on the host, one Python call
per kernel.  Inputs are resident in HBM before timing starts; one pair of
HIP events brackets the timed steps (an event pair per step costs 8-9 us per
step).

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

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("dense-equiv TFLOP/s & HBM GB/s vs activation sparsity; per-model latency @1 GPU")
HBM_PEAK_GBS = 8000.0
M_LIST = (1, 8, 64)
RHO_LIST = (0.0, 0.5, 0.8, 0.95)
PATTERNS = ("iid", "block")
K = N = 4096
INTENSITY_THR = 315.0   # bf16 ridge point of MI355X: 2.5 PFLOP/s / 8 TB/s (datasheet)
SKIP_MARGIN = 0.97      # calibration: a skip path must beat dense by 3 % to count as a win
THRESHOLDS_FILE = os.path.join(ROOT, "calibration", "fc_sweep_thresholds.json")
# model stacks: name -> (layer table builder (stacks module), dtype name)
STACKS = {"resnet50_b1_bf16": ("resnet50", 1, "bf16"),
          "resnet50_b32_bf16": ("resnet50", 32, "bf16"),
          "mobilenet_v2_b32_fp16": ("mobilenet_v2", 32, "f16"),
          "ffn12_2048x768_fp16": ("ffn", None, "f16")}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--cpu-seconds", type=float, default=20.0,
                   help="bound on the oracle CPU-baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--thresholds", default=None,
                   help='JSON {m: [sparsity_thr, intensity_thr]}, or a file holding it (or a '
                        'calibration record with "thresholds_per_m"); default: the committed '
                        'calibration/fc_sweep_thresholds.json')
    p.add_argument("--calibrate", action="store_true",
                   help="calibrate the thresholds from this run's forced-path timings instead "
                        "of reading them")
    p.add_argument("--calibrate-out", default=None, metavar="FILE",
                   help="with --calibrate: write the thresholds and the timings they come from")
    p.add_argument("--no-layers", action="store_true",
                   help="skip the per-layer tables of the model stacks")
    p.add_argument("--stack", default=None, choices=sorted(STACKS),
                   help="only replay one model stack's routed pass as a HIP graph (--steps "
                        "times) and print its layer table: the program rocprofv3 profiles")
    p.add_argument("--stack-summary", default=None, metavar="DIR",
                   help="no GPU: turn the rocprofv3 outputs of the --stack runs under DIR into "
                        "profiles/<stack>_layers.md")
    p.add_argument("--bw-kernels", action="store_true",
                   help="only run the bandwidth-bound kernels on large model tensors (standalone "
                        "measurement, depthwise with fused measurement, pointwise), --steps "
                        "calls each: the program rocprofv3 profiles for --bw-summary")
    p.add_argument("--bw-summary", default=None, metavar="DIR",
                   help="no GPU: turn the rocprofv3 outputs of the --bw-kernels runs under DIR "
                        "into profiles/bandwidth_kernels.md")
    p.add_argument("--cases-out", default=None, help="write the per-case table (JSON) here")
    p.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                   help="only run 5 plain device-to-device copies of MIB MiB and exit (the "
                        "reference kernel that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    p.add_argument("--no-models", action="store_true",
                   help="skip the per-model latency runs (ResNet-50, MobileNetV2, FFN stacks)")
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the forced-path and per-operator timings (needs --thresholds): "
                        "only the step kernels run, e.g. under a profiler")
    p.add_argument("--profile-summary", default=None, metavar="DIR",
                   help="no GPU: turn the rocprofv3 outputs under DIR (prof_bench/, "
                        "pmc_{bench,copy}_{FETCH,WRITE}_SIZE/ and their .log files) into "
                        "profiles/fc_sweep_step_kernels.md and profiles/fc_sweep_traffic.json")
    p.add_argument("--crossover", action="store_true",
                   help="f2 sweep instead of the benchmark: whole-path time of every forced "
                        "path at block sparsity 0 .. 0.99 (step 0.05) for each m and zero "
                        "pattern; prints one JSON line with the skip/dense crossovers")
    p.add_argument("--mode", choices=("graph", "eager", "host"), default="eager",
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
    for f in ("fc_bw.hip", "measure.hip", "gemm.hip"):
        with open(os.path.join(ROOT, "paper_2511_19457_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(digest, family, alg_per_launch):
    """HBM traffic per operator of one kernel family measured by rocprofv3
    counters (profiles/fc_sweep_traffic.json), if taken on the current kernel
    sources and on the same operators and paths (same algorithmic bytes per
    operator)."""
    path = os.path.join(ROOT, "profiles", "fc_sweep_traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != digest:
        return None
    # one entry per routing outcome profiled (calibration may route a
    # borderline class either way from run to run)
    for fam in t.get("families", {}).get(family, []):
        if fam.get("alg_bytes_per_launch") == alg_per_launch:
            return fam.get("bytes_per_launch")
    return None


# ---------------------------------------------------------------------------
# rocprofv3 summaries (host only).  The commands below are run from /tmp on the
# GPU machine with REPO the repository root; THR is the thresholds JSON the
# step runs with (--thresholds), so the profiled step is the timed one.
PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats -d $REPO/gpurun_out/prof_bench -o bench -- "
             "python3 $REPO/bench.py --steps 20 --warmup 3 --no-cpu-baseline --no-sweep "
             "--no-models --thresholds \"$THR\"",
    "pmc_bench": "rocprofv3 --pmc {C} --output-format csv -d $REPO/gpurun_out/pmc_bench_{C} -o pmc "
                 "-- python3 $REPO/bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-sweep "
                 "--no-models --thresholds \"$THR\"",
    "pmc_copy": "rocprofv3 --pmc {C} --output-format csv -d $REPO/gpurun_out/pmc_copy_{C} -o pmc "
                "-- python3 $REPO/bench.py --copy-probe {MIB}",
}


def _bench_line(log_path, key="metric"):
    with open(log_path) as f:
        for line in reversed(f.read().splitlines()):
            if line.startswith("{") and f'"{key}"' in line:
                return json.loads(line)
    raise ValueError(f"no bench JSON line in {log_path}")


def _short(name):
    return name.replace("sparoa::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def profile_summary(d, copy_mib):
    """Writes the two profile summaries from rocprofv3 outputs under d."""
    import csv
    import glob
    import sqlite3
    from collections import defaultdict

    # kernel trace of the timed step
    line = _bench_line(os.path.join(d, "prof_bench.log"))
    thr = json.dumps(line["config"]["thresholds_per_m"])
    db = sorted(glob.glob(os.path.join(d, "prof_bench", "**", "*.db"), recursive=True))[0]
    rows = sqlite3.connect(db).execute("select name, start, end from kernels").fetchall()
    agg = defaultdict(list)
    for name, t0, t1 in rows:
        agg[_short(name)].append((t1 - t0) / 1e3)
    tot = sum(sum(v) for v in agg.values())
    out = [f"# FC sweep step: kernel trace ({line['ms_per_step']} ms/step in this run)", "",
           "Command (from /tmp on the GPU machine, REPO = repository root):", "", "```",
           "THR='" + thr + "'", PROFILE_COMMANDS["trace"], "```", "",
           f"Kernel dispatches: {len(rows)}; total kernel time {tot / 1e3:.2f} ms (all phases "
           "of the run: eager reference, warm-up, timed steps, per-family calls).", "",
           "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{k}` | {len(v)} | {sum(v) / 1e3:.3f} | {sum(v) / len(v):.2f} | "
                   f"{min(v):.2f} | {max(v):.2f} | {100 * sum(v) / tot:.1f} |")
    out += ["", "bench.py's own figures in the same run (HIP events around back-to-back "
            "executor calls per family):", ""]
    for fam, r in [("dominant", line["roofline"])] + list(line.get("roofline_other_families", {}).items()):
        out.append(f"- {fam}: `{r['kernel']}`, {r['operators']} operators in {r['launches']} "
                   f"launches, avg {r['avg_launch_us']} us per launch, {r['achieved']} GB/s "
                   "algorithmic")
    with open(os.path.join(ROOT, "profiles", "fc_sweep_step_kernels.md"), "w") as f:
        f.write("\n".join(out) + "\n")

    # HBM traffic per operator of each family, counters scaled by a plain copy
    def counters(sub):
        with open(os.path.join(d, sub, "pmc_counter_collection.csv")) as f:
            return [(r["Kernel_Name"], float(r["Counter_Value"])) for r in csv.DictReader(f)]

    pline = _bench_line(os.path.join(d, "pmc_bench_FETCH_SIZE.log"))
    fams = {pline["roofline"]["kernel"]: pline["roofline"]}
    fams.update({r["kernel"]: r for r in pline.get("roofline_other_families", {}).values()})
    res = dict(workload="FC sweep step (24 operators)",
               source_digest=pline["roofline"]["source_digest"],   # sources the counters ran on
               scale_reading="a plain device-to-device copy of known size reads FETCH_SIZE and "
                             "WRITE_SIZE; each counter is scaled by known bytes / measured",
               families={}, commands=[])
    out_path = os.path.join(ROOT, "profiles", "fc_sweep_traffic.json")
    try:      # keep the entries of other routing outcomes taken on the same sources
        with open(out_path) as f:
            old = json.load(f)
        if old.get("source_digest") == res["source_digest"]:
            res["families"] = {k: [e for e in v if e.get("thresholds") != thr]
                               for k, v in old.get("families", {}).items()
                               if isinstance(v, list)}
            res["commands"] = old.get("commands", [])
    except (OSError, ValueError):
        pass
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        cp = sorted(v for n, v in counters(f"pmc_copy_{c}") if "copyBuffer" in n)[-5:]
        scale[c] = copy_mib * 1024.0 / (sum(cp) / len(cp))
        res[f"copy_{c.lower()}_kib"] = round(sum(cp) / len(cp), 3)
        res[f"scale_{c.lower()}"] = round(scale[c], 4)
    per = {c: counters(f"pmc_bench_{c}") for c in ("FETCH_SIZE", "WRITE_SIZE")}
    for kernel, r in fams.items():
        mfma = "igemm" in kernel
        name = "dense_mfma" if mfma else "dense_bw"
        kib = {}
        for c, rows_c in per.items():
            if mfma:   # per operator: its GEMM and its share of the grouped measurement
                ops = sum(1 for n, _ in rows_c if "igemm_kernel<" in n)    # and reduction
                tot_c = sum(v for n, v in rows_c if any(k in n for k in (
                    "measure_init", "measure_lanebit", "igemm_kernel<", "split_reduce")))
            else:      # one launch = one grouped self-measuring streaming-FC dispatch
                sel = [v for n, v in rows_c if "fc_bw_measured_group<" in n]
                ops, tot_c = len(sel), sum(sel)
            kib[c] = (tot_c / max(ops, 1), ops)
        res["families"].setdefault(name, []).append(dict(
            thresholds=thr,
            kernel=kernel, operators=r["operators"], alg_bytes_per_launch=r["alg_bytes_per_launch"],
            bytes_per_launch=int(sum(kib[c][0] * 1024 * scale[c] for c in kib)),
            fetch_kib_per_launch=round(kib["FETCH_SIZE"][0], 3),
            write_kib_per_launch=round(kib["WRITE_SIZE"][0], 3),
            launches_counted=kib["FETCH_SIZE"][1]))
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        for cmd in ("THR='" + thr + "' " + PROFILE_COMMANDS["pmc_bench"].format(C=c),
                    PROFILE_COMMANDS["pmc_copy"].format(C=c, MIB=copy_mib)):
            if cmd not in res["commands"]:
                res["commands"].append(cmd)
    with open(out_path, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res["families"], indent=1))


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
        # skip granularity of each kernel family; the mask fits either
        c.block = {fam: abi.sparoa_fc_skip_block(c.desc, fam | 1)
                   for fam in (abi.PATH_DENSE_BW, abi.PATH_DENSE_MFMA)}
        c.counts = torch.zeros(4, dtype=torch.int64, device=dev)
        c.mask = torch.zeros(max(abi.sparoa_mask_words(m, K, br, bc) for br, bc in c.block.values()),
                             dtype=torch.int32, device=dev)
        ws = max(abi.sparoa_fc_workspace_size(c.desc, p) for p in range(4))
        c.ws = torch.zeros(max(16, ws), dtype=torch.uint8, device=dev)
        c.y = torch.empty(m, N, dtype=torch.bfloat16, device=dev)
        c.path_dev = torch.zeros(1, dtype=torch.int32, device=dev)
        cases.append(c)
    torch.cuda.synchronize()
    return cases


def family(c):
    """Kernel family the operator's intensity threshold selects."""
    return abi_mod().PATH_DENSE_BW if c.inten["intensity"] < c.c_thr else abi_mod().PATH_DENSE_MFMA


def abi_mod():
    from paper_2511_19457_amd import abi
    return abi


def run_case(abi, c):
    """One operator through the whole path with the host route (counts read
    back, sparoa_route, fixed-path call); returns the routed path."""
    br, bc = c.block[family(c)]
    counts = abi.sparoa_measure_sparsity_sync(c.x, c.m, K, br, bc, 0, c.counts, c.mask)
    path = abi.sparoa_route(counts, c.inten, 0, c.s_thr, c.c_thr)
    w = c.wp if abi.sparoa_fc_uses_packed(c.desc, path) else c.w
    abi.sparoa_fc(c.desc, path, c.x, w, None, None, abi.ACT_NONE, c.mask if path & 1 else None,
                  c.y, c.ws)
    c.counts_host = counts
    return path


def forced_times(abi, torch, cases, paths, rounds=5):
    """Duration (us) of every case's whole path (sparoa_fc_measured: measure,
    route, execute) with the route forced onto each path by its thresholds
    (intensity threshold 0 or 1e30 picks the family, sparsity threshold 0 or 2
    the skip bit), so a family is charged the measurement it needs (the
    streaming kernel measures inside its one launch; the GEMM family measures
    in a launch of its own).  Cold weights: one call per case in case order
    (each case streams its own 32 MiB of weights, so the 24 cases overflow the
    Infinity Cache), a pair of HIP events around each call, best of `rounds`
    (five: a single slow sample of one case would move a class's threshold).
    Also records each case's block sparsity at each family's granularity."""
    for c in cases:
        c.forced = {}
        c.rho_b = {}
    for p in paths:
        fam = p & 2
        s_thr = 0.0 if p & 1 else 2.0
        c_thr = 1e30 if fam else 0.0
        best = [None] * len(cases)
        for _ in range(rounds):
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in cases]
            # an untimed call first: the first launch of a round runs cold
            # (code and translation caches), which would skew case 0
            c = cases[-1]
            abi.sparoa_fc_measured(c.desc, s_thr, c_thr, abi.ROUTE_BLOCK, c.x, c.w, c.wp, None,
                                   None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws, c.path_dev)
            for c, (e0, e1) in zip(cases, ev):
                e0.record()
                abi.sparoa_fc_measured(c.desc, s_thr, c_thr, abi.ROUTE_BLOCK, c.x, c.w, c.wp,
                                       None, None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws,
                                       c.path_dev)
                e1.record()
            torch.cuda.synchronize()
            for i, (e0, e1) in enumerate(ev):
                t = e0.elapsed_time(e1) * 1e3
                best[i] = t if best[i] is None else min(best[i], t)
        for c, t in zip(cases, best):
            c.forced[p] = t
            assert int(c.path_dev.item()) == p, "forced thresholds must force the path"
            z, _, zb, nb = c.counts.cpu().tolist()
            c.rho_b[fam] = zb / nb


def family_batch_times(abi, torch, cases, reps=10):
    """Per operator class (m) and kernel family: duration (us) of the class's
    operators issued as one executor batch (sparoa_fc_ops_run, captured in a
    HIP graph, as the step issues them) with the family forced on every
    operator (intensity threshold 1e30 or 0, dense paths).  Median of `reps`
    replays between HIP events; weights stay cold across the classes' 8 x 32
    MiB."""
    out = {}
    for m in M_LIST:
        cs = [c for c in cases if c.m == m]
        for fam, c_thr in ((abi.PATH_DENSE_BW, 1e30), (abi.PATH_DENSE_MFMA, 0.0)):
            arr = abi.fc_op_array([
                abi.fc_op(c.desc, c.x, c.w, c.wp, None, None, abi.ACT_NONE, c.counts, c.mask,
                          c.y, c.ws, c.path_dev, (2.0, c_thr, abi.ROUTE_BLOCK)) for c in cs])
            cap = torch.cuda.Stream()
            cap.wait_stream(torch.cuda.current_stream())
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(cap):
                with torch.cuda.graph(g):
                    abi.sparoa_fc_ops_run(arr)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert all(int(c.path_dev.item()) == fam for c in cs), "forced family"
            ts = []
            for _ in range(reps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                g.replay()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            out[(m, fam)] = sorted(ts)[reps // 2]
            del g
    return out


def path_times(abi, torch, cases, rounds=3):
    """Duration (us) of each operator's whole path (sparoa_fc_measured:
    measure, route and FC) with cold weights: one call per case in case
    order between a pair of HIP events, best of `rounds`."""
    best = [None] * len(cases)
    for _ in range(rounds):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in cases]
        c = cases[-1]  # untimed first call, as in forced_times
        abi.sparoa_fc_measured(c.desc, c.s_thr, c.c_thr, abi.ROUTE_BLOCK, c.x, c.w, c.wp, None,
                               None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws, c.path_dev)
        for c, (e0, e1) in zip(cases, ev):
            e0.record()
            abi.sparoa_fc_measured(c.desc, c.s_thr, c.c_thr, abi.ROUTE_BLOCK, c.x, c.w, c.wp,
                                   None, None, abi.ACT_NONE, c.counts, c.mask, c.y, c.ws,
                                   c.path_dev)
            e1.record()
        torch.cuda.synchronize()
        for i, (e0, e1) in enumerate(ev):
            t = e0.elapsed_time(e1) * 1e3
            best[i] = t if best[i] is None else min(best[i], t)
    for c, t in zip(cases, best):
        c.path_us = t


def alg_bytes(c, path, mask_host):
    """Algorithmic HBM bytes of one operator's FC: x, y and the weight rows the
    path must read.  Bandwidth skip path: the rows of input columns that are
    nonzero in some row (mask at block (m, 1)).  MFMA skip path: the 64-row
    channel chunks in which some row of the (single, m <= 64) row tile is
    nonzero (mask at block (1, 8)).  Dense paths: all K rows."""
    rows = K
    if path & 1:
        bits = np.unpackbits(mask_host.view(np.uint8), bitorder="little")
        if path & 2:
            rows = int(bits[:K].sum())
        else:
            per_row = bits[:c.m * (K // 8)].reshape(c.m, K // 8).any(axis=0)
            rows = int(per_row.reshape(K // 64, 8).any(axis=1).sum()) * 64
    return 2 * (c.m * K + c.m * N) + 2 * rows * N


def crossover_sweep(abi, torch, synth, dev, n_w=12):
    """f2: the sparsity at which each family's skip path starts to beat its
    dense path, per operator class.  x [m, 4096] at rho = 0, 0.05, .., 0.95,
    0.99 (i.i.d. or 16 x 16 block zeros), w [4096, 4096] bf16 from a pool of
    n_w matrices used in turn (cold: the pool exceeds the Infinity Cache).
    Each point: the whole path (sparoa_fc_measured) forced onto each of the
    four paths, median of one call per pool matrix."""
    rhos = [round(0.05 * i, 2) for i in range(20)] + [0.99]
    ws_nk, ws_p = [], []
    d0 = abi.fc_desc(1, K, N, abi.BF16)
    for i in range(n_w):
        w = synth.normal((N, K), "bf16", synth.seed_for(6, 900 + i), std=1.0 / 64.0).to(dev)
        wp = torch.empty(abi.sparoa_fc_packed_bytes(d0) // 2, dtype=torch.bfloat16, device=dev)
        abi.sparoa_fc_pack_weights(d0, w, wp)
        ws_nk.append(w)
        ws_p.append(wp)
    out = {}
    for m in M_LIST:
        d = abi.fc_desc(m, K, N, abi.BF16)
        blocks = {fam: abi.sparoa_fc_skip_block(d, fam | 1)
                  for fam in (abi.PATH_DENSE_BW, abi.PATH_DENSE_MFMA)}
        counts = torch.zeros(4, dtype=torch.int64, device=dev)
        mask = torch.zeros(max(abi.sparoa_mask_words(m, K, br, bc) for br, bc in blocks.values()),
                           dtype=torch.int32, device=dev)
        ws = torch.zeros(max(16, max(abi.sparoa_fc_workspace_size(d, p) for p in range(4))),
                         dtype=torch.uint8, device=dev)
        y = torch.empty(m, N, dtype=torch.bfloat16, device=dev)
        path = torch.zeros(1, dtype=torch.int32, device=dev)
        for pat in PATTERNS:
            rows = []
            for j, rho in enumerate(rhos):
                x = synth.sparse_matrix(m, K, rho, pat, "bf16",
                                        synth.seed_for(6, 100 * m + 10 * j + len(pat))).to(dev)
                row = dict(rho=rho)
                for p in (abi.PATH_DENSE_BW, abi.PATH_SKIP_BW, abi.PATH_DENSE_MFMA,
                          abi.PATH_SKIP_MFMA):
                    s_thr, c_thr = (0.0 if p & 1 else 2.0), (1e30 if p & 2 else 0.0)
                    ev = [(torch.cuda.Event(enable_timing=True),
                           torch.cuda.Event(enable_timing=True)) for _ in range(n_w)]
                    for i, (e0, e1) in enumerate(ev):
                        e0.record()
                        abi.sparoa_fc_measured(d, s_thr, c_thr, abi.ROUTE_BLOCK, x, ws_nk[i],
                                               ws_p[i], None, None, abi.ACT_NONE, counts, mask, y,
                                               ws, path)
                        e1.record()
                    torch.cuda.synchronize()
                    ts = sorted(e0.elapsed_time(e1) * 1e3 for e0, e1 in ev)
                    row[abi.PATH_NAMES[p] + "_us"] = round(ts[len(ts) // 2], 2)
                    z, _, zb, nb = counts.cpu().tolist()
                    row["rho_b_" + ("bw" if p & 2 else "mfma")] = round(zb / nb, 4)
                rows.append(row)
            cross = {}
            for fam, tag in ((abi.PATH_DENSE_BW, "bw"), (abi.PATH_DENSE_MFMA, "mfma")):
                dn, sk = abi.PATH_NAMES[fam] + "_us", abi.PATH_NAMES[fam | 1] + "_us"
                c = None           # smallest block sparsity from which skip always wins
                for r in reversed(sorted(rows, key=lambda r: r["rho_b_" + tag])):
                    if r[sk] < r[dn]:
                        c = r["rho_b_" + tag]
                    else:
                        break
                cross[tag] = c
            out[f"m{m}_{pat}"] = dict(crossover_rho_b=cross, points=rows)
            print(f"bench: crossover m={m} {pat}: {cross}", file=sys.stderr, flush=True)
    return out


def model_latencies(abi, torch, synth, reps=10):
    """Per-model latency at one GPU: the whole stack (measure, device-side
    route, execute, glue per layer) captured once in a HIP graph and replayed;
    HIP events around each replay, median over `reps`.  Weights He-normal,
    inputs N(0, 1) (seeded)."""
    from paper_2511_19457_amd import stacks
    from paper_2511_19457_amd.driver import Engine
    out = {}
    specs = [("resnet50_b1_bf16", stacks.resnet50(1), torch.bfloat16),
             ("resnet50_b8_bf16", stacks.resnet50(8), torch.bfloat16),
             ("resnet50_b32_bf16", stacks.resnet50(32), torch.bfloat16),
             ("mobilenet_v2_b32_fp16", stacks.mobilenet_v2(32), torch.float16),
             ("ffn12_2048x768_fp16", stacks.ffn(), torch.float16)]
    for name, layers, dt in specs:
        eng = Engine(layers, dt, "cuda", seed=synth.seed_for(3, 0), sparsity_thr=0.5)
        x = synth.normal(stacks.input_shape(layers), dt, synth.seed_for(3, 1)).cuda()
        eng.forward_routed(x)                       # warm-up, eager
        torch.cuda.synchronize()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(cap):
            with torch.cuda.graph(g):
                eng.forward_routed(x)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        ts.sort()
        flops = sum(2 * eng.st[i]["inten"]["macs"] for i, L in enumerate(layers)
                    if L.kind != "maxpool")
        ms = ts[len(ts) // 2]
        out[name] = dict(ms=round(ms, 3), dense_equiv_tflops=round(flops / (ms * 1e-3) / 1e12, 2),
                         layers=len(layers))
        print(f"bench: model {name}: {ms:.3f} ms", file=sys.stderr, flush=True)
        del g, eng, x
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def load_thresholds(arg):
    """Thresholds per operator class {m: (sparsity_thr, intensity_thr)} from a
    JSON object, or from a file holding one or a calibration record."""
    text = arg
    if not arg.lstrip().startswith("{"):
        with open(arg) as f:
            text = f.read()
    obj = json.loads(text)
    obj = obj.get("thresholds_per_m", obj)
    return {int(k): (float(v[0]), float(v[1])) for k, v in obj.items()}


def calibrate(abi, cases, batch=None):
    """Thresholds per operator class (m): the kernel family whose dense path
    is faster -- over the class's operators issued as one executor batch when
    `batch` (family_batch_times) is given, else summed over the cold
    single-operator forced-path timings -- (intensity threshold: the class's
    own intensity when the MFMA family wins, the bf16 ridge point otherwise),
    and the smallest block sparsity at or above which that family's skip path
    beats its dense path (by more than 3 %) in every case of the class (1.0
    when it never does)."""
    out = {}
    for m in M_LIST:
        cs = [c for c in cases if c.m == m]
        if batch is not None:
            bw, mf = batch[(m, abi.PATH_DENSE_BW)], batch[(m, abi.PATH_DENSE_MFMA)]
        else:
            bw = sum(c.forced[abi.PATH_DENSE_BW] for c in cs)
            mf = sum(c.forced[abi.PATH_DENSE_MFMA] for c in cs)
        fam = abi.PATH_DENSE_MFMA if mf < bw else abi.PATH_DENSE_BW
        c_thr = cs[0].inten["intensity"] if fam == abi.PATH_DENSE_MFMA else INTENSITY_THR
        # the skip path wins a case when it is faster by more than the timing
        # noise (3 %), so that near-ties resolve the same way in every run
        pts = sorted((c.rho_b[fam], c.forced[fam | 1] < SKIP_MARGIN * c.forced[fam]) for c in cs)
        s_thr = 1.0
        for rb, wins in reversed(pts):
            if not wins:
                break
            s_thr = rb
        out[m] = (max(s_thr, 1e-9), c_thr)
    return out


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
        br, bc = c.block[family(c)]
        st = oracle.measure(c.x_cpu, c.m, K, br, bc)
        path = oracle.route(st["zeros"], st["numel"], st["zero_blocks"], st["num_blocks"],
                            c.inten["intensity"], 0, c.s_thr, c.c_thr)
        oracle.fc(c.x_cpu, w_cpu, c.m, K, N,
                  skip_mask=st["mask"] if path & 1 else None, skip_rows=br, skip_cols=bc)
        elapsed += time.perf_counter() - t1
        flops += 2 * c.m * K * N
        done.append(f"m{c.m}/rho{c.rho}/{c.pattern}")
        if elapsed > budget_s:
            break
    return flops, elapsed, done


# ---------------------------------------------------------------------------
# Single 3x3 conv workload, per-layer tables of the model stacks, and the
# oracle's CPU timings beside them.

FP32_PEAK_TFLOPS = 157.3
MFMA16_PEAK_TFLOPS = 2500.0


def _roof_us(flops, nbytes, dtype_bits):
    """Roofline time (us) of an operator: max of its flops at the dtype's
    dense peak and its compulsory bytes at the HBM peak."""
    peak = FP32_PEAK_TFLOPS if dtype_bits == 32 else MFMA16_PEAK_TFLOPS
    return max(flops / (peak * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e6


def _graph_us(torch, fn, reps):
    """Median duration (us) of `fn` captured once in a HIP graph and replayed
    `reps` times, HIP events around every replay."""
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g):
            fn()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    del g
    return sorted(ts)[len(ts) // 2]


def _queued_us(torch, fn, reps, cyc):
    """Median GPU time (us) of the kernels `fn` enqueues: a spin kernel first,
    so the host has enqueued all of them before the GPU reaches the first of
    the two HIP events around them."""
    ts = []
    for _ in range(reps):
        torch.cuda._sleep(cyc)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    return sorted(ts)[len(ts) // 2]


def config1_single_conv(abi, torch, synth, reps=50):
    """The single 3x3 conv workload: x = ReLU(N(0,1)) fp32 [1,56,56,64]
    (NHWC), w ~ N(0, 2/576) [64,3,3,64], bias 0.  Timed: the whole path
    (zero count and bitmap of x, device-side route, routed conv) and its
    parts, each as a HIP graph replayed `reps` times (median).  Launch-latency
    bound at this size: reported in us, with the fp32 roofline for context."""
    dev = torch.device("cuda")
    d = abi.conv_desc(1, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, dtype=abi.F32)
    x = synth.relu_normal((1, 56, 56, 64), "f32", synth.seed_for(1, 0)).to(dev)
    w = synth.he_normal((64, 3, 3, 64), 576, "f32", synth.seed_for(1, 1)).to(dev)
    inten = abi.sparoa_op_intensity_conv(d)
    counts = torch.zeros(4, dtype=torch.int64, device=dev)
    mask = torch.zeros(abi.sparoa_mask_words(56 * 56, 64, 1, 8), dtype=torch.int32, device=dev)
    ws = torch.empty(max(16, max(abi.sparoa_conv2d_workspace_size(d, p) for p in range(4))),
                     dtype=torch.uint8, device=dev)
    y = torch.empty(1, 56, 56, 64, dtype=torch.float32, device=dev)
    path = torch.zeros(1, dtype=torch.int32, device=dev)
    s_thr, c_thr = 0.5, 20.0          # fp32 ridge point: 157.3 TFLOP/s / 8 TB/s

    def measure():
        abi.sparoa_measure_sparsity(x, 56 * 56, 64, 1, 8, 0, counts, mask)

    def whole():
        measure()
        abi.sparoa_conv2d_routed(d, s_thr, c_thr, abi.ROUTE_BLOCK, counts, x, w, None, None,
                                 abi.ACT_NONE, mask, y, ws, path)

    def conv_dense():
        abi.sparoa_conv2d(d, abi.PATH_DENSE_MFMA, x, w, None, None, abi.ACT_NONE, None, y, ws)

    cyc = _sleep_cycles(torch)
    whole_us = _queued_us(torch, whole, reps, cyc)
    meas_us = _queued_us(torch, measure, reps, cyc)
    conv_us = _queued_us(torch, conv_dense, reps, cyc)
    graph_us = _graph_us(torch, whole, reps)
    c = dict(zip(("zeros", "numel", "zero_blocks", "num_blocks"), counts.cpu().tolist()))
    roof = _roof_us(inten["flops"], inten["bytes"], 32)
    return dict(workload="single 3x3 conv, x ReLU(N(0,1)) fp32 [1,56,56,64] NHWC, w N(0,2/576) "
                         "[64,3,3,64], bias 0; measure + device route + conv",
                path=abi.PATH_NAMES[int(path.item())], zeros=c["zeros"], numel=c["numel"],
                macs=inten["macs"], bytes=inten["bytes"], intensity=round(inten["intensity"], 3),
                whole_path_us=round(whole_us, 2), measure_us=round(meas_us, 2),
                conv_dense_us=round(conv_us, 2),
                conv_tflops=round(inten["flops"] / conv_us / 1e6, 2),
                fp32_roofline_us=round(roof, 3), conv_roofline_frac=round(roof / conv_us, 4),
                whole_path_graph_replay_us=round(graph_us, 2),
                timing=f"each piece queued behind a spin kernel, HIP events around it, median of "
                       f"{reps} (warm); whole_path_graph_replay_us: the whole path as one HIP "
                       f"graph, events around each replay (includes the graph launch)")


def _sleep_cycles(torch):
    """A torch.cuda._sleep argument that keeps the GPU busy for about 300 us
    (long enough for the host to enqueue a whole layer behind it)."""
    n = 100000
    for _ in range(12):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.cuda._sleep(n)
        e1.record()
        e1.synchronize()
        us = e0.elapsed_time(e1) * 1e3
        if us >= 300.0:
            return n
        n = int(n * max(2.0, 330.0 / max(us, 1.0)))
    return n


def layer_table(abi, torch, synth, name, layers, dtype, reps=5):
    """Per layer of one model stack: its routed path alone (input measurement
    where not fused in its producer, device route, kernel, output
    measurement where fused), timed after a full routed pass has left every
    activation and counter in place.  Each rep restores the counters the
    layer reads and writes to their values before the layer, then (cold
    mode) overwrites a 512 MiB buffer to evict the Infinity Cache, queues a
    spin kernel so the host has enqueued the whole layer before the GPU
    reaches the first event, and brackets the layer with HIP events.  Median
    of `reps` per mode.  Algorithmic bytes and flops are the layer's Eq. 2
    figures (compulsory traffic of input, weights and output; 2 * MACs)."""
    from paper_2511_19457_amd.driver import Engine
    from paper_2511_19457_amd.stacks import input_shape, output_shape
    eng = Engine(layers, dtype, "cuda", seed=synth.seed_for(3, 0), sparsity_thr=0.5)
    x = synth.normal(input_shape(layers), dtype, synth.seed_for(3, 1)).cuda()
    eng.forward_routed(x)
    torch.cuda.synchronize()
    recs = eng.records_from_device()
    final = eng.ctr.clone()
    tmpl = eng.ctr_template
    base = eng.ctr.data_ptr()
    bits = 32 if dtype == torch.float32 else 16
    esz = bits // 8
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cyc = _sleep_cycles(torch)
    rows = []
    for i, L in enumerate(layers):
        pre = final.clone()
        if L.kind != "maxpool":
            pre[i] = tmpl[i]                       # the layer's own input-measurement counters
        out = eng.tmeas.get(i + 1)
        if out is not None:                        # its fused / standalone output counters
            r = (out["counts"].data_ptr() - base) // (16 * 8)
            pre[r] = tmpl[r]
        times = {}
        for mode in ("warm", "cold"):
            ts = []
            for _ in range(reps):
                eng.ctr.copy_(pre)
                if mode == "cold":
                    scrub.fill_(len(ts) & 255)
                torch.cuda._sleep(cyc)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                eng.run_layer_routed(i)
                e1.record()
                e1.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            times[mode] = sorted(ts)[len(ts) // 2]
        rec = recs[i]
        if L.kind == "maxpool":
            s = L.shape
            n_in = s["n"] * s["h"] * s["w"] * s["c"]
            oshape = output_shape(L)
            n_out = oshape[0] * oshape[1] * oshape[2] * oshape[3]
            flops, nbytes, path, inten = 0, (n_in + n_out) * esz, "glue", 0.0
        else:
            assert int(eng.st[i]["path"].item()) == rec.path, (name, L.name, "path changed")
            flops, nbytes = 2 * rec.macs, rec.bytes
            path, inten = abi.PATH_NAMES[rec.path], rec.intensity
        roof = _roof_us(flops, nbytes, bits)
        bound = "mfma" if flops and inten >= (315.0 if bits == 16 else 20.0) else "hbm"
        t = times["warm"] if bound == "mfma" else times["cold"]
        rows.append(dict(layer=L.name, kind=L.kind, rho_e=round(rec.rho_e, 4),
                         rho_b=round(rec.rho_b, 4), intensity=round(inten, 2), path=path,
                         us_warm=round(times["warm"], 2), us_cold=round(times["cold"], 2),
                         gbps=round(nbytes / t / 1e3, 1), tflops=round(flops / t / 1e6, 2),
                         bound=bound, roofline_frac=round(roof / t, 4)))
    del eng, x, scrub
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    tot_w = sum(r["us_warm"] for r in rows)
    return dict(rows=rows, sum_us_warm=round(tot_w, 1),
                sum_us_cold=round(sum(r["us_cold"] for r in rows), 1),
                timing=("each layer alone after a full routed pass, HIP events after a spin "
                        "kernel; median of %d reps; warm = back to back, cold = after a 512 MiB "
                        "overwrite; roofline_frac and rates use the warm time for layers at or "
                        "above the ridge point (mfma) and the cold time otherwise (hbm)" % reps))


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_timings(torch, synth, budget_s=8.0):
    """The oracle (plain C, double precision) on the host cores, one core and
    all cores: the single 3x3 conv in full, and sampled outputs of
    representative layers of the three stacks (conv2d_at on seeded output
    offsets), scaled to each stack's whole pass by its MAC count.  A baseline
    only (no BLAS, no vectorisation)."""
    import oracle
    from paper_2511_19457_amd import stacks
    all_cores = oracle.set_threads(0)
    out = dict(cpu_model=cpu_model(), nproc=os.cpu_count(), threads_all_cores=all_cores)
    x1 = synth.relu_normal((1, 56, 56, 64), "f32", synth.seed_for(1, 0))
    w1 = synth.he_normal((64, 3, 3, 64), 576, "f32", synth.seed_for(1, 1))
    cfg1 = {}
    for label, nt in (("one_core", 1), ("all_cores", all_cores)):
        oracle.set_threads(nt)
        t0 = time.perf_counter()
        _, _, macs = oracle.conv2d(x1, w1, 1, 64, 56, 56, 64, 3, 3, ph=1, pw=1)
        cfg1[label + "_s"] = round(time.perf_counter() - t0, 3)
    cfg1["macs"] = macs
    out["single_conv"] = cfg1
    specs = [("resnet50_b32_bf16", stacks.resnet50(32), torch.bfloat16,
              ("s2b1.c2", "s3b2.c1", "s4b1.c3")),
             ("mobilenet_v2_b32_fp16", stacks.mobilenet_v2(32), torch.float16,
              ("b2.1.expand", "b2.1.dw", "b4.2.project")),
             ("ffn12_2048x768_fp16", stacks.ffn(), torch.float16, ("ffn1.fc1", "ffn1.fc2"))]
    for name, layers, dt, picks in specs:
        pass_macs = 0
        for L in layers:
            s = L.shape
            if L.kind == "conv":
                ho = (s["h"] + 2 * s["ph"] - s["kh"]) // s["sh"] + 1
                wo = (s["w"] + 2 * s["pw"] - s["kw"]) // s["sw"] + 1
                pass_macs += s["n"] * ho * wo * s["cout"] * (s["cin"] // s["groups"]) * \
                    s["kh"] * s["kw"]
            elif L.kind == "fc":
                pass_macs += s["m"] * s["k"] * s["n"]
        res = dict(pass_macs=pass_macs, sampled_layers=list(picks))
        for label, nt in (("one_core", 1), ("all_cores", all_cores)):
            oracle.set_threads(nt)
            macs_done, secs = 0, 0.0
            for L in layers:
                if L.name not in picks:
                    continue
                s = L.shape
                if L.kind == "conv":    # one image: the MAC rate does not depend on the batch
                    n, cin, h, w, cout, k = 1, s["cin"], s["h"], s["w"], s["cout"], s["kh"]
                    ho = (h + 2 * s["ph"] - k) // s["sh"] + 1
                    wo = (w + 2 * s["pw"] - k) // s["sw"] + 1
                    cin_g = cin // s["groups"]
                    x = synth.relu_normal((n, h, w, cin), dt, 77)
                    wt = synth.he_normal((cout, k, k, cin_g), k * k * cin_g, dt, 78)
                    total, per = n * ho * wo * cout, cin_g * k * k
                    args = (n, cin, h, w, cout, k, k, s["sh"], s["sw"], s["ph"], s["pw"], 1, 1,
                            s["groups"])
                else:
                    x = synth.relu_normal((s["m"], s["k"]), dt, 77)
                    wt = synth.normal((s["n"], 1, 1, s["k"]), dt, 78)
                    total, per = s["m"] * s["n"], s["k"]
                    args = (s["m"], s["k"], 1, 1, s["n"], 1, 1)
                count = max(256, min(total, int(4e7 / per / (8 if nt == 1 else 1))))
                idx = synth.rng(79).integers(0, total, size=count)
                t0 = time.perf_counter()
                oracle.conv2d_at(x, wt, idx, *args)
                secs += time.perf_counter() - t0
                macs_done += count * per
                if secs > budget_s:
                    break
            rate = macs_done / secs
            res[label] = dict(mmac_per_s=round(rate / 1e6, 1),
                              est_pass_s=round(pass_macs / rate, 1),
                              sampled_macs=macs_done, seconds=round(secs, 2))
        out[name] = res
    oracle.set_threads(all_cores)
    return out



# ---------------------------------------------------------------------------
# Model-stack profiles: the program rocprofv3 runs (--stack) and the summary
# of its outputs (--stack-summary).

STACK_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --output-format csv -d $REPO/gpurun_out/stk_trace_{S} "
             "-o trace -- python3 $REPO/bench.py --stack {S} --steps 10",
    "pmc": "rocprofv3 --pmc {C} --output-format csv -d $REPO/gpurun_out/stk_pmc_{S}_{T} -o pmc "
           "-- python3 $REPO/bench.py --stack {S} --steps 3",
    "copy": "rocprofv3 --pmc {C} --output-format csv -d $REPO/gpurun_out/pmc_copy_{C} -o pmc "
            "-- python3 $REPO/bench.py --copy-probe 256",
}
STACK_PMC = {"fetch": "FETCH_SIZE", "write": "WRITE_SIZE",
             "mfma": "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 "
                     "SQ_INSTS_VALU_MFMA_MOPS_F16 GRBM_GUI_ACTIVE"}


def _stack_layers(torch, name):
    from paper_2511_19457_amd import stacks
    fn, n, dt = STACKS[name]
    layers = getattr(stacks, fn)(n) if n is not None else getattr(stacks, fn)()
    return layers, {"bf16": torch.bfloat16, "f16": torch.float16}[dt]


def _graph_nodes(torch, fn):
    """Kernels `fn` enqueues: nodes of a HIP graph it is captured into."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    g = torch.cuda.CUDAGraph(keep_graph=True)
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g):
            fn()
    torch.cuda.synchronize()
    n = ctypes.c_size_t(0)
    rc = hip.hipGraphGetNodes(ctypes.c_void_p(g.raw_cuda_graph()), None, ctypes.byref(n))
    assert rc == 0, f"hipGraphGetNodes: {rc}"
    del g
    return int(n.value)


def stack_profile_run(abi, torch, synth, name, reps):
    """One model stack's routed pass (counter reset, then measure + device
    route + execute per layer) captured once as a HIP graph and replayed
    `reps` times, after counting the kernels of each layer (its routed call
    captured alone).  Prints the layer table the summary needs."""
    from paper_2511_19457_amd.driver import Engine
    from paper_2511_19457_amd.stacks import input_shape
    layers, dt = _stack_layers(torch, name)
    eng = Engine(layers, dt, "cuda", seed=synth.seed_for(3, 0), sparsity_thr=0.5)
    x = synth.normal(input_shape(layers), dt, synth.seed_for(3, 1)).cuda()
    eng.forward_routed(x)
    torch.cuda.synchronize()
    recs = eng.records_from_device()
    counts = [_graph_nodes(torch, lambda i=i: eng.run_layer_routed(i)) for i in range(len(layers))]
    reset = _graph_nodes(torch, eng.reset_counters)
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g):
            eng.forward_routed(x)
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    rows = []
    for L, rec, k in zip(layers, recs, counts):
        if L.kind == "maxpool":      # glue: input + output bytes
            from paper_2511_19457_amd.stacks import output_shape
            sh, o = L.shape, output_shape(L)
            rec.bytes = (sh["n"] * sh["h"] * sh["w"] * sh["c"] + o[0] * o[1] * o[2] * o[3]) * \
                torch.tensor([], dtype=dt).element_size()
        rows.append(dict(layer=L.name, kind=L.kind, kernels=k,
                         path=abi.PATH_NAMES.get(rec.path, "glue") if L.kind != "maxpool" else "glue",
                         macs=rec.macs, bytes=rec.bytes, rho_e=round(rec.rho_e, 4),
                         rho_b=round(rec.rho_b, 4), intensity=round(rec.intensity, 2)))
    print(json.dumps(dict(stack=name, reps=reps, reset_kernels=reset,
                          kernels_per_pass=reset + sum(counts), ms=sorted(ts)[len(ts) // 2],
                          layers=rows)), flush=True)


def _csv_rows(d, pattern):
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(d, "**", pattern), recursive=True))
    if not files:
        raise FileNotFoundError(f"no {pattern} under {d}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def stack_summary(d):
    """profiles/<stack>_layers.md from the --stack runs under d: per layer
    its kernels' average duration per pass (kernel trace of 10 replays), its
    HBM bytes per pass (FETCH_SIZE and WRITE_SIZE, each scaled by what it
    reads for a plain 256 MiB copy), and its MFMA busy fraction
    (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE x 4 SIMDs x 256 CUs)."""
    from collections import defaultdict
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = _csv_rows(os.path.join(d, f"pmc_copy_{c}"), "*counter_collection.csv")
        vals = sorted(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])
        vals = vals[-5:]
        scale[c] = 256 * 1024.0 / (sum(vals) / len(vals))
    for name in STACKS:
        try:
            line = _bench_line(os.path.join(d, f"stk_{name}.log"), key="stack")
        except (OSError, ValueError):
            continue
        per = line["kernels_per_pass"]
        # kernel trace: the last reps passes, dispatch order
        tr = _csv_rows(os.path.join(d, f"stk_trace_{name}"), "*kernel_trace.csv")
        tr.sort(key=lambda r: int(r["Dispatch_Id"]))
        tr = tr[-line["reps"] * per:]
        dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in tr]
        names = [r["Kernel_Name"] for r in tr]
        # counters per dispatch: the last passes of each run
        def pmc(tag):
            rows = _csv_rows(os.path.join(d, f"stk_pmc_{name}_{tag}"), "*counter_collection.csv")
            by = defaultdict(dict)
            for r in rows:
                by[int(r["Dispatch_Id"])][r["Counter_Name"]] = \
                    by[int(r["Dispatch_Id"])].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            ids = sorted(by)
            reps_c = len(ids) // per
            ids = ids[-per * min(reps_c, 3):]
            return [by[i] for i in ids], min(reps_c, 3)
        fetch, nf = pmc("fetch")
        write, nw = pmc("write")
        mf, nm = pmc("mfma")
        out = [f"# {name}: per-layer kernel time, HBM traffic and MFMA use", "",
               f"One routed pass (counter reset, then per layer: input measurement where not "
               f"fused in its producer, device-side route, the layer's kernel with fused output "
               f"measurement where available) captured as a HIP graph; {per} kernels per pass; "
               f"graph replay median {line['ms']:.3f} ms in the traced run (profiler attached).",
               "", "Commands (from /tmp on the GPU machine, REPO = repository root):", "", "```",
               STACK_COMMANDS["trace"].format(S=name)]
        for tag, c in STACK_PMC.items():
            out.append(STACK_COMMANDS["pmc"].format(S=name, T=tag, C=c))
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            out.append(STACK_COMMANDS["copy"].format(C=c))
        out += ["```", "",
                f"Counter scale (plain 256 MiB copy): FETCH_SIZE x {scale['FETCH_SIZE']:.4f}, "
                f"WRITE_SIZE x {scale['WRITE_SIZE']:.4f}.  Algorithmic bytes: the layer's Eq. 2 "
                "compulsory traffic (input, weights, output); a residual read adds to the counted "
                "bytes only (max pool: input + output).  Rates use the traced kernel time; "
                "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES (summed over SIMDs) / (one XCD's "
                "GRBM_GUI_ACTIVE x 1024 SIMDs), over the layer's kernels.", "",
                "| layer | path | kernels | us | alg MB | counted MB | counted/alg | GB/s (counted) "
                "| TFLOP/s | MFMA busy % | roofline % | kernels (avg us) |",
                "|---|---|---|---|---|---|---|---|---|---|---|---|"]
        tot_us = tot_alg = tot_cnt = 0.0
        pos = line["reset_kernels"]
        bits = 32 if name.endswith("fp32") else 16
        for L in line["layers"]:
            k = L["kernels"]
            us = sum(dur[p * per + pos + j] for p in range(line["reps"]) for j in range(k)) / \
                line["reps"]
            def cnt(rows, n_rep, c):
                return sum(rows[p * per + pos + j].get(c, 0.0) for p in range(n_rep)
                           for j in range(k)) / max(n_rep, 1)
            counted = (cnt(fetch, nf, "FETCH_SIZE") * scale["FETCH_SIZE"] +
                       cnt(write, nw, "WRITE_SIZE") * scale["WRITE_SIZE"]) * 1024
            busy = cnt(mf, nm, "SQ_VALU_MFMA_BUSY_CYCLES")
            # GRBM_GUI_ACTIVE arrives summed over the 8 XCDs: one XCD's
            # active cycles is the sum / 8
            gui = sum(max(mf[p * per + pos + j].get("GRBM_GUI_ACTIVE", 0.0), 1.0) / 8
                      for p in range(nm) for j in range(k)) / max(nm, 1)
            kn = defaultdict(list)
            for j in range(k):
                kn[_short(names[pos + j])].append(
                    sum(dur[p * per + pos + j] for p in range(line["reps"])) / line["reps"])
            flops = 2 * L["macs"]
            roof = _roof_us(flops, L["bytes"], bits) if L["kind"] != "maxpool" else \
                L.get("bytes", 0) / (HBM_PEAK_GBS * 1e3)
            frac = roof / us if us else 0.0
            out.append(f"| {L['layer']} | {L['path']} | {k} | {us:.2f} | {L['bytes'] / 1e6:.1f} | "
                       f"{counted / 1e6:.1f} | {counted / max(L['bytes'], 1):.2f} | "
                       f"{counted / us / 1e3:.0f} | {flops / us / 1e6:.1f} | "
                       f"{100 * busy / (gui * 1024):.1f} | {100 * frac:.1f} | " +
                       ", ".join(f"`{kk}` {sum(v) / len(v):.1f}" for kk, v in kn.items()) + " |")
            tot_us += us
            tot_alg += L["bytes"]
            tot_cnt += counted
            pos += k
        out += ["", f"Sum of kernel time per pass: {tot_us:.1f} us; algorithmic {tot_alg / 1e6:.1f} "
                f"MB, counted {tot_cnt / 1e6:.1f} MB."]
        with open(os.path.join(ROOT, "profiles", f"{name}_layers.md"), "w") as f:
            f.write("\n".join(out) + "\n")
        print(f"wrote profiles/{name}_layers.md", file=sys.stderr)

# ---------------------------------------------------------------------------
# Bandwidth-bound kernels on large model tensors: the program rocprofv3 runs
# (--bw-kernels) and the summary of its outputs (--bw-summary).

BW_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --output-format csv -d $REPO/gpurun_out/bw_trace -o trace "
             "-- python3 $REPO/bench.py --bw-kernels --steps 20",
    "pmc": "rocprofv3 --pmc {C} --output-format csv -d $REPO/gpurun_out/bw_pmc_{C} -o pmc -- "
           "python3 $REPO/bench.py --bw-kernels --steps 3",
}


def bw_workloads(abi, torch, synth):
    """(name, kernel-name substrings of one call, algorithmic bytes, callable) of
    each bandwidth-bound workload, on MobileNetV2 / ResNet-50 N = 32 tensors."""
    dev = torch.device("cuda")
    out = []

    def measure(shape, dt):
        x = synth.relu_normal(shape, dt, synth.seed_for(4, len(out))).to(dev)
        rows, cols = x.numel() // shape[-1], shape[-1]
        nb = rows * cols // 8
        preset = torch.tensor([0, rows * cols, nb, nb], dtype=torch.int64, device=dev)
        c = preset.clone()
        m = torch.zeros(abi.sparoa_mask_words(rows, cols, 1, 8), dtype=torch.int32, device=dev)
        cw = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)

        def f():
            abi.sparoa_measure_sparsity_preset(x, rows, cols, 1, 8, c, m, commit=cw)
        name = f"measurement {list(shape)} {dt} at (1, 8), preset counters, commit words"
        out.append((name, ["measure_lanebit"], x.numel() * x.element_size() + m.numel() * 4, f))

    def depthwise(n, c, h, s, dt):
        tdt = torch.float16 if dt == "f16" else torch.bfloat16
        d = abi.conv_desc(n, c, h, h, c, 3, 3, s, s, 1, 1, 1, 1, c, tdt, has_bias=True)
        ho = (h - 1) // s + 1
        seed = synth.seed_for(4, 10 + len(out))
        x = synth.relu_normal((n, h, h, c), dt, seed).to(dev)
        w = synth.he_normal((c, 3, 3, 1), 9, dt, seed + 1).to(dev)
        b = synth.normal((c,), dt, seed + 2).to(dev)
        y = torch.empty(n, ho, ho, c, dtype=tdt, device=dev)
        cnt = torch.zeros(4, dtype=torch.int64, device=dev)
        rows = n * ho * ho
        yc = torch.tensor([0, rows * c, rows * c // 8, rows * c // 8], dtype=torch.int64,
                          device=dev)
        cw = torch.zeros(abi.COMMIT_WORDS_BYTES // 8, dtype=torch.int64, device=dev)
        ws = torch.zeros(16, dtype=torch.uint8, device=dev)

        def f():
            abi.sparoa_conv2d_routed_measured(d, 2.0, 0.0, abi.ROUTE_BLOCK, cnt, x, w, b, None,
                                              abi.ACT_RELU6, None, y, yc, None, ws, None, cw)
        name = (f"depthwise 3x3/{s} [{n},{h},{h},{c}] {dt}, ReLU6, counts-only output "
                "measurement fused")
        out.append((name, ["dw3x3_kernel"], (x.numel() + y.numel() + w.numel() + c) * 2, f))

    def pointwise(n, cin, h, cout, dt, residual):
        tdt = torch.float16 if dt == "f16" else torch.bfloat16
        d = abi.conv_desc(n, cin, h, h, cout, 1, 1, 1, 1, 0, 0, 1, 1, 1, tdt)
        seed = synth.seed_for(4, 20 + len(out))
        x = synth.relu_normal((n, h, h, cin), dt, seed).to(dev)
        w = synth.he_normal((cout, 1, 1, cin), cin, dt, seed + 1).to(dev)
        r = synth.normal((n, h, h, cout), dt, seed + 2).to(dev) if residual else None
        y = torch.empty(n, h, h, cout, dtype=tdt, device=dev)
        ws = torch.zeros(16, dtype=torch.uint8, device=dev)
        assert abi.sparoa_conv2d_tiling(d, abi.PATH_DENSE_BW) == (16, 32)   # the pointwise kernel

        def f():
            abi.sparoa_conv2d(d, abi.PATH_DENSE_BW, x, w, None, r, abi.ACT_RELU, None, y, ws)
        alg = (x.numel() + y.numel() + w.numel() + (r.numel() if residual else 0)) * 2
        name = (f"pointwise 1x1 [{n},{h},{h},{cin}] -> {cout} {dt}"
                + (", residual" if residual else ""))
        out.append((name, ["pointwise_kernel"], alg, f))

    measure((32, 56, 56, 256), "bf16")
    measure((32, 112, 112, 96), "f16")
    depthwise(32, 32, 112, 1, "f16")
    depthwise(32, 96, 112, 2, "f16")
    depthwise(32, 144, 56, 1, "f16")
    pointwise(32, 16, 112, 96, "f16", False)
    pointwise(32, 64, 56, 256, "bf16", True)
    return out


def bw_kernels_run(abi, torch, synth, reps):
    """Each workload: 2 warm-up calls, then `reps` calls; prints the JSON line
    the summary reads (workload order, kernel names, algorithmic bytes)."""
    work = bw_workloads(abi, torch, synth)
    torch.cuda.synchronize()
    rows = []
    for name, kern, alg, f in work:
        for _ in range(2 + reps):
            f()
        torch.cuda.synchronize()
        rows.append(dict(name=name, kernels=kern, alg_bytes=alg, calls=2 + reps))
    print(json.dumps(dict(bw_kernels=rows, reps=reps)), flush=True)


def bw_summary(d):
    """profiles/bandwidth_kernels.md from the --bw-kernels runs under d: per
    workload the kernel's average duration over its timed calls (kernel
    trace) and its HBM bytes per call (FETCH_SIZE and WRITE_SIZE, each scaled
    by what it reads for a plain 256 MiB copy)."""
    from collections import defaultdict
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = _csv_rows(os.path.join(d, f"pmc_copy_{c}"), "*counter_collection.csv")
        vals = sorted(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])
        vals = vals[-5:]
        scale[c] = 256 * 1024.0 / (sum(vals) / len(vals))

    def walk(dispatches, line):
        """Dispatches (dispatch order) of each workload's calls, by kernel name."""
        res, i = [], 0
        for w in line["bw_kernels"]:
            got = []
            while i < len(dispatches) and len(got) < w["calls"]:
                if any(k in dispatches[i][0] for k in w["kernels"]):
                    got.append(dispatches[i])
                i += 1
            res.append(got[2:])   # the timed calls
        return res

    line_t = _bench_line(os.path.join(d, "bw_trace.log"), key="bw_kernels")
    tr = _csv_rows(os.path.join(d, "bw_trace"), "*kernel_trace.csv")
    tr.sort(key=lambda r: int(r["Dispatch_Id"]))
    disp = [(r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
            for r in tr]
    times = walk(disp, line_t)
    cnt = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        line_c = _bench_line(os.path.join(d, f"bw_pmc_{c}.log"), key="bw_kernels")
        rows = _csv_rows(os.path.join(d, f"bw_pmc_{c}"), "*counter_collection.csv")
        by = defaultdict(float)
        names = {}
        for r in rows:
            by[int(r["Dispatch_Id"])] += float(r["Counter_Value"])
            names[int(r["Dispatch_Id"])] = r["Kernel_Name"]
        disp_c = [(names[k], by[k]) for k in sorted(by)]
        cnt[c] = walk(disp_c, line_c)
    out = ["# Bandwidth-bound kernels on large model tensors: kernel time and HBM traffic", "",
           "Each workload runs 2 warm-up calls and then the timed calls back to back on one "
           "stream (warm: the tensors stay in the 256 MB Infinity Cache where they fit).",
           "", "Commands (from /tmp on the GPU machine, REPO = repository root):", "", "```",
           BW_COMMANDS["trace"]]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        out.append(BW_COMMANDS["pmc"].format(C=c))
        out.append(STACK_COMMANDS["copy"].format(C=c))
    out += ["```", "",
            f"Counter scale (plain 256 MiB copy): FETCH_SIZE x {scale['FETCH_SIZE']:.4f}, "
            f"WRITE_SIZE x {scale['WRITE_SIZE']:.4f}.  Algorithmic bytes: input + output (+ "
            "weights, residual, bitmap) once.  Rates use the traced kernel time; the roofline "
            f"fraction is against {HBM_PEAK_GBS / 1000:.0f} TB/s.", "",
            "| workload | kernel | calls | avg us | alg MB | counted MB | GB/s (alg) | "
            "fraction of HBM peak |", "|---|---|---|---|---|---|---|---|"]
    for w, ts, fe, wr in zip(line_t["bw_kernels"], times, cnt["FETCH_SIZE"], cnt["WRITE_SIZE"]):
        if not ts:
            continue
        us = sum(t for _, t in ts) / len(ts)
        kb = {c: (sum(v for _, v in cc) / len(cc) if cc else 0.0)
              for c, cc in (("FETCH_SIZE", fe), ("WRITE_SIZE", wr))}
        counted = sum(kb[c] * 1024 * scale[c] for c in kb)
        gbs = w["alg_bytes"] / us / 1e3
        out.append(f"| {w['name']} | `{_short(ts[0][0])}` | {len(ts)} | {us:.2f} | "
                   f"{w['alg_bytes'] / 1e6:.1f} | {counted / 1e6:.1f} | {gbs:.0f} | "
                   f"{gbs / HBM_PEAK_GBS:.3f} |")
    with open(os.path.join(ROOT, "profiles", "bandwidth_kernels.md"), "w") as f:
        f.write("\n".join(out) + "\n")
    print("wrote profiles/bandwidth_kernels.md", file=sys.stderr)


def main():
    args = parse()
    if args.profile_summary:
        profile_summary(args.profile_summary, args.copy_probe or 256)
        return
    if args.stack_summary:
        stack_summary(args.stack_summary)
        return
    if args.bw_summary:
        bw_summary(args.bw_summary)
        return
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
    if args.stack:
        stack_profile_run(abi, torch, synth, args.stack, args.steps)
        return
    if args.bw_kernels:
        bw_kernels_run(abi, torch, synth, args.steps)
        return
    if args.crossover:
        print(json.dumps(dict(sweep="f2 crossover", workload="x [m,4096] x w [4096,4096] bf16, "
                              "whole path forced per path", data="synthetic",
                              results=crossover_sweep(abi, torch, synth, dev))), flush=True)
        return
    print("bench: building 24 FC operators (packing weights)", file=sys.stderr, flush=True)
    cases = build_cases(abi, torch, synth, dev)

    # Forced-path timings per case (untimed phase, cold weights): the sparsity
    # sweep of the metric, and the data the thresholds are calibrated from.
    paths_swept = (abi.PATH_DENSE_BW, abi.PATH_SKIP_BW, abi.PATH_DENSE_MFMA, abi.PATH_SKIP_MFMA)
    thr_source = args.thresholds
    if thr_source is None and not args.calibrate:
        if os.path.exists(THRESHOLDS_FILE):
            thr_source = THRESHOLDS_FILE
        else:
            print(f"bench: {THRESHOLDS_FILE} missing: calibrating from this run", file=sys.stderr)
    if thr_source is None and args.no_sweep:
        print("bench.py: --no-sweep needs thresholds (--thresholds or the committed file)",
              file=sys.stderr)
        sys.exit(2)
    batch_times = None
    if args.no_sweep:
        for c in cases:
            c.forced, c.rho_b = {}, {}
    else:
        print("bench: forced-path sweep", file=sys.stderr, flush=True)
        forced_times(abi, torch, cases, paths_swept)
        batch_times = family_batch_times(abi, torch, cases)
    calibrated = calibrate(abi, cases, batch_times) if not args.no_sweep else None
    thresholds = calibrated if thr_source is None else load_thresholds(thr_source)
    if args.calibrate_out and calibrated is not None:
        rec = dict(thresholds_per_m={str(k): list(v) for k, v in calibrated.items()},
                   rule="per operator class m: kernel family by the faster dense path of the "
                        "class's operators issued as one executor batch (intensity threshold = "
                        "the class's intensity when the MFMA family wins, else the bf16 ridge "
                        "point 315); sparsity threshold = the smallest block sparsity from "
                        "which the family's skip path beats its dense path by more than 3 % "
                        "in every case of the class (1.0 when it never does)",
                   family_batch_us={f"m={m} {abi.PATH_NAMES[f]}": round(t, 2)
                                    for (m, f), t in batch_times.items()},
                   forced_path_us=[dict(m=c.m, rho=c.rho, pattern=c.pattern,
                                        rho_b_bw=round(c.rho_b[abi.PATH_DENSE_BW], 4),
                                        rho_b_mfma=round(c.rho_b[abi.PATH_DENSE_MFMA], 4),
                                        **{abi.PATH_NAMES[p]: round(c.forced[p], 2)
                                           for p in paths_swept}) for c in cases],
                   source_digest=source_digest(),
                   workload="FC sweep: x [m,4096] bf16, w [4096,4096] bf16, cold weights; whole "
                            "path (sparoa_fc_measured) forced onto each path, best of 5")
        with open(args.calibrate_out, "w") as f:
            json.dump(rec, f, indent=1)
    for c in cases:
        c.s_thr, c.c_thr = thresholds[c.m]
    print(f"bench: warmup {args.warmup} steps, thresholds per m (sparsity, intensity): "
          f"{thresholds}", file=sys.stderr, flush=True)

    # the executor's batch: one sparoa_fc_measured per operator, own thresholds
    def batch(sel):
        return abi.fc_op_array([
            abi.fc_op(c.desc, c.x, c.w, c.wp, None, None, abi.ACT_NONE, c.counts, c.mask, c.y,
                      c.ws, c.path_dev, (c.s_thr, c.c_thr, abi.ROUTE_BLOCK)) for c in sel])
    op_array = batch(cases)

    def executor_step():
        abi.sparoa_fc_ops_run(op_array)

    # reference outputs: the timed steps must reproduce them
    executor_step()
    torch.cuda.synchronize()
    y_ref = [c.y.clone() for c in cases]

    def capture(fn):
        cap = torch.cuda.Stream()                   # default priority
        cap.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(cap):
            with torch.cuda.graph(g):
                fn()
        torch.cuda.synchronize()
        return g

    graph = capture(executor_step) if args.mode == "graph" else None

    def step():
        if args.mode == "graph":
            graph.replay()
        elif args.mode == "eager":
            executor_step()
        else:
            for c in cases:
                run_case(abi, c)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # one pair of HIP events brackets the timed steps on the stream they run on
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for s in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    paths = [int(c.path_dev.item()) for c in cases] if args.mode != "host" else \
        [run_case(abi, c) for c in cases]
    torch.cuda.synchronize()
    masks = []
    for i, c in enumerate(cases):
        c.counts_host = dict(zip(("zeros", "numel", "zero_blocks", "num_blocks"),
                                 c.counts.cpu().tolist()))
        masks.append(c.mask.cpu().numpy())
        # the device decision must be the host rule's on the same counts
        assert paths[i] == abi.sparoa_route(c.counts_host, c.inten, 0, c.s_thr, c.c_thr)
        assert torch.equal(c.y, y_ref[i]), f"operator {i}: step output differs from eager run"
    step_s = (t1 - t0) / args.steps
    print(f"bench: timed {args.steps} steps, {step_s * 1e3:.3f} ms/step", file=sys.stderr,
          flush=True)

    flops_step = sum(2 * c.m * K * N for c in cases)
    value = flops_step / step_s / 1e12
    step_gpu_us = ev0.elapsed_time(ev1) * 1e3 / args.steps
    if args.no_sweep:
        for c in cases:
            c.path_us = None
    else:           # per-operator view: the whole path of one operator, cold weights
        path_times(abi, torch, cases)
    table = []
    for i, c in enumerate(cases):
        ch = c.counts_host
        c.alg = alg_bytes(c, paths[i], masks[i])
        row = dict(m=c.m, rho=c.rho, pattern=c.pattern, rho_e=round(ch["zeros"] / ch["numel"], 4),
                   rho_b=round(ch["zero_blocks"] / ch["num_blocks"], 4),
                   path=abi.PATH_NAMES[paths[i]], alg_bytes=c.alg)
        if c.path_us is not None:
            row.update(us=round(c.path_us, 2), gbps=round(c.alg / c.path_us / 1e3, 1),
                       dense_equiv_tflops=round(2 * c.m * K * N / c.path_us / 1e6, 2))
        for p in paths_swept:   # whole path (measure, route, execute) forced onto p
            if p in c.forced:
                row[abi.PATH_NAMES[p] + "_path_us"] = round(c.forced[p], 2)
        table.append(row)
    tot_bytes = sum(c.alg for c in cases)

    # Roofline of each kernel family's launches: the step's operators of one
    # family issued by back-to-back executor calls on the current stream, one
    # pair of HIP events around all of them (the launches run back to back).
    fam_rows = {}
    for fam in (abi.PATH_DENSE_BW, abi.PATH_DENSE_MFMA):
        sel = [c for c in cases if family(c) == fam]
        if not sel:
            continue
        arr = batch(sel)
        abi.sparoa_fc_ops_run(arr)
        torch.cuda.synchronize()
        reps = max(10, args.steps)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            abi.sparoa_fc_ops_run(arr)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        fam_rows[fam] = (sel, us)
    dominant = max(fam_rows, key=lambda f: fam_rows[f][1])
    digest = source_digest()

    def roofline_of(fam):
        sel, us = fam_rows[fam]
        nb = sum(c.alg for c in sel)
        achieved = nb / (us * 1e-6) / 1e9
        if fam == abi.PATH_DENSE_BW:
            # one grouped launch per 16 operators of one dtype
            keys = {}
            for c in sel:
                keys[c.desc.dtype] = keys.get(c.desc.dtype, 0) + 1
            launches = sum(-(-v // 16) for v in keys.values())
            kernel = ("fc_bw_measured_group (self-measuring weight-streaming FC; the family's "
                      "operators in grouped launches of up to 16)")
        else:
            launches = len(sel)
            kernel = ("igemm_kernel (per operator; the family's measurements and split-K "
                      "reductions run as grouped launches)")
        per_launch = int(nb / launches)
        traffic = load_traffic(digest, abi.PATH_NAMES[fam], per_launch)
        return dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(achieved / HBM_PEAK_GBS, 4), traffic=traffic, kernel=kernel,
                    operators=len(sel), launches=launches, alg_bytes_per_launch=per_launch,
                    avg_launch_us=round(us / launches, 3),
                    timing="this family's operators of the step issued by back-to-back "
                           "executor calls, one pair of HIP events around them all (gaps "
                           "between launches included)",
                    source_digest=digest)

    roofline = roofline_of(dominant)
    others = {abi.PATH_NAMES[f]: roofline_of(f) for f in fam_rows if f != dominant}

    line = dict(
        metric=METRIC, value=round(value, 3), unit="TFLOP/s", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(step_s * 1e3, 4), higher_is_better=True,
        scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
        config=dict(workload="fc_sweep: 24 FC operators, x [m,4096] (m in 1,8,64; sparsity "
                             "0/0.5/0.8/0.95 i.i.d. or 16x16 blocks) x w [4096,4096] bf16, "
                             "one weight matrix per operator; measure+route+execute each",
                    global_batch=sum(M_LIST) * len(RHO_LIST) * len(PATTERNS),
                    thresholds_per_m={str(k): v for k, v in thresholds.items()},
                    thresholds_source=(os.path.relpath(thr_source, ROOT)
                                       if thr_source and os.path.exists(thr_source) else
                                       "command line" if thr_source else "calibrated in this run"),
                    route_mode="block", issue=args.mode),
        hbm_gbps_step=round(tot_bytes / step_s / 1e9, 1),
        step_gpu_us=round(step_gpu_us, 2),
        roofline=roofline,
        roofline_other_families=others,
        family_batch_us=None if batch_times is None else {
            f"m={m} {abi.PATH_NAMES[f]}": round(t, 2) for (m, f), t in batch_times.items()},
        sweep=table,
    )
    if not args.no_models:
        line["models"] = model_latencies(abi, torch, synth)
        print("bench: single 3x3 conv", file=sys.stderr, flush=True)
        line["single_conv"] = config1_single_conv(abi, torch, synth)
    if not args.no_models and not args.no_layers:
        from paper_2511_19457_amd import stacks
        line["layers"] = {}
        for name, layers, dt in (("resnet50_b32_bf16", stacks.resnet50(32), torch.bfloat16),
                                 ("mobilenet_v2_b32_fp16", stacks.mobilenet_v2(32), torch.float16),
                                 ("ffn12_2048x768_fp16", stacks.ffn(), torch.float16)):
            print(f"bench: per-layer table {name}", file=sys.stderr, flush=True)
            line["layers"][name] = layer_table(abi, torch, synth, name, layers, dt)
    if not args.no_cpu_baseline:
        import oracle
        print("bench: oracle CPU baseline", file=sys.stderr, flush=True)
        cores = oracle.set_threads(0)
        flops, elapsed, done = cpu_baseline_timed(cases, args.cpu_seconds)
        oracle.set_threads(1)
        flops1, elapsed1, done1 = cpu_baseline_timed(cases, args.cpu_seconds / 4)
        oracle.set_threads(cores)
        line["cpu_baseline"] = dict(
            value=round(flops / elapsed / 1e12, 6), unit="TFLOP/s", cores=cores, kind="oracle",
            sample=f"first {len(done)} of 24 sweep operators in case order "
                   f"({done[0]} .. {done[-1]}): oracle measure + route + FC in double, "
                   f"{elapsed:.1f} s",
            one_core=dict(value=round(flops1 / elapsed1 / 1e12, 6), unit="TFLOP/s",
                          sample=f"first {len(done1)} sweep operators, {elapsed1:.1f} s"),
            cpu_model=cpu_model(), nproc=os.cpu_count())
        if not args.no_models:
            print("bench: oracle timings of the other workloads", file=sys.stderr, flush=True)
            line["oracle_timings"] = oracle_timings(torch, synth)
    else:
        line["cpu_baseline"] = None
    if args.cases_out:
        with open(args.cases_out, "w") as f:
            json.dump(table, f, indent=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
