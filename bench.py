"""Throughput of the mini-batch GNN hot path on one MI355X.

A step is one mini-batch through the whole path: sample_blocks (fan-out
sampling + dedup/relabel into blocks), gather_features (input rows) and
sage_forward (GraphSAGE-mean, 3 layers), in order on one stream.  Like the
paper's sampling workers that overlap mini-batch production with training
(Section III-D), consecutive batches run on --streams streams (default 4),
each with its own sampler state and workspaces.  Default
workload: the 2.4M-node power-law graph (shape of Table I's product graph),
fp32 features of dim 100, model 100-256-256-47, fan-outs 15/10/5, batch 1000,
one epoch over a random 8% training set (196 batches).

--mode train times the whole training iteration instead: the same
sampling and gather, run ahead on loader streams, then forward, softmax
cross-entropy, backward and SGD on one compute stream (the overlap of
sampling with training of Section III-D), with per-stage event times of a
one-stream pass and the oracle's training iteration as CPU baseline.

Prints one JSON line.  value = seeds/s over the timed steps; sampled edges/s
and gather GB/s ride along, and so does the rate of the forward with the
feature pull folded into layer 0 (`fused_forward`); `roofline` covers the
dominant kernel, measured with HIP events on the stream the kernels run on;
`cpu_baseline` times the CPU oracle on a bounded sample of the same batches
(one batch per host thread, up to 16, plus a one-thread figure).

--summarize-profile, --summarize-pmc and --summarize-counters turn the
rocprofv3 output of runs of this script into the tables kept in profiles/.
"""
from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=196)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="products2m")
    ap.add_argument("--cpu-batches", type=int, default=4,
                    help="batches the CPU oracle runs for the baseline (0 = skip)")
    ap.add_argument("--summarize-profile", metavar="PREFIX",
                    help="print a markdown summary of a rocprofv3 CSV run of this script "
                         "(PREFIX_kernel_stats.csv, PREFIX_kernel_trace.csv) and exit; --steps "
                         "and --warmup must match that run")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM traffic of the gather and copy kernels from two rocprofv3 "
                         "--pmc runs of this script (FETCH_SIZE, then WRITE_SIZE; CSV output "
                         "under each directory) as JSON and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                    help="print a markdown table of per-kernel hardware counters from rocprofv3 --pmc "
                         "runs of this script (CSV output under each directory; one counter set per run) "
                         "and exit")
    ap.add_argument("--streams", type=int, default=4,
                    help="mini-batches in flight: batch i runs on stream i %% streams, each stream "
                         "with its own sampler state and workspaces")
    ap.add_argument("--mode", choices=("infer", "train"), default="infer",
                    help="infer: sample + gather + forward (the default); train: the whole "
                         "training iteration, + loss, backward and SGD (bf16 workloads: fp32 master weights)")
    ap.add_argument("--lr", type=float, default=0.01, help="SGD step size of --mode train")
    ap.add_argument("--embed", action="store_true",
                    help="--mode train: the layer-0 inputs are learnable vertex embeddings (a table "
                         "initialised from the features), updated by sparse SGD every iteration")
    ap.add_argument("--fused", action="store_true",
                    help="--mode train: the forward with the feature pull folded into layer 0 "
                         "(only the destination rows gathered)")
    return ap.parse_args()


PASS_A_RUNS = 3   # the headline is the median of this many timed passes


def host_info() -> dict:
    """The host the oracle baseline runs on."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        nodes = len([d for d in os.listdir("/sys/devices/system/node") if d.startswith("node") and d[4:].isdigit()])
    except OSError:
        nodes = None
    return {"nproc": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0)), "cpu_model": model,
            "numa_nodes": nodes}


def gemm_check(torch, dev) -> dict:
    """fp32 matrix throughput of the library GEMM (torch.mm, no TF32) on this
    GPU in the same run: the practical ceiling the linear layers are held to
    next to the published 157.3 TFLOP/s."""
    torch.backends.cuda.matmul.allow_tf32 = False
    n = 8192
    a = torch.randn(n, n, device=dev)
    b = torch.randn(n, n, device=dev)
    c = a @ b
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    reps = 5
    for _ in range(reps):
        torch.mm(a, b, out=c)
    ev[1].record()
    torch.cuda.synchronize()
    tf = reps * 2 * n ** 3 / (ev[0].elapsed_time(ev[1]) / 1e3) / 1e12
    del a, b, c
    return {"torch_fp32_gemm_8192_TFLOPs": tf}


def oracle_threads() -> int:
    """Host threads for the oracle's all-cores figure: the usable CPUs, at
    most 16 (a one-GPU share of the host)."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def alg_sample_bytes(sizes, wide: bool) -> int:
    """Algorithmic bytes of sampling + relabel for one batch: per hop, the
    destination ids, their row-offset pairs, the sampled neighbour ids, the
    block row offsets, the local ids and the source ids."""
    w = 8 if wide else 4
    total = 0
    for n_dst, n_src, nnz in sizes:
        total += 4 * n_dst + 2 * w * n_dst + 4 * nnz + 4 * (n_dst + 1) + 4 * nnz + 4 * n_src
    return total


def quiet_gc() -> None:
    """The timed passes run with Python's cyclic garbage collector off and
    the objects made so far frozen out of its scans: a full collection over
    the generated workload's objects takes tens of milliseconds, and one
    landing inside a single-run timed loop inflated it several times over."""
    gc.collect()
    gc.freeze()
    gc.disable()


def alg_gather_bytes(n_in: int, dim: int, es: int) -> int:
    """Rows read + rows written + ids read."""
    return n_in * (2 * dim * es + 4)


GATHER_SETS = 16


def gather_launch_time(gmb, torch, csr, batches, fanouts, wl, cfg, feats, x_out, K, es, dev):
    """The gather kernel's average launch duration for the roofline: the
    first GATHER_SETS batches of the epoch sampled into workspaces of their
    own (untimed), then K gathers back to back on one stream, cycling over
    them, between one pair of HIP events on that stream.  The average holds
    the gap between consecutive kernels but no event per launch (an event
    pair around every launch, as in the per-stage pass, adds its own
    dispatch latency of several microseconds).  16 batches' rows are about
    2 GB on the 2.4M-node workload, far more than the caches hold.  Returns
    (seconds per launch, algorithmic bytes per launch)."""
    n = min(GATHER_SETS, len(batches))
    nbytes = gmb.sample_workspace_bytes(cfg.batch, fanouts, cfg.num_nodes)
    sets = []
    for b in range(n):
        ws = gmb._aligned_bytes(nbytes, dev)[1]
        blocks = gmb.sample_blocks(csr, batches[b], fanouts, wl.batch_key(b), workspace=ws)
        sets.append((ws, blocks, alg_gather_bytes(blocks.sizes()[0][1], cfg.feat_dim, es)))
    for _, blocks, _ in sets:   # warm-up
        gmb.gather_features(blocks, feats, out=x_out)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(K):
        gmb.gather_features(sets[i % n][1], feats, out=x_out)
    ev[1].record()
    torch.cuda.synchronize()
    csr.check_status()
    total = sum(sets[i % n][2] for i in range(K))
    return ev[0].elapsed_time(ev[1]) / 1e3 / K, total / K


def alg_forward_bytes(sizes, dims, es: int) -> int:
    """Per layer: each source row read once, block CSR, mean rows written
    and read, weight matrices, output rows."""
    total = 0
    for l, (n_dst, n_src, nnz) in enumerate(sizes):
        d, o = dims[l], dims[l + 1]
        total += n_src * d * es + 4 * nnz + 4 * (n_dst + 1) + 2 * n_dst * d * es
        total += 2 * d * o * es + 4 * o + n_dst * o * (4 if l == len(sizes) - 1 else es)
    return total


def linear_flops(sizes, dims) -> int:
    return sum(2 * n_dst * 2 * dims[l] * dims[l + 1] for l, (n_dst, _, _) in enumerate(sizes))


def summarize_profile(args):
    """Markdown summary of `rocprofv3 --kernel-trace --stats --output-format
    csv -- python bench.py ... --cpu-batches 0`: the per-kernel statistics of
    the whole run, the gather kernel over the launches of pass B (isolated,
    one stream, per-stage events) and of pass G (the run's last `steps`
    gathers, back to back on one stream: what `roofline.avg_launch_ms`
    measures), and pass B's kernels step by step."""
    import csv
    pre = args.summarize_profile
    stats = list(csv.DictReader(open(pre + "_kernel_stats.csv")))
    trace = list(csv.DictReader(open(pre + "_kernel_trace.csv")))
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    out = ["| kernel | calls | avg us | min us | max us | share % |", "|---|---:|---:|---:|---:|---:|"]
    for r in stats:
        name = r["Name"].replace("gmb::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                   f"{float(r['Percentage']):.1f} |")
    g = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace if "k_gather" in r["Kernel_Name"]]
    lo = args.warmup + PASS_A_RUNS * args.steps
    hi = lo + args.steps
    sel = g[lo:hi]
    out.append("")
    out.append(f"k_gather launches in the run: {len(g)}; pass B (isolated, launches {lo}..{hi - 1}): "
               f"{len(sel)} launches, average {sum(sel) / max(len(sel), 1) / 1e3:.2f} us, "
               f"min {min(sel) / 1e3:.2f} us, max {max(sel) / 1e3:.2f} us" if sel else "no pass-B launches")
    gt = [r for r in trace if "k_gather" in r["Kernel_Name"]][-args.steps:]
    if len(gt) == args.steps:
        dur = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in gt]
        span = (int(gt[-1]["End_Timestamp"]) - int(gt[0]["Start_Timestamp"])) / len(gt)
        out.append(f"pass G (the last {len(gt)} launches, back to back): kernel average {sum(dur) / len(dur) / 1e3:.2f} us, "
                   f"min {min(dur) / 1e3:.2f} us, max {max(dur) / 1e3:.2f} us; first start to last end "
                   f"{span / 1e3:.2f} us per launch (kernel plus the gap to the next)")
    # pass B step by step: kernels between the seed kernels that start each
    # step, median duration of each position over the complete steps
    gi = [i for i, r in enumerate(trace) if "k_gather" in r["Kernel_Name"]]
    if len(gi) >= hi:
        window = trace[gi[lo - 1] + 1:gi[hi - 1] + 1]
        steps, cur = [], None
        for r in window:
            name = r["Kernel_Name"].replace("gmb::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
            if name.startswith("k_seed_scan"):
                cur = []
                steps.append(cur)
            if cur is not None:
                cur.append((name, int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
        if steps:
            import statistics
            n = statistics.mode(len(st) for st in steps[:-1] or steps)
            full = [st for st in steps if len(st) == n]
            out.append("")
            out.append(f"Pass B, one stream: the kernels of a step in launch order, median over "
                       f"{len(full)} complete steps:")
            out.append("")
            out.append("| # | kernel | median us |")
            out.append("|---:|---|---:|")
            tot = 0.0
            for k in range(n):
                m = statistics.median(st[k][1] for st in full) / 1e3
                tot += m
                out.append(f"| {k} | `{full[0][k][0]}` | {m:.2f} |")
            out.append(f"| | sum | {tot:.1f} |")
    print("\n".join(out))


COPY_BYTES = 1 << 30   # the plain copy that calibrates bandwidth and HBM counters


def traffic_file(workload: str) -> str:
    """Stored counter summary of the gather kernel on one workload."""
    return os.path.join(ROOT, "profiles", f"k_gather_{workload}_traffic.json")

GATHER_SOURCE = os.path.join(ROOT, "paper_2010_05337_amd", "csrc", "gather.hip")


def _source_digest(path: str) -> str:
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _pmc_per_dispatch(d: str, counter: str):
    """{kernel name: [value of `counter` per dispatch]} from the
    counter_collection CSV files rocprofv3 wrote under `d`."""
    import csv
    import glob
    acc = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r.get("Counter_Name") != counter:
                continue
            name = r["Kernel_Name"].replace("gmb::(anonymous namespace)::", "").replace("void ", "")
            per = acc.setdefault(name, {})
            key = int(r.get("Dispatch_Id", len(per)))
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    return {k: [v[i] for i in sorted(v)] for k, v in acc.items()}   # in dispatch order


SIMDS = 256 * 4          # MI355X: 256 CUs of 4 SIMDs
CLOCK_HZ = 2.4e9


def summarize_counters(args):
    """Per kernel, the median over its dispatches of each counter found in
    the rocprofv3 --pmc runs under the given directories, and derived
    figures: MFMA busy share of all SIMD cycles over the dispatch
    (SQ_VALU_MFMA_BUSY_CYCLES summed over the SIMDs), VALU and vector-read
    instructions per wave, the share of wave time spent waiting, and HBM
    read and write megabytes per dispatch: FETCH_SIZE and WRITE_SIZE (KiB)
    each scaled by the factor that makes it read COPY_BYTES on the plain
    copy of the same run (the copy-kernel dispatches within 20% of the
    largest)."""
    import csv
    import glob
    import statistics
    per = {}      # kernel -> counter -> {dispatch: value}
    dur = {}      # kernel -> {dispatch: ns}
    for d in args.summarize_counters:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                name = r["Kernel_Name"].replace("gmb::(anonymous namespace)::", "").replace("void ", "")
                name = name.split("(")[0]
                if name.startswith("Cijk_"):
                    name = "library GEMM (the bench's MFMA check)"
                # one row per launch shape: a kernel that serves several
                # layers runs each with a grid of its own
                name = (name, int(r["Grid_Size"]) // max(1, int(r["Workgroup_Size"])))
                key = (d, r.get("Dispatch_Id", ""))
                c = per.setdefault(name, {}).setdefault(r["Counter_Name"], {})
                c[key] = c.get(key, 0.0) + float(r["Counter_Value"])
                dur.setdefault(name, {})[key] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])

    def med(name, counter):
        v = per[name].get(counter)
        return statistics.median(v.values()) if v else None

    scale = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        v = [x for k in per if "copyBuffer" in k[0] for x in per[k].get(counter, {}).values()]
        # only a copy of the calibration size (a run without one has small
        # copies alone, whose counts say nothing about the scale)
        if v and max(v) * 1024.0 >= COPY_BYTES / 4:
            big = [x for x in v if x >= 0.8 * max(v)]
            scale[counter] = COPY_BYTES / (1024.0 * statistics.mean(big))

    rows = []
    for name in per:
        if name[0].startswith("at::") or "copyBuffer" in name[0] or "fillBuffer" in name[0]:
            continue
        t_ns = statistics.median(dur[name].values())
        waves = med(name, "SQ_WAVES")
        mfma = med(name, "SQ_VALU_MFMA_BUSY_CYCLES")
        row = {"kernel": name[0], "workgroups": name[1],
               "dispatches": max(len(v) for v in per[name].values()),
               "us": t_ns / 1e3 if t_ns else None}
        if mfma is not None and t_ns:
            row["mfma_busy"] = mfma / (SIMDS * t_ns * 1e-9 * CLOCK_HZ)
        for c, k in (("SQ_INSTS_VALU", "valu_per_wave"), ("SQ_INSTS_VMEM_RD", "vmem_rd_per_wave")):
            v = med(name, c)
            if v is not None and waves:
                row[k] = v / waves
        wait, wc = med(name, "SQ_WAIT_ANY"), med(name, "SQ_WAVE_CYCLES")
        if wait is not None and wc:
            row["wait_share"] = wait / wc
        for c, k in (("FETCH_SIZE", "hbm_read_MB"), ("WRITE_SIZE", "hbm_write_MB")):
            v = med(name, c)
            if v is not None and c in scale:
                row[k] = v * 1024.0 * scale[c] / 1e6
        if "hbm_read_MB" in row and "hbm_write_MB" in row and t_ns:
            row["hbm_GBps"] = (row["hbm_read_MB"] + row["hbm_write_MB"]) * 1e6 / t_ns
        v = med(name, "SQ_LDS_BANK_CONFLICT")
        if v is not None:
            row["lds_bank_conflict_cycles"] = v
        rows.append(row)
    rows.sort(key=lambda r: -(r["us"] or 0) * r["dispatches"])
    print(f"counter scale from the {COPY_BYTES / 2**30:.0f} GiB copy: "
          + (", ".join(f"{c} x{f:.3f}" for c, f in scale.items()) or "no such copy in these runs") + "\n")
    cols = ["kernel", "workgroups", "dispatches", "us", "mfma_busy", "valu_per_wave", "vmem_rd_per_wave",
            "wait_share", "hbm_read_MB", "hbm_write_MB", "hbm_GBps", "lds_bank_conflict_cycles"]
    print("| " + " | ".join(cols) + " |")
    print("|" + "---|" * len(cols))
    for r in rows:
        cells = []
        for c in cols:
            v = r.get(c)
            if v is None:
                cells.append("")
            elif c == "kernel":
                cells.append(f"`{v}`")
            elif isinstance(v, float):
                cells.append(f"{v:.3f}" if v < 10 else f"{v:,.0f}")
            else:
                cells.append(str(v))
        print("| " + " | ".join(cells) + " |")


def summarize_pmc(args):
    """HBM bytes per launch of the gather kernel from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), each scaled by the factor that makes the
    same counter read the known size of the plain copy (COPY_BYTES read,
    COPY_BYTES written) in the same run.  The gather's dispatches are the
    run's last `--steps` ones: pass G, the launches `roofline` divides its
    algorithmic bytes over (the earlier passes hold smaller batches too).
    The copy's dispatches are the copy-kernel dispatches within 20% of the
    largest."""
    fetch = _pmc_per_dispatch(args.summarize_pmc[0], "FETCH_SIZE")
    write = _pmc_per_dispatch(args.summarize_pmc[1], "WRITE_SIZE")

    def gather(tab):
        ks = [k for k in tab if "k_gather" in k]
        if len(ks) != 1:
            raise SystemExit(f"expected one gather kernel in the counter files, found {len(ks)}")
        v = tab[ks[0]][-args.steps:]
        if len(v) < args.steps:
            raise SystemExit(f"{len(v)} gather dispatches, fewer than --steps {args.steps}")
        return ks[0].split("(")[0], sum(v) / len(v), len(v)

    def copy(tab):
        v = [x for k in tab if "copyBuffer" in k for x in tab[k]]
        if not v:
            raise SystemExit("no copy-kernel dispatches in the counter files")
        big = [x for x in v if x >= 0.8 * max(v)]
        return sum(big) / len(big), len(big)
    gk, g_fetch, n_gf = gather(fetch)
    _, g_write, n_gw = gather(write)
    c_fetch, n_cf = copy(fetch)
    c_write, n_cw = copy(write)
    f_fetch = COPY_BYTES / (1024.0 * c_fetch)
    f_write = COPY_BYTES / (1024.0 * c_write)
    out = {"kernel": gk, "copy_bytes": COPY_BYTES,
           "fetch_kib_per_launch": g_fetch, "write_kib_per_launch": g_write,
           "gather_dispatches": [n_gf, n_gw], "copy_dispatches": [n_cf, n_cw],
           "copy_fetch_kib": c_fetch, "copy_write_kib": c_write,
           "fetch_scale": f_fetch, "write_scale": f_write,
           "traffic_bytes_per_launch": 1024.0 * (g_fetch * f_fetch + g_write * f_write),
           "gather_source_sha256_16": _source_digest(GATHER_SOURCE)}
    # the benchmark line of the FETCH_SIZE run, if saved next to its CSV
    try:
        with open(os.path.join(args.summarize_pmc[0], "bench.json")) as f:
            line = json.loads(f.read().strip().splitlines()[-1])
        alg = line["roofline"]["alg_bytes_per_launch"]
        out["workload"] = line["config"]["workload"].split(":")[0]
        out["alg_bytes_per_launch"] = alg
        out["traffic_over_alg"] = out["traffic_bytes_per_launch"] / alg
    except (OSError, ValueError, KeyError, IndexError):
        pass
    print(json.dumps(out, indent=1))


def gather_traffic(workload: str):
    """Measured HBM bytes per gather launch and where they come from: the
    stored counter summary of this workload, if it was taken on the current
    gather kernel (digest of its source); otherwise (None, reason)."""
    path = traffic_file(workload)
    try:
        with open(path) as f:
            t = json.load(f)
    except OSError:
        return None, f"no counter run stored for the {workload} workload"
    except ValueError:
        return None, f"unreadable counter summary {os.path.relpath(path, ROOT)}"
    if t.get("workload", "products2m") != workload:
        return None, f"{os.path.relpath(path, ROOT)} was taken on another workload"
    digest = _source_digest(GATHER_SOURCE)
    if t.get("gather_source_sha256_16") != digest:
        return None, "the stored counter summary predates the current gather kernel"
    return t["traffic_bytes_per_launch"], (
        f"not measured in this run: {os.path.relpath(path, ROOT)}, two rocprofv3 --pmc runs "
        f"(FETCH_SIZE, WRITE_SIZE) of the command recorded there, calibrated by a 1 GiB copy; "
        f"gather.hip digest {digest} matches")


def main():
    args = parse()
    if args.summarize_profile:
        summarize_profile(args)
        return
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the path has no multi-GPU sharding; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2010_05337_amd as gmb
    from datagen.configs import CONFIGS, make_workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    cfg = CONFIGS[args.workload]
    t_gen = time.perf_counter()
    wl = make_workload(args.workload)
    t_gen = time.perf_counter() - t_gen
    g = wl.graph
    wide = g.num_edges > 0x7FFFFFFF
    dev = torch.device("cuda:0")
    ip = torch.from_numpy(g.indptr if wide else g.indptr.astype(np.int32)).to(dev)
    ix = torch.from_numpy(g.indices).to(dev)
    csr = gmb.CSRGraph(ip, ix)
    bf16 = cfg.feat_dtype == "bf16"
    es = 2 if bf16 else 4
    if bf16:
        feats = torch.from_numpy(wl.feats.view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        feats = torch.from_numpy(wl.feats).to(dev)

    def mat(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(a).to(dev)
    w = wl.weights
    weights = gmb.SageWeights([mat(a) for a in w.w_self], [mat(a) for a in w.w_neigh],
                              [torch.from_numpy(b).to(dev) for b in w.bias])
    fanouts = list(cfg.fanouts)
    batches = [torch.from_numpy(b).to(dev) for b in wl.batches]
    nb = len(batches)
    if args.mode == "train":
        if bf16 and args.embed:
            print("--embed runs fp32 workloads only (the embeddings are fp32)", file=sys.stderr)
            sys.exit(2)
        run_train(args, wl, csr, ip, ix, feats, weights, batches, t_gen)
        return

    # one set of buffers per stream, sized for a full batch and reused by
    # every step that runs on that stream
    S = max(1, args.streams)
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(S - 1)]
    lanes = []
    for k in range(S):
        c = csr if k == 0 else gmb.CSRGraph(ip, ix)
        ws_s = gmb._aligned_bytes(gmb.sample_workspace_bytes(cfg.batch, fanouts, g.num_nodes), dev)[1]
        probe = gmb.sample_blocks(c, batches[0], fanouts, wl.batch_key(0), workspace=ws_s)
        lanes.append(dict(
            csr=c, ws_sample=ws_s,
            x=torch.empty((probe.input_capacity, cfg.feat_dim), dtype=feats.dtype, device=dev),
            x_dst=torch.empty((gmb.dst_capacity(probe), cfg.feat_dim), dtype=feats.dtype, device=dev),
            ws_fwd=gmb._aligned_bytes(gmb.forward_workspace_bytes(probe, weights), dev)[1],
            logits=torch.empty((cfg.batch, cfg.dims[-1]), dtype=torch.float32, device=dev)))
    torch.cuda.synchronize()
    for ln in lanes:
        ln["csr"].check_status()
    ws_sample, x_buf, ws_fwd = lanes[0]["ws_sample"], lanes[0]["x"], lanes[0]["ws_fwd"]

    def step(i, nstreams, ev=None):
        b = i % nb
        ln = lanes[i % nstreams]
        st = streams[i % nstreams]
        with torch.cuda.stream(st):
            if ev is not None:
                ev[0].record(st)
            blocks = gmb.sample_blocks(ln["csr"], batches[b], fanouts, wl.batch_key(b),
                                       workspace=ln["ws_sample"])
            if ev is not None:
                ev[1].record(st)
            x = gmb.gather_features(blocks, feats, out=ln["x"])
            if ev is not None:
                ev[2].record(st)
            gmb.sage_forward(blocks, x, weights, workspace=ln["ws_fwd"],
                             logits=ln["logits"][:batches[b].numel()])
            if ev is not None:
                ev[3].record(st)
        return blocks

    quiet_gc()
    for i in range(args.warmup):
        step(i, S)
    torch.cuda.synchronize()

    # pass A (the headline): K steps, S streams in flight, no events; the
    # median of PASS_A_RUNS timed passes
    K = args.steps
    runs = []
    for _ in range(PASS_A_RUNS):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            step(i, S)
        T_enq = time.perf_counter() - t0
        torch.cuda.synchronize()
        runs.append(time.perf_counter() - t0)
    T = sorted(runs)[len(runs) // 2]
    for ln in lanes:
        ln["csr"].check_status()

    # pass B (isolated launches): the same K steps on one stream with HIP
    # events around every stage, for per-stage times and the roofline
    stage = {"sample": 0.0, "gather": 0.0, "forward": 0.0}
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(K):
        step(i, 1, evs[i])
    torch.cuda.synchronize()
    T1 = time.perf_counter() - t1
    csr.check_status()
    for e in evs:
        stage["sample"] += e[0].elapsed_time(e[1])
        stage["gather"] += e[1].elapsed_time(e[2])
        stage["forward"] += e[2].elapsed_time(e[3])

    # pass C: sampling + gather only, S streams in flight (a mini-batch
    # loader that runs ahead of the model)
    def step_sg(i, nstreams):
        b = i % nb
        ln = lanes[i % nstreams]
        with torch.cuda.stream(streams[i % nstreams]):
            ln["blocks"] = gmb.sample_blocks(ln["csr"], batches[b], fanouts, wl.batch_key(b),
                                             workspace=ln["ws_sample"])
            gmb.gather_features(ln["blocks"], feats, out=ln["x"])
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for i in range(K):
        step_sg(i, S)
    torch.cuda.synchronize()
    T2 = time.perf_counter() - t2
    for ln in lanes:
        ln["csr"].check_status()

    # pass C split: the same K steps with only the sampling, then with only
    # the gather (each lane gathering the batch it sampled last), S streams
    # in flight; together with pass C they show whether the two stages
    # overlap or compete for the memory system
    def step_s(i, nstreams):
        b = i % nb
        ln = lanes[i % nstreams]
        with torch.cuda.stream(streams[i % nstreams]):
            ln["blocks"] = gmb.sample_blocks(ln["csr"], batches[b], fanouts, wl.batch_key(b),
                                             workspace=ln["ws_sample"])

    def step_g(i, nstreams):
        ln = lanes[i % nstreams]
        with torch.cuda.stream(streams[i % nstreams]):
            gmb.gather_features(ln["blocks"], feats, out=ln["x"])
    split = {}
    for what, fn in (("sample_only", step_s), ("gather_only", step_g)):
        torch.cuda.synchronize()
        t = time.perf_counter()
        for i in range(K):
            fn(i, S)
        torch.cuda.synchronize()
        split[what] = time.perf_counter() - t
    for ln in lanes:
        ln["csr"].check_status()

    # pass D: the fused path (sampling, then the forward that reads layer
    # 0's neighbour rows from the feature table and gathers only the
    # destination rows), S streams in flight, median of PASS_A_RUNS
    def step_fused(i, nstreams):
        b = i % nb
        ln = lanes[i % nstreams]
        with torch.cuda.stream(streams[i % nstreams]):
            blocks = gmb.sample_blocks(ln["csr"], batches[b], fanouts, wl.batch_key(b),
                                       workspace=ln["ws_sample"])
            gmb.sage_forward_fused(blocks, feats, weights, x_dst=ln["x_dst"], workspace=ln["ws_fwd"],
                                   logits=ln["logits"][:batches[b].numel()])
    for i in range(args.warmup):
        step_fused(i, S)
    runs_d = []
    for _ in range(PASS_A_RUNS):
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        for i in range(K):
            step_fused(i, S)
        torch.cuda.synchronize()
        runs_d.append(time.perf_counter() - t3)
    T3 = sorted(runs_d)[len(runs_d) // 2]
    for ln in lanes:
        ln["csr"].check_status()

    copy_GBps = stream_copy(torch, dev)

    # sizes per batch (sampling is a pure function of the batch and its key)
    seeds_total = edges_total = 0
    b_sample = b_gather = b_fwd = flops = 0
    for i in range(K):
        b = i % nb
        blocks = gmb.sample_blocks(csr, batches[b], fanouts, wl.batch_key(b), workspace=ws_sample)
        sizes = blocks.sizes()
        seeds_total += batches[b].numel()
        edges_total += sum(s[2] for s in sizes)
        b_sample += alg_sample_bytes(sizes, wide)
        b_gather += alg_gather_bytes(sizes[0][1], cfg.feat_dim, es)
        b_fwd += alg_forward_bytes(sizes, cfg.dims, es)
        flops += linear_flops(sizes, cfg.dims)

    seeds_per_s = seeds_total / T
    res = {
        "metric": "sampled edges/s + seeds/s (sample+gather+SAGE fwd); gather GB/s vs HBM peak",
        "value": seeds_per_s,
        "unit": "seeds/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * T / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {cfg.num_nodes}-node "
                               f"{'R-MAT' if 'rmat' in cfg.graph else 'ER'} graph, {g.num_edges} edges, "
                               f"feats {cfg.feat_dtype} x{cfg.feat_dim}, SAGE {'-'.join(map(str, cfg.dims))}, "
                               f"fanouts {fanouts}, batch {cfg.batch}, {nb} batches per epoch",
                   "batch": cfg.batch, "fanouts": fanouts, "num_nodes": cfg.num_nodes,
                   "num_edges": g.num_edges, "dims": list(cfg.dims), "batches_per_epoch": nb},
        "sampled_edges_per_s": edges_total / T,
        "pass_a_runs_seeds_per_s": [seeds_total / t for t in runs],
        "streams": S,
        "host_enqueue_ms_per_step": 1e3 * T_enq / K,
        "seeds": seeds_total,
        "sampled_edges": edges_total,
        "datagen_s": t_gen,
    }
    ts, tg, tf = stage["sample"] / 1e3, stage["gather"] / 1e3, stage["forward"] / 1e3
    res["single_stream"] = {"seeds_per_s": seeds_total / T1, "ms_per_step": 1e3 * T1 / K,
                            "stage_ms_per_step": {k: v / K for k, v in stage.items()}}
    res["gather_GBps"] = b_gather / tg / 1e9
    res["sampling_edges_per_s"] = edges_total / ts
    # isolated: stage times of pass B; pipelined: pass C wall time
    res["sample_gather_hbm"] = {"alg_bytes": b_sample + b_gather,
                                "GBps": (b_sample + b_gather) / (ts + tg) / 1e9,
                                "frac_of_peak": (b_sample + b_gather) / (ts + tg) / 1e9 / HBM_PEAK_GBPS,
                                "pipelined_GBps": (b_sample + b_gather) / T2 / 1e9,
                                "pipelined_frac_of_peak": (b_sample + b_gather) / T2 / 1e9 / HBM_PEAK_GBPS,
                                "pipelined_streams": S,
                                "pipelined_us_per_batch": 1e6 * T2 / K,
                                "pipelined_sample_only_us_per_batch": 1e6 * split["sample_only"] / K,
                                "pipelined_gather_only_us_per_batch": 1e6 * split["gather_only"] / K}
    res["stream_copy_GBps"] = copy_GBps
    peak = BF16_MFMA_PEAK_TFLOPS if bf16 else FP32_MFMA_PEAK_TFLOPS
    res["forward"] = {"alg_bytes": b_fwd, "linear_flops": flops,
                      "linear_TFLOPs_lower_bound": flops / tf / 1e12, "mfma_peak_TFLOPs": peak,
                      "linear_arithmetic": ("bf16 operands, v_mfma_f32_16x16x32_bf16, fp32 accumulation" if bf16 else
                                            "fp32 operands cut exactly into three bf16 parts, six part products "
                                            "per fp32 product on v_mfma_f32_16x16x32_bf16, fp32 accumulation "
                                            "(K = 2 d_in <= 512; wider layers on many rows: v_mfma_f32_16x16x4_f32)")}
    res["gemm_check"] = gemm_check(torch, dev)
    res["fused_forward"] = {"seeds_per_s": seeds_total / T3, "ms_per_step": 1e3 * T3 / K,
                            "runs_seeds_per_s": [seeds_total / t for t in runs_d], "streams": S,
                            "what": "sample_blocks + sage_forward_fused (layer-0 mean from the feature "
                                    "table, only block 0's destination rows gathered)"}
    # dominant kernel of the path: the feature gather, K launches back to
    # back on one stream (pass G, after the size pass)
    t_launch, b_launch = gather_launch_time(gmb, torch, csr, batches, fanouts, wl, cfg, feats, x_buf, K, es, dev)
    traffic, traffic_source = gather_traffic(args.workload)
    res["roofline"] = {"kernel": "k_gather", "bound": "hbm",
                       "achieved": b_launch / t_launch / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                       "frac": b_launch / t_launch / 1e9 / HBM_PEAK_GBPS, "traffic": traffic,
                       "traffic_source": traffic_source,
                       "alg_bytes_per_launch": b_launch, "avg_launch_ms": 1e3 * t_launch,
                       "launches": f"the last {K} k_gather launches (pass G: {min(GATHER_SETS, nb)} batches "
                                   "cycled, back to back on one stream)",
                       "pass_b_event_bracket_ms": 1e3 * tg / K}

    if args.cpu_batches > 0:
        res["cpu_baseline"], res["parity"] = cpu_baseline(args, wl, csr, batches, fanouts, feats,
                                                          weights, ws_sample, x_buf, ws_fwd)
    print(json.dumps(res), flush=True)


def backward_flops(sizes, dims) -> int:
    """The products of the backward: per layer [H | M]^T dZ, and for layers
    >= 1 also dZ [W_self; W_neigh]^T."""
    total = 0
    for l, (n_dst, _, _) in enumerate(sizes):
        total += 2 * n_dst * 2 * dims[l] * dims[l + 1]
        if l > 0:
            total += 2 * n_dst * 2 * dims[l] * dims[l + 1]
    return total


def stream_copy(torch, dev):
    """GB/s of a plain device copy of COPY_BYTES (read + write): the
    bandwidth a streaming kernel reaches on this GPU, and, under a
    counter run, the calibration of the HBM byte counters."""
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    ce = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ce[0].record()
    for _ in range(5):
        dst.copy_(src)
    ce[1].record()
    torch.cuda.synchronize()
    return 5 * 2 * COPY_BYTES / (ce[0].elapsed_time(ce[1]) / 1e3) / 1e9


def run_train(args, wl, csr, ip, ix, feats, weights, batches, t_gen):
    """Training iterations: sample + gather of batch i on loader stream
    i % S (its own sampler state and buffers), then forward, loss, backward
    and SGD on one compute stream (each step needs the weights the previous
    one left).  Events order the two: the compute stream waits for the
    batch's gather, a loader stream waits until the compute stream is done
    with the buffers it is about to reuse."""
    import torch
    import paper_2010_05337_amd as gmb
    from datagen import labels as vertex_labels
    cfg, g = wl.cfg, wl.graph
    dev = feats.device
    fanouts = list(cfg.fanouts)
    nb = len(batches)
    C = cfg.dims[-1]
    lab_all = vertex_labels(g.num_nodes, C, cfg.seeds[2] + 1)
    labels = [torch.from_numpy(lab_all[b]).to(dev) for b in wl.batches]
    if args.embed:
        # the table the layer-0 inputs come from, trained in place (loaders
        # gather from it while the compute stream updates it: Hogwild)
        feats = feats.clone()
    S = max(1, args.streams)
    comp = torch.cuda.current_stream()
    lanes = []
    for k in range(S):
        c = csr if k == 0 else gmb.CSRGraph(ip, ix)
        ws_s = gmb._aligned_bytes(gmb.sample_workspace_bytes(cfg.batch, fanouts, g.num_nodes), dev)[1]
        probe = gmb.sample_blocks(c, batches[0], fanouts, wl.batch_key(0), workspace=ws_s)
        rows = gmb.dst_capacity(probe) if args.fused else probe.input_capacity
        lanes.append(dict(csr=c, ws_sample=ws_s, stream=torch.cuda.Stream(),
                          x=torch.empty((rows, cfg.feat_dim), dtype=feats.dtype, device=dev),
                          ready=torch.cuda.Event(), done=torch.cuda.Event()))
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(probe, weights), dev)[1]
    ws_bwd = gmb._aligned_bytes((gmb.backward_embedding_workspace_bytes if args.embed
                                 else gmb.backward_workspace_bytes)(probe, weights), dev)[1]
    emb = dict(embedding=feats, emb_lr=args.lr) if args.embed else {}
    logits = torch.empty((cfg.batch, C), dtype=torch.float32, device=dev)
    grads = gmb.SageGrads(weights)
    # a bf16 model trains fp32 master weights and keeps its bf16 matrices as
    # their rounded copies
    master = weights.master() if weights.dtype == gmb.GMB_BF16 else None
    K, W = args.steps, args.warmup
    losses = torch.zeros(W + 2 * K, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()

    def forward(blocks, x, b):
        if args.fused:   # x: the destination rows, gathered by the forward itself
            return gmb.sage_forward_fused(blocks, feats, weights, x_dst=x, workspace=ws_fwd,
                                          logits=logits[:batches[b].numel()])[0]
        return gmb.sage_forward(blocks, x, weights, workspace=ws_fwd, logits=logits[:batches[b].numel()])

    def model(blocks, x, b, i):
        lg = forward(blocks, x, b)
        gmb.sage_backward(blocks, x, weights, lg, labels[b], ws_fwd, grads=grads, loss=losses[i:i + 1],
                          workspace=ws_bwd, **emb)
        if master is not None:
            gmb.sgd_update_bf16(weights, master, grads, args.lr)
        else:
            gmb.sgd_update(weights, grads, args.lr)

    def step(i):
        b = i % nb
        ln = lanes[i % S]
        st = ln["stream"]
        with torch.cuda.stream(st):
            st.wait_event(ln["done"])
            blocks = gmb.sample_blocks(ln["csr"], batches[b], fanouts, wl.batch_key(b), workspace=ln["ws_sample"])
            x = ln["x"] if args.fused else gmb.gather_features(blocks, feats, out=ln["x"])
            ln["ready"].record(st)
        comp.wait_event(ln["ready"])
        model(blocks, x, b, i)
        ln["done"].record(comp)

    quiet_gc()
    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    # pass A (the figure): K iterations, loaders S batches ahead; the median
    # of PASS_A_RUNS timed passes (each pass continues the training)
    runs = []
    for r in range(PASS_A_RUNS):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(W, W + K):
            step(i)
        torch.cuda.synchronize()
        runs.append(time.perf_counter() - t0)
    T = sorted(runs)[len(runs) // 2]
    for ln in lanes:
        ln["csr"].check_status()
    # pass B: the same iterations on the compute stream alone, events
    # around every stage
    names = ("sample", "gather", "forward", "backward", "sgd")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(K)]
    ln0 = lanes[0]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for j in range(K):
        i = W + K + j
        b = i % nb
        e = evs[j]
        e[0].record(comp)
        blocks = gmb.sample_blocks(ln0["csr"], batches[b], fanouts, wl.batch_key(b), workspace=ln0["ws_sample"])
        e[1].record(comp)
        x = ln0["x"] if args.fused else gmb.gather_features(blocks, feats, out=ln0["x"])
        e[2].record(comp)
        lg = forward(blocks, x, b)
        e[3].record(comp)
        gmb.sage_backward(blocks, x, weights, lg, labels[b], ws_fwd, grads=grads, loss=losses[i:i + 1],
                          workspace=ws_bwd, **emb)
        e[4].record(comp)
        if master is not None:
            gmb.sgd_update_bf16(weights, master, grads, args.lr)
        else:
            gmb.sgd_update(weights, grads, args.lr)
        e[5].record(comp)
    torch.cuda.synchronize()
    T1 = time.perf_counter() - t1
    csr.check_status()
    stage = {n: sum(e[k].elapsed_time(e[k + 1]) for e in evs) for k, n in enumerate(names)}
    loss_h = losses.cpu().numpy()
    if not np.isfinite(loss_h).all():
        raise RuntimeError("non-finite loss in the training run")

    seeds_total = edges_total = 0
    b_gather = fwd_flops = bwd_flops = 0
    for j in range(K):
        b = (W + j) % nb
        blocks = gmb.sample_blocks(csr, batches[b], fanouts, wl.batch_key(b), workspace=lanes[0]["ws_sample"])
        sizes = blocks.sizes()
        seeds_total += batches[b].numel()
        edges_total += sum(s[2] for s in sizes)
        b_gather += alg_gather_bytes(sizes[0][1], cfg.feat_dim, 2 if master is not None else 4)
        fwd_flops += linear_flops(sizes, cfg.dims)
        bwd_flops += backward_flops(sizes, cfg.dims)
    tf, tb = stage["forward"] / 1e3, stage["backward"] / 1e3
    res = {
        "metric": "seeds/s of the training iteration (sample+gather+SAGE fwd+loss+bwd+SGD)"
                  + (", gather folded into the forward" if args.fused else "")
                  + (", learnable vertex embeddings" if args.embed else ""),
        "value": seeds_total / T,
        "unit": "seeds/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": 1e3 * T / K,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.feat_dtype, "data": "synthetic",
        "config": {"workload": f"{args.workload}: {cfg.num_nodes}-node graph, {g.num_edges} edges, feats "
                               f"{cfg.feat_dtype} "
                               f"x{cfg.feat_dim}, SAGE {'-'.join(map(str, cfg.dims))}, fanouts {fanouts}, batch "
                               f"{cfg.batch}, {nb} batches per epoch, SGD lr {args.lr}",
                   "batch": cfg.batch, "fanouts": fanouts, "dims": list(cfg.dims), "batches_per_epoch": nb,
                   "mode": "train", "fused": bool(args.fused), "embed": bool(args.embed),
                   "weights": "bf16 matrices, fp32 master weights, fp32 backward" if master is not None else "f32"},
        "epoch_s": nb * T / K,
        "pass_a_runs_seeds_per_s": [seeds_total / t for t in runs],
        "sampled_edges_per_s": edges_total / T,
        "loader_streams": S,
        "single_stream": {"seeds_per_s": seeds_total / T1, "ms_per_step": 1e3 * T1 / K,
                          "stage_ms_per_step": {k: v / K for k, v in stage.items()}},
        "forward_linear_TFLOPs_lower_bound": fwd_flops / tf / 1e12,
        "backward_products_TFLOPs_lower_bound": bwd_flops / tb / 1e12,
        "mfma_peak_TFLOPs": FP32_MFMA_PEAK_TFLOPS,
        "products_arithmetic": "fp32 operands cut exactly into three bf16 parts, six part products per fp32 "
                               "product on v_mfma_f32_16x16x32_bf16, fp32 accumulation (forward linear, input "
                               "gradients, and the weight gradient of layers with a launch of their own); the "
                               "weight gradients of layers with an input gradient on v_mfma_f32_16x16x4_f32",
        "gemm_check": gemm_check(torch, dev),
        "stream_copy_GBps": stream_copy(torch, dev),
        "gather_GBps": None if args.fused else b_gather / (stage["gather"] / 1e3) / 1e9,
        "loss": {"first": float(loss_h[0]), "last_of_pass_A": float(loss_h[W + K - 1]),
                 "last": float(loss_h[-1])},
        "datagen_s": t_gen,
    }
    # the gather is the one kernel of the iteration bracketed alone by events
    # (in the fused form it runs inside the forward stage: no line)
    if not args.fused:
        es = 2 if master is not None else 4
        t_launch, b_launch = gather_launch_time(gmb, torch, csr, batches, fanouts, wl, cfg, feats,
                                                lanes[0]["x"], K, es, dev)
        res["roofline"] = {"kernel": "k_gather", "bound": "hbm", "achieved": b_launch / t_launch / 1e9,
                           "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": b_launch / t_launch / 1e9 / HBM_PEAK_GBPS,
                           "traffic": None, "alg_bytes_per_launch": b_launch, "avg_launch_ms": 1e3 * t_launch,
                           "launches": f"the last {K} k_gather launches (pass G: {min(GATHER_SETS, nb)} batches "
                                       "cycled, back to back on one stream)",
                           "pass_b_event_bracket_ms": stage["gather"] / K}
    else:
        del res["gather_GBps"]   # no gather stage of its own
    if args.cpu_batches > 0:
        res["cpu_baseline"] = cpu_baseline_train(args, wl, fanouts)
    print(json.dumps(res), flush=True)


def _oracle_train_batch(wl, fanouts, lab_all, lr, b, weights=None):
    import oracle
    g = wl.graph
    ws, wn, bs = weights if weights is not None else wl.weights.as_f64()
    seeds_np = wl.batches[b]
    ref = oracle.sample_blocks(g.indptr, g.indices, seeds_np, fanouts, wl.batch_key(b))
    X = oracle.widen(oracle.gather(wl.feats, ref[0].src), wl.cfg.feat_dtype)
    return oracle.sage_train_step(ref, X, ws, wn, bs, lab_all[seeds_np], lr)


def cpu_baseline_train(args, wl, fanouts):
    """The oracle's training iteration (plain C, fp64): one thread over the
    first batches of the epoch (weights carried from step to step), then
    independent batches spread over the host's threads (each from the
    initial weights: the same work per batch)."""
    from datagen import labels as vertex_labels
    g, cfg = wl.graph, wl.cfg
    lab_all = vertex_labels(g.num_nodes, cfg.dims[-1], cfg.seeds[2] + 1)
    n = min(args.cpu_batches, len(wl.batches))
    seeds_done, t = 0, 0.0
    w = wl.weights.as_f64()
    for b in range(n):
        t0 = time.perf_counter()
        _, _, _, w = _oracle_train_batch(wl, fanouts, lab_all, args.lr, b, w)
        t += time.perf_counter() - t0
        seeds_done += len(wl.batches[b])
    nt = oracle_threads()
    nb_all = min(len(wl.batches), nt)
    t_all, nt = _all_cores(lambda b: _oracle_train_batch(wl, fanouts, lab_all, args.lr, b), nb_all)
    seeds_all = sum(len(wl.batches[b]) for b in range(nb_all))
    return {"value": seeds_all / t_all, "unit": "seeds/s", "cores": nt, "kind": "oracle",
            "sample": f"first {nb_all} of {len(wl.batches)} batches of the epoch ({seeds_all} seeds), one batch per "
                      f"thread on {nt} threads, sample+gather+forward+loss+backward+SGD in fp64 plain C, "
                      f"{t_all:.1f} s wall",
            "single_thread": {"value": seeds_done / t, "unit": "seeds/s", "cores": 1,
                              "sample": f"first {n} batches one after another, {t:.1f} s"},
            "host": host_info()}


def _oracle_infer_batch(wl, fanouts, b):
    import oracle
    g, cfg = wl.graph, wl.cfg
    ws64, wn64, b64 = wl.weights.as_f64()
    ref = oracle.sample_blocks(g.indptr, g.indices, wl.batches[b], fanouts, wl.batch_key(b))
    X = oracle.gather(wl.feats, ref[0].src)
    logits, _ = oracle.sage_forward(ref, oracle.widen(X, cfg.feat_dtype), ws64, wn64, b64)
    return ref, X, logits


def _all_cores(work, n_batches: int):
    """Runs work(b) for b < n_batches on oracle_threads() threads (the
    oracle's C calls release the interpreter lock); returns (seconds,
    threads)."""
    from concurrent.futures import ThreadPoolExecutor
    import oracle
    oracle.lib()
    nt = oracle_threads()
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=nt) as ex:
        list(ex.map(work, range(n_batches)))
    return time.perf_counter() - t0, nt


def cpu_baseline(args, wl, csr, batches, fanouts, feats, weights, ws_sample, x_buf, ws_fwd):
    """The oracle (plain C, fp64) on the first batches of the same epoch:
    one thread, timed batch by batch (its results double as a parity check
    of the GPU run on those batches), then independent batches spread over
    the host's threads (the aggregate figure)."""
    import torch
    import paper_2010_05337_amd as gmb
    n = min(args.cpu_batches, len(batches))
    seeds_done = 0
    t = 0.0
    per_batch = []
    bitexact = True
    max_err = 0.0
    import oracle
    ws64, wn64, bs64 = wl.weights.as_f64()
    stage = {"sample_relabel": [], "gather": [], "forward": []}
    hubs = getattr(wl.graph, "hubs", None)
    hub_rows = []
    for b in range(n):
        # the same steps as _oracle_infer_batch, each timed on its own
        t0 = time.perf_counter()
        ref = oracle.sample_blocks(wl.graph.indptr, wl.graph.indices, wl.batches[b], fanouts, wl.batch_key(b))
        t1 = time.perf_counter()
        X = oracle.gather(wl.feats, ref[0].src)
        t2 = time.perf_counter()
        logits, _ = oracle.sage_forward(ref, oracle.widen(X, wl.cfg.feat_dtype), ws64, wn64, bs64)
        t3 = time.perf_counter()
        stage["sample_relabel"].append(t1 - t0)
        stage["gather"].append(t2 - t1)
        stage["forward"].append(t3 - t2)
        per_batch.append(t3 - t0)
        t += per_batch[-1]
        seeds_done += len(wl.batches[b])
        if hubs is not None and len(hubs):
            # hub occurrences per hop (hop h samples layer L-1-h): hubs among
            # the hop's destinations, edges sampled from hub rows, edges
            # that sampled a hub
            L = len(ref)
            row = []
            for h in range(L):
                r = ref[L - 1 - h]
                dst = r.src[:r.n_dst]
                is_hub_dst = np.isin(dst, hubs)
                from_hub = int(np.diff(r.indptr)[is_hub_dst].sum())
                row.append({"hop": h, "layer": L - 1 - h, "n_dst": int(r.n_dst), "nnz": int(r.nnz),
                            "hub_dsts": int(is_hub_dst.sum()), "edges_from_hub_rows": from_hub,
                            "edges_to_hubs": int(np.isin(r.nbr, hubs).sum())})
            hub_rows.append(row)
        # the GPU result of the same batch
        blocks = gmb.sample_blocks(csr, batches[b], fanouts, wl.batch_key(b), workspace=ws_sample)
        x = gmb.gather_features(blocks, feats, out=x_buf)
        lg = gmb.sage_forward(blocks, x, weights, workspace=ws_fwd)
        got = blocks.blocks()
        for a, r in zip(got, ref):
            bitexact &= (a.n_dst, a.n_src, a.nnz) == (r.n_dst, r.n_src, r.nnz)
            bitexact &= bool(np.array_equal(a.nbr.cpu().numpy(), r.nbr))
            bitexact &= bool(np.array_equal(a.indices.cpu().numpy(), r.local))
            bitexact &= bool(np.array_equal(a.src_ids.cpu().numpy(), r.src))
        xb = x[:ref[0].n_src]
        xb = xb.view(torch.int16).cpu().numpy().view(np.uint16) if xb.dtype == torch.bfloat16 \
            else xb.cpu().numpy()
        bitexact &= xb.tobytes() == X.tobytes()
        out = lg.float().cpu().numpy().astype(np.float64)
        err = (np.abs(out - logits).max(axis=1) / np.maximum(np.abs(logits).max(axis=1), 1e-30)).max()
        max_err = max(max_err, float(err))
    nt = oracle_threads()
    nb_all = min(len(batches), nt)
    t_all, nt = _all_cores(lambda b: _oracle_infer_batch(wl, fanouts, b), nb_all)
    seeds_all = sum(len(wl.batches[b]) for b in range(nb_all))
    base = {"value": seeds_all / t_all, "unit": "seeds/s", "cores": nt, "kind": "oracle",
            "sample": f"first {nb_all} of {len(batches)} batches of the epoch ({seeds_all} seeds), one batch per "
                      f"thread on {nt} threads, sample+gather+forward in fp64 plain C, {t_all:.1f} s wall",
            "single_thread": {"value": seeds_done / t, "unit": "seeds/s", "cores": 1,
                              "batch_s_median": float(np.median(per_batch)),
                              "stage_s_median": {k: float(np.median(v)) for k, v in stage.items()},
                              "sample": f"first {n} batches one after another, {t:.1f} s"},
            "host": host_info()}
    if hub_rows:
        # per hop, the median over the timed batches
        base["hub_occurrences_per_hop"] = [
            {k: (int(np.median([r[h][k] for r in hub_rows])) if k not in ("hop", "layer") else hub_rows[0][h][k])
             for k in hub_rows[0][h]} for h in range(len(hub_rows[0]))]
    par = {"batches": n, "sample_relabel_gather_bitexact": bitexact, "logits_max_rel_err": max_err}
    return base, par


if __name__ == "__main__":
    main()
