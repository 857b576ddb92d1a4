"""Benchmark of the RSLM IVF hot path on one MI355X.

Workload (default): a text-embedding shaped collection of N = 10,000,000
float32 vectors of dimension 768 (anisotropic Gaussian, power-law variance
spectrum with exponent 1, shared mean offset, not normalised), nlist = 4096
Euclidean k-means partitions (10 iterations on 256 points per centre),
4-bit RSLM codes with global scaling and SQ8 codes of the second residual for
rescoring; 10,000 queries from the same distribution in batches of 256,
nprobe = 64, top-100 from the scan, rescored to top-10.

A step is one pass of the whole path over one batch: query rotation,
probing, scan + top-k, rescoring, and the encoding of 65,536 new vectors
into scan records and SQ8 rescoring codes (the collection's fitted ranges).
``value`` is the number of scored (query, candidate) pairs per second of
whole-step time, inputs resident in HBM.  The JSON line also carries the
roofline of the scan kernel, per-stage times, encode throughput and the CPU
oracle's throughput on a bounded sample of the same workload.
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

METRIC = "scored candidates/sec + achieved HBM GB/s, 4-bit d=768 IVF scan, 1 GPU"
HBM_PEAK_GBPS = 8000.0
# The scan's arithmetic: decoded centroids (exact in float16) times the
# rotated query split into two float16 halves (hi + lo, about 22 significant
# bits) on the matrix cores, products exact, accumulated in float32.
SCAN_DTYPE = "split-f16 mfma, f32 accumulate"
# Queries of a batch that probe the same list are scored together, up to
# this many per work item: a list's records leave HBM once per such group.
SCAN_GROUP_Q = 8


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--n", type=int, default=10_000_000)
    ap.add_argument("--dim", type=int, default=768)
    ap.add_argument("--nlist", type=int, default=4096)
    ap.add_argument("--nprobe", type=int, default=64)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--nq", type=int, default=10_000)
    ap.add_argument("--k", type=int, default=100)
    ap.add_argument("--k-out", type=int, default=10)
    ap.add_argument("--bits", type=int, default=4)
    ap.add_argument("--kmeans-iters", type=int, default=10)
    ap.add_argument("--encode-chunk", type=int, default=65536)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lite", action="store_true",
                    help="text768 workload with Rslm4Lite records (scales in the codes)")
    ap.add_argument("--workload", choices=("text768", "mid", "capacity", "sweep", "onetomany"),
                    default="text768",
                    help="text768 (default): the metric's configuration; mid: 1M x 96 unit-norm "
                         "Gaussian mixture (1,024 components), nlist 1,024, 4-bit two-pass RSLM "
                         "+ SQ8 rescoring, nprobe 32; capacity: 100M x 768 "
                         "at nlist 16,384 with 2-bit RSLM rescoring records; sweep: 10M x 1,024 "
                         "unit-norm at 1, 2, 3 and 4 bits with recall@10; onetomany: the paper's "
                         "codec microbenchmarks (OneToMany scoring at D = 256, contiguous and "
                         "gathered from a 128M-record pool, and compression at D = 2049)")
    ap.add_argument("--counter-summary", nargs=2, metavar=("SQ_A_CSV", "SQ_B_CSV"),
                    help="print a markdown summary of the two SQ counter runs and exit")
    ap.add_argument("--copy-calib", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration) and exit")
    ap.add_argument("--stats-summary", nargs=2, metavar=("KERNEL_STATS_CSV", "BENCH_JSON"),
                    help="print a markdown summary of a rocprofv3 --stats run and exit")
    ap.add_argument("--traffic-summary", nargs=5,
                    metavar=("FETCH_CSV", "WRITE_CSV", "CALIB_FETCH_CSV", "CALIB_WRITE_CSV",
                             "BENCH_JSON"),
                    help="print the scan kernel's HBM traffic per launch from rocprofv3 "
                         "FETCH_SIZE / WRITE_SIZE runs and a copy calibration, and exit")
    args = ap.parse_args()
    if args.workload == "mid":
        # the mid-size, non-power-of-two configuration (both rotation passes)
        args.n, args.dim, args.nlist, args.nprobe = 1_000_000, 96, 1024, 32
    return args


# ------------------------------------------------------------------ profile summaries
PROFILE_CMDS = {
    "stats": ("cd /tmp && export TMPDIR=/tmp && rocprofv3 --kernel-trace --stats "
              "--output-format csv -d /tmp/p_stats -o run -- python3 $REPO/bench.py "
              "--no-cpu-baseline"),
    "fetch": ("cd /tmp && rocprofv3 --pmc FETCH_SIZE --output-format csv -d /tmp/p_fetch -o run "
              "-- python3 $REPO/bench.py --steps 5 --warmup 1 --no-cpu-baseline"),
    "write": ("cd /tmp && rocprofv3 --pmc WRITE_SIZE --output-format csv -d /tmp/p_write -o run "
              "-- python3 $REPO/bench.py --steps 5 --warmup 1 --no-cpu-baseline"),
    "calib_fetch": ("cd /tmp && rocprofv3 --pmc FETCH_SIZE --output-format csv -d /tmp/p_cf -o run "
                    "-- python3 $REPO/bench.py --copy-calib"),
    "calib_write": ("cd /tmp && rocprofv3 --pmc WRITE_SIZE --output-format csv -d /tmp/p_cw -o run "
                    "-- python3 $REPO/bench.py --copy-calib"),
    "sq_a": ("cd /tmp && rocprofv3 --pmc SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_INST_ANY "
             "SQ_ACTIVE_INST_VALU SQ_INSTS_VALU SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE "
             "--output-format csv -d /tmp/p_a -o run -- python3 $REPO/bench.py --steps 5 "
             "--warmup 1 --no-cpu-baseline"),
    "sq_b": ("cd /tmp && rocprofv3 --pmc SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_LDS "
             "SQ_WAIT_INST_LDS SQ_INSTS_VMEM_RD SQ_THREAD_CYCLES_VALU SQ_ACTIVE_INST_ANY "
             "SQ_LDS_ADDR_CONFLICT GRBM_GUI_ACTIVE --output-format csv -d /tmp/p_b -o run -- "
             "python3 $REPO/bench.py --steps 5 --warmup 1 --no-cpu-baseline"),
}

STEP_KERNELS = ("k_scan<", "k_topk_stream", "k_dots", "k_probe_select", "k_rescore_sq8",
                "k_encode", "k_rotate", "k_plan")


def stats_summary(stats_csv, bench_json):
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    b = json.load(open(bench_json))
    r = b["roofline"]
    out = ["# rocprofv3 kernel statistics: RSLM IVF scan, text-embedding workload "
           "(10M x 768, 4-bit)", "",
           "Command (run from /tmp on one MI355X; `$REPO` is the repository root):", "",
           "```", PROFILE_CMDS["stats"], "```", "",
           f"Kernel sources hash: `{csrc_hash()}` (scan kernel sources `{scan_src_hash()}`).  The bench run under the profiler reported: "
           f"value {b['value']:.3e} scored candidates/s, {b['ms_per_step']:.3f} ms/step, scan "
           f"kernel {r['kernel_ms'] * 1e3:.1f} us by HIP events ({r['achieved']:.0f} GB/s "
           f"algorithmic, {100 * r['frac']:.1f}% of 8 TB/s).", "",
           "The run covers index construction (assignment and encoding of 10M vectors, SQ8 "
           f"fit/encode) and {b['warmup']} warm-up + {b['steps']} timed steps; the per-step "
           "kernels of the hot path are listed first (their averages include the one large "
           "build-time call of the encoder).", "",
           "| Kernel | Calls | Average (us) | Min (us) | Total (ms) | % |",
           "|---|---|---|---|---|---|"]
    step = [x for x in rows if any(k in x["Name"] for k in STEP_KERNELS)]
    other = [x for x in rows if x not in step]
    for x in step + other[:8]:
        name = x["Name"].replace("|", "\\|")
        name = name if len(name) <= 90 else name[:87] + "..."
        out.append(f"| `{name}` | {x['Calls']} | {float(x['AverageNs']) / 1e3:.1f} | "
                   f"{float(x['MinNs']) / 1e3:.1f} | {float(x['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(x['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def counter_summary(a_csv, b_csv, n_steps=5):
    """Per-kernel SQ counters of the timed steps (the last n_steps dispatches
    of each kernel), with derived utilisations.  Chip-wide cycles of a
    dispatch = GRBM_GUI_ACTIVE / 8 (the counter sums the 8 XCDs); the SQ_*
    cycle counters sum over the 1,024 SIMDs; a wave64 VALU instruction
    occupies its SIMD for 4 cycles."""
    import collections
    import csv

    def load(path):
        d = collections.OrderedDict()
        for r in csv.DictReader(open(path)):
            key = (r["Dispatch_Id"], r["Kernel_Name"])
            d.setdefault(key, collections.Counter())[r["Counter_Name"]] += float(r["Counter_Value"])
        return d
    da, db = load(a_csv), load(b_csv)
    kern = [("k_scan<", "scan (a3+a4)"), ("k_topk_stream", "top-k (a5)"),
            ("k_plan_a", "planning, queries (a3-a5)"), ("k_plan_b", "planning, items (a3-a5)"),
            ("k_dots_tiled", "probe dots (a2)"), ("k_probe_select_reg", "probe selection (a2)"),
            ("k_rotate_reg", "query rotation (a1)"), ("k_rescore_sq8", "rescore (a6)"),
            ("k_encode_rows<6, 4, 2,", "encode with SQ8 codes (a7)")]

    def avg(d, part):
        ds = [v for (i, n), v in d.items() if part in n][-n_steps:]
        if not ds:
            return None
        return {c: sum(x[c] for x in ds) / len(ds) for c in ds[0]}
    out = ["# rocprofv3 SQ counters of the step's kernels: RSLM IVF scan, text-embedding workload "
           "(10M x 768, 4-bit)", "",
           "Commands (run from /tmp on one MI355X; `$REPO` is the repository root):", "",
           "```", PROFILE_CMDS["sq_a"], PROFILE_CMDS["sq_b"], "```", "",
           f"Kernel sources hash: `{csrc_hash()}`.  Averages over the last 5 dispatches of each "
           "kernel (steps of the same workload).  Chip cycles "
           "= GRBM_GUI_ACTIVE / 8; VALU busy = 4 x SQ_ACTIVE_INST_VALU / 1,024 SIMDs / chip "
           "cycles; VALU lane use = SQ_THREAD_CYCLES_VALU / (64 x SQ_ACTIVE_INST_VALU); MFMA busy = "
           "SQ_VALU_MFMA_BUSY_CYCLES / 1,024 / chip cycles; LDS bank-conflict share = "
           "SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS; wait share = SQ_WAIT_INST_ANY / "
           "SQ_WAVE_CYCLES.", "",
           "| Kernel | chip cycles | waves | VALU instr / wave | VALU busy | VALU lane use | MFMA "
           "busy | LDS instr / wave | LDS bank-conflict share | wait share |",
           "|---|---|---|---|---|---|---|---|---|---|"]
    for part, label in kern:
        a, b = avg(da, part), avg(db, part)
        if a is None or b is None:
            continue
        cyc = a["GRBM_GUI_ACTIVE"] / 8
        waves = max(a["SQ_WAVES"], 1)
        valu_busy = 4 * a["SQ_ACTIVE_INST_VALU"] / 1024 / cyc
        lane_use = b["SQ_THREAD_CYCLES_VALU"] / max(64 * a["SQ_ACTIVE_INST_VALU"], 1)
        mfma = b["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / cyc
        lds_conf = a["SQ_LDS_BANK_CONFLICT"] / max(b["SQ_ACTIVE_INST_LDS"], 1)
        wait = a["SQ_WAIT_INST_ANY"] / max(a["SQ_WAVE_CYCLES"], 1)
        out.append(f"| {label} `{part.split('<')[0]}` | {cyc:,.0f} | {waves:,.0f} | "
                   f"{a['SQ_INSTS_VALU'] / waves:,.0f} | {100 * valu_busy:.0f}% | "
                   f"{100 * lane_use:.0f}% | {100 * mfma:.0f}% | "
                   f"{a['SQ_INSTS_LDS'] / waves:,.0f} | {100 * lds_conf:.1f}% | {100 * wait:.0f}% |")
    return "\n".join(out) + "\n"


def _pmc_per_dispatch(csv_path, name_part, counter):
    import csv
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(csv_path))
            if name_part in r["Kernel_Name"] and r["Counter_Name"] == counter]
    return vals


def traffic_summary(fetch_csv, write_csv, cf_csv, cw_csv, bench_json):
    b = json.load(open(bench_json))
    fetch = _pmc_per_dispatch(fetch_csv, "k_scan<", "FETCH_SIZE")
    write = _pmc_per_dispatch(write_csv, "k_scan<", "WRITE_SIZE")
    # calibration: the largest copy dispatch of the 1 GiB device copy
    cf = max(_pmc_per_dispatch(cf_csv, "", "FETCH_SIZE"))
    cw = max(_pmc_per_dispatch(cw_csv, "", "WRITE_SIZE"))
    calib = 1 << 30
    ff, wf = calib / (cf * 1024), calib / (cw * 1024)
    # the scan's launches of the timed steps: after the warm-up launches (the
    # stage-breakdown and recall passes follow them)
    n, w0 = b["steps"], b["warmup"]
    fk, wk = sum(fetch[w0:w0 + n]) / n, sum(write[w0:w0 + n]) / n
    rd, wr = fk * 1024 * ff, wk * 1024 * wf
    return {
        "kernel": b["roofline"]["kernel"],
        "workload": ("10,000,000 x 768 anisotropic Gaussian, nlist 4096, 4-bit RSLM global, "
                     "batch 256, nprobe 64"),
        "scan_src_sha": scan_src_hash(),
        "fetch_KiB_per_launch": fk,
        "write_KiB_per_launch": wk,
        "copy_calibration": {"bytes": calib, "fetch_KiB": cf, "write_KiB": cw,
                             "fetch_factor": ff, "write_factor": wf},
        "hbm_bytes_per_launch": rd + wr,
        "hbm_read_bytes_per_launch": rd,
        "hbm_write_bytes_per_launch": wr,
        "algorithmic_read_bytes_per_launch_same_run": b["roofline"]["algorithmic_bytes_per_launch"],
        "commands": [PROFILE_CMDS[k] for k in ("fetch", "write", "calib_fetch", "calib_write")],
    }


def csrc_hash():
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2608_30384_amd", "csrc")
    for f in sorted(os.listdir(d)):
        with open(os.path.join(d, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


SCAN_SOURCES = ("paper_2608_30384_amd/csrc/scan.hip", "paper_2608_30384_amd/csrc/select_dev.h",
                "paper_2608_30384_amd/csrc/rslm_internal.h", "include/rslm.h")


def scan_src_hash():
    """Hash of the files the scan kernel is compiled from."""
    h = hashlib.sha256()
    for f in SCAN_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def traffic_from_profiles(streamed_records_per_launch):
    """HBM bytes per scan launch from committed rocprofv3 counters, if they
    were taken on the current kernel sources; else None."""
    p = os.path.join(ROOT, "profiles", "scan_traffic_text768.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    if t.get("scan_src_sha") != scan_src_hash():
        return None
    return t.get("hbm_bytes_per_launch")


def calibrate_read(torch, lib, x, reps=5):
    """Best read bandwidth (GB/s) of the calibration kernel over the first
    4 GiB of x, across grid sizes and with / without non-temporal loads."""
    import ctypes
    flat = x.view(-1)[: min(x.numel(), 1 << 30)]
    nbytes = flat.numel() * 4
    out = torch.empty(1 << 16, dtype=torch.int32, device=x.device)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    best = (0.0, None)
    for nt in (0, 1):
        for grid in (2048, 8192, 32768, 65536):
            call = lambda: lib.rslm_calibrate_read(ctypes.c_void_p(flat.data_ptr()), nbytes,
                                                   ctypes.c_void_p(out.data_ptr()), grid, nt,
                                                   stream)
            for _ in range(2):
                call()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                st = call()
                assert st == 0, st
            e1.record()
            torch.cuda.synchronize()
            bw = reps * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9
            if bw > best[0]:
                best = (bw, {"grid": grid, "nontemporal": bool(nt)})
    return best


# ------------------------------------------------------------------ CPU baseline
_CPU = {}


def _cpu_query(i):
    """One query of the batch through the oracle: its probed lists' canonical
    records are unpacked and their scales decoded (input preparation, timed
    apart), then the LUT-route scan and the top-k (timed)."""
    import oracle
    d = _CPU
    t0 = time.perf_counter()
    lists = []
    for L in d["pid"][i]:
        o, n = int(d["offs"][L]), int(d["sizes"][L])
        if n == 0:
            continue
        sc = d["scales"][o:o + n]
        lists.append((oracle.unpack_canonical(d["canon"][o:o + n], d["bits"], d["n_sub"]),
                      d["dec_s"][sc & 0xFFFF], d["dec_g"][sc >> 16], d["ids"][o:o + n]))
    t1 = time.perf_counter()
    all_s, all_i = [], []
    pairs = 0
    j = 0
    for jj, L in enumerate(d["pid"][i]):
        if int(d["sizes"][L]) == 0:
            continue
        codes, sh, gh, ids = lists[j]
        j += 1
        s = oracle.scan_scores_lut(d["qrot"][i], d["pdot"][i, jj], codes, sh, gh, d["C"])
        all_s.append(s)
        all_i.append(ids)
        pairs += len(s)
    if all_s:
        oracle.topk(np.concatenate(all_s), np.concatenate(all_i), d["k"])
    return pairs, time.perf_counter() - t1, t1 - t0, os.getpid()


def _cpu_encode(lo_hi):
    """Rows [lo, hi) of the encode sample through the oracle: codes and
    scales, the rotated second residual and its SQ8 codes."""
    import oracle
    d = _CPU
    lo, hi = lo_hi
    t0 = time.perf_counter()
    xs = d["xe"][lo:hi]
    cen = d["cen"][d["ae"][lo:hi]]
    enc = oracle.encode(xs, d["Rm"], d["C"], d["bits"], centroids=cen, scale_mode="global")
    ra = oracle.first_stage_rotated(enc["codes"], enc["s_code"], enc["g_code"], d["C"], d["Rm"],
                                    cen)
    r2 = xs @ d["Rm"].T - ra
    oracle.sq8_encode(r2, d["sq8_lo"], d["sq8_hi"])
    return hi - lo, time.perf_counter() - t0, os.getpid()


def _per_worker_wall(res, t_index, pid_index):
    """The busiest worker's summed time: the wall time of the timed parts."""
    tot = {}
    for r in res:
        tot[r[pid_index]] = tot.get(r[pid_index], 0.0) + r[t_index]
    return max(tot.values())


def cpu_baseline(R, plan, index, qrot, pid, pdot, k, xe_rows, cen, n_encode=1 << 17):
    """The oracle on the host cores, on bounded samples of the workload:
    (1) the LUT-route scan + top-k of every query of the first batch over its
    probed lists (the index's records unpacked to the oracle's canonical
    codes); (2) the encode of the first n_encode collection vectors (codes,
    scales, rotated second residual, SQ8 codes), against the oracle's own
    assignment of them, computed beforehand."""
    import multiprocessing as mp

    import oracle
    import synth

    workers = max(1, min(16, os.cpu_count() or 1))
    K, g = oracle.codec_shape(plan.bits)
    n_sub = -(-plan.dim // g)
    total = index.ids.numel()
    canon = R.rslm_unpack_codes(plan, index.codes, total).cpu().numpy()
    Rm = oracle.rotation_matrix(plan.dim, plan.passes, synth.sign_table(),
                                synth.permutation_table())
    xe = xe_rows.cpu().numpy().astype(np.float64)
    cen_h = cen.cpu().numpy().astype(np.float64)
    ae, _ = oracle.assign_l2_expanded(xe, cen_h)
    # SQ8 ranges of the sample's own second residuals (oracle), as fitted ranges
    enc0 = oracle.encode(xe[:4096], Rm, synth.codebook(plan.bits), plan.bits,
                         centroids=cen_h[ae[:4096]], scale_mode="global")
    ra0 = oracle.first_stage_rotated(enc0["codes"], enc0["s_code"], enc0["g_code"],
                                     synth.codebook(plan.bits), Rm, cen_h[ae[:4096]])
    sq8_lo, sq8_hi = oracle.sq8_fit(xe[:4096] @ Rm.T - ra0)
    _CPU.update(pid=pid.cpu().numpy(), pdot=pdot.cpu().numpy().astype(np.float64),
                qrot=qrot.cpu().numpy().astype(np.float64), canon=canon,
                scales=index.scales.cpu().numpy().astype(np.uint32),
                ids=index.ids.cpu().numpy().astype(np.int64),
                offs=index.list_offsets.cpu().numpy(), sizes=index.list_sizes.cpu().numpy(),
                bits=plan.bits, n_sub=n_sub, C=synth.codebook(plan.bits), k=k, xe=xe,
                # the oracle's scale decoders tabulated over all 2^16 codes
                dec_s=np.array([oracle.dec_ue7m9(u) for u in range(1 << 16)]),
                dec_g=np.array([oracle.dec_ue4m12(u) for u in range(1 << 16)]),
                cen=cen_h, ae=ae, Rm=Rm, sq8_lo=sq8_lo, sq8_hi=sq8_hi)
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    ctx = mp.get_context("fork")
    nq = qrot.shape[0]
    with ctx.Pool(workers) as pool:
        t0 = time.perf_counter()
        res = pool.map(_cpu_query, range(nq), chunksize=1)
        wall_q = time.perf_counter() - t0
        chunk = 2048
        t0 = time.perf_counter()
        res_e = pool.map(_cpu_encode, [(a, min(len(xe), a + chunk))
                                       for a in range(0, len(xe), chunk)], chunksize=1)
        wall_e = time.perf_counter() - t0
    pairs = sum(r[0] for r in res)
    scan_wall = _per_worker_wall(res, 1, 3)
    enc_wall = _per_worker_wall(res_e, 1, 2)
    _CPU.clear()
    return {"value": pairs / scan_wall, "unit": "scored candidates/s", "cores": workers,
            "kind": "oracle",
            "sample": (f"oracle LUT-route scan + top-{k} (float64 NumPy) of all {nq} queries of "
                       f"the first batch over their probed {plan.dim}-d {plan.bits}-bit lists "
                       f"({pairs} pairs); rate = pairs / the busiest of {workers} worker "
                       f"processes' summed scan time ({scan_wall:.1f} s; {wall_q:.1f} s wall "
                       f"including the per-query unpacking of canonical records)"),
            "encode": {"value": len(xe) / enc_wall, "unit": "vectors/s", "cores": workers,
                       "sample": (f"oracle encode (codes, UE7M9/UE4M12 scales, rotated second "
                                  f"residual, SQ8 codes; float64 NumPy, dense rotation) of the "
                                  f"first {len(xe)} collection vectors against the oracle's own "
                                  f"assignment, {workers} worker processes, {enc_wall:.1f} s "
                                  f"(busiest worker), {wall_e:.1f} s wall")}}


# ------------------------------------------------------------------ main
def main():
    args = parse()
    if args.stats_summary:
        sys.stdout.write(stats_summary(*args.stats_summary))
        return
    if args.counter_summary:
        sys.stdout.write(counter_summary(*args.counter_summary))
        return
    if args.traffic_summary:
        print(json.dumps(traffic_summary(*args.traffic_summary), indent=1))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only (the scan has no multi-GPU path); run with --gpus 1"}))
        sys.exit(2)
    if args.workload == "capacity":
        return run_capacity(args)
    if args.workload == "sweep":
        return run_sweep(args)
    if args.workload == "onetomany":
        return run_onetomany(args)
    import torch

    import synth
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import _lib as LL
    from paper_2608_30384_amd import ivf

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    if args.copy_calib:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calib_bytes": a.numel() * 4}))
        return

    N, D, nlist = args.n, args.dim, args.nlist
    mid = args.workload == "mid"
    t_setup = time.time()
    log(f"generating {N} x {D} vectors")
    if mid:
        # unit-norm Gaussian mixture of 1,024 components (host generator)
        x = torch.from_numpy(synth.gmix(N, D, 1024, seed=100)).to(dev)
        q_all = torch.from_numpy(synth.queries_like("gmix", args.nq, D, data_seed=100,
                                                    query_seed=200, n_comp=1024)).to(dev)
    else:
        x = synth.aniso_torch(N, D, alpha=1.0, seed=100, device=dev)
        q_all = torch.from_numpy(synth.queries_like("aniso", args.nq, D, data_seed=100,
                                                    query_seed=200)).to(dev)
    torch.cuda.synchronize()
    log(f"k-means: {nlist} lists, {args.kmeans_iters} iterations on {min(N, 256 * nlist)} points")
    t0 = time.time()
    cen = ivf.kmeans(x, nlist, iters=args.kmeans_iters, seed=0, sample=256 * nlist)
    torch.cuda.synchronize()
    log(f"k-means done in {time.time() - t0:.1f} s")
    # the mid-size configuration exercises the block-wise cascade: two passes
    plan = R.Plan(D, args.bits, passes=2 if mid else -1, scale_mode="global", lite=args.lite)
    resid = torch.empty_like(x)
    t0 = time.time()
    index, crot, assign = ivf.build_index(plan, x, cen, resid_rot=resid)
    torch.cuda.synchronize()
    log(f"assign + layout + encode of {N} vectors: {time.time() - t0:.1f} s; "
        f"max list {index.max_list_size}, records {index.ids.numel()}")
    codes2, lo, hi = ivf.build_sq8(resid)
    del resid
    torch.cuda.synchronize()
    # a chunk of new vectors for the per-step encode (row a7)
    if mid:
        xe = torch.from_numpy(synth.gmix(args.encode_chunk, D, 1024, seed=300,
                                         mean_seed=100)).to(dev)
    else:
        xe = synth.aniso_torch(args.encode_chunk, D, alpha=1.0, seed=300, device=dev)
    ae, _ = R.ivf_assign_probe(xe, cen, 1, R.IVF_ASSIGN_L2)
    codes_e = torch.empty(plan.code_bytes(args.encode_chunk), dtype=torch.uint8, device=dev)
    scales_e = torch.empty(args.encode_chunk, dtype=torch.int32, device=dev)
    sq8_e = torch.empty((args.encode_chunk, D), dtype=torch.uint8, device=dev)
    log(f"setup {time.time() - t_setup:.1f} s")

    # context: the read bandwidth a plain streaming kernel sustains on this
    # device (rslm_calibrate_read over 4 GiB of the collection, best grid)
    stream_read_GBps, stream_read_cfg = calibrate_read(torch, LL.lib(), x)

    batches = [q_all[i:i + args.batch].contiguous() for i in range(0, args.nq, args.batch)]
    sizes = index.list_sizes.long()
    rec_bytes = D * args.bits // 8 + (0 if args.lite else 4)
    # per-batch work, computed outside the timed region from the probe result
    work = []
    for qb in batches:
        pid, _ = R.ivf_assign_probe(qb, cen, args.nprobe, R.IVF_PROBE_IP)
        pl = pid.long().reshape(-1)
        pairs = int(sizes[pl].sum().item())
        m = torch.bincount(pl, minlength=nlist)
        groups = (m + SCAN_GROUP_Q - 1) // SCAN_GROUP_Q
        streamed = int((groups * sizes).sum().item())
        distinct = int(sizes[m > 0].sum().item())     # records of the lists probed at all
        work.append((pairs, streamed, distinct))

    ws_scan = torch.empty(R.rslm_scan_topk_workspace(plan, index, args.batch, args.nprobe, args.k),
                          dtype=torch.uint8, device=dev)
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def step(b, timers):
        """One pass of every row over one batch: rotate, probe, scan + top-k,
        rescore, and the encode of new vectors into scan records and SQ8
        rescoring codes (row a7), in this order on one stream.  (The encode
        on a second stream shortens the step by about 3 %, but its
        workgroups then share the CUs with the scan, whose own time grows by
        about 6 %; in order, the scan's figure is the kernel's alone.)"""
        qb = batches[b % len(batches)]
        mark = (lambda i: timers[i].record()) if timers else (lambda i: None)
        mark(0)
        qrot = R.rslm_fwht(plan, qb)
        mark(1)
        pid, pdot = R.ivf_assign_probe(qb, cen, args.nprobe, R.IVF_PROBE_IP)
        mark(2)
        s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, args.k, ws=ws_scan)
        mark(3)
        R.rslm_rescore(codes2, lo, hi, qrot, s1, i1, args.k_out)
        mark(4)
        R.rslm_encode_sq8(plan, xe, codes_e, scales_e, lo, hi, sq8_e, rec_list=ae, centroids=cen,
                          centroids_rot=crot)
        mark(5)
        return qrot, pid, pdot

    lib = LL.lib()
    for w in range(args.warmup):
        step(w, None)
    torch.cuda.synchronize()
    scan_ev = []
    for s in range(args.steps):
        scan_ev.append([ev() for _ in range(4)])
        for e in scan_ev[-1]:
            e.record()          # materialise the HIP events before handing them over
    torch.cuda.synchronize()
    # timed region: the steps, with the library's HIP events around the scan
    # and top-k kernels only (stage events would add their own gaps)
    t0 = time.perf_counter()
    for s in range(args.steps):
        se = scan_ev[s]
        lib.rslm_set_timer(0, se[0]._as_parameter_, se[1]._as_parameter_)
        lib.rslm_set_timer(1, se[2]._as_parameter_, se[3]._as_parameter_)
        step(args.warmup + s, None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    lib.rslm_set_timer(0, None, None)
    lib.rslm_set_timer(1, None, None)

    # per-stage breakdown: the same steps again, events between the stages
    names = ["rotate", "probe", "scan_topk", "rescore", "encode"]
    stage = {n: 0.0 for n in names}
    all_ev = [[ev() for _ in range(6)] for _ in range(args.steps)]
    for s in range(args.steps):
        step(args.warmup + s, all_ev[s])
    torch.cuda.synchronize()
    for e in all_ev:
        for i, n in enumerate(names):
            stage[n] += e[i].elapsed_time(e[i + 1])
    t_scan = sum(se[0].elapsed_time(se[1]) for se in scan_ev) / args.steps
    t_topk = sum(se[2].elapsed_time(se[3]) for se in scan_ev) / args.steps
    steps_b = [(args.warmup + s) % len(batches) for s in range(args.steps)]
    pairs_total = sum(work[b][0] for b in steps_b)
    streamed_avg = sum(work[b][1] for b in steps_b) / args.steps
    distinct_avg = sum(work[b][2] for b in steps_b) / args.steps
    pairs_avg = pairs_total / args.steps
    ms_per_step = wall * 1e3 / args.steps
    value = pairs_total / wall
    achieved = streamed_avg * rec_bytes / (t_scan * 1e-3) / 1e9
    traffic = None if (mid or args.lite) else traffic_from_profiles(streamed_avg)
    enc_ms = stage["encode"] / args.steps
    enc_bytes = args.encode_chunk * (4 * D + rec_bytes + D)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "scored candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": SCAN_DTYPE,
        "data": "synthetic",
        "config": {
            "workload": ((f"mid-size IVF scan: N={N:,} x d={D} unit-norm Gaussian mixture "
                          f"(1,024 components, sigma 0.3), " if mid else
                          f"text-embedding shaped IVF scan: N={N:,} x d={D} anisotropic Gaussian "
                          f"(power-law spectrum, exponent 1, mean offset, unnormalised), ") +
                         f"nlist={nlist}, {args.bits}-bit RSLM{'4Lite' if args.lite else ''} "
                         f"global scale ({plan.passes} rotation passes) + SQ8 rescore, "
                         f"batches of {args.batch} queries, nprobe={args.nprobe}, "
                         f"top-{args.k} -> top-{args.k_out}; each step also encodes "
                         f"{args.encode_chunk:,} vectors"),
            "N": N, "dim": D, "nlist": nlist, "nprobe": args.nprobe, "batch": args.batch,
            "k": args.k, "k_out": args.k_out, "bits": args.bits, "passes": plan.passes,
        },
        "hbm_GBps": achieved,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "kernel": f"k_scan<{args.bits},{plan.d_pad // 32}>",
            "algorithmic_bytes_per_launch": streamed_avg * rec_bytes,
            "kernel_ms": t_scan,
            "stream_read_GBps_measured": stream_read_GBps,
            "stream_read_kernel": stream_read_cfg,
            "frac_of_measured_stream": achieved / stream_read_GBps,
            # the same kernel time under the two other byte models: every
            # scored (query, candidate) pair reading its record, and every
            # record of a list the batch probes read once
            "frac_pair_equivalent": pairs_avg * rec_bytes / (t_scan * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "frac_min_bytes": distinct_avg * rec_bytes / (t_scan * 1e-3) / 1e9 / HBM_PEAK_GBPS,
            "min_bytes_per_launch": distinct_avg * rec_bytes,
        },
        "scan": {
            "pairs_per_step": pairs_avg,
            "streamed_records_per_step": streamed_avg,
            "record_bytes": rec_bytes,
            "candidates_per_s_scan_kernel": pairs_avg / (t_scan * 1e-3),
            "pair_equivalent_GBps": pairs_avg * rec_bytes / (t_scan * 1e-3) / 1e9,
            "topk_kernel_ms": t_topk,
        },
        "stages_ms": {n: stage[n] / args.steps for n in names},
        "stages_from": "a second pass over the same steps with HIP events between the stages",
        "encode": {
            "vectors": args.encode_chunk,
            "ms": enc_ms,
            "vectors_per_s": args.encode_chunk / (enc_ms * 1e-3),
            "GBps": enc_bytes / (enc_ms * 1e-3) / 1e9,
        },
        "kernel_sources": csrc_hash(),
        "scan_sources": scan_src_hash(),
    }
    # two-stage encode (4-bit scan codes + 2-bit RSLM rescoring codes, the
    # capacity configuration's records) of the same chunk, outside the step
    plan2 = R.Plan(D, 2, passes=0, scale_mode="global")
    codes2_e = torch.empty((args.encode_chunk, plan2.canon_bytes), dtype=torch.uint8, device=dev)
    scales2_e = torch.empty(args.encode_chunk, dtype=torch.int32, device=dev)

    def enc2():
        R.rslm_encode_two_stage(plan, plan2, xe, codes_e, scales_e, codes2_e, scales2_e,
                                rec_list=ae, centroids=cen, centroids_rot=crot)
    for _ in range(2):
        enc2()
    e0, e1 = ev(), ev()
    e0.record()
    for _ in range(10):
        enc2()
    e1.record()
    torch.cuda.synchronize()
    t2 = e0.elapsed_time(e1) / 10
    b2 = args.encode_chunk * (4 * D + rec_bytes + plan2.canon_bytes + 4)
    out["encode_two_stage"] = {
        "vectors": args.encode_chunk, "ms": t2,
        "vectors_per_s": args.encode_chunk / (t2 * 1e-3),
        "GBps": b2 / (t2 * 1e-3) / 1e9,
        "record_bytes": [rec_bytes, plan2.canon_bytes + 4],
    }
    # quality of what the step returns, outside the timed region: recall@10
    # of the rescored top-k_out and of the scan's own first k_out, against
    # exact float32 MIPS over the raw vectors (torch matmul on the device:
    # the reference of a quality figure, not of a kernel)
    hits_final = hits_scan = nq_rec = 0
    for b in range(min(2, len(batches))):
        qb = batches[b]
        qrot = R.rslm_fwht(plan, qb)
        pid, pdot = R.ivf_assign_probe(qb, cen, args.nprobe, R.IVF_PROBE_IP)
        s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, args.k, ws=ws_scan)
        _, i2 = R.rslm_rescore(codes2, lo, hi, qrot, s1, i1, args.k_out)
        ex = torch.topk(torch.matmul(qb, x.T), args.k_out, dim=1).indices.int()
        hits_final += int((i2[:, :, None] == ex[:, None, :]).any(2).sum().item())
        hits_scan += int((i1[:, :args.k_out, None] == ex[:, None, :]).any(2).sum().item())
        nq_rec += qb.shape[0]
    out["quality"] = {
        "queries": nq_rec,
        f"recall_at_{args.k_out}": hits_final / (nq_rec * args.k_out),
        f"recall_at_{args.k_out}_scan_only": hits_scan / (nq_rec * args.k_out),
        "reference": "exact float32 inner products over the raw vectors (torch matmul)",
    }
    if not args.no_cpu_baseline and not args.lite:
        log("CPU oracle baseline")
        qrot, pid, pdot = step(0, None)
        torch.cuda.synchronize()
        del codes2
        torch.cuda.empty_cache()
        out["cpu_baseline"] = cpu_baseline(R, plan, index, qrot, pid, pdot, args.k,
                                           x[:min(N, 1 << 17)], cen)
    print(json.dumps(out), flush=True)


# ------------------------------------------------------------------ other workloads
def _timed_batches(torch, batches, fn, warmup):
    """Runs fn over every batch (after `warmup` untimed ones); returns the
    wall time of the timed pass (host clock between synchronisations)."""
    for i in range(warmup):
        fn(batches[i % len(batches)])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for qb in batches:
        fn(qb)
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def _streamed(torch, R, cen, batches, nprobe, sizes, nlist):
    """Scored pairs and streamed records (lists read once per group of
    <= SCAN_GROUP_Q queries) of each batch, computed outside the timed
    region."""
    out = []
    for qb in batches:
        pid, _ = R.ivf_assign_probe(qb, cen, nprobe, R.IVF_PROBE_IP)
        pl = pid.long().reshape(-1)
        m = torch.bincount(pl, minlength=nlist)
        out.append((int(sizes[pl].sum().item()),
                    int((((m + SCAN_GROUP_Q - 1) // SCAN_GROUP_Q) * sizes).sum().item())))
    return out


def run_capacity(args):
    """Capacity configuration: 100,000,000 x 768 anisotropic vectors (raw
    float32 never resident: generated, assigned and encoded in blocks of
    2^22 rows), nlist 16,384, 4-bit RSLM scan records + 2-bit RSLM rescoring
    records (two-stage encode, global scales) resident in HBM; 100,000 queries
    in batches of 1,024, nprobe 128, top-100 from the scan rescored to top-10.
    Reports the scan path's throughput over every batch and the bulk
    two-stage encode rate on a device-resident block."""
    import torch

    import synth
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import _lib as LL
    from paper_2608_30384_amd import ivf

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    N, D, nlist, nprobe, B = 100_000_000, 768, 16384, 128, 1024
    nq, k, k_out = 100_000, 100, 10
    BLK = synth.TORCH_BLOCK
    t_setup = time.time()
    plan = R.Plan(D, 4, passes=-1, scale_mode="global")
    plan2 = R.Plan(D, 2, passes=0, scale_mode="global")
    xb = torch.empty((BLK, D), dtype=torch.float32, device=dev)

    def block(b):
        synth.aniso_torch_block(b, D, seed=100, out=xb)
        rows = min(BLK, N - b * BLK)
        return xb[:rows]

    log(f"k-means: {nlist} lists on the first {256 * nlist} rows, {args.kmeans_iters} iterations")
    sample = block(0)[: 256 * nlist].contiguous()
    cen = ivf.kmeans(sample, nlist, iters=args.kmeans_iters, seed=0)
    del sample
    torch.cuda.synchronize()
    t_km = time.time()
    log(f"k-means done at {t_km - t_setup:.0f} s; assigning {N} rows")
    t_as = None

    def assigned():
        nonlocal t_as
        torch.cuda.synchronize()
        t_as = time.time()
        log(f"assignment done at {t_as - t_setup:.0f} s")
    index, codes2, scales2, crot = ivf.build_two_stage_blocked(plan, plan2, block, N, BLK, cen,
                                                               on_assigned=assigned)
    torch.cuda.synchronize()
    resident = (index.codes.numel() + index.scales.numel() * 4 + codes2.numel() +
                scales2.numel() * 4 + index.ids.numel() * 4)
    t_built = time.time()
    log(f"index built at {t_built - t_setup:.0f} s: {index.ids.numel()} records, max list "
        f"{index.max_list_size}, {resident / 1e9:.1f} GB resident")

    # bulk two-stage encode rate on one device-resident block (records = rows)
    xs = block(0)
    a0, _ = R.ivf_assign_probe(xs, cen, 1, R.IVF_ASSIGN_L2)
    c_e = torch.empty(plan.code_bytes(len(xs)), dtype=torch.uint8, device=dev)
    s_e = torch.empty(len(xs), dtype=torch.int32, device=dev)
    c2_e = torch.empty((len(xs), plan2.canon_bytes), dtype=torch.uint8, device=dev)
    s2_e = torch.empty(len(xs), dtype=torch.int32, device=dev)
    enc = lambda: R.rslm_encode_two_stage(plan, plan2, xs, c_e, s_e, c2_e, s2_e, rec_list=a0,
                                          centroids=cen, centroids_rot=crot)
    enc()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(3):
        enc()
    e1.record()
    torch.cuda.synchronize()
    t_enc = e0.elapsed_time(e1) / 3
    del c_e, s_e, c2_e, s2_e, xb, xs
    torch.cuda.empty_cache()

    q_all = torch.from_numpy(synth.queries_like("aniso", nq, D, data_seed=100,
                                                query_seed=200)).to(dev)
    batches = [q_all[i:i + B].contiguous() for i in range(0, nq, B)]
    work = _streamed(torch, R, cen, batches, nprobe, index.list_sizes.long(), nlist)
    ws = torch.empty(R.rslm_scan_topk_workspace(plan, index, B, nprobe, k), dtype=torch.uint8,
                     device=dev)
    log(f"setup {time.time() - t_setup:.0f} s; scan workspace {ws.numel() / 1e9:.1f} GB")

    def query(qb):
        qrot = R.rslm_fwht(plan, qb)
        pid, pdot = R.ivf_assign_probe(qb, cen, nprobe, R.IVF_PROBE_IP)
        s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, k, ws=ws)
        R.rslm_rescore_rslm(plan2, codes2, scales2, qrot, s1, i1, k_out)

    wall = _timed_batches(torch, batches, query, args.warmup)
    # the scan kernel alone (HIP events around its launch), on every batch
    lib = LL.lib()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in batches]
    for a, b_ in evs:
        a.record()
        b_.record()
    torch.cuda.synchronize()
    for (a, b_), qb in zip(evs, batches):
        lib.rslm_set_timer(0, a._as_parameter_, b_._as_parameter_)
        query(qb)
    torch.cuda.synchronize()
    lib.rslm_set_timer(0, None, None)
    t_scan = sum(a.elapsed_time(b_) for a, b_ in evs) * 1e-3
    pairs = sum(w[0] for w in work)
    streamed = sum(w[1] for w in work)
    rec_bytes = D * 4 // 8 + 4
    achieved = streamed * rec_bytes / t_scan / 1e9
    out = {
        "metric": METRIC,
        "value": pairs / wall,
        "unit": "scored candidates/s",
        "n_gpus": 1, "steps": len(batches), "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / len(batches),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": SCAN_DTYPE, "data": "synthetic",
        "config": {"workload": ("capacity: N=100,000,000 x d=768 anisotropic Gaussian, "
                                "nlist=16384, 4-bit RSLM global + 2-bit RSLM global rescoring "
                                "records resident, 100,000 queries in batches of 1,024, "
                                "nprobe=128, top-100 -> top-10"),
                   "N": N, "dim": D, "nlist": nlist, "nprobe": nprobe, "batch": B,
                   "k": k, "k_out": k_out, "bits": 4, "rescore_bits": 2},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "k_scan<4,24>", "kernel_ms_per_batch": t_scan * 1e3 / len(batches),
                     "algorithmic_bytes_per_batch": streamed * rec_bytes / len(batches)},
        "scan": {"pairs_per_batch": pairs / len(batches),
                 "streamed_records_per_batch": streamed / len(batches),
                 "candidates_per_s_scan_kernel": pairs / t_scan},
        "resident_index_GB": resident / 1e9,
        "max_list_size": index.max_list_size,
        "encode_two_stage": {"vectors": BLK, "ms": t_enc, "vectors_per_s": BLK / (t_enc * 1e-3),
                             "GBps": BLK * (4 * D + rec_bytes + plan2.canon_bytes + 4) /
                             (t_enc * 1e-3) / 1e9},
        "build_s": t_built - t_setup,
        "build_phases_s": {
            "kmeans": t_km - t_setup, "assign": t_as - t_km, "layout_and_encode": t_built - t_as,
            "kmeans_rows": min(N, 256 * nlist), "kmeans_iters": args.kmeans_iters,
            "assign_TFLOPs": 2.0 * N * D * nlist / (t_as - t_km) / 1e12,
        },
        "kernel_sources": csrc_hash(),
    }
    print(json.dumps(out), flush=True)


def run_sweep(args):
    """Bit-width sweep: 10,000,000 x 1,024 anisotropic unit-norm vectors,
    nlist 4,096, RSLM codes at 1, 2, 3 and 4 bits (global scales) of the same
    data; 10,000 queries in batches of 256, nprobe 64, top-10.  Per bit
    width: scored candidates/s over every batch, the scan kernel's
    algorithmic GB/s, and recall@10 against exact float32 MIPS over the raw
    vectors (torch matmul on the device; the reference of a quality figure,
    not of a kernel)."""
    import torch

    import synth
    import paper_2608_30384_amd as R
    from paper_2608_30384_amd import _lib as LL
    from paper_2608_30384_amd import ivf

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    N, D, nlist, nprobe, B, nq, k = 10_000_000, 1024, 4096, 64, 256, 10_000, 10
    t_setup = time.time()
    x = synth.aniso_torch(N, D, alpha=1.0, seed=100, normalize=True, device=dev)
    cen = ivf.kmeans(x, nlist, iters=args.kmeans_iters, seed=0, sample=256 * nlist)
    assign, _ = R.ivf_assign_probe(x, cen, 1, R.IVF_ASSIGN_L2)
    q_all = torch.from_numpy(synth.queries_like("aniso", nq, D, data_seed=100, query_seed=200,
                                                normalize=True)).to(dev)
    batches = [q_all[i:i + B].contiguous() for i in range(0, nq, B)]
    # exact top-10 by float32 inner product over the raw vectors
    exact = []
    for qb in batches:
        s = torch.matmul(qb, x.T)
        exact.append(torch.topk(s, k, dim=1).indices.int())
        del s
    torch.cuda.synchronize()
    log(f"data, partitions and exact top-{k} in {time.time() - t_setup:.0f} s")
    lib = LL.lib()
    res = {}
    for bits in (1, 2, 3, 4):
        plan = R.Plan(D, bits, passes=-1, scale_mode="global")
        index, crot, _ = ivf.build_index(plan, x, cen, assign=assign)
        sizes = index.list_sizes.long()
        work = _streamed(torch, R, cen, batches, nprobe, sizes, nlist)
        ws = torch.empty(R.rslm_scan_topk_workspace(plan, index, B, nprobe, k),
                         dtype=torch.uint8, device=dev)
        found = []

        def query(qb, keep=False):
            qrot = R.rslm_fwht(plan, qb)
            pid, pdot = R.ivf_assign_probe(qb, cen, nprobe, R.IVF_PROBE_IP)
            s1, i1 = R.rslm_scan_topk(plan, index, qrot, pid, pdot, k, ws=ws)
            if keep:
                found.append(i1)
        wall = _timed_batches(torch, batches, query, args.warmup)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in batches]
        for a, b_ in evs:
            a.record()
            b_.record()
        torch.cuda.synchronize()
        for (a, b_), qb in zip(evs, batches):
            lib.rslm_set_timer(0, a._as_parameter_, b_._as_parameter_)
            query(qb, keep=True)
        torch.cuda.synchronize()
        lib.rslm_set_timer(0, None, None)
        t_scan = sum(a.elapsed_time(b_) for a, b_ in evs) * 1e-3
        hits = 0
        for f, e in zip(found, exact):
            hits += int((f[:, :, None] == e[:, None, :]).any(2).sum().item())
        pairs = sum(w[0] for w in work)
        streamed = sum(w[1] for w in work)
        rec_bytes = D * bits // 8 + 4
        res[str(bits)] = {
            "scored_candidates_per_s": pairs / wall,
            "scan_kernel_candidates_per_s": pairs / t_scan,
            "scan_kernel_GBps": streamed * rec_bytes / t_scan / 1e9,
            "scan_kernel_frac_of_8TBps": streamed * rec_bytes / t_scan / 1e9 / HBM_PEAK_GBPS,
            "record_bytes": rec_bytes,
            "recall_at_10": hits / (nq * k),
            "ms_per_batch": wall * 1e3 / len(batches),
        }
        log(f"{bits}-bit: {res[str(bits)]}")
        del index, ws, found
        torch.cuda.empty_cache()
    out = {
        "metric": "scored candidates/s, GB/s and recall@10 per bit width, d=1024 IVF scan, 1 GPU",
        "value": res["4"]["scored_candidates_per_s"], "unit": "scored candidates/s",
        "n_gpus": 1, "steps": len(batches), "warmup": args.warmup,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": SCAN_DTYPE, "data": "synthetic",
        "config": {"workload": ("bit-width sweep: N=10,000,000 x d=1024 anisotropic Gaussian, "
                                "unit norm, nlist=4096, RSLM 1/2/3/4-bit global, 10,000 queries "
                                "in batches of 256, nprobe=64, top-10"),
                   "N": N, "dim": D, "nlist": nlist, "nprobe": nprobe, "batch": B, "k": k},
        "per_bits": res,
        "setup_s": time.time() - t_setup,
        "kernel_sources": csrc_hash(),
    }
    print(json.dumps(out), flush=True)


# The paper's CPU figures for the same shapes (M items/s; AMD Milan / Intel
# Cascade Lake), quoted as context only.
PAPER_ONETOMANY = {
    "Rslm1": {"contiguous": (388.31, 233.57), "largepool": (175.06, 153.24)},
    "Rslm2": {"contiguous": (225.47, 168.78), "largepool": (103.29, 80.15)},
    "Rslm3": {"contiguous": (58.49, 41.60), "largepool": (38.13, 21.53)},
    "Rslm4": {"contiguous": (151.61, 93.68), "largepool": (55.88, 43.33)},
    "Rslm4Lite": {"contiguous": (137.43, 104.98), "largepool": (105.58, 61.46)},
}
PAPER_COMPRESS_2049 = 0.128   # M items/s, Rslm4 on AMD Milan


def run_onetomany(args):
    """The paper's codec microbenchmarks on one GPU.  OneToMany: one rotated
    query scored against 16,777,216 packed records of D = 256 (codes + 2-byte
    UE7M9 suffix; Rslm4Lite: ceil(D/2) bytes with the scale embedded), either
    contiguous or gathered at uniformly random positions of a pool of
    134,217,728 records ("LargePool 128M").  Records are real encodings of
    isotropic Gaussian unit vectors, encoded block by block.  Compress: Rslm4
    encoding (rotation, Lloyd-Max codes, norm correction, packed records) of
    1,048,576 device-resident vectors of D = 2049 (block-wise cascaded FWHT
    with an overlap block)."""
    import torch

    import synth
    import paper_2608_30384_amd as R

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    D, POOL, N = 256, 1 << 27, 1 << 24
    BLK = synth.TORCH_BLOCK
    reps = 10
    t_setup = time.time()
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    ids = torch.randint(0, POOL, (N,), generator=gen, device=dev, dtype=torch.int64)
    q = torch.from_numpy(synth.aniso(1, D, alpha=0.0, seed=77, normalize=True)).to(dev)
    xb = torch.empty((BLK, D), dtype=torch.float32, device=dev)
    codecs = [("Rslm1", 1, False), ("Rslm2", 2, False), ("Rslm3", 3, False), ("Rslm4", 4, False),
              ("Rslm4Lite", 4, True)]
    res = {}

    def timed(fn):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3
    for name, bits, lite in codecs:
        plan = R.Plan(D, bits, passes=-1, scale_mode="local", lite=lite)
        rb = plan.record_bytes
        pool = torch.empty((POOL, rb), dtype=torch.uint8, device=dev)
        tiles = torch.empty(plan.code_bytes(BLK), dtype=torch.uint8, device=dev)
        sc = torch.empty(BLK, dtype=torch.int32, device=dev)
        for b in range(POOL // BLK):
            synth.aniso_torch_block(b, D, alpha=0.0, seed=100, normalize=True, out=xb)
            R.rslm_encode(plan, xb, tiles, sc)
            pool[b * BLK:(b + 1) * BLK] = R.rslm_pack_records(plan, tiles, sc, BLK)
        del tiles, sc
        qrot = R.rslm_fwht(plan, q)
        out = torch.empty((1, N), dtype=torch.float32, device=dev)
        t_c = timed(lambda: R.rslm_score(plan, pool, qrot, n=N, out=out))
        t_g = timed(lambda: R.rslm_score(plan, pool, qrot, ids=ids, out=out))
        # 128-byte lines a gathered record touches, on average
        off = (ids[: 1 << 20] * rb) % 128
        lines = float(((off + rb + 127) // 128).float().mean().item())
        res[name] = {
            "record_bytes": rb,
            "contiguous": {"M_items_per_s": N / t_c / 1e6, "GBps": N * rb / t_c / 1e9,
                           "paper_M_items_per_s_milan_cascadelake":
                               PAPER_ONETOMANY[name]["contiguous"]},
            "largepool": {"M_items_per_s": N / t_g / 1e6, "record_GBps": N * rb / t_g / 1e9,
                          "lines_per_record": lines,
                          "line_GBps": N * lines * 128 / t_g / 1e9,
                          "paper_M_items_per_s_milan_cascadelake":
                              PAPER_ONETOMANY[name]["largepool"]},
        }
        log(f"{name}: {res[name]}")
        del pool, out
        torch.cuda.empty_cache()
    del xb
    # compress at D = 2049
    D2, n2 = 2049, 1 << 20
    plan = R.Plan(D2, 4, passes=-1, scale_mode="local")
    x2 = synth.aniso_torch(n2, D2, alpha=0.0, seed=5, normalize=True, device=dev)
    tiles = torch.empty(plan.code_bytes(n2), dtype=torch.uint8, device=dev)
    sc = torch.empty(n2, dtype=torch.int32, device=dev)

    def compress():
        R.rslm_encode(plan, x2, tiles, sc)
        R.rslm_pack_records(plan, tiles, sc, n2)
    t_e = timed(compress)
    out = {
        "metric": "OneToMany scored items/s (D = 256) and Rslm4 compress items/s (D = 2049), 1 GPU",
        "value": res["Rslm4"]["contiguous"]["M_items_per_s"] * 1e6, "unit": "items/s",
        "n_gpus": 1, "higher_is_better": True, "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": ("codec microbenchmarks: one query vs 16,777,216 packed D=256 "
                                "records, contiguous and gathered from a 134,217,728-record pool; "
                                "Rslm4 compress of 1,048,576 vectors at D=2049"),
                   "dim": D, "pool": POOL, "n": N, "queries": 1},
        "onetomany": res,
        "compress_2049": {"codec": "Rslm4", "vectors": n2, "ms": t_e * 1e3,
                          "M_items_per_s": n2 / t_e / 1e6,
                          "paper_M_items_per_s_milan": PAPER_COMPRESS_2049,
                          "GBps": n2 * (4 * D2 + plan.record_bytes) / t_e / 1e9},
        "setup_s": time.time() - t_setup,
        "kernel_sources": csrc_hash(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
