"""Text summaries of rocprofv3 runs of bench.py, for the profiles/ folder.

  python -m paper_1606_07822_amd.profile_summary stats STATS_CSV BENCH_JSON OUT_TXT --command CMD
      kernel table from `rocprofv3 --kernel-trace --stats` (run_kernel_stats.csv) next to the
      bench.py line of the same run.

  python -m paper_1606_07822_amd.profile_summary traffic FETCH_CSV WRITE_CSV BENCH_JSON OUT_JSON OUT_TXT
         --workload NAME --command-fetch CMD --command-write CMD [--sq SQ_CSV --command-sq CMD]
      HBM bytes of the training kernel from `rocprofv3 --pmc FETCH_SIZE` and `--pmc WRITE_SIZE`
      (run_counter_collection.csv, KiB per dispatch) of `bench.py --copy-calibration`. Each counter
      is scaled by what it reads for a dispatch of known size in the same run, made of the same
      per-lane dword row accesses as the training kernel: every row of a 1e6 x 320 float matrix
      written once (k_probe<3, ...>) for WRITE_SIZE, then read once (k_probe<2, ...>) for FETCH_SIZE.
      OUT_JSON carries the source hash of the training kernel; bench.py reports the traffic only
      while that hash matches.
"""
from __future__ import annotations

import argparse
import csv
import json
import os


def _hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ("train.hip", "w2v_internal.h"):
        with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _short(name: str) -> str:
    name = name.replace("w2v::(anonymous namespace)::", "")
    return name if len(name) <= 70 else name[:67] + "..."


def _bench_line(path: str) -> dict:
    with open(path) as fh:
        lines = [ln for ln in fh if ln.strip().startswith("{")]
    return json.loads(lines[-1])


def stats(args):
    rows = list(csv.DictReader(open(args.csv)))
    b = _bench_line(args.bench)
    title = args.title or f"{b['config']['workload']} (default bench)"
    out = [f"# rocprofv3 kernel statistics: {title}", "",
           "Command (repository root, MI355X):", f"  {args.command}", "",
           f"bench.py: --steps {b['steps']} --warmup {b['warmup']}; one step = {b['config']['step']}.", "",
           f"{'kernel':<72}{'calls':>6}{'total ms':>12}{'avg ms':>12}{'%':>7}"]
    for r in rows:
        out.append(f"{_short(r['Name']):<72}{int(r['Calls']):>6}{float(r['TotalDurationNs']) / 1e6:>12.2f}"
                   f"{float(r['AverageNs']) / 1e6:>12.3f}{float(r['Percentage']):>7.2f}")
    train = [r for r in rows if "k_train" in r["Name"] and "<" in r["Name"]]
    out += ["", "bench.py line of the same run (HIP events on the training kernel's stream):",
            f"  train_kernel_ms = {b['train_kernel_ms']:.1f}"
            + (f"  (rocprofv3 average of the training kernel above: {float(train[0]['AverageNs']) / 1e6:.1f})"
               if train else ""),
            f"  value = {b['value']:.4g} {b['unit']}, ms_per_step = {b['ms_per_step']:.1f}",
            f"  roofline = {json.dumps(b['roofline'])}"]
    if b.get("memory_probe"):
        out.append(f"  memory_probe = {json.dumps(b['memory_probe'])}")
    if b.get("cpu_baseline"):
        out.append(f"  cpu_baseline = {json.dumps(b['cpu_baseline'])}")
    with open(args.out, "w") as fh:
        fh.write("\n".join(out) + "\n")


def _dispatches(path: str) -> list[dict]:
    return list(csv.DictReader(open(path)))


def _train_row(rows):
    t = [r for r in rows if "k_train<" in r["Kernel_Name"]]
    if len(t) != 1:
        raise SystemExit(f"expected one training dispatch, found {len(t)}")
    return t[0]


def traffic(args):
    fr, wr = _dispatches(args.fetch), _dispatches(args.write)
    tf, tw = _train_row(fr), _train_row(wr)
    b = _bench_line(args.bench)
    cal = b.get("counter_calibration")
    if not cal:
        raise SystemExit("no counter_calibration in the bench line (run bench.py with --copy-calibration)")
    known = cal["rows"] * cal["row_bytes"]
    reads = [r for r in _dispatches(args.calib_fetch or args.fetch) if "k_probe<2," in r["Kernel_Name"]]
    writes = [r for r in wr if "k_probe<3," in r["Kernel_Name"]]
    if not reads or not writes:
        raise SystemExit("calibration dispatches k_probe<2> / k_probe<3> missing")
    read_factor = float(reads[-1]["Counter_Value"]) * 1024 / known
    write_factor = float(writes[-1]["Counter_Value"]) * 1024 / known
    f_kib, w_kib = float(tf["Counter_Value"]), float(tw["Counter_Value"])
    rd, wt = f_kib * 1024 / read_factor, w_kib * 1024 / write_factor
    ms = (int(tf["End_Timestamp"]) - int(tf["Start_Timestamp"])) / 1e6
    settings = {k: b["config"].get(k, 0) for k in ("cache_k", "flush_every", "flush_policy", "write_policy",
                                                   "cache_mode")}
    res = {"workload": args.workload, "kernel": tf["Kernel_Name"], "kernel_source": _hash(), "settings": settings,
           "fetch_kib_raw": f_kib, "write_kib_raw": w_kib, "read_factor": read_factor, "write_factor": write_factor,
           "hbm_read_bytes_per_launch": rd, "hbm_write_bytes_per_launch": wt, "hbm_bytes_per_launch": rd + wt,
           "kernel_ms_under_counters": ms}
    with open(args.out_json, "w") as fh:
        json.dump(res, fh, indent=1)
    alg = b.get("algorithmic_bytes_per_launch")
    out = [f"# rocprofv3 counters: k_train, {args.workload} (one launch)", "",
           "Commands (repository root, MI355X), one pass each:",
           f"  {args.command_fetch}", f"  {args.command_write}"]
    if args.sq:
        out.append(f"  {args.command_sq}")
    for c in args.command_tcc or []:
        out.append(f"  {c}")
    out += ["", f"kernel: {tf['Kernel_Name']}", f"  grid {tf['Grid_Size']} threads, workgroup {tf['Workgroup_Size']}, "
            f"arch VGPR {tf['VGPR_Count']}, LDS {tf['LDS_Block_Size']} B", f"  duration under counters: {ms:.1f} ms", "",
            "HBM bytes (fabric side of L2):",
            f"  FETCH_SIZE {f_kib:.4g} KiB raw; calibration: reading {known / 1e9:.3f} GB once (k_probe<2>) counts "
            f"{read_factor * known / 1024:.0f} KiB -> factor {read_factor:.3f}",
            f"  WRITE_SIZE {w_kib:.4g} KiB raw; calibration: writing {known / 1e9:.3f} GB once (k_probe<3>) counts "
            f"{write_factor * known / 1024:.0f} KiB -> factor {write_factor:.3f}",
            f"  read {rd / 1e12:.3f} TB + write {wt / 1e12:.3f} TB = {(rd + wt) / 1e12:.3f} TB per launch -> "
            f"{(rd + wt) / (ms / 1e3) / 1e12:.2f} TB/s"]
    if alg:
        out.append(f"  algorithmic bytes of the same launch (byte model): {alg / 1e12:.3f} TB")
    if args.sq:
        sq = [r for r in _dispatches(args.sq) if "k_train<" in r["Kernel_Name"]]
        vals = {r["Counter_Name"]: float(r["Counter_Value"]) for r in sq}
        out += ["", "SQ counters (sum over the device):"]
        out += [f"  {k:<22} {v:.4g}" for k, v in sorted(vals.items())]
        nodes = b.get("stats", {}).get("node_updates")
        if nodes and "SQ_INSTS_VALU" in vals:
            out.append(f"  VALU instructions per node update: {vals['SQ_INSTS_VALU'] / nodes:.1f} ({nodes:.4g} updates)")
        if "SQ_INSTS_LDS" in vals and vals["SQ_INSTS_LDS"] and "SQ_LDS_BANK_CONFLICT" in vals:
            out.append(f"  LDS bank conflicts per LDS instruction: "
                       f"{vals['SQ_LDS_BANK_CONFLICT'] / vals['SQ_INSTS_LDS']:.4f}")
    if args.tcc:
        vals = {}
        for f in args.tcc:
            vals.update({r["Counter_Name"]: float(r["Counter_Value"]) for r in _dispatches(f) if "k_train<" in r["Kernel_Name"]})
        out += ["", "L2 (TCC) counters (sum over the device):"]
        out += [f"  {k:<36} {v:.4g}" for k, v in sorted(vals.items())]
        if vals.get("TCC_HIT_sum") and vals.get("TCC_MISS_sum"):
            h, m = vals["TCC_HIT_sum"], vals["TCC_MISS_sum"]
            out.append(f"  L2 hit rate: {h / (h + m):.3f}")
        if vals.get("TCC_EA0_RDREQ_LEVEL_sum") and vals.get("TCC_EA0_RDREQ_sum"):
            out.append(f"  mean read latency past L2 (queue level / requests): "
                       f"{vals['TCC_EA0_RDREQ_LEVEL_sum'] / vals['TCC_EA0_RDREQ_sum']:.0f} cycles")
        if vals.get("TCC_EA0_WRREQ_LEVEL_sum") and vals.get("TCC_EA0_WRREQ_sum"):
            out.append(f"  mean write latency past L2: "
                       f"{vals['TCC_EA0_WRREQ_LEVEL_sum'] / vals['TCC_EA0_WRREQ_sum']:.0f} cycles")
    with open(args.out_txt, "w") as fh:
        fh.write("\n".join(out) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("bench")
    s.add_argument("out")
    s.add_argument("--command", required=True)
    s.add_argument("--title", default="")
    t = sub.add_parser("traffic")
    for a in ("fetch", "write", "bench", "out_json", "out_txt"):
        t.add_argument(a)
    t.add_argument("--workload", required=True)
    t.add_argument("--command-fetch", required=True)
    t.add_argument("--command-write", required=True)
    t.add_argument("--calib-fetch", help="FETCH_SIZE csv holding k_probe<2> if not FETCH_CSV")
    t.add_argument("--sq")
    t.add_argument("--command-sq", default="")
    t.add_argument("--tcc", action="append", help="L2 counter csv (repeatable)")
    t.add_argument("--command-tcc", action="append")
    args = ap.parse_args()
    stats(args) if args.cmd == "stats" else traffic(args)


if __name__ == "__main__":
    main()
