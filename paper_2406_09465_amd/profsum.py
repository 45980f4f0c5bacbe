"""Summarizes rocprofv3 outputs into the short text files kept under profiles/.

  python -m paper_2406_09465_amd.profsum stats <rocprof dir> <out.md> --cmd "<command>"
      kernel-trace statistics (*_kernel_stats.csv) as a markdown table.

  python -m paper_2406_09465_amd.profsum counters <pmc dir>... --out <out.md> --cmd "<command>"...
      MFMA / LDS counters (SQ_VALU_MFMA_BUSY_CYCLES, SQ_LDS_BANK_CONFLICT, ...)
      of a plan's kernels with the derived utilisations.

  python -m paper_2406_09465_amd.profsum pmc --workload mlp --fetch <dir> --write <dir>
         --calib-mib 256 --out profiles/pmc_traffic.json --cmd-fetch "..." --cmd-write "..."
      FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of every kernel of the
      workload's fused plan, each scaled by the ratio between the known bytes of
      a plain streaming kernel (dst = src + 1 over calib-mib MiB, uint8) and
      what the same counter reads for it; records the generated source's hash
      so a stale figure is never reported for a changed kernel.
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics


def _rows(d, pattern):
    out = []
    for f in glob.glob(os.path.join(d, "**", pattern), recursive=True):
        out.extend(csv.DictReader(open(f)))
    return out


def stats(args):
    rows = _rows(args.dir, "*_kernel_stats.csv")
    lines = [f"# {args.title or os.path.basename(args.out)}", "", "Command:", "", "```", args.cmd, "```", "",
             "| kernel | calls | average (us) | min (us) | max (us) | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['Name']} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                     f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f}% |")
    open(args.out, "w").write("\n".join(lines) + "\n")


def _counter(d, name):
    per = {}
    for r in _rows(d, "*counter_collection.csv"):
        if r.get("Counter_Name") != name:
            continue
        per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: statistics.median(v) for k, v in per.items()}


def pmc(args):
    from . import graphs
    fetch = _counter(args.fetch, "FETCH_SIZE")
    write = _counter(args.write, "WRITE_SIZE")
    calib = [k for k in fetch if "elementwise" in k and fetch[k] > 1000]
    if not calib:
        raise SystemExit("no calibration kernel found")
    ck = max(calib, key=lambda k: fetch[k])
    known_kib = args.calib_mib * 1024.0
    f_fetch = known_kib / fetch[ck]
    f_write = known_kib / write[ck]
    w = graphs.build(args.workload)
    if args.bench_json:
        # the plan bench.py ran (e.g. the measured-cost choice), by node names
        d = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
        w, ks = graphs.plan_from_record(w, d["chosen_plan"])
        p = graphs.Plan(w.graph, ks)
    else:
        p = w.plan(args.plan)
    p.compile()
    res = {"workload": args.workload, "plan": args.plan, "calibration_kernel": ck[:80],
           "fetch_factor": f_fetch, "write_factor": f_write, "cmd_fetch": args.cmd_fetch, "cmd_write": args.cmd_write,
           "kernels": {}}
    old = {}
    if os.path.exists(args.out):
        old = json.load(open(args.out)).get("kernels", {})
    for k in range(p.num_kernels()):
        name = p.kernel_name(k)
        if name not in fetch or name not in write:
            continue
        fam, ab, af = p.kernel_info(k)
        h = hashlib.sha256(p.kernel_source(k).encode()).hexdigest()[:16]
        hbm = (fetch[name] * f_fetch + write[name] * f_write) * 1024.0
        res["kernels"][f"{args.workload}/{name}"] = {
            "workload": args.workload, "family": fam, "source_hash": h, "fetch_kib": fetch[name],
            "write_kib": write[name], "hbm_bytes_per_launch": hbm, "alg_bytes": ab,
            "traffic_over_alg": hbm / ab if ab else None}
    for k, v in old.items():  # keep other workloads' records
        if v.get("workload") != args.workload:
            res["kernels"].setdefault(k, v)
    json.dump(res, open(args.out, "w"), indent=1)
    md = os.path.splitext(args.out)[0] + ".md"
    lines = ["# HBM traffic per launch (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             f"Calibration: `{res['calibration_kernel'][:60]}` over {args.calib_mib} MiB (uint8, dst = src + 1) reads "
             f"FETCH_SIZE x {f_fetch:.3f} and WRITE_SIZE x {f_write:.3f} of the known bytes; every figure below "
             "is scaled by those factors.", "", "Commands (run once per workload `<w>`):", "", "```",
             args.cmd_fetch, args.cmd_write, "```", "",
             "| kernel | family | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes | algorithmic bytes | ratio | source hash |",
             "|---|---|---|---|---|---|---|---|"]
    for k, v in sorted(res["kernels"].items()):
        lines.append(f"| {k} | {v['family']} | {v['fetch_kib']:.0f} | {v['write_kib']:.0f} | "
                     f"{v['hbm_bytes_per_launch']:.0f} | {v['alg_bytes']:.0f} | {v['traffic_over_alg']:.3f} | "
                     f"{v['source_hash']} |")
    open(md, "w").write("\n".join(lines) + "\n")


def _dispatches(d):
    """{(dispatch id, kernel name): {counter: value, "_ns": duration}} of a --pmc run."""
    out = {}
    for r in _rows(d, "*counter_collection.csv"):
        k = (r["Dispatch_Id"], r["Kernel_Name"])
        e = out.setdefault(k, {})
        e[r["Counter_Name"]] = float(r["Counter_Value"])
        e["_ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    return out


def counters(args):
    """MFMA and LDS counters of a plan's kernels (medians over dispatches) from
    --pmc runs, with the derived utilisations.  SQ counters are totals over
    the whole GPU; SQ_VALU_MFMA_BUSY_CYCLES counts 16 cycles per 16x16x32 MFMA
    on its SIMD; GRBM_GUI_ACTIVE sums the busy cycles of the 8 XCDs."""
    per = {}
    for d in args.dirs:
        for (_, name), e in _dispatches(d).items():
            if not name.startswith(args.prefix):
                continue
            for c, v in e.items():
                per.setdefault(name, {}).setdefault(c, []).append(v)
    med = {k: {c: statistics.median(v) for c, v in cs.items()} for k, cs in per.items()}
    lines = [f"# {args.title}", "", "Commands (one rocprofv3 pass per counter group):", "", "```"] + args.cmd + ["```", "",
             f"Medians over the dispatches of each kernel (durations are those under counter collection, longer "
             f"than in the timed bench).  `MFMA busy` = SQ_VALU_MFMA_BUSY_CYCLES / ({args.simds} SIMDs x "
             f"{args.ghz} GHz x duration), the matrix cores' busy fraction against the nominal clock of the "
             "published peak; `MFMA TFLOP/s` = SQ_INSTS_VALU_MFMA_MOPS_F16 (+ _BF16) x 512 / duration.  `LDS "
             "conflict` = SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS (stall cycles per LDS-instruction cycle).  `wait "
             "LDS`, `wait any`, `VALU active` = SQ_WAIT_INST_LDS, SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_VALU / "
             "SQ_WAVE_CYCLES (shares of the waves' lifetime).", ""]
    cols = ["kernel", "duration us", "MFMA busy", "MFMA TFLOP/s", "LDS conflict", "wait LDS", "wait any",
            "VALU active"]
    lines += ["| " + " | ".join(cols) + " |", "|" + "---|" * len(cols)]
    for k in sorted(med):
        m = med[k]
        dur = m.get("_ns", 0.0) / 1e3
        busy = m.get("SQ_VALU_MFMA_BUSY_CYCLES")
        mops = m.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) + m.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        wave = m.get("SQ_WAVE_CYCLES")

        def f(x, fmt="{:.3f}"):
            return fmt.format(x) if x is not None else ""

        def share(c):
            return m[c] / wave if wave and c in m else None
        row = [k, f(dur, "{:.2f}"),
               f(busy / (args.simds * args.ghz * 1e3 * dur) if busy is not None and dur else None),
               f(mops * 512 / (dur * 1e-6) / 1e12 if mops and dur else None, "{:.0f}"),
               f(m["SQ_LDS_BANK_CONFLICT"] / m["SQ_ACTIVE_INST_LDS"] if m.get("SQ_ACTIVE_INST_LDS") else None),
               f(share("SQ_WAIT_INST_LDS")), f(share("SQ_WAIT_INST_ANY")), f(share("SQ_ACTIVE_INST_VALU"))]
        lines.append("| " + " | ".join(row) + " |")
    if any("TCP_TCC_READ_REQ" in m or "TCC_HIT" in m for m in med.values()):
        # memory-side counters: TCP counters sum over the compute units' L1s,
        # TCC over the L2 channels, GRBM_GUI_ACTIVE over the XCDs
        lines += ["", "Memory side: `L2 round trip` = TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ (clocks from an L1 "
                  "miss to its L2 answer, averaged over requests); `L1 pending stall` = TCP_PENDING_STALL_CYCLES / "
                  f"({args.cus} L1s x GRBM_GUI_ACTIVE / {args.xcds}), the share of the kernel's cycles an L1 could not "
                  "accept requests because too many were in flight; `L2 hit` = TCC_HIT / (TCC_HIT + TCC_MISS); "
                  "`L2 to memory` = TCC_EA0_RDREQ (read requests from L2 to the Infinity Fabric).", "",
                  "| kernel | L2 round trip (clk) | L1 pending stall | L2 hit | L2 to memory |", "|---|---|---|---|---|"]
        for k in sorted(med):
            m = med[k]
            gui = m.get("GRBM_GUI_ACTIVE")
            rt = m["TCP_TCC_READ_REQ_LATENCY"] / m["TCP_TCC_READ_REQ"] if m.get("TCP_TCC_READ_REQ") else None
            ps = (m["TCP_PENDING_STALL_CYCLES"] / (args.cus * gui / args.xcds)
                  if "TCP_PENDING_STALL_CYCLES" in m and gui else None)
            hit = m["TCC_HIT"] / (m["TCC_HIT"] + m["TCC_MISS"]) if m.get("TCC_HIT") is not None and "TCC_MISS" in m else None
            ea = m.get("TCC_EA0_RDREQ")
            lines.append("| " + " | ".join([k, "" if rt is None else f"{rt:.0f}", "" if ps is None else f"{ps:.3f}",
                                            "" if hit is None else f"{hit:.3f}", "" if ea is None else f"{ea:.0f}"]) + " |")
    lines += ["", "Raw medians:", "", "| kernel | counter | value |", "|---|---|---|"]
    for k in sorted(med):
        for c in sorted(med[k]):
            if c != "_ns":
                lines.append(f"| {k} | {c} | {med[k][c]:.0f} |")
    open(args.out, "w").write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("out")
    s.add_argument("--cmd", required=True)
    s.add_argument("--title", default="")
    p = sub.add_parser("pmc")
    p.add_argument("--workload", default="mlp")
    p.add_argument("--plan", default="fused")
    p.add_argument("--fetch", required=True)
    p.add_argument("--write", required=True)
    p.add_argument("--calib-mib", type=int, default=256)
    p.add_argument("--out", required=True)
    p.add_argument("--cmd-fetch", default="")
    p.add_argument("--cmd-write", default="")
    p.add_argument("--bench-json", default="", help="bench.py output line whose chosen_plan to use")
    c = sub.add_parser("counters")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--out", required=True)
    c.add_argument("--title", default="MFMA and LDS counters")
    c.add_argument("--prefix", default="korch_k")
    c.add_argument("--simds", type=int, default=1024)
    c.add_argument("--ghz", type=float, default=2.4)
    c.add_argument("--cus", type=int, default=256)
    c.add_argument("--xcds", type=int, default=8)
    c.add_argument("--cmd", action="append", default=[])
    a = ap.parse_args()
    {"stats": stats, "pmc": pmc, "counters": counters}[a.mode](a)


if __name__ == "__main__":
    main()
