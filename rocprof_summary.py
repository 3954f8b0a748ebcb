"""Writes the short text summaries under profiles/ from rocprofv3 result databases.

    python rocprof_summary.py trace DB --cmd CMD --title TITLE --out profiles/kernel_trace_X.md [--note NOTE]
    python rocprof_summary.py counters FETCH_DB WRITE_DB --cmd-template TMPL --title TITLE \\
        --name X --workload WORKLOAD --sources SRC...

`trace` reads a `rocprofv3 --kernel-trace --stats` database and tabulates calls,
mean / median / min duration, grid, block, LDS and registers per kernel.
`counters` reads two `rocprofv3 --pmc` databases (FETCH_SIZE, then WRITE_SIZE,
taken on a run that starts with a plain device copy of 256 MiB,
`bench.py --calib-copy-mib 256`) and writes profiles/counters_X.md and
profiles/traffic_X.json: per kernel the median counter per dispatch, scaled to
bytes by what the same counter reads for the copy (the largest copy dispatch
of the run), keyed by the library's stage names, with the sha256 of the
kernel sources the counters were taken on (bench.py reports the traffic as
unknown once those sources change).  Every kernel is mapped to its stage; an
unknown kernel name is an error.
"""
import argparse
import hashlib
import json
import os
import sqlite3
import statistics

ROOT = os.path.dirname(os.path.abspath(__file__))


def short(name):
    return name.split("(")[0].replace("void ", "").replace("gdn::", "")


def stage_of(kernel):
    """The library's stage name for a kernel (token path: wy, group_transfer,
    group_scan, chunk_states, output; frame-wise path: summaries, reduce, scan,
    output)."""
    k = short(kernel)
    if k.startswith("gdn_frame_summary"):          # gdn_frame_summary_kernel, fused variant too
        return "summaries"
    if k.startswith("gdn_frame_reduce"):
        return "reduce"
    if k.startswith("gdn_frame_scan"):
        return "scan"
    if k.startswith("gdn_frame_output"):           # gdn_frame_output_kernel, gdn_frame_output_fused_kernel
        return "output"
    if k.startswith("gdn_wy_kernel"):
        return "wy"
    if k.startswith("gdn_groupscan_kernel"):
        return "group_scan"
    if k.startswith("gdn_output_kernel"):
        return "output"
    if k.startswith("gdn_chunkscan_kernel"):
        args = [a.strip() for a in k.split("<", 1)[1].rstrip(">").split(",")]
        return "group_transfer" if args[3] == "0" else "chunk_states"
    raise ValueError(f"no stage for kernel {k!r}")


def kernel_rows(db):
    cur = sqlite3.connect(db).cursor()
    return cur.execute("select name, duration, grid_x, grid_y, workgroup_x, lds_size, vgpr_count, "
                       "accum_vgpr_count from kernels").fetchall()


def trace_md(db, cmd, title, note=""):
    by = {}
    for n, d, gx, gy, wx, lds, vg, ag in kernel_rows(db):
        by.setdefault(short(n), []).append((d, gx, gy, wx, lds, vg, ag))
    lines = [f"# {title}", "", "Command (from the repository root, on one MI355X):", "", "```", cmd, "```", "",
             "| kernel | stage | calls | avg (us) | median (us) | min (us) | grid (threads) | block | LDS (B) | "
             "arch VGPR | acc VGPR |", "|---|---|---|---|---|---|---|---|---|---|---|"]
    for n, v in sorted(by.items(), key=lambda kv: -sum(x[0] for x in kv[1])):
        if not n.startswith("gdn"):
            continue
        ds = [x[0] / 1e3 for x in v]
        x = v[0]
        lines.append(f"| `{n}` | {stage_of(n)} | {len(ds)} | {statistics.mean(ds):.2f} | "
                     f"{statistics.median(ds):.2f} | {min(ds):.2f} | ({x[1]},{x[2]}) | {x[3]} | {x[4]} | {x[5]} | "
                     f"{x[6]} |")
    return "\n".join(lines) + "\n" + (f"\n{note}\n" if note else "")


def pmc_medians(db):
    cur = sqlite3.connect(db).cursor()
    cols = [d[0] for d in cur.execute("select * from counters_collection limit 1").description]
    ci = {c: i for i, c in enumerate(cols)}
    per = {}
    for r in cur.execute("select * from counters_collection").fetchall():
        key = (short(r[ci["kernel_name"]]), r[ci["counter_name"]])
        per.setdefault(key, {}).setdefault(r[ci["dispatch_id"]], 0.0)
        per[key][r[ci["dispatch_id"]]] += r[ci["value"]]
    return {k: statistics.median(v.values()) for k, v in per.items()}


def copy_reading(db, counter):
    """The counter's value for the largest plain copy dispatch of the run."""
    cur = sqlite3.connect(db).cursor()
    cols = [d[0] for d in cur.execute("select * from counters_collection limit 1").description]
    ci = {c: i for i, c in enumerate(cols)}
    per = {}
    for r in cur.execute("select * from counters_collection").fetchall():
        if "copyBuffer" in r[ci["kernel_name"]] and r[ci["counter_name"]] == counter:
            per[r[ci["dispatch_id"]]] = per.get(r[ci["dispatch_id"]], 0.0) + r[ci["value"]]
    return max(per.values())


def counters(fetch_db, write_db, tmpl, title, workload, sources):
    f, w = pmc_medians(fetch_db), pmc_medians(write_db)
    copy_f, copy_w = copy_reading(fetch_db, "FETCH_SIZE"), copy_reading(write_db, "WRITE_SIZE")
    ff, wf = 262144.0 / copy_f, 262144.0 / copy_w           # 256 MiB in KiB
    cmds = [tmpl.format(counters="FETCH_SIZE"), tmpl.format(counters="WRITE_SIZE")]
    lines = [f"# {title}", "", "Each counter is its own run:", "", "```", *cmds, "```", "",
             f"Calibration: a plain 256 MiB device copy (the largest copy dispatch of the run) reads "
             f"FETCH_SIZE = {copy_f:.0f} KiB and WRITE_SIZE = {copy_w:.0f} KiB, so FETCH_SIZE is scaled by "
             f"{ff:.3f} and WRITE_SIZE by {wf:.3f}.", "",
             "| kernel | stage | FETCH_SIZE raw (KiB) | WRITE_SIZE raw (KiB) | read (MB) | written (MB) | total (MB) |",
             "|---|---|---|---|---|---|---|"]
    stages = {}
    total = 0.0
    for (k, c), v in sorted(f.items()):
        if not k.startswith("gdn"):
            continue
        wv = w.get((k, "WRITE_SIZE"), 0.0)
        rd, wr = v * ff * 1024, wv * wf * 1024
        st = stage_of(k)
        stages[st] = {"kernel": k, "fetch_kib_raw": v, "write_kib_raw": wv, "hbm_bytes_per_launch": rd + wr}
        total += rd + wr
        lines.append(f"| `{k}` | {st} | {v:.0f} | {wv:.0f} | {rd / 1e6:.1f} | {wr / 1e6:.1f} | "
                     f"{(rd + wr) / 1e6:.1f} |")
    lines += ["", f"Whole call (sum over the kernels): {total / 1e6:.1f} MB."]
    h = hashlib.sha256()
    for s in sources:
        h.update(open(os.path.join(ROOT, s), "rb").read())
    rec = {"workload": workload, "sources": list(sources), "source_sha256": h.hexdigest(),
           "fetch_scale": ff, "write_scale": wf, "commands": cmds, "stages": stages}
    return "\n".join(lines) + "\n", rec


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="what", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("--cmd", required=True)
    t.add_argument("--title", required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--note", default="")
    c = sub.add_parser("counters")
    c.add_argument("fetch_db")
    c.add_argument("write_db")
    c.add_argument("--cmd-template", required=True, help="the rocprofv3 command with {counters}")
    c.add_argument("--title", required=True)
    c.add_argument("--name", required=True)
    c.add_argument("--workload", required=True)
    c.add_argument("--sources", nargs="+", required=True)
    c.add_argument("--outdir", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args()
    if a.what == "trace":
        open(a.out, "w").write(trace_md(a.db, a.cmd, a.title, a.note))
    else:
        md, rec = counters(a.fetch_db, a.write_db, a.cmd_template, a.title, a.workload, a.sources)
        os.makedirs(a.outdir, exist_ok=True)
        open(os.path.join(a.outdir, f"counters_{a.name}.md"), "w").write(md)
        open(os.path.join(a.outdir, f"traffic_{a.name}.json"), "w").write(json.dumps(rec, indent=1) + "\n")


if __name__ == "__main__":
    main()
