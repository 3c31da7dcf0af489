"""Turns rocprofv3 output into the short summaries kept under profiles/.

  kernels <stats.csv> <title> <command> [note]
      --kernel-trace --stats CSV -> markdown table of per-kernel times.
  by_grid <kernel_trace.csv> <name-substring,...>
      --kernel-trace CSV -> markdown rows of median / min time per (kernel,
      workgroups launched), for runs whose calls of one kernel differ in size.
  traffic <F.csv> <W.csv> <CF.csv> <CW.csv> <kernel-substring> <name> <workload> <source_hash>
      two --pmc runs (FETCH_SIZE, WRITE_SIZE) of a workload and the same two
      of the 256 MiB device copy (bench.py --calibrate-copy) -> the JSON
      record bench.py reads (HBM bytes per launch of one kernel, each
      counter scaled by what it reads for the copy).
"""
import csv
import json
import sys

COPY_KIB = 256 * 1024  # the calibration copy moves 256 MiB each way


def short_name(name: str) -> str:
    name = name.replace("void ", "").replace("hstu::(anonymous namespace)::", "")
    return name.split("(")[0]


def kernels(csv_path: str, title: str, command: str, note: str = "") -> str:
    rows = list(csv.DictReader(open(csv_path)))
    out = [f"# {title}", "", "Command (on the GPU host, from /tmp with TMPDIR=/tmp):", "", "```",
           command, "```", ""]
    if note:
        out += [note, ""]
    out += ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def by_grid(trace_csv: str, subs: str) -> str:
    groups = {}
    for r in csv.DictReader(open(trace_csv)):
        name = short_name(r["Kernel_Name"])
        if not any(x in name for x in subs.split(",")):
            continue
        wg = int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"])
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups.setdefault((name, wg), []).append(us)
    out = ["| kernel | workgroups | launches | median us | min us |", "|---|---|---|---|---|"]
    for (name, wg), v in sorted(groups.items()):
        v.sort()
        out.append(f"| `{name}` | {wg} | {len(v)} | {v[len(v) // 2]:.1f} | {v[0]:.1f} |")
    return "\n".join(out) + "\n"


def _mean_kib(path: str, counter: str, kernel_sub: str) -> float:
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path))
            if r["Counter_Name"] == counter and kernel_sub in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no {counter} rows for {kernel_sub!r} in {path}")
    return sum(vals) / len(vals)


def traffic(f_csv, w_csv, cf_csv, cw_csv, kernel_sub, name, workload, source_hash) -> str:
    fetch = _mean_kib(f_csv, "FETCH_SIZE", kernel_sub)
    write = _mean_kib(w_csv, "WRITE_SIZE", kernel_sub)
    ff = COPY_KIB / _mean_kib(cf_csv, "FETCH_SIZE", "copyBuffer")
    wf = COPY_KIB / _mean_kib(cw_csv, "WRITE_SIZE", "copyBuffer")
    rec = {"kernel": name, "workload": workload, "source_hash": source_hash,
           "fetch_kib": fetch, "write_kib": write, "fetch_factor": ff, "write_factor": wf,
           "hbm_bytes_per_launch": (fetch * ff + write * wf) * 1024.0,
           "summary": f"profiles/traffic_{workload}.md"}
    return json.dumps(rec, indent=1) + "\n"


if __name__ == "__main__":
    cmd, args = sys.argv[1], sys.argv[2:]
    print({"kernels": kernels, "traffic": traffic, "by_grid": by_grid}[cmd](*args), end="")
