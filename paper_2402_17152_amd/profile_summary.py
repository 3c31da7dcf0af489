"""Turns a rocprofv3 --stats kernel CSV into a short markdown table."""
import csv
import sys


def short_name(name: str) -> str:
    name = name.replace("void ", "").replace("hstu::(anonymous namespace)::", "")
    return name.split("(")[0]


def main(csv_path: str, title: str, command: str, note: str = "") -> str:
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


if __name__ == "__main__":
    print(main(*sys.argv[1:]), end="")
