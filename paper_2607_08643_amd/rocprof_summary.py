"""Short text summaries of rocprofv3 CSV output (kernel-trace statistics and
per-dispatch counter values), for the figures kept under profiles/.

  python -m paper_2607_08643_amd.rocprof_summary stats DIR [NAME_SUBSTRING ...]
      mean / min / max duration and call count per kernel, from the
      *_kernel_stats.csv that `rocprofv3 --kernel-trace --stats
      --output-format csv` writes under DIR.

  python -m paper_2607_08643_amd.rocprof_summary trace DIR [NAME_SUBSTRING ...]
      the same per (kernel, grid size), from the per-dispatch
      *_kernel_trace.csv (one kernel launched with different grids, e.g. the
      projection groups of a block, is then told apart).

  python -m paper_2607_08643_amd.rocprof_summary counters DIR COUNTER NAME_SUBSTRING ...
      mean value of COUNTER per dispatch, per (kernel, grid size), from the
      *_counter_collection.csv that `rocprofv3 --pmc COUNTER
      --output-format csv` writes under DIR.

Only the standard library is used; nothing here touches a GPU.
"""
from __future__ import annotations

import collections
import csv
import glob
import os
import sys


def _find(d: str, suffix: str) -> list[str]:
    return sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))


def _col(header: list[str], *names: str) -> int:
    low = [h.strip().lower() for h in header]
    for n in names:
        if n.lower() in low:
            return low.index(n.lower())
    raise KeyError(f"none of {names} in {header}")


def stats(d: str, subs: list[str]) -> str:
    out = []
    for path in _find(d, "kernel_stats.csv"):
        with open(path, newline="") as f:
            rows = list(csv.reader(f))
        h, body = rows[0], rows[1:]
        i_n, i_c = _col(h, "Name"), _col(h, "Calls")
        i_avg, i_min, i_max = _col(h, "AverageNs"), _col(h, "MinNs"), _col(h, "MaxNs")
        i_tot = _col(h, "TotalDurationNs")
        out.append(f"# {os.path.basename(path)}")
        out.append("# calls  mean_us  min_us  max_us  total_us  kernel")
        for r in body:
            if subs and not any(s in r[i_n] for s in subs):
                continue
            out.append(f"{int(r[i_c]):6d} {float(r[i_avg]) / 1e3:8.2f} {float(r[i_min]) / 1e3:7.2f} "
                       f"{float(r[i_max]) / 1e3:7.2f} {float(r[i_tot]) / 1e3:9.1f}  {r[i_n][:110]}")
    return "\n".join(out)


def trace(d: str, subs: list[str]) -> str:
    out = []
    for path in _find(d, "kernel_trace.csv"):
        with open(path, newline="") as f:
            rows = list(csv.reader(f))
        h, body = rows[0], rows[1:]
        i_n = _col(h, "Kernel_Name", "kernel_name", "Name")
        i_s, i_e = _col(h, "Start_Timestamp", "start_timestamp"), _col(h, "End_Timestamp", "end_timestamp")
        try:
            i_g = _col(h, "Grid_Size", "grid_size", "Grid_Size_X")
        except KeyError:
            i_g = None
        agg = collections.defaultdict(list)
        for r in body:
            if subs and not any(s in r[i_n] for s in subs):
                continue
            g = r[i_g] if i_g is not None else "?"
            agg[(r[i_n][:110], g)].append((int(r[i_e]) - int(r[i_s])) / 1e3)
        out.append(f"# {os.path.basename(path)}: duration per dispatch (us)")
        out.append("# dispatches  mean  min  max  grid_size  kernel")
        for (name, g), vs in sorted(agg.items()):
            out.append(f"{len(vs):6d} {sum(vs) / len(vs):8.2f} {min(vs):8.2f} {max(vs):8.2f} {g}  {name}")
    return "\n".join(out)


def counters(d: str, counter: str, subs: list[str]) -> str:
    out = []
    for path in _find(d, "counter_collection.csv"):
        with open(path, newline="") as f:
            rows = list(csv.reader(f))
        h, body = rows[0], rows[1:]
        i_n = _col(h, "Kernel_Name", "kernel_name", "Name")
        i_c = _col(h, "Counter_Name", "counter_name")
        i_v = _col(h, "Counter_Value", "counter_value", "Value")
        i_d = _col(h, "Dispatch_Id", "dispatch_id", "Correlation_Id")
        try:
            i_g = _col(h, "Grid_Size", "grid_size")
        except KeyError:
            i_g = None
        per = collections.defaultdict(float)   # (kernel, grid, dispatch) -> value summed over instances
        for r in body:
            if r[i_c].strip() != counter or not any(s in r[i_n] for s in subs):
                continue
            g = r[i_g] if i_g is not None else "?"
            per[(r[i_n][:110], g, r[i_d])] += float(r[i_v])
        agg = collections.defaultdict(list)
        for (name, g, _), v in per.items():
            agg[(name, g)].append(v)
        out.append(f"# {os.path.basename(path)}: {counter} per dispatch")
        out.append("# dispatches  mean  min  max  grid_size  kernel")
        for (name, g), vs in sorted(agg.items()):
            out.append(f"{len(vs):6d} {sum(vs) / len(vs):.6g} {min(vs):.6g} {max(vs):.6g} {g}  {name}")
    return "\n".join(out)


def main(argv: list[str]) -> int:
    if len(argv) >= 2 and argv[0] == "stats":
        print(stats(argv[1], argv[2:]))
        return 0
    if len(argv) >= 2 and argv[0] == "trace":
        print(trace(argv[1], argv[2:]))
        return 0
    if len(argv) >= 4 and argv[0] == "counters":
        print(counters(argv[1], argv[2], argv[3:]))
        return 0
    print(__doc__, file=sys.stderr)
    return 2


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
