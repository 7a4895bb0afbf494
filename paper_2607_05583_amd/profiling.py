"""Short text summaries of rocprofv3 output for the ``profiles/`` folder.

rocprofv3 (ROCm 7) writes one SQLite database per run (``*_results.db``).  This
module reads the ``kernels`` and ``pmc_events`` views of such databases and
writes the few figures that the benchmark line cites:

  kernel-trace  per kernel name and grid size: launches, average / min / max
                duration (from ``rocprofv3 --kernel-trace --stats``);
  traffic       HBM bytes per launch of the single-pass forward kernel from a
                ``FETCH_SIZE`` run and a ``WRITE_SIZE`` run, each scaled by what the
                same counter reads for the runtime's plain buffer copy of known
                size in the same process (``bench.py --counters``);
  counters      every counter of several ``--pmc`` runs per dispatch of the
                kernels named (``bench.py --counters bwd|decode``).

Usage:
  python -m paper_2607_05583_amd.profiling kernel-trace DB_DIR OUT.md --command "..." \
      [--prefill-launches N]
  python -m paper_2607_05583_amd.profiling traffic FETCH_DIR WRITE_DIR OUT.json \
      --copy-bytes N --command "..."
  python -m paper_2607_05583_amd.profiling counters OUT.md DB_DIR [DB_DIR ...] \
      --kernels PATTERN[,PATTERN] --command "..."
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sqlite3

PKG = os.path.dirname(os.path.abspath(__file__))
FUSED = "fwd_stream_kernel"
COPY = "copyBuffer"


# the streaming forward kernel, its launcher and the entry point that sizes its grid
SEG_SOURCES = ("api.hip", "common.h", "fwd.hip", "stream.h", "tile_io.h")


def source_hash() -> str:
    """Hash of the sources the streaming forward kernel is built and launched from: a counter
    summary is valid only for the code it was taken on."""
    h = hashlib.sha256()
    csrc = os.path.join(PKG, "csrc")
    for f in SEG_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def _db(path: str) -> sqlite3.Connection:
    if os.path.isdir(path):
        fs = sorted(glob.glob(os.path.join(path, "**", "*_results.db"), recursive=True))
        if not fs:
            raise FileNotFoundError(f"no *_results.db under {path}")
        path = fs[0]
    return sqlite3.connect(path)


def short_name(name: str) -> str:
    n = name.split("(")[0]
    return n.replace("void ", "").strip()


def kernel_rows(db_path: str):
    cur = _db(db_path).cursor()
    q = ("select name, grid_x, workgroup_x, count(*), avg(duration), min(duration), max(duration), "
         "sum(duration) from kernels group by name, grid_x, workgroup_x order by sum(duration) desc")
    return [dict(name=r[0], grid=r[1], wg=r[2], calls=r[3], avg_us=r[4] / 1e3, min_us=r[5] / 1e3,
                 max_us=r[6] / 1e3, total_us=r[7] / 1e3) for r in cur.execute(q)]


def first_launches(db_path: str, pattern: str, n: int):
    """Durations (us) of the first n launches of the kernels matching pattern, in launch order."""
    cur = _db(db_path).cursor()
    q = "select duration from kernels where name like ? order by start limit ?"
    return [r[0] / 1e3 for r in cur.execute(q, (f"%{pattern}%", n))]


def write_kernel_trace(db_dir: str, out: str, command: str, top: int = 20, prefill_launches: int = 0):
    rows = kernel_rows(db_dir)
    tot = sum(r["total_us"] for r in rows)
    lines = ["# rocprofv3 kernel trace", "", "Command (from the repository root, on one MI355X):", "",
             "```", command, "```", "",
             "| kernel | grid (threads) | block | launches | avg us | min us | max us | total % |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        lines.append(f"| `{short_name(r['name'])}` | {r['grid']} | {r['wg']} | {r['calls']} | "
                     f"{r['avg_us']:.2f} | {r['min_us']:.2f} | {r['max_us']:.2f} | "
                     f"{100 * r['total_us'] / tot:.1f} |")
    lines.append("")
    if prefill_launches > 0:
        # the bench runs the prefill first: its warmup and timed launches are the
        # first ones of the forward kernel (later ones belong to other workloads)
        d = first_launches(db_dir, FUSED, prefill_launches)
        lines += [f"Prefill workload only (the first {len(d)} `{FUSED}` launches: warm-up and both timed loops of steps):",
                  "", "| launches | avg us | min us | max us |", "|---:|---:|---:|---:|",
                  f"| {len(d)} | {sum(d) / len(d):.2f} | {min(d):.2f} | {max(d):.2f} |", ""]
    with open(out, "w") as f:
        f.write("\n".join(lines))
    return rows


def _counter(db_dir: str, counter: str, pattern: str):
    cur = _db(db_dir).cursor()
    q = ("select dispatch_id, sum(counter_value) from pmc_events where counter_name = ? and name like ? "
         "group by dispatch_id order by dispatch_id")
    return [r[1] for r in cur.execute(q, (counter, f"%{pattern}%"))]


def write_traffic(fetch_dir: str, write_dir: str, out: str, command: str, copy_bytes: int):
    """FETCH_SIZE and WRITE_SIZE are in KiB per dispatch.  The copy moves copy_bytes in
    and copy_bytes out; the ratio of that to its counter reading is the scale applied
    to the forward kernel's readings."""
    fetch_copy = _counter(fetch_dir, "FETCH_SIZE", COPY)
    write_copy = _counter(write_dir, "WRITE_SIZE", COPY)
    fetch_fwd = _counter(fetch_dir, "FETCH_SIZE", FUSED)
    write_fwd = _counter(write_dir, "WRITE_SIZE", FUSED)
    if not (fetch_copy and write_copy and fetch_fwd and write_fwd):
        raise RuntimeError("counter rows missing for the copy or the forward kernel")
    # the largest copy dispatch is the calibration copy (smaller ones move inputs)
    fc, wc = max(fetch_copy), max(write_copy)
    f_scale = copy_bytes / (fc * 1024.0)
    w_scale = copy_bytes / (wc * 1024.0)
    # skip the first forward launch (it also faults in the workspace)
    ff = fetch_fwd[1:] if len(fetch_fwd) > 1 else fetch_fwd
    wf = write_fwd[1:] if len(write_fwd) > 1 else write_fwd
    fetch_b = sum(ff) / len(ff) * 1024.0 * f_scale
    write_b = sum(wf) / len(wf) * 1024.0 * w_scale
    res = {
        "kernel": FUSED,
        "workload": "prefill_bf16_B4_L32768_D256_M8",
        "command": command,
        "copy_bytes": copy_bytes,
        "copy_fetch_kib": fc, "copy_write_kib": wc,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "fwd_launches": len(ff),
        "fwd_fetch_kib_avg": sum(ff) / len(ff), "fwd_write_kib_avg": sum(wf) / len(wf),
        "fetch_bytes_per_launch": fetch_b, "write_bytes_per_launch": write_b,
        "bytes_per_launch": fetch_b + write_b,
        "source_hash": source_hash(),
    }
    with open(out, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    return res


def _all_counters(db_dir: str):
    """{kernel short name: {counter: average per dispatch}} (instances of a counter
    summed per dispatch) and {kernel: dispatches} of one --pmc run."""
    cur = _db(db_dir).cursor()
    q = ("select name, counter_name, dispatch_id, sum(counter_value) from pmc_events "
         "group by name, counter_name, dispatch_id")
    acc, disp = {}, {}
    for name, cn, did, v in cur.execute(q):
        k = short_name(name)
        acc.setdefault(k, {}).setdefault(cn, []).append(v)
        disp.setdefault(k, set()).add(did)
    return {k: {cn: sum(v) / len(v) for cn, v in d.items()} for k, d in acc.items()}, \
        {k: len(v) for k, v in disp.items()}


def write_counters(db_dirs, out: str, command: str, kernels, copy_bytes: int):
    """A table of every counter of the given --pmc runs, per dispatch of each kernel
    whose name contains one of the patterns; FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch) are also given in bytes, scaled by the same counters' reading for
    the runtime's buffer copy of copy_bytes in the same run."""
    rows, ndisp, scale = {}, {}, {}
    for d in db_dirs:
        c, n = _all_counters(d)
        for k, vals in c.items():
            if COPY in k:
                for cn in ("FETCH_SIZE", "WRITE_SIZE"):
                    if cn in vals:
                        scale[cn] = copy_bytes / (max(_counter(d, cn, COPY)) * 1024.0)
                continue
            if not any(p in k for p in kernels):
                continue
            rows.setdefault(k, {}).update(vals)
            ndisp[k] = max(ndisp.get(k, 0), n[k])
    names = sorted({cn for v in rows.values() for cn in v})
    lines = ["# rocprofv3 counters", "", "Commands (from the repository root, on one MI355X), one per counter set:",
             "", "```", command, "```", "",
             "Per dispatch, averaged over the dispatches of each kernel (instances of a counter summed). "
             "SQ cycle and busy counters are as the hardware reports them (summed over the shader engines).", "",
             "| kernel | dispatches | " + " | ".join(names) + " |",
             "|---|---:|" + "---:|" * len(names)]
    for k in sorted(rows):
        lines.append(f"| `{k}` | {ndisp[k]} | " + " | ".join(f"{rows[k].get(cn, float('nan')):.4g}" for cn in names)
                     + " |")
    if scale:
        lines += ["", "HBM bytes per dispatch (counter KiB x 1024 x the copy's scale: "
                  + ", ".join(f"{cn} {v:.3f}" for cn, v in sorted(scale.items())) + "):", "",
                  "| kernel | fetch MB | write MB |", "|---|---:|---:|"]
        for k in sorted(rows):
            f = rows[k].get("FETCH_SIZE", float("nan")) * 1024 * scale.get("FETCH_SIZE", float("nan")) / 1e6
            w = rows[k].get("WRITE_SIZE", float("nan")) * 1024 * scale.get("WRITE_SIZE", float("nan")) / 1e6
            lines.append(f"| `{k}` | {f:.2f} | {w:.2f} |")
    lines.append("")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    return rows


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("kernel-trace")
    a.add_argument("db_dir")
    a.add_argument("out")
    a.add_argument("--command", required=True)
    a.add_argument("--prefill-launches", type=int, default=0,
                   help="also summarise the first N launches of the forward kernel (the prefill)")
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("out")
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--command", required=True)
    c = sub.add_parser("counters")
    c.add_argument("out")
    c.add_argument("db_dirs", nargs="+")
    c.add_argument("--kernels", required=True, help="comma-separated name patterns")
    c.add_argument("--copy-bytes", type=int, default=256 << 20)
    c.add_argument("--command", required=True)
    args = ap.parse_args()
    if args.cmd == "counters":
        rows = write_counters(args.db_dirs, args.out, args.command, args.kernels.split(","), args.copy_bytes)
        for k, v in rows.items():
            print(k, {cn: round(x, 1) for cn, x in v.items()})
        return
    if args.cmd == "kernel-trace":
        for r in write_kernel_trace(args.db_dir, args.out, args.command,
                                    prefill_launches=args.prefill_launches)[:8]:
            print(f"{short_name(r['name'])[:60]:60s} grid {r['grid']:>8} n {r['calls']:>6} avg {r['avg_us']:.2f} us")
    else:
        print(json.dumps(write_traffic(args.fetch_dir, args.write_dir, args.out, args.command,
                                       args.copy_bytes), indent=1))


if __name__ == "__main__":
    main()
