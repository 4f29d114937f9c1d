"""Summaries of rocprofv3 output for the extend-attention kernel.

Turns the CSV files rocprofv3 writes (``--stats --output-format csv`` and
``--pmc ... --output-format csv``) into the short text summaries kept under
``profiles/``:

* ``stats``   -- per-kernel call count and average / total duration;
* ``traffic`` -- HBM bytes per extend launch from ``FETCH_SIZE`` and
  ``WRITE_SIZE`` (KiB per dispatch), each divided by what the same counter
  reads per byte for a plain copy kernel of known size run in the same
  process (bench.py ``--calibrate-copy-mib``);
* ``counters`` -- any other counters, averaged per dispatch.

The traffic summary carries the SHA-256 of the kernel sources it was taken
on; bench.py reports the figure only while the sources still match.

  python -m paper_2609_39819_amd.profiling stats CSV --cmd CMD --out FILE
  python -m paper_2609_39819_amd.profiling traffic --fetch CSV --write CSV --copy-mib N --cmd CMD --out FILE
  python -m paper_2609_39819_amd.profiling counters CSV... --cmd CMD --out FILE
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os
from typing import Dict, List

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXTEND_SOURCES = ("paper_2609_39819_amd/csrc/kvt_extend.hip", "paper_2609_39819_amd/csrc/kvt_device.h",
                  "paper_2609_39819_amd/csrc/kvt_internal.h")
DECODE_SOURCES = ("paper_2609_39819_amd/csrc/kvt_decode.hip", "paper_2609_39819_amd/csrc/kvt_device.h",
                  "paper_2609_39819_amd/csrc/kvt_internal.h")
APPEND_SOURCES = ("paper_2609_39819_amd/csrc/kvt_append.hip", "paper_2609_39819_amd/csrc/kvt_internal.h")
EXTEND_KERNEL = "extend_fwd_kernel"
DECODE_KERNEL = "decode_kernel"
APPEND_KERNEL = "append_kv_kernel"
COPY_KERNEL = "neg_kernel"
SOURCES = {EXTEND_KERNEL: EXTEND_SOURCES, DECODE_KERNEL: DECODE_SOURCES, APPEND_KERNEL: APPEND_SOURCES}
WHAT = {EXTEND_KERNEL: "extend", DECODE_KERNEL: "decode", APPEND_KERNEL: "append"}


def source_sha(paths=EXTEND_SOURCES) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def demangle(name: str) -> str:
    """Readable form of this library's kernel symbols (c++filt does not know
    the bf16 mangling DF16b)."""
    import re
    m = re.search(r"(extend_fwd_kernel|extend_combine_kernel|decode_kernel)I(DF16b|f)Li(\d+)E", name)
    if m:
        return f"{m.group(1)}<{'bf16' if m.group(2) == 'DF16b' else 'float'}, {m.group(3)}>"
    return name


def short_name(name: str) -> str:
    name = demangle(name)
    for key in ("extend_fwd_kernel", "extend_combine_kernel", "decode_kernel", "append_kv_kernel"):
        if key in name:
            tmpl = name[name.find(key):]
            return tmpl.split("(")[0].replace("kvt::(anonymous namespace)::", "")
    return name if len(name) < 70 else name[:67] + "..."


def per_dispatch(paths: List[str]) -> Dict[str, Dict[str, float]]:
    """Counter values averaged over the dispatches of each kernel (each file
    is one profiling pass; its counters are averaged over its own dispatches)."""
    out: Dict[str, Dict[str, float]] = collections.defaultdict(dict)
    for p in paths:
        sums: Dict[str, Dict[str, float]] = collections.defaultdict(lambda: collections.defaultdict(float))
        disp: Dict[str, set] = collections.defaultdict(set)
        with open(p) as f:
            for r in csv.DictReader(f):
                k = r["Kernel_Name"]
                sums[k][r["Counter_Name"]] += float(r["Counter_Value"])
                disp[k].add(r["Dispatch_Id"])
        for k, v in sums.items():
            for c, x in v.items():
                out[k][c] = x / len(disp[k])
    return out


def cmd_stats(args) -> str:
    rows = list(csv.DictReader(open(args.csv)))
    lines = [f"# Kernel time: {args.title}", "", f"Command: `{args.cmd}`", "",
             "| kernel | calls | avg (us) | min (us) | max (us) | total (ms) | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| {} | {} | {:.1f} | {:.1f} | {:.1f} | {:.3f} | {:.1f} |".format(
            short_name(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, float(r["TotalDurationNs"]) / 1e6, float(r["Percentage"])))
    return "\n".join(lines) + "\n"


def cmd_traffic(args) -> str:
    f = per_dispatch([args.fetch])
    w = per_dispatch([args.write])
    copy_bytes = args.copy_mib * 1024 * 1024

    def find(d, key):
        ks = [k for k in d if key in k]
        if not ks:
            raise SystemExit(f"no kernel matching {key!r} in the counter file")
        return d[ks[0]]

    fc = find(f, COPY_KERNEL)["FETCH_SIZE"] * 1024 / copy_bytes    # counter bytes per true byte
    wc = find(w, COPY_KERNEL)["WRITE_SIZE"] * 1024 / copy_bytes
    fe = find(f, args.kernel)["FETCH_SIZE"] * 1024 / fc
    we = find(w, args.kernel)["WRITE_SIZE"] * 1024 / wc
    what = WHAT[args.kernel]
    lines = [
        f"# HBM traffic per {what} launch: {args.title}", "",
        f"Command (FETCH_SIZE pass): `{args.cmd.replace('{C}', 'FETCH_SIZE')}`",
        f"Command (WRITE_SIZE pass): `{args.cmd.replace('{C}', 'WRITE_SIZE')}`", "",
        f"Calibration: a {args.copy_mib} MiB fp32 copy kernel (torch.neg) in the same process reads "
        f"FETCH_SIZE x{fc:.3f} and WRITE_SIZE x{wc:.3f} of its true bytes; the {what} figures are divided by those factors.",
        "",
        "| quantity | value |", "|---|---|",
        f"| fetch bytes per launch | {fe / 1e6:.1f} MB |",
        f"| write bytes per launch | {we / 1e6:.1f} MB |",
        (f"| algorithmic bytes per launch ({ALGO[what]}) | {args.algorithmic / 1e6:.1f} MB |"
         if args.algorithmic else ""),
        "",
        f"source_sha256: {source_sha(SOURCES[args.kernel])}",
        f"hbm_bytes_per_launch: {int(fe + we)}",
        f"fetch_bytes_per_launch: {int(fe)}",
        f"write_bytes_per_launch: {int(we)}",
    ]
    return "\n".join(l for l in lines if l is not None) + "\n"


ALGO = {"extend": "K/V once + Q + out", "decode": "K/V once + Q + out", "append": "new K/V read + written"}


def cmd_counters(args) -> str:
    d = per_dispatch(args.csv)
    lines = [f"# Counters per dispatch: {args.title}", "", f"Command: `{args.cmd}`", ""]
    for k, v in d.items():
        if args.kernel and args.kernel not in k:
            continue
        lines += [f"## {short_name(k)}", "", "| counter | per dispatch |", "|---|---|"]
        for c in sorted(v):
            lines.append(f"| {c} | {v[c]:.6g} |")
        lines.append("")
    return "\n".join(lines)


def read_traffic(path: str):
    """(source sha, HBM bytes per launch) from a traffic summary, or None."""
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.split(":")[0] in ("source_sha256", "hbm_bytes_per_launch"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if "source_sha256" not in vals or "hbm_bytes_per_launch" not in vals:
        return None
    return vals["source_sha256"], int(vals["hbm_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats"); s.add_argument("csv")
    t = sub.add_parser("traffic"); t.add_argument("--fetch", required=True); t.add_argument("--write", required=True)
    t.add_argument("--kernel", default=EXTEND_KERNEL, choices=sorted(SOURCES))
    t.add_argument("--copy-mib", type=int, required=True); t.add_argument("--algorithmic", type=float, default=0)
    c = sub.add_parser("counters"); c.add_argument("csv", nargs="+"); c.add_argument("--kernel", default=EXTEND_KERNEL)
    for p in (s, t, c):
        p.add_argument("--cmd", required=True); p.add_argument("--out", required=True)
        p.add_argument("--title", default="long ReAct turn (131072 reused + 2048 new tokens, Hq=96, Hkv=8, D=128, bf16)")
    args = ap.parse_args()
    text = {"stats": cmd_stats, "traffic": cmd_traffic, "counters": cmd_counters}[args.what](args)
    with open(args.out, "w") as f:
        f.write(text)
    print(text)


if __name__ == "__main__":
    main()
