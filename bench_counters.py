"""HBM traffic of bench.py's dominant kernel class from rocprofv3 counters.

Two subcommands:

  cast --n N
      Runs the library's fp32 -> bf16 cast once over N elements: a plain
      streaming kernel that reads exactly 4N and writes exactly 2N bytes.
      Profiled with --pmc FETCH_SIZE (then WRITE_SIZE), it calibrates what
      the counters read for a known number of bytes.

  summarize --class NAME --kernel PATTERN [...] --launches-per-step L
            --steps S --fetch CSV --write CSV --cal-fetch CSV --cal-write CSV
            --n N --sources FILE [...]
      Sums FETCH_SIZE / WRITE_SIZE (KiB per dispatch) over the dispatches whose
      kernel name contains one of the patterns, divides by the S profiled
      steps and the class's L launches per step, scales each by the cast's
      counter-to-byte factor, and records the result in profiles/counters.json
      under NAME together with a digest of the kernel sources (bench.py reports
      the figure only while the sources are unchanged).
"""

import argparse
import csv
import json
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def run_cast(n):
    import torch
    from paper_1904_10584_amd import binding as am
    src = torch.rand(n, dtype=torch.float32, device="cuda")
    dst = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    am.cast_f32_to_bf16(src, dst)
    torch.cuda.synchronize()
    print(f"cast of {n} elements: {4 * n} bytes read, {2 * n} bytes written", flush=True)


def counter_kib(path, counter, patterns):
    """Sum of `counter` over the dispatches whose kernel matches a pattern,
    and the number of such dispatches."""
    total, seen = 0.0, set()
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r.get("Counter_Name") != counter:
                continue
            name = r.get("Kernel_Name", "")
            if any(p in name for p in patterns):
                total += float(r["Counter_Value"])
                seen.add(r.get("Dispatch_Id"))
    return total, len(seen)


def summarize(a):
    from bench import kernel_sources_digest
    cal_f, nf = counter_kib(a.cal_fetch, "FETCH_SIZE", ["cast_kernel"])
    cal_w, nw = counter_kib(a.cal_write, "WRITE_SIZE", ["cast_kernel"])
    if nf != 1 or nw != 1:
        sys.exit(f"expected one cast dispatch per calibration run, got {nf} and {nw}")
    k_fetch = cal_f * 1024 / (4 * a.n)   # counter bytes per real byte read
    k_write = cal_w * 1024 / (2 * a.n)
    f, df = counter_kib(a.fetch, "FETCH_SIZE", a.kernel)
    w, dw = counter_kib(a.write, "WRITE_SIZE", a.kernel)
    launches = a.steps * a.launches_per_step
    fetch_b = f * 1024 / k_fetch / launches
    write_b = w * 1024 / k_write / launches
    path = os.path.join(ROOT, "profiles", "counters.json")
    table = json.load(open(path)) if os.path.exists(path) else {}
    table[a.cls] = {
        "kernels": a.kernel,
        "dispatches": [df, dw],
        "launches": launches,
        "fetch_bytes_per_launch": round(fetch_b),
        "write_bytes_per_launch": round(write_b),
        "hbm_bytes_per_launch": round(fetch_b + write_b),
        "calibration": {"kernel": "cast_kernel", "n": a.n,
                        "fetch_factor": round(k_fetch, 4), "write_factor": round(k_write, 4)},
        "sources": a.sources,
        "sources_sha": kernel_sources_digest(a.sources),
    }
    with open(path, "w") as fh:
        json.dump(table, fh, indent=1)
    print(json.dumps(table[a.cls]))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("cast")
    c.add_argument("--n", type=int, default=1 << 28)
    s = sub.add_parser("summarize")
    s.add_argument("--class", dest="cls", required=True)
    s.add_argument("--kernel", action="append", required=True)
    s.add_argument("--launches-per-step", type=int, required=True)
    s.add_argument("--steps", type=int, required=True)
    s.add_argument("--fetch", required=True)
    s.add_argument("--write", required=True)
    s.add_argument("--cal-fetch", required=True)
    s.add_argument("--cal-write", required=True)
    s.add_argument("--n", type=int, default=1 << 28)
    s.add_argument("--sources", nargs="+", required=True)
    a = ap.parse_args()
    if a.cmd == "cast":
        run_cast(a.n)
    else:
        summarize(a)


if __name__ == "__main__":
    main()
