"""Summaries of rocprofv3 CSV output for the GSQ kernels (kept short, as text, under profiles/).

    python -m paper_2604_18556_amd.rocprof_summary stats  STATS_CSV  --cmd "..." > out.txt
    python -m paper_2604_18556_amd.rocprof_summary pmc    COUNTER_CSV [...] --cmd "..." > out.txt
    python -m paper_2604_18556_amd.rocprof_summary traffic --fetch F.csv --write W.csv \
        --copy-fetch CF.csv --copy-write CW.csv --copy-bytes N --kernel backward \
        --workload NAME --cmd "..." [--json profiles/traffic.json] > out.txt

FETCH_SIZE and WRITE_SIZE are in KiB per dispatch.  ``traffic`` scales each by the ratio of
the known byte count of a plain device copy (bench.py --copy-calibration) to what the same
counter reports for that copy, and records the HBM bytes per launch of one GSQ kernel,
together with the SHA-256 of the kernel's source file, into a JSON file that bench.py reads
(it reports the traffic only while the source is unchanged).
"""
import argparse
import collections
import csv
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
KERNEL_MATCH = {  # short name -> (substring of the mangled / demangled kernel name, source file)
    "forward": ("k_forward", "gsq_elem.hip"),
    "backward": ("k_backward", "gsq_elem.hip"),
    "contract": ("k_contract_bf16", "gsq_contract.hip"),
    "contract_f32": ("k_contract_f32", "gsq_contract.hip"),
    "harden": ("k_harden", "gsq_elem.hip"),
}


def short(name):
    for k, (sub, _) in KERNEL_MATCH.items():
        if sub in name:
            return k
    return name[:70]


def per_kernel_counters(path):
    agg = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        agg[(short(r["Kernel_Name"]), r["Counter_Name"])].append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in agg.items()}


def cmd_stats(a):
    print(f"# rocprofv3 kernel statistics\n# command: {a.cmd}\n")
    print(f"{'kernel':<72} {'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'share%':>7}")
    for r in csv.DictReader(open(a.csv)):
        print(f"{short(r['Name']):<72} {int(r['Calls']):>6} {float(r['AverageNs']) / 1e3:>10.2f} "
              f"{float(r['MinNs']) / 1e3:>10.2f} {float(r['MaxNs']) / 1e3:>10.2f} "
              f"{float(r['Percentage']):>7.2f}")


def cmd_pmc(a):
    print(f"# rocprofv3 counters, average per dispatch\n# command: {a.cmd}\n")
    for path in a.csv:
        for (k, c), (v, n) in sorted(per_kernel_counters(path).items()):
            if k.startswith("__amd") or "at::native" in k or k.startswith("Cijk"):
                continue
            print(f"{k:<40} {c:<24} {v:>16.3f}  (n={n})")


def cmd_traffic(a):
    f = per_kernel_counters(a.fetch)
    w = per_kernel_counters(a.write)
    cf = per_kernel_counters(a.copy_fetch)
    cw = per_kernel_counters(a.copy_write)
    copy_kib = a.copy_bytes / 1024.0
    # the device-to-device copy of the calibration run is the runtime's copy kernel
    ck = [k for (k, c) in cf if "copyBuffer" in k][0]
    sf = copy_kib / cf[(ck, "FETCH_SIZE")][0]
    sw = copy_kib / cw[(ck, "WRITE_SIZE")][0]
    fk = f[(a.kernel, "FETCH_SIZE")][0] * sf * 1024
    wk = w[(a.kernel, "WRITE_SIZE")][0] * sw * 1024
    src = KERNEL_MATCH[a.kernel][1]
    sha = hashlib.sha256(open(os.path.join(PKG, "csrc", src), "rb").read()).hexdigest()
    print(f"# HBM traffic of one {a.kernel} launch, workload {a.workload}\n# command: {a.cmd}\n")
    print(f"copy calibration: {a.copy_bytes} bytes read and written; FETCH_SIZE scale {sf:.4f}, "
          f"WRITE_SIZE scale {sw:.4f}")
    print(f"{a.kernel}: FETCH_SIZE {f[(a.kernel, 'FETCH_SIZE')][0]:.1f} KiB/dispatch -> {fk / 1e6:.2f} MB")
    print(f"{a.kernel}: WRITE_SIZE {w[(a.kernel, 'WRITE_SIZE')][0]:.1f} KiB/dispatch -> {wk / 1e6:.2f} MB")
    print(f"{a.kernel}: traffic {(fk + wk) / 1e6:.2f} MB per launch; source {src} sha256 {sha[:16]}...")
    if a.json:
        data = json.load(open(a.json)) if os.path.exists(a.json) else {}
        data[f"{a.kernel}:{a.workload}"] = {"bytes_per_launch": fk + wk, "fetch_bytes": fk,
                                             "write_bytes": wk, "fetch_scale": sf, "write_scale": sw,
                                             "source": src, "source_sha256": sha, "command": a.cmd}
        json.dump(data, open(a.json, "w"), indent=1, sort_keys=True)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--cmd", default="")
    p = sub.add_parser("pmc")
    p.add_argument("csv", nargs="+")
    p.add_argument("--cmd", default="")
    t = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy_fetch", "copy_write", "kernel", "workload"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--json")
    t.add_argument("--cmd", default="")
    a = ap.parse_args(argv)
    {"stats": cmd_stats, "pmc": cmd_pmc, "traffic": cmd_traffic}[a.what](a)


if __name__ == "__main__":
    sys.exit(main())
