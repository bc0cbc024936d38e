"""Summaries of rocprofv3 CSV output for the GSQ kernels (kept short, as text, under profiles/).

    python -m paper_2604_18556_amd.rocprof_summary stats  STATS_CSV  --cmd "..." > out.txt
    python -m paper_2604_18556_amd.rocprof_summary pmc    COUNTER_CSV [...] --cmd "..." > out.txt
    python -m paper_2604_18556_amd.rocprof_summary traffic --fetch F.csv --write W.csv \
        --copy-fetch CF.csv --copy-write CW.csv --copy-bytes N --kernel backward \
        --workload NAME --cmd "..." [--json profiles/traffic.json] > out.txt
    python -m paper_2604_18556_amd.rocprof_summary mfma COUNTER_CSV --agent AGENT_CSV --cmd "..."

FETCH_SIZE and WRITE_SIZE are in KiB per dispatch.  ``traffic`` scales each by the ratio of
the known byte count of a plain device copy (bench.py --copy-calibration) to what the same
counter reports for that copy, and records the HBM bytes per launch of one GSQ kernel,
together with the SHA-256 of the kernel's source file, into a JSON file that bench.py reads
(it reports the traffic only while the source is unchanged).

``mfma`` reads one counter pass holding SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16 and
GRBM_GUI_ACTIVE, and gives for the contraction: the clock while the GPU is active
(GRBM_GUI_ACTIVE per XCC over the dispatch time), the share of those cycles the matrix cores
are busy (rocprofv3's MfmaUtil), the bf16 flops (512 per MOPS unit) and the rate they make.
Contractions dispatched after the first harden kernel are gsq_harden's hard-loss ones and are
listed apart from the step's.
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


def per_kernel_counters(path, steps_only=False):
    """{(kernel, counter): (mean per dispatch, dispatches)}.  With steps_only, only the dispatches
    before the first harden kernel count: the optimisation steps, not gsq_harden's hard-loss
    contractions."""
    rows = list(csv.DictReader(open(path)))
    cut = float("inf")
    if steps_only:
        cut = min((int(r["Dispatch_Id"]) for r in rows if short(r["Kernel_Name"]) == "harden"),
                  default=float("inf"))
    agg = collections.defaultdict(list)
    for r in rows:
        if int(r["Dispatch_Id"]) < cut:
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


PEAK_BF16_TFLOPS, NOMINAL_GHZ = 2500.0, 2.4   # MI355X dense bf16 matrix peak and its clock


def gpu_agent(path):
    for r in csv.DictReader(open(path)):
        if r["Agent_Type"] == "GPU":
            return int(r["Num_Xcc"]), int(r["Simd_Count"])
    raise SystemExit(f"no GPU agent in {path}")


def median(v):
    v = sorted(v)
    n = len(v)
    return v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2])


def cmd_mfma(a):
    n_xcc, n_simd = gpu_agent(a.agent)
    per, meta = collections.defaultdict(dict), {}
    for r in csv.DictReader(open(a.csv)):
        d = int(r["Dispatch_Id"])
        per[d][r["Counter_Name"]] = float(r["Counter_Value"])
        meta[d] = (short(r["Kernel_Name"]),
                   (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    first_harden = min((d for d, (k, _) in meta.items() if k == "harden"), default=float("inf"))
    groups = collections.defaultdict(list)
    for d, (k, t) in sorted(meta.items()):
        if k == "contract" or "k_contract_fixup" in k:
            groups[(k if k == "contract" else "fixup", "step" if d < first_harden else "hard loss")].append(d)
    print(f"# rocprofv3 MFMA counters of the contraction, median over dispatches\n# command: {a.cmd}\n"
          f"# GPU: {n_xcc} XCCs, {n_simd} SIMDs; peak {PEAK_BF16_TFLOPS:.0f} TFLOP/s bf16 at "
          f"{NOMINAL_GHZ} GHz\n")
    print(f"{'kernel':<10} {'calls':<10} {'n':>3} {'us':>9} {'clock_GHz':>10} {'mfma_busy':>10} "
          f"{'GFLOP':>9} {'TFLOP/s':>8} {'frac':>6} {'frac@clock':>10} {'lds_conflict':>12}")
    for (k, kind), ds in sorted(groups.items()):
        us = median([meta[d][1] * 1e6 for d in ds])
        if k == "fixup":
            print(f"{k:<10} {kind:<10} {len(ds):>3} {us:>9.1f}")
            continue
        ghz = median([per[d]["GRBM_GUI_ACTIVE"] / n_xcc / meta[d][1] / 1e9 for d in ds])
        busy = median([per[d]["SQ_VALU_MFMA_BUSY_CYCLES"] / (per[d]["GRBM_GUI_ACTIVE"] / n_xcc * n_simd)
                       for d in ds])
        gf = median([per[d]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 / 1e9 for d in ds])
        tf = median([per[d]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 / meta[d][1] / 1e12 for d in ds])
        conf = median([per[d].get("SQ_LDS_BANK_CONFLICT", float("nan")) for d in ds])
        print(f"{k:<10} {kind:<10} {len(ds):>3} {us:>9.1f} {ghz:>10.3f} {busy:>10.3f} {gf:>9.1f} "
              f"{tf:>8.0f} {tf / PEAK_BF16_TFLOPS:>6.3f} {tf / (PEAK_BF16_TFLOPS * ghz / NOMINAL_GHZ):>10.3f} "
              f"{conf:>12.0f}")
    print("\nclock_GHz: GRBM_GUI_ACTIVE per XCC / dispatch time.  mfma_busy: SQ_VALU_MFMA_BUSY_CYCLES / "
          "(active cycles x SIMDs) (rocprofv3 MfmaUtil).\nfrac: of the nominal peak; frac@clock: of the "
          "peak at the measured clock.  lds_conflict: SQ_LDS_BANK_CONFLICT cycles per dispatch.")


def cmd_traffic(a):
    f = per_kernel_counters(a.fetch, steps_only=True)
    w = per_kernel_counters(a.write, steps_only=True)
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
    print(f"# HBM traffic of one {a.kernel} launch of the optimisation steps, workload {a.workload}"
          f"\n# command: {a.cmd}\n")
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


def cmd_l2(a):
    """L2 (TCC) hit rate and the bytes read past the L2 (TCC_EA0_RDREQ_DRAM_32B x 32) per step
    dispatch of the step kernels, beside the algorithmic R + H bytes of the contraction."""
    c = per_kernel_counters(a.csv, steps_only=True)
    print(f"# L2 counters per step dispatch\n# command: {a.cmd}\n")
    print(f"{'kernel':<10} {'L2 hit':>7} {'requests':>12} {'read past L2 MB':>16}")
    for k in ("contract", "backward"):
        if (k, "TCC_HIT_sum") not in c:
            continue
        hit, miss = c[(k, "TCC_HIT_sum")][0], c[(k, "TCC_MISS_sum")][0]
        rd = c[(k, "TCC_EA0_RDREQ_DRAM_32B_sum")][0] * 32
        print(f"{k:<10} {hit / (hit + miss):>7.3f} {hit + miss:>12.4g} {rd / 1e6:>16.1f}")
    if a.rh_bytes:
        print(f"\ncontraction operands R + H: {a.rh_bytes / 1e6:.1f} MB per step")


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--cmd", default="")
    p = sub.add_parser("pmc")
    p.add_argument("csv", nargs="+")
    p.add_argument("--cmd", default="")
    m = sub.add_parser("mfma")
    m.add_argument("csv")
    m.add_argument("--agent", required=True)
    m.add_argument("--cmd", default="")
    l2 = sub.add_parser("l2")
    l2.add_argument("csv")
    l2.add_argument("--rh-bytes", type=float, default=0.0)
    l2.add_argument("--cmd", default="")
    t = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy_fetch", "copy_write", "kernel", "workload"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--json")
    t.add_argument("--cmd", default="")
    a = ap.parse_args(argv)
    {"stats": cmd_stats, "pmc": cmd_pmc, "mfma": cmd_mfma, "traffic": cmd_traffic,
     "l2": cmd_l2}[a.what](a)


if __name__ == "__main__":
    sys.exit(main())
