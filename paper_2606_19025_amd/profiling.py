"""Summaries of rocprofv3 output for the kernels of the resident-expert layer.

Three summaries, written as short text files:

* ``kernel-stats``: the ``--kernel-trace --stats`` table (``*_kernel_stats.csv``)
  with every kernel symbol mapped to the name the library's own HIP-event
  timing uses (``moe_timing_collect``), so the two can be compared launch for
  launch.
* ``mfma``: the bf16 MFMA flops each GEMM launch executed and its MFMA busy
  share, from a ``--pmc MfmaFlopsBF16 MfmaUtil`` run, beside the algorithmic
  flops a bench.py run counts for the same launch.
* ``traffic``: HBM bytes per launch from two ``--pmc`` runs of the same
  command (``FETCH_SIZE``, then ``WRITE_SIZE``; both in KiB per dispatch).
  Each counter is scaled by the factor that makes it read exactly the known
  size of a plain device-to-device copy made in the same run (``bench.py
  --traffic-calibration`` copies ``CALIBRATION_BYTES``).  Every row carries
  the digest of the kernel's source file, so a reader (``bench.py``) can tell
  when the kernel has changed since the counters were taken.

    python -m paper_2606_19025_amd.profiling kernel-stats STATS_CSV OUT --command "..."
    python -m paper_2606_19025_amd.profiling traffic FETCH_CSV WRITE_CSV OUT --command "..."
    python -m paper_2606_19025_amd.profiling mfma COUNTERS_CSV BENCH_JSON OUT --command "..."
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")

CALIBRATION_BYTES = 1 << 30  # the plain copy bench.py makes for the counter scale

GEMM_KINDS = ["gemm_gu_fwd", "gemm_down_fwd", "gemm_dhh_bwd", "gemm_dx_bwd", "gemm_dwd",
              "gemm_dwgu", "gemm_up_fwd", "gemm_dh_bwd"]

# launches of two GEMM kinds (the backward's dHh with dW_d, dX with dW_gu)
_MERGED = {(2, 4): "gemm_dhh_dwd", (7, 4): "gemm_dh_dwd", (3, 5): "gemm_dx_dwgu"}


def _gemm_launch_name(ka: int, kb: int) -> str:
    return GEMM_KINDS[ka] if ka == kb else _MERGED.get((ka, kb), "gemm_merged")


# kernel symbol (demangled, as rocprofv3 prints it) -> timing name
_SYMBOLS = [
    (r"gemm_bf16_kernel(?:<|ILi)(\d)(?:, |ELi)(\d)", lambda m: _gemm_launch_name(int(m.group(1)), int(m.group(2)))),
    (r"gemm_bf16_kernel(?:<|ILi)(\d)", lambda m: GEMM_KINDS[int(m.group(1))]),
    (r"gemm_f32_kernel(?:<|ILi)(\d)", lambda m: GEMM_KINDS[int(m.group(1))]),
    (r"route_fwd_kernel", lambda m: "route_fwd"),
    (r"route_dz_kernel", lambda m: "route_dz"),
    (r"route_bwd_mfma_kernel", lambda m: "route_bwd_mfma"),
    (r"route_dw_partial_kernel", lambda m: "route_dw_partial"),
    (r"route_dw_reduce_kernel", lambda m: "route_dw_reduce"),
    (r"route_dx_kernel", lambda m: "route_dx"),
    (r"dispatch_count_kernel", lambda m: "dispatch_count"),
    (r"dispatch_scan_kernel", lambda m: "dispatch_scan"),
    (r"dispatch_scatter_kernel", lambda m: "dispatch_scatter"),
    (r"gather_rows_kernel", lambda m: "dispatch_gather"),
    (r"dispatch_place_kernel", lambda m: "dispatch_place"),
    (r"combine_fwd_kernel", lambda m: "combine_fwd"),
    (r"combine_bwd_kernel", lambda m: "combine_bwd"),
    (r"combine_bwd_rows_kernel", lambda m: "combine_bwd"),
    (r"unpermute_kernel", lambda m: "unpermute"),
    (r"expert_delta_kernel", lambda m: "expert_delta"),
    (r"splitk_reduce_kernel", lambda m: "splitk_reduce"),
    (r"splitk_rows_reduce_kernel", lambda m: "splitk_rows_reduce"),
    (r"zero_counters_kernel", lambda m: "zero_counters"),
    (r"adamw_kernel", lambda m: "adamw_step"),
    (r"outer_nesterov_kernel", lambda m: "outer_nesterov"),
    (r"replica_mean_kernel", lambda m: "replica_mean"),
    (r"copy_expert_rows_kernel", lambda m: "copy_expert_rows"),
]

# timing name prefix -> source file that holds the kernel
_SOURCES = [("gemm_", "gemm.hip"), ("splitk_", "gemm.hip"), ("zero_counters", "gemm.hip"), ("route_", "route.hip"), ("dispatch_", "dispatch.hip"),
            ("combine_", "dispatch.hip"), ("unpermute", "dispatch.hip"),
            ("expert_delta", "dispatch.hip"), ("adamw", "optim.hip"), ("outer_", "optim.hip"),
            ("replica_", "optim.hip"),
            ("copy_expert_rows", "placement.hip")]


def timing_name(symbol: str) -> str | None:
    """Library timing name of a kernel symbol (demangled or mangled), or None
    for kernels not ours."""
    if "moe::" not in symbol and "_ZN3moe" not in symbol:
        return None
    for pat, fn in _SYMBOLS:
        m = re.search(pat, symbol)
        if m:
            return fn(m)
    return None


def _code_only(src: str) -> str:
    """C++ source without comments and with whitespace runs collapsed, so that
    editing a comment does not count as changing the kernel."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def source_digest(name: str) -> str | None:
    """sha256 (16 hex digits) of the code of the kernel's source file and the
    shared header (comments and layout ignored)."""
    for prefix, fname in _SOURCES:
        if name.startswith(prefix):
            h = hashlib.sha256()
            for f in (fname, "common.h"):
                with open(os.path.join(CSRC, f)) as fh:
                    h.update(_code_only(fh.read()).encode())
            return h.hexdigest()[:16]
    return None


def _is_copy(symbol: str) -> bool:
    return "copyBuffer" in symbol or "copy_kernel" in symbol


def _mangled_kernel_name(sym: str) -> str:
    """The *_kernel component of an Itanium-mangled nested name
    (_ZN<len><id><len><id>...), or sym itself."""
    i = sym.find("N") + 1 if sym.startswith("_ZN") else 2
    found = sym
    while i < len(sym) and sym[i].isdigit():
        j = i
        while j < len(sym) and sym[j].isdigit():
            j += 1
        n = int(sym[i:j])
        comp = sym[j:j + n]
        if comp.endswith("_kernel"):
            found = comp
        i = j + n
    return found


def kernel_stats(stats_csv: str, out: str, command: str) -> None:
    rows = list(csv.DictReader(open(stats_csv)))
    agg = collections.OrderedDict()
    for r in rows:
        nm = timing_name(r["Name"])
        if nm is None:
            continue
        calls, tot = int(r["Calls"]), float(r["TotalDurationNs"])
        mn, mx = float(r["MinNs"]), float(r["MaxNs"])
        a = agg.setdefault(nm, [0, 0.0, float("inf"), 0.0, set()])
        a[0] += calls
        a[1] += tot
        a[2] = min(a[2], mn)
        a[3] = max(a[3], mx)
        sym = r["Name"].replace("void ", "").replace("moe::(anonymous namespace)::", "")
        if sym.startswith("_Z"):  # mangled (templates on bf16): the kernel's own name
            sym = _mangled_kernel_name(sym)
        a[4].add(re.sub(r"\(.*", "", sym))
    total = sum(v[1] for v in agg.values())
    with open(out, "w") as f:
        f.write("# rocprofv3 --kernel-trace --stats summary (durations in microseconds)\n")
        f.write(f"# command: {command}\n")
        f.write("# name = the library's timing name (bench.py 'kernels' keys); one name can\n")
        f.write("# cover several launches per step (e.g. routed and shared experts)\n\n")
        f.write(f"{'name':18s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} "
                f"{'total_ms':>9s} {'share':>6s}  symbol\n")
        for nm, (calls, tot, mn, mx, syms) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
            f.write(f"{nm:18s} {calls:6d} {tot / calls / 1e3:9.1f} {mn / 1e3:9.1f} "
                    f"{mx / 1e3:9.1f} {tot / 1e6:9.3f} {100 * tot / total:5.1f}%  "
                    f"{','.join(sorted(syms))}\n")


def _per_dispatch(csv_path: str, counter: str):
    """{symbol: [values per dispatch]} of one counter (summed over its dimensions)."""
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        per[r["Kernel_Name"]][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
    return {k: list(v.values()) for k, v in per.items()}


def traffic(fetch_csv: str, write_csv: str, out: str, command: str) -> None:
    fetch = _per_dispatch(fetch_csv, "FETCH_SIZE")
    write = _per_dispatch(write_csv, "WRITE_SIZE")
    kib = 1024.0

    def calib(per):
        best = max((v for k, vals in per.items() if _is_copy(k) for v in vals), default=None)
        if not best:
            raise SystemExit("no calibration copy found: run bench.py with --traffic-calibration")
        return CALIBRATION_BYTES / (best * kib), best

    f_fetch, c_fetch = calib(fetch)
    f_write, c_write = calib(write)

    def by_name(per):
        agg = collections.defaultdict(list)
        for sym, vals in per.items():
            nm = timing_name(sym)
            if nm:
                agg[nm] += vals
        return agg

    fn, wn = by_name(fetch), by_name(write)
    with open(out, "w") as f:
        f.write("# HBM traffic per launch from rocprofv3 --pmc (one counter per run)\n")
        f.write(f"# fetch command: {command.replace('{COUNTER}', 'FETCH_SIZE')}\n")
        f.write(f"# write command: {command.replace('{COUNTER}', 'WRITE_SIZE')}\n")
        f.write(f"# calibration: a plain {CALIBRATION_BYTES} B device-to-device copy read "
                f"FETCH_SIZE {c_fetch:.0f} KiB and WRITE_SIZE {c_write:.0f} KiB\n")
        f.write(f"# scale: fetch x {f_fetch:.5f}, write x {f_write:.5f} (one factor per counter for "
                "every kernel: it assumes each kernel's requests are sized like the copy's; "
                "partial-line or scattered reads may be overstated)\n")
        f.write("# columns: name launches fetch_kib write_kib bytes_per_launch source_digest\n")
        for nm in sorted(set(fn) | set(wn)):
            fv, wv = fn.get(nm, []), wn.get(nm, [])
            fa = sum(fv) / len(fv) if fv else 0.0
            wa = sum(wv) / len(wv) if wv else 0.0
            b = fa * kib * f_fetch + wa * kib * f_write
            f.write(f"{nm} {max(len(fv), len(wv))} {fa:.1f} {wa:.1f} {b:.0f} "
                    f"{source_digest(nm)}\n")


def mfma(counters_csv: str, bench_json: str, out: str, command: str) -> None:
    """Per GEMM launch: the bf16 MFMA flops the hardware executed (rocprofv3's
    MfmaFlopsBF16 = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) against the algorithmic
    flops bench.py counts for the same launch (executed rows only), and the
    MFMA busy share (MfmaUtil = MFMA busy cycles over all SIMDs / (GPU active
    cycles x SIMDs))."""
    import json
    per = collections.defaultdict(lambda: collections.defaultdict(lambda: collections.defaultdict(float)))
    for r in csv.DictReader(open(counters_csv)):
        nm = timing_name(r["Kernel_Name"])
        if nm is None or not nm.startswith("gemm_"):
            continue
        per[nm][r["Counter_Name"]][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
    bench = {}
    for line in open(bench_json):
        line = line.strip()
        if line.startswith("{"):
            bench = json.loads(line)
    kern = bench.get("kernels", {})
    with open(out, "w") as f:
        f.write("# bf16 MFMA work and busy share per GEMM launch (rocprofv3 --pmc, derived counters)\n")
        f.write(f"# command: {command}\n")
        f.write("# algorithmic flops per launch: bench.py 'kernels' per_launch of the run\n")
        f.write(f"#   {bench_json.split('/')[-1]} (executed routes only; config {bench.get('config', {}).get('workload')})\n")
        f.write("# executed/algorithmic above 1 is tile padding: rows of partial m-tiles and\n")
        f.write("# columns past N in the last n-tile still run MFMAs\n")
        f.write("# columns: name launches executed_gflop algorithmic_gflop executed/algorithmic mfma_util_pct\n")
        for nm in sorted(per):
            fl = per[nm].get("MfmaFlopsBF16", {})
            ut = per[nm].get("MfmaUtil", {})
            n = max(len(fl), len(ut))
            ex = sum(fl.values()) / len(fl) if fl else float("nan")
            u = sum(ut.values()) / len(ut) if ut else float("nan")
            alg = kern.get(nm, {}).get("per_launch")
            ratio = ex / alg if alg else float("nan")
            f.write(f"{nm} {n} {ex / 1e9:.1f} {(alg or float('nan')) / 1e9:.1f} {ratio:.3f} {u:.1f}\n")


def load_traffic(path: str) -> dict:
    """{name: (bytes_per_launch, digest)} from a traffic summary; {} if absent."""
    res = {}
    if not os.path.exists(path):
        return res
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        nm, _launches, _f, _w, b, dg = line.split()
        res[nm] = (float(b), dg)
    return res


def main() -> None:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    k = sub.add_parser("kernel-stats")
    k.add_argument("stats_csv")
    k.add_argument("out")
    k.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_csv")
    t.add_argument("write_csv")
    t.add_argument("out")
    t.add_argument("--command", required=True, help="the pmc command with {COUNTER}")
    m = sub.add_parser("mfma")
    m.add_argument("counters_csv")
    m.add_argument("bench_json", help="a bench.py JSON line of the same workload (kernel timing on)")
    m.add_argument("out")
    m.add_argument("--command", required=True)
    a = ap.parse_args()
    if a.cmd == "kernel-stats":
        kernel_stats(a.stats_csv, a.out, a.command)
    elif a.cmd == "mfma":
        mfma(a.counters_csv, a.bench_json, a.out, a.command)
    else:
        traffic(a.fetch_csv, a.write_csv, a.out, a.command)


if __name__ == "__main__":
    main()
