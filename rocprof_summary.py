"""Summarise rocprofv3 result databases (rocpd SQLite) of bench.py runs.

  python rocprof_summary.py trace <kt_results.db>
      per-kernel call count, total and average duration (kernel-trace run)
  python rocprof_summary.py counter <results.db> <COUNTER> [<kernel substring> ...]
      per-kernel average of a per-dispatch counter (e.g. FETCH_SIZE, WRITE_SIZE,
      in KiB), and the same counter for the plain 256 MiB copy that
      `bench.py --copy-calibration` runs first, as the calibration factor
      measured KiB / 262144 KiB.
  python rocprof_summary.py decode-traffic <fetch_results.db> <write_results.db>
      calibrated HBM bytes per launch of the W1/W3 and W2 decode kernels
      (FETCH_SIZE + WRITE_SIZE), tagged with the hash of the kernel source
      that bench.py checks before it reports them as roofline.traffic.
"""
import os
import sqlite3
import sys
from collections import defaultdict


def _short(name: str) -> str:
    for key in ("decode13_kernel", "decode_kernel<true", "decode_kernel<false", "xprep_kernel", "bgemm_kernel", "gemm_kernel",
                "combine_kernel", "gate_kernel", "topk_kernel", "hist_perm_kernel",
                "schedule_kernel", "pack_kernel", "chunk_kernel", "route_kernel", "to_bf16_kernel"):
        if key in name:
            return name[name.find(key):][:90]
    return name[:90]


def trace(db):
    con = sqlite3.connect(db)
    rows = con.execute("select name, duration from kernels").fetchall()
    agg = defaultdict(list)
    for name, dur in rows:
        agg[_short(name)].append(dur)
    print(f"{'kernel':92s} {'calls':>6s} {'total_us':>10s} {'avg_us':>9s}")
    for name, durs in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        print(f"{name:92s} {len(durs):6d} {sum(durs) / 1e3:10.1f} {sum(durs) / len(durs) / 1e3:9.2f}")


def _per_kernel(db, cname):
    """Calibration factor and per-kernel average of a per-dispatch counter."""
    con = sqlite3.connect(db)
    cols = [r[1] for r in con.execute("pragma table_info('counters_collection')")]
    rows = con.execute("select * from counters_collection").fetchall()
    ix = {c: i for i, c in enumerate(cols)}
    name_col = "kernel_name" if "kernel_name" in ix else "name"
    per_disp = defaultdict(float)
    names = {}
    for r in rows:
        if r[ix["counter_name"]] == cname:
            per_disp[r[ix["dispatch_id"]]] += float(r[ix["value"]])
            names[r[ix["dispatch_id"]]] = r[ix[name_col]]
    cal = sorted(v for d, v in per_disp.items() if "copyBuffer" in names[d] and v > 0.25 * 262144)
    factor = cal[len(cal) // 2] / 262144.0
    agg = defaultdict(list)
    for key, v in per_disp.items():
        agg[_short(names[key])].append(v)
    return factor, {k: sum(v) / len(v) for k, v in agg.items()}


def decode_traffic(fetch_db, write_db):
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    from bench import kernel_source_hash
    total = defaultdict(float)
    for db, cname in ((fetch_db, "FETCH_SIZE"), (write_db, "WRITE_SIZE")):
        factor, avg = _per_kernel(db, cname)
        for name, kib in avg.items():
            total[name] += kib / factor * 1024
    def w13_kernel(k):  # W1/W3 + SwiGLU: decode13_kernel<..., true> or decode_kernel<true, ...>
        return k.startswith("decode_kernel<true") or (k.startswith("decode13_kernel") and "true>" in k)

    def w2_kernel(k):
        return k.startswith("decode_kernel<false") or (k.startswith("decode13_kernel") and "false>" in k)

    w13 = [v for k, v in total.items() if w13_kernel(k)]
    w2 = [v for k, v in total.items() if w2_kernel(k)]
    print("traffic per launch (FETCH + WRITE, calibrated), used by bench.py as roofline.traffic:")
    print(f"kernel_source_sha256_16: {kernel_source_hash()}")
    print(f"traffic_w13_bytes: {int(round(sum(w13) / len(w13)))}")
    print(f"traffic_w2_bytes: {int(round(sum(w2) / len(w2)))}")


def counter(db, cname, subs):
    con = sqlite3.connect(db)
    cols = [r[1] for r in con.execute("pragma table_info('counters_collection')")]
    rows = con.execute("select * from counters_collection").fetchall()
    ix = {c: i for i, c in enumerate(cols)}
    name_col = "kernel_name" if "kernel_name" in ix else "name"
    per_disp = defaultdict(float)
    names = {}
    for r in rows:
        if r[ix["counter_name"]] != cname:
            continue
        key = r[ix["dispatch_id"]]
        per_disp[key] += float(r[ix["value"]])
        names[key] = r[ix[name_col]]
    # the three 256 MiB device-to-device copies of `bench.py --copy-calibration`
    # run as the runtime's copy kernel; each reads and writes 262144 KiB
    cal = sorted(v for d, v in per_disp.items()
                 if "copyBuffer" in names[d] and v > 0.25 * 262144)
    factor = cal[len(cal) // 2] / 262144.0 if cal else None
    if cal:
        print(f"calibration: {len(cal)} copies of 262144 KiB read and written, median "
              f"{cname} {cal[len(cal) // 2]:.1f} KiB -> factor {factor:.4f} (counter / bytes)")
    agg = defaultdict(list)
    for key, v in per_disp.items():
        agg[_short(names[key])].append(v)
    print(f"{'kernel':92s} {'dispatches':>10s} {'KiB_avg':>12s} {'MB_avg_calibrated':>18s}")
    for name, vals in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        if subs and not any(s in name for s in subs):
            continue
        avg = sum(vals) / len(vals)
        calib = f"{avg / factor * 1024 / 1e6:18.2f}" if factor else f"{'-':>18s}"
        print(f"{name:92s} {len(vals):10d} {avg:12.1f} {calib}")


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(sys.argv[2])
    elif sys.argv[1] == "decode-traffic":
        decode_traffic(sys.argv[2], sys.argv[3])
    else:
        counter(sys.argv[2], sys.argv[3], sys.argv[4:])
