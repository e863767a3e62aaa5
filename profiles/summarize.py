"""Turn rocprofv3 outputs of bench.py into the short summaries kept in this
folder (kernel-time table, calibrated HBM traffic of the attention kernel).

    python profiles/summarize.py <gpurun_out dir>

Inputs (from the commands written into the summaries): a --kernel-trace --stats
run, FETCH_SIZE and WRITE_SIZE --pmc runs of the workload, and the same two
counters for `bench.py --copy-probe` (a plain 1 GiB copy per launch), which
give the factor from counter units to bytes.
"""
import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def rows(pattern):
    f = glob.glob(pattern, recursive=True)
    if not f:
        raise SystemExit(f"missing {pattern}")
    return list(csv.DictReader(open(f[0])))


def counter_avg(rs, kernel_prefix):
    v = [float(r["Counter_Value"]) for r in rs if r["Kernel_Name"].startswith(kernel_prefix)]
    return sum(v) / len(v), len(v)


def main(out):
    stats = rows(f"{out}/prof_factory/**/*kernel_stats.csv")
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# Kernel-time summary: factory_b256 workload (256 ragged requests, pi0-shaped expert, bf16)", "",
             "Command (one MI355X, repository root, library built in-tree; one lane, so every dispatch",
             "runs alone as in bench.py's per-kernel timing pass):", "", "```",
             "export TMPDIR=/tmp; rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_factory "
             "-o factory -- python -u bench.py --steps 3 --warmup 1 --no-cpu-baseline --lanes 1", "```", "",
             "The profiled process runs 1 warm-up + 3 timed + 2 per-kernel-timing generate calls (6 calls).",
             "Table from `factory_kernel_stats.csv`, sorted by total time.", "",
             "| Kernel | Calls | Avg (us) | Total (ms) | % |", "|---|---:|---:|---:|---:|"]
    for r in stats:
        name = r["Name"].split("(")[0]
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    open(os.path.join(HERE, "kernel_stats_factory_b256.md"), "w").write("\n".join(lines) + "\n")

    fetch, nf = counter_avg(rows(f"{out}/pmc_fetch/**/*counter_collection.csv"), "void rosa::attention_bf16")
    write, nw = counter_avg(rows(f"{out}/pmc_write/**/*counter_collection.csv"), "void rosa::attention_bf16")
    cf, _ = counter_avg(rows(f"{out}/pmc_cfetch/**/*counter_collection.csv"), "__amd_rocclr_copyBuffer")
    cw, _ = counter_avg(rows(f"{out}/pmc_cwrite/**/*counter_collection.csv"), "__amd_rocclr_copyBuffer")
    gib_kib = float(1 << 20)
    ff, wf = gib_kib / cf, gib_kib / cw
    rd, wr = fetch * ff * 1024, write * wf * 1024
    sha = hashlib.sha256(open(os.path.join(ROOT, "paper_2607_01088_amd", "csrc", "k_attn.hip"), "rb").read())
    t = {"kernel": "attention", "workload": "factory_b256", "source_sha": sha.hexdigest()[:16], "dispatches": nf,
         "fetch_size_kib_avg": round(fetch, 1), "write_size_kib_avg": round(write, 1),
         "copy_probe_fetch_kib": round(cf, 1), "copy_probe_write_kib": round(cw, 1),
         "fetch_factor": round(ff, 4), "write_factor": round(wf, 4), "hbm_bytes_per_launch": int(rd + wr)}
    json.dump(t, open(os.path.join(HERE, "traffic_attention_factory_b256.json"), "w"), indent=1)
    md = ["# HBM traffic of the attention kernel, factory_b256 workload", "",
          "Commands (one MI355X, repository root, library built in-tree; one counter per run, one lane):", "", "```",
          "export TMPDIR=/tmp",
          "timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE --output-format csv -d gpurun_out/pmc_fetch -o f -- "
          "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
          "timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE --output-format csv -d gpurun_out/pmc_write -o w -- "
          "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
          "timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv -d gpurun_out/pmc_cfetch -o f -- "
          "python -u bench.py --copy-probe",
          "timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv -d gpurun_out/pmc_cwrite -o w -- "
          "python -u bench.py --copy-probe",
          "python profiles/summarize.py gpurun_out", "```", "",
          f"Calibration: the copy probe reads and writes 1 GiB (1048576 KiB) per launch; FETCH_SIZE reads "
          f"{cf:.1f} KiB and WRITE_SIZE {cw:.1f} KiB per dispatch, so FETCH_SIZE is scaled by {ff:.4f} and "
          f"WRITE_SIZE by {wf:.4f}.", "",
          "| Kernel | Dispatches | FETCH_SIZE (KiB, avg) | WRITE_SIZE (KiB, avg) | HBM read (MB) | HBM write (MB) |",
          "|---|---:|---:|---:|---:|---:|",
          f"| `rosa::attention_bf16_kernel<256, 1>` | {nf} | {fetch:.1f} | {write:.1f} | {rd / 1e6:.1f} | {wr / 1e6:.1f} |",
          "", f"Per launch: {(rd + wr) / 1e6:.1f} MB of HBM traffic.  Algorithmic bytes per launch (each active "
          "request's prefix K and V of the layer read once) are 174 MB averaged over the 180 launches of one call; "
          "queries, action keys and the output add about 26 MB written and 30 MB read.", "",
          f"Kernel source sha256 (first 16 hex digits) of `k_attn.hip` when measured: `{t['source_sha']}`."]
    open(os.path.join(HERE, "traffic_attention_factory_b256.md"), "w").write("\n".join(md) + "\n")
    print(json.dumps(t))


if __name__ == "__main__":
    main(sys.argv[1] if len(sys.argv) > 1 else os.path.join(ROOT, "gpurun_out"))
