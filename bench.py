"""Benchmark: batched action-chunk generation on one MI355X.

One step = one rosa_generate_actions call over the whole factory-fleet batch
(256 ragged robot requests, pi0-shaped action expert, bf16): every request runs
its own 5 or 10 Euler steps over 18 layers with attention over its own cached
prefix.  Prefix KV, noise and weights are resident in HBM before timing.

Prints one JSON line (rank 0): throughput in action chunks/s, p50/p99 batch
latency, the roofline of the dominant kernel (timed live with HIP events on
the library's stream), and the CPU oracle timed on this host's cores on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0    # MI355X dense bf16 MFMA
PROFILES = os.path.join(ROOT, "profiles")


def algorithmic_work(shape, reqs):
    """Per-call algorithmic work by kernel class, from the request shapes.

    GEMM flops: 2 * rows * (in * out) for the four projections of every layer
    at every step.  Attention: prefix K and V bytes streamed once per
    layer-step (L * 2 * n_kv * hd * 2 bytes per prefix token), and
    4 * n_q * hd * H * (P + H) flops per layer-step."""
    L, d, nq, nkv, hd, dff = (shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                              shape.head_dim, shape.d_mlp)
    qkv = (nq + 2 * nkv) * hd
    tok_steps = sum(r.horizon * r.steps for r in reqs)
    w = {
        "gemm_qkv": 2.0 * tok_steps * d * qkv * L,
        "gemm_o": 2.0 * tok_steps * nq * hd * d * L,
        "gemm_up": 2.0 * tok_steps * d * dff * L,
        "gemm_down": 2.0 * tok_steps * dff * d * L,
    }
    if getattr(shape, "attention_layout", 0) == 1:
        # alternating: the (L + 1) // 2 even layers read the prefix, the odd
        # layers attend over the request's own action keys only
        lc, ls = (L + 1) // 2, L // 2
        attn_bytes = sum(r.prefix_len * r.steps for r in reqs) * lc * 2 * nkv * hd * 2
        attn_flops = sum(4.0 * nq * hd * r.horizon * (lc * r.prefix_len + ls * r.horizon) * r.steps for r in reqs)
    else:
        attn_bytes = sum(r.prefix_len * r.steps for r in reqs) * L * 2 * nkv * hd * 2
        attn_flops = sum(4.0 * nq * hd * r.horizon * (r.prefix_len + r.horizon) * r.steps for r in reqs) * L
    return w, float(attn_bytes), float(attn_flops), tok_steps


def kernel_source_hash(name: str) -> str:
    src = {"attention": "k_attn.hip"}.get(name, "k_gemm.hip")
    with open(os.path.join(ROOT, "paper_2607_01088_amd", "csrc", src), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(name: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary of this
    kernel on this workload, if it was taken on the current kernel source."""
    path = os.path.join(PROFILES, f"traffic_{name}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_sha") != kernel_source_hash(name):
        return None
    return t.get("hbm_bytes_per_launch")


def cpu_baseline(preset, weights, reqs_meta, budget_s: float):
    """The oracle on a stratified sample of the workload's requests; its
    throughput is extrapolated to the whole batch by algorithmic GEMM +
    attention flops (the oracle's cost is additive over requests)."""
    from oracle import OracleModel
    from synthetic import make_requests
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    cores = len(os.sched_getaffinity(0))
    om = OracleModel(weights, preset.shape)
    classes = {}
    for i, m in enumerate(reqs_meta):
        classes.setdefault((m.horizon, m.steps), []).append(i)
    order = []
    pools = [sorted(v) for _, v in sorted(classes.items())]
    for j in range(max(len(p) for p in pools)):
        for p in pools:
            if j < len(p):
                order.append(p[j])

    def flops(m):
        sh = preset.shape
        per_tok = 2.0 * sh.n_layers * (sh.d_model * sh.qkv_dim + sh.n_q_heads * sh.head_dim * sh.d_model
                                       + 2 * sh.d_model * sh.d_mlp)
        if getattr(sh, "attention_layout", 0) == 1:
            att = 4.0 * sh.n_q_heads * sh.head_dim * m.horizon * (
                (sh.n_layers + 1) // 2 * m.prefix_len + sh.n_layers // 2 * m.horizon)
        else:
            att = 4.0 * sh.n_layers * sh.n_q_heads * sh.head_dim * m.horizon * (m.prefix_len + m.horizon)
        return (per_tok * m.horizon + att) * m.steps

    done, t_used = [], 0.0
    for i in order:
        r = make_requests(preset, indices=[i], threads=1)[0]
        t0 = time.perf_counter()
        om.generate([r])
        t_used += time.perf_counter() - t0
        done.append(i)
        if t_used >= budget_s and len(done) >= len(pools):
            break
    f_sample = sum(flops(reqs_meta[i]) for i in done)
    f_total = sum(flops(m) for m in reqs_meta)
    batch_s = t_used * f_total / f_sample
    return {
        "value": len(reqs_meta) / batch_s,
        "unit": "chunks/s",
        "cores": int(blas_threads),          # threads the oracle's matrix products ran on
        "host_cores_available": cores,
        "kind": "oracle",
        "sample": (f"{len(done)} of {len(reqs_meta)} requests (stratified over horizon x steps), "
                   f"{t_used:.1f} s measured, scaled to the whole batch by algorithmic flops "
                   f"(extrapolated batch time {batch_s:.1f} s); NumPy float64"),
    }


def _csv_rows(pattern):
    import csv
    import glob
    f = glob.glob(pattern, recursive=True)
    if not f:
        raise SystemExit(f"missing {pattern}")
    return list(csv.DictReader(open(f[0])))


def _counter_avg(rs, kernel_prefix):
    v = [float(r["Counter_Value"]) for r in rs if r["Kernel_Name"].startswith(kernel_prefix)]
    return sum(v) / len(v), len(v)


def _summarize_prefill(out):
    """Kernel-time table of the prefix producer from a --kernel-trace --stats
    run of `bench.py --prefill` (prof_prefill/)."""
    stats = _csv_rows(f"{out}/prof_prefill/**/*kernel_stats.csv")
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# Kernel-time summary: vlm_prefill_b32 workload (32 robots' prefixes, 26,173 tokens, "
             "18-layer width-2048 VLM backbone, bf16)", "",
             "Command (one MI355X, repository root, library built in-tree):", "", "```",
             f"export TMPDIR=/tmp; rocprofv3 --kernel-trace --stats --output-format csv -d {out}/prof_prefill "
             "-o prefill -- python3 -u bench.py --prefill --steps 3 --warmup 1 --no-cpu-baseline",
             f"python bench.py --summarize-profiles {out}", "```", "",
             "The profiled process runs 1 warm-up + 3 timed + 2 per-kernel-timing prefill calls (6 calls); each "
             "call is 18 QKV projections and K/V scatters and 17 attention, output-projection and MLP layers "
             "(the last layer's caches need only its K and V).",
             "Table from `prefill_kernel_stats.csv`, sorted by total time.", "",
             "| Kernel | Calls | Avg (us) | Total (ms) | % |", "|---|---:|---:|---:|---:|"]
    for r in stats:
        name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0]
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    open(os.path.join(PROFILES, "kernel_stats_vlm_prefill_b32.md"), "w").write("\n".join(lines) + "\n")


PMC_UTIL = ("MfmaUtil VALUBusy LdsUtil LDSBankConflict SQ_WAIT_INST_LDS SQ_WAVE_CYCLES SQ_BUSY_CYCLES "
            "SQ_LDS_DATA_FIFO_FULL GRBM_GUI_ACTIVE")
PMC_INST = ("SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS SQ_INSTS_SALU SQ_WAIT_ANY SQ_INSTS_VALU_MFMA_MOPS_BF16 "
            "SQ_LDS_CMD_FIFO_FULL SQ_ACTIVE_INST_LDS GRBM_GUI_ACTIVE")
PROJ_ORDER = ("gemm_qkv", "attention", "gemm_o", "gemm_up", "gemm_down")


def _classify_dispatches(rows):
    """Dispatch id -> kernel role for a one-lane bf16 generate run.  Per layer
    the expert launches modnorm, the QKV projection, attention (and, for split
    keys, the merge), the output projection, modnorm, MLP up, MLP down; a split
    product's reduce kernel belongs to the projection before it, and when that
    reduce also takes the following norm, or an unsplit output projection or
    MLP-down defers it to the next product, no modnorm launch follows."""
    names = {}
    for r in rows:
        names[int(r["Dispatch_Id"])] = r["Kernel_Name"]
    role, prev, last_gemm = {}, "", ""
    for d in sorted(names):
        n = names[d]
        if "attention_bf16" in n:
            cur = "attention"
        elif "gemm_split_reduce" in n:
            cur = prev if prev.startswith("gemm_") else "other"
        elif "gemm_bf16_kernel" in n:
            if prev in ("attention", "attn_merge"):
                cur = "gemm_o"
            elif prev == "gemm_up":
                cur = "gemm_down"
            elif prev == "modnorm":
                cur = "gemm_up" if last_gemm == "gemm_o" else "gemm_qkv"
            elif prev == "gemm_o":
                cur = "gemm_up"
            elif prev == "gemm_down":
                cur = "gemm_qkv"
            else:
                cur = "other"
            last_gemm = cur
        elif "attn_merge" in n:
            cur = "attn_merge"
        elif "modnorm" in n:
            cur = "modnorm"
        else:
            cur = "other"
        role[d] = cur
        prev = cur
    return role


def _pmc_by_role(rows, role):
    """{role: {counter: [values per dispatch]}} and {role: {dispatch: GRBM_GUI_ACTIVE}}."""
    agg, grbm = {}, {}
    for r in rows:
        k = role.get(int(r["Dispatch_Id"]), "other")
        v = float(r["Counter_Value"])
        agg.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(v)
        if r["Counter_Name"] == "GRBM_GUI_ACTIVE":
            grbm.setdefault(k, {})[int(r["Dispatch_Id"])] = v
    return agg, grbm


def _summarize_pmc(out):
    """Utilisation counters per kernel role (pmc_util/, pmc_inst/ runs)."""
    util = _csv_rows(f"{out}/pmc_util/**/*counter_collection.csv")
    inst = _csv_rows(f"{out}/pmc_inst/**/*counter_collection.csv")
    ua, ug = _pmc_by_role(util, _classify_dispatches(util))
    ia, _ = _pmc_by_role(inst, _classify_dispatches(inst))

    def wavg(agg, grbm, role, name):
        # time-weighted over dispatches (weights: GRBM_GUI_ACTIVE of the dispatch)
        rows = [r for r in util if r["Counter_Name"] == name]
        role_of = _classify_dispatches(util)
        num = den = 0.0
        for r in rows:
            d = int(r["Dispatch_Id"])
            if role_of.get(d) != role:
                continue
            w = grbm.get(role, {}).get(d, 0.0)
            num += w * float(r["Counter_Value"])
            den += w
        return num / den if den else float("nan")

    def tot(agg, role, name):
        return sum(agg.get(role, {}).get(name, [0.0]))

    lines = ["# Utilisation counters per kernel, factory_b256 workload", "",
             "Commands (one MI355X, repository root, library built in-tree; one lane, so every dispatch runs "
             "alone; two counter sets, each in its own run):", "", "```", "export TMPDIR=/tmp",
             f"timeout -s KILL 300 rocprofv3 --pmc {PMC_UTIL} --output-format csv -d {out}/pmc_util -o u -- "
             "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
             f"timeout -s KILL 300 rocprofv3 --pmc {PMC_INST} --output-format csv -d {out}/pmc_inst -o i -- "
             "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
             f"python bench.py --summarize-profiles {out}", "```", "",
             "Dispatches are assigned to projections by their place in the per-layer launch sequence "
             "(modnorm, QKV, attention, output projection, modnorm, MLP up, MLP down).  MfmaUtil, VALUBusy, "
             "LdsUtil and LDSBankConflict are rocprofv3's derived metrics (percent of the kernel's active GPU "
             "cycles: MFMA busy cycles per SIMD, VALU issue per CU, LDS indexed-access cycles per CU, LDS "
             "bank-conflict stall cycles per CU), averaged over dispatches weighted by GRBM_GUI_ACTIVE.  "
             "LDS wait = SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES (share of resident-wave time spent waiting to issue "
             "an LDS instruction); any wait = SQ_WAIT_ANY / SQ_WAVE_CYCLES.  Instruction counts are per MFMA "
             "instruction (every MFMA here is a 32x32x16 bf16 one, 32 busy cycles).", "",
             "| Kernel | Dispatches | MfmaUtil % | VALUBusy % | LdsUtil % | LDS bank conflict % | LDS wait | "
             "any wait | VALU / MFMA | LDS / MFMA | SALU / MFMA | LDS data FIFO full / active cycle | "
             "GFLOP / dispatch |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    res = {}
    for role in PROJ_ORDER:
        if role not in ua:
            continue
        n = len(ug.get(role, {}))
        mf = wavg(ua, ug, role, "MfmaUtil")
        vb = wavg(ua, ug, role, "VALUBusy")
        lu = wavg(ua, ug, role, "LdsUtil")
        bc = wavg(ua, ug, role, "LDSBankConflict")
        wc = tot(ua, role, "SQ_WAVE_CYCLES")
        lw = tot(ua, role, "SQ_WAIT_INST_LDS") / wc if wc else float("nan")
        mfma = tot(ia, role, "SQ_INSTS_MFMA")
        aw_wc = tot(ia, role, "SQ_WAIT_ANY")
        # SQ_WAIT_ANY comes from the second run; its wave cycles are taken as the first run's
        any_w = aw_wc / wc if wc else float("nan")
        per = lambda c: tot(ia, role, c) / mfma if mfma else float("nan")
        fifo = tot(ua, role, "SQ_LDS_DATA_FIFO_FULL") / max(tot(ua, role, "SQ_BUSY_CYCLES"), 1.0)
        gfl = tot(ia, role, "SQ_INSTS_VALU_MFMA_MOPS_BF16") * 512 / max(len(ia.get(role, {}).get("SQ_INSTS_MFMA", [1])), 1) / 1e9
        res[role] = dict(dispatches=n, mfma_util=round(mf, 1), valu_busy=round(vb, 1), lds_util=round(lu, 1),
                         lds_bank_conflict=round(bc, 2), lds_wait=round(lw, 3), any_wait=round(any_w, 3),
                         valu_per_mfma=round(per("SQ_INSTS_VALU"), 2), lds_per_mfma=round(per("SQ_INSTS_LDS"), 3),
                         salu_per_mfma=round(per("SQ_INSTS_SALU"), 3), gflop_per_dispatch=round(gfl, 2))
        lines.append(f"| {role} | {n} | {mf:.1f} | {vb:.1f} | {lu:.1f} | {bc:.2f} | {lw:.3f} | {any_w:.3f} | "
                     f"{per('SQ_INSTS_VALU'):.2f} | {per('SQ_INSTS_LDS'):.3f} | {per('SQ_INSTS_SALU'):.3f} | "
                     f"{fifo:.3f} | {gfl:.2f} |")
    srcs = {f: hashlib.sha256(open(os.path.join(ROOT, "paper_2607_01088_amd", "csrc", f), "rb").read()).hexdigest()[:16]
            for f in ("k_attn.hip", "k_gemm.hip")}
    lines += ["", "Kernel source sha256 (first 16 hex digits) when measured: " +
              ", ".join(f"`{f}` `{h}`" for f, h in srcs.items()) + "."]
    open(os.path.join(PROFILES, "pmc_factory_b256.md"), "w").write("\n".join(lines) + "\n")
    json.dump({"workload": "factory_b256", "sources": srcs, "kernels": res},
              open(os.path.join(PROFILES, "pmc_factory_b256.json"), "w"), indent=1)


def _traffic_rows(out, ff, wf):
    """Per-projection rows of the traffic table (dispatches assigned by launch order)."""
    fr = _csv_rows(f"{out}/pmc_fetch/**/*counter_collection.csv")
    wr_ = _csv_rows(f"{out}/pmc_write/**/*counter_collection.csv")
    fa, _ = _pmc_by_role(fr, _classify_dispatches(fr))
    wa, _ = _pmc_by_role(wr_, _classify_dispatches(wr_))
    rows = []
    for role in ("gemm_qkv", "gemm_o", "gemm_up", "gemm_down"):
        f = fa.get(role, {}).get("FETCH_SIZE", [])
        w = wa.get(role, {}).get("WRITE_SIZE", [])
        if not f or not w:
            continue
        fk, wk = sum(f) / len(f), sum(w) / len(w)
        rows.append(f"| {role} (all tile configurations) | {len(f)} | {fk:.1f} | {wk:.1f} | "
                    f"{fk * ff * 1024 / 1e6:.1f} | {wk * wf * 1024 / 1e6:.1f} |")
    return rows


def _summarize_presets(out):
    """One line per workload from `bench.py --workload W` runs whose JSON
    lines were saved as bench_W.log under `out` (with the oracle's timing on
    the host cores when the run measured it)."""
    rows = []
    for w in ("factory_b256", "factory_b256_alternating", "pi0_b1", "pi0_b32", "stress_b512"):
        f = f"{out}/bench_{w}.log"
        if not os.path.exists(f):
            continue
        try:
            j = json.loads(open(f).read().strip().splitlines()[-1])
        except (ValueError, IndexError):
            continue
        if j.get("config", {}).get("workload") == w:
            rows.append((w, j))
    if not rows:
        return
    lines = ["# Whole-call results per workload (one MI355X, bf16)", "",
             "Commands (repository root, library built in-tree), one per workload:", "", "```",
             "export TMPDIR=/tmp",
             *[f"timeout -k 10 400 python -u bench.py --workload {w.replace('_alternating', '')}"
               + ("" if "cpu_baseline" in j else " --no-cpu-baseline")
               + (" --attention-layout alternating" if w.endswith("_alternating") else "") + f" > {out}/bench_{w}.log"
               for w, j in rows],
             f"python bench.py --summarize-profiles {out}", "```", "",
             "Each line: 3 warm-up + 20 timed calls; chunks/s = requests x calls / wall time; per-call kernel time "
             "from the library's per-launch events (one extra pass).", "",
             "| Workload | Requests | Action tokens | Prefix tokens | chunks/s | ms per call | p50 ms | p99 ms | "
             "attention ms/call | GEMMs ms/call | attention GB/s (frac of 8 TB/s) | GEMM TFLOP/s (frac of 2.5 PF) | "
             "oracle chunks/s (host threads) |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for w, j in rows:
        k = j.get("kernels", {})
        att = k.get("attention", {})
        gm = sum(v.get("ms_per_call", 0) for n, v in k.items() if n.startswith("gemm_"))
        lines.append(f"| {w} | {j['config']['requests']} | {j['config']['action_tokens']} | "
                     f"{j['config']['prefix_tokens']} | {j['value']} | {j['ms_per_step']} | {j['p50_ms']} | "
                     f"{j['p99_ms']} | {att.get('ms_per_call', 0):.2f} | {gm:.2f} | "
                     f"{att.get('achieved', 0):.0f} ({att.get('frac', 0):.3f}) | "
                     f"{j['gemm_all']['achieved']} ({j['gemm_all']['frac']:.3f}) | "
                     + (f"{j['cpu_baseline']['value']:.3g} ({j['cpu_baseline']['cores']}) |" if "cpu_baseline" in j
                        else "- |"))
    samples = [(w, j["cpu_baseline"]["sample"]) for w, j in rows if "cpu_baseline" in j]
    if samples:
        lines += ["", "Oracle samples (float64 NumPy on the GPU box's host cores, scaled to the whole batch):"]
        lines += [f"- {w}: {smp}" for w, smp in samples]
    srcs = {f: hashlib.sha256(open(os.path.join(ROOT, "paper_2607_01088_amd", "csrc", f), "rb").read()).hexdigest()[:16]
            for f in ("k_attn.hip", "k_gemm.hip")}
    lines += ["", "Kernel source sha256 (first 16 hex digits) when measured: " +
              ", ".join(f"`{f}` `{h}`" for f, h in srcs.items()) + "."]
    open(os.path.join(PROFILES, "bench_workloads.md"), "w").write("\n".join(lines) + "\n")


_CALL_TRACES = {
    # directory under `out`: (file under profiles/, title, bench arguments)
    "tr_b1": ("kernel_trace_pi0_b1.md", "one single-robot call: pi0_b1 workload (1 request, prefix 816, "
              "horizon 50, 10 Euler steps, bf16)", "--workload pi0_b1"),
    "tr_b16": ("kernel_trace_factory_first16.md", "one 16-robot call: the first 16 requests of the factory_b256 "
               "batch (horizons 16/50, 5/10 Euler steps, bf16)", "--workload factory_b256 --first 16"),
}


def _summarize_call_trace(out, sub):
    """Per-kernel durations and launch gaps of one timed generate call from a
    --kernel-trace run of bench.py (`out`/`sub`/)."""
    import collections
    fname, title, bench_args = _CALL_TRACES[sub]
    rows = _csv_rows(f"{out}/{sub}/**/*kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    starts = [i for i, r in enumerate(rows) if "time_embedding" in r["Kernel_Name"]]
    if len(starts) < 4:
        raise SystemExit(f"{sub}: fewer than 4 generate calls in the trace")
    call = rows[starts[2]:starts[3]]              # the first timed call (after 1 warm-up)
    span = (int(call[-1]["End_Timestamp"]) - int(call[0]["Start_Timestamp"])) / 1e3
    dur = collections.defaultdict(list)
    gap = collections.defaultdict(list)
    prev_end = None
    for r in call:
        name = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0]
        t0, t1 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        dur[name].append((t1 - t0) / 1e3)
        if prev_end is not None:
            gap[name].append((t0 - prev_end) / 1e3)
        prev_end = t1
    busy = sum(sum(v) for v in dur.values())
    lines = [f"# Kernel trace of {title}", "",
             "Command (one MI355X, repository root, library built in-tree):", "", "```",
             f"export TMPDIR=/tmp; rocprofv3 --kernel-trace --output-format csv -d {out}/{sub} -o t -- "
             f"python -u bench.py {bench_args} --steps 3 --warmup 1 --no-cpu-baseline",
             f"python bench.py --summarize-profiles {out}", "```", "",
             f"The first timed call: {len(call)} kernels, {busy / 1e3:.2f} ms of kernel time, {span / 1e3:.2f} ms "
             "from its first kernel's start to its last kernel's end under the tracer (the untraced call takes "
             "about the kernel time: the tracer widens the gaps between dependent launches).  Per layer-step "
             "the call launches QKV, attention (and, for split key ranges, their merge), the output "
             "projection, MLP up and MLP down, with the two modulated norms either as launches of their own "
             "or, after a K-split output or MLP-down projection, fused into its slice reduction, or, "
             "after an unsplit one of at most 1,024 rows, completed in the next product's epilogue.", "",
             "| Kernel | Launches | Avg (us) | Min (us) | Total (ms) | Avg gap before (us) |",
             "|---|---:|---:|---:|---:|---:|"]
    for name, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        g = gap.get(name, [])
        lines.append(f"| `{name}` | {len(v)} | {sum(v) / len(v):.2f} | {min(v):.2f} | {sum(v) / 1e3:.3f} | "
                     f"{(sum(g) / len(g)) if g else 0.0:.2f} |")
    open(os.path.join(PROFILES, fname), "w").write("\n".join(lines) + "\n")


def summarize_profiles(out):
    """Turn rocprofv3 outputs of this script into the summaries under
    profiles/ (kernel-time table, calibrated HBM traffic of the attention
    kernel).  `out` holds a --kernel-trace --stats run (prof_factory/),
    FETCH_SIZE and WRITE_SIZE --pmc runs (pmc_fetch/, pmc_write/) and the same
    counters for --copy-probe (pmc_cfetch/, pmc_cwrite/); the commands are
    written into the summaries."""
    import glob
    if glob.glob(f"{out}/prof_prefill/**/*kernel_stats.csv", recursive=True):
        _summarize_prefill(out)
    if glob.glob(f"{out}/pmc_util/**/*counter_collection.csv", recursive=True):
        _summarize_pmc(out)
    for sub in _CALL_TRACES:
        if glob.glob(f"{out}/{sub}/**/*kernel_trace.csv", recursive=True):
            _summarize_call_trace(out, sub)
    _summarize_presets(out)
    if not glob.glob(f"{out}/prof_factory/**/*kernel_stats.csv", recursive=True):
        return
    stats = _csv_rows(f"{out}/prof_factory/**/*kernel_stats.csv")
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# Kernel-time summary: factory_b256 workload (256 ragged requests, pi0-shaped expert, bf16)", "",
             "Command (one MI355X, repository root, library built in-tree; one lane, so every dispatch",
             "runs alone as in bench.py's per-kernel timing pass):", "", "```",
             f"export TMPDIR=/tmp; rocprofv3 --kernel-trace --stats --output-format csv -d {out}/prof_factory "
             "-o factory -- python -u bench.py --steps 3 --warmup 1 --no-cpu-baseline --lanes 1", "```", "",
             "The profiled process runs 1 warm-up + 3 timed + 2 per-kernel-timing generate calls (6 calls).",
             "Table from `factory_kernel_stats.csv`, sorted by total time.", "",
             "| Kernel | Calls | Avg (us) | Total (ms) | % |", "|---|---:|---:|---:|---:|"]
    for r in stats:
        name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0]
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    open(os.path.join(PROFILES, "kernel_stats_factory_b256.md"), "w").write("\n".join(lines) + "\n")

    fetch, nf = _counter_avg(_csv_rows(f"{out}/pmc_fetch/**/*counter_collection.csv"), "void rosa::attention_bf16")
    write, nw = _counter_avg(_csv_rows(f"{out}/pmc_write/**/*counter_collection.csv"), "void rosa::attention_bf16")
    cf, _ = _counter_avg(_csv_rows(f"{out}/pmc_cfetch/**/*counter_collection.csv"), "__amd_rocclr_copyBuffer")
    cw, _ = _counter_avg(_csv_rows(f"{out}/pmc_cwrite/**/*counter_collection.csv"), "__amd_rocclr_copyBuffer")
    gib_kib = float(1 << 20)
    ff, wf = gib_kib / cf, gib_kib / cw
    rd, wr = fetch * ff * 1024, write * wf * 1024
    sha = hashlib.sha256(open(os.path.join(ROOT, "paper_2607_01088_amd", "csrc", "k_attn.hip"), "rb").read())
    t = {"kernel": "attention", "workload": "factory_b256", "source_sha": sha.hexdigest()[:16], "dispatches": nf,
         "fetch_size_kib_avg": round(fetch, 1), "write_size_kib_avg": round(write, 1),
         "copy_probe_fetch_kib": round(cf, 1), "copy_probe_write_kib": round(cw, 1),
         "fetch_factor": round(ff, 4), "write_factor": round(wf, 4), "hbm_bytes_per_launch": int(rd + wr)}
    json.dump(t, open(os.path.join(PROFILES, "traffic_attention_factory_b256.json"), "w"), indent=1)
    md = ["# HBM traffic of the attention kernel, factory_b256 workload", "",
          "Commands (one MI355X, repository root, library built in-tree; one counter per run, one lane):", "", "```",
          "export TMPDIR=/tmp",
          f"timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE --output-format csv -d {out}/pmc_fetch -o f -- "
          "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
          f"timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE --output-format csv -d {out}/pmc_write -o w -- "
          "python -u bench.py --steps 1 --warmup 0 --no-cpu-baseline --lanes 1",
          f"timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv -d {out}/pmc_cfetch -o f -- "
          "python -u bench.py --copy-probe",
          f"timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv -d {out}/pmc_cwrite -o w -- "
          "python -u bench.py --copy-probe",
          f"python bench.py --summarize-profiles {out}", "```", "",
          f"Calibration: the copy probe reads and writes 1 GiB (1048576 KiB) per launch; FETCH_SIZE reads "
          f"{cf:.1f} KiB and WRITE_SIZE {cw:.1f} KiB per dispatch, so FETCH_SIZE is scaled by {ff:.4f} and "
          f"WRITE_SIZE by {wf:.4f}.", "",
          "| Kernel | Dispatches | FETCH_SIZE (KiB, avg) | WRITE_SIZE (KiB, avg) | HBM read (MB) | HBM write (MB) |",
          "|---|---:|---:|---:|---:|---:|",
          f"| `rosa::attention_bf16_kernel<256, 1, false>` | {nf} | {fetch:.1f} | {write:.1f} | {rd / 1e6:.1f} | {wr / 1e6:.1f} |",
          *_traffic_rows(out, ff, wf),
          "", f"Per launch: {(rd + wr) / 1e6:.1f} MB of HBM traffic.  Algorithmic bytes per launch (each active "
          "request's prefix K and V of the layer read once) are 174 MB averaged over the 180 launches of one call; "
          "queries, action keys and the output add about 26 MB written and 30 MB read.", "",
          f"Kernel source sha256 (first 16 hex digits) of `k_attn.hip` when measured: `{t['source_sha']}`."]
    open(os.path.join(PROFILES, "traffic_attention_factory_b256.md"), "w").write("\n".join(md) + "\n")
    print(json.dumps(t))


def copy_probe(torch):
    """A plain copy of known size: each launch reads and writes exactly 1 GiB.
    Its FETCH_SIZE / WRITE_SIZE readings give the factor that turns those
    counters into bytes for the other kernels."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read_per_launch": n, "copy_probe_bytes_written_per_launch": n,
                      "launches": 5}), flush=True)


def measured_peaks(torch, rosa):
    """Attainable peaks on this GPU, taken after the timed region: a plain
    512 MiB device-to-device copy (read + write bytes per second, best of 5)
    and the library's MFMA-only loop (dense bf16, rosa_debug_mfma_peak)."""
    n = 512 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = 0.0
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, 2 * n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del src, dst
    return {"hbm_copy_gbs": round(best, 1), "mfma_bf16_tflops": round(rosa.mfma_peak(torch.cuda.current_device()), 1),
            "how": "best of 5 timed 512 MiB device-to-device copies (2 x bytes / time); "
                   "rosa_debug_mfma_peak (back-to-back 32x32x16 bf16 MFMAs, 2 waves per SIMD on every CU)"}


def batch_profile(torch, rosa, expert, db, reqs, preset, args):
    """Latency / throughput of one call per batch size B (the first B requests
    of the workload, the System-1 batching profile of the paper's scheduler),
    then the library's batch-size choice for closed-loop fleets."""
    sizes, rows = [], []
    B = len(reqs)
    b = 1
    while b <= B:
        sizes.append(b)
        b *= 2
    stream = torch.cuda.current_stream()
    for b in sizes:
        sub = db.structs[:b]
        for _ in range(max(2, args.warmup)):
            expert.generate(sub)
        n = max(5, args.steps)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        torch.cuda.synchronize()
        for e0, e1 in evs:
            e0.record(stream)
            expert.generate(sub)
            e1.record(stream)
        torch.cuda.synchronize()
        lat = np.array([e0.elapsed_time(e1) for e0, e1 in evs])
        rows.append({"batch": b, "p50_ms": round(float(np.percentile(lat, 50)), 3),
                     "p99_ms": round(float(np.percentile(lat, 99)), 3),
                     "chunks_per_s": round(b / (lat.mean() * 1e-3), 1),
                     "actions_per_s": round(sum(r.horizon for r in reqs[:b]) / (lat.mean() * 1e-3), 1)})
        print(f"[bench] B={b}: p50 {rows[-1]['p50_ms']} ms, {rows[-1]['chunks_per_s']} chunks/s",
              file=sys.stderr, flush=True)
    ms = [r["p50_ms"] for r in rows]
    choices = []
    for robots in [1, 16, 64, 256]:
        for t_act in [50.0, 200.0]:
            for slo in [0.0, 200.0]:
                best, outs = rosa.s1_select_batch(sizes, ms, robots, t_act, slo, 2000)
                entry = {"robots": robots, "t_act_ms": t_act, "slo_ms": slo,
                         "batch": None if best is None else sizes[best]}
                if best is not None:
                    o = outs[best]
                    one = outs[0]
                    entry.update({"action_rate_hz": round(o["action_rate_hz"], 2),
                                  "throughput_hz": round(o["throughput_hz"], 1),
                                  "p99_ms": round(o["latency_p99_ms"], 2),
                                  "gain_vs_batch1": round(o["throughput_hz"] / one["throughput_hz"], 2)
                                  if one["feasible"] else None})
                choices.append(entry)
    # Homogeneous fleet schedules on a node of 8 such GPUs: System-1 latency
    # profiles L(b, rate) simulated from the measured call times, then the
    # binary search on the shared action rate (System 1 only: no System-2 or
    # obligation models are served here).
    profile = [(b, rosa.rate_profile(b, t, n_rates=10, n_requests=max(4000, 40 * b), seed=1))
               for b, t in zip(sizes, ms)]
    schedules = []
    for robots in [16, 64, 256, 1024]:
        for t_act in [50.0, 200.0]:
            s1 = {"role": rosa.ROSA_ROLE_S1, "deadline_ms": 200.0, "profile": profile}
            t0 = time.perf_counter()
            out = rosa.schedule_homogeneous({"robots": robots, "servers": 8, "t_act_ms": t_act, "horizon": 1,
                                             "eps_hz": 1e-2}, [s1])
            solve_s = time.perf_counter() - t0
            servers = {}
            for _, (b, k, mean, slo) in out["assignment"]:
                servers.setdefault((b, k), [0, mean, slo])[0] += 1
            schedules.append({"robots": robots, "t_act_ms": t_act, "feasible": out["feasible"],
                              "f_hz": round(out["f_hz"], 3), "l_s1_ms": round(out["l_s1_ms"], 2),
                              "fleet_chunks_per_s": round(out["f_hz"] * robots, 1),
                              "bound_zero_latency_hz": round(1000.0 / t_act, 3),
                              "servers": [{"batch": b, "streams": k, "count": c, "mean_ms": round(mn, 2),
                                           "p99_ms": round(sl, 2)} for (b, k), (c, mn, sl) in sorted(servers.items())],
                              "solve_s": round(solve_s, 3)})
            print(f"[bench] schedule robots={robots} t_act={t_act}: f={out['f_hz']:.2f} Hz "
                  f"({solve_s:.2f} s)", file=sys.stderr, flush=True)
    print(json.dumps({"kind": "s1_batch_profile", "workload": preset.name, "dtype": preset.dtype,
                      "profile": rows, "choices": choices, "homogeneous_schedules": schedules,
                      "schedule_model": "8 servers (GPUs) like this one, System 1 only, p99 deadline 200 ms; "
                                        "L(b, rate) simulated from the measured p50 call times (Poisson arrivals, "
                                        "a batch waits for b requests), ten rates per batch size",
                      "server_model": "closed loop, FIFO, a batch starts when the worker is idle and B "
                                      "requests wait; batch latency = measured p50"}), flush=True)


def step_batching(torch, rosa, expert, db, reqs, preset, args, n_req=1024, seed=0):
    """One worker serving requests that arrive at exponential intervals (the
    workload's request mix, cycling over its resident prefixes).  The clock is
    virtual: it advances by each call's measured duration (HIP events), so
    every call runs on the GPU and queueing follows from the measurements.
      whole: when idle, the worker takes every waiting request (up to the
        handle's capacity) and runs their whole chunks (rosa_generate_actions);
      step: every call advances all requests in flight by one Euler step
        (rosa_generate_steps); arrivals join, finished requests leave, between
        calls.
    Latency = completion - arrival."""
    rng = np.random.default_rng(seed)
    arrive = np.cumsum(rng.exponential(1000.0 / args.arrival_rate, n_req))     # ms
    src = [i % len(reqs) for i in range(n_req)]
    outs = [torch.empty_like(db.noise[j]) for j in src]
    cap_n = len(reqs)
    cap_tok = sum(r.horizon for r in reqs)
    stream = torch.cuda.current_stream()

    def struct(i, done):
        j = src[i]
        r = reqs[j]
        return rosa.request_struct(db.k[j], db.v[j], db.noise[j] if done == 0 else None, outs[i],
                                   r.prefix_len, r.horizon, r.steps, done)

    def timed_call(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1)

    def run(mode):
        t, nxt = 0.0, 0
        waiting, flight, done_steps = [], [], {}
        finish = np.zeros(n_req)
        calls, sizes = 0, []
        while nxt < n_req or waiting or flight:
            while nxt < n_req and arrive[nxt] <= t:
                waiting.append(nxt)
                nxt += 1
            if mode == "whole":
                if not waiting:
                    t = arrive[nxt]
                    continue
                batch, tok = [], 0
                while waiting and len(batch) < cap_n and tok + reqs[src[waiting[0]]].horizon <= cap_tok:
                    tok += reqs[src[waiting[0]]].horizon
                    batch.append(waiting.pop(0))
                t += timed_call(lambda: expert.generate([struct(i, 0) for i in batch]))
                finish[batch] = t
                sizes.append(len(batch))
            else:
                tok = sum(reqs[src[i]].horizon for i in flight)
                while waiting and len(flight) < cap_n and tok + reqs[src[waiting[0]]].horizon <= cap_tok:
                    tok += reqs[src[waiting[0]]].horizon
                    i = waiting.pop(0)
                    done_steps[i] = 0
                    flight.append(i)
                if not flight:
                    t = arrive[nxt]
                    continue
                t += timed_call(lambda: expert.generate_steps([struct(i, done_steps[i]) for i in flight], 1))
                sizes.append(len(flight))
                keep = []
                for i in flight:
                    done_steps[i] += 1
                    if done_steps[i] == reqs[src[i]].steps:
                        finish[i] = t
                    else:
                        keep.append(i)
                flight = keep
            calls += 1
        lat = finish - arrive
        return {"chunks_per_s": round(n_req / ((finish.max() - arrive[0]) * 1e-3), 1),
                "latency_mean_ms": round(float(lat.mean()), 2),
                "latency_p50_ms": round(float(np.percentile(lat, 50)), 2),
                "latency_p99_ms": round(float(np.percentile(lat, 99)), 2),
                "calls": calls, "mean_requests_per_call": round(float(np.mean(sizes)), 1)}

    for _ in range(2):                         # warm-up of both paths
        expert.generate([struct(0, 0)])
        expert.generate_steps([struct(0, 0)], 1)
    torch.cuda.synchronize()
    res = {m: run(m) for m in ["whole", "step"]}
    print(json.dumps({"kind": "step_batching", "workload": preset.name, "requests": n_req,
                      "arrival_rate_per_s": args.arrival_rate, "whole_chunk_batches": res["whole"],
                      "step_level_batches": res["step"],
                      "clock": "virtual: advanced by each call's measured duration"}), flush=True)


def visible_keys(P: int, c: int) -> float:
    """Sum over a job's tokens of the keys each sees: P^2 when bidirectional;
    with a causal segment of the last c tokens, b^2 + (b+1) + ... + P for
    b = P - c."""
    b = P - c
    return float(b) * b + (float(P) * (P + 1) - float(b) * (b + 1)) / 2.0


def prefill_work(shape, lens, head_layers: int = 0, causal=None):
    """Algorithmic flops of one prefix-producer call by kernel class.  Per-layer
    form: every layer's QKV projection; the attention, output projection and
    MLP of all layers but the last (its caches need only its K and V).
    Context form (head_layers > 0): every layer in full, plus the context
    projection for every head layer (counted with the QKV class, the same
    kernel class).  Attention: 4 * n_q * hd * (visible keys summed over the
    job's tokens: P^2 without a causal segment) per job and layer."""
    L, d, nq, nkv, hd, dff = (shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                              shape.d_mlp)
    M = float(sum(lens))
    Lb = L if head_layers else L - 1
    return {
        "gemm_qkv": 2.0 * M * d * shape.qkv_dim * L + 2.0 * M * d * head_layers * 2 * nkv * hd,
        "gemm_o": 2.0 * M * nq * hd * d * Lb,
        "gemm_up": 2.0 * M * d * dff * Lb,
        "gemm_down": 2.0 * M * dff * d * Lb,
        "attention": 4.0 * nq * hd * sum(visible_keys(P, c) for P, c in zip(lens, causal or [0] * len(lens))) * Lb,
    }


def prefill_cpu_baseline(shape, weights, xs, lens, budget_s: float, wctx=None, causal=None):
    """The oracle backbone on a bounded sample: whole jobs of the batch, in
    order, until budget_s seconds have been spent; scaled to the whole batch by
    algorithmic flops (the oracle's cost is additive over jobs)."""
    from oracle import prefill, prefill_context
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    # the oracle runs every layer in full: 2 * (qkv + o + up + down) per token and layer, plus attention
    per_tok = 2.0 * (shape.d_model * shape.qkv_dim + shape.n_q_heads * shape.head_dim * shape.d_model
                     + 2 * shape.d_model * shape.d_mlp)
    ctx_tok = 0.0 if wctx is None else 2.0 * shape.d_model * wctx.shape[0] * wctx.shape[2]
    causal = causal or [0] * len(lens)
    flops = lambda P, c: (shape.n_layers * (per_tok * P + 4.0 * shape.n_q_heads * shape.head_dim * visible_keys(P, c))
                          + ctx_tok * P)
    t_used, done = 0.0, 0
    for x, c in zip(xs, causal):
        t0 = time.perf_counter()
        if wctx is None:
            prefill(x, weights, shape, causal_len=c)
        else:
            prefill_context(x, weights, shape, wctx, causal_len=c)
        t_used += time.perf_counter() - t0
        done += 1
        if t_used >= budget_s:
            break
    batch_s = t_used * (sum(flops(P, c) for P, c in zip(lens, causal))
                        / sum(flops(P, c) for P, c in zip(lens[:done], causal[:done])))
    return {"value": sum(lens) / batch_s, "unit": "prefix tokens/s", "cores": int(blas_threads),
            "host_cores_available": len(os.sched_getaffinity(0)), "kind": "oracle",
            "sample": (f"{done} of {len(lens)} jobs ({sum(lens[:done])} tokens, all {shape.n_layers} layers), "
                       f"{t_used:.1f} s measured, scaled to the whole batch by algorithmic flops "
                       f"(extrapolated batch time {batch_s:.1f} s); NumPy float64")}


def prefill_bench(torch, rosa, args):
    """The prefix producer (a PaliGemma-sized VLM backbone, bf16) over one
    batch of robots' embedded prefixes; value = prefix tokens/s."""
    from synthetic import PI0_VLM, make_context_weights, make_prefix_embeddings, make_vlm_weights, prefill_lengths
    shape = PI0_VLM
    if args.prefill_rope:
        import dataclasses
        shape = dataclasses.replace(shape, rope_base=args.prefill_rope)
    lens = prefill_lengths()
    context = args.prefill_cache == "context"
    head_layers = 18
    cache_layers = head_layers if context else shape.n_layers
    t0 = time.time()
    weights = make_vlm_weights(shape, "bf16")
    wctx = make_context_weights(shape, head_layers, "bf16") if context else None
    xs = [make_prefix_embeddings(shape, P, "bf16", 4000 + i) for i, P in enumerate(lens)]
    print(f"[bench] generated backbone weights and {len(lens)} prefixes in {time.time() - t0:.1f} s",
          file=sys.stderr, flush=True)
    emb = [torch.from_numpy(x).to(torch.bfloat16).cuda() for x in xs]
    kc = [torch.empty((cache_layers, P, shape.n_kv_heads, shape.head_dim), dtype=torch.bfloat16,
                      device="cuda") for P in lens]
    vc = [torch.empty_like(k) for k in kc]
    causal = [min(args.prefill_causal, P) for P in lens]
    jobs = [rosa.prefix_job(e, k, v, P, c) for e, k, v, P, c in zip(emb, kc, vc, lens, causal)]
    pp = rosa.PrefixProducer(shape, "bf16", weights, len(lens), sum(lens), context_weights=wctx)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        pp.run(jobs)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t_start = time.perf_counter()
    for a, b in evs:
        a.record(stream)
        pp.run(jobs)
        b.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    lat = np.array([a.elapsed_time(b) for a, b in evs])
    print(f"[bench] timed {args.steps} prefill calls: {elapsed:.3f} s", file=sys.stderr, flush=True)

    pp.set_profiling(True)
    n_prof = 2
    for _ in range(n_prof):
        pp.run(jobs)
    prof = pp.profile()
    pp.set_profiling(False)
    work = prefill_work(shape, lens, head_layers if context else 0, causal)
    kernels = {}
    for name, (launches, ms) in prof.items():
        if launches == 0:
            continue
        per_call = launches / n_prof
        avg_ms = ms / launches
        entry = {"launches_per_call": per_call, "avg_launch_ms": avg_ms, "ms_per_call": ms / n_prof}
        if name in work:
            ach = work[name] / per_call / (avg_ms * 1e-3) / 1e12
            entry.update({"bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                          "frac": ach / MFMA_BF16_PEAK_TFS})
        kernels[name] = entry
    dom = max((k for k in kernels if "bound" in kernels[k]), key=lambda k: kernels[k]["ms_per_call"])
    d = kernels[dom]
    total_flops = sum(work.values())
    ms_per_step = elapsed / args.steps * 1e3
    out = {
        "metric": "prefix tokens/s of the VLM prefix producer (per-layer K/V caches for the action expert)",
        "value": round(sum(lens) * args.steps / elapsed, 1),
        "unit": "prefix tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "vlm_prefill_b32" + ("_context" if context else "")
                   + (f"_causal{args.prefill_causal}" if args.prefill_causal else "")
                   + ("_rope" if args.prefill_rope else ""), "jobs": len(lens),
                   "prefix_tokens": int(sum(lens)), "cache_form": args.prefill_cache,
                   "causal_segment_tokens": args.prefill_causal, "rope_base": args.prefill_rope,
                   "backbone": "18 layers, width 2048, 8 query heads / 1 KV head of 256, MLP 16384"},
        "jobs_per_s": round(len(lens) * args.steps / elapsed, 2),
        "p50_ms": round(float(np.percentile(lat, 50)), 3),
        "p99_ms": round(float(np.percentile(lat, 99)), 3),
        "roofline": {"kernel": dom, "bound": d["bound"], "achieved": round(d["achieved"], 2), "peak": d["peak"],
                     "unit": d["unit"], "frac": round(d["frac"], 4), "traffic": None},
        "all_mfma": {"achieved": round(total_flops / (ms_per_step * 1e-3) / 1e12, 1), "peak": MFMA_BF16_PEAK_TFS,
                     "unit": "TFLOP/s", "frac": round(total_flops / (ms_per_step * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4)},
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kernels.items()},
    }
    pp.close()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = prefill_cpu_baseline(shape, weights, xs, lens, args.cpu_budget, wctx, causal)
    print(json.dumps(out), flush=True)


def pipeline_bench(torch, rosa, args):
    """The whole System-1 path for a batch of robots: the VLM backbone fills
    their prefix caches, then the action expert generates their chunks from
    them, back to back on one stream (32 robots, prefixes of 600..1024
    tokens, horizon 50, 10 Euler steps).  value = robot requests served per
    second; the two phases are timed separately too."""
    from synthetic import PI0_SHAPE, PI0_VLM, make_prefix_embeddings, make_vlm_weights, make_weights, prefill_lengths
    lens = prefill_lengths()
    H, K, A = 50, 10, PI0_SHAPE.action_dim
    vw = make_vlm_weights(PI0_VLM, "bf16")
    ew = make_weights(PI0_SHAPE, "bf16")
    emb = [torch.from_numpy(make_prefix_embeddings(PI0_VLM, P, "bf16", 4000 + i)).to(torch.bfloat16).cuda()
           for i, P in enumerate(lens)]
    kc = [torch.empty((PI0_SHAPE.n_layers, P, 1, PI0_SHAPE.head_dim), dtype=torch.bfloat16, device="cuda")
          for P in lens]
    vc = [torch.empty_like(k) for k in kc]
    rng = np.random.default_rng(5)
    nz = [torch.from_numpy(rng.standard_normal((H, A)).astype(np.float32)).cuda() for _ in lens]
    out = [torch.empty_like(n) for n in nz]
    pp = rosa.PrefixProducer(PI0_VLM, "bf16", vw, len(lens), sum(lens))
    ex = rosa.ActionExpert(PI0_SHAPE, "bf16", ew, rosa.capacity(len(lens), H, H * len(lens), K, sum(lens)))
    jobs = [rosa.prefix_job(e, k, v, P) for e, k, v, P in zip(emb, kc, vc, lens)]
    reqs = [rosa.request_struct(k, v, n, o, P, H, K) for k, v, n, o, P in zip(kc, vc, nz, out, lens)]
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        pp.run(jobs)
        ex.generate(reqs)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b, c in evs:
        a.record(stream)
        pp.run(jobs)
        b.record(stream)
        ex.generate(reqs)
        c.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    pre = np.array([a.elapsed_time(b) for a, b, _ in evs])
    gen = np.array([b.elapsed_time(c) for _, b, c in evs])
    tot = np.array([a.elapsed_time(c) for a, _, c in evs])
    pp.close()
    ex.close()
    print(json.dumps({
        "metric": "robot requests/s through VLM prefill + action generation (System-1 path)",
        "value": round(len(lens) * args.steps / elapsed, 2), "unit": "requests/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "s1_pipeline_b32", "robots": len(lens), "prefix_tokens": int(sum(lens)),
                   "horizon": H, "steps": K},
        "prefill_ms_p50": round(float(np.percentile(pre, 50)), 3),
        "generate_ms_p50": round(float(np.percentile(gen, 50)), 3),
        "total_ms_p50": round(float(np.percentile(tot, 50)), 3),
        "total_ms_p99": round(float(np.percentile(tot, 99)), 3)}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="factory_b256")
    ap.add_argument("--first", type=int, default=0, metavar="N",
                    help="only the first N requests of the workload (a smaller batch of the same mix)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lanes", type=int, default=0,
                    help="concurrent sub-batches per call (0: the library default); the per-kernel timing "
                         "pass always runs one lane")
    ap.add_argument("--batch-profile", action="store_true",
                    help="System-1 batch-size profile: latency and throughput of one call on the first B "
                         "requests of the workload for B = 1, 2, 4, ..., then the batch size the library "
                         "chooses for a few robot fleets (prints its own JSON line)")
    ap.add_argument("--step-batching", action="store_true",
                    help="open-loop request arrivals served by one worker with whole-chunk batches vs "
                         "step-level batches (rosa_generate_steps); prints its own JSON line")
    ap.add_argument("--arrival-rate", type=float, default=2000.0, help="requests per second for --step-batching")
    ap.add_argument("--attention-layout", choices=["joint", "alternating"], default="joint",
                    help="the expert's attention layout: joint prefix + action attention in every layer, or "
                         "alternating cross-attention (even layers) and self-attention (odd layers)")
    ap.add_argument("--prefill", action="store_true",
                    help="the prefix producer instead: a VLM backbone over 32 robots' prefixes "
                         "(prints its own JSON line)")
    ap.add_argument("--pipeline", action="store_true",
                    help="the whole System-1 path: VLM prefill then action generation for 32 robots "
                         "(prints its own JSON line)")
    ap.add_argument("--prefill-causal", type=int, default=0, metavar="C",
                    help="with --prefill: each job's last C tokens (at most P) form a causal segment")
    ap.add_argument("--prefill-rope", type=float, default=0.0, metavar="BASE",
                    help="with --prefill: rotary position embedding of the backbone's queries and keys")
    ap.add_argument("--prefill-cache", choices=["per_layer", "context"], default="per_layer",
                    help="with --prefill: per-layer backbone K/V, or the context form (the backbone's "
                         "normalised output projected for every layer of an 18-layer cross-attending head)")
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="write the profiles/ summaries from rocprofv3 outputs under DIR and exit (no GPU)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (calibrates HBM byte counters)")
    args = ap.parse_args()
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported (requests shard across GPUs "
              "with no exchange, so each GPU's share is measured on its own).", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe:
        copy_probe(torch)
        return
    from paper_2607_01088_amd import rosa
    if args.prefill:
        prefill_bench(torch, rosa, args)
        return
    if args.pipeline:
        pipeline_bench(torch, rosa, args)
        return
    from synthetic import PRESETS, make_metadata, make_requests, make_weights

    preset = PRESETS[args.workload]
    workload = preset.name
    if args.attention_layout == "alternating":
        import dataclasses
        preset = dataclasses.replace(preset, shape=dataclasses.replace(preset.shape, attention_layout=1))
        workload += "_alternating"
    t0 = time.time()
    weights = make_weights(preset.shape, preset.dtype)
    meta = make_metadata(preset)
    reqs = make_requests(preset, threads=16)
    if args.first > 0:
        reqs, meta = reqs[:args.first], meta[:args.first]
        workload += f"_first{args.first}"
    print(f"[bench] generated inputs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    cap = rosa.capacity(len(reqs), max(r.horizon for r in reqs), sum(r.horizon for r in reqs),
                        max(r.steps for r in reqs), sum(r.prefix_len for r in reqs))
    expert = rosa.ActionExpert(preset.shape, preset.dtype, weights, cap)
    if args.lanes > 0:
        expert.set_lanes(args.lanes)
    db = rosa.DeviceBatch(reqs, preset.dtype)
    kv_bytes = sum(k.numel() * k.element_size() * 2 for k in db.k if k is not None)
    torch.cuda.synchronize()
    print(f"[bench] uploaded (prefix KV {kv_bytes / 1e9:.2f} GB resident)", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    if args.batch_profile:
        batch_profile(torch, rosa, expert, db, reqs, preset, args)
        expert.close()
        return
    if args.step_batching:
        step_batching(torch, rosa, expert, db, reqs, preset, args)
        expert.close()
        return
    for _ in range(args.warmup):
        expert.generate(db.structs)
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for a, b in evs:
        a.record(stream)
        expert.generate(db.structs)
        b.record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    lat = np.array([a.elapsed_time(b) for a, b in evs])
    print(f"[bench] timed {args.steps} calls: {elapsed:.3f} s", file=sys.stderr, flush=True)

    # Per-kernel durations, live, with HIP events on the library's stream.
    expert.set_profiling(True)
    n_prof = 2
    for _ in range(n_prof):
        expert.generate(db.structs)
    prof = expert.profile()
    expert.set_profiling(False)

    gemm_flops, attn_bytes, attn_flops, tok_steps = algorithmic_work(preset.shape, reqs)
    kernels = {}
    for name, (launches, ms) in prof.items():
        if launches == 0:
            continue
        per_call_launches = launches / n_prof
        avg_ms = ms / launches
        entry = {"launches_per_call": per_call_launches, "avg_launch_ms": avg_ms, "ms_per_call": ms / n_prof}
        if name in gemm_flops:
            per_launch = gemm_flops[name] / per_call_launches
            ach = per_launch / (avg_ms * 1e-3) / 1e12
            entry.update({"bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                          "frac": ach / MFMA_BF16_PEAK_TFS})
        elif name == "attention":
            per_launch = attn_bytes / per_call_launches
            ach = per_launch / (avg_ms * 1e-3) / 1e9
            entry.update({"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": ach / HBM_PEAK_GBS,
                          "mfma_tflops": attn_flops / per_call_launches / (avg_ms * 1e-3) / 1e12})
        kernels[name] = entry
    dom = max((k for k in kernels if "bound" in kernels[k]), key=lambda k: kernels[k]["ms_per_call"])
    d = kernels[dom]
    roofline = {"kernel": dom, "bound": d["bound"], "achieved": round(d["achieved"], 2), "peak": d["peak"],
                "unit": d["unit"], "frac": round(d["frac"], 4),
                "traffic": load_traffic(dom, workload)}
    gemm_total_ms = sum(kernels[k]["ms_per_call"] for k in gemm_flops if k in kernels)
    gemm_all = sum(gemm_flops.values()) / (gemm_total_ms * 1e-3) / 1e12

    peaks = measured_peaks(torch, rosa)
    mpeak = peaks["hbm_copy_gbs"] if roofline["bound"] == "hbm" else peaks["mfma_bf16_tflops"]
    roofline["frac_of_measured_peak"] = round(roofline["achieved"] / mpeak, 4) if mpeak else None

    B = len(reqs)
    ms_per_step = elapsed / args.steps * 1e3
    value = B * args.steps / elapsed
    out = {
        "metric": "action chunks/sec + p50/p99 batch latency at B=256; % HBM and MFMA peak",
        "value": round(value, 2),
        "unit": "chunks/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": workload, "requests": B, "attention_layout": args.attention_layout,
                   "action_tokens": int(sum(r.horizon for r in reqs)),
                   "prefix_tokens": int(sum(r.prefix_len for r in reqs)),
                   "token_steps": int(tok_steps)},
        "actions_per_s": round(sum(r.horizon for r in reqs) * args.steps / elapsed, 1),
        "p50_ms": round(float(np.percentile(lat, 50)), 3),
        "p99_ms": round(float(np.percentile(lat, 99)), 3),
        "roofline": roofline,
        "gemm_all": {"achieved": round(gemm_all, 1), "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                     "frac": round(gemm_all / MFMA_BF16_PEAK_TFS, 4),
                     "frac_of_measured_peak": round(gemm_all / peaks["mfma_bf16_tflops"], 4)
                     if peaks["mfma_bf16_tflops"] else None},
        "measured_peaks": peaks,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kernels.items()},
        "prefix_kv_gb": round(kv_bytes / 1e9, 3),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(preset, weights, meta, args.cpu_budget)
    expert.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
