"""Decode-step MoE benchmark on one MI355X.

One step = one decode token through every MoE layer of the stack: router GEMV
+ softmax top-k, predictor verify/update and next-layer prediction, expert
residency, and the bf16 SwiGLU expert FFN.  Inputs (router rows, expert
weights, every token's hidden states) are resident in HBM before timing.

Default workload: the Mixtral-8x7B-shaped stack (32 layers, hidden 4096,
intermediate 14336, 8 experts top-2, bf16, batch 1), seeded synthetic data.

Besides the timed HBM-resident run the JSON line carries:
  roofline      the gate/up FFN kernel's algorithmic bytes per launch over its
                event-timed average duration, against 8 TB/s
  offload       the same stack with the HBM cache capped (3 experts per layer
                for Mixtral shapes) and the other experts in pinned host
                memory: decode tokens/s on demand and with prediction-driven
                prefetch, stall per token, predictor hit rates, cache counts
  cpu_baseline  the CPU oracle timed on a bounded sample of the same workload

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config mixtral]
                       [--offload-tokens N] [--cpu-tokens S]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
#: the FFN launches of every TIMING_EVERY-th token of the timed region carry HIP events
TIMING_EVERY = 25


def timing_cadence(steps):
    """Tokens between event-timed tokens: TIMING_EVERY, or half the timed
    region when that is shorter (at least two timed tokens), 1 for a region
    of one to three tokens."""
    return max(1, min(TIMING_EVERY, steps // 2))


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="mixtral")
    ap.add_argument("--offload-tokens", type=int, default=16,
                    help="decode tokens per capped-cache mode (0 skips the offload runs)")
    ap.add_argument("--pinned-gb", type=float, default=56.0,
                    help="pinned host pool budget; larger stacks alias experts onto it")
    ap.add_argument("--cpu-tokens", type=int, default=64,
                    help="at most this many decode tokens of the CPU oracle sample (0 skips it)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="the CPU oracle sample stops after the token that reaches this much timed work")
    ap.add_argument("--offload-only", default=None, metavar="VARIANT[,VARIANT...]",
                    help="run only these capped-cache variants (and on-demand loading)")
    ap.add_argument("--pool", choices=("host", "hbm"), default="host",
                    help="backing pool of the capped cache: pinned host memory (PCIe) or the HBM-resident "
                         "stack (device-to-device copies, a faster tier)")
    ap.add_argument("--hbm-pool-gb", type=float, default=80.0,
                    help="for a stack larger than HBM: distinct expert blobs generated in HBM "
                         "(expert (l, e) reads blob (l*E + e) mod their number)")
    ap.add_argument("--attention-sweep", default=None, metavar="CTX1,CTX2,...",
                    help="capped cache with a decode-attention stand-in of these context lengths (markdown)")
    ap.add_argument("--handoff-probe", action="store_true",
                    help="producer -> consumer handoff as two launches or inside one launch (markdown) and exit")
    ap.add_argument("--copy-sweep", default=None, metavar="W1,W2,...",
                    help="capped cache with device decisions at these copy-kernel workgroup counts: the expert "
                         "tier's bandwidth as a measured sweep (markdown table; with --pool hbm up to TB/s)")
    ap.add_argument("--offload-sweep", default=None, metavar="C1,C2,...",
                    help="capped-cache sweep over these per-layer budgets (markdown table; no JSON line)")
    ap.add_argument("--counters", action="store_true",
                    help="run the fixed workload profiled by the rocprofv3 --pmc passes and exit")
    ap.add_argument("--counters-meta", default=None, metavar="JSON",
                    help="where --counters writes the profiled workload's shapes and call counts "
                         "(default counters_<config>.json in the working directory)")
    ap.add_argument("--predictor-sweep", action="store_true",
                    help="replay planted traces through the GPU predictor for every config and the paper's "
                         "Table 1 shapes; print recall/precision per ablation mode and exit")
    ap.add_argument("--predictor-spread", action="store_true",
                    help="recall/precision of the full predictor per workload over three trace seeds (markdown) "
                         "and exit")
    ap.add_argument("--ffn-sweep", action="store_true",
                    help="time moe_expert_ffn on every config shape, weights in no cache (markdown table on "
                         "stdout) and exit")
    ap.add_argument("--largest-tokens", type=int, default=10,
                    help="with the default workload, also decode the Qwen3-235B shapes (batch 16, HBM-resident "
                         "stand-in) for this many tokens after 2 warm-up tokens and report them in the JSON "
                         "line's 'largest_config' (0 skips)")
    ap.add_argument("--largest-capped-tokens", type=int, default=3,
                    help="tokens of the largest workload's capped-cache runs in 'largest_config' (0 skips)")
    ap.add_argument("--read-floor", action="store_true",
                    help="time one streaming-read launch per size, bytes in no cache (markdown table) and exit")
    ap.add_argument("--reread-probe", action="store_true",
                    help="streaming reads of bytes in no cache against bytes the Infinity Cache may hold (phase "
                         "order as markdown; durations from a kernel trace) and exit")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("KERNEL_TRACE_CSV", "TITLE", "COMMAND"),
                    help="median kernel durations per kernel and grid size of a rocprofv3 kernel trace")
    ap.add_argument("--summarize-mfma", nargs=2, metavar=("COUNTER_CSV", "COMMAND"),
                    help="MfmaUtil / bf16 MFMA operations of the MFMA kernels in a rocprofv3 --pmc pass")
    ap.add_argument("--summarize-policy", metavar="POLICY_BOUND_MD",
                    help="pivot a --policy-bound table by workload, link rate and attention window")
    ap.add_argument("--summarize-floor", nargs=2, metavar=("READ_FLOOR_TRACE_CSV", "FFN_SWEEP_TRACE_CSV"),
                    help="the read floor by size beside the FFN sweep's kernels (markdown)")
    ap.add_argument("--summarize-stats", nargs=3, metavar=("STATS_CSV", "TITLE", "COMMAND"),
                    help="print a markdown table of a rocprofv3 kernel_stats.csv and exit")
    ap.add_argument("--summarize-overlap", nargs=2, metavar=("KERNEL_CSV", "COPY_CSV"),
                    help="copy/compute overlap of the capped-cache runs in a rocprofv3 trace")
    ap.add_argument("--summarize-offload", nargs="+", metavar="BENCH_JSON",
                    help="print a markdown table of the capped-cache runs in bench JSON lines and exit")
    ap.add_argument("--policy-bound", default=None, metavar="CONFIG[,CONFIG...]",
                    help="time-model bound of one-layer-lookahead prefetch policies on the planted traces")
    ap.add_argument("--policy-attn", default="0", metavar="MS1,MS2,...",
                    help="attention windows (ms per layer) for --policy-bound")
    ap.add_argument("--policy-link", default="measured", metavar="GBPS1,GBPS2,...",
                    help="link rates for --policy-bound: 'measured' and/or GB/s (copy time = blob bytes / rate)")
    ap.add_argument("--summarize-gaps", nargs=3, metavar=("KERNEL_TRACE_CSV", "TITLE", "COMMAND"),
                    help="print the compute-queue gap analysis of a rocprofv3 kernel trace as markdown")
    ap.add_argument("--summarize-counters", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "META_JSON"),
                    help="print the markdown counter summary of two rocprofv3 --pmc runs and exit")
    return ap.parse_args()


COUNTERS_MD = os.path.join(ROOT, "profiles", "ffn_gate_up_mixtral8x7b_b1_counters.md")
POOL_TIER = "host"      # set from --pool
FFN_SOURCES = [os.path.join(ROOT, "paper_2606_15453_amd", "csrc", f)
               for f in ("expert_ffn.hip", "gating_dev.h", "common.h")]
CALIB_BYTES = 1 << 30
COUNTER_TOKENS = 20


def strip_c_comments(text):
    """C/C++ source without its comments (// to the end of the line and
    /* ... */), string and character literals kept as they are."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return "".join(out)


def ffn_source_sha():
    """Hash of the code the gate/up kernel is built from (the FFN kernels,
    the gating steps of their routing prologue, the shared helpers), comments
    removed: an edit of a comment leaves the kernel and its counters as
    they were."""
    import hashlib
    h = hashlib.sha256()
    for path in FFN_SOURCES:
        with open(path, encoding="utf-8") as f:
            h.update(strip_c_comments(f.read()).encode())
    return h.hexdigest()[:16]


def committed_traffic():
    """HBM bytes per ffn_gate_up launch from the committed counter summary, if
    it was taken on the current kernel source; else None."""
    try:
        lines = open(COUNTERS_MD).read().splitlines()
    except OSError:
        return None
    kv = dict(l.split(": ", 1) for l in lines if l.startswith(("traffic_bytes_per_launch: ", "expert_ffn_source_sha: ")))
    if kv.get("expert_ffn_source_sha") != ffn_source_sha():
        return None
    return int(kv["traffic_bytes_per_launch"])


def counter_means(path, counter):
    """Mean counter value per kernel name from a rocprofv3 counter_collection.csv."""
    import csv
    acc = {}
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") != counter:
            continue
        name = r["Kernel_Name"]
        v = float(r["Counter_Value"])
        s, n = acc.get(name, (0.0, 0))
        acc[name] = (s + v, n + 1)
    return {k: (s / n, n) for k, (s, n) in acc.items()}


def summarize_mfma(path, cmd):
    """Markdown: MfmaUtil and bf16 MFMA operations of the MFMA kernels in a
    rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_BF16 pass, per kernel
    and grid (one row per shape of the FFN sweep)."""
    import csv
    acc = {}
    for r in csv.DictReader(open(path)):
        name = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        if "mfma" not in name:
            continue
        key = (name.replace("stmoe::", ""), r.get("Grid_Size", "?"))
        d = acc.setdefault(key, {})
        s, n = d.get(r["Counter_Name"], (0.0, 0))
        d[r["Counter_Name"]] = (s + float(r["Counter_Value"]), n + 1)
    print("MFMA utilisation of the batched kernels (one counter pass over the FFN sweep):\n")
    print(f"```\n{cmd}\n```\n")
    print("| kernel | grid (threads) | dispatches | MfmaUtil (% of SIMD cycles with the MFMA unit busy) | "
          "MFMA bf16 flops per dispatch (MOPS x 512) |")
    print("|---|---|---|---|---|")
    for (name, grid), d in acc.items():
        u, n = d.get("MfmaUtil", (0.0, 0))
        m, nm = d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", (0.0, 0))
        print(f"| `{name}` | {grid} | {n} | {u / max(n, 1):.2f} | {m / max(nm, 1) * 512 / 1e9:.2f} G |")


def summarize_counters(fetch_csv, write_csv, meta_json):
    """Markdown summary of the FETCH_SIZE / WRITE_SIZE passes over the counters
    workload; meta_json is the file counters_workload wrote (shapes, FFN calls
    and distinct experts of the profiled tokens)."""
    meta = json.load(open(meta_json))
    f = counter_means(fetch_csv, "FETCH_SIZE")
    w = counter_means(write_csv, "WRITE_SIZE")

    def pick(d, key):
        m = [(k, v) for k, v in d.items() if key in k]
        if not m:
            raise SystemExit(f"no {key} dispatches in the counter file")
        return m[0][1]

    cf, _ = pick(f, "calib_copy_kernel")
    cw, _ = pick(w, "calib_copy_kernel")
    gf, n_g = pick(f, "ffn_gate_up")
    gw, _ = pick(w, "ffn_gate_up")
    df, _ = pick(f, "ffn_down")
    dw, _ = pick(w, "ffn_down")
    kf = CALIB_BYTES / (cf * 1024.0)
    kw = CALIB_BYTES / (cw * 1024.0)
    up_bytes = gf * 1024 * kf + gw * 1024 * kw
    dn_bytes = df * 1024 * kf + dw * 1024 * kw
    # algorithmic weight bytes per FFN call: distinct routed experts (+ shared)
    per_call = (meta["n_experts"] + meta["n_calls"] * meta["n_shared"]) / meta["n_calls"]
    mat = meta["H"] * meta["I"] * meta["esz"]
    alg_up = per_call * 2 * mat
    alg_dn = per_call * mat
    cfg = meta["config"]
    cmd_f = (f"rocprofv3 --pmc FETCH_SIZE -d $OUT/pmc_fetch -o fetch --output-format csv "
             f"-- python -u $R/bench.py --counters --config {cfg} --counters-meta $OUT/counters_{cfg}.json")
    cmd_w = cmd_f.replace("FETCH_SIZE", "WRITE_SIZE").replace("pmc_fetch", "pmc_write").replace("-o fetch", "-o write")
    out = [
        f"# HBM traffic counters: ffn_gate_up / ffn_down, {meta['title']}",
        "",
        "Commands (run from `/tmp` with `TMPDIR=/tmp`, repository at `$R`, output directory `$OUT`), one "
        "counter per run:",
        "",
        "```", cmd_f, cmd_w,
        f"python bench.py --summarize-counters <fetch counter_collection.csv> <write counter_collection.csv> "
        f"$OUT/counters_{cfg}.json",
        "```",
        "",
        f"The profiled workload runs {COUNTER_TOKENS} decode tokens of the HBM-resident stack ({per_call:.2f} "
        f"experts per FFN call on average, shared included) and then {CALIB_BYTES >> 30} GiB copies with "
        f"`stmoe_calib_copy` (reads and writes exactly {CALIB_BYTES} bytes each).  Counters are in KiB per "
        f"dispatch.",
        "",
        "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB |",
        "|---|---|---|---|",
        f"| `calib_copy_kernel` (1 GiB) | - | {cf:.0f} | {cw:.0f} |",
        f"| `ffn_gate_up` | {n_g} | {gf:.0f} | {gw:.0f} |",
        f"| `ffn_down` | - | {df:.0f} | {dw:.0f} |",
        "",
        f"Scale factors from the copy kernel: fetch {kf:.4f} bytes per counted byte, write {kw:.4f}.",
        "",
        f"ffn_gate_up: measured {up_bytes / 1e6:.2f} MB per launch against {alg_up / 1e6:.2f} MB algorithmic "
        f"({up_bytes / alg_up:.4f}x).",
        f"ffn_down: measured {dn_bytes / 1e6:.2f} MB per launch against {alg_dn / 1e6:.2f} MB algorithmic "
        f"({dn_bytes / alg_dn:.4f}x).",
        "",
        f"traffic_bytes_per_launch: {int(round(up_bytes))}",
        f"expert_ffn_source_sha: {ffn_source_sha()}",
    ]
    print("\n".join(out))


DECODE_KERNELS = ("route_logits_kernel", "route_tail_kernel", "route_update_predict_kernel", "ffn_gate_up",
                  "ffn_down", "ffn_reduce", "update_predict", "decide_kernel", "blit_kernel", "set_table_kernel")


def summarize_gaps(trace_csv, title, cmd, skip_frac=0.25):
    """Kernel-trace gap analysis of the decode layer on the compute queue:
    per kernel its average duration and the average idle time between the
    previous decode kernel's end and its start.  The window runs from the
    first to the last decode kernel on that queue; its first `skip_frac` of
    dispatches (warm-up) is dropped."""
    import csv
    rows = list(csv.DictReader(open(trace_csv)))
    key_q = "Queue_Id" if "Queue_Id" in rows[0] else "Stream_Id"

    def short(n):
        n = n.replace("(anonymous namespace)::", "").replace("void ", "").replace("stmoe::", "")
        return n.split("(")[0].split("<")[0]

    rows = [dict(name=short(r["Kernel_Name"]), q=r[key_q], s=int(r["Start_Timestamp"]),
                 e=int(r["End_Timestamp"])) for r in rows if r.get("End_Timestamp")]
    rows.sort(key=lambda r: r["s"])
    is_dec = lambda r: r["name"].startswith(DECODE_KERNELS)
    ffn_q = max(set(r["q"] for r in rows if r["name"].startswith("ffn_gate_up")),
                key=lambda q: sum(1 for r in rows if r["q"] == q))
    comp = [r for r in rows if r["q"] == ffn_q]
    idx = [i for i, r in enumerate(comp) if is_dec(r)]
    comp = [r for r in comp[idx[0]:idx[-1] + 1] if is_dec(r)]
    comp = comp[int(len(comp) * skip_frac):]
    while comp and not comp[0]["name"].startswith(("route", "ffn_gate_up")):
        comp = comp[1:]
    acc = {}
    for prev, cur in zip(comp, comp[1:]):
        d = acc.setdefault(cur["name"], [0, 0.0, 0.0])
        d[0] += 1
        d[1] += (cur["e"] - cur["s"]) / 1e3
        d[2] += max(cur["s"] - prev["e"], 0) / 1e3
    span = (comp[-1]["e"] - comp[0]["e"]) / 1e3
    busy = sum((r["e"] - r["s"]) / 1e3 for r in comp[1:])
    n_up = max(sum(1 for r in comp[1:] if r["name"].startswith("ffn_gate_up")), 1)
    out = [f"# {title}", "",
           "Command (run from `/tmp` with `TMPDIR=/tmp`, repository at `$R`):", "", "```", cmd,
           f"python bench.py --summarize-gaps <kernel_trace.csv> '<title>' '<command>'", "```", "",
           f"Compute queue, decode kernels only (the timed run's window, first {int(skip_frac * 100)}% dropped): "
           f"{len(comp)} dispatches, {n_up} layers.", "",
           "| kernel | dispatches | avg duration us | avg idle before it us |", "|---|---|---|---|"]
    for name, (n, dur, gap) in sorted(acc.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| `{name}` | {n} | {dur / n:.2f} | {gap / n:.2f} |")
    out += ["", f"Per layer: {span / n_up:.2f} us of wall time on the compute queue, {busy / n_up:.2f} us of it "
                f"inside kernels ({busy / span:.3f})."]
    print("\n".join(out))


def _union(iv):
    """Merge intervals [(s, e)] into disjoint sorted ones."""
    out = []
    for s_, e_ in sorted(iv):
        if out and s_ <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e_)
        else:
            out.append([s_, e_])
    return out


def _intersect_len(a, b):
    """Total length of the intersection of two disjoint sorted interval lists."""
    i = j = 0
    tot = 0
    while i < len(a) and j < len(b):
        lo, hi = max(a[i][0], b[j][0]), min(a[i][1], b[j][1])
        if hi > lo:
            tot += hi - lo
        if a[i][1] < b[j][1]:
            i += 1
        else:
            j += 1
    return tot


def summarize_overlap(kernel_csv, copy_csv):
    """Copy/compute overlap per capped-cache run of a rocprofv3 trace.

    A run is a cluster of routing launches (gaps under 300 ms); its window runs
    from its first routing launch to its last kernel, so the cache warm-up
    copies before it are excluded.  Expert copies are the host-to-device
    copies longer than 1 ms.  Overlap = time an expert copy is in flight while
    an FFN kernel runs, over the time any expert copy is in flight."""
    import csv
    ks = [(r["Kernel_Name"], int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
          for r in csv.DictReader(open(kernel_csv)) if "stmoe" in r["Kernel_Name"]]
    cs = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in csv.DictReader(open(copy_csv))
          if r["Direction"].endswith("HOST_TO_DEVICE")]
    cs = [c for c in cs if c[1] - c[0] > 1_000_000]
    routes = sorted(s_ for n, s_, e_ in ks if "route" in n)
    runs, cur = [], []
    for t in routes:
        if cur and t - cur[-1] > 300_000_000:
            runs.append(cur)
            cur = []
        cur.append(t)
    if cur:
        runs.append(cur)
    print("| run | window ms | expert copies | copy busy ms | FFN busy ms | copy time overlapped by FFN | "
          "FFN time overlapped by copies |")
    print("|---|---|---|---|---|---|---|")
    for n_run, r in enumerate(runs):
        w0 = r[0]
        w1 = max(e_ for n, s_, e_ in ks if s_ >= w0 and s_ <= r[-1] + 300_000_000)
        cp = _union([(max(a, w0), min(b, w1)) for a, b in cs if b > w0 and a < w1])
        if not cp:
            continue
        ffn = _union([(s_, e_) for n, s_, e_ in ks if "ffn_" in n and e_ > w0 and s_ < w1])
        cbusy = sum(b - a for a, b in cp)
        fbusy = sum(b - a for a, b in ffn)
        ov = _intersect_len(cp, ffn)
        n_cp = sum(1 for a, b in cs if a >= w0 and a < w1)
        print(f"| {n_run} | {(w1 - w0) / 1e6:.1f} | {n_cp} | {cbusy / 1e6:.1f} | {fbusy / 1e6:.1f} | "
              f"{ov / max(cbusy, 1):.3f} | {ov / max(fbusy, 1):.3f} |")


def summarize_offload(paths):
    """Markdown table of the capped-cache runs in bench JSON lines (one file
    per workload): per variant, tokens/s, stall beyond the HBM-resident step,
    its reduction against on-demand loading, copies and prediction quality."""
    print("| workload | C of E | variant | tokens/s | ms per token | stall ms per token | stall reduction "
          "vs on-demand | vs on-demand, same decisions and eviction | demand / overflow / prefetch (useful, "
          "wasted) copies | H2D GB/s | recall l>=1 / l=0 / precision |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for p in paths:
        d = json.loads(open(p).read().strip().splitlines()[-1])
        o = d.get("offload")
        if not o:
            continue
        cfg = d["config"]
        red = o.get("stall_reduction", {})
        runs = {n: r for n, r in o.items() if isinstance(r, dict) and "tokens_per_s" in r}

        def policy(r):
            return (r.get("device_decisions"), r.get("graph_replay"), r.get("eviction", "least recently used"))
        base = {policy(r): r for n, r in runs.items() if n.startswith("on_demand")}
        for name, r in runs.items():
            c = r["cache"]
            pq = (f"{r['recall_layers_ge1']:.3f} / {r['recall_layer0']:.3f} / {r['precision']:.3f}"
                  if "recall_layers_ge1" in r else "-")
            rd = red.get(name)
            b = base.get(policy(r))
            same = ("-" if name.startswith("on_demand") or b is None or b["stall_ms_per_token"] <= 0 else
                    f"{1.0 - r['stall_ms_per_token'] / b['stall_ms_per_token']:+.3f}")
            print(f"| {cfg['workload']} | {o['cache_slots_per_layer']} of {cfg['experts']} | {name} | "
                  f"{r['tokens_per_s']} | {r['ms_per_token']} | {r['stall_ms_per_token']} | "
                  f"{'-' if rd is None else f'{rd:+.3f}'} | {same} | {c['demand']} / {c['overflow']} / "
                  f"{c['prefetch']} ({c['useful']}, {c['wasted']}) | {r['h2d_gbps']} | {pq} |")


def summarize_stats(path, title, cmd):
    import csv
    print(f"# {title}\n")
    print(f"Command (run from `/tmp` with `TMPDIR=/tmp`, repository at `$R`):\n\n```\n{cmd}\n```\n")
    print("| kernel | calls | avg us | min us | max us | % of GPU time |")
    print("|---|---|---|---|---|---|")
    for r in csv.DictReader(open(path)):
        name = r["Name"].replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        if len(name) > 70:
            name = name[:67] + "..."
        print(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
              f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")


def counters_workload(config="mixtral", meta_path=None):
    """Fixed workload for the rocprofv3 --pmc passes: decode tokens of the
    resident stack of `config` (Mixtral shapes by default), then calibration
    copies of known size.  Writes the shapes, FFN calls and distinct experts
    of the profiled tokens as JSON to meta_path (default
    counters_<config>.json in the working directory)."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS[config]
    if cfg.L * cfg.E * cfg.blob_bytes > 0.8 * torch.cuda.get_device_properties(0).total_memory:
        raise SystemExit(f"--counters: the {cfg.name} stack does not fit in HBM; only resident stacks are profiled")
    wl = Workload(cfg)
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(wl.prof)
    ctx = make_ctx(wl, pred)
    ctx.set_predictor_batch(True)
    ctx.set_timing(1)
    y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device="cuda:0")
    run_tokens(ctx, wl, 0, COUNTER_TOKENS, y, S.MODE_STMOE)
    torch.cuda.synchronize()
    _, _, n_calls, n_experts = ctx.timing()
    src = torch.empty(CALIB_BYTES, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        S.calib_copy(src, dst, CALIB_BYTES)
    torch.cuda.synchronize()
    ctx.close()
    pred.close()
    meta = dict(config=config, title=f"{cfg.name}, batch {cfg.B}", H=cfg.H, I=cfg.I, esz=cfg.wbytes,
                n_shared=cfg.n_shared, n_calls=int(n_calls), n_experts=int(n_experts))
    path = meta_path or f"counters_{config}.json"
    if os.path.dirname(path):
        os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        json.dump(meta, f)
    log("counters workload done")


def predictor_spread(seed_offsets=(0, 100, 200)):
    """Recall and precision of the full predictor (CCT + HT, online update)
    per workload over planted traces drawn with three seeds (the workload's,
    +100, +200): mean and range.  Markdown lines."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    dev = "cuda:0"
    out = ["| workload | seeds | recall l>=1 mean (min-max) | recall l0 mean (min-max) | precision mean (min-max) |",
           "|---|---|---|---|---|"]
    for name in ("tiny", "mixtral", "qwen30b", "qwen30b-b8", "dsv2lite", "qwen235b"):
        vals = []
        for off in seed_offsets:
            cfg = W.CONFIGS[name].scaled(seed=W.CONFIGS[name].seed + off)
            T = min(cfg.T, 128)
            sel = W.planted_trace(cfg, n_tokens=cfg.P + T)
            dsel = torch.from_numpy(np.ascontiguousarray(sel[cfg.P:].transpose(0, 2, 1, 3))).to(dev)
            p = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
            p.profile(sel[:cfg.P])
            p.predict(-1, None, use=S.USE_HT)
            for t in range(T):
                for l in range(cfg.L):
                    cur = dsel[t, l]
                    p.update(l, dsel[t, l - 1] if l else None, cur)
                    if l + 1 < cfg.L:
                        p.predict(l, cur, use=S.USE_BOTH)
                    else:
                        p.predict(-1, None, use=S.USE_HT)
            st = p.stats()
            p.close()
            vals.append((st[1:, 0].sum() / max(st[1:, 1].sum(), 1), st[0, 0] / max(st[0, 1], 1),
                         st[:, 0].sum() / max(st[:, 2].sum(), 1)))
        v = np.array(vals)
        cells = [f"{v[:, i].mean():.3f} ({v[:, i].min():.3f}-{v[:, i].max():.3f})" for i in range(3)]
        base = W.CONFIGS[name].seed
        out.append(f"| {W.CONFIGS[name].name} | {', '.join(str(base + o) for o in seed_offsets)} | "
                   + " | ".join(cells) + " |")
        log(f"predictor spread {name} done")
    return out


def predictor_sweep():
    """Prediction quality of the GPU predictor (stmoe_update / stmoe_predict)
    on planted routing traces, per prediction source and with the online CCT
    update on or off.  Recall = sum|A n P| / sum|A| (layers >= 1 and layer 0),
    precision = sum|A n P| / sum|P|, |P| = mean predicted set per row."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    dev = "cuda:0"
    cfgs = [W.CONFIGS[n] for n in ("tiny", "mixtral", "qwen30b", "qwen30b-b8", "dsv2lite", "qwen235b")]
    cfgs += [W.table1_config(n) for n in W.TABLE1_SHAPES]
    modes = [("CCT+HT", S.USE_BOTH, True), ("CCT+HT, no online update", S.USE_BOTH, False),
             ("HT only", S.USE_HT, True), ("CCT only", S.USE_CCT, True)]
    print("| workload | B | tokens | overlap / (K^2/E) | mode | recall l>=1 | recall l0 | precision | mean set |")
    print("|---|---|---|---|---|---|---|---|---|")
    for cfg in cfgs:
        T = min(cfg.T, 128)
        sel = W.planted_trace(cfg, n_tokens=cfg.P + T)
        dec = sel[cfg.P:]
        ov = np.mean([len(set(dec[t, b, l]) & set(dec[t - 1, b, l])) for t in range(1, T)
                      for b in range(cfg.B) for l in range(cfg.L)])
        ratio = ov / (cfg.K * cfg.K / cfg.E)
        dsel = torch.from_numpy(np.ascontiguousarray(dec.transpose(0, 2, 1, 3))).to(dev)   # [T][L][B][K]
        for mname, use, online in modes:
            p = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
            p.profile(sel[:cfg.P])
            p.predict(-1, None, use=use & S.USE_HT)
            for t in range(T):
                for l in range(cfg.L):
                    cur = dsel[t, l]
                    p.update(l, dsel[t, l - 1] if l else None, cur, online=online)
                    if l + 1 < cfg.L:
                        p.predict(l, cur, use=use)
                    else:
                        p.predict(-1, None, use=use & S.USE_HT)
            st = p.stats()
            p.close()
            r1 = st[1:, 0].sum() / max(st[1:, 1].sum(), 1)
            r0 = st[0, 0] / max(st[0, 1], 1)
            prec = st[:, 0].sum() / max(st[:, 2].sum(), 1)
            mset = st[:, 2].sum() / max(st[:, 1].sum() / cfg.K, 1)
            print(f"| {cfg.name} | {cfg.B} | {T} | {ratio:.2f} | {mname} | {r1:.3f} | {r0:.3f} | {prec:.3f} | "
                  f"{mset:.1f} |", flush=True)


SWEEP_CONFIGS = ("tiny", "mixtral", "qwen30b", "qwen30b-b8", "dsv2lite", "qwen235b")


def sweep_routing(cfg):
    """The FFN sweep's seeded routing of one config: B rows of K distinct
    experts, their weights, and the sorted distinct experts."""
    rng = np.random.default_rng(cfg.seed)
    idx = np.stack([rng.choice(cfg.E, cfg.K, replace=False) for _ in range(cfg.B)]).astype(np.int32)
    w = rng.random((cfg.B, cfg.K)).astype(np.float32)
    return rng, idx, w, sorted(set(idx.ravel().tolist()))


def ffn_sweep(calls=60, cold_bytes=2 << 30):
    """Event-timed moe_expert_ffn per config shape: one seeded routing of B
    tokens (top-K of E).  Each call reads a different copy of the selected
    experts' blobs, cycling over at least `cold_bytes` (well above the 256 MB
    Infinity Cache), so no call finds its weights in a cache, as in decode,
    where every layer reads other experts.  The per-call time includes the
    launch gaps; the kernel durations come from a kernel trace of this run."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    dev = "cuda:0"
    print("| workload | B | distinct experts (+shared) | bytes per call | copies cycled | us per call | GB/s | "
          "of 8 TB/s | path |")
    print("|---|---|---|---|---|---|---|---|---|")
    for name in SWEEP_CONFIGS:
        cfg = W.CONFIGS[name]
        rng, idx, w, sel = sweep_routing(cfg)
        nb = len(sel) + cfg.n_shared
        n_sets = max(2, -(-cold_bytes // (nb * cfg.blob_bytes)))
        tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        store = torch.empty((n_sets, nb, cfg.blob_elems), dtype=tdt, device=dev)
        for k, e in enumerate(sel):
            W.expert_blob_torch(cfg, 0, e, store[0, k])
        for sh in range(cfg.n_shared):
            W.expert_blob_torch(cfg, 0, sh, store[0, len(sel) + sh], shared=True)
        for c in range(1, n_sets):
            store[c].copy_(store[0])
        eptr, sptr = [], []
        for c in range(n_sets):
            ptrs = [store[c, 0].data_ptr()] * cfg.E
            for k, e in enumerate(sel):
                ptrs[e] = store[c, k].data_ptr()
            eptr.append(torch.tensor(ptrs, dtype=torch.int64, device=dev))
            sptr.append(torch.tensor([store[c, len(sel) + sh].data_ptr() for sh in range(cfg.n_shared)],
                                     dtype=torch.int64, device=dev) if cfg.n_shared else None)
        dt = S.BF16 if cfg.dtype == "bf16" else S.F32
        x = Workload._dev(W.to_storage(cfg, rng.normal(0, 1, (cfg.B, cfg.H))))
        y = torch.empty((cfg.B, cfg.H), dtype=torch.float32, device=dev)
        ws = torch.zeros(S.ffn_workspace_bytes(cfg.B, cfg.K, cfg.E, cfg.H, cfg.I, cfg.n_shared, dt),
                         dtype=torch.uint8, device=dev)
        ti, tw = torch.from_numpy(idx).to(dev), torch.from_numpy(w).to(dev)

        def call(c):
            S.expert_ffn(x, ti, tw, cfg.H, cfg.I, cfg.E, dt, eptr[c % n_sets], y, ws, shared_ptrs=sptr[c % n_sets],
                         n_shared=cfg.n_shared)

        for c in range(2):
            call(c)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for c in range(2, 2 + calls):
            call(c)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / calls
        nbytes = nb * cfg.blob_bytes
        gbps = nbytes / us / 1e3
        path = "MFMA" if (cfg.B >= 8 and cfg.dtype == "bf16") else "GEMV"
        print(f"| {cfg.name} | {cfg.B} | {len(sel)} (+{cfg.n_shared}) | {nbytes} | {n_sets} | {us:.1f} | {gbps:.0f} | "
              f"{gbps / PEAK_HBM_GBPS:.3f} | {path} |", flush=True)
        del store


READ_FLOOR_MIB = (24, 48, 96, 144, 224, 448)


def read_floor(sizes_mib=READ_FLOOR_MIB, reps=40, buf_bytes=4 << 30):
    """The shortest time one launch needs to stream n bytes that are in no
    cache: stmoe_calib_read with 32 KiB (pattern 2) and 256 KiB (pattern 1)
    per workgroup, every launch on a different region of a 4 GiB buffer.
    Event-timed over back-to-back launches (launch gaps included); the kernel
    durations come from a kernel trace of this run."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    dev = "cuda:0"
    src = torch.empty(buf_bytes, dtype=torch.uint8, device=dev)
    src.zero_()
    top = max(sizes_mib) << 20
    out = torch.empty(max(S.calib_read_out_words(top, 2), S.calib_read_out_words(top, 1)), dtype=torch.int32,
                      device=dev)
    print("| MiB per launch | bytes per workgroup | workgroups | us per launch (events, gaps included) | GB/s |")
    print("|---|---|---|---|---|")
    for mib in sizes_mib:
        n = mib << 20
        for pattern, region in ((2, 32 << 10), (1, 256 << 10)):
            offs = [((k * n) % (buf_bytes - n)) & ~((256 << 10) - 1) for k in range(reps + 2)]
            assert all(o + n <= buf_bytes for o in offs)
            for o in offs[:2]:
                S.calib_read(src[o:], n, out, pattern=pattern)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for o in offs[2:]:
                S.calib_read(src[o:], n, out, pattern=pattern)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            print(f"| {mib} | {region >> 10} KiB | {S.calib_read_out_words(n, pattern)} | {us:.2f} | "
                  f"{n / us / 1e3:.0f} |", flush=True)
    del src


def reread_probe(sizes_mib=(24, 48, 96), reps=20, buf_bytes=4 << 30, other_mib=72):
    """One stmoe_calib_read launch (32 KiB per workgroup) on bytes in no
    cache, against the same bytes once the Infinity Cache may hold them: read
    again by the same kernel, first read by a plain-load kernel (torch's sum),
    and first read that way with `other_mib` MiB of other data streamed in
    between (what a prefetch one layer ahead would leave for the next
    layer).  Phases are separated by idle time so that a kernel trace of this
    run splits them (--summarize-trace); the order is printed."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    dev = "cuda:0"
    src = torch.empty(buf_bytes, dtype=torch.uint8, device=dev)
    src.zero_()
    other = torch.empty(buf_bytes // 2, dtype=torch.uint8, device=dev)
    other.zero_()
    on = other_mib << 20
    top = max(max(sizes_mib) << 20, on)
    out = torch.empty(S.calib_read_out_words(top, 2), dtype=torch.int32, device=dev)
    acc = torch.zeros((), dtype=torch.int64, device=dev)
    run = 0

    def pause(label):
        nonlocal run
        torch.cuda.synchronize()
        time.sleep(0.01)
        print(f"| {run} | {label} |", flush=True)
        run += 1

    print("| trace run | phase |")
    print("|---|---|")
    for mib in sizes_mib:
        n = mib << 20
        offs = [((k * n) % (buf_bytes - n)) & ~((256 << 10) - 1) for k in range(reps)]
        assert all(o + n <= buf_bytes for o in offs)
        for o in offs:
            S.calib_read(src[o:], n, out, pattern=2)
        pause(f"{mib} MiB, bytes in no cache")
        for _ in range(reps):
            S.calib_read(src[offs[-1]:], n, out, pattern=2)
        pause(f"{mib} MiB, the same bytes read again")
        for o in offs:
            acc += src[o:o + n].view(torch.int32).sum()
            S.calib_read(src[o:], n, out, pattern=2)
        pause(f"{mib} MiB, first read by torch's sum")
        for k, o in enumerate(offs):
            acc += src[o:o + n].view(torch.int32).sum()
            oo = ((k * (on + (8 << 20))) % (buf_bytes // 2 - on)) & ~((256 << 10) - 1)
            assert oo + on <= buf_bytes // 2
            S.calib_read(other[oo:], on, out, pattern=2)
            S.calib_read(src[o:], n, out, pattern=2)
        pause(f"{mib} MiB, first read by torch's sum, then {other_mib} MiB of other data streamed")
    del src, other


def trace_groups(path, pause_ns=1_000_000):
    """This library's kernels in a rocprofv3 kernel trace, grouped by run
    (launches separated by more than `pause_ns` of idle time start a new
    one: input generation between shapes), kernel and workgroup count, in
    order of appearance: {(run, name, workgroups): [durations in us]}."""
    import csv
    groups = {}
    run, last_end = 0, None
    for r in sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"])):
        name = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        if not name.startswith("stmoe::"):
            continue
        t0, t1 = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
        if last_end is not None and t0 - last_end > pause_ns:
            run += 1
        last_end = t1
        wgs = int(r["Grid_Size_X"]) // max(int(r["Workgroup_Size_X"]), 1)
        groups.setdefault((run, name, wgs), []).append((t1 - t0) / 1e3)
    return groups


def _median_kept(t):
    kept = sorted(t[len(t) // 4:])
    return kept[len(kept) // 2], kept


def summarize_floor(rf_csv, fs_csv):
    """Markdown: the read floor by bytes per launch (32 KiB per workgroup
    launches of --read-floor) beside every FFN kernel of --ffn-sweep, both
    from kernel traces (median duration per group)."""
    from paper_2606_15453_amd import workload as W
    pts = sorted((wgs * (32 << 10), _median_kept(t)[0]) for (_, n, wgs), t in trace_groups(rf_csv).items()
                 if n.endswith("<2048ul>"))

    def floor_us(nbytes):     # above the largest size: that size's rate
        if nbytes >= pts[-1][0]:
            return pts[-1][1] * nbytes / pts[-1][0]
        for (b0, t0), (b1, t1) in zip(pts, pts[1:]):
            if b0 <= nbytes <= b1:
                return t0 + (t1 - t0) * (nbytes - b0) / (b1 - b0)

    print("Read floor (one `stmoe_calib_read` launch, 32 KiB per workgroup, bytes in no cache):\n")
    print("| MiB per launch | median us | GB/s | of 8 TB/s |")
    print("|---|---|---|---|")
    for b, t in pts:
        print(f"| {b >> 20} | {t:.2f} | {b / t / 1e3:.0f} | {b / t / 1e3 / PEAK_HBM_GBPS:.3f} |")
    groups = trace_groups(fs_csv)
    runs = sorted({k[0] for k in groups})
    assert len(runs) == len(SWEEP_CONFIGS), (len(runs), "runs in the FFN sweep trace")
    print("\nExpert FFN kernels of the sweep (weights in no cache; floor interpolated linearly between the sizes "
          "above, none below the smallest):\n")
    print("| workload | kernel | workgroups | algorithmic MB | median us | GB/s | floor us | of floor | of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|---|")
    for run, name in zip(runs, SWEEP_CONFIGS):
        cfg = W.CONFIGS[name]
        _, _, _, sel = sweep_routing(cfg)
        esz = 2 if cfg.dtype == "bf16" else 4
        nb = len(sel) + cfg.n_shared
        for (r, kname, wgs), t in groups.items():
            if r != run or "reduce" in kname:
                continue
            nbytes = nb * (2 if "gate_up" in kname else 1) * cfg.H * cfg.I * esz
            med = _median_kept(t)[0]
            short = kname.replace("stmoe::", "")
            fl = f"{floor_us(nbytes):.2f} | {floor_us(nbytes) / med:.3f}" if nbytes >= pts[0][0] else "- | -"
            print(f"| {cfg.name} | `{short}` | {wgs} | {nbytes / 1e6:.1f} | {med:.2f} | {nbytes / med / 1e3:.0f} | "
                  f"{fl} | {nbytes / med / 1e3 / PEAK_HBM_GBPS:.3f} |")


def summarize_trace(path, title, cmd, pause_ns=1_000_000):
    """Median kernel durations of this library's kernels in a rocprofv3
    kernel trace, per run, kernel and grid size (see trace_groups); the first
    quarter of each group's launches is dropped (first touch of the
    buffers)."""
    groups = trace_groups(path, pause_ns)
    print(f"# {title}\n")
    print(f"Command (run from `/tmp` with `TMPDIR=/tmp`, repository at `$R`):\n\n```\n{cmd}\n```\n")
    print("| kernel | workgroups | launches | median us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for (_, name, wgs), t in groups.items():
        med, kept = _median_kept(t)
        print(f"| `{name}` | {wgs} | {len(kept)} | {med:.2f} | {kept[0]:.2f} | {kept[-1]:.2f} |")


def achievable_read_gbps(nbytes=4 << 30, reps=10, pattern=0):
    """Streaming-read bandwidth of stmoe_calib_read with the FFN's loads, event-timed:
    pattern 0 a grid-stride sweep, 1 a contiguous 256 KiB region per workgroup."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    src.zero_()
    out = torch.empty(S.calib_read_out_words(nbytes, pattern), dtype=torch.int32, device="cuda:0")
    S.calib_read(src, nbytes, out, pattern=pattern)
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    for _ in range(reps):
        S.calib_read(src, nbytes, out, pattern=pattern)
    s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1)
    del src
    return nbytes * reps / (ms * 1e-3) / 1e9


class Workload:
    """Seeded synthetic inputs of one config, placed in HBM.

    hbm_blobs: for a stack whose experts do not fit in HBM (Qwen3-235B shapes,
    454 GB), only this many distinct expert blobs are generated and expert
    (l, e) reads blob (l*E + e) mod hbm_blobs.  Within a layer the E experts
    stay distinct, so every timed read streams distinct HBM bytes; the values
    are those of the first hbm_blobs experts.  x_tokens: hidden states for the
    first x_tokens decode tokens only (their routing trace is unchanged)."""

    def __init__(self, cfg, hbm_blobs=None, x_tokens=None):
        import torch
        from paper_2606_15453_amd import stmoe as S
        from paper_2606_15453_amd import workload as W
        self.cfg = cfg
        dev = "cuda:0"
        self.dt = S.BF16 if cfg.dtype == "bf16" else S.F32
        tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        self.n_blobs = cfg.L * cfg.E if hbm_blobs is None else min(cfg.L * cfg.E, hbm_blobs)
        assert self.n_blobs >= cfg.E
        self.T = cfg.T if x_tokens is None else min(cfg.T, x_tokens)
        t0 = time.time()
        self.sel = W.planted_trace(cfg)
        self.prof = W.profiling_selections(cfg, self.sel)
        self.warm = S.warm_sets(self.prof, cfg.E, cfg.C)
        log(f"planted trace {self.sel.shape} in {time.time() - t0:.1f}s")
        t0 = time.time()
        self.wg_f64 = [W.router_rows_f64(cfg, l) for l in range(cfg.L)]
        self.wg = [self._dev(W.to_storage(cfg, g)) for g in self.wg_f64]
        xs = np.stack([np.stack([W.to_storage(cfg, W.hidden_f64(cfg, self.sel, cfg.P + t, l, self.wg_f64[l]))
                                 for l in range(cfg.L)]) for t in range(self.T)])
        self.x_store = xs
        self.x = self._dev(xs)                              # [T][L][B][H]
        log(f"router rows + hidden states for {self.T} tokens in {time.time() - t0:.1f}s")
        t0 = time.time()
        self.blobs = torch.empty((self.n_blobs, cfg.blob_elems), dtype=tdt, device=dev)
        for i in range(self.n_blobs):
            l, e = divmod(i, cfg.E)
            W.expert_blob_torch(cfg, l, e, self.blobs[i])
        self.shared = None
        if cfg.n_shared:
            self.shared = torch.empty((cfg.L * cfg.n_shared, cfg.blob_elems), dtype=tdt, device=dev)
            for l in range(cfg.L):
                for s in range(cfg.n_shared):
                    W.expert_blob_torch(cfg, l, s, self.shared[l * cfg.n_shared + s], shared=True)
        torch.cuda.synchronize()
        gb = self.blobs.numel() * self.blobs.element_size() / 1e9
        log(f"{self.n_blobs} of {cfg.L * cfg.E} expert blobs ({gb:.1f} GB) generated in HBM in "
            f"{time.time() - t0:.1f}s")

    @staticmethod
    def _dev(a):
        import torch
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to("cuda:0").view(torch.bfloat16)
        return torch.from_numpy(a).to("cuda:0")

    @property
    def aliased(self):
        return self.n_blobs < self.cfg.L * self.cfg.E

    def blob(self, l, e):
        return self.blobs[(l * self.cfg.E + e) % self.n_blobs]

    def blob_ptr(self, l, e):
        return self.blob(l, e).data_ptr()

    def shared_ptrs(self):
        if self.shared is None:
            return None
        return [self.shared[i].data_ptr() for i in range(self.shared.shape[0])]


def make_ctx(wl, pred, cache=None):
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    resident = None if cache else [wl.blob_ptr(l, e) for l in range(cfg.L) for e in range(cfg.E)]
    return S.DecodeContext(cfg.L, cfg.E, cfg.K, cfg.B, cfg.H, cfg.I, wl.dt, [g.data_ptr() for g in wl.wg],
                           predictor=pred, cache=cache, resident_ptrs=resident,
                           shared_ptrs=wl.shared_ptrs(), n_shared=cfg.n_shared)


def run_tokens(ctx, wl, first, n, y, mode):
    T = wl.T
    for i in range(n):
        t = first + i
        ctx.token(t, wl.x[t % T], y, mode=mode)


def repeat_summary(tokens, seconds):
    """tokens/s of back-to-back timed runs of the same length (the first is
    `value`), their median and their spread (max - min over the median)."""
    rates = sorted(tokens / t for t in seconds)
    med = rates[len(rates) // 2]
    return {"runs": len(seconds), "tokens_per_s": [round(tokens / t, 3) for t in seconds],
            "median": round(med, 3), "spread": round((rates[-1] - rates[0]) / med, 4)}


def hbm_resident(wl, steps, warmup):
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(wl.prof)
    ctx = make_ctx(wl, pred)
    ctx.set_predictor_batch(True)     # the predictor's layers in one side-stream launch per token
    y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device="cuda:0")
    run_tokens(ctx, wl, 0, warmup, y, S.MODE_STMOE)
    torch.cuda.synchronize()
    # host cost of issuing one layer (a short burst, so launches never block
    # on a full queue): below the GPU time per layer means the GPU is the bound
    n_issue = min(8, max(1, warmup))
    t0 = time.perf_counter()
    run_tokens(ctx, wl, 0, n_issue, y, S.MODE_STMOE)
    host_us = (time.perf_counter() - t0) * 1e6 / (n_issue * cfg.L)
    torch.cuda.synchronize()
    # event-time every TIMING_EVERY-th token, or every token of a short run
    # (the cadence counts from the first timed token)
    every = timing_cadence(steps)
    ctx.set_timing(every)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_tokens(ctx, wl, warmup, steps, y, S.MODE_STMOE)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    up_ms, down_ms, n_calls, n_exp = ctx.timing()
    route_ms, _, ffn_ms, pred_ms, n_timed = ctx.stage_timing()
    stats = pred.stats()
    # the same timed run twice more (next tokens of the trace): the spread of
    # the rate; the statistics above cover the first run only
    repeats = []
    for k in range(2):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run_tokens(ctx, wl, warmup + (k + 1) * steps, steps, y, S.MODE_STMOE)
        torch.cuda.synchronize()
        repeats.append(time.perf_counter() - t0)
    ctx.close()
    pred.close()
    per = 1e3 / max(n_timed, 1)
    stages = {"route_logits": round(route_ms * per, 2), "ffn_with_routing": round(ffn_ms * per, 2),
              "predict_side_stream": round(pred_ms * per, 2)}
    return dict(seconds=dt, up_ms=up_ms, down_ms=down_ms, n_calls=n_calls, n_experts=n_exp, stats=stats,
                host_issue_us_per_layer=host_us, stages_us=stages, repeat_seconds=repeats)


def largest_config(steps, warmup, hbm_pool_gb, capped_tokens, pinned_gb):
    """The largest workload, Qwen3-235B-A22B shapes at batch 16, decoded with
    its experts in HBM.  Its stack does not fit, so a pool of distinct blobs
    stands in (expert (l, e) reads blob (l*E + e) mod the pool's size): the
    timing of the real stack, not its values.  tokens/s with two repeats, the
    gate/up kernel's event-timed rate and the predictor's hit rates; with
    capped_tokens > 0 also the config's capped cache (45 of 128 experts per
    layer in HBM, the rest in pinned host memory) for that many tokens:
    on-demand loading and ST-MoE prefetch (into slots and staged), decisions
    on the device."""
    import torch
    from paper_2606_15453_amd import workload as W
    cfg = W.CONFIGS["qwen235b"]
    wl = Workload(cfg, hbm_blobs=int(hbm_pool_gb * 1e9) // cfg.blob_bytes, x_tokens=warmup + steps)
    r = hbm_resident(wl, steps, warmup)
    esz = cfg.wbytes
    up_bytes = r["n_experts"] * 2 * cfg.H * cfg.I * esz + r["n_calls"] * cfg.n_shared * 2 * cfg.H * cfg.I * esz
    dn_bytes = r["n_experts"] * cfg.H * cfg.I * esz + r["n_calls"] * cfg.n_shared * cfg.H * cfg.I * esz
    up_gbps = up_bytes / (r["up_ms"] * 1e-3) / 1e9
    dn_gbps = dn_bytes / (r["down_ms"] * 1e-3) / 1e9
    stats = r["stats"]
    out = {
        "workload": cfg.name,
        "mode": (f"HBM-resident stand-in: {wl.n_blobs} distinct expert blobs in HBM, expert (l, e) reads blob "
                 f"(l*E + e) mod {wl.n_blobs}; ST-MoE predictor on"),
        "steps": steps, "warmup": warmup,
        "tokens_per_s": round(cfg.B * steps / r["seconds"], 3),
        "ms_per_step": round(1e3 * r["seconds"] / steps, 3),
        "repeats": repeat_summary(cfg.B * steps, [r["seconds"]] + r["repeat_seconds"]),
        "ffn_gate_up": {"achieved_gbps": round(up_gbps, 1), "frac": round(up_gbps / PEAK_HBM_GBPS, 4),
                        "avg_launch_us": round(1e3 * r["up_ms"] / max(r["n_calls"], 1), 3),
                        "launches": r["n_calls"]},
        "ffn_down": {"achieved_gbps": round(dn_gbps, 1), "frac": round(dn_gbps / PEAK_HBM_GBPS, 4),
                     "avg_launch_us": round(1e3 * r["down_ms"] / max(r["n_calls"], 1), 3)},
        "layer_us": round(1e6 * r["seconds"] / steps / cfg.L, 2),
        "prediction": {
            "recall_layers_ge1": round(float(stats[1:, 0].sum() / max(stats[1:, 1].sum(), 1)), 4),
            "recall_layer0": round(float(stats[0, 0] / max(stats[0, 1], 1)), 4),
            "precision": round(float(stats[:, 0].sum() / max(stats[:, 2].sum(), 1)), 4),
        },
    }
    if capped_tokens > 0:
        out["capped"] = offload(wl, capped_tokens, out["ms_per_step"], pinned_gb,
                                "on_demand_device,st_moe_device,st_moe_staged_device")
    del wl
    torch.cuda.empty_cache()
    return out


#: host-to-HBM copy rate (GB/s): the latest on-demand run's copied bytes over its time
LINK_GBPS = [55.0]


def attn_window_s(attn):
    """Seconds per layer of the decode-attention stand-in (kv buffer, bytes, out): its bytes
    at the HBM streaming rate."""
    return attn[1] / (6.0e12)


def expert_pool(wl, pinned_gb, tier):
    """The backing pool the capped cache copies from: pinned host memory over
    PCIe ("host"), or the HBM-resident stack itself ("hbm", copies device to
    device), which models a backing tier much faster than the host link."""
    if tier == "hbm":
        cfg = wl.cfg
        return None, [wl.blob_ptr(l, e) for l in range(cfg.L) for e in range(cfg.E)], wl.n_blobs
    return host_pool(wl, pinned_gb)


def host_pool(wl, pinned_gb):
    """Pinned host copies of the expert blobs.  The pool holds M = min(L*E,
    pinned budget / blob) distinct blobs; expert (l, e) is copied from pool
    slot (l*E + e) mod M.  Every copy still moves a whole blob over PCIe, so
    the timing is that of distinct experts."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    blob = cfg.blob_bytes
    n_all = cfg.L * cfg.E
    M = min(wl.n_blobs, int(pinned_gb * 1e9) // blob)
    t0 = time.time()
    pool = S.PinnedHost(M * blob)
    host = pool.tensor()
    for i in range(M):
        host[i * blob:(i + 1) * blob].copy_(wl.blobs[i].view(torch.uint8))
    log(f"pinned host pool {pool.nbytes / 1e9:.1f} GB ({M} of {n_all} blobs) filled in {time.time() - t0:.1f}s")
    ptrs = [pool.ptr + (i % M) * blob for i in range(n_all)]
    return pool, ptrs, M


def offload_run(wl, C, arena, ptrs, streams, v, n_tokens, resident_ms_per_token, attn=None):
    """One capped-cache decode run: C slots per layer, the rest streamed from
    the pinned host pool, with the settings of `v` (see variant()).  attn =
    (kv buffer, bytes, out): a decode-attention stand-in that streams `bytes`
    of KV cache on the compute stream before every MoE layer (layers are then
    issued one by one)."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    blob = cfg.blob_bytes
    name, mode, min_score, online, after_demand = v["name"], v["mode"], v["min_score"], v["online"], v["after_demand"]
    device, staged, head, graph, freq = v["device"], v["staged"], v["head"], v["graph"], v["freq"]
    max_pf = C if v["max_pf"] is None else v["max_pf"]
    n_stage = staging_slots(cfg, C)
    demand, side = streams
    if head < 0:
        # the layer's compute window (routing, FFN, attention) at the link's
        # rate, shared by the experts staged for one layer
        window_s = resident_ms_per_token / cfg.L * 1e-3 + (attn_window_s(attn) if attn else 0.0)
        head = min(blob, max(1 << 16, int(LINK_GBPS[0] * 1e9 * window_s / max(staged, 1)) // 4096 * 4096))
    y = torch.empty((cfg.L, cfg.B, cfg.H), dtype=torch.float32, device="cuda:0")
    cache = S.ExpertCache(cfg.L, cfg.E, C, blob, n_stage, arena, ptrs, demand, side)
    cache.warm(W_warm(wl, C))
    cache.set_prefetch_order(after_demand)
    if freq:
        cache.set_counts(S.use_counts(wl.prof, cfg.E))
    cache.set_device_policy(device)
    if v.get("copy_wgs"):
        cache.set_copy_workgroups(v["copy_wgs"], v["copy_wgs"])
    if staged:
        cache.set_staged_prefetch(staged, head)
    pred = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(wl.prof)
    ctx = make_ctx(wl, pred, cache)
    ctx.set_prefetch(min_score, max_pf)
    ctx.set_online_update(online)
    if graph:
        ctx.set_graph(True)     # event timing would run the tokens eagerly: no stage times
    else:
        ctx.set_timing(1)       # events on every layer: negligible next to ms-scale copies
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if attn is None:
        run_tokens(ctx, wl, 0, n_tokens, y, mode)
    else:
        kv, nbytes, out = attn
        T = wl.T
        for t in range(n_tokens):
            for l in range(cfg.L):
                S.calib_read(kv, nbytes, out)
                ctx.layer(t, l, wl.x[t % T][l], y[l], mode)
    torch.cuda.synchronize()
    demand.synchronize()
    side.synchronize()
    dt = time.perf_counter() - t0
    route_ms, miss_ms, ffn_ms, _, n_timed = ctx.stage_timing()
    cst = cache.stats()
    st = pred.stats()
    copies = cst["demand"] + cst["overflow"] + cst["prefetch"]
    # bytes moved over the link: whole blobs, except staged copies (host decisions: the head of
    # every staged expert, the rest of the used ones; device decisions: cancelled copies stop
    # at an unrecorded point, so no byte count)
    if not staged:
        h2d_bytes = copies * blob
    elif not device:
        hb = head if 0 < head < blob else blob
        h2d_bytes = (cst["demand"] + cst["overflow"]) * blob + cst["prefetch"] * hb + cst["useful"] * (blob - hb)
    else:
        h2d_bytes = None
    rec = dict(tokens=n_tokens, seconds=round(dt, 4), prefetch_min_score=min_score, staged_per_layer=staged,
               staged_head_bytes=(head if staged and not device else None), graph_replay=bool(graph),
               prefetch_max_per_layer=max_pf, online_update=bool(online),
               prefetch_after_demand=bool(after_demand), device_decisions=bool(device),
               eviction="frequency-aware" if freq else "least recently used",
               tokens_per_s=round(cfg.B * n_tokens / dt, 3),
               ms_per_token=round(1e3 * dt / n_tokens, 3),
               stall_ms_per_token=round(1e3 * dt / n_tokens - resident_ms_per_token, 3),
               h2d_copies=copies, h2d_gbps=(None if h2d_bytes is None else round(h2d_bytes / dt / 1e9, 2)),
               cache=cst,
               stages_us_per_layer={"route_and_predict": round(1e3 * route_ms / max(n_timed, 1), 1),
                                    "record_wait_and_missed_loads": round(1e3 * miss_ms / max(n_timed, 1), 1),
                                    "ffn": round(1e3 * ffn_ms / max(n_timed, 1), 1)})
    if mode != S.MODE_ON_DEMAND:
        rec["recall_layers_ge1"] = round(float(st[1:, 0].sum() / max(st[1:, 1].sum(), 1)), 4)
        rec["recall_layer0"] = round(float(st[0, 0] / max(st[0, 1], 1)), 4)
        rec["precision"] = round(float(st[:, 0].sum() / max(st[:, 2].sum(), 1)), 4)
        rec["mean_predicted_per_row"] = round(float(st[:, 2].sum() / max(st[:, 1].sum() / cfg.K, 1)), 3)
    if mode == S.MODE_ON_DEMAND and not device and copies > 0:
        LINK_GBPS[0] = rec["h2d_gbps"]
    log(f"offload C={C} {name}: {rec['tokens_per_s']} tok/s, {rec['ms_per_token']} ms/token, cache {cst}")
    ctx.close()
    pred.close()
    cache.close()
    return rec


def W_warm(wl, C):
    """Warm start for C slots per layer: the C experts most selected in profiling."""
    from paper_2606_15453_amd import stmoe as S
    if C == wl.cfg.C:
        return wl.warm
    return S.warm_sets(wl.prof, wl.cfg.E, C)


def variant(name, mode, min_score=2, max_pf=None, online=1, after_demand=0, device=0, staged=0, head=0,
            graph=0, freq=0, copy_wgs=0):
    """One capped-cache run's settings: prediction mode, admission (min score,
    at most max_pf prefetches per layer; None = the cache's slots), online
    CCT update, prefetch copies after the missed loads, device-side
    decisions, staged prefetches per layer (0: prefetch into evicted slots),
    bytes of each staged expert copied up front with host decisions (-1: the
    layer's compute window at the link's rate, shared by the staged experts;
    0: all of it), HIP graph replay of each token, frequency-aware eviction
    (use counts seeded from profiling) instead of least recently used, and the
    copy kernels' workgroups with device decisions (0: the defaults)."""
    return dict(name=name, mode=mode, min_score=min_score, max_pf=max_pf, online=online,
                after_demand=after_demand, device=device, staged=staged, head=head, graph=graph, freq=freq,
                copy_wgs=copy_wgs)


def offload_variants(cfg):
    from paper_2606_15453_amd import stmoe as S
    n_st = STAGED_PER_LAYER(cfg)
    return [variant("on_demand", S.MODE_ON_DEMAND),
            variant("st_moe", S.MODE_STMOE),
            variant("st_moe_after_demand", S.MODE_STMOE, after_demand=1),
            variant("st_moe_score4_maxK", S.MODE_STMOE, 4, cfg.K),
            variant("st_moe_score4_maxK_after_demand", S.MODE_STMOE, 4, cfg.K, after_demand=1),
            variant("ht_only", S.MODE_HT_ONLY),
            variant("cct_only", S.MODE_CCT_ONLY),
            variant("st_moe_staged_host", S.MODE_STMOE, after_demand=1, staged=n_st, head=-1),
            variant("st_moe_staged_host1", S.MODE_STMOE, after_demand=1, staged=1, head=-1),
            variant("on_demand_device", S.MODE_ON_DEMAND, device=1),
            variant("st_moe_device", S.MODE_STMOE, device=1),
            variant("st_moe_score4_maxK_after_demand_device", S.MODE_STMOE, 4, cfg.K, after_demand=1, device=1),
            variant("st_moe_staged_device", S.MODE_STMOE, after_demand=1, device=1, staged=n_st),
            variant("on_demand_device_graph", S.MODE_ON_DEMAND, device=1, graph=1),
            variant("st_moe_staged_device_graph", S.MODE_STMOE, after_demand=1, device=1, staged=n_st, graph=1),
            variant("on_demand_freq", S.MODE_ON_DEMAND, freq=1),
            variant("on_demand_device_freq", S.MODE_ON_DEMAND, device=1, freq=1),
            variant("st_moe_staged_host_freq", S.MODE_STMOE, after_demand=1, staged=n_st, head=-1, freq=1)]


def STAGED_PER_LAYER(cfg):
    """Staged prefetches per layer: two (the time model gains little beyond two)."""
    return min(cfg.K, 2)


def staging_slots(cfg, C):
    """Staging slots of the cache arena: the host path's overflow ring, and two
    sets of staged prefetches."""
    return max(0, min(cfg.B * cfg.K, cfg.E) - C) + 2 * STAGED_PER_LAYER(cfg)


def offload(wl, n_tokens, resident_ms_per_token, pinned_gb, only=None):
    """Capped HBM cache over a pinned host pool: on-demand vs ST-MoE prefetch."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    pool, ptrs, M = expert_pool(wl, pinned_gb, POOL_TIER)
    n_stage = staging_slots(cfg, cfg.C)
    arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, cfg.blob_bytes, n_stage), dtype=torch.uint8,
                        device="cuda:0")
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    keep = None if only is None else set(only.split(",")) | {"on_demand"}
    variants = [v for v in offload_variants(cfg) if keep is None or v["name"] in keep]
    out = {}
    for v in variants:
        out[v["name"]] = offload_run(wl, cfg.C, arena, ptrs, streams, v, n_tokens, resident_ms_per_token)
    od = out["on_demand"]["stall_ms_per_token"]
    out["stall_reduction"] = {v["name"]: (round(1.0 - out[v["name"]]["stall_ms_per_token"] / od, 4) if od > 0
                                          else None) for v in variants if v["name"] != "on_demand"}
    # prefetch against on-demand loading with the same decision site, graph use and eviction rule
    base_of = {(v["device"], v["graph"], v["freq"]): v["name"] for v in variants if v["mode"] == S.MODE_ON_DEMAND}
    same = {}
    for v in variants:
        b = base_of.get((v["device"], v["graph"], v["freq"]))
        if v["mode"] != S.MODE_ON_DEMAND and b is not None:
            ob = out[b]["stall_ms_per_token"]
            same[v["name"]] = {"against": b, "reduction": round(1.0 - out[v["name"]]["stall_ms_per_token"] / ob, 4)
                               if ob > 0 else None}
    out["stall_reduction_vs_same_policy_on_demand"] = same
    out["cache_slots_per_layer"] = cfg.C
    out["host_pool"] = {"distinct_blobs": M, "experts": cfg.L * cfg.E, "slot_of_expert": "(l*E + e) mod distinct_blobs"}
    out["h2d_link"] = ("PCIe, pinned host memory, hipMemcpyAsync on demand/side streams" if POOL_TIER == "host" else
                       "device-to-device copies from the HBM-resident stack (a backing tier faster than PCIe)")
    out["pool_tier"] = POOL_TIER
    del arena
    del pool
    return out


# KV-cache bytes per context token per layer (K and V, bf16) of the models
# whose expert shapes the configs use: grouped-query attention with 8 KV heads
# of 128 (Mixtral-8x7B), 4 of 128 (Qwen3-30B-A3B), 4 of 128 (Qwen3-235B-A22B),
# and DeepSeek-V2-Lite's compressed latent (512 + 64 rope dims, one head).
KV_BYTES_PER_TOKEN = {"mixtral": 2 * 8 * 128 * 2, "qwen30b": 2 * 4 * 128 * 2, "qwen30b-b8": 2 * 4 * 128 * 2,
                      "qwen235b": 2 * 4 * 128 * 2, "dsv2lite": (512 + 64) * 2, "tiny": 2 * 2 * 64 * 4}


def attention_sweep(wl, key, n_tokens, resident_ms_per_token, pinned_gb, contexts):
    """Capped cache with a decode-attention stand-in between MoE layers: the
    prefetch issued after layer l overlaps layer l+1's attention.  Returns
    markdown lines."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    pool, ptrs, M = expert_pool(wl, pinned_gb, POOL_TIER)
    n_stage = staging_slots(cfg, cfg.C)
    arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, cfg.blob_bytes, n_stage), dtype=torch.uint8,
                        device="cuda:0")
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    per_tok = KV_BYTES_PER_TOKEN[key] * cfg.B
    rows = []
    for ctx_len in contexts:
        nbytes = (ctx_len * per_tok + 4095) // 4096 * 4096
        attn = None
        attn_us = 0.0
        if nbytes:
            kv = torch.zeros(nbytes, dtype=torch.uint8, device="cuda:0")
            out = torch.empty(S.calib_read_out_words(nbytes), dtype=torch.int32, device="cuda:0")
            attn = (kv, nbytes, out)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            S.calib_read(kv, nbytes, out)
            e0.record()
            for _ in range(20):
                S.calib_read(kv, nbytes, out)
            e1.record()
            torch.cuda.synchronize()
            attn_us = e0.elapsed_time(e1) * 1e3 / 20
        base_ms = resident_ms_per_token + attn_us * cfg.L / 1e3
        recs = {}
        for v in offload_variants(cfg):
            if v["name"] not in ("on_demand", "st_moe", "st_moe_score4_maxK_after_demand", "on_demand_device",
                                 "st_moe_staged_host", "st_moe_staged_host1", "st_moe_staged_device",
                                 "on_demand_device_freq"):
                continue
            recs[v["name"]] = offload_run(wl, cfg.C, arena, ptrs, streams, v, n_tokens, base_ms, attn)
        od = recs["on_demand"]["stall_ms_per_token"]
        for name, rec in recs.items():
            red = 1.0 - rec["stall_ms_per_token"] / od if od > 0 else float("nan")
            rows.append(f"| {ctx_len} | {nbytes / 1e6:.1f} | {attn_us:.1f} | {name} | {rec['tokens_per_s']} | "
                        f"{rec['ms_per_token']} | {rec['stall_ms_per_token']} | {red:+.3f} |")
    del arena
    del pool
    head = ["| context tokens | KV MB per layer | attention stand-in us per layer | variant | tokens/s | "
            "ms/token | stall ms/token (beyond resident + attention) | stall reduction vs on-demand |",
            "|---|---|---|---|---|---|---|---|"]
    return head + rows


def offload_sweep(wl, n_tokens, resident_ms_per_token, pinned_gb, budgets):
    """Cache budget x predictor variant (with the online update on and off):
    one markdown table of tokens/s, stall and copies."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    pool, ptrs, M = expert_pool(wl, pinned_gb, POOL_TIER)
    cmax = max(budgets)
    n_stage = staging_slots(cfg, min(budgets))
    arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cmax, cfg.blob_bytes, n_stage), dtype=torch.uint8,
                        device="cuda:0")
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    rows = []
    for C in budgets:
        variants = [v for v in offload_variants(cfg) if not v["graph"]]
        variants.insert(3, variant("st_moe_frozen_cct", S.MODE_STMOE, online=0))
        base = None
        for v in variants:
            rec = offload_run(wl, C, arena, ptrs, streams, v, n_tokens, resident_ms_per_token)
            if v["name"] == "on_demand":
                base = rec["stall_ms_per_token"]
            red = 1.0 - rec["stall_ms_per_token"] / base if base and base > 0 else float("nan")
            cst = rec["cache"]
            rows.append(f"| {C} | {v['name']} | {rec['tokens_per_s']} | {rec['stall_ms_per_token']} | {red:+.3f} | "
                        f"{cst['hits']} | {cst['demand'] + cst['overflow']} | {cst['prefetch']} | "
                        f"{cst['useful']} | {rec.get('recall_layers_ge1', '-')} | {rec.get('precision', '-')} |")
    del arena
    del pool
    head = [f"| C per layer | variant | tokens/s | stall ms/token | stall reduction vs on-demand | hits | "
            f"demand + overflow copies | prefetch copies | useful prefetches | recall (l >= 1) | precision |",
            "|---|---|---|---|---|---|---|---|---|---|---|"]
    return head + rows


def handoff_probe(iters=60, n_chunks=40, reps=2):
    """Markdown: the handoff a single gate/up + down launch would need, at the
    shape of a Qwen3-30B layer at batch 1 (1536 producer workgroups streaming
    32 KiB each, 1024 consumer workgroups streaming 24 KiB each into registers
    and then reading all 1536 published words), as two launches and as one
    launch with write-through stores or release/acquire, every consumer polling
    the count, or with the count's last producer (mode 4: counted in 64 group
    words first) setting flag copies that the consumers poll.  Every iteration uses
    another of n_chunks copies of the data (3 GB in all: no cache holds it);
    each mode's last output is checked against the two-launch result."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    P, Q, C1, C2 = 1536, 1024, 32 << 10, 24 << 10
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(2606)
    w1 = torch.randint(-2 ** 31, 2 ** 31 - 1, (n_chunks * P * C1 // 4,), dtype=torch.int32, device=dev, generator=g)
    w2 = torch.randint(-2 ** 31, 2 ** 31 - 1, (n_chunks * Q * C2 // 4,), dtype=torch.int32, device=dev, generator=g)
    act = torch.zeros(P, dtype=torch.int32, device=dev)
    out = torch.zeros(Q, dtype=torch.int32, device=dev)
    ref = torch.zeros(Q, dtype=torch.int32, device=dev)
    sync = torch.zeros(S.HANDOFF_SYNC_WORDS, dtype=torch.int32, device=dev)
    n1, n2 = P * C1 // 4, Q * C2 // 4
    target = 0
    names = {0: "two launches", 1: "one launch, write-through stores + relaxed counter",
             2: "one launch, release/acquire counter",
             3: "one launch, relaxed counter, the last producer sets 64 flag copies",
             4: "one launch, 64 group counters, the last group sets 64 flag copies"}
    times = {m: [] for m in names}
    checks = {}
    torch.cuda.synchronize()
    for _ in range(reps):
        for mode in names:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for it in range(iters):
                k = it % n_chunks
                if mode:
                    target += P
                S.calib_handoff(w1[k * n1:(k + 1) * n1], C1, P, w2[k * n2:(k + 1) * n2], C2, Q, mode, act, out,
                                sync, target)
            e1.record()
            torch.cuda.synchronize()
            times[mode].append(1e3 * e0.elapsed_time(e1) / iters)
            k = (iters - 1) % n_chunks
            S.calib_handoff(w1[k * n1:(k + 1) * n1], C1, P, w2[k * n2:(k + 1) * n2], C2, Q, 0, act, ref, sync,
                            target)
            torch.cuda.synchronize()
            checks[mode] = (bool(torch.equal(out, ref)), int(sync[1].item()))
    mb = (P * C1 + Q * C2) / 1e6
    lines = ["Producer -> consumer handoff (`stmoe_calib_handoff`), Qwen3-30B batch-1 FFN shape: "
             f"{P} x {C1 >> 10} KiB producers, {Q} x {C2 >> 10} KiB consumers, {mb:.1f} MB per iteration, "
             f"{iters} iterations per run over {n_chunks} copies of the data:", "",
             "| mode | us per iteration (runs) | GB/s | output equal to two launches | wait error word |",
             "|---|---|---|---|---|"]
    for m, name in names.items():
        best = min(times[m])
        lines.append(f"| {name} | {' / '.join(f'{t:.2f}' for t in times[m])} | {mb * 1e3 / best:.0f} | "
                     f"{'yes' if checks[m][0] else 'NO'} | {checks[m][1]} |")
    return lines


def copy_sweep(wl, n_tokens, resident_ms_per_token, pinned_gb, workgroups):
    """The expert tier's bandwidth as a measured sweep: with device decisions
    the copy kernels' workgroup count sets the copy rate (from the pinned host
    pool, or from the HBM pool with --pool hbm, up to TB/s).  Per count: the
    rate of stmoe_calib_copy_grid on the same pool, then on-demand loading,
    ST-MoE prefetch (into slots and staged) and frequency-aware on-demand
    loading, all with that many copy workgroups.  Markdown lines."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    cfg = wl.cfg
    pool, ptrs, M = expert_pool(wl, pinned_gb, POOL_TIER)
    n_stage = staging_slots(cfg, cfg.C)
    arena = torch.empty(S.cache_arena_bytes(cfg.L, cfg.E, cfg.C, cfg.blob_bytes, n_stage), dtype=torch.uint8,
                        device="cuda:0")
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    dst = torch.empty(cfg.blob_bytes, dtype=torch.uint8, device="cuda:0")
    n_st = STAGED_PER_LAYER(cfg)
    rows = []
    for n in workgroups:
        srcs = [ptrs[(7919 * i) % len(ptrs)] for i in range(8)]
        S.calib_copy_grid(srcs[0], dst.data_ptr(), cfg.blob_bytes, n)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for src in srcs:
            S.calib_copy_grid(src, dst.data_ptr(), cfg.blob_bytes, n)
        e1.record()
        torch.cuda.synchronize()
        gbps = len(srcs) * cfg.blob_bytes / (e0.elapsed_time(e1) * 1e-3) / 1e9
        vs = [variant("on_demand_device", S.MODE_ON_DEMAND, device=1, copy_wgs=n),
              variant("st_moe_device", S.MODE_STMOE, device=1, copy_wgs=n),
              variant("st_moe_staged_device", S.MODE_STMOE, after_demand=1, device=1, staged=n_st, copy_wgs=n),
              variant("on_demand_device_freq", S.MODE_ON_DEMAND, device=1, freq=1, copy_wgs=n)]
        base = None
        for v in vs:
            rec = offload_run(wl, cfg.C, arena, ptrs, streams, v, n_tokens, resident_ms_per_token)
            if base is None:
                base = rec["stall_ms_per_token"]
            red = 1.0 - rec["stall_ms_per_token"] / base if base > 0 else float("nan")
            c = rec["cache"]
            rows.append(f"| {n} | {gbps:.1f} | {v['name']} | {rec['tokens_per_s']} | {rec['stall_ms_per_token']} | "
                        f"{red:+.3f} | {c['demand']} / {c['overflow']} / {c['prefetch']} ({c['useful']}, "
                        f"{c['wasted']}) |")
            log(f"copy sweep {n} workgroups ({gbps:.1f} GB/s) {v['name']}: {rec['tokens_per_s']} tok/s")
    del arena, dst
    del pool
    head = [f"HBM-resident reference: {resident_ms_per_token:.3f} ms/token; {n_tokens} tokens per run; pool: "
            f"{POOL_TIER}",
            "| copy workgroups | copy GB/s | variant | tokens/s | stall ms/token | stall reduction vs on-demand "
            "(same copy rate) | demand / overflow / prefetch (useful, wasted) copies |",
            "|---|---|---|---|---|---|---|"]
    return head + rows


def near_tie_rows(wl, warmup, steps, eps=1e-4):
    """Routed rows of the timed tokens whose K-th and (K+1)-th router logits
    (fp64) differ by less than eps: their expert set may legitimately differ
    between fp32 and fp64 arithmetic."""
    cfg = wl.cfg
    if cfg.K >= cfg.E:
        return {"rows": 0, "of": 0, "eps": eps}
    from paper_2606_15453_amd import workload as W

    def exact(a):   # stored values (bf16 bits or fp32) as float64
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64) if a.dtype == np.uint16 \
            else a.astype(np.float64)

    wg = [exact(W.to_storage(cfg, g)) for g in wl.wg_f64]
    n, rows = 0, 0
    for i in range(steps):
        t = (warmup + i) % wl.T
        for l in range(cfg.L):
            z = np.sort(exact(wl.x_store[t][l]) @ wg[l].T, axis=1)[:, ::-1]
            n += int(np.sum(z[:, cfg.K - 1] - z[:, cfg.K] < eps))
            rows += z.shape[0]
    return {"rows": n, "of": rows, "eps": eps}


# ---------------------------------------------------------------------------
# Policy bound: what prefetching with one layer of lookahead can win on this
# link, priced by a time model (CPU arithmetic on the routing trace and the
# GPU predictor's predictions; no kernel timing beyond the measured inputs).
# ---------------------------------------------------------------------------

class _Link:
    """One host-to-device link serving copies first in, first out."""

    def __init__(self, copy_ms):
        self.copy_ms = copy_ms
        self.free = 0.0

    def put(self, t, ms=None):
        ms = self.copy_ms if ms is None else ms
        self.free = max(self.free, t) + ms
        return self.free


class _Lru:
    """Per-layer C-slot cache: least recently used with protection of the
    current set (the library's policy), or the offline optimum (evict the
    expert whose next use in this layer is farthest), or, for the online
    alternatives, the least frequently used (counts seeded from profiling,
    +1 per token that selects the expert) or the lowest score of a given
    per-expert vector, ties by least recent use."""

    def __init__(self, warm, C, future=None, counts=None):
        self.slots = [list(w) for w in warm]
        self.last = [[0] * C for _ in warm]
        self.C = C
        self.future = future          # future[l] = list over tokens of sets, for the offline optimum
        self.freq = None if counts is None else [list(r) for r in counts]

    def victim(self, l, keep, t=None, score=None):
        cands = [c for c in range(self.C) if self.slots[l][c] < 0 or self.slots[l][c] not in keep]
        if not cands:
            return -1
        if score is not None or self.freq is not None:
            val = score if score is not None else self.freq[l]
            return min(cands, key=lambda c: (val[self.slots[l][c]] if self.slots[l][c] >= 0 else -1,
                                             self.last[l][c], c))
        if self.future is None:
            return min(cands, key=lambda c: (self.last[l][c], c))

        def nxt(e):
            for tt in range(t + 1, len(self.future[l])):
                if e in self.future[l][tt]:
                    return tt
            return 1 << 30
        return max(cands, key=lambda c: (nxt(self.slots[l][c]) if self.slots[l][c] >= 0 else 1 << 31, -c))

    def acquire(self, l, U, stamp, t=None, score=None):
        keep = set(U)
        misses, overflow = [], []
        for f in U:
            if f in self.slots[l]:
                self.last[l][self.slots[l].index(f)] = stamp
                continue
            c = self.victim(l, keep, t, score)
            if c < 0:
                overflow.append(f)
                continue
            self.slots[l][c] = f
            self.last[l][c] = stamp
            misses.append(f)
        if self.freq is not None:
            for f in U:
                self.freq[l][f] += 1
        return misses, overflow

    def prefetch(self, l, ranked, stamp, t=None):
        ranked = ranked[:self.C]
        keep = set(ranked)
        out = []
        for f in ranked:
            if f in self.slots[l]:
                continue
            c = self.victim(l, keep, t)
            if c < 0:
                break
            self.slots[l][c] = f
            self.last[l][c] = stamp
            out.append(f)
        return out


NO_PREFETCH = ("demand", "optimum", "demand_lfu", "demand_cct")


def simulate_policy(trace, preds, L, C, warm, copy_ms, layer_ms, attn_ms, policy, max_staged=None,
                    counts=None, cct=None):
    """Time model of the capped decode loop.  trace[t][l]: distinct selected
    experts; preds[t][l]: the admitted ranking for the layer after (t, l).
    Per layer: the attention window (attn_ms), routing and decisions, the
    missed copies on the link (the FFN waits for every copy it needs), the FFN
    (layer_ms covers routing and FFN), and the next layer's prefetches queued
    on the link behind this layer's missed copies.

    policy: "demand" (no prefetch), "evict" (prefetch into LRU victims, the
    copies run to the end), "staged" (prefetch into spare buffers without
    eviction, cancelled when the next layer's routing shows them unused),
    "perfect_evict" / "perfect_staged" (the same with the exact next-layer
    selection as the prediction), "optimum" (offline-optimal replacement, no
    prefetch); online replacement alternatives without prefetch: "demand_lfu"
    (least frequently used, counts[l][e] seeds), "demand_cct" (evict the
    expert with the lowest Eq. 1 spatial score from the previous layer's
    current selection through cct = (cct_idx, cct_conf); layer 0 by counts).
    Returns (stall ms per token, copies started, copy-ms wasted)."""
    T = len(trace)
    future = [[trace[t][l] for t in range(T)] for l in range(L)] if policy == "optimum" else None
    cache = _Lru(warm, C, future, counts if policy == "demand_lfu" else None)
    link = _Link(copy_ms)
    clock, copies, wasted = 0.0, 0, 0.0
    pend = {}                     # layer -> [(expert, start, end)] prefetch copies issued for it
    perfect = policy.startswith("perfect")
    staged = policy.endswith("staged")
    for t in range(T):
        for l in range(L):
            clock += attn_ms
            route_end = clock + 0.05 * layer_ms
            U = trace[t][l]
            stamp = t * L + l + 1
            jobs = pend.pop(l, [])
            ready = route_end
            if staged:
                # the link at route_end: unused staged copies stop there; the used ones go on
                keep = [j for j in jobs if j[0] in U]
                drop = [j for j in jobs if j[0] not in U]
                for f, s0, e0 in drop:
                    wasted += max(0.0, min(e0, route_end) - s0)
                # only this layer's staged copies can still be on the link here
                link.free = min(link.free, route_end)
                for f, s0, e0 in keep:
                    rest = e0 - max(s0, route_end) if e0 > route_end else 0.0
                    end = link.put(route_end, rest) if rest > 0 else e0
                    ready = max(ready, end)
                staged_ok = {j[0] for j in keep}
                misses, overflow = cache.acquire(l, U, stamp, t)
                for f in misses + overflow:
                    if f in staged_ok:
                        continue
                    ready = max(ready, link.put(route_end))
                    copies += 1
            else:
                inflight = {f: e0 for f, _, e0 in jobs}
                for f, s0, e0 in jobs:
                    if f not in U:
                        wasted += e0 - s0
                score = None
                if policy == "demand_cct":
                    if l == 0:
                        score = list(counts[0])
                    else:
                        sc = np.zeros(len(counts[l]))
                        for f in trace[t][l - 1]:
                            np.add.at(sc, np.asarray(cct[0][l - 1][f], np.int64), np.asarray(cct[1][l - 1][f]))
                        score = sc.tolist()
                misses, overflow = cache.acquire(l, U, stamp, t, score)
                for f in U:
                    if f in inflight and f not in misses:
                        ready = max(ready, inflight[f])
                for f in misses + overflow:
                    ready = max(ready, link.put(route_end))
                    copies += 1
            clock = ready + 0.95 * layer_ms
            # prefetch for the next layer, behind this layer's missed copies
            if policy in NO_PREFETCH:
                continue
            nl, nt = (l + 1) % L, t + (l + 1) // L
            if perfect:
                if nt >= T:
                    continue
                ranked = [f for f in trace[nt][nl]]
            else:
                ranked = preds[t][l]
            if staged:
                resident = set(cache.slots[nl])
                cand = [f for f in ranked if f not in resident][:max_staged or C]
                out = []
                for f in cand:
                    end = link.put(route_end)
                    out.append((f, end - copy_ms, end))
                    copies += 1
                pend[nl] = out
            else:
                got = cache.prefetch(nl, ranked, stamp, t)
                out = []
                for f in got:
                    end = link.put(route_end)
                    out.append((f, end - copy_ms, end))
                    copies += 1
                pend[nl] = out
    ideal = T * L * (attn_ms + layer_ms)
    return (clock - ideal) / T, copies, wasted


POLICIES = ("demand", "evict", "staged", "perfect_evict", "perfect_staged", "optimum", "demand_lfu", "demand_cct")


def policy_bound(names, n_tokens, attn_list, links=("measured",)):
    """Markdown table of simulate_policy over the planted traces, with the GPU
    predictor's rankings (paper threshold) and measured inputs: the H2D copy
    time of one expert (pinned host -> HBM, event-timed) and the layer time of
    the HBM-resident decode (router + FFN, event-timed on one layer's call).
    links: "measured" and/or link rates in GB/s; a rate replaces the measured
    copy time by blob bytes / rate (the sensitivity of each policy to the
    bandwidth of the tier the experts come from)."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    dev = "cuda:0"
    out = ["| workload | link GB/s | copy ms | attention ms/layer | policy | copies | wasted copy-ms | "
           "stall ms/token | stall vs on-demand |", "|---|---|---|---|---|---|---|---|---|"]
    for name in names:
        cfg = W.CONFIGS[name]
        T = min(n_tokens, cfg.T)
        sel = W.planted_trace(cfg, n_tokens=cfg.P + T)
        prof = sel[:cfg.P]
        dec = sel[cfg.P:]
        trace = [[sorted(set(int(v) for b in range(cfg.B) for v in dec[t, b, l])) for l in range(cfg.L)]
                 for t in range(T)]
        # the GPU predictor's admitted rankings (paper threshold, capped at C)
        p = S.Predictor(cfg.L, cfg.E, cfg.K, cfg.B)
        p.profile(prof)
        _, cct_idx, cct_conf, _ = p.export()          # the profiled tables, for demand_cct
        counts = np.zeros((cfg.L, cfg.E), np.int64)     # profiling tokens that select each expert
        for t in range(cfg.P):
            for l in range(cfg.L):
                counts[l, np.unique(prof[t, :, l])] += 1
        ranked = torch.zeros(cfg.E, dtype=torch.int32, device=dev)
        nr = torch.zeros(1, dtype=torch.int32, device=dev)
        dsel = torch.from_numpy(np.ascontiguousarray(dec.transpose(0, 2, 1, 3))).to(dev)
        preds = []
        for t in range(T):
            row = []
            for l in range(cfg.L):
                cur = dsel[t, l]
                p.update(l, dsel[t, l - 1] if l else None, cur)
                if l + 1 < cfg.L:
                    p.predict(l, cur, use=S.USE_BOTH, ranked=ranked, n_ranked=nr)
                else:
                    p.predict(-1, None, use=S.USE_HT, ranked=ranked, n_ranked=nr)
                n = int(nr.item())
                row.append(ranked[:n].cpu().tolist())
            preds.append(row)
        p.close()
        # measured inputs: one expert's H2D copy, one layer's resident routing + FFN
        blob = cfg.blob_bytes
        host = torch.empty(blob, dtype=torch.uint8).pin_memory()
        devb = torch.empty(blob, dtype=torch.uint8, device=dev)
        devb.copy_(host, non_blocking=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            devb.copy_(host, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        copy_ms = e0.elapsed_time(e1) / 5
        del host, devb
        layer_ms = ffn_layer_ms(cfg)
        warm = S.warm_sets(prof, cfg.E, cfg.C)
        log(f"policy bound {name}: copy {copy_ms:.3f} ms, layer {layer_ms:.4f} ms, {T} tokens")
        for link in links:
            cms = copy_ms if link == "measured" else blob / (float(link) * 1e6)
            rate = f"{blob / cms / 1e6:.0f}" + (" (measured)" if link == "measured" else "")
            for attn in attn_list:
                base = None
                for pol in POLICIES:
                    stall, copies, wasted = simulate_policy(trace, preds, cfg.L, cfg.C, warm, cms, layer_ms,
                                                            attn, pol, max_staged=cfg.C, counts=counts,
                                                            cct=(cct_idx, cct_conf))
                    if base is None:
                        base = stall
                    rel = f"{1 - stall / base:+.3f}" if base > 1e-9 else "-"
                    out.append(f"| {cfg.name} (layer {layer_ms:.3f} ms) | {rate} | {cms:.4f} | {attn:.2f} | {pol} | "
                               f"{copies} | {wasted:.1f} | {stall:.2f} | {rel} |")
    return out


def summarize_policy(path):
    """Pivot of a --policy-bound table: per workload, link rate and attention
    window, the on-demand stall and each policy's stall reduction against it."""
    tab = {}
    for line in open(path):
        c = [x.strip() for x in line.strip().strip("|").split("|")]
        if len(c) != 9 or c[0] == "workload" or c[0].startswith("---"):
            continue
        key = (c[0].split(" (")[0], c[1].split(" ")[0] + (" (measured)" if "measured" in c[1] else ""), c[3])
        tab.setdefault(key, {})[c[4]] = (float(c[7]), c[8])
    pols = [p for p in POLICIES[1:] if any(p in v for v in tab.values())]
    print("| workload | link GB/s | attention ms/layer | on-demand stall ms/token | "
          + " | ".join(pols) + " |")
    print("|---" * (4 + len(pols)) + "|")
    for (w, link, attn), v in tab.items():
        print(f"| {w} | {link} | {attn} | {v['demand'][0]:.2f} | " + " | ".join(v[p][1] for p in pols) + " |")


def ffn_layer_ms(cfg, reps=20):
    """Event-timed routing + expert FFN of one layer at the config's shape
    (the distinct experts of one seeded routing generated in HBM)."""
    import torch
    from paper_2606_15453_amd import stmoe as S
    from paper_2606_15453_amd import workload as W
    dev = "cuda:0"
    rng = np.random.default_rng(cfg.seed)
    idx = np.stack([rng.choice(cfg.E, cfg.K, replace=False) for _ in range(cfg.B)]).astype(np.int32)
    w = rng.random((cfg.B, cfg.K)).astype(np.float32)
    selx = sorted(set(idx.ravel().tolist()))
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    store = torch.empty((len(selx) + cfg.n_shared, cfg.blob_elems), dtype=tdt, device=dev)
    for k, e in enumerate(selx):
        W.expert_blob_torch(cfg, 0, e, store[k])
    for sh in range(cfg.n_shared):
        W.expert_blob_torch(cfg, 0, sh, store[len(selx) + sh], shared=True)
    ptrs = [store[0].data_ptr()] * cfg.E
    for k, e in enumerate(selx):
        ptrs[e] = store[k].data_ptr()
    eptr = torch.tensor(ptrs, dtype=torch.int64, device=dev)
    sptr = (torch.tensor([store[len(selx) + sh].data_ptr() for sh in range(cfg.n_shared)], dtype=torch.int64,
                         device=dev) if cfg.n_shared else None)
    dt = S.BF16 if cfg.dtype == "bf16" else S.F32
    x = Workload._dev(W.to_storage(cfg, rng.normal(0, 1, (cfg.B, cfg.H))))
    wg = Workload._dev(W.router_rows(cfg, 0))
    y = torch.empty((cfg.B, cfg.H), dtype=torch.float32, device=dev)
    ws = torch.zeros(S.ffn_workspace_bytes(cfg.B, cfg.K, cfg.E, cfg.H, cfg.I, cfg.n_shared, dt),
                     dtype=torch.uint8, device=dev)
    rws = torch.zeros(S.route_workspace_bytes(cfg.B, cfg.E), dtype=torch.uint8, device=dev)
    ti, tw = torch.from_numpy(idx).to(dev), torch.from_numpy(w).to(dev)
    ri, rw = torch.empty_like(ti), torch.empty_like(tw)

    def call():
        S.route_topk(x, wg, cfg.K, ri, rw, rws, dtype=dt)
        S.expert_ffn(x, ti, tw, cfg.H, cfg.I, cfg.E, dt, eptr, y, ws, shared_ptrs=sptr, n_shared=cfg.n_shared)

    for _ in range(3):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    del store
    return e0.elapsed_time(e1) / reps


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline_run(wl, max_tokens, target_s):
    """The CPU oracle on the first decode tokens of the same workload, until
    `target_s` seconds of timed work (at most max_tokens tokens).

    Timed: routing, predictor update/predict, cache policy and the fp64 FFN of
    every layer.  Not timed: preparing each layer's fp64 expert matrices (the
    generator's GPU blobs widened to fp64 on the GPU and copied into pinned
    host buffers)."""
    import torch
    from oracle.stmoe_oracle import STPredictor, CacheSim, admitted, decode_storage, moe_ffn, route, \
        warm_from_profile
    cfg = wl.cfg
    pred = STPredictor(cfg.L, cfg.E, cfg.K, cfg.B)
    pred.profile(wl.prof)
    cache = CacheSim(cfg.L, cfg.E, cfg.C, warm_from_profile(wl.prof, cfg.L, cfg.E, cfg.C))
    timed = 0.0
    n, Hh, Ii = cfg.H * cfg.I, cfg.H, cfg.I
    n_bufs = min(cfg.B * cfg.K, cfg.E) + cfg.n_shared
    bufs = [torch.empty(cfg.blob_elems, dtype=torch.float64, pin_memory=True) for _ in range(n_bufs)]
    used = [0]

    def mats(blob):
        buf = bufs[used[0]]
        used[0] += 1
        buf.copy_(blob.to(torch.float64))
        b = buf.numpy()
        return b[:n].reshape(Ii, Hh), b[n:2 * n].reshape(Ii, Hh), b[2 * n:].reshape(Hh, Ii)

    n_tokens = 0
    for t in range(min(max_tokens, wl.T)):
        if timed >= target_s:
            break
        n_tokens += 1
        prev = None
        for l in range(cfg.L):
            x = decode_storage(wl.x_store[t][l])
            t0 = time.perf_counter()
            r = route(x, wl.wg_f64[l], cfg.K)
            cur = [sorted(int(v) for v in r["idx"][b]) for b in range(cfg.B)]
            pred.update(l, prev, cur)
            P_next = pred.predict(l, cur) if l + 1 < cfg.L else pred.predict(-1, None)
            U = sorted(set(v for s in cur for v in s))
            cache.acquire(l, U, t * cfg.L + l + 1)
            timed += time.perf_counter() - t0
            used[0] = 0
            experts = {e: mats(wl.blob(l, e)) for e in U}
            shared = [mats(wl.shared[l * cfg.n_shared + s]) for s in range(cfg.n_shared)]
            t0 = time.perf_counter()
            moe_ffn(x, r["idx"], r["w"], lambda e: experts[e], shared=shared)
            cache.prefetch((l + 1) % cfg.L, admitted(P_next), t * cfg.L + l + 1)
            timed += time.perf_counter() - t0
            prev = cur
            del experts
    del bufs
    return n_tokens, timed


def cpu_baseline(wl, max_tokens, target_s):
    """The oracle timed twice on the host: with every core its BLAS library
    uses, and single-threaded (BLAS limited to one thread)."""
    cfg = wl.cfg
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except ImportError:
        threadpool_info = threadpool_limits = None
    cores = os.cpu_count()
    if threadpool_info is not None:
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    n_all, t_all = cpu_baseline_run(wl, max_tokens, target_s)
    single = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            n_one, t_one = cpu_baseline_run(wl, max_tokens, target_s)
        single = dict(value=round(cfg.B * n_one / t_one, 4), seconds=round(t_one, 3), tokens=n_one, cores=1)
    return dict(value=round(cfg.B * n_all / t_all, 4), unit="tokens/s", cores=int(cores),
                kind="oracle", seconds=round(t_all, 3), single_thread=single,
                host_cpus=os.cpu_count(), cpu_model=cpu_model(),
                sample=f"first {n_all} decode token(s) x {cfg.L} layers x batch {cfg.B} of the same "
                       f"workload: fp64 routing, predictor, cache policy and SwiGLU FFN, {t_all:.1f} s of "
                       f"timed CPU work on {cores} BLAS threads (expert matrix preparation not timed); "
                       f"single_thread: the same with BLAS limited to one thread")


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.summarize_gaps:
        summarize_gaps(*args.summarize_gaps)
        return
    if args.summarize_overlap:
        summarize_overlap(*args.summarize_overlap)
        return
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.summarize_floor:
        summarize_floor(*args.summarize_floor)
        return
    if args.summarize_policy:
        summarize_policy(args.summarize_policy)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return
    if args.summarize_offload:
        summarize_offload(args.summarize_offload)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported (this implementation has no "
              f"multi-GPU path)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_15453_amd import workload as W
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.counters:
        counters_workload(args.config, args.counters_meta)
        return
    if args.policy_bound:
        lines = policy_bound(args.policy_bound.split(","), max(args.offload_tokens, 1),
                             [float(a) for a in args.policy_attn.split(",")], args.policy_link.split(","))
        print("\n".join(lines), flush=True)
        return
    if args.ffn_sweep:
        ffn_sweep()
        return
    if args.read_floor:
        read_floor()
        return
    if args.reread_probe:
        reread_probe()
        return
    if args.handoff_probe:
        print("\n".join(handoff_probe()), flush=True)
        return
    if args.predictor_sweep:
        predictor_sweep()
        return
    if args.predictor_spread:
        print("\n".join(predictor_spread()), flush=True)
        return
    global POOL_TIER
    POOL_TIER = args.pool
    cfg = W.CONFIGS[args.config]
    log(f"workload {cfg.name}")
    total = torch.cuda.get_device_properties(0).total_memory
    if cfg.L * cfg.E * cfg.blob_bytes > 0.8 * total:
        # the stack does not fit in HBM: alias a pool of distinct blobs, and
        # generate hidden states only for the tokens this run decodes
        n_tok = max(args.warmup + args.steps, args.offload_tokens, 1)
        wl = Workload(cfg, hbm_blobs=int(args.hbm_pool_gb * 1e9) // cfg.blob_bytes, x_tokens=n_tok)
    else:
        wl = Workload(cfg)
    if args.attention_sweep:
        contexts = [int(c) for c in args.attention_sweep.split(",")]
        r = hbm_resident(wl, 40, 5)
        res_ms = 1e3 * r["seconds"] / 40
        lines = attention_sweep(wl, args.config, max(args.offload_tokens, 1), res_ms, args.pinned_gb, contexts)
        print(f"HBM-resident reference: {res_ms:.3f} ms/token; {max(args.offload_tokens, 1)} tokens per run")
        print("\n".join(lines), flush=True)
        return
    if args.copy_sweep:
        r = hbm_resident(wl, 40, 5)
        res_ms = 1e3 * r["seconds"] / 40
        lines = copy_sweep(wl, max(args.offload_tokens, 1), res_ms, args.pinned_gb,
                           [int(c) for c in args.copy_sweep.split(",")])
        print("\n".join(lines), flush=True)
        return
    if args.offload_sweep:
        budgets = [int(c) for c in args.offload_sweep.split(",")]
        r = hbm_resident(wl, 40, 5)
        res_ms = 1e3 * r["seconds"] / 40
        lines = offload_sweep(wl, max(args.offload_tokens, 1), res_ms, args.pinned_gb, budgets)
        print(f"HBM-resident reference: {res_ms:.3f} ms/token; {max(args.offload_tokens, 1)} tokens per run")
        print("\n".join(lines), flush=True)
        return
    r = hbm_resident(wl, args.steps, args.warmup)
    ms_per_step = 1e3 * r["seconds"] / args.steps
    value = cfg.B * args.steps / r["seconds"]
    log(f"HBM-resident: {value:.2f} tok/s, {ms_per_step:.3f} ms/token, "
        f"host issue {r['host_issue_us_per_layer']:.1f} us/layer")
    esz = cfg.wbytes
    up_bytes = r["n_experts"] * 2 * cfg.H * cfg.I * esz + r["n_calls"] * cfg.n_shared * 2 * cfg.H * cfg.I * esz
    dn_bytes = r["n_experts"] * cfg.H * cfg.I * esz + r["n_calls"] * cfg.n_shared * cfg.H * cfg.I * esz
    up_gbps = up_bytes / (r["up_ms"] * 1e-3) / 1e9
    dn_gbps = dn_bytes / (r["down_ms"] * 1e-3) / 1e9
    ffn_gbps = (up_bytes + dn_bytes) / ((r["up_ms"] + r["down_ms"]) * 1e-3) / 1e9
    stats = r["stats"]
    out = {
        "metric": "MoE decode tokens/s; expert-weight HBM GB/s vs peak; prefetch hit rate",
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "repeats": repeat_summary(cfg.B * args.steps, [r["seconds"]] + r["repeat_seconds"]),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "accum_dtype": "f32",
        "data": "synthetic (seeded planted-Markov routing, N(0, 0.02) expert weights)",
        "config": {"workload": cfg.name, "layers": cfg.L, "hidden": cfg.H, "intermediate": cfg.I,
                   "experts": cfg.E, "shared_experts": cfg.n_shared, "top_k": cfg.K, "global_batch": cfg.B,
                   "mode": ("all experts HBM-resident, ST-MoE predictor on" if not wl.aliased else
                            f"HBM-resident stand-in: {wl.n_blobs} distinct expert blobs in HBM, expert (l, e) "
                            f"reads blob (l*E + e) mod {wl.n_blobs} (the stack does not fit in HBM); "
                            f"ST-MoE predictor on"),
                   "parallelism": "none (1 GPU)",
                   "launch": "eager launches; the predictor's update/predict of every layer in one side-stream "
                             "launch per token, overlapping the next token"},
        "roofline": {
            "bound": "hbm", "kernel": "ffn_gate_up",
            "achieved": round(up_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(up_gbps / PEAK_HBM_GBPS, 4),
            "traffic": committed_traffic() if cfg.name == W.CONFIGS["mixtral"].name else None,
            "bytes_per_launch": int(up_bytes / max(r["n_calls"], 1)),
            "avg_launch_us": round(1e3 * r["up_ms"] / max(r["n_calls"], 1), 3),
            "launches": r["n_calls"],
            "event_sampling": ("HIP events around the FFN launches of "
                               + (f"every {timing_cadence(args.steps)}th token" if timing_cadence(args.steps) > 1
                                  else "every token") + " of the timed region"),
        },
        "ffn_down": {"achieved_gbps": round(dn_gbps, 1), "frac": round(dn_gbps / PEAK_HBM_GBPS, 4),
                     "avg_launch_us": round(1e3 * r["down_ms"] / max(r["n_calls"], 1), 3)},
        "ffn_hbm_gbps": round(ffn_gbps, 1),
        # expert-weight bytes per token from the event-timed tokens, over the whole timed region
        "step_hbm_gbps": round((up_bytes + dn_bytes) / max(r["n_calls"] / cfg.L, 1e-9) * args.steps
                               / r["seconds"] / 1e9, 1),
        "layer_us": round(1e6 * r["seconds"] / args.steps / cfg.L, 2),
        # event-timed stages per layer (every TIMING_EVERY-th token); the side-stream
        # predictor overlaps the FFN and the next router
        "stages_us_per_layer": r["stages_us"],
        "routing_near_tie_rows": near_tie_rows(wl, warmup=args.warmup, steps=args.steps),
        "host_issue_us_per_layer": round(r["host_issue_us_per_layer"], 2),
        "prediction": {
            "recall_layers_ge1": round(float(stats[1:, 0].sum() / max(stats[1:, 1].sum(), 1)), 4),
            "recall_layer0": round(float(stats[0, 0] / max(stats[0, 1], 1)), 4),
            "precision": round(float(stats[:, 0].sum() / max(stats[:, 2].sum(), 1)), 4),
        },
    }
    read_stride = achievable_read_gbps(pattern=0)
    read_blocked = achievable_read_gbps(pattern=1)
    read_gbps = max(read_stride, read_blocked)
    out["achievable_read_gbps"] = {"grid_stride": round(read_stride, 1), "contiguous_per_workgroup":
                                   round(read_blocked, 1)}
    out["roofline"]["frac_of_achievable_read"] = round(up_gbps / read_gbps, 4)
    log(f"streaming-read probes: grid stride {read_stride:.0f} GB/s, contiguous per workgroup "
        f"{read_blocked:.0f} GB/s")
    if args.offload_tokens > 0:
        out["offload"] = offload(wl, args.offload_tokens, ms_per_step, args.pinned_gb, args.offload_only)
    if args.cpu_tokens > 0:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_tokens, args.cpu_seconds)
        log(f"cpu baseline {out['cpu_baseline']['value']} tok/s in {time.time() - t0:.1f}s wall")
    if args.largest_tokens > 0 and args.config == "mixtral":
        del wl
        torch.cuda.empty_cache()
        t0 = time.time()
        out["largest_config"] = largest_config(args.largest_tokens, 2, args.hbm_pool_gb, args.largest_capped_tokens,
                                               args.pinned_gb)
        log(f"largest config {out['largest_config']['workload']}: {out['largest_config']['tokens_per_s']} tok/s "
            f"({time.time() - t0:.1f}s wall)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
