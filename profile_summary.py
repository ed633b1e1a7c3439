"""Summaries of rocprofv3 runs of bench.py, written into profiles/.

Two kinds of run are summarised (commands as recorded in each summary):

  trace     rocprofv3 --kernel-trace --stats --output-format csv -d DIR -o run --
                python3 bench.py --workload WL [bench flags]
            -> profiles/step_kernels_WL.md: per-step kernel table of the timed
               (graph-replayed) pass, step/draft/verify/tail spans between the
               step's wall-clock stamp kernels, and the verify GEMM launches of
               the timed and the eager (event-timed) pass, per GEMM role.

  counters  rocprofv3 --pmc <counters> --output-format csv -d DIR/<name> -o run --
                python3 bench.py --workload WL --counter-sample
            for <name> in fetch (FETCH_SIZE), write (WRITE_SIZE) and
            sq (SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES
            SQ_BUSY_CYCLES GRBM_GUI_ACTIVE)
            -> profiles/counters_WL.md, and for the 7B 512-token workload the
               record bench.py reads (verify_gemm_llama7b_p512_traffic.json).

Steps are found through the stamp kernels every decode step launches (four
per step: draft start, verify start, verify end, step end).  A speculative
step is told from a plain greedy one by its verify GEMMs covering more than one
16-row tile block.  The byte counters are scaled by what they read for the
sample's three 1 GiB device copies (2^20 KiB read and 2^20 KiB written).

  attn      rocprofv3 --pmc <counters> --output-format csv -d DIR/<name> -o run --
                python3 bench.py --workload WL --counter-sample --counter-prompt P
            for <name> in sq (ATTN_COUNTERS) and optionally fetch (FETCH_SIZE)
            and write (WRITE_SIZE)
            -> profiles/attn_counters_WL.md: instruction mix and HBM bytes of
               the verify pass's two tree-attention kernels per dispatch.

usage: python profile_summary.py trace DIR WORKLOAD WARMUP STEPS "COMMAND"
       python profile_summary.py counters DIR WORKLOAD "FETCH_CMD" "WRITE_CMD" "SQ_CMD"
       python profile_summary.py attn DIR WORKLOAD "SQ_CMD" ["FETCH_CMD" "WRITE_CMD"]
"""
from __future__ import annotations

import collections
import csv
import hashlib
import json
import os
import re
import statistics
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

OUT_DIR = os.environ.get("PROFILES_DIR", os.path.join(ROOT, "profiles"))
HBM_PEAK = 8.0e12
BF16_PEAK = 2.5e15
GEMM_SOURCES = ["paper_2402_15758_amd/csrc/kernels_gemm.hip", "paper_2402_15758_amd/csrc/common.h",
                "paper_2402_15758_amd/csrc/kernels.h", "paper_2402_15758_amd/build.py"]
GEMM_RE = re.compile(r"gemm_kernel<[^,]+, (\d+), (\d+)")


def short(name):
    name = name.replace("void ", "").replace("(anonymous namespace)::", "")
    return re.sub(r"\(.*", "", name)


def gemm_mb(name):
    m = GEMM_RE.search(name)
    return int(m.group(1)) if m else 0


def sources_sha():
    h = hashlib.sha256()
    for src in GEMM_SOURCES:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    return h.hexdigest()


def verify_roles(cfg, M):
    """(role, N, K, algorithmic bytes) of the verify GEMM launches in launch
    order: QKV, output projection, gate/up, down per layer, then the LM head.
    Bytes: the weight once, the M input rows, the M fp32 output rows."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, F, V, hdim = cfg.d_model, cfg.d_ffn, cfg.vocab, cfg.n_heads * cfg.head_dim
    shapes = [("QKV", 3 * hdim, d), ("O", d, hdim), ("gate/up", 2 * F, d), ("down", d, F)]
    out = []
    for _ in range(cfg.n_layers):
        out += shapes
    out.append(("LM head", V, d))
    return [(r, n, k, n * k * es + M * k * es + M * n * 4) for r, n, k in out]


def step_groups(rows, is_stamp, name_of):
    """Indices of the stamp kernels, grouped four per decode step."""
    st = [i for i, r in enumerate(rows) if is_stamp(r)]
    if len(st) % 4:
        raise SystemExit(f"{len(st)} stamp kernels: not a whole number of steps")
    return [st[i:i + 4] for i in range(0, len(st), 4)]


# --------------------------------------------------------------------------
def trace(d, wl_name, warmup, steps, cmd):
    import synth
    wl = synth.WORKLOADS[wl_name]
    cfg = wl.model
    B = len(wl.prompts())
    N = len(synth.TREES[wl.tree]) + 1  # the root and the tree's nodes
    M = B * N
    rows = list(csv.DictReader(open(os.path.join(d, "run_kernel_trace.csv"))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    t = lambda r, k: int(r[k])
    groups = step_groups(rows, lambda r: "stamp_kernel" in r["Kernel_Name"], None)
    spec = [g for g in groups if any(gemm_mb(rows[i]["Kernel_Name"]) > 1 for i in range(g[1] + 1, g[2]))]
    if len(spec) < warmup + 3 * steps:
        raise SystemExit(f"{len(spec)} speculative steps in the trace, expected at least {warmup + 3 * steps}")
    passes = {"timed (graph replay, pipelined)": spec[warmup:warmup + steps],
              "one call per step (graph replay)": spec[warmup + steps:warmup + 2 * steps],
              "eager, event-timed": spec[warmup + 2 * steps:warmup + 3 * steps]}
    roles = verify_roles(cfg, M)
    out = [f"# Decode step kernels, workload `{wl_name}` — rocprofv3 kernel-trace summary\n\n",
           f"One MI355X (gfx950). Model: {cfg.n_layers} layers, d {cfg.d_model}, {cfg.n_heads} heads x "
           f"{cfg.head_dim}, F {cfg.d_ffn}, vocab {cfg.vocab}, {cfg.dtype}; batch {B}, tree of {N} nodes "
           f"({M} verify rows). Made by\n\n```\n{cmd}\npython profile_summary.py trace <DIR> {wl_name} "
           f"{warmup} {steps} \"<command>\"\n```\n\n"
           "Steps are delimited by the library's wall-clock stamp kernels (draft start, verify start, "
           "verify end, step end); spans below run from the end of one stamp kernel to the start of the "
           "next, so they include the launch gaps inside the span.\n\n"
           "| pass | steps | step us | draft us | verify us | tail us | verify GEMM launches/step | "
           "verify GEMM avg us | verify GEMM us/step |\n|---|---:|---:|---:|---:|---:|---:|---:|---:|\n"]
    role_us = {}
    for label, sel in passes.items():
        ph = [[], [], [], []]
        vg = []
        per_role = collections.defaultdict(list)
        for g in sel:
            for p in range(3):
                ph[p].append((t(rows[g[p + 1]], "Start_Timestamp") - t(rows[g[p]], "End_Timestamp")) / 1e3)
            ph[3].append((t(rows[g[3]], "Start_Timestamp") - t(rows[g[0]], "End_Timestamp")) / 1e3)
            launches = [rows[i] for i in range(g[1] + 1, g[2]) if "gemm_kernel" in rows[i]["Kernel_Name"]]
            if len(launches) != len(roles):
                raise SystemExit(f"{len(launches)} GEMM launches in a verify span, expected {len(roles)}")
            for (role, _, _, _), r in zip(roles, launches):
                us = (t(r, "End_Timestamp") - t(r, "Start_Timestamp")) / 1e3
                vg.append(us)
                per_role[role].append(us)
        med = [statistics.median(x) for x in ph]
        out.append(f"| {label} | {len(sel)} | {med[3]:.1f} | {med[0]:.1f} | {med[1]:.1f} | {med[2]:.1f} | "
                   f"{len(vg) / len(sel):.0f} | {sum(vg) / len(vg):.2f} | {sum(vg) / len(sel):.1f} |\n")
        role_us[label] = per_role
    out.append("\n(medians over the pass's steps; GEMM columns are means)\n")

    # verify GEMMs per role, timed pass and eager pass
    out.append("\n## Verify GEMMs per role\n\nAlgorithmic bytes per launch: the weight once, the input rows "
               "(bf16) and the fp32 output rows. Fraction of the 8 TB/s HBM peak.\n\n"
               "| role | N x K | launches/step | MB/launch | timed avg us | timed frac | eager avg us | eager frac |\n"
               "|---|---|---:|---:|---:|---:|---:|---:|\n")
    seen = collections.OrderedDict()
    for role, n, k, b in roles:
        seen.setdefault(role, (n, k, b, 0))
        n0, k0, b0, c = seen[role]
        seen[role] = (n0, k0, b0, c + 1)
    tot = {"t": [0.0, 0.0], "e": [0.0, 0.0]}
    labels = list(passes)
    for role, (n, k, b, c) in seen.items():
        ut = statistics.mean(role_us[labels[0]][role])
        ue = statistics.mean(role_us[labels[2]][role])
        tot["t"][0] += b * c
        tot["t"][1] += ut * c
        tot["e"][0] += b * c
        tot["e"][1] += ue * c
        out.append(f"| {role} | {n} x {k} | {c} | {b / 1e6:.2f} | {ut:.2f} | {b / (ut * 1e-6) / HBM_PEAK:.3f} | "
                   f"{ue:.2f} | {b / (ue * 1e-6) / HBM_PEAK:.3f} |\n")
    out.append(f"| all | | {len(roles)} | {tot['t'][0] / len(roles) / 1e6:.2f} | {tot['t'][1] / len(roles):.2f} | "
               f"{tot['t'][0] / (tot['t'][1] * 1e-6) / HBM_PEAK:.3f} | {tot['e'][1] / len(roles):.2f} | "
               f"{tot['e'][0] / (tot['e'][1] * 1e-6) / HBM_PEAK:.3f} |\n")

    # whole-step kernel table of the timed pass
    sel = passes[labels[0]]
    agg = collections.defaultdict(lambda: [0.0, 0])
    busy = 0.0
    for g in sel:
        for i in range(g[0] + 1, g[3]):
            r = rows[i]
            if "stamp_kernel" in r["Kernel_Name"]:
                continue
            us = (t(r, "End_Timestamp") - t(r, "Start_Timestamp")) / 1e3
            key = f"{short(r['Kernel_Name'])} grid {r['Grid_Size_X']}x{r['Grid_Size_Y']}x{r['Grid_Size_Z']}"
            agg[key][0] += us
            agg[key][1] += 1
            busy += us
    ns = len(sel)
    out.append(f"\n## Kernels of the timed pass, per step\n\nKernel busy time {busy / ns:.1f} us/step "
               f"(sum of kernel durations between the first and the last stamp).\n\n"
               "| us/step | launches/step | avg us | kernel |\n|---:|---:|---:|---|\n")
    for key, (us, c) in sorted(agg.items(), key=lambda kv: -kv[1][0]):
        out.append(f"| {us / ns:.1f} | {c / ns:.1f} | {us / c:.2f} | `{key}` |\n")
    stats = os.path.join(d, "run_kernel_stats.csv")
    if os.path.exists(stats):
        srows = sorted(csv.DictReader(open(stats)), key=lambda r: -float(r["TotalDurationNs"]))
        out.append("\n## rocprofv3 --stats, whole run (all passes, prefills and side measurements)\n\n"
                   "| calls | total ms | avg us | min us | max us | kernel |\n|---:|---:|---:|---:|---:|---|\n")
        for r in srows[:16]:
            out.append(f"| {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['AverageNs']) / 1e3:.2f} | "
                       f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | `{short(r['Name'])}` |\n")
    path = os.path.join(OUT_DIR, f"step_kernels_{wl_name}.md")
    open(path, "w").write("".join(out))
    print("".join(out))


# --------------------------------------------------------------------------
def load_counters(path):
    by = collections.OrderedDict()
    for r in csv.DictReader(open(path)):
        key = int(r["Dispatch_Id"])
        e = by.setdefault(key, {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"]),
                                "dur": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [by[k] for k in sorted(by)]


def verify_gemms(ds):
    """Per speculative step: the verify GEMM dispatches, in launch order."""
    st = [i for i, e in enumerate(ds) if "stamp_kernel" in e["name"]]
    out = []
    for g in (st[i:i + 4] for i in range(0, len(st) - 3, 4)):
        launches = [ds[i] for i in range(g[1] + 1, g[2]) if "gemm_kernel" in ds[i]["name"]]
        if any(gemm_mb(e["name"]) > 1 for e in launches):
            out.append(launches)
    return out


def copy_scale(ds, counter):
    c = [e[counter] for e in ds if "copyBuffer" in e["name"] and e["grid"] >= (1 << 17)][-3:]
    if len(c) != 3:
        raise SystemExit(f"expected three 1 GiB copies, found {len(c)}")
    return 1048576.0 / statistics.mean(c), c


def counters(d, wl_name, cmd_f, cmd_w, cmd_sq):
    import synth
    wl = synth.WORKLOADS[wl_name]
    cfg = wl.model
    B = len(wl.prompts())
    N = len(synth.TREES[wl.tree]) + 1  # the root and the tree's nodes
    M = B * N
    roles = verify_roles(cfg, M)
    fd = load_counters(os.path.join(d, "fetch", "run_counter_collection.csv"))
    wd = load_counters(os.path.join(d, "write", "run_counter_collection.csv"))
    sd = load_counters(os.path.join(d, "sq", "run_counter_collection.csv"))
    ff, fc = copy_scale(fd, "FETCH_SIZE")
    wf, wc = copy_scale(wd, "WRITE_SIZE")
    fs, ws, ss = verify_gemms(fd), verify_gemms(wd), verify_gemms(sd)
    for s in (fs, ws, ss):
        if not s or any(len(x) != len(roles) for x in s):
            raise SystemExit("verify GEMM launches do not match the model's layer count")
    agg = collections.OrderedDict()
    for role, n, k, b in roles:
        agg.setdefault(role, {"n": n, "k": k, "alg": b, "f": [], "w": [], "mops": [], "busy": [], "gui": [],
                              "sqb": [], "dur": []})
    for step in fs:
        for (role, *_), e in zip(roles, step):
            agg[role]["f"].append(e["FETCH_SIZE"] * ff * 1024)
    for step in ws:
        for (role, *_), e in zip(roles, step):
            agg[role]["w"].append(e["WRITE_SIZE"] * wf * 1024)
    for step in ss:
        for (role, *_), e in zip(roles, step):
            a = agg[role]
            a["mops"].append(e["SQ_INSTS_VALU_MFMA_MOPS_BF16"])
            a["busy"].append(e["SQ_VALU_MFMA_BUSY_CYCLES"])
            a["gui"].append(e["GRBM_GUI_ACTIVE"])
            a["sqb"].append(e["SQ_BUSY_CYCLES"])
            a["dur"].append(e["dur"])
    out = [f"# Verify GEMM hardware counters, workload `{wl_name}` — rocprofv3 --pmc summary\n\n",
           f"One MI355X (gfx950). Verify rows M = {M} (batch {B} x {N} tree nodes); model d {cfg.d_model}, "
           f"F {cfg.d_ffn}, {cfg.n_layers} layers, {cfg.dtype}. The sample (`bench.py --counter-sample`) runs "
           "the workload's model and tree on 64-token prompts, three steps launched kernel by kernel, then "
           "three 1 GiB device copies; the verify GEMMs see the same shapes as in the full workload. Made by\n\n"
           f"```\n{cmd_f}\n{cmd_w}\n{cmd_sq}\npython profile_summary.py counters <DIR> {wl_name} \"<fetch command>\" "
           "\"<write command>\" \"<sq command>\"\n```\n\n",
           f"- byte-counter scale: the three copies read FETCH_SIZE {', '.join(f'{x:.0f}' for x in fc)} KiB and "
           f"WRITE_SIZE {', '.join(f'{x:.0f}' for x in wc)} KiB for 1048576 KiB each way: factors "
           f"{ff:.4f} (fetch) and {wf:.4f} (write)\n",
           "- MFMA FLOPs = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
           "(GRBM_GUI_ACTIVE / 8 x 256 CUs x 4 SIMDs): the CSV's GRBM_GUI_ACTIVE is the sum over the 8 XCDs "
           "(8 x 2.4 GHz x the duration)\n",
           "- durations are the counter runs' own (kernels serialised by the profiler), so rates use them\n\n",
           "| role | N x K | launches | alg MB | HBM fetch MB | HBM write MB | traffic / alg | dur us | "
           "HBM TB/s | GFLOP | TFLOP/s | frac bf16 peak | MFMA busy |\n"
           "|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|\n"]
    tot = collections.Counter()
    for role, a in agg.items():
        c = len(a["f"])
        f, w = statistics.mean(a["f"]), statistics.mean(a["w"])
        dur = statistics.mean(a["dur"]) / 1e9
        flops = statistics.mean(a["mops"]) * 512
        busy = statistics.mean(a["busy"]) * 8 / (statistics.mean(a["gui"]) * 1024)
        out.append(f"| {role} | {a['n']} x {a['k']} | {c} | {a['alg'] / 1e6:.2f} | {f / 1e6:.2f} | {w / 1e6:.2f} | "
                   f"{(f + w) / a['alg']:.3f} | {dur * 1e6:.2f} | {(f + w) / dur / 1e12:.2f} | {flops / 1e9:.2f} | "
                   f"{flops / dur / 1e12:.1f} | {flops / dur / BF16_PEAK:.3f} | {100 * busy:.1f}% |\n")
        n_role = sum(1 for r in roles if r[0] == role)
        tot["alg"] += a["alg"] * n_role
        tot["f"] += f * n_role
        tot["w"] += w * n_role
        tot["dur"] += dur * n_role
        tot["flops"] += flops * n_role
        tot["busy_w"] += busy * dur * n_role
    n = len(roles)
    out.append(f"| all (per launch) | | {n}/step | {tot['alg'] / n / 1e6:.2f} | {tot['f'] / n / 1e6:.2f} | "
               f"{tot['w'] / n / 1e6:.2f} | {(tot['f'] + tot['w']) / tot['alg']:.3f} | {tot['dur'] / n * 1e6:.2f} | "
               f"{(tot['f'] + tot['w']) / tot['dur'] / 1e12:.2f} | {tot['flops'] / n / 1e9:.2f} | "
               f"{tot['flops'] / tot['dur'] / 1e12:.1f} | {tot['flops'] / tot['dur'] / BF16_PEAK:.3f} | "
               f"{100 * tot['busy_w'] / tot['dur']:.1f}% |\n")
    out.append(f"\nGEMM sources ({', '.join(GEMM_SOURCES)}) sha256 {sources_sha()}\n")
    open(os.path.join(OUT_DIR, f"counters_{wl_name}.md"), "w").write("".join(out))
    if wl_name == "llama7b_p512":
        rec = {"kernel": "verify GEMMs", "workload": wl_name, "sources": GEMM_SOURCES,
               "sources_sha256": sources_sha(),
               "fetch_bytes_per_launch": tot["f"] / n, "write_bytes_per_launch": tot["w"] / n,
               "traffic_bytes_per_launch": (tot["f"] + tot["w"]) / n,
               "fetch_factor": ff, "write_factor": wf,
               "commands": [cmd_f, cmd_w]}
        json.dump(rec, open(os.path.join(OUT_DIR, "verify_gemm_llama7b_p512_traffic.json"), "w"), indent=1)
    print("".join(out))


# --------------------------------------------------------------------------
ATTN_COUNTERS = ["SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_LDS",
                 "SQ_INSTS_SALU", "SQ_LDS_BANK_CONFLICT", "GRBM_GUI_ACTIVE"]
ATTN_KERNELS = ["tree_attn_shared", "tree_attn_window"]


def attn(d, wl_name, cmd_sq, cmd_f=None, cmd_w=None):
    """Instruction mix of the verify pass's tree-attention kernels (the
    dispatches between each step's verify stamps) from DIR/sq, and, when
    DIR/fetch and DIR/write hold FETCH_SIZE and WRITE_SIZE passes of the same
    sample, their HBM bytes scaled by the sample's 1 GiB copies."""

    def verify_attn(ds):
        st = [i for i, e in enumerate(ds) if "stamp_kernel" in e["name"]]
        per = {k: [] for k in ATTN_KERNELS}
        for g in (st[i:i + 4] for i in range(0, len(st) - 3, 4)):
            for i in range(g[1] + 1, g[2]):
                for k in ATTN_KERNELS:
                    if k in ds[i]["name"]:
                        per[k].append(ds[i])
        if not per["tree_attn_shared"]:
            raise SystemExit("no verify-pass attention dispatches between step stamps")
        return per

    per = verify_attn(load_counters(os.path.join(d, "sq", "run_counter_collection.csv")))
    mean = lambda rows, c: statistics.mean(r[c] for r in rows)
    cmds = "\n".join(c for c in (cmd_sq, cmd_f, cmd_w) if c)
    args = " ".join(f'"<{n} command>"' for n, c in (("sq", cmd_sq), ("fetch", cmd_f), ("write", cmd_w)) if c)
    out = [f"# Tree attention counters, workload `{wl_name}` — rocprofv3 --pmc summary\n\n",
           "One MI355X (gfx950). The verify pass's two attention kernels (shared MFMA pass over 64-position "
           "chunks, per-query window pass) in the counter sample of `bench.py` (the workload's model and "
           "tree, the given prompt length, three steps launched kernel by kernel, then three 1 GiB device "
           "copies). Made by\n\n"
           f"```\n{cmds}\npython profile_summary.py attn <DIR> {wl_name} {args}\n```\n\n"
           "- counts are rocprofv3's per-dispatch totals over all waves; per-wave figures divide by SQ_WAVES\n"
           "- a shared-pass wave issues exactly 64 MFMAs per 64-key chunk (16 for S^T = K Q^T, 48 for the "
           "three-term P V), so SQ_INSTS_MFMA / 64 counts (chunk, wave) pairs and the instructions per 64 "
           "MFMAs are those of one chunk of one wave, with the pass's prologue and epilogue spread over its "
           "chunks\n"
           "- LDS bank conflicts are SQ_LDS_BANK_CONFLICT cycles per LDS instruction\n\n"
           "| kernel | dispatches | dur us | waves | VALU / wave | MFMA / wave | LDS / wave | SALU / wave | "
           "VALU per 64 MFMA | LDS per 64 MFMA | conflict cycles / LDS instr |\n"
           "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|\n"]
    for k in ATTN_KERNELS:
        rows = per[k]
        if not rows:
            continue
        waves = mean(rows, "SQ_WAVES")
        valu, mfma = mean(rows, "SQ_INSTS_VALU"), mean(rows, "SQ_INSTS_MFMA")
        lds, salu = mean(rows, "SQ_INSTS_LDS"), mean(rows, "SQ_INSTS_SALU")
        conf = mean(rows, "SQ_LDS_BANK_CONFLICT")
        dur = statistics.mean(r["dur"] for r in rows) / 1e3
        chunk = f"{64 * valu / mfma:.0f}" if mfma > 0 else "–"
        lchunk = f"{64 * lds / mfma:.1f}" if mfma > 0 else "–"
        out.append(f"| `{k}` | {len(rows)} | {dur:.2f} | {waves:.0f} | {valu / waves:.1f} | {mfma / waves:.1f} | "
                   f"{lds / waves:.1f} | {salu / waves:.1f} | {chunk} | {lchunk} | "
                   f"{conf / lds if lds else 0:.3f} |\n")
    if cmd_f and cmd_w:
        fd = load_counters(os.path.join(d, "fetch", "run_counter_collection.csv"))
        wd = load_counters(os.path.join(d, "write", "run_counter_collection.csv"))
        ff, fc = copy_scale(fd, "FETCH_SIZE")
        wf, wc = copy_scale(wd, "WRITE_SIZE")
        pf, pw = verify_attn(fd), verify_attn(wd)
        out.append(f"\nHBM bytes per dispatch (FETCH_SIZE x {ff:.4f}, WRITE_SIZE x {wf:.4f}, the factors at which "
                   "the three 1 GiB copies read 1 GiB each way; durations from the fetch pass):\n\n"
                   "| kernel | dispatches | fetch MB | write MB | dur us | HBM TB/s |\n|---|---:|---:|---:|---:|---:|\n")
        for k in ATTN_KERNELS:
            if not pf[k]:
                continue
            f = statistics.mean(r["FETCH_SIZE"] for r in pf[k]) * ff * 1024
            w = statistics.mean(r["WRITE_SIZE"] for r in pw[k]) * wf * 1024
            dur = statistics.mean(r["dur"] for r in pf[k]) / 1e9
            out.append(f"| `{k}` | {len(pf[k])} | {f / 1e6:.2f} | {w / 1e6:.2f} | {dur * 1e6:.2f} | "
                       f"{(f + w) / dur / 1e12:.2f} |\n")
    open(os.path.join(OUT_DIR, f"attn_counters_{wl_name}.md"), "w").write("".join(out))
    print("".join(out))


if __name__ == "__main__":
    if len(sys.argv) >= 7 and sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3], int(sys.argv[4]), int(sys.argv[5]), sys.argv[6])
    elif len(sys.argv) >= 7 and sys.argv[1] == "counters":
        counters(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6])
    elif len(sys.argv) in (5, 7) and sys.argv[1] == "attn":
        attn(sys.argv[2], sys.argv[3], *sys.argv[4:])
    else:
        raise SystemExit(__doc__)
