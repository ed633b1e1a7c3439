"""Benchmark of the Chimera decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline]

A step is one chimera_step: draft chain, tree assembly, the target's verify
pass over the whole candidate tree, greedy acceptance and KV compaction.
The default workload is the Llama-7B-shaped bf16 model (random N(0, 0.02)
weights), batch 1, a uniform random 512-token prompt, the 64-node tree and
forced acceptance p = 0.7 (the paper's datasets and trained drafts are
replaced by synthetic prompts and a seeded acceptance bias).  W untimed
steps run first, then exactly K steps are timed; the line printed is

  value = accepted (committed) tokens / timed seconds.

Also reported: the verify GEMM kernel's achieved HBM bandwidth from HIP
events around each of its launches in the timed steps (roofline), the whole
verify pass's fraction of HBM peak, the plain greedy decoding rate of the
same GPU path (tree of one node), the CPU oracle on a bounded sample, and
side measurements of the trigram lookup cache, branch-conditioned drafting
and typical decoding.
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

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama7b_p512")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--no-typical", action="store_true", help="skip the typical-decoding (T = 1) measurement")
    ap.add_argument("--no-branch", action="store_true", help="skip the branch-conditioned drafting measurement")
    ap.add_argument("--trigram-cache", type=int, default=65536,
                    help="entries of the trigram lookup cache measured after the headline passes (0: skip)")
    return ap.parse_args()


def forcing_tables(wl, prompts, ar_streams, stride):
    """Reference greedy stream and seeded success bits per sequence."""
    import synth
    B = len(prompts)
    ref = np.full((B, stride), -1, dtype=np.int32)
    ok = np.zeros((B, stride), dtype=np.uint8)
    ps = wl.accept_probs()
    for b in range(B):
        n0 = len(prompts[b])
        a = ar_streams[b][: stride - n0]
        ref[b, n0:n0 + len(a)] = a
        ok[b] = synth.force_table(ps[b], wl.force_seed, b, stride)
    return ref, ok


def drafted_per_level(tree):
    """Tree nodes with children at each depth: the draft queries per sequence
    of each level under branch-conditioned drafting."""
    internal = {r[:-1] for r in tree}
    K = max(len(r) for r in tree)
    return [sum(1 for r in internal if len(r) == k) for k in range(K)]


def cpu_baseline(wl, weights_gpu, prompt, accept_len):
    """The oracle on a bounded sample of the workload: one decode step of
    the full draft and of the first two target layers plus the LM head,
    after a prefill of the same prompt; the target part is scaled to all
    layers.  Reported in accepted tokens/s with the realised mean accepted
    length of the GPU run."""
    import dataclasses

    import oracle
    import synth
    cfg = wl.model
    n_sample = 2
    sub = dataclasses.replace(cfg, n_layers=n_sample)
    keep = [n for n, _, _ in synth.tensor_specs(sub)]
    w = synth.weights_to_numpy({k: weights_gpu[k] for k in keep})
    threads = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp:
        threads = min(threads, int(omp))
    orc = oracle.Oracle(sub, w, compute=np.float32)
    dec = oracle.Decoder(orc, synth.TREES[wl.tree])
    t0 = time.perf_counter()
    dec.prefill(list(prompt))
    t_prefill = time.perf_counter() - t0
    t0 = time.perf_counter()
    lists, _ = dec.draft()
    t_draft = time.perf_counter() - t0
    toks = dec.assemble(lists)
    t0 = time.perf_counter()
    logits, h, tkv = dec.verify(toks)
    t_verify = time.perf_counter() - t0
    t0 = time.perf_counter()
    _ = h @ orc.w("lm_head")
    t_head = time.perf_counter() - t0
    t_layers = max(t_verify - t_head, 0.0)
    t_step = t_draft + t_layers * (cfg.n_layers / n_sample) + t_head
    return {
        "value": accept_len / t_step,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"one float32 oracle step (draft + {n_sample} of {cfg.n_layers} target layers + LM head, "
                   f"64-node tree, context {len(prompt)}), target layers scaled x{cfg.n_layers // n_sample}; "
                   f"prefill {t_prefill:.1f}s excluded; step {t_step:.2f}s"),
    }


def counter_traffic():
    """HBM bytes per verify-GEMM launch from the committed rocprofv3 counter
    summary, if the GEMM's sources (the kernel file, the headers it
    includes and the build script with its compiler flags) still have the
    hash they were measured with."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "verify_gemm_llama7b_p512_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if "sources" not in rec:
        return None
    h = hashlib.sha256()
    for src in rec["sources"]:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if h.hexdigest() != rec["sources_sha256"]:
        return None
    return rec["traffic_bytes_per_launch"]


def main():
    a = parse()
    if a.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(the decode step of one sequence batch lives on one MI355X)", file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    from paper_2402_15758_amd import Session

    wl = synth.WORKLOADS[a.workload]
    cfg = wl.model
    prompts = wl.prompts()
    K_levels = max(len(r) for r in synth.TREES[wl.tree])
    total_steps = a.warmup + 2 * a.steps  # warmup, timed pass, profiled pass
    max_len = max(len(p) for p in prompts) + total_steps * (K_levels + 1) + 128
    max_len = (max_len + 63) // 64 * 64
    torch.cuda.init()
    dev = torch.device("cuda:0")
    log(f"[bench] workload {wl.name}: generating weights on the GPU")
    t0 = time.perf_counter()
    weights = synth.make_weights(cfg, wl.target_seed, wl.draft_seed, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] weights ready in {time.perf_counter() - t0:.1f}s; loading")
    spec = Session(cfg, weights, synth.TREES[wl.tree], max_batch=len(prompts), max_len=max_len)
    ar = Session(cfg, None, (), max_batch=len(prompts), max_len=max_len, share_model=spec)
    torch.cuda.synchronize()

    # greedy reference stream (plain decoding through the same kernels)
    n_ref = total_steps * (K_levels + 1) + K_levels + 2
    log(f"[bench] greedy decoding {n_ref} tokens for the forcing reference")
    streams = [[int(t)] for t in ar.prefill(prompts)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while min(len(s) for s in streams) < n_ref:
        toks, n, _ = ar.step()
        for b in range(len(prompts)):
            streams[b] += [int(x) for x in toks[b, : n[b]]]
    torch.cuda.synchronize()
    ar_rate = len(prompts) * (n_ref - 1) / (time.perf_counter() - t0)
    stride = max_len + 8
    ref, ok = forcing_tables(wl, prompts, streams, stride)
    spec.set_forcing(torch.from_numpy(ref).to(dev), torch.from_numpy(ok).to(dev))

    log(f"[bench] spec: prefill, {a.warmup} warmup steps, {a.steps} timed steps")
    first = spec.prefill(prompts)
    out = [[int(t)] for t in first]
    for _ in range(a.warmup):
        toks, n, _ = spec.step()
        for b in range(len(prompts)):
            out[b] += [int(x) for x in toks[b, : n[b]]]
    # timed pass: exactly K steps, no per-kernel events
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    accepted = 0
    for _ in range(a.steps):
        toks, n, _ = spec.step()
        accepted += int(n.sum())
        for b in range(len(prompts)):
            out[b] += [int(x) for x in toks[b, : n[b]]]
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    # profiled pass: K more steps with HIP events on the stream the kernels
    # run on: around each phase, and recorded by each verify GEMM kernel's
    # own dispatch at its start and end (kernels launched one by one here)
    spec.set_graph(False)
    spec.profile(True)
    accepted_p = 0
    for _ in range(a.steps):
        toks, n, _ = spec.step()
        accepted_p += int(n.sum())
        for b in range(len(prompts)):
            out[b] += [int(x) for x in toks[b, : n[b]]]
    torch.cuda.synchronize()
    prof = spec.profile_read()
    spec.profile(False)
    spec.set_graph(True)
    lossless = all(out[b] == streams[b][: len(out[b])] for b in range(len(prompts)))

    tri = None
    if a.trigram_cache:
        # trigram lookup cache: a cold pass (cache filled only by the prompt and
        # the run itself) and a warm pass (the same run again, so every draft
        # trigram is cached); both must reproduce the stream above exactly
        spec.trigram_cache(a.trigram_cache)
        tri = {"entries": a.trigram_cache}
        for label in ("cold", "warm"):
            first = spec.prefill(prompts)
            out2 = [[int(t)] for t in first]
            for _ in range(a.warmup):
                toks, n, _ = spec.step()
                for b in range(len(prompts)):
                    out2[b] += [int(x) for x in toks[b, : n[b]]]
            l0, h0 = spec.trigram_stats()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            acc2 = 0
            for _ in range(a.steps):
                toks, n, _ = spec.step()
                acc2 += int(n.sum())
                for b in range(len(prompts)):
                    out2[b] += [int(x) for x in toks[b, : n[b]]]
            torch.cuda.synchronize()
            dt2 = time.perf_counter() - t0
            l1, h1 = spec.trigram_stats()
            same = all(out2[b] == out[b][: len(out2[b])] for b in range(len(prompts)))
            tri[label] = {"tokens_per_s": round(acc2 / dt2, 2), "ms_per_step": round(dt2 / a.steps * 1e3, 4),
                          "lookups": l1 - l0, "hits": h1 - h0,
                          "hit_rate": round((h1 - h0) / max(l1 - l0, 1), 4), "same_stream": same}
            log(f"[bench] trigram cache {label}: {tri[label]}")
        spec.trigram_cache(0)
    br = None
    if not a.no_branch and K_levels > 0:
        # branch-conditioned drafting: every internal tree node drafts along its
        # own path.  Forcing keeps the accepted path on the rank-0 chain, so the
        # stream must equal the one above; the cost is the draft at more rows.
        spec.set_drafting(True)
        first = spec.prefill(prompts)
        out3 = [[int(t)] for t in first]
        for _ in range(a.warmup):
            toks, n, _ = spec.step()
            for b in range(len(prompts)):
                out3[b] += [int(x) for x in toks[b, : n[b]]]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        acc4 = 0
        for _ in range(a.steps):
            toks, n, _ = spec.step()
            acc4 += int(n.sum())
            for b in range(len(prompts)):
                out3[b] += [int(x) for x in toks[b, : n[b]]]
        torch.cuda.synchronize()
        dt4 = time.perf_counter() - t0
        spec.set_graph(False)
        spec.profile(True)
        for _ in range(a.steps):
            toks, n, _ = spec.step()
            for b in range(len(prompts)):
                out3[b] += [int(x) for x in toks[b, : n[b]]]
        torch.cuda.synchronize()
        pb = spec.profile_read()
        spec.profile(False)
        spec.set_graph(True)
        spec.set_drafting(False)
        same = all(out3[b] == out[b][: len(out3[b])] for b in range(len(prompts)))
        br = {"tokens_per_s": round(acc4 / dt4, 2), "ms_per_step": round(dt4 / a.steps * 1e3, 4),
              "draft_ms": round(pb.ms_draft / pb.steps, 4), "chain_draft_ms": round(prof.ms_draft / prof.steps, 4),
              "queries_per_level": [len(prompts) * r for r in drafted_per_level(synth.TREES[wl.tree])],
              "same_stream": same}
        log(f"[bench] branch-conditioned drafting: {br}")
    value = accepted / dt
    gemm_gbs = prof.gemm_verify_bytes / (prof.ms_gemm_verify * 1e-3) / 1e9
    verify_gbs = prof.verify_bytes / (prof.ms_verify * 1e-3) / 1e9
    per_launch_bytes = prof.gemm_verify_bytes / max(prof.gemm_verify_launches, 1)
    per_launch_us = prof.ms_gemm_verify * 1e3 / max(prof.gemm_verify_launches, 1)
    log(f"[bench] {value:.1f} tok/s, {dt / a.steps * 1e3:.3f} ms/step, accept {accepted / a.steps / len(prompts):.3f}, "
        f"verify {prof.ms_verify / prof.steps:.3f} ms ({verify_gbs:.0f} GB/s), draft {prof.ms_draft / prof.steps:.3f} ms, "
        f"gemm {gemm_gbs:.0f} GB/s, lossless={lossless}")

    if a.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy calibration: 3 x 1 GiB device copies")
        del src, dst
    cpu = None
    if not a.no_cpu_baseline and len(prompts) == 1:
        log("[bench] CPU oracle baseline (bounded sample)")
        try:
            cpu = cpu_baseline(wl, weights, prompts[0], accepted / a.steps)
        except MemoryError:
            cpu = None
    typ = None
    if not a.no_typical:
        # typical decoding at T = 1 (sampling, not lossless): accepted length and
        # rate of the speculative session, against plain sampling (no draft)
        spec.set_decoding(True, 1.0, 0.09, 0.3, seed=17)
        ar.set_decoding(True, 1.0, 0.09, 0.3, seed=17)
        spec.prefill(prompts)
        for _ in range(a.warmup):
            spec.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        acc3 = 0
        for _ in range(a.steps):
            _, n, _ = spec.step()
            acc3 += int(n.sum())
        torch.cuda.synchronize()
        dt3 = time.perf_counter() - t0
        ar.prefill(prompts)
        for _ in range(a.warmup):
            ar.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(a.steps):
            ar.step()
        torch.cuda.synchronize()
        dt4 = time.perf_counter() - t0
        spec.set_decoding(False)
        ar.set_decoding(False)
        typ = {"temperature": 1.0, "eps": 0.09, "delta": 0.3,
               "tokens_per_s": round(acc3 / dt3, 2), "accept_len_mean": round(acc3 / a.steps / len(prompts), 3),
               "sampling_tokens_per_s": round(a.steps * len(prompts) / dt4, 2),
               "speedup_vs_sampling": round((acc3 / dt3) / (a.steps * len(prompts) / dt4), 3)}
        log(f"[bench] typical decoding: {typ}")
    line = {
        "metric": "accepted tokens/sec at batch 1 (Llama-7B-shape bf16); verify-pass % of HBM peak",
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(dt / a.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "target": f"{cfg.n_layers}L d{cfg.d_model} {cfg.n_heads}x{cfg.head_dim} F{cfg.d_ffn} V{cfg.vocab}",
            "draft": f"trigram MLP + 1 encoder layer + {cfg.n_draft_heads} heads",
            "batch": len(prompts),
            "prompt_len": [len(p) for p in prompts] if len(prompts) > 1 else len(prompts[0]),
            "tree": wl.tree,
            "accept_p": wl.accept_p[0] if wl.accept_p and len(prompts) == 1 else wl.accept_p,
            "page_size": 16,
        },
        "roofline": {
            "kernel": "verify GEMMs (QKV, O, gate/up, down, LM head)",
            "bound": "hbm",
            "achieved": round(gemm_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gemm_gbs / HBM_PEAK_GBS, 4),
            "traffic": (round(counter_traffic()) if counter_traffic() and wl.name == "llama7b_p512" else None),
            "bytes_per_launch": round(per_launch_bytes),
            "us_per_launch": round(per_launch_us, 2),
        },
        "verify_pass": {
            "ms": round(prof.ms_verify / prof.steps, 4),
            "bytes": round(prof.verify_bytes / prof.steps),
            "achieved_gbs": round(verify_gbs, 1),
            "frac_hbm_peak": round(verify_gbs / HBM_PEAK_GBS, 4),
        },
        "draft_ms": round(prof.ms_draft / prof.steps, 4),
        "tail_ms": round(prof.ms_tail / prof.steps, 4),
        "accept_len_mean": round(accepted / a.steps / len(prompts), 4),
        "lossless_vs_greedy": lossless,
        "trigram_cache": tri,
        "typical_decoding": typ,
        "branch_drafting": br,
        "greedy_tokens_per_s": round(ar_rate, 2),
        "speedup_vs_greedy": round(value / ar_rate, 3),
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    spec.close()
    ar.close()


if __name__ == "__main__":
    main()
