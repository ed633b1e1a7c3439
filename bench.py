"""Benchmark of the Chimera decode step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline]

A step is one chimera_step: draft chain, tree assembly, the target's verify
pass over the whole candidate tree, greedy acceptance and KV compaction.
The default workload is the Llama-7B-shaped bf16 model (random N(0, 0.02)
weights), batch 1, a uniform random 512-token prompt, the 64-node tree and
forced acceptance p = 0.7 (the paper's datasets and trained drafts are
replaced by synthetic prompts and a seeded acceptance bias).  W untimed
steps run first, then exactly K steps are timed (HIP graph replay, the
launch mode of the library); the line printed is

  value = accepted (committed) tokens / timed seconds,

the K steps enqueued back to back (chimera_steps: one host synchronisation
per up to 64 steps; the same steps one chimera_step call each are reported
beside it).

Also reported:
  verify_pass  the verify pass (tree pass + LM head + argmax) timed by device
               wall-clock stamps inside the replayed step graph, median over
               K steps, against its algorithmic bytes (weights + KV read +
               tree KV write) and against HBM peak and a measured device copy;
  roofline     the verify GEMM kernels' achieved HBM bandwidth, from HIP
               events recorded by each launch's own dispatch (K steps with the
               kernels launched one by one);
  generation   the workload's whole generation (G tokens after the prefill),
               timed three times, median tokens/s;
  cpu_baseline the CPU oracle's own decode steps on this host, timed;
and the plain greedy decoding rate of the same GPU path (tree of one node),
plus side measurements of the trigram lookup cache, branch-conditioned
drafting and typical decoding.
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
    ap.add_argument("--no-generation", action="store_true", help="skip the three whole-generation timings")
    ap.add_argument("--counter-sample", action="store_true",
                    help="only a short sample for hardware-counter passes: the workload's model and tree, "
                         "64-token prompts, three steps launched kernel by kernel, then three 1 GiB device "
                         "copies (the counters' scale reference); prints no benchmark line")
    ap.add_argument("--counter-prompt", type=int, default=64,
                    help="prompt tokens of the counter sample (the attention passes' context)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--no-typical", action="store_true", help="skip the typical-decoding (T = 1) measurement")
    ap.add_argument("--no-branch", action="store_true", help="skip the branch-conditioned drafting measurement")
    ap.add_argument("--torch-gemm-reference", action="store_true",
                    help="also time torch's bf16 linear (hipBLASLt) on the verify GEMM shapes, as a library reference")
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


def cpu_baseline(wl, weights_gpu, prompt, ref_row, ok_row, n_steps=8):
    """The CPU oracle on a bounded sample of the workload: after an untimed
    prefill of the same prompt and one untimed step (which also converts the
    draft weights), n_steps of its own decode steps (draft, tree verify over
    every target layer, acceptance and commit) with the same forced-acceptance
    tables as the GPU run, timed.  Reported in accepted tokens/s."""
    import oracle
    import synth
    cfg = wl.model
    threads = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp:
        threads = min(threads, int(omp))
    orc = oracle.Oracle(cfg, synth.weights_to_numpy(weights_gpu), compute=np.float32)
    dec = oracle.Decoder(orc, synth.TREES[wl.tree], forcing=oracle.Forcing(ref_row, ok_row))
    t0 = time.perf_counter()
    dec.prefill([int(x) for x in prompt])
    t_prefill = time.perf_counter() - t0
    log(f"[bench] oracle prefill {t_prefill:.1f}s")
    dec.step()
    t0 = time.perf_counter()
    accepted = 0
    for i in range(n_steps):
        accepted += len(dec.step()["new_tokens"])
        log(f"[bench] oracle step {i}: {time.perf_counter() - t0:.1f}s")
    t_steps = time.perf_counter() - t0
    return {
        "value": accepted / t_steps,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{n_steps} float32 oracle decode steps of the workload (all {cfg.n_layers} target layers, "
                   f"draft, {wl.tree} tree, context {len(prompt)}+, same forcing), {accepted} tokens accepted in "
                   f"{t_steps:.1f}s ({t_steps / n_steps:.2f} s/step); prefill {t_prefill:.1f}s and one warm-up "
                   f"step not timed"),
    }


def copy_bandwidth(torch, dev, nbytes=1 << 30, reps=5):
    """Device-to-device copy of nbytes (read + write) timed with HIP events:
    the streaming reference bandwidth of this GPU, in GB/s."""
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del src, dst
    return 2.0 * nbytes / (best * 1e-3) / 1e9


def torch_gemm_reference(torch, dev, cfg, M, reps=40):
    """Microseconds per torch linear layer (the vendor BLAS) on each verify
    GEMM shape with M rows, bf16 in and out, weights rotated over copies that
    exceed the 256 MB Infinity Cache.  A reference for the library's own
    kernels, not part of the decode step."""
    hdim = cfg.n_heads * cfg.head_dim
    roles = [("QKV", cfg.d_model, 3 * hdim), ("O", hdim, cfg.d_model), ("gate/up", cfg.d_model, 2 * cfg.d_ffn),
             ("down", cfg.d_ffn, cfg.d_model), ("LM head", cfg.d_model, cfg.vocab)]
    lin = torch.nn.functional.linear  # y = x W^T with W stored [N][K], as a linear layer holds it
    out = {}
    for name, K, N in roles:
        copies = min(8, max(2, int(700e6 // (K * N * 2)) + 1))
        ws = [torch.randn(N, K, device=dev, dtype=torch.bfloat16) for _ in range(copies)]
        x = torch.randn(M, K, device=dev, dtype=torch.bfloat16)
        for i in range(4):
            y = lin(x, ws[i % copies])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(reps):
            y = lin(x, ws[i % copies])
        e1.record()
        e1.synchronize()
        out[name] = round(e0.elapsed_time(e1) * 1e3 / reps, 2)
        del ws, x, y
    torch.cuda.empty_cache()
    return out


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


def run_steps(spec, n, out):
    """n steps, one chimera_step call each; appends each sequence's committed
    tokens to out; returns the accepted count."""
    acc = 0
    for _ in range(n):
        toks, nn, _ = spec.step()
        acc += int(nn.sum())
        for b in range(len(out)):
            out[b] += [int(x) for x in toks[b, : nn[b]]]
    return acc


def run_pipelined(spec, n, out, chunk=64):
    """n steps enqueued back to back (chimera_steps, up to `chunk` per call);
    appends each sequence's committed tokens to out; returns the accepted
    count."""
    acc, done = 0, 0
    while done < n:
        c = min(chunk, n - done)
        toks, nn, _ = spec.steps(c)
        acc += int(nn.sum())
        for i in range(c):
            for b in range(len(out)):
                out[b] += [int(x) for x in toks[i, b, : nn[i, b]]]
        done += c
    return acc


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
    B = len(prompts)
    K_levels = max(len(r) for r in synth.TREES[wl.tree])
    total_steps = a.warmup + 3 * a.steps  # warmup, timed pass, one-call-per-step pass, eager-profiled pass
    horizon = max(total_steps * (K_levels + 1), wl.gen_tokens + K_levels + 1)
    max_len = max(len(p) for p in prompts) + horizon + 128
    max_len = (max_len + 63) // 64 * 64
    torch.cuda.init()
    dev = torch.device("cuda:0")
    log(f"[bench] workload {wl.name}: generating weights on the GPU")
    t0 = time.perf_counter()
    weights = synth.make_weights(cfg, wl.target_seed, wl.draft_seed, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] weights ready in {time.perf_counter() - t0:.1f}s; loading")
    spec = Session(cfg, weights, synth.TREES[wl.tree], max_batch=B, max_len=max_len)
    if a.counter_sample:
        # the same verify-pass kernels at the workload's rows (batch x tree
        # nodes); a short context keeps the number of dispatches small
        spec.set_graph(False)
        spec.prefill([p[:a.counter_prompt] for p in prompts])
        for _ in range(3):
            spec.step()
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] counter sample: {wl.name}, {B} x {a.counter_prompt}-token prompts, 3 eager steps, "
            "3 x 1 GiB copies")
        spec.close()
        return
    ar = Session(cfg, None, (), max_batch=B, max_len=max_len, share_model=spec)
    torch.cuda.synchronize()

    # greedy reference stream (plain decoding through the same kernels)
    n_ref = horizon + K_levels + 2
    log(f"[bench] greedy decoding {n_ref} tokens for the forcing reference")
    streams = [[int(t)] for t in ar.prefill(prompts)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_pipelined(ar, n_ref - 1, streams)  # one token per greedy step
    torch.cuda.synchronize()
    ar_rate = B * (n_ref - 1) / (time.perf_counter() - t0)
    stride = max_len + 8
    ref, ok = forcing_tables(wl, prompts, streams, stride)
    spec.set_forcing(torch.from_numpy(ref).to(dev), torch.from_numpy(ok).to(dev))

    log(f"[bench] spec: prefill, {a.warmup} warmup steps, {a.steps} timed steps")
    out = [[int(t)] for t in spec.prefill(prompts)]
    run_steps(spec, a.warmup, out)
    # timed pass: exactly K steps, graph replay, enqueued back to back
    # (chimera_steps).  Every step carries one-lane wall-clock stamp kernels
    # at its phase boundaries (draft | verify | tail); the library reports the
    # per-step medians of exactly these steps.
    spec.profile_read()  # opens the stamp window
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    accepted = run_pipelined(spec, a.steps, out)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    prof_g = spec.profile_read()
    # the same K steps with one host round trip per step (chimera_step)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    accepted_1 = run_steps(spec, a.steps, out)
    torch.cuda.synchronize()
    dt_1 = time.perf_counter() - t0
    # eager-profiled pass: kernels launched one by one, each verify GEMM
    # launch recording HIP events at its own dispatch start and end
    spec.set_graph(False)
    spec.profile(True)
    spec.profile_read()
    run_steps(spec, a.steps, out)
    torch.cuda.synchronize()
    prof = spec.profile_read()
    spec.profile(False)
    spec.set_graph(True)
    lossless = all(out[b] == streams[b][: len(out[b])] for b in range(B))

    # the whole generation: G tokens per sequence after the prefill, three times
    gen = []
    for rep in range(0 if a.no_generation else 3):
        o = [[int(t)] for t in spec.prefill(prompts)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        steps = 0
        while min(len(x) for x in o) < wl.gen_tokens:
            # every step commits 1 .. K+1 tokens: enqueue as many steps as the
            # remainder surely needs
            need = wl.gen_tokens - min(len(x) for x in o)
            c = max(1, -(-need // (K_levels + 1)))
            run_pipelined(spec, c, o)
            steps += c
        torch.cuda.synchronize()
        t_gen = time.perf_counter() - t0
        committed = sum(len(x) - 1 for x in o)
        gen.append((committed / t_gen, steps, committed, t_gen))
        lossless = lossless and all(o[b] == streams[b][: len(o[b])] for b in range(B))
    gen_sorted = sorted(gen)
    generation = None if not gen else {"tokens": wl.gen_tokens, "reps": 3,
                  "tokens_per_s_median": round(gen_sorted[1][0], 2),
                  "tokens_per_s": [round(g[0], 2) for g in gen],
                  "steps": [g[1] for g in gen], "committed": [g[2] for g in gen],
                  "timing": "pipelined steps (chimera_steps), first launch to the last synchronisation, prefill excluded"}
    if generation:
        log(f"[bench] generation of {wl.gen_tokens} tokens x3: {generation['tokens_per_s']} tok/s")

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
        spec.profile_read()  # opens the stamp window
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
        pb = spec.profile_read()
        spec.set_drafting(False)
        same = all(out3[b] == out[b][: len(out3[b])] for b in range(len(prompts)))
        br = {"tokens_per_s": round(acc4 / dt4, 2), "ms_per_step": round(dt4 / a.steps * 1e3, 4),
              "draft_ms": round(pb.ms_draft_median, 4), "chain_draft_ms": round(prof_g.ms_draft_median, 4),
              "queries_per_level": [len(prompts) * r for r in drafted_per_level(synth.TREES[wl.tree])],
              "same_stream": same}
        log(f"[bench] branch-conditioned drafting: {br}")
    value = accepted / dt
    verify_bytes_step = prof_g.verify_bytes / max(prof_g.steps, 1)
    verify_ms = prof_g.ms_verify_median
    verify_gbs = verify_bytes_step / (verify_ms * 1e-3) / 1e9
    gemm_gbs = prof.gemm_verify_bytes / (prof.ms_gemm_verify * 1e-3) / 1e9
    per_launch_bytes = prof.gemm_verify_bytes / max(prof.gemm_verify_launches, 1)
    per_launch_us = prof.ms_gemm_verify * 1e3 / max(prof.gemm_verify_launches, 1)
    copy_gbs = copy_bandwidth(torch, dev)
    log(f"[bench] {value:.1f} tok/s, {dt / a.steps * 1e3:.3f} ms/step, accept {accepted / a.steps / B:.3f}, "
        f"verify {verify_ms:.3f} ms in the graph ({verify_gbs:.0f} GB/s), draft {prof_g.ms_draft_median:.3f} ms, "
        f"gemm {gemm_gbs:.0f} GB/s, copy {copy_gbs:.0f} GB/s, lossless={lossless}")

    if a.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy calibration: 3 x 1 GiB device copies")
        del src, dst
    torch_ref = None
    if a.torch_gemm_reference:
        rows = B * (len(synth.TREES[wl.tree]) + 1)  # the verify pass's rows: root and tree nodes per sequence
        torch_ref = {"rows": rows, "us_per_launch": torch_gemm_reference(torch, dev, cfg, rows)}
        log(f"[bench] torch matmul reference: {torch_ref}")
    cpu = None
    if not a.no_cpu_baseline and B == 1:
        log("[bench] CPU oracle baseline (8 timed oracle steps)")
        try:
            cpu = cpu_baseline(wl, weights, prompts[0], ref[0], ok[0])
        except MemoryError:
            cpu = None
        log(f"[bench] CPU oracle: {cpu}")
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
            "batch": B,
            "prompt_len": [len(p) for p in prompts] if B > 1 else len(prompts[0]),
            "tree": wl.tree,
            "accept_p": wl.accept_p[0] if wl.accept_p and B == 1 else wl.accept_p,
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
            "launches_per_step": round(prof.gemm_verify_launches / max(prof.steps, 1), 2),
        },
        "verify_pass": {
            "ms": round(verify_ms, 4),
            "ms_mean": round(prof_g.ms_verify / max(prof_g.steps, 1), 4),
            "bytes": round(verify_bytes_step),
            "achieved_gbs": round(verify_gbs, 1),
            "frac_hbm_peak": round(verify_gbs / HBM_PEAK_GBS, 4),
            "frac_copy_bw": round(verify_gbs / copy_gbs, 4),
            "timing": "device wall-clock stamps around the verify pass inside the replayed step graph, median over the timed steps",
        },
        "step_ms_stamped_median": round(prof_g.ms_step_median, 4),
        "one_call_per_step": {"tokens_per_s": round(accepted_1 / dt_1, 2),
                              "ms_per_step": round(dt_1 / a.steps * 1e3, 4)},
        "copy_bw_gbs": round(copy_gbs, 1),
        "draft_ms": round(prof_g.ms_draft_median, 4),
        "tail_ms": round(prof_g.ms_tail / max(prof_g.steps, 1), 4),
        "accept_len_mean": round(accepted / a.steps / B, 4),
        "generation": generation,
        "lossless_vs_greedy": lossless,
        "trigram_cache": tri,
        "typical_decoding": typ,
        "branch_drafting": br,
        "greedy_tokens_per_s": round(ar_rate, 2),
        "speedup_vs_greedy": round(value / ar_rate, 3),
        "cpu_baseline": cpu,
    }
    if torch_ref:
        line["torch_gemm_reference"] = torch_ref
    print(json.dumps(line), flush=True)
    spec.close()
    ar.close()


if __name__ == "__main__":
    main()
