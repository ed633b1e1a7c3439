"""Verify-logit error of the full-depth models against the oracle (a report,
not a test: pytest does not collect it).

    python tests/report_full_depth_error.py [--models llama7b,llama13b,vicuna33b]

For each model at its full depth, one teacher-forced decode step on a
70-token prompt with the 64-node tree: the GPU's verify logits are compared
node by node with the oracle's, relative to each node's logit range (the
bf16 tolerance of the numeric contract is 2e-2 of that range).  The 7B and
13B oracles run in float64; the 33B one in float32, because float64 weights
of 33B parameters would not fit the host memory.  Prints one markdown table.
"""
from __future__ import annotations

import argparse
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402
from gpu_helpers import TieLog, check_step, gpu_step, make_session  # noqa: E402

MODELS = {"llama7b": (synth.LLAMA7B, np.float64), "llama13b": (synth.LLAMA13B, np.float64),
          "vicuna33b": (synth.VICUNA33B, np.float32)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--models", default="llama7b,llama13b,vicuna33b")
    a = ap.parse_args()
    import torch
    rows = []
    for name in a.models.split(","):
        cfg, ct = MODELS[name]
        t0 = time.perf_counter()
        print(f"[report] {name}: {cfg.n_layers} layers, weights on the GPU", file=sys.stderr, flush=True)
        w = synth.make_weights(cfg, device="cuda")
        prompt = synth.make_prompt(70, cfg.vocab, 43)
        sess = make_session(cfg, w, synth.TREE_T64, max_len=192)
        first = sess.prefill([prompt])
        print(f"[report] {name}: {np.dtype(ct).name} oracle prefill", file=sys.stderr, flush=True)
        orc = oracle.Oracle(cfg, synth.weights_to_numpy(w), compute=ct, cache_weights=False)
        dec = oracle.Decoder(orc, synth.TREE_T64)
        f_o = dec.prefill(list(prompt))
        if int(first[0]) != f_o:  # a first-token near-tie: the oracle follows the GPU
            dec.pending = int(first[0])
            dec.seq[-1] = int(first[0])
        ties = TieLog()
        print(f"[report] {name}: one teacher-forced step", file=sys.stderr, flush=True)
        _, err = check_step(gpu_step(sess), 0, dec, 1.0, ties)
        rows.append((name, cfg.n_layers, np.dtype(ct).name, err, ties.argmax_ties, ties.list_ties,
                     time.perf_counter() - t0))
        print(f"[report] {name}: max verify rel err {err:.3e}", file=sys.stderr, flush=True)
        sess.close()
        del sess, w, orc, dec
        torch.cuda.empty_cache()
    print("| model | layers | oracle | max verify error / logit range | argmax differences | draft-list differences | s |")
    print("|---|---:|---|---:|---:|---:|---:|")
    for name, L, ct, err, ta, tl, s in rows:
        print(f"| {name} | {L} | {ct} | {err:.3e} | {ta} | {tl} | {s:.0f} |")


if __name__ == "__main__":
    main()
