"""Parity at the Llama-7B shape (32 layers, d 4096, 32 x 128 heads, F 11008,
V 32000, bf16, 4 draft heads, 64-node tree) in the launch configuration the
benchmark times.

* The benchmark workload itself, checked node by node: the 512-token
  prompt, the 64-node tree and forced acceptance p = 0.7, for 8
  teacher-forced steps against a float64 oracle holding every 7B weight
  (drafted lists, tree assembly, verify logits, argmax, path, committed
  tokens and bonus).
* Branch-conditioned drafting: two teacher-forced steps after a 130-token
  prompt with every drafted node's list checked.
* Properties that hold at any size, on the benchmark workload, on the
  4096-token paged context and on the ragged batch of 8 (prompts
  U[256, 2048], T32, p_b ~ U[0.4, 0.9]): the speculative stream equals the
  GPU's greedy stream token for token, and every step accepts exactly
  1 + (consecutive seeded successes) tokens along the rank-0 chain.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import (TieLog, check_step, forced_lossless_run, gpu_step, log, make_session, tau,
                         teacher_forced_config)

pytestmark = pytest.mark.gpu

CFG = synth.LLAMA7B


@pytest.fixture(scope="module")
def w7b():
    log("llama7b: generating weights on the GPU")
    return synth.make_weights(CFG, device="cuda")


@pytest.fixture(scope="module")
def orc7b(w7b):
    log("llama7b: float64 oracle weights")
    return oracle.Oracle(CFG, synth.weights_to_numpy(w7b), compute=np.float64)


def test_llama7b_p512_teacher_forced_vs_float64_oracle(w7b, orc7b):
    wl = synth.WORKLOADS["llama7b_p512"]
    err, ties, lens = teacher_forced_config(CFG, w7b, wl.prompts(), synth.TREE_T64, wl.accept_probs(), 8,
                                            label="llama7b_p512", orc=orc7b)
    assert err <= tau(CFG)
    assert max(lens) > 1


def test_llama7b_branch_teacher_forced_vs_oracle(w7b, orc7b):
    branch = True
    log("llama7b: prompt 130, T64, branch-conditioned drafting, 2 teacher-forced steps vs float64 oracle")
    prompt = synth.make_prompt(130, CFG.vocab, 41)
    sess = make_session(CFG, w7b, synth.TREE_T64, max_len=256)
    sess.set_drafting(branch)
    first = sess.prefill([prompt])
    orc = orc7b
    dec = oracle.Decoder(orc, synth.TREE_T64, branch=branch)
    f_o = dec.prefill(list(prompt))
    log(f"llama7b: oracle prefill done (first token gpu {int(first[0])}, oracle {f_o})")
    ties = TieLog()
    if int(first[0]) != f_o:  # admissible only as a tie of the oracle's own logits
        logits, _, _ = orc.causal_forward(list(prompt))
        z = logits[-1]
        assert abs(z[int(first[0])] - z[f_o]) <= 2 * tau(CFG) * (z.max() - z.min())
        dec.pending = int(first[0])
        dec.seq[-1] = int(first[0])
        ties.argmax_ties += 1
    for i in range(2):
        _, err = check_step(gpu_step(sess), 0, dec, tau(CFG), ties)
        log(f"llama7b: step {i} verify rel err {err:.2e}")
    log(f"llama7b: ties argmax {ties.argmax_ties}, lists {ties.list_ties}")
    sess.close()


def test_llama7b_p512_lossless_and_forced_acceptance(w7b):
    import torch
    wl = synth.WORKLOADS["llama7b_p512"]
    prompt = wl.prompts()[0]
    n0, steps, max_len = len(prompt), 24, 768
    log("llama7b_p512: greedy reference, then 24 forced speculative steps")
    ar = make_session(CFG, w7b, (), max_len=max_len)
    out_a, _ = ar.generate([prompt], steps * 5 + 8)
    ar.close()
    stride = max_len + 8
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, n0:n0 + len(out_a[0])] = out_a[0]
    ok = synth.force_table(wl.accept_probs()[0], wl.force_seed, 0, stride)[None]
    sp = make_session(CFG, w7b, synth.TREE_T64, max_len=max_len)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    first = sp.prefill([prompt])
    out = [int(first[0])]
    n = n0
    chain = [0] + [sp_idx for sp_idx in range(1, 64) if synth.TREE_T64[sp_idx - 1] == (0,) * len(synth.TREE_T64[sp_idx - 1])]
    for _ in range(steps):
        toks, nn, path = sp.step()
        L = int(nn[0])
        run = 0
        while run < 4 and ok[0, n + 1 + run]:
            run += 1
        assert L == 1 + run
        assert list(path[0, :L]) == chain[:L]
        out += [int(t) for t in toks[0, :L]]
        n += L
    assert out == out_a[0][: len(out)]
    log(f"llama7b_p512: {len(out)} tokens lossless, mean accepted {len(out) / steps:.2f}")
    sp.close()


def test_llama7b_p512_branch_drafting_lossless_and_forced_acceptance(w7b):
    forced_lossless_run(CFG, w7b, synth.WORKLOADS["llama7b_p512"], steps=16, branch=True)


def test_llama7b_p4096_lossless_and_forced_acceptance(w7b):
    forced_lossless_run(CFG, w7b, synth.WORKLOADS["llama7b_p4096"], steps=16)


def test_llama7b_batch8_ragged_lossless_and_forced_acceptance(w7b):
    forced_lossless_run(CFG, w7b, synth.WORKLOADS["llama7b_b8"], steps=16)


def test_llama7b_batch8_ragged_t8_lossless_and_forced_acceptance(w7b):
    forced_lossless_run(CFG, w7b, synth.WORKLOADS["llama7b_b8_t8"], steps=16)
