"""Teacher-forced oracle parity at the shapes the workloads run, node by
node, through the C ABI in the launch configuration the benchmark times
(HIP graph replay).

Each model keeps its full width (d_model, heads of 128, FFN, 32000-token
vocabulary, 4 draft heads) and the workload's real prompts, tree, page size
and forced acceptance; the target is cut to two layers so that the CPU
oracle, computing in float64 between the bf16 storage points, finishes in
about a minute.  The full-depth 7B benchmark workload itself is checked
against a float64 oracle in test_gpu_llama7b.py.

* 4096-token prompt (page size 16): the shared attention pass reaches the
  far groups of four chunks past position 1024 with bf16 head_dim 128.
* 13B width, 1024-token prompt, forced p = 0.5 and 0.8; the p = 0.8 run has
  the trigram lookup cache (Sec. 4.1.1) attached, which must be exact.
* Batch 8 with ragged prompts U[256, 2048], the 32-node tree and per-sequence
  p_b ~ U[0.4, 0.9]: ragged accepted lengths and ragged compaction.
* 33B width (d 6656, 52 heads, F 17920), 512-token prompt.

Every step checks, per sequence: the drafted lists, the tree tokens as the
assembly of those lists (Sec. 4.4), the verify logits within 2e-2 of each
node's logit range, each node's argmax, the accepted path, the committed
tokens and the bonus (argmax and list choices under the tie rule).
"""
import dataclasses

import numpy as np
import pytest

import synth
from gpu_helpers import log, teacher_forced_config

pytestmark = pytest.mark.gpu


def reduced(cfg, n_layers=2):
    return dataclasses.replace(cfg, n_layers=n_layers)


def run(wl_name, steps, accept_p=None, **kw):
    wl = synth.WORKLOADS[wl_name]
    cfg = reduced(wl.model)
    log(f"{wl_name} (2-layer, full width): generating weights on the GPU")
    w = synth.make_weights(cfg, device="cuda")
    prompts = wl.prompts()
    ps = accept_p if accept_p is not None else wl.accept_probs()
    err, ties, lens = teacher_forced_config(cfg, w, prompts, synth.TREES[wl.tree], ps, steps,
                                            compute=np.float64, page_size=wl.page_size, label=wl_name, **kw)
    assert err <= 2e-2
    return err, ties, lens


def test_llama7b_p4096_teacher_forced():
    run("llama7b_p4096", steps=6)


@pytest.mark.parametrize("name,tri", [("llama13b_p1024_a05", 0), ("llama13b_p1024_a08", 65536)],
                         ids=["p0.5", "p0.8_trigram_cache"])
def test_llama13b_p1024_teacher_forced(name, tri):
    _, _, lens = run(name, steps=8, trigram_entries=tri)
    assert max(lens) > 1  # forcing made some steps accept draft tokens


def test_llama7b_batch8_ragged_teacher_forced():
    _, _, lens = run("llama7b_b8", steps=4)
    assert len(set(lens)) > 1  # ragged accepted lengths across the batch


def test_vicuna33b_width_teacher_forced():
    run("vicuna33b_p512", steps=6)
