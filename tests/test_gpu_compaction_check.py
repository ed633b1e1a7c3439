"""The compaction check (debug mode, race detection for the in-place KV
compaction after acceptance): after every step, slot n+d of every sequence
and layer must hold the pre-compaction K/V row of the accepted path's node
path[d], and attaching the check must not change what a step computes."""
import numpy as np
import pytest

import synth
from gpu_helpers import log, make_session

pytestmark = pytest.mark.gpu

SMALL = synth.small_config(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
                           n_draft_heads=4)


def _forcing(cfg, w, prompts, p_b, max_len, n_ref=90):
    """Forcing tables toward the GPU greedy stream of the same prompts."""
    ar = make_session(cfg, w, (), max_batch=len(prompts), max_len=max_len)
    out, _ = ar.generate(prompts, n_ref)
    ar.close()
    stride = max_len + 8
    ref = np.full((len(prompts), stride), -1, dtype=np.int32)
    for b, p in enumerate(prompts):
        ref[b, len(p):len(p) + n_ref] = out[b]
    ok = np.stack([synth.force_table(p, 5, b, stride) for b, p in enumerate(p_b)])
    return ref, ok


def _run(cfg, w, tree, prompts, ref, ok, steps, max_len, *, check, graph, branch, page_order=None):
    import torch
    sp = make_session(cfg, w, tree, max_batch=len(prompts), max_len=max_len, page_order=page_order)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    sp.set_graph(graph)
    if branch:
        sp.set_drafting(True)
    if check:
        sp.compaction_check(True)
    sp.prefill(prompts)
    rec = []
    for _ in range(steps):
        toks, n, path = sp.step()
        rec.append((toks.copy(), n.copy(), path.copy()))
    counts = sp.compaction_check_read() if check else None
    sp.close()
    return rec, counts


@pytest.mark.parametrize("graph,branch", [(True, False), (False, True)], ids=["graph_chain", "eager_branch"])
def test_compaction_check_small_bf16_batch(small_weights, graph, branch):
    """Batch of 3 ragged sequences, T32, forced p_b in {0.5, 0.8, 0.95}: the
    check compares every accepted row of every layer, finds no difference,
    and the steps are bit-identical to the same run without it."""
    w = small_weights
    log(f"compaction check: small bf16, batch 3, graph={graph}, branch drafting={branch}, 14 steps")
    lens = [70, 130, 200]
    prompts = [synth.make_prompt(n, SMALL.vocab, 700 + n) for n in lens]
    max_len = 512
    ref, ok = _forcing(SMALL, w, prompts, [0.5, 0.8, 0.95], max_len)
    base, _ = _run(SMALL, w, synth.TREE_T32, prompts, ref, ok, 14, max_len, check=False, graph=graph, branch=branch)
    got, (rows, bad) = _run(SMALL, w, synth.TREE_T32, prompts, ref, ok, 14, max_len, check=True, graph=graph,
                            branch=branch)
    accepted = sum(int(n.sum()) for _, n, _ in got)
    log(f"compaction check: {rows} rows compared, {bad} differing chunks, {accepted} tokens committed")
    assert bad == 0
    # one row per accepted path position, per sequence, layer and K/V
    assert rows == accepted * SMALL.n_layers * 2
    assert max(int(n.max()) for _, n, _ in got) > 2  # paths that really move rows
    for (t0, n0, p0), (t1, n1, p1) in zip(base, got):
        assert np.array_equal(n0, n1) and np.array_equal(t0, t1) and np.array_equal(p0, p1)


def test_compaction_check_tiny_shuffled_pages():
    """fp32 tiny model, T8, every forced draft accepted (p = 1), shuffled page
    order so that the moved rows cross page boundaries."""
    cfg = synth.TINY
    w = synth.make_weights(cfg, device="cpu")
    prompt = synth.WORKLOADS["tiny"].prompts()[0]
    log("compaction check: tiny fp32, T8, p = 1, shuffled pages, 12 steps")
    max_len = 256
    ref, ok = _forcing(cfg, w, [prompt], [1.0], max_len, n_ref=60)
    n_pages = int(np.ceil((max_len + 64) / 16))
    order = np.random.default_rng(3).permutation(n_pages).astype(np.int32)
    got, (rows, bad) = _run(cfg, w, synth.TREE_T8, [prompt], ref, ok, 12, max_len, check=True, graph=True,
                            branch=False, page_order=order)
    log(f"compaction check: {rows} rows compared, {bad} differing chunks")
    assert bad == 0
    assert all(int(n[0]) == 4 for _, n, _ in got)  # K + 1 tokens every step
    assert rows == sum(int(n.sum()) for _, n, _ in got) * cfg.n_layers * 2


@pytest.fixture(scope="module")
def small_weights():
    return synth.make_weights(SMALL, std=0.06, device="cpu")
