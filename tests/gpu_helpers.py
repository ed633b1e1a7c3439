"""Shared pieces of the GPU parity tests: sessions built from the synthetic
workloads, and a teacher-forced comparison of one GPU step with the oracle.

Parity rule (numeric contract): verify logits within tau * (max - min) of the
oracle's per node (tau = 1e-4 for f32 models, 2e-2 for bf16); tokens, tree
node ids and the accepted path bit-exact.  For bf16 models a differing
argmax or top-s choice is admissible only when the oracle's own margin
between the two ids is <= 2 tau * range; such ties are counted and the
oracle then follows the GPU's choice.
"""
from __future__ import annotations

import sys

import numpy as np

import oracle
import synth
from oracle import chimera_oracle as co


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def tau(cfg):
    return 2e-2 if cfg.dtype == "bf16" else 1e-4


def make_session(cfg, weights, tree, max_batch=1, max_len=512, page_order=None):
    from paper_2402_15758_amd import Session
    return Session(cfg, weights, tree, max_batch=max_batch, max_len=max_len, page_order=page_order)


class TieLog:
    def __init__(self):
        self.argmax_ties = 0
        self.list_ties = 0


def compare_lists(gpu_list, o_list, z, t, ties: TieLog, forced_first: bool):
    """Compare a GPU top-s list with the oracle's for one draft head."""
    if list(gpu_list) == list(o_list):
        return
    rng = float(z.max() - z.min())
    for r, (a, b) in enumerate(zip(gpu_list, o_list)):
        if a == b:
            continue
        assert not (forced_first and r == 0), "forced rank-0 token differs"
        assert abs(float(z[a]) - float(z[b])) <= 2 * t * rng, (
            f"draft rank {r}: gpu {a} vs oracle {b}, margin {abs(z[a] - z[b]):.3g} > {2 * t * rng:.3g}")
        ties.list_ties += 1


def gpu_step(sess):
    """One GPU step plus the debug buffers the comparison needs."""
    from paper_2402_15758_amd import binding as B
    toks, n, path = sess.step()
    art = dict(toks=toks, n=n, path=path, tree=sess.debug(B.DBG_TREE_TOKENS),
               logits=sess.debug(B.DBG_VERIFY_LOGITS).reshape(sess.batch, sess.n_nodes, -1))
    if sess.K:
        art["lists"] = sess.debug(B.DBG_DRAFT_LISTS)
    return art


def check_step(art, b: int, dec: oracle.Decoder, t: float, ties: TieLog, forced=None):
    """Check sequence b of a GPU step against the oracle driven along the
    GPU's state; the oracle then commits what the GPU committed."""
    L = int(art["n"][b])
    tree_g = art["tree"][b]
    logits_g = art["logits"][b]
    if dec.K and dec.branch:
        # branch-conditioned drafting: every drafted node's list, with the
        # oracle's paths following the GPU's tree tokens
        tt = dec.tree
        for v in range(1, tt.n):
            assert int(tree_g[v]) == int(art["lists"][b, tt.parent[v], tt.ranks[v][-1]]), v
        lists_o, dz = dec.draft_branches(tree_tokens=[int(x) for x in tree_g])
        for k in range(dec.K):
            ff = forced is not None and bool(forced.ok[dec.n + 1 + k])
            for u in dec.drafted[k]:
                compare_lists(art["lists"][b, u, : dec.s[k]], lists_o[u], dz[u], t, ties, ff)
    elif dec.K:
        # the oracle's draft chain follows the GPU's rank-0 tokens (each checked
        # against the oracle's own list below, with the tie rule)
        lists_o, dz = dec.draft(chain_tokens=[int(art["lists"][b, k, 0]) for k in range(dec.K)])
        for k in range(dec.K):
            ff = forced is not None and bool(forced.ok[dec.n + 1 + k])
            compare_lists(art["lists"][b, k, : dec.s[k]], lists_o[k], dz[k], t, ties, ff)
    assert int(tree_g[0]) == dec.pending
    logits_o, h_o, tkv = dec.verify(list(tree_g))
    rngs = logits_o.max(-1) - logits_o.min(-1)
    err = float(np.max(np.abs(logits_g - logits_o) / rngs[:, None]))
    assert err <= t, f"verify logits rel err {err:.3g} > {t}"
    amax_g = logits_g.argmax(-1)
    amax_o = logits_o.argmax(-1)
    for u in range(len(tree_g)):
        if amax_g[u] != amax_o[u]:
            z = logits_o[u]
            assert abs(z[amax_g[u]] - z[amax_o[u]]) <= 2 * t * rngs[u], f"node {u} argmax differs beyond tie"
            ties.argmax_ties += 1
    path_o, bonus_o = dec.accept(list(tree_g), list(amax_g))
    assert list(art["path"][b, :L]) == path_o, (list(art["path"][b, :L]), path_o)
    new_o = [int(tree_g[u]) for u in path_o[1:]] + [int(bonus_o)]
    assert list(art["toks"][b, :L]) == new_o
    dec.commit(path_o, bonus_o, list(tree_g), h_o, tkv)
    return new_o, err


def used_lists(lists, tree_ranks, branch: bool):
    """The slots of a DBG_DRAFT_LISTS array [B][64][8] that a step fills:
    per drafted row (level k for chain drafting, internal tree node for
    branch-conditioned drafting) its first s_k entries, concatenated."""
    t = co.Tree(tree_ranks)
    K = t.levels if t.n > 1 else 0
    s_k = [max(r[k] for r in tree_ranks if len(r) > k) + 1 for k in range(K)]
    if branch:
        rows = [(u, s_k[t.depth[u]]) for u in range(t.n) if u in t.parent]
    else:
        rows = [(k, s_k[k]) for k in range(K)]
    return np.concatenate([lists[:, r, :s] for r, s in rows], axis=1)


def chain_nodes(tree_ranks):
    """Node ids of the rank-0 chain (root, then (0,), (0, 0), ...)."""
    return [0] + [i + 1 for i, r in enumerate(tree_ranks) if all(x == 0 for x in r)]


def forced_lossless_run(cfg, weights, wl, steps: int, extra: int = 128, branch: bool = False):
    """Run the workload's forced speculative decoding for `steps` steps and
    check, per sequence, the properties that hold at any size: the stream
    equals the GPU's greedy stream token for token, and every step accepts
    exactly 1 + (consecutive seeded successes) tokens along the rank-0
    chain.  Returns the mean accepted length."""
    import torch
    prompts = wl.prompts()
    tree = synth.TREES[wl.tree]
    K = max(len(r) for r in tree)
    B = len(prompts)
    max_len = max(len(p) for p in prompts) + steps * (K + 1) + extra
    max_len = (max_len + 63) // 64 * 64
    log(f"{wl.name}: greedy reference for {B} sequence(s), max_len {max_len}")
    ar = make_session(cfg, weights, (), max_batch=B, max_len=max_len)
    n_ref = steps * (K + 1) + K + 2
    streams = [[int(t)] for t in ar.prefill(prompts)]
    while min(len(s) for s in streams) < n_ref:
        toks, n, _ = ar.step()
        for b in range(B):
            streams[b] += [int(x) for x in toks[b, : n[b]]]
    ar.close()
    del ar  # release its weight arena before the speculative session loads
    stride = max_len + 8
    ref = np.full((B, stride), -1, dtype=np.int32)
    ok = np.zeros((B, stride), dtype=np.uint8)
    ps = wl.accept_probs()
    for b in range(B):
        n0 = len(prompts[b])
        a = streams[b][: stride - n0]
        ref[b, n0:n0 + len(a)] = a
        ok[b] = synth.force_table(ps[b], wl.force_seed, b, stride)
    log(f"{wl.name}: {steps} forced speculative steps, tree {wl.tree}, "
        f"{'branch-conditioned' if branch else 'chain'} drafting")
    sp = make_session(cfg, weights, tree, max_batch=B, max_len=max_len)
    sp.set_drafting(branch)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    first = sp.prefill(prompts)
    out = [[int(t)] for t in first]
    pos = [len(p) for p in prompts]
    chain = chain_nodes(tree)
    total = 0
    for _ in range(steps):
        toks, nn, path = sp.step()
        for b in range(B):
            L = int(nn[b])
            run = 0
            while run < K and ok[b, pos[b] + 1 + run]:
                run += 1
            assert L == 1 + run, (b, pos[b], L, run)
            assert list(path[b, :L]) == chain[:L], (b, list(path[b, :L]))
            out[b] += [int(t) for t in toks[b, :L]]
            pos[b] += L
            total += L
    sp.close()
    for b in range(B):
        assert out[b] == streams[b][: len(out[b])], f"sequence {b} differs from greedy decoding"
    mean = total / (steps * B)
    log(f"{wl.name}: lossless over {B} x {steps} steps, mean accepted {mean:.2f}")
    return mean
