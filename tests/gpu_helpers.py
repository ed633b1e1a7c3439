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


# Set by the autouse fixture in conftest.py to the test's capsys: progress
# lines then reach the terminal even while pytest captures output, so a long
# GPU test shows it is alive between its steps.
_PROGRESS_SINK = None


def log(*a):
    sink = _PROGRESS_SINK
    if sink is not None:
        with sink.disabled():
            print(*a, flush=True)
    else:
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
        # every tree token is the oracle's assembly (Sec. 4.4) of the GPU's own
        # per-head lists: node (r_0..r_k) holds rank r_k of head k
        lists_g = [[int(x) for x in art["lists"][b, k, : dec.s[k]]] for k in range(dec.K)]
        want = dec.assemble(lists_g)
        assert [int(x) for x in tree_g] == want, "tree tokens are not the assembly of the drafted lists"
        # the oracle's draft chain follows the GPU's rank-0 tokens (each checked
        # against the oracle's own list below, with the tie rule)
        lists_o, dz = dec.draft(chain_tokens=[lst[0] for lst in lists_g])
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


class GreedyRef:
    """The oracle's own greedy stream from a decoder's state after prefill,
    extended on demand one token per step through a root-only tree (the
    decoder itself is left untouched).  tokens[i] is the token at absolute
    position n0 + i, tokens[0] the pending token."""

    def __init__(self, dec: oracle.Decoder):
        self.ar = oracle.Decoder(dec.o, ())
        for name in ("seq", "kv", "n", "pending", "h_last", "llm_k", "llm_v", "tri_k", "tri_v"):
            setattr(self.ar, name, getattr(dec, name))
        self.n0 = dec.n
        self.tokens = [int(dec.pending)]

    def upto(self, pos: int):
        """Extend the stream to cover absolute position pos."""
        while self.n0 + len(self.tokens) <= pos:
            self.tokens += [int(x) for x in self.ar.step()["new_tokens"]]
        return self.tokens


def oracle_greedy_ref(dec: oracle.Decoder, n_tokens: int):
    """The pending token and the n_tokens - 1 greedy tokens after it."""
    r = GreedyRef(dec)
    return r.upto(dec.n + n_tokens - 1)[:n_tokens]


def teacher_forced_config(cfg, w_gpu, prompts, tree, accept_p, steps: int, *, compute=np.float32,
                          page_size: int = 16, trigram_entries: int = 0, force_seed: int = 3,
                          label: str = "", cache_weights: bool = True, orc=None):
    """Teacher-forced node-by-node parity of `steps` GPU steps at a workload's
    shape (batch = len(prompts)).

    Forcing (the synthetic stand-in for a trained draft) biases both sides
    toward the oracle's own greedy stream with per-sequence success
    probabilities accept_p[b]; the same tables go to the GPU and to the
    oracle.  Every step checks, per sequence: the drafted lists (tie rule),
    the tree tokens as the assembly of those lists, the verify logits within
    tau of the oracle's, the argmax per node (tie rule), the accepted path,
    the committed tokens and the bonus.  Returns (max logit error, ties,
    accepted lengths).  ``orc`` reuses an oracle already holding these weights."""
    import torch
    t = tau(cfg)
    B = len(prompts)
    K = max(len(r) for r in tree)
    max_len = max(len(p) for p in prompts) + steps * (K + 1) + K + 2 + 64
    max_len = (max_len + 63) // 64 * 64
    stride = max_len + 8
    if orc is None:
        orc = oracle.Oracle(cfg, synth.weights_to_numpy(w_gpu), compute=compute, cache_weights=cache_weights)
    log(f"{label}: oracle ({np.dtype(orc.ct).name}) prefill of {B} prompt(s) {[len(p) for p in prompts]}")
    ref = np.full((B, stride), -1, dtype=np.int32)
    ok = np.zeros((B, stride), dtype=np.uint8)
    decs, grefs = [], []
    for b, p in enumerate(prompts):
        d = oracle.Decoder(orc, tree)
        d.prefill([int(x) for x in p])
        ok[b] = synth.force_table(float(accept_p[b]), force_seed, b, stride)
        d.forcing = oracle.Forcing(ref[b], ok[b])  # views: later reference tokens show up here
        decs.append(d)
        grefs.append(GreedyRef(d))
        log(f"{label}: sequence {b}: oracle prefill done")
    sess = make_session(cfg, w_gpu, tree, max_batch=B, max_len=max_len)
    if page_size != 16:
        raise ValueError("sessions here use 16-token pages")
    if trigram_entries:
        sess.trigram_cache(trigram_entries)
    ref_dev, ok_dev = torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda()
    sess.set_forcing(ref_dev, ok_dev)
    first = sess.prefill([np.asarray(p, dtype=np.int32) for p in prompts])
    ties = TieLog()
    for b, d in enumerate(decs):
        if int(first[b]) != d.pending:  # admissible only as a tie of the oracle's own logits
            logits, _, _ = d.o.causal_forward(d.seq[: d.n])
            z = logits[-1]
            assert abs(z[int(first[b])] - z[d.pending]) <= 2 * t * (z.max() - z.min())
            d.pending = int(first[b])
            d.seq[-1] = int(first[b])
            ties.argmax_ties += 1

    def extend_reference():
        # a step with committed length n reads the forcing at n+1 .. n+K
        for b, d in enumerate(decs):
            g = grefs[b].upto(d.n + K + 1)
            n0 = grefs[b].n0
            ref[b, n0:n0 + len(g)] = g
            ref_dev[b, n0:n0 + len(g)] = torch.from_numpy(ref[b, n0:n0 + len(g)].copy())
        torch.cuda.synchronize()

    errs, lens = [], []
    for i in range(steps):
        extend_reference()
        art = gpu_step(sess)
        for b, d in enumerate(decs):
            new, err = check_step(art, b, d, t, ties, forced=d.forcing)
            errs.append(err)
            lens.append(len(new))
        log(f"{label}: step {i}: max verify rel err {max(errs[-B:]):.2e}, accepted {lens[-B:]}")
    if trigram_entries:
        lookups, hits = sess.trigram_stats()
        log(f"{label}: trigram cache {hits}/{lookups} hits")
    sess.close()
    log(f"{label}: {steps} steps x {B} sequence(s) match the oracle; max err {max(errs):.2e}, "
        f"ties argmax {ties.argmax_ties}, lists {ties.list_ties}, mean accepted {np.mean(lens):.2f}")
    return max(errs), ties, lens
