"""Pins of the oracle's branch-conditioned drafting (the tree reading of
Sec. 4.4): every depth-k node with children runs the draft along its own
root-to-node tokens, with the encoder query masked to its ancestors.

What fixes it, other than the oracle itself:
* on a chain-shaped tree it is chain drafting, exactly;
* each drafted node's logits equal a fresh, unmasked encoder run over that
  node's path alone (brute force per path, the draft-side analogue of the
  tree-pass check of the verify);
* a node's list depends on the tokens of its own path only;
* the stream stays the greedy stream (lossless), with the forced-acceptance
  closed form L = 1 + consecutive successes.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import chimera_oracle as co

CFG = synth.TINY
CHAIN3 = [(0,), (0, 0), (0, 0, 0)]
# several drafted nodes per level, a rank-1 and a rank-2 parent, ranks up to 2
WIDE = [(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (1, 2), (2, 0), (0, 0, 0), (0, 1, 0), (1, 0, 0), (1, 2, 1)]


def tiny_oracle(std=0.06, seed=0):
    w = synth.weights_to_numpy(synth.make_weights(CFG, target_seed=seed, draft_seed=seed + 1, std=std))
    return oracle.Oracle(CFG, w)


@pytest.fixture(scope="module")
def orc():
    return tiny_oracle()


def _state(o, tree, branch, n_steps=2, seed=11, forcing=None):
    dec = oracle.Decoder(o, tree, forcing, branch=branch)
    dec.prefill(list(synth.make_prompt(20, CFG.vocab, seed)))
    for _ in range(n_steps):
        dec.step()
    return dec


def test_drafted_nodes_are_the_internal_nodes():
    dec = oracle.Decoder(tiny_oracle(), WIDE, branch=True)
    t = dec.tree
    idx = {r: i for i, r in enumerate(t.ranks)}
    assert dec.drafted == [[0], [idx[(0,)], idx[(1,)], idx[(2,)]],
                           [idx[(0, 0)], idx[(0, 1)], idx[(1, 0)], idx[(1, 2)]]]
    assert dec.s == [3, 3, 2]


def test_chain_tree_branch_drafting_is_chain_drafting(orc):
    a = _state(orc, CHAIN3, branch=False)
    b = _state(orc, CHAIN3, branch=True)
    assert a.seq == b.seq and a.n == b.n
    la, za = a.draft()
    lb, zb = b.draft_branches()
    for k in range(a.K):
        u = b.drafted[k][0]
        assert u == (0 if k == 0 else k)  # the chain's node at depth k
        assert la[k] == lb[u]
        assert np.array_equal(za[k], zb[u])
    prompt = list(synth.make_prompt(24, CFG.vocab, 5))
    oa, sa = oracle.Decoder(orc, CHAIN3).generate(prompt, 30)
    ob, sb = oracle.Decoder(orc, CHAIN3, branch=True).generate(prompt, 30)
    assert oa == ob
    assert [s["tree_tokens"] for s in sa] == [s["tree_tokens"] for s in sb]


@pytest.mark.parametrize("tree", ["T8", "WIDE"])
def test_branch_lists_equal_fresh_encoder_runs_per_path(orc, tree):
    """Recompute every drafted node from a fresh memory built over its own
    path: the committed tokens, the pending token and the node's path tokens
    as one plain sequence, all of its trigram entries encoded again, no mask."""
    ranks = synth.TREE_T8 if tree == "T8" else WIDE
    dec = _state(orc, ranks, branch=True)
    lists, dl = dec.draft_branches()
    toks = dec.assemble(lists)
    n, t = dec.n, dec.tree
    _, h, _ = orc.causal_forward(dec.seq[:n])
    lk, lv = orc.encoder_kv(h, np.arange(n))
    checked = 0
    for k in range(dec.K):
        j = n + k
        for u in dec.drafted[k]:
            seq = dec.seq[: n + 1] + [toks[a] for a in t.anc[u][1:]]
            assert len(seq) == j + 1
            ht = orc.trigram_encode(orc.trigram_inputs(seq, list(range(j + 1))))
            tk, tv = orc.encoder_kv(ht, np.arange(j + 1))
            hf = orc.encoder_query(ht[j], j, np.concatenate([lk, tk]), np.concatenate([lv, tv]))
            z = orc.head_logits(k, h[-1], hf)
            np.testing.assert_allclose(dl[u], z, rtol=1e-10, atol=1e-12)
            assert lists[u] == co.top_s(z, dec.s[k])
            checked += 1
    assert checked == sum(len(x) for x in dec.drafted)
    # children carry their parent's own candidates
    for v in range(1, t.n):
        assert toks[v] == lists[t.parent[v]][t.ranks[v][-1]]


def test_branch_lists_depend_only_on_their_path(orc):
    dec = _state(orc, WIDE, branch=True)
    lists, dl = dec.draft_branches()
    toks = dec.assemble(lists)
    t = dec.tree
    u = t.ranks.index((1, 2))  # drafted at level 2; its path is root, (1,), (1, 2)
    off = [v for v in range(1, t.n) if v not in t.anc[u]]
    moved = list(toks)
    for v in off:
        moved[v] = (moved[v] + 17) % CFG.vocab
    l2, d2 = dec.draft_branches(tree_tokens=moved)
    assert np.array_equal(d2[u], dl[u]) and l2[u] == lists[u]
    # and it does depend on its own path
    on = list(toks)
    on[t.ranks.index((1,))] = (on[t.ranks.index((1,))] + 17) % CFG.vocab
    _, d3 = dec.draft_branches(tree_tokens=on)
    assert not np.allclose(d3[u], dl[u])


@pytest.mark.parametrize("std", [0.02, 0.06])
@pytest.mark.parametrize("tree", ["T8", "WIDE"])
def test_branch_lossless_unforced(std, tree):
    o = tiny_oracle(std=std)
    ranks = synth.TREE_T8 if tree == "T8" else WIDE
    prompt = list(synth.WORKLOADS["tiny"].prompts()[0])
    ar = o.greedy_ar(prompt, 32)
    out, _ = oracle.Decoder(o, ranks, branch=True).generate(prompt, 32)
    assert out == ar


@pytest.mark.parametrize("p", [0.7, 1.0])
def test_branch_lossless_forced_and_acceptance_closed_form(orc, p):
    prompt = list(synth.WORKLOADS["tiny"].prompts()[0])
    G, n0 = 40, len(prompt)
    ar = orc.greedy_ar(prompt, G + 8)
    g = np.zeros(n0 + G + 8, dtype=np.int64)
    g[n0:] = ar
    ok = synth.force_table(p, 3, 0, n0 + G + 8)
    dec = oracle.Decoder(orc, WIDE, oracle.Forcing(g, ok), branch=True)
    out, steps = dec.generate(prompt, G)
    assert out == ar[:G]
    K = dec.K
    for a in steps:
        run = 0
        while run < K and ok[a["n"] + 1 + run]:
            run += 1
        assert len(a["new_tokens"]) == 1 + run
        assert a["path"] == [0] + [dec.tree.ranks.index((0,) * d) for d in range(1, run + 1)]
    if p == 1.0:
        assert all(len(a["new_tokens"]) == K + 1 for a in steps[:-1])
