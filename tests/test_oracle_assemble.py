"""Pins of the oracle's candidate-tree assembly (Sec. 4.4: the candidates are
built from the per-head top-k lists).

Each drafted list holds sentinel ids that name where they came from, so a
tree token says which list and which rank it was taken from.  The expected
tokens below are written out by hand from the rule, not computed by it:

* chain drafting: node (r_0, ..., r_k) takes rank r_k of head k's list;
* branch-conditioned drafting: it takes rank r_k of its parent's own list.

Plausible slips (the first rank instead of the last, a level off by one,
the node's own list instead of its parent's) are planted in copies of the
oracle's method and must fail the same check.
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import chimera_oracle as co

PENDING = 7


class _Stub:
    """The parts of an Oracle that Decoder.__init__ reads."""

    def __init__(self, K):
        self.cfg = synth.small_config(n_draft_heads=K)


def _decoder(tree, branch):
    K = max(len(r) for r in tree)
    d = oracle.Decoder(_Stub(K), tree, branch=branch)
    d.pending = PENDING
    return d


def chain_lists(K, s=8):
    # head k's rank-r candidate is the id 100 * (k + 1) + r
    return [[100 * (k + 1) + r for r in range(s)] for k in range(K)]


def branch_lists(tree):
    # drafted node u's rank-r candidate is the id 1000 + 10 * u + r
    t = co.Tree(tree)
    return {u: [1000 + 10 * u + r for r in range(8)] for u in range(t.n) if u in t.parent}


# T8 (nodes 1..7 = (0,) (1,) (2,) (0,0) (0,3) (1,0) (0,0,0)), written out by hand
T8_CHAIN = [PENDING, 100, 101, 102, 200, 203, 200, 300]
#   parents:          -    0    0    0    1    1    2    4
T8_BRANCH = [PENDING, 1000, 1001, 1002, 1010, 1013, 1020, 1040]

# the first 24 nodes of T64, (0,) .. (4,0) then (0,0,0)
T64_CHAIN_HEAD = [PENDING, 100, 101, 102, 103, 104,
                  200, 201, 202, 203, 204, 200, 201, 202, 203, 204,
                  200, 201, 203, 204, 200, 203, 204, 200, 300]
T64_BRANCH_HEAD = [PENDING, 1000, 1001, 1002, 1003, 1004,
                   1010, 1011, 1012, 1013, 1014, 1020, 1021, 1022, 1023, 1024,
                   1030, 1031, 1033, 1034, 1040, 1043, 1044, 1050, 1060]


def check_chain(assemble_fn):
    d = _decoder(synth.TREE_T8, False)
    assert assemble_fn(d, chain_lists(3)) == T8_CHAIN
    d = _decoder(synth.TREE_T64, False)
    got = assemble_fn(d, chain_lists(4))
    assert got[:25] == T64_CHAIN_HEAD
    # the four-deep nodes of T64 all end in head 3's list; the all-zeros chain
    # is the rank-0 token of every head in turn
    assert got[-15:] == [400, 401, 402, 403, 404, 400, 400, 400, 400, 400, 400, 400, 400, 400, 400]
    chain = [i + 1 for i, r in enumerate(synth.TREE_T64) if all(x == 0 for x in r)]
    assert [got[u] for u in chain] == [100, 200, 300, 400]


def check_branch(assemble_fn):
    d = _decoder(synth.TREE_T8, True)
    assert assemble_fn(d, branch_lists(synth.TREE_T8)) == T8_BRANCH
    d = _decoder(synth.TREE_T64, True)
    assert assemble_fn(d, branch_lists(synth.TREE_T64))[:25] == T64_BRANCH_HEAD


def test_chain_assembly_takes_head_k_rank_rk():
    check_chain(lambda d, lists: d.assemble(lists))


def test_branch_assembly_takes_the_parents_list():
    check_branch(lambda d, lists: d.assemble(lists))


def _planted(kind):
    """Decoder.assemble with one slip planted."""

    def fn(d, lists):
        t = d.tree
        toks = [d.pending]
        for u in range(1, t.n):
            r = t.ranks[u]
            if kind == "first_rank":
                src, rank = lists[len(r) - 1], r[0]
            elif kind == "level_plus_one":
                src, rank = lists[min(len(r), len(lists) - 1)], r[-1]
            elif kind == "level_minus_one":
                src, rank = lists[max(len(r) - 2, 0)], r[-1]
            elif kind == "own_list":
                src, rank = lists.get(u, lists[t.parent[u]]), r[-1]
            elif kind == "grandparent":
                gp = t.parent[t.parent[u]]
                src, rank = lists[gp if gp >= 0 else 0], r[-1]
            else:
                raise ValueError(kind)
            toks.append(int(src[rank]))
        return toks

    return fn


@pytest.mark.parametrize("kind", ["first_rank", "level_plus_one", "level_minus_one"])
def test_planted_chain_slips_fail(kind):
    with pytest.raises(AssertionError):
        check_chain(_planted(kind))


@pytest.mark.parametrize("kind", ["own_list", "grandparent"])
def test_planted_branch_slips_fail(kind):
    with pytest.raises(AssertionError):
        check_branch(_planted(kind))


def test_step_uses_assemble_on_its_own_lists():
    """In a full oracle step the tree tokens are the assembly of the step's
    own draft lists (chain and branch-conditioned drafting)."""
    cfg = synth.TINY
    w = synth.weights_to_numpy(synth.make_weights(cfg, device="cpu", std=0.06))
    orc = oracle.Oracle(cfg, w)
    prompt = list(synth.make_prompt(20, cfg.vocab, 5))
    for branch in (False, True):
        d = oracle.Decoder(orc, synth.TREE_T8, branch=branch)
        d.prefill(prompt)
        for _ in range(2):
            pending = d.pending
            art = d.step()
            lists = art["lists"]
            t = d.tree
            for u in range(1, t.n):
                r = t.ranks[u]
                src = lists[t.parent[u]] if branch else lists[len(r) - 1]
                assert art["tree_tokens"][u] == src[r[-1]]
            assert art["tree_tokens"][0] == pending
            # siblings have distinct ranks, so their tokens are distinct
            for p in range(t.n):
                kids = [art["tree_tokens"][u] for u in range(1, t.n) if t.parent[u] == p]
                assert len(kids) == len(set(kids))
