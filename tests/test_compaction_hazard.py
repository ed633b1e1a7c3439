"""Hazard analysis of the in-place KV compaction after acceptance (CPU).

After a step accepts the path (path[0] = root, path[1], ..., path[L-1]), the
tree slot of node path[d] (position n + path[d]) is moved to position n + d.
The kernel does this in place, for d = 1 .. L-1 in increasing order, with no
staging buffer.  That is safe because tree nodes are numbered in
breadth-first order, so a node at depth d has id >= d: every source slot lies
at or above its destination, and every destination below it has already
been read.  This test checks the claim on every root-to-node path of every
tree the workloads use, and that the opposite order would corrupt some path.
"""
import pytest

import synth


def _nodes(tree):
    """Rank tuples in node-id order, the root first."""
    return [()] + list(tree)


def _paths(tree):
    nodes = _nodes(tree)
    idx = {r: i for i, r in enumerate(nodes)}
    for r in nodes:
        yield [idx[r[:d]] for d in range(len(r) + 1)]


def _compact(path, order):
    slots = list(range(max(path) + 1))  # slot n+u holds node u's row
    ds = range(1, len(path)) if order == "increasing" else range(len(path) - 1, 0, -1)
    for d in ds:
        slots[d] = slots[path[d]]
    return slots[: len(path)]


TREES = {"T8": synth.TREE_T8, "T32": synth.TREES["T32"], "T64": synth.TREES["T64"]}


@pytest.mark.parametrize("name", sorted(TREES))
def test_sources_never_below_destinations(name):
    for path in _paths(TREES[name]):
        assert all(path[d] >= d for d in range(len(path))), path


@pytest.mark.parametrize("name", sorted(TREES))
def test_increasing_order_compacts_every_path(name):
    for path in _paths(TREES[name]):
        assert _compact(path, "increasing") == path, path


@pytest.mark.parametrize("name", sorted(TREES))
def test_decreasing_order_would_corrupt_a_path(name):
    bad = [p for p in _paths(TREES[name]) if _compact(p, "decreasing") != p]
    assert bad, "the reverse order is hazardous on some path of every tree"
