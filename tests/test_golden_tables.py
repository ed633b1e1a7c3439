"""Workload definitions against the values the paper prints (Table 1 model
shapes, Table 5 head accuracies that shape the candidate trees)."""
import os

import synth

HERE = os.path.join(os.path.dirname(__file__), "golden", "paper_tables.txt")


def _rows(tag):
    with open(HERE) as f:
        return [l.split()[1:] for l in f if l.startswith(tag + " ")]


def test_table1_shapes():
    rows = {r[0]: tuple(int(x) for x in r[1:]) for r in _rows("table1")}
    for name, cfg in (("Vicuna-7B", synth.LLAMA7B), ("LlaMA-2-chat-13B", synth.LLAMA13B),
                      ("Vicuna-33B", synth.VICUNA33B)):
        layers, hidden, heads = rows[name]
        assert (cfg.n_layers, cfg.d_model, cfg.n_heads) == (layers, hidden, heads)
        assert cfg.head_dim * cfg.n_heads == hidden


def test_table5_accuracies_drive_trees():
    rows = [tuple(float(x) for x in r[1:]) for r in _rows("table5")]
    assert tuple(rows) == synth.HEAD_TOPK_ACC
    for r in rows:  # top-k accuracy is non-decreasing in k
        assert all(a <= b for a, b in zip(r, r[1:]))
