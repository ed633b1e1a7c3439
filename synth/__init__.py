"""Seeded synthetic inputs for the Chimera decode step.

This module is shared by the CPU oracle's tests, the GPU tests and the
benchmark.  It holds workload *definitions* and seeded random inputs only --
model shapes, candidate-tree shapes, random-init weights, prompts and the
forced-acceptance tables -- and none of the method's arithmetic (no norms,
attention, projections, acceptance or KV handling).

Workloads follow the paper's backbones (Table 1: Vicuna/LLaMA-2 7B and 13B
shapes) with random weights; the paper's datasets (ShareGPT, MT-bench,
Vicuna-bench; Experiment Setup, "Datasets") are not available, so uniform
random prompts plus seeded forced acceptance stand in for them.
"""
from __future__ import annotations

import dataclasses
import itertools
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Model shapes
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """Shape of the target decoder and of the Chimera draft attached to it.

    The target is a Llama-style decoder (pre-RMSNorm, multi-head attention
    with rotary positions, SwiGLU feed-forward, untied LM head).  The draft is
    the trigram encoder (Sec. 4.1.1, Eq. 2), one full-context encoder block at
    the target's width (Sec. 4.1.2, Eq. 3) and ``n_draft_heads`` residual
    decoding heads (Sec. 4.1.3, Eq. 4).
    """

    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    n_draft_heads: int
    dtype: str  # "f32" or "bf16": storage type of weights and activations
    rope_base: float = 10000.0
    rms_eps: float = 1e-5

    def __post_init__(self):
        assert self.n_heads * self.head_dim == self.d_model
        assert self.dtype in ("f32", "bf16")


TINY = ModelConfig(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=1024,
                   vocab=1024, n_draft_heads=3, dtype="f32")
LLAMA7B = ModelConfig(n_layers=32, d_model=4096, n_heads=32, head_dim=128,
                      d_ffn=11008, vocab=32000, n_draft_heads=4, dtype="bf16")
LLAMA13B = ModelConfig(n_layers=40, d_model=5120, n_heads=40, head_dim=128,
                       d_ffn=13824, vocab=32000, n_draft_heads=4, dtype="bf16")
# Vicuna-33B shape (Table 1): 60 layers, d 6656, 52 heads of 128, F 17920
VICUNA33B = ModelConfig(n_layers=60, d_model=6656, n_heads=52, head_dim=128,
                        d_ffn=17920, vocab=32000, n_draft_heads=4, dtype="bf16")


def small_config(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512,
                 vocab=2048, n_draft_heads=4, dtype="bf16") -> ModelConfig:
    """A small bf16 model with the 7B head size, used for fast parity tests."""
    return ModelConfig(n_layers=n_layers, d_model=d_model, n_heads=n_heads,
                       head_dim=head_dim, d_ffn=d_ffn, vocab=vocab,
                       n_draft_heads=n_draft_heads, dtype=dtype)


# ---------------------------------------------------------------------------
# Candidate trees
# ---------------------------------------------------------------------------
# Per-rank acceptance probabilities of the draft heads, derived from the top-k
# head accuracies of Chimera on Vicuna-7B (Table 5): q_k(r) = Acc_k(top-(r+1))
# - Acc_k(top-r).  They only shape the static candidate trees.
HEAD_TOPK_ACC = (
    (0.66, 0.78, 0.83, 0.87, 0.90),
    (0.49, 0.55, 0.60, 0.68, 0.75),
    (0.38, 0.44, 0.49, 0.55, 0.62),
    (0.33, 0.38, 0.43, 0.46, 0.54),
)

# Explicit rank-tuple trees (root excluded).  A node (r_0..r_k) holds the
# rank-r_k candidate of draft head k and sits at depth k+1.
TREE_T8 = ((0,), (1,), (2,), (0, 0), (0, 3), (1, 0), (0, 0, 0))
TREE_T32 = (
    (0,), (1,), (2,), (3,), (4,), (0, 0), (0, 1), (0, 2), (0, 3), (0, 4),
    (1, 0), (1, 3), (1, 4), (2, 0), (3, 0), (4, 0), (0, 0, 0), (0, 0, 1),
    (0, 0, 2), (0, 0, 3), (0, 0, 4), (0, 1, 0), (0, 2, 0), (0, 3, 0),
    (0, 4, 0), (1, 0, 0), (2, 0, 0), (3, 0, 0), (0, 0, 0, 0), (0, 0, 0, 4),
    (0, 0, 4, 0))
TREE_T64 = (
    (0,), (1,), (2,), (3,), (4,), (0, 0), (0, 1), (0, 2), (0, 3), (0, 4),
    (1, 0), (1, 1), (1, 2), (1, 3), (1, 4), (2, 0), (2, 1), (2, 3), (2, 4),
    (3, 0), (3, 3), (3, 4), (4, 0), (0, 0, 0), (0, 0, 1), (0, 0, 2),
    (0, 0, 3), (0, 0, 4), (0, 1, 0), (0, 1, 4), (0, 2, 0), (0, 3, 0),
    (0, 3, 1), (0, 3, 3), (0, 3, 4), (0, 4, 0), (0, 4, 1), (0, 4, 4),
    (1, 0, 0), (1, 0, 1), (1, 0, 2), (1, 0, 3), (1, 0, 4), (1, 3, 0),
    (1, 4, 0), (2, 0, 0), (3, 0, 0), (4, 0, 0), (0, 0, 0, 0), (0, 0, 0, 1),
    (0, 0, 0, 2), (0, 0, 0, 3), (0, 0, 0, 4), (0, 0, 1, 0), (0, 0, 2, 0),
    (0, 0, 3, 0), (0, 0, 4, 0), (0, 1, 0, 0), (0, 2, 0, 0), (0, 3, 0, 0),
    (0, 4, 0, 0), (1, 0, 0, 0), (2, 0, 0, 0))

TREES = {"T8": TREE_T8, "T32": TREE_T32, "T64": TREE_T64}


def derive_tree(n_nodes: int, n_levels: int, max_rank: int = 5) -> Tuple[Tuple[int, ...], ...]:
    """Greedy static tree: the ``n_nodes - 1`` rank tuples with the highest
    product of per-rank acceptance probabilities (Table 5), ties broken by
    (shorter, lexicographically smaller), then ordered by (depth, tuple)."""
    q = [[round(acc[r] - (acc[r - 1] if r else 0.0), 10) for r in range(max_rank)]
         for acc in HEAD_TOPK_ACC]
    cands = []
    for depth in range(1, n_levels + 1):
        for t in itertools.product(range(max_rank), repeat=depth):
            p = 1.0
            for k, r in enumerate(t):
                p *= q[k][r]
            cands.append((-p, depth, t))
    cands.sort()
    sel = [c[2] for c in cands[: n_nodes - 1]]
    sel.sort(key=lambda t: (len(t), t))
    return tuple(sel)


def tree_top_s(tree: Sequence[Tuple[int, ...]], n_levels: int) -> List[int]:
    """Number of candidates each draft head must supply: 1 + the largest rank
    that the tree uses at that level."""
    s = [1] * n_levels
    for t in tree:
        k = len(t) - 1
        s[k] = max(s[k], t[-1] + 1)
    return s


def chain_tree(n_levels: int) -> Tuple[Tuple[int, ...], ...]:
    """The all-rank-0 chain of ``n_levels`` draft tokens."""
    return tuple((0,) * d for d in range(1, n_levels + 1))


# ---------------------------------------------------------------------------
# Weights
# ---------------------------------------------------------------------------
INIT_STD = 0.02


def tensor_specs(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Canonical tensor list: (name, shape, group).  Matrices are stored
    [d_in, d_out] so that a projection reads y = x @ W, the paper's notation
    (e.g. W_1 in R^{3d x d}, Eq. 2).  ``group`` is "target" or "draft";
    norm gains have group "gain" (all ones)."""
    d, F, V = cfg.d_model, cfg.d_ffn, cfg.vocab
    hd = cfg.n_heads * cfg.head_dim
    out = [("tok_embed", (V, d), "target")]

    def block(prefix, group):
        return [
            (prefix + "attn_norm", (d,), "gain"),
            (prefix + "wq", (d, hd), group),
            (prefix + "wk", (d, hd), group),
            (prefix + "wv", (d, hd), group),
            (prefix + "wo", (hd, d), group),
            (prefix + "ffn_norm", (d,), "gain"),
            (prefix + "w_gate", (d, F), group),
            (prefix + "w_up", (d, F), group),
            (prefix + "w_down", (F, d), group),
        ]

    for l in range(cfg.n_layers):
        out += block(f"layers.{l}.", "target")
    out += [("final_norm", (d,), "gain"), ("lm_head", (d, V), "target")]
    out += [("draft.tri_w1", (3 * d, d), "draft"), ("draft.tri_w2", (d, d), "draft")]
    out += block("draft.enc.", "draft")
    for k in range(cfg.n_draft_heads):
        out += [(f"draft.heads.{k}.a", (2 * d, d), "draft"),
                (f"draft.heads.{k}.theta", (d, V), "draft")]
    return out


def _splitmix64(x: int) -> int:
    """SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014)."""
    m = (1 << 64) - 1
    z = (x + 0x9E3779B97F4A7C15) & m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def tensor_seed(seed: int, index: int) -> int:
    return _splitmix64(_splitmix64(seed) ^ index) & ((1 << 63) - 1)


def make_weights(cfg: ModelConfig, target_seed: int = 0, draft_seed: int = 1,
                 device: str = "cpu", names: Optional[Sequence[str]] = None,
                 std: float = INIT_STD):
    """Random-init weights N(0, std) (std 0.02 by default; larger values give
    less repetitive greedy streams for tests), one torch generator per tensor seeded
    from (group seed, tensor index).  bf16 configs round by RNE.  Returns an
    ordered dict name -> torch tensor on ``device``.  The values depend on the
    device kind of the generator (CPU and GPU generators differ)."""
    import torch

    tdt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    out: Dict[str, "torch.Tensor"] = {}
    for idx, (name, shape, group) in enumerate(tensor_specs(cfg)):
        if names is not None and name not in names:
            continue
        if group == "gain":
            out[name] = torch.ones(shape, dtype=torch.float32, device=device)
            continue
        seed = target_seed if group == "target" else draft_seed
        g = torch.Generator(device=device)
        g.manual_seed(tensor_seed(seed, idx))
        t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        t.mul_(std)
        out[name] = t.to(tdt)
    return out


def weights_to_numpy(weights) -> Dict[str, np.ndarray]:
    """float32 tensors -> float32 arrays; bfloat16 tensors -> uint16 arrays of
    their bit patterns (the oracle upcasts them exactly)."""
    import torch

    out = {}
    for k, t in weights.items():
        t = t.detach().cpu()
        if t.dtype == torch.bfloat16:
            out[k] = t.view(torch.int16).numpy().view(np.uint16).copy()
        else:
            out[k] = t.numpy().astype(np.float32, copy=True)
    return out


# ---------------------------------------------------------------------------
# Prompts and forced acceptance
# ---------------------------------------------------------------------------


def make_prompt(n: int, vocab: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, size=n).astype(np.int32)


def make_prompt_lengths(batch: int, lo: int, hi: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(lo, hi + 1, size=batch).astype(np.int32)


def force_table(p: float, seed: int, batch_index: int, length: int) -> np.ndarray:
    """Per-position success bits of the forced-acceptance bias: position j
    succeeds iff (splitmix64(splitmix64(splitmix64(seed) ^ b) ^ j) >> 11) <
    floor(p * 2^53).  Returned as uint8 [length]."""
    thr = int(np.floor(p * float(1 << 53)))
    base = _splitmix64(_splitmix64(seed) ^ batch_index)
    return np.array([1 if (_splitmix64(base ^ j) >> 11) < thr else 0 for j in range(length)],
                    dtype=np.uint8)


# ---------------------------------------------------------------------------
# Workloads
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    tree: str
    batch: int
    prompt_len: int           # single length (batch 1) or upper bound
    gen_tokens: int
    accept_p: Optional[Tuple[float, ...]]  # forced-acceptance probabilities, None = unforced
    prompt_len_lo: Optional[int] = None     # ragged batches: U[lo, prompt_len]
    target_seed: int = 0
    draft_seed: int = 1
    prompt_seed: int = 2
    force_seed: int = 3
    length_seed: int = 4
    p_seed: int = 5
    page_size: int = 16

    def prompts(self) -> List[np.ndarray]:
        V = self.model.vocab
        if self.batch == 1:
            return [make_prompt(self.prompt_len, V, self.prompt_seed)]
        lens = make_prompt_lengths(self.batch, self.prompt_len_lo, self.prompt_len, self.length_seed)
        return [make_prompt(int(n), V, self.prompt_seed * 1000 + b) for b, n in enumerate(lens)]

    def accept_probs(self) -> Optional[List[float]]:
        if self.accept_p is None:
            return None
        if len(self.accept_p) == 2 and self.batch > 1:
            lo, hi = self.accept_p
            return list(np.random.default_rng(self.p_seed).uniform(lo, hi, size=self.batch))
        return [float(self.accept_p[0])] * self.batch


WORKLOADS = {
    # tiny fp32, CPU-checkable: 32-token prompt, 64 generated tokens, T8
    "tiny": Workload("tiny", TINY, "T8", 1, 32, 64, None),
    # Llama-7B shape, 512-token prompt, 256 tokens, T64, p = 0.7
    "llama7b_p512": Workload("llama7b_p512", LLAMA7B, "T64", 1, 512, 256, (0.7,)),
    # Llama-7B shape, 4096-token prompt (long paged context)
    "llama7b_p4096": Workload("llama7b_p4096", LLAMA7B, "T64", 1, 4096, 256, (0.7,)),
    # Llama-13B shape, 1024-token prompt, p = 0.5 and p = 0.8
    "llama13b_p1024_a05": Workload("llama13b_p1024_a05", LLAMA13B, "T64", 1, 1024, 256, (0.5,)),
    "llama13b_p1024_a08": Workload("llama13b_p1024_a08", LLAMA13B, "T64", 1, 1024, 256, (0.8,)),
    # Vicuna-33B shape, 512-token prompt, T64, p = 0.7
    "vicuna33b_p512": Workload("vicuna33b_p512", VICUNA33B, "T64", 1, 512, 256, (0.7,)),
    # batch 8, ragged prompts U[256, 2048], T32, p_b ~ U[0.4, 0.9]
    "llama7b_b8": Workload("llama7b_b8", LLAMA7B, "T32", 8, 2048, 128, (0.4, 0.9), prompt_len_lo=256),
    # the same batch with the 8-node tree: 64 verify rows, as many as one sequence's T64
    "llama7b_b8_t8": Workload("llama7b_b8_t8", LLAMA7B, "T8", 8, 2048, 128, (0.4, 0.9), prompt_len_lo=256),
}
