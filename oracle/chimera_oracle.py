"""CPU oracle for one Chimera decode step (Zeng et al., "Chimera: A Lossless
Decoding Method for Accelerating Large Language Models Inference by Fusing
all Tokens", arXiv 2402.15758).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke entry point and the
benchmark's CPU-baseline leg may import this module; the GPU product path
never calls it and shares no code with it.

It is a plain, slow, NumPy implementation of what one decode step computes:

* the target LLM (Sec. 3.1, Eq. 1), a Llama-style decoder;
* the draft: trigram encoder (Sec. 4.1.1, Eq. 2), full-context encoder
  (Sec. 4.1.2, Eq. 3) and residual decoding heads (Sec. 4.1.3, Eq. 4);
* candidate construction from per-head top-k lists (Sec. 4.4);
* verification of the whole candidate tree in one target pass with
  tree-structured attention (Sec. 4.3);
* greedy acceptance of the longest matching path (Sec. 4.3, Sec. 4.4) and
  the commit of the accepted tokens' keys/values.

Arithmetic runs in float64 (``compute=np.float64``, the default) or float32.
Models whose storage type is bf16 round to bf16 (round-to-nearest-even) at
the storage points of the numeric contract: GEMM inputs, Q/K/V, the KV
caches, the attention output and the SwiGLU product.  The residual streams,
norms, softmax and logits stay in the compute type.

Readings of points the paper leaves open (all documented next to the code
that takes them):

* the first two trigrams are left zero-padded (Sec. 4.1.1 collapses them to a
  unigram and a bigram, which cannot feed W_1 in R^{3d x d});
* no biases anywhere; the draft shares the target's token embeddings;
* the full-context encoder is one Llama decoder block at the target's width;
  every encoder entry carries its sequence position; at inference the query
  at trigram position j sees all target-state entries 0..n-1 and trigram
  entries 0..j, and only that query's output is used;
* each residual head is MLP = A_k (2d -> d), SiLU, Theta_k (d -> V);
* h^LLM is the target's post-final-norm last-layer state;
* the draft runs as a chain: head k reads the encoder output at the position
  reached by the rank-0 tokens of heads 0..k-1; its top-s list is shared by
  every tree branch at depth k+1;
* branch-conditioned drafting (the tree reading of Sec. 4.4, optional): level
  k runs the draft once for every depth-k tree node that has children, along
  that node's own root-to-node tokens; the encoder query of such a node sees
  the target-state entries 0..n-1, the trigram entries 0..n-1 and the
  trigram entries of its ancestors-or-self (the tree mask of Sec. 4.3
  applied to the encoder), and a child of rank r takes the rank-r token of
  its parent's own list.  On a chain-shaped tree it is chain drafting;
* greedy acceptance takes the longest root-to-node path whose every non-root
  token equals the target's argmax at its parent, then the bonus token;
* argmax ties go to the lowest id; top-s orders by (value desc, id asc);
* typical decoding (Sec. 4.3, Sec. 5.1, T = 1): a draft node passes when the
  target's probability of its token at its parent exceeds
  min(eps, delta * exp(-H)), H that distribution's entropy (the paper defers
  the rule and its thresholds to Medusa; eps = 0.09, delta = 0.3 by default);
  the chosen node is the deepest whose whole path passes, then the highest
  path log-probability, then the lowest index; the bonus token and the first
  token after the prompt are sampled by the Gumbel-max trick from a
  SplitMix64 chain keyed by (seed, sequence, position, token).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Elementary pieces
# ---------------------------------------------------------------------------


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bit patterns (uint16) to float32."""
    return (u16.astype(np.uint32) << 16).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bf16 value, ties to even, after rounding to
    float32 (the GPU rounds float32 accumulators).  Returns the rounded
    values in the input's float type (float64 for non-float input)."""
    x = np.asarray(x)
    f = x.astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = (((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16).astype(np.uint32)
    out = np.where(np.isnan(f), f, r.view(np.float32))
    return out.astype(x.dtype if x.dtype.kind == "f" else np.float64)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x * sigmoid(x), the activation of Eq. 2 and Eq. 4."""
    return x / (1.0 + np.exp(-x))


def rope_cos_sin(positions: np.ndarray, head_dim: int, base: float):
    """Rotary tables for the given positions: angle(p, i) = p * base^(-2i/hd),
    i < hd/2, evaluated in float64 and rounded to float32."""
    half = head_dim // 2
    inv = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    return (np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32))


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding of x [M, H, hd]: dims (i, i + hd/2) form
    the pair rotated by angle(p, i).  cos/sin are [M, hd/2]."""
    half = x.shape[-1] // 2
    c = cos[:, None, :].astype(x.dtype)
    s = sin[:, None, :].astype(x.dtype)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def masked_attention(q, k, v, visible, rows_per_block: int = 256):
    """Multi-head scaled dot-product attention.
    q [M, H, hd]; k, v [P, H, hd]; visible [M, P] bool.  Returns [M, H, hd].

    softmax(q k^T / sqrt(hd)) v per head, over the keys each query may see.
    Query rows are independent, so they are evaluated in blocks of
    ``rows_per_block``; a block reads the keys up to the last one any of its
    rows can see (the keys after it would only add exact zeros)."""
    M, H, hd = q.shape
    out = np.zeros((M, H, v.shape[-1]), dtype=np.result_type(q, v))
    kh = np.ascontiguousarray(np.transpose(k, (1, 2, 0)))  # [H, hd, P]
    vh = np.ascontiguousarray(np.transpose(v, (1, 0, 2)))  # [H, P, hd]
    for r0 in range(0, M, rows_per_block):
        r1 = min(M, r0 + rows_per_block)
        vis = visible[r0:r1]
        cols = np.nonzero(vis.any(axis=0))[0]
        if cols.size == 0:
            continue
        p_end = int(cols[-1]) + 1
        qh = np.ascontiguousarray(np.transpose(q[r0:r1], (1, 0, 2)))  # [H, m, hd]
        s = np.matmul(qh, kh[:, :, :p_end])
        s /= np.sqrt(hd)
        s += np.where(vis[:, :p_end], 0.0, -np.inf).astype(s.dtype)[None, :, :]
        s -= np.max(s, axis=-1, keepdims=True)
        np.exp(s, out=s)
        s /= np.sum(s, axis=-1, keepdims=True)
        out[r0:r1] = np.transpose(np.matmul(s, vh[:, :p_end]), (1, 0, 2))
    return out


def argmax_lowest(z: np.ndarray) -> int:
    """argmax over a 1-D array; ties resolve to the lowest index."""
    return int(np.argmax(z))  # numpy returns the first maximal index


def top_s(z: np.ndarray, s: int, exclude: Optional[int] = None) -> List[int]:
    """Ids of the s largest entries, ordered by (value desc, id asc)."""
    order = np.lexsort((np.arange(z.shape[0]), -z))
    if exclude is not None:
        order = order[order != exclude]
    return [int(i) for i in order[:s]]


# ---------------------------------------------------------------------------
# Typical decoding (Sec. 4.3: candidates chosen by their probability under the
# original model; Sec. 5.1: temperature T = 1)
# ---------------------------------------------------------------------------
_M64 = (1 << 64) - 1


def splitmix64(x: int) -> int:
    """One output of SplitMix64 (Steele, Lea and Flood, 2014) for state x:
    advance by the golden-ratio increment, then two xor-shift-multiply
    rounds and a final xor-shift."""
    z = (x + 0x9E3779B97F4A7C15) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def sample_uniform(seed: int, b: int, pos: int, v: int) -> float:
    """Uniform draw in (0, 1) for token v of the sample at position pos of
    sequence b: the top 53 bits of a chain of SplitMix64 outputs, centred
    in their interval."""
    z = splitmix64(splitmix64(splitmix64(splitmix64(seed) ^ b) ^ pos) ^ v)
    return ((z >> 11) + 0.5) * 2.0 ** -53


def gumbel_sample(z: np.ndarray, seed: int, b: int, pos: int) -> int:
    """Exact sample from softmax(z) by the Gumbel-max trick: the index of
    the largest z_v - log(-log(u_v)) (ties to the lowest index)."""
    g = np.array([-np.log(-np.log(sample_uniform(seed, b, pos, v))) for v in range(len(z))])
    return argmax_lowest(np.asarray(z, dtype=np.float64) + g)


def log_probs_entropy(z: np.ndarray):
    """log softmax(z) and the entropy -sum p log p of softmax(z)."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max()
    lp = z - (m + np.log(np.exp(z - m).sum()))
    return lp, float(-(np.exp(lp) * lp).sum())


class Typical:
    """Typical acceptance settings: temperature, the hard threshold eps, the
    entropy-scaled threshold delta, and the sampler's seed."""

    def __init__(self, temperature: float = 1.0, eps: float = 0.09, delta: float = 0.3, seed: int = 0):
        self.T = float(temperature)
        self.eps = float(eps)
        self.delta = float(delta)
        self.seed = int(seed)


def typical_accept(tree: "Tree", tree_tokens: Sequence[int], logits: np.ndarray, typ: Typical, n: int,
                   b: int = 0):
    """Typical acceptance over a verified tree.  Node u (depth >= 1) passes
    when p_parent(tok_u) > min(eps, delta * exp(-H_parent)) with p the
    target distribution at temperature T; the chosen node is the deepest
    whose whole root path passes, then the highest path log-probability,
    then the lowest index; the bonus token is sampled from the chosen
    node's distribution for position n + depth + 1.  Returns (path, bonus,
    per-node pass flags, per-node token log-probabilities)."""
    stats = [log_probs_entropy(np.asarray(r, dtype=np.float64) / typ.T) for r in logits]
    ok = [True] * tree.n
    lp = [0.0] * tree.n
    for u in range(1, tree.n):
        lpp, H = stats[tree.parent[u]]
        thr = min(typ.eps, typ.delta * float(np.exp(-H)))
        lp[u] = float(lpp[tree_tokens[u]])
        ok[u] = thr <= 0.0 or lp[u] > float(np.log(thr))
    best, best_key = 0, None
    for u in range(tree.n):
        if not all(ok[a] for a in tree.anc[u]):
            continue
        key = (tree.depth[u], sum(lp[a] for a in tree.anc[u]), -u)
        if best_key is None or key > best_key:
            best, best_key = u, key
    pos = n + tree.depth[best] + 1
    bonus = gumbel_sample(np.asarray(logits[best], dtype=np.float64) / typ.T, typ.seed, b, pos)
    return list(tree.anc[best]), int(bonus), ok, lp


# ---------------------------------------------------------------------------
# Candidate tree metadata (Sec. 4.3 tree attention; Sec. 4.4 candidates)
# ---------------------------------------------------------------------------


class Tree:
    """Static candidate tree from rank tuples.  Node 0 is the root (the
    pending token); node i >= 1 is rank tuple ``ranks[i-1]`` at depth
    len(tuple), holding the rank-r_k candidate of draft head k.  Nodes are
    ordered by (depth, tuple), so every parent precedes its children."""

    def __init__(self, ranks: Sequence[Tuple[int, ...]]):
        self.ranks: List[Tuple[int, ...]] = [()] + [tuple(r) for r in ranks]
        index = {r: i for i, r in enumerate(self.ranks)}
        self.n = len(self.ranks)
        self.depth = [len(r) for r in self.ranks]
        self.parent = [-1] + [index[r[:-1]] for r in self.ranks[1:]]
        # ancestor-or-self sets: the nodes whose keys node u may attend to
        self.anc: List[List[int]] = []
        for u in range(self.n):
            path = []
            w = u
            while w >= 0:
                path.append(w)
                w = self.parent[w]
            self.anc.append(sorted(path, key=lambda x: self.depth[x]))
        self.levels = max(self.depth)

    def mask(self) -> np.ndarray:
        """visible[u, v] = v is an ancestor of u or u itself."""
        m = np.zeros((self.n, self.n), dtype=bool)
        for u in range(self.n):
            m[u, self.anc[u]] = True
        return m


# ---------------------------------------------------------------------------
# Networks
# ---------------------------------------------------------------------------


class Oracle:
    """Target and draft networks on the CPU.

    ``weights`` maps the canonical tensor names to float32 arrays (f32
    models) or uint16 bf16 bit patterns (bf16 models); matrices are stored
    [d_in, d_out] so that a projection is y = x @ W.
    """

    def __init__(self, cfg, weights: Dict[str, np.ndarray], compute=np.float64,
                 cache_weights: bool = True):
        self.cfg = cfg
        self.raw = weights
        self.ct = compute
        self.cache_weights = cache_weights
        self._cache: Dict[str, np.ndarray] = {}
        self.H, self.hd, self.d = cfg.n_heads, cfg.head_dim, cfg.d_model
        self.bf16 = cfg.dtype == "bf16"

    # -- storage -----------------------------------------------------------
    def w(self, name: str) -> np.ndarray:
        if name in self._cache:
            return self._cache[name]
        a = self.raw[name]
        a = bf16_bits_to_f32(a) if a.dtype == np.uint16 else a
        a = a.astype(self.ct)
        if self.cache_weights:
            self._cache[name] = a
        return a

    def st(self, x: np.ndarray) -> np.ndarray:
        """Value at a storage point: rounded to bf16 for bf16 models."""
        x = np.asarray(x, dtype=self.ct)
        return round_bf16(x).astype(self.ct) if self.bf16 else x

    def embed(self, tokens: Sequence[int]) -> np.ndarray:
        """Token embeddings x_i (Sec. 4.1.1) -- rows of the target's table."""
        return self.w("tok_embed")[np.asarray(tokens, dtype=np.int64)]

    def rope(self, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
        c, s = rope_cos_sin(pos, self.hd, self.cfg.rope_base)
        return apply_rope(x, c, s)

    # -- one Llama decoder block (target layers and the encoder block) ------
    def block_kv(self, prefix: str, x: np.ndarray, pos: np.ndarray):
        """Pre-norm K/V of the entries x [M, d] at positions pos."""
        xn = self.st(rms_norm(x, self.w(prefix + "attn_norm"), self.cfg.rms_eps))
        k = (xn @ self.w(prefix + "wk")).reshape(-1, self.H, self.hd)
        v = (xn @ self.w(prefix + "wv")).reshape(-1, self.H, self.hd)
        return xn, self.st(self.rope(k, pos)), self.st(v)

    def block(self, prefix: str, x: np.ndarray, pos: np.ndarray,
              k_past: np.ndarray, v_past: np.ndarray, visible: np.ndarray):
        """One decoder block over M new rows.  x [M, d] residual; keys are the
        P past entries followed by the M new rows; visible [M, P + M].
        Returns (x_out, k_new, v_new)."""
        xn, k, v = self.block_kv(prefix, x, pos)
        q = self.st(self.rope((xn @ self.w(prefix + "wq")).reshape(-1, self.H, self.hd), pos))
        kk = np.concatenate([k_past, k], axis=0)
        vv = np.concatenate([v_past, v], axis=0)
        o = self.st(masked_attention(q, kk, vv, visible)).reshape(-1, self.H * self.hd)
        x = x + o @ self.w(prefix + "wo")
        xn2 = self.st(rms_norm(x, self.w(prefix + "ffn_norm"), self.cfg.rms_eps))
        g = xn2 @ self.w(prefix + "w_gate")
        u = xn2 @ self.w(prefix + "w_up")
        f = self.st(silu(g) * u)
        x = x + f @ self.w(prefix + "w_down")
        return x, k, v

    # -- target (Eq. 1) ------------------------------------------------------
    def target_rows(self, tokens, pos, past: List[Tuple[np.ndarray, np.ndarray]],
                    visible: np.ndarray):
        """Target forward over new rows ``tokens`` at ``pos`` given per-layer
        past K/V and the visibility mask [M, P + M].  Returns
        (logits [M, V], h^LLM [M, d] (post-final-norm, stored), new K/V)."""
        x = self.embed(tokens).astype(self.ct)
        pos = np.asarray(pos, dtype=np.int64)
        new_kv = []
        for l in range(self.cfg.n_layers):
            kp, vp = past[l]
            x, k, v = self.block(f"layers.{l}.", x, pos, kp, vp, visible)
            new_kv.append((k, v))
        h = self.st(rms_norm(x, self.w("final_norm"), self.cfg.rms_eps))
        logits = h @ self.w("lm_head")
        return logits, h, new_kv

    def empty_past(self):
        z = np.zeros((0, self.H, self.hd), dtype=self.ct)
        return [(z, z) for _ in range(self.cfg.n_layers)]

    def causal_forward(self, tokens: Sequence[int]):
        """Plain causal forward over a whole sequence (no cache): the
        definition the tree pass must reproduce."""
        n = len(tokens)
        vis = np.tril(np.ones((n, n), dtype=bool))
        return self.target_rows(tokens, np.arange(n), self.empty_past(), vis)

    def greedy_ar(self, prompt: Sequence[int], n_new: int) -> List[int]:
        """Greedy autoregressive decoding x_{t+1} = argmax M(x | x_<=t)
        (Eq. 1 with the argmax choice), recomputed from scratch per token."""
        seq = list(int(t) for t in prompt)
        out = []
        for _ in range(n_new):
            logits, _, _ = self.causal_forward(seq)
            nxt = argmax_lowest(logits[-1])
            out.append(nxt)
            seq.append(nxt)
        return out

    # -- draft: trigram encoder (Eq. 2) --------------------------------------
    def trigram_inputs(self, seq: Sequence[int], js: Sequence[int]) -> np.ndarray:
        """t_j = [x_{j-2}; x_{j-1}; x_j] (embeddings), with zero vectors
        standing in for positions before the sequence start."""
        E = self.w("tok_embed")
        out = np.zeros((len(js), 3 * self.d), dtype=self.ct)
        for r, j in enumerate(js):
            for s, i in enumerate((j - 2, j - 1, j)):
                if i >= 0:
                    out[r, s * self.d:(s + 1) * self.d] = E[seq[i]]
        return out

    def trigram_encode(self, t: np.ndarray) -> np.ndarray:
        """h^tri = MLP(SiLU(MLP(t))) with W_1 in R^{3d x d}, W_2 in R^{d x d}."""
        a = self.st(silu(self.st(t) @ self.w("draft.tri_w1")))
        return a @ self.w("draft.tri_w2")

    # -- draft: full-context encoder (Eq. 3) ---------------------------------
    def encoder_kv(self, u: np.ndarray, pos: np.ndarray):
        """K/V that the encoder block derives from entries u [M, d]."""
        _, k, v = self.block_kv("draft.enc.", u.astype(self.ct), np.asarray(pos))
        return k, v

    def encoder_query(self, u: np.ndarray, pos: int, k_mem: np.ndarray, v_mem: np.ndarray):
        """Output of the encoder block for one query entry u [d] at ``pos``
        attending to the memory k_mem/v_mem [P, H, hd] (which must already
        hold the query's own K/V).  Returns h^full [d]."""
        x = u.astype(self.ct)[None, :]
        p = np.array([pos])
        pre = "draft.enc."
        xn = self.st(rms_norm(x, self.w(pre + "attn_norm"), self.cfg.rms_eps))
        q = self.st(self.rope((xn @ self.w(pre + "wq")).reshape(1, self.H, self.hd), p))
        vis = np.ones((1, k_mem.shape[0]), dtype=bool)
        o = self.st(masked_attention(q, k_mem, v_mem, vis)).reshape(1, -1)
        y = x + o @ self.w(pre + "wo")
        yn = self.st(rms_norm(y, self.w(pre + "ffn_norm"), self.cfg.rms_eps))
        f = self.st(silu(yn @ self.w(pre + "w_gate")) * (yn @ self.w(pre + "w_up")))
        return (y + f @ self.w(pre + "w_down"))[0]

    # -- draft: residual decoding heads (Eq. 4) ------------------------------
    def head_logits(self, k: int, h_llm: np.ndarray, h_full: np.ndarray) -> np.ndarray:
        """Logits of head k: Theta_k^T SiLU(A_k^T [h^LLM_n; h^full_{n+1+k}]).
        Softmax is monotone, so selection works on these logits."""
        z = np.concatenate([self.st(h_llm), self.st(h_full)])
        a = self.st(silu(z @ self.w(f"draft.heads.{k}.a")))
        return a @ self.w(f"draft.heads.{k}.theta")


# ---------------------------------------------------------------------------
# Decoding state machine (prefill, draft, verify, accept, commit)
# ---------------------------------------------------------------------------


class Forcing:
    """Forced-acceptance bias: at draft level k the predicted position is
    j = n + 1 + k.  If ok[j], the level list becomes [g_j] + the top-(s-1)
    of the rest; otherwise the top-s excluding g_j.  ``g`` and ``ok`` are
    indexed by absolute position; a negative g_j means no reference there
    (plain top-s)."""

    def __init__(self, g: np.ndarray, ok: np.ndarray):
        self.g = np.asarray(g)
        self.ok = np.asarray(ok)


class Decoder:
    """One sequence decoded with Chimera's draft-then-verify loop (Sec. 3.1,
    Sec. 4.3, Sec. 4.4).  With an empty tree (root only) the step is plain
    greedy autoregressive decoding through the same cache path."""

    def __init__(self, oracle: Oracle, tree_ranks: Sequence[Tuple[int, ...]],
                 forcing: Optional[Forcing] = None, typical: Optional[Typical] = None,
                 branch: bool = False):
        self.o = oracle
        self.tree = Tree(tree_ranks)
        self.K = self.tree.levels if self.tree.n > 1 else 0
        if self.K > oracle.cfg.n_draft_heads:
            raise ValueError("tree deeper than the number of draft heads")
        self.s = [1] * self.K
        for r in self.tree.ranks[1:]:
            self.s[len(r) - 1] = max(self.s[len(r) - 1], r[-1] + 1)
        self.forcing = forcing
        self.typical = typical
        self.branch = branch
        # branch-conditioned drafting: the nodes drafted at level k are the
        # depth-k nodes with children, in node order
        t = self.tree
        self.drafted = [[u for u in range(t.n) if t.depth[u] == k and u in t.parent] for k in range(self.K)]

    # -- state -----------------------------------------------------------
    def prefill(self, prompt: Sequence[int]) -> int:
        """Run the target over the prompt, fill the target KV and the draft's
        encoder memory, and return the first generated token."""
        o = self.o
        self.seq: List[int] = [int(t) for t in prompt]
        n = len(self.seq)
        logits, h, kv = o.causal_forward(self.seq)
        self.kv = [(k.copy(), v.copy()) for k, v in kv]  # target K/V, positions 0..n-1
        self.n = n
        if self.typical is not None:
            ty = self.typical
            self.pending = gumbel_sample(np.asarray(logits[-1], dtype=np.float64) / ty.T, ty.seed, 0, n)
        else:
            self.pending = argmax_lowest(logits[-1])
        self.seq.append(self.pending)
        self.h_last = h[-1].copy()
        # draft encoder memory: target-state entries 0..n-1, trigram entries 0..n-1
        pos = np.arange(n)
        self.llm_k, self.llm_v = o.encoder_kv(h, pos)
        htri = o.trigram_encode(o.trigram_inputs(self.seq, list(range(n))))
        self.tri_k, self.tri_v = o.encoder_kv(htri, pos)
        return self.pending

    # -- draft (Sec. 4.1, Sec. 4.4) ----------------------------------------
    def draft(self, chain_tokens: Optional[Sequence[int]] = None):
        """Chain drafting: K sequential encoder queries along the rank-0
        chain.  Returns (level lists [K][s_k], per-head logits [K, V]).
        ``chain_tokens`` (teacher forcing) replaces each level's rank-0 token
        as the next chain token, e.g. by another run's choice at a tie."""
        o, n = self.o, self.n
        chain = list(self.seq[: n + 1])  # committed tokens and the pending one
        tri_k, tri_v = self.tri_k, self.tri_v
        lists, all_logits = [], []
        for k in range(self.K):
            j = n + k
            t = o.trigram_inputs(chain, [j])
            htri = o.trigram_encode(t)
            kj, vj = o.encoder_kv(htri, np.array([j]))
            tri_k = np.concatenate([tri_k[:j], kj], axis=0)
            tri_v = np.concatenate([tri_v[:j], vj], axis=0)
            k_mem = np.concatenate([self.llm_k[:n], tri_k[: j + 1]], axis=0)
            v_mem = np.concatenate([self.llm_v[:n], tri_v[: j + 1]], axis=0)
            hfull = o.encoder_query(htri[0], j, k_mem, v_mem)
            z = o.head_logits(k, self.h_last, hfull)
            all_logits.append(z)
            lst = self._select(z, self.s[k], n + 1 + k)
            lists.append(lst)
            chain.append(lst[0] if chain_tokens is None else int(chain_tokens[k]))
        return lists, (np.stack(all_logits) if all_logits else np.zeros((0, o.cfg.vocab)))

    def draft_branches(self, tree_tokens: Optional[Sequence[int]] = None):
        """Branch-conditioned drafting.  Level k runs the draft for every
        depth-k node u with children: the trigram at position n+k is built
        from u's own path tokens, its encoder query attends to the target
        entries 0..n-1, the trigram entries 0..n-1 and the trigram entries of
        u's ancestors-or-self (root first), and head k's top-s list becomes
        the candidates of u's children.  Returns ({u: list}, {u: logits}).
        ``tree_tokens`` (teacher forcing) supplies the path tokens instead of
        the lists, e.g. another run's tree."""
        o, n, t = self.o, self.n, self.tree
        forced_path = tree_tokens is not None
        toks = [int(x) for x in tree_tokens] if forced_path else [self.pending] + [-1] * (t.n - 1)
        ent_k, ent_v = {}, {}
        lists, all_logits = {}, {}
        for k in range(self.K):
            j = n + k
            for u in self.drafted[k]:
                path = t.anc[u]
                seq = list(self.seq[: n + 1]) + [toks[a] for a in path[1:]]
                htri = o.trigram_encode(o.trigram_inputs(seq, [j]))
                kj, vj = o.encoder_kv(htri, np.array([j]))
                ent_k[u], ent_v[u] = kj[0], vj[0]
                k_mem = np.concatenate([self.llm_k[:n], self.tri_k[:n], np.stack([ent_k[a] for a in path])])
                v_mem = np.concatenate([self.llm_v[:n], self.tri_v[:n], np.stack([ent_v[a] for a in path])])
                hfull = o.encoder_query(htri[0], j, k_mem, v_mem)
                z = o.head_logits(k, self.h_last, hfull)
                lists[u] = self._select(z, self.s[k], n + 1 + k)
                all_logits[u] = z
            if not forced_path:
                for v in range(t.n):
                    if t.depth[v] == k + 1:
                        toks[v] = int(lists[t.parent[v]][t.ranks[v][-1]])
        return lists, all_logits

    def _select(self, z: np.ndarray, s: int, j: int) -> List[int]:
        f = self.forcing
        if f is None:
            return top_s(z, s)
        gj = int(f.g[j])
        if gj < 0 or gj >= z.shape[0]:
            return top_s(z, s)  # no reference token at this position: no bias
        if f.ok[j]:
            return [gj] + top_s(z, s - 1, exclude=gj)
        return top_s(z, s, exclude=gj)

    def assemble(self, lists) -> List[int]:
        """Tree tokens: root = pending; node (r_0..r_k) = lists[k][r_k] for
        chain drafting, or the rank-r_k token of its parent's own list for
        branch-conditioned drafting."""
        t = self.tree
        toks = [self.pending]
        for u in range(1, t.n):
            r = t.ranks[u]
            src = lists[t.parent[u]] if self.branch else lists[len(r) - 1]
            toks.append(int(src[r[-1]]))
        return toks

    # -- verify (Sec. 4.3) ------------------------------------------------
    def verify(self, tree_tokens: Sequence[int]):
        """One target pass over all tree nodes: node u sits at position
        n + depth(u) and sees the whole committed cache plus its ancestors.
        Returns (logits [N, V], h^LLM [N, d], per-layer tree K/V)."""
        t, n = self.tree, self.n
        vis = np.concatenate([np.ones((t.n, n), dtype=bool), t.mask()], axis=1)
        pos = n + np.asarray(t.depth)
        return self.o.target_rows(tree_tokens, pos, self.kv, vis)

    def brute_force_node_logits(self, tree_tokens: Sequence[int], u: int) -> np.ndarray:
        """Logits of node u from a plain causal forward over the committed
        tokens followed by the root-to-u path (no tree mask, no cache)."""
        path = [tree_tokens[a] for a in self.tree.anc[u]]
        logits, _, _ = self.o.causal_forward(self.seq[: self.n] + path)
        return logits[-1]

    # -- accept (Sec. 4.3 greedy; Sec. 4.4) ---------------------------------
    def accept(self, tree_tokens: Sequence[int], amax: Sequence[int]):
        """Longest root-to-node path whose every non-root token equals the
        target argmax at its parent.  Returns (path node ids, bonus token)."""
        t = self.tree
        good = [u == 0 or tree_tokens[u] == amax[t.parent[u]] for u in range(t.n)]
        best = 0
        for u in range(t.n):
            if all(good[a] for a in t.anc[u]) and t.depth[u] > t.depth[best]:
                best = u
        return list(t.anc[best]), int(amax[best])

    # -- commit ------------------------------------------------------------
    def commit(self, path: Sequence[int], bonus: int, tree_tokens, h_tree, tree_kv):
        """Append the accepted path's keys/values at positions n..n+L-1,
        extend the encoder memory, and advance to the bonus token."""
        o, n, L = self.o, self.n, len(path)
        idx = np.asarray(path)
        self.kv = [(np.concatenate([k[:n], kt[idx]]), np.concatenate([v[:n], vt[idx]]))
                   for (k, v), (kt, vt) in zip(self.kv, tree_kv)]
        self.seq = self.seq[: n + 1] + [int(tree_tokens[u]) for u in path[1:]]
        self.seq.append(int(bonus))
        pos = np.arange(n, n + L)
        hk, hv = o.encoder_kv(h_tree[idx], pos)
        self.llm_k = np.concatenate([self.llm_k[:n], hk])
        self.llm_v = np.concatenate([self.llm_v[:n], hv])
        htri = o.trigram_encode(o.trigram_inputs(self.seq, list(range(n, n + L))))
        tk, tv = o.encoder_kv(htri, pos)
        self.tri_k = np.concatenate([self.tri_k[:n], tk])
        self.tri_v = np.concatenate([self.tri_v[:n], tv])
        self.h_last = h_tree[path[-1]].copy()
        self.n = n + L
        self.pending = int(bonus)

    def step(self, tree_tokens_override: Optional[Sequence[int]] = None,
             accept_override: Optional[Sequence[int]] = None) -> dict:
        """One draft -> verify -> accept -> commit iteration.  Returns the
        newly generated tokens (accepted draft tokens then the bonus) and
        the step's artefacts.  The overrides let a test drive the oracle
        along another run's tree tokens or accepted path."""
        if not self.K:
            lists, dlogits = [], None
        elif self.branch:
            lists, dlogits = self.draft_branches()
        else:
            lists, dlogits = self.draft()
        toks = self.assemble(lists) if tree_tokens_override is None else list(tree_tokens_override)
        logits, h, tkv = self.verify(toks)
        amax = [argmax_lowest(r) for r in logits]
        if self.typical is not None:
            path, bonus, _, _ = typical_accept(self.tree, toks, logits, self.typical, self.n)
        else:
            path, bonus = self.accept(toks, amax)
        if accept_override is not None:
            path = list(accept_override)
            bonus = amax[path[-1]]
        art = dict(n=self.n, lists=lists, draft_logits=dlogits, tree_tokens=toks,
                   logits=logits, argmax=amax, path=path, bonus=bonus,
                   new_tokens=[toks[u] for u in path[1:]] + [bonus])
        self.commit(path, bonus, toks, h, tkv)
        return art

    def generate(self, prompt: Sequence[int], n_new: int):
        """Generate n_new tokens: the prefill's token, then draft/verify steps
        until enough are committed; the last step's excess is dropped."""
        out = [self.prefill(prompt)]
        steps = []
        while len(out) < n_new:
            a = self.step()
            steps.append(a)
            out += a["new_tokens"]
        return out[:n_new], steps
