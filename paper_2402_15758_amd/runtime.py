"""A decode session on one GPU: model, paged KV and decode context created
through the C ABI, with every arena allocated by torch on the device and
every launch on torch's current stream.  The loop around chimera_step is
plain orchestration; all of the step's work runs in the library's kernels."""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import binding as B


def tree_arrays(ranks: Sequence[Sequence[int]]) -> Tuple[np.ndarray, np.ndarray]:
    """(parent, rank) arrays of a tree given by rank tuples (root excluded,
    ordered by depth): node i >= 1 is ranks[i-1]; its parent is the node of
    the tuple without its last rank."""
    nodes = [()] + [tuple(r) for r in ranks]
    index = {r: i for i, r in enumerate(nodes)}
    parent = np.array([-1] + [index[r[:-1]] for r in nodes[1:]], dtype=np.int32)
    rank = np.array([0] + [r[-1] for r in nodes[1:]], dtype=np.int32)
    return parent, rank


class Session:
    """Chimera decode state for up to ``max_batch`` sequences.

    ``cfg`` provides n_layers, d_model, n_heads, head_dim, d_ffn, vocab,
    n_draft_heads, rope_base, rms_eps and dtype ("f32" | "bf16");
    ``weights`` maps the canonical tensor names to torch tensors."""

    def __init__(self, cfg, weights: Optional[Dict[str, "object"]], tree_ranks, max_batch: int = 1,
                 max_len: int = 1024, page_size: int = 16, page_order: Optional[np.ndarray] = None,
                 device: str = "cuda", share_model: Optional["Session"] = None):
        import torch

        self.torch = torch
        self.device = torch.device(device)
        self.cfg = cfg
        self.dt = B.CHIMERA_BF16 if cfg.dtype == "bf16" else B.CHIMERA_F32
        self.max_batch, self.max_len = max_batch, max_len
        c = B.chimera_config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ffn, cfg.vocab,
                             cfg.n_draft_heads, float(cfg.rope_base), float(cfg.rms_eps), self.dt, max_len + 128)
        self._c = c
        self._owner = share_model is None
        if share_model is not None:
            # another decode state over the same loaded weights
            if share_model.cfg != cfg or share_model.max_len < max_len:
                raise ValueError("shared model has another config or a shorter rotary table")
            self.w_arena, self.model = share_model.w_arena, share_model.model
            self._c = share_model._c
        else:
            wb = B.chimera_weight_bytes(c)
            self.w_arena = torch.empty(wb, dtype=torch.uint8, device=self.device)
            names, tensors = [], []
            for name, t in weights.items():
                # the library reads device memory only
                t = t.to(self.device).contiguous()
                nb = name.encode()
                names.append((nb, t))
                dt = B.CHIMERA_F32 if t.dtype == torch.float32 else B.CHIMERA_BF16
                tensors.append(B.chimera_tensor(nb, t.data_ptr(), t.numel(), dt, 1 if t.is_cuda else 0))
            self.model = B.chimera_load(c, tensors, self.w_arena.data_ptr(), wb, self.stream())
            del names, tensors
        self.page_size = page_size
        self.n_pages = max_batch * math.ceil((max_len + 64) / page_size)
        if page_order is not None:
            page_order = np.ascontiguousarray(page_order, dtype=np.int32)
        kb = B.chimera_kv_bytes(self.model, max_batch, max_len, self.n_pages, page_size)
        self.kv_arena = torch.empty(kb, dtype=torch.uint8, device=self.device)
        self.kv = B.chimera_kv_create(self.model, max_batch, max_len, self.n_pages, page_size, page_order,
                                      self.kv_arena.data_ptr(), kb)
        parent, rank = tree_arrays(tree_ranks)
        self.n_nodes = len(parent)
        self.K = max((len(r) for r in tree_ranks), default=0)
        cb = B.chimera_ctx_bytes(self.model, self.kv, self.n_nodes)
        self.ctx_arena = torch.empty(cb, dtype=torch.uint8, device=self.device)
        self.ctx = B.chimera_ctx_create(self.model, self.kv, parent, rank, self.ctx_arena.data_ptr(), cb)
        self.batch = 0
        self._forcing = None

    def stream(self) -> int:
        return self.torch.cuda.current_stream(self.device).cuda_stream

    # -- decoding ----------------------------------------------------------
    def prefill(self, prompts: List[np.ndarray]) -> np.ndarray:
        lens = np.array([len(p) for p in prompts], dtype=np.int32)
        toks = np.ascontiguousarray(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts]))
        first = np.zeros(len(prompts), dtype=np.int32)
        B.chimera_prefill(self.model, self.kv, self.ctx, toks, lens, first, self.stream())
        self.batch = len(prompts)
        return first

    def step(self):
        K1 = self.K + 1
        toks = np.zeros((self.batch, K1), dtype=np.int32)
        n = np.zeros(self.batch, dtype=np.int32)
        path = np.zeros((self.batch, K1), dtype=np.int32)
        B.chimera_step(self.model, self.kv, self.ctx, toks, n, path, self.stream())
        return toks, n, path

    def steps(self, n: int):
        """n pipelined steps (chimera_steps, at most CHIMERA_MAX_PIPELINED_STEPS
        per call): arrays [n][batch][K+1], [n][batch], [n][batch][K+1]."""
        K1 = self.K + 1
        toks = np.zeros((n, self.batch, K1), dtype=np.int32)
        nn = np.zeros((n, self.batch), dtype=np.int32)
        path = np.zeros((n, self.batch, K1), dtype=np.int32)
        B.chimera_steps(self.model, self.kv, self.ctx, n, toks, nn, path, self.stream())
        return toks, nn, path

    def generate(self, prompts: List[np.ndarray], n_new: int):
        """Prefill, then step until every sequence has n_new tokens; returns
        (per-sequence token lists truncated to n_new, per-step records)."""
        first = self.prefill(prompts)
        out = [[int(t)] for t in first]
        steps = []
        while min(len(o) for o in out) < n_new:
            toks, n, path = self.step()
            steps.append((toks.copy(), n.copy(), path.copy()))
            for b in range(self.batch):
                out[b] += [int(t) for t in toks[b, : n[b]]]
        return [o[:n_new] for o in out], steps

    def set_forcing(self, ref, ok):
        """ref: int32 [batch][stride], ok: uint8 [batch][stride] device
        tensors (kept alive here); None disables forcing."""
        if ref is None:
            B.chimera_set_forcing(self.ctx, None, None, 0)
            self._forcing = None
            return
        assert ref.is_cuda and ok.is_cuda and ref.dtype == self.torch.int32 and ok.dtype == self.torch.uint8
        ref, ok = ref.contiguous(), ok.contiguous()
        self._forcing = (ref, ok)
        B.chimera_set_forcing(self.ctx, ref.data_ptr(), ok.data_ptr(), ref.shape[1])

    def set_tree_tokens(self, tokens: np.ndarray):
        B.chimera_set_tree_tokens(self.ctx, np.ascontiguousarray(tokens, dtype=np.int32), self.batch)

    # -- inspection -------------------------------------------------------
    def debug(self, what: int) -> np.ndarray:
        Bn, N, K, V = max(self.batch, 1), self.n_nodes, self.K, self.cfg.vocab
        shapes = {
            B.DBG_VERIFY_LOGITS: ((Bn * N, V), np.float32),
            B.DBG_DRAFT_LOGITS: ((Bn, K, V), np.float32),
            B.DBG_TREE_TOKENS: ((Bn, N), np.int32),
            B.DBG_DRAFT_LISTS: ((Bn, 64, 8), np.int32),
            B.DBG_SEQ_LEN: ((Bn,), np.int32),
            B.DBG_TOKENS: ((Bn, self.max_len + 8), np.int32),
        }
        shape, dt = shapes[what]
        out = np.zeros(shape, dtype=dt)
        B.chimera_debug_copy(self.ctx, what, out.ctypes.data, out.nbytes)
        return out

    def kv_read(self, layer: int, b: int, pos0: int, count: int):
        """Target K and V at positions pos0..pos0+count-1 of sequence b:
        float32 arrays, or uint16 bf16 bit patterns for bf16 models."""
        dt = np.uint16 if self.dt == B.CHIMERA_BF16 else np.float32
        shape = (count, self.cfg.n_heads, self.cfg.head_dim)
        k = np.zeros(shape, dtype=dt)
        v = np.zeros(shape, dtype=dt)
        B.chimera_kv_read(self.kv, layer, b, pos0, count, k.ctypes.data, v.ctypes.data)
        return k, v

    def set_graph(self, enable: bool):
        B.chimera_set_graph(self.ctx, enable)

    def set_drafting(self, branch: bool):
        """Chain drafting (branch=False) or branch-conditioned drafting."""
        B.chimera_set_drafting(self.ctx, B.CHIMERA_DRAFT_BRANCH if branch else B.CHIMERA_DRAFT_CHAIN)

    def set_decoding(self, typical: bool, temperature: float = 1.0, eps: float = 0.09, delta: float = 0.3,
                     seed: int = 0):
        """Greedy verification (typical=False) or typical acceptance with sampling."""
        B.chimera_set_decoding(self.ctx, B.CHIMERA_DECODE_TYPICAL if typical else B.CHIMERA_DECODE_GREEDY,
                               temperature, eps, delta, seed)

    def trigram_cache(self, n_entries: int):
        """Attach an empty trigram lookup cache of n_entries outputs (0 detaches)."""
        import torch
        if not n_entries:
            B.chimera_set_trigram_cache(self.ctx, None, 0, 0)
            self.tri_arena = None
            return
        nb = B.chimera_trigram_cache_bytes(self.model, n_entries)
        self.tri_arena = torch.empty(nb + 256, dtype=torch.uint8, device=self.device)
        base = (self.tri_arena.data_ptr() + 255) // 256 * 256
        B.chimera_set_trigram_cache(self.ctx, base, nb, n_entries)

    def trigram_stats(self):
        """(lookups, hits) of draft-level trigram rows since the cache was attached."""
        return B.chimera_trigram_cache_stats(self.ctx)

    def compaction_check(self, enable: bool):
        """Attach (or detach) the compaction check's side arena: every step then
        copies the tree's K/V rows before compaction and compares the accepted
        path's slots with them after it."""
        import torch
        if not enable:
            B.chimera_set_compaction_check(self.ctx, None, 0)
            self.cc_arena = None
            return
        nb = B.chimera_compaction_check_bytes(self.ctx)
        self.cc_arena = torch.empty(nb + 256, dtype=torch.uint8, device=self.device)
        base = (self.cc_arena.data_ptr() + 255) // 256 * 256
        B.chimera_set_compaction_check(self.ctx, base, nb)

    def compaction_check_read(self):
        """(rows compared, 16-byte chunks that differed) since the check was attached."""
        return B.chimera_compaction_check_read(self.ctx)

    def profile(self, enable: bool):
        B.chimera_profile_enable(self.ctx, enable)

    def profile_read(self):
        return B.chimera_profile_read(self.ctx)

    def close(self):
        if getattr(self, "ctx", None):
            B.chimera_set_trigram_cache(self.ctx, None, 0, 0)
            B.chimera_set_compaction_check(self.ctx, None, 0)
            B.chimera_ctx_free(self.ctx)
            self.ctx = None
        if getattr(self, "kv", None):
            B.chimera_kv_free(self.kv)
            self.kv = None
        if getattr(self, "model", None):
            if self._owner:
                B.chimera_free(self.model)
            self.model = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
