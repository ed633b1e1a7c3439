"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a library
implementation of the same block (Hugging Face's Llama, torch's attention),
a closed form, an invariant, brute force on tiny inputs, or the lossless
property (speculative output == greedy autoregressive output).
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import chimera_oracle as co

CFG = synth.TINY


def tiny_oracle(std=0.06, seed=0, cfg=CFG, compute=np.float64):
    w = synth.weights_to_numpy(synth.make_weights(cfg, target_seed=seed, draft_seed=seed + 1, std=std))
    return oracle.Oracle(cfg, w, compute=compute)


@pytest.fixture(scope="module")
def orc():
    return tiny_oracle()


@pytest.fixture(scope="module")
def orc_exact():
    """The tiny workload's own weights (std 0.02)."""
    return tiny_oracle(std=0.02)


# ---------------------------------------------------------------------------
# Elementary closed forms
# ---------------------------------------------------------------------------


def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-8, 8, 20000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.005859375, 65504.0, 1e-40]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = co.round_bf16(x)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_rms_norm_closed_form():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 256)) * 3.0
    y = co.rms_norm(x, np.ones(256), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-12)
    # a constant row c maps to sign(c) * gain / sqrt(1 + eps / c^2)
    c = np.full((1, 8), -2.0)
    np.testing.assert_allclose(co.rms_norm(c, np.arange(8.0), 1e-5)[0], -np.arange(8.0) / np.sqrt(1 + 1e-5 / 4))


def test_silu_closed_form():
    x = np.linspace(-20, 20, 401)
    s = co.silu(x)
    np.testing.assert_allclose(s - co.silu(-x), x, atol=1e-12)  # x*sig(x) - (-x)*sig(-x) = x
    assert co.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(s, torch.nn.functional.silu(torch.from_numpy(x)).numpy(), rtol=1e-14)


def test_rope_preserves_norm_and_is_relative():
    rng = np.random.default_rng(2)
    hd = 64
    q = rng.standard_normal((1, 1, hd))
    k = rng.standard_normal((1, 1, hd))
    def rot(x, p):
        c, s = co.rope_cos_sin(np.array([p]), hd, 10000.0)
        return co.apply_rope(x, c.astype(np.float64), s.astype(np.float64))
    for p in (0, 1, 17, 4095):
        np.testing.assert_allclose(np.linalg.norm(rot(q, p)), np.linalg.norm(q), rtol=1e-6)
    # <R(m) q, R(n) k> depends only on m - n (up to the float32 tables)
    d1 = np.sum(rot(q, 100) * rot(k, 90))
    d2 = np.sum(rot(q, 1010) * rot(k, 1000))
    np.testing.assert_allclose(d1, d2, rtol=1e-4)
    # position 0 is the identity
    np.testing.assert_array_equal(rot(q, 0), q)


def test_softmax_and_attention_vs_torch_sdpa():
    rng = np.random.default_rng(3)
    M, P, H, hd = 5, 11, 3, 16
    q, k, v = (rng.standard_normal((M, H, hd)), rng.standard_normal((P, H, hd)), rng.standard_normal((P, H, hd)))
    vis = rng.random((M, P)) < 0.6
    vis[:, 0] = True
    got = co.masked_attention(q, k, v, vis)
    tq, tk, tv = (torch.from_numpy(a).permute(1, 0, 2) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=torch.from_numpy(vis))
    np.testing.assert_allclose(got, ref.permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(co.softmax_rows(rng.standard_normal((4, 9))).sum(-1), 1.0, rtol=1e-14)


def test_argmax_and_top_s_tie_rules():
    z = np.array([1.0, 3.0, 3.0, 2.0, 3.0, -1.0])
    assert co.argmax_lowest(z) == 1
    assert co.top_s(z, 4) == [1, 2, 4, 3]
    assert co.top_s(z, 3, exclude=2) == [1, 4, 3]
    rng = np.random.default_rng(4)
    r = rng.standard_normal(1000)
    assert co.top_s(r, 5) == [int(i) for i in np.argsort(-r)[:5]]


# ---------------------------------------------------------------------------
# Target decoder vs an independent library implementation (Hugging Face Llama)
# ---------------------------------------------------------------------------


def hf_llama(orc_):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = orc_.cfg
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_heads, head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps,
                     rope_theta=cfg.rope_base, max_position_embeddings=4096, tie_word_embeddings=False,
                     attention_bias=False, mlp_bias=False)
    m = LlamaForCausalLM(hc).double().eval()
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a.T))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(torch.from_numpy(orc_.w("tok_embed")))
        for l in range(cfg.n_layers):
            L = m.model.layers[l]
            p = f"layers.{l}."
            L.self_attn.q_proj.weight.copy_(T(orc_.w(p + "wq")))
            L.self_attn.k_proj.weight.copy_(T(orc_.w(p + "wk")))
            L.self_attn.v_proj.weight.copy_(T(orc_.w(p + "wv")))
            L.self_attn.o_proj.weight.copy_(T(orc_.w(p + "wo")))
            L.mlp.gate_proj.weight.copy_(T(orc_.w(p + "w_gate")))
            L.mlp.up_proj.weight.copy_(T(orc_.w(p + "w_up")))
            L.mlp.down_proj.weight.copy_(T(orc_.w(p + "w_down")))
            L.input_layernorm.weight.copy_(torch.from_numpy(orc_.w(p + "attn_norm")))
            L.post_attention_layernorm.weight.copy_(torch.from_numpy(orc_.w(p + "ffn_norm")))
        m.model.norm.weight.copy_(torch.from_numpy(orc_.w("final_norm")))
        m.lm_head.weight.copy_(T(orc_.w("lm_head")))
    return m


def test_target_matches_hf_llama(orc):
    m = hf_llama(orc)
    toks = synth.make_prompt(40, CFG.vocab, 7)
    logits, _, _ = orc.causal_forward(list(toks))
    with torch.no_grad():
        ref = m(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].numpy()
    rng_ = ref.max(-1) - ref.min(-1)
    # HF's RMSNorm computes in float32; everything else is float64
    assert np.max(np.abs(logits - ref) / rng_[:, None]) < 1e-5


def test_encoder_block_matches_hf_decoder_layer(orc):
    """The full-context encoder (Eq. 3) is one Transformer block over
    [H^LLM; H^tri] whose entries carry their sequence positions; the query at
    trigram position j sees everything.  A one-layer HF Llama run on the
    concatenated inputs with those position ids and a causal mask gives the
    same last row."""
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer, LlamaRotaryEmbedding
    cfg = orc.cfg
    rng = np.random.default_rng(5)
    n, j = 9, 11
    h_llm = rng.standard_normal((n, cfg.d_model))
    h_tri = rng.standard_normal((j + 1, cfg.d_model))
    pos = np.concatenate([np.arange(n), np.arange(j + 1)])
    lk, lv = orc.encoder_kv(h_llm, np.arange(n))
    tk, tv = orc.encoder_kv(h_tri, np.arange(j + 1))
    got = orc.encoder_query(h_tri[-1], j, np.concatenate([lk, tk]), np.concatenate([lv, tv]))

    hc = LlamaConfig(hidden_size=cfg.d_model, intermediate_size=cfg.d_ffn, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_heads, head_dim=cfg.head_dim, rms_norm_eps=cfg.rms_eps,
                     rope_theta=cfg.rope_base, max_position_embeddings=4096)
    hc._attn_implementation = "eager"
    layer = LlamaDecoderLayer(hc, 0).double().eval()
    T = lambda a: torch.from_numpy(np.ascontiguousarray(orc.w("draft.enc." + a).T))
    with torch.no_grad():
        layer.self_attn.q_proj.weight.copy_(T("wq"))
        layer.self_attn.k_proj.weight.copy_(T("wk"))
        layer.self_attn.v_proj.weight.copy_(T("wv"))
        layer.self_attn.o_proj.weight.copy_(T("wo"))
        layer.mlp.gate_proj.weight.copy_(T("w_gate"))
        layer.mlp.up_proj.weight.copy_(T("w_up"))
        layer.mlp.down_proj.weight.copy_(T("w_down"))
        x = torch.from_numpy(np.concatenate([h_llm, h_tri]))[None]
        pid = torch.from_numpy(pos)[None]
        cos, sin = LlamaRotaryEmbedding(hc)(x, pid)
        L = x.shape[1]
        mask = torch.full((L, L), float("-inf"), dtype=torch.float64).triu(1)[None, None]
        out = layer(x, attention_mask=mask, position_ids=pid, position_embeddings=(cos, sin))
        out = out[0] if isinstance(out, tuple) else out
    ref = out[0, -1].numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-6)


# ---------------------------------------------------------------------------
# Draft modules: special cases with closed forms
# ---------------------------------------------------------------------------


def test_trigram_zero_padding_and_locality(orc):
    seq = list(synth.make_prompt(12, CFG.vocab, 8))
    t = orc.trigram_inputs(seq, [0, 1, 2, 7])
    E, d = orc.w("tok_embed"), CFG.d_model
    np.testing.assert_array_equal(t[0], np.concatenate([np.zeros(d), np.zeros(d), E[seq[0]]]))
    np.testing.assert_array_equal(t[1], np.concatenate([np.zeros(d), E[seq[0]], E[seq[1]]]))
    np.testing.assert_array_equal(t[2], np.concatenate([E[seq[0]], E[seq[1]], E[seq[2]]]))
    # h^tri_j depends on tokens j-2..j only
    seq2 = list(seq)
    seq2[3] = (seq2[3] + 1) % CFG.vocab
    seq2[8] = (seq2[8] + 1) % CFG.vocab
    h1 = orc.trigram_encode(orc.trigram_inputs(seq, [7]))
    h2 = orc.trigram_encode(orc.trigram_inputs(seq2, [7]))
    np.testing.assert_array_equal(h1, h2)
    h3 = orc.trigram_encode(orc.trigram_inputs(seq2, [8]))
    assert not np.array_equal(orc.trigram_encode(orc.trigram_inputs(seq, [8])), h3)


def test_trigram_mlp_special_weights():
    """With W_1 = [0; 0; I] and W_2 = I the encoder returns SiLU(x_j): this
    fixes the block order of the concatenation and SiLU between the layers."""
    o = tiny_oracle()
    d = CFG.d_model
    w1 = np.zeros((3 * d, d))
    w1[2 * d:] = np.eye(d)
    o._cache["draft.tri_w1"] = w1
    o._cache["draft.tri_w2"] = np.eye(d)
    seq = [5, 9, 13]
    h = o.trigram_encode(o.trigram_inputs(seq, [2]))
    np.testing.assert_allclose(h[0], co.silu(o.w("tok_embed")[13]), rtol=1e-14)
    w1 = np.zeros((3 * d, d))
    w1[:d] = np.eye(d)
    o._cache["draft.tri_w1"] = w1
    h = o.trigram_encode(o.trigram_inputs(seq, [2]))
    np.testing.assert_allclose(h[0], co.silu(o.w("tok_embed")[5]), rtol=1e-14)


def test_head_special_weights_and_separation():
    """Head k is Theta_k(SiLU(A_k [h^LLM; h^full])): with A_k = [I; 0] it sees
    only h^LLM, with [0; I] only h^full; other heads' weights are unused."""
    o = tiny_oracle()
    d, V = CFG.d_model, CFG.vocab
    rng = np.random.default_rng(9)
    hl, hf = rng.standard_normal(d), rng.standard_normal(d)
    a = np.zeros((2 * d, d))
    a[:d] = np.eye(d)
    o._cache["draft.heads.1.a"] = a
    theta = o.w("draft.heads.1.theta")
    np.testing.assert_allclose(o.head_logits(1, hl, hf), co.silu(hl) @ theta, rtol=1e-12)
    a = np.zeros((2 * d, d))
    a[d:] = np.eye(d)
    o._cache["draft.heads.1.a"] = a
    np.testing.assert_allclose(o.head_logits(1, hl, hf), co.silu(hf) @ theta, rtol=1e-12)
    z0 = o.head_logits(0, hl, hf)
    o._cache["draft.heads.2.theta"] = theta * 7.0
    o._cache["draft.heads.1.a"] = a * 3.0
    np.testing.assert_array_equal(o.head_logits(0, hl, hf), z0)


def test_encoder_key_order_independence(orc):
    rng = np.random.default_rng(10)
    u = rng.standard_normal((14, CFG.d_model))
    k, v = orc.encoder_kv(u, np.arange(14))
    perm = rng.permutation(14)
    a = orc.encoder_query(u[-1], 13, k, v)
    b = orc.encoder_query(u[-1], 13, k[perm], v[perm])
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# Tree metadata
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("name", ["T8", "T32", "T64"])
def test_tree_mask_invariants(name):
    t = oracle.Tree(synth.TREES[name])
    m = t.mask()
    for u in range(t.n):
        assert m[u, u] and m[u, 0]
        assert m[u].sum() == t.depth[u] + 1
        if u:
            assert t.parent[u] < u
            assert np.all(m[u] >= m[t.parent[u]])  # anc(u) contains anc(parent)
    assert np.array_equal(m, np.tril(m))  # lower-triangular in node order
    for u, v in itertools.combinations(range(1, t.n), 2):
        if t.parent[u] == t.parent[v]:
            assert not m[u, v] and not m[v, u]  # siblings invisible to each other
    chain = oracle.Tree(synth.chain_tree(5))
    assert np.array_equal(chain.mask(), np.tril(np.ones((6, 6), dtype=bool)))


def test_trees_follow_table5_derivation():
    assert synth.derive_tree(8, 3) == synth.TREE_T8
    assert synth.derive_tree(32, 4) == synth.TREE_T32
    assert synth.derive_tree(64, 4) == synth.TREE_T64
    assert synth.tree_top_s(synth.TREE_T8, 3) == [3, 4, 1]
    assert synth.tree_top_s(synth.TREE_T64, 4) == [5, 5, 5, 5]


# ---------------------------------------------------------------------------
# Verify, accept, commit: brute force and the lossless property
# ---------------------------------------------------------------------------


def _state_after_steps(o, tree, n_steps=3, forcing=None, seed=11):
    dec = oracle.Decoder(o, tree, forcing)
    dec.prefill(list(synth.make_prompt(20, CFG.vocab, seed)))
    for _ in range(n_steps):
        dec.step()
    return dec


def test_tree_pass_equals_brute_force_per_node(orc):
    dec = _state_after_steps(orc, synth.TREE_T8)
    lists, _ = dec.draft()
    toks = dec.assemble(lists)
    logits, _, _ = dec.verify(toks)
    for u in range(dec.tree.n):
        ref = dec.brute_force_node_logits(toks, u)
        assert np.max(np.abs(logits[u] - ref)) <= 1e-12 * (ref.max() - ref.min())


def test_tree_pass_brute_force_random_tokens(orc):
    """Random (non-draft) tokens in a 32-node tree, after a ragged history."""
    dec = _state_after_steps(orc, synth.TREE_T32[:12], n_steps=2, seed=12)
    rng = np.random.default_rng(13)
    toks = [dec.pending] + list(rng.integers(0, CFG.vocab, dec.tree.n - 1))
    logits, _, _ = dec.verify(toks)
    for u in range(dec.tree.n):
        ref = dec.brute_force_node_logits(toks, u)
        assert np.max(np.abs(logits[u] - ref)) <= 1e-12 * (ref.max() - ref.min())


def test_accept_equals_brute_force_over_paths(orc):
    """Acceptance = the longest candidate sequence (root-to-node path) that
    greedy decoding itself would produce from the committed prefix."""
    t3 = tuple(r for r in synth.TREE_T32 if len(r) <= CFG.n_draft_heads)
    dec = _state_after_steps(orc, t3, n_steps=1)
    rng = np.random.default_rng(14)
    t = dec.tree
    for trial in range(30):
        amax = list(rng.integers(0, 4, t.n))
        toks = [dec.pending] + list(rng.integers(0, 4, t.n - 1))
        path, bonus = dec.accept(toks, amax)
        best = [0]
        for u in range(t.n):
            p = t.anc[u]
            if all(toks[p[i + 1]] == amax[p[i]] for i in range(len(p) - 1)) and len(p) > len(best):
                best = p
        assert path == best and bonus == amax[best[-1]]


def test_commit_equals_prefill_of_committed_tokens(orc):
    dec = _state_after_steps(orc, synth.TREE_T8, n_steps=4)
    _, _, kv = orc.causal_forward(dec.seq[: dec.n])
    for (k, v), (kr, vr) in zip(dec.kv, kv):
        np.testing.assert_allclose(k, kr, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(v, vr, rtol=1e-12, atol=1e-14)
    # the draft's encoder memory equals a fresh build from the committed stream
    logits, h, _ = orc.causal_forward(dec.seq[: dec.n])
    lk, lv = orc.encoder_kv(h, np.arange(dec.n))
    np.testing.assert_allclose(dec.llm_k, lk, rtol=1e-12, atol=1e-14)
    ht = orc.trigram_encode(orc.trigram_inputs(dec.seq, list(range(dec.n))))
    tk, tv = orc.encoder_kv(ht, np.arange(dec.n))
    np.testing.assert_allclose(dec.tri_v, tv, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dec.h_last, h[-1], rtol=1e-12, atol=1e-14)


def test_draft_chain_equals_fresh_encoder_runs(orc):
    """Head k's list comes from the encoder query at trigram position n+k
    along the rank-0 chain; recompute each from a fresh memory."""
    dec = _state_after_steps(orc, synth.TREE_T8, n_steps=2)
    lists, dl = dec.draft()
    n = dec.n
    chain = dec.seq[: n + 1] + [l[0] for l in lists]
    _, h, _ = orc.causal_forward(dec.seq[:n])
    for k in range(dec.K):
        j = n + k
        ht = orc.trigram_encode(orc.trigram_inputs(chain, list(range(j + 1))))
        lk, lv = orc.encoder_kv(h, np.arange(n))
        tk, tv = orc.encoder_kv(ht, np.arange(j + 1))
        hf = orc.encoder_query(ht[j], j, np.concatenate([lk, tk]), np.concatenate([lv, tv]))
        z = orc.head_logits(k, h[-1], hf)
        np.testing.assert_allclose(dl[k], z, rtol=1e-10, atol=1e-12)
        assert lists[k] == co.top_s(z, dec.s[k])


@pytest.mark.parametrize("std", [0.02, 0.06])
def test_lossless_unforced(std):
    o = tiny_oracle(std=std)
    prompt = list(synth.WORKLOADS["tiny"].prompts()[0])
    ar = o.greedy_ar(prompt, 40)
    out, steps = oracle.Decoder(o, synth.TREE_T8).generate(prompt, 40)
    assert out == ar


@pytest.mark.parametrize("p", [0.0, 0.7, 1.0])
def test_lossless_forced_and_acceptance_closed_form(orc, p):
    prompt = list(synth.WORKLOADS["tiny"].prompts()[0])
    G, n0 = 48, len(prompt)
    ar = orc.greedy_ar(prompt, G + 8)
    g = np.zeros(n0 + G + 8, dtype=np.int64)
    g[n0:] = ar
    ok = synth.force_table(p, 3, 0, n0 + G + 8)
    dec = oracle.Decoder(orc, synth.TREE_T8, oracle.Forcing(g, ok))
    out, steps = dec.generate(prompt, G)
    assert out == ar[:G]
    K = dec.K
    for a in steps:
        n = a["n"]
        run = 0
        while run < K and ok[n + 1 + run]:
            run += 1
        assert len(a["new_tokens"]) == 1 + run  # L = 1 + consecutive successes
        assert a["path"] == [0] + [dec.tree.ranks.index((0,) * d) for d in range(1, run + 1)]
    if p == 0.0:
        assert all(len(a["new_tokens"]) == 1 for a in steps)
    if p == 1.0:
        assert all(len(a["new_tokens"]) == K + 1 for a in steps[:-1])


def test_forcing_table_rate_matches_closed_form():
    """Success bits are i.i.d. Bernoulli(p); the expected accepted length per
    step is sum_{j=0..K} p^j (2.7731 at p=0.7, K=4)."""
    for p in (0.5, 0.7, 0.8):
        ok = synth.force_table(p, 3, 0, 20000)
        assert abs(ok.mean() - p) < 4 * np.sqrt(p * (1 - p) / 20000)
        K = 4
        Ls, n = [], 0
        while n + K + 1 < len(ok):
            run = 0
            while run < K and ok[n + 1 + run]:
                run += 1
            Ls.append(1 + run)
            n += 1 + run
        closed = sum(p ** j for j in range(K + 1))
        assert abs(np.mean(Ls) - closed) < 0.05 * closed
    assert abs(sum(0.7 ** j for j in range(5)) - 2.7731) < 1e-4


def test_ar_tree_is_plain_greedy(orc):
    """With a root-only tree the step is greedy decoding through the cache."""
    prompt = list(synth.make_prompt(16, CFG.vocab, 15))
    out, steps = oracle.Decoder(orc, ()).generate(prompt, 12)
    assert out == orc.greedy_ar(prompt, 12)
    assert all(len(a["new_tokens"]) == 1 for a in steps)


def test_bf16_contract_rounds_storage_points():
    cfg = synth.small_config(n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ffn=256, vocab=512)
    w = synth.weights_to_numpy(synth.make_weights(cfg, std=0.06))
    o = oracle.Oracle(cfg, w)
    xn, k, v = o.block_kv("layers.0.", np.random.default_rng(0).standard_normal((3, 256)), np.arange(3))
    for a in (xn, k, v):
        assert np.array_equal(co.round_bf16(a), a)
    prompt = list(synth.make_prompt(10, cfg.vocab, 1))
    out, _ = oracle.Decoder(o, synth.TREE_T8).generate(prompt, 12)
    assert out == o.greedy_ar(prompt, 12)


# ---------------------------------------------------------------------------
# Typical decoding (Sec. 4.3, Sec. 5.1)
# ---------------------------------------------------------------------------
def test_splitmix64_published_output():
    # first output of SplitMix64 from state 0 (the generator's reference value)
    assert co.splitmix64(0) == 16294208416658607535
    assert co.splitmix64(0) == 0xE220A8397B1DCDAF


def test_gumbel_sampling_matches_softmax():
    """Over many positions the Gumbel-max samples follow softmax(z)."""
    z = np.array([0.0, 1.0, 2.0, -1.0, 0.5])
    p = np.exp(z - z.max())
    p /= p.sum()
    n = 6000
    counts = np.zeros(len(z))
    for pos in range(n):
        counts[co.gumbel_sample(z, 7, 0, pos)] += 1
    sd = np.sqrt(n * p * (1 - p))
    assert np.all(np.abs(counts - n * p) <= 4.5 * sd), (counts, n * p)


def test_sampling_is_keyed_by_sequence_position_and_seed():
    z = np.zeros(64)
    a = [co.gumbel_sample(z, 1, 0, pos) for pos in range(40)]
    assert a == [co.gumbel_sample(z, 1, 0, pos) for pos in range(40)]
    assert a != [co.gumbel_sample(z, 2, 0, pos) for pos in range(40)]
    assert a != [co.gumbel_sample(z, 1, 1, pos) for pos in range(40)]


def test_entropy_closed_forms():
    for V in (2, 7, 1000):
        lp, H = co.log_probs_entropy(np.zeros(V))
        assert abs(H - np.log(V)) < 1e-12
        assert np.allclose(np.exp(lp), 1.0 / V)
    _, H = co.log_probs_entropy(np.array([300.0, 0.0, 0.0]))
    assert H < 1e-100 + 1e-12


def _random_tree_case(seed, V=40):
    rng = np.random.default_rng(seed)
    tree = co.Tree(synth.TREE_T8)
    toks = [int(x) for x in rng.integers(0, V, size=tree.n)]
    logits = rng.normal(0, 1.5, size=(tree.n, V))
    return tree, toks, logits


def test_typical_zero_thresholds_take_the_most_probable_deepest_path():
    """With eps = delta = 0 every node passes: the chosen node is, by brute
    force over all nodes, the deepest one with the largest path probability."""
    for seed in range(5):
        tree, toks, logits = _random_tree_case(seed)
        typ = co.Typical(1.0, 0.0, 0.0, seed=3)
        path, bonus, ok, _ = co.typical_accept(tree, toks, logits, typ, n=50)
        assert all(ok)
        best, best_key = None, None
        for u in range(tree.n):
            prob = 1.0
            for a in tree.anc[u][1:]:
                q = np.exp(logits[tree.parent[a]] - logits[tree.parent[a]].max())
                prob *= q[toks[a]] / q.sum()
            key = (tree.depth[u], prob)
            if best_key is None or key > best_key:
                best, best_key = u, key
        assert path == list(tree.anc[best])
        assert bonus == co.gumbel_sample(logits[best], 3, 0, 50 + tree.depth[best] + 1)


def test_typical_unreachable_threshold_keeps_only_the_root():
    tree, toks, logits = _random_tree_case(11)
    typ = co.Typical(1.0, 1.5, 1e9, seed=5)
    path, bonus, ok, _ = co.typical_accept(tree, toks, logits, typ, n=9)
    assert path == [0] and not any(ok[1:])
    assert bonus == co.gumbel_sample(logits[0], 5, 0, 10)


def test_typical_acceptance_is_monotone_in_the_thresholds():
    """Raising eps or delta never lets more nodes pass."""
    for seed in range(4):
        tree, toks, logits = _random_tree_case(20 + seed, V=6)
        prev = None
        for eps, delta in [(0.0, 0.0), (0.05, 0.1), (0.09, 0.3), (0.2, 0.6), (0.5, 2.0)]:
            _, _, ok, _ = co.typical_accept(tree, toks, logits, co.Typical(1.0, eps, delta), n=0)
            if prev is not None:
                assert all(p or not q for p, q in zip(prev, ok))
            prev = ok


def test_typical_sampling_without_draft_is_plain_sampling(orc):
    """With no draft (a one-node tree) typical decoding is autoregressive
    sampling: every token is the Gumbel-max sample of a plain causal forward
    at its position."""
    prompt = list(synth.make_prompt(9, CFG.vocab, 4))
    dec = oracle.Decoder(orc, (), typical=co.Typical(1.0, seed=9))
    out = [dec.prefill(prompt)]
    for _ in range(5):
        out += dec.step()["new_tokens"]
    seq = list(prompt)
    want = []
    for _ in range(6):
        logits, _, _ = orc.causal_forward(seq)
        t = co.gumbel_sample(logits[-1], 9, 0, len(seq))
        want.append(t)
        seq.append(t)
    assert out == want
