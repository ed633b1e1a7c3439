"""GPU parity of the Chimera decode step against the CPU oracle, through the
C ABI.  Each test prints the case it runs before touching the GPU."""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import (TieLog, check_step, compare_lists, gpu_step, log, make_session, tau,
                         teacher_forced_config, used_lists)
from oracle import chimera_oracle as co

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# GEMM unit (repack + MFMA GEMM), including row-count invariance
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,N,K", [(1, 64, 256), (8, 192, 512), (64, 4096, 4096), (100, 1024, 1536), (256, 128, 11008), (37, 12288, 4096)])
def test_gemm_matches_fp64(dtype, M, N, K):
    import torch
    from paper_2402_15758_amd import binding as B
    if dtype == "f32" and K % 16:
        pytest.skip("K must be a multiple of 16")
    log(f"gemm {dtype} M={M} N={N} K={K}")
    g = torch.Generator().manual_seed(M * 7 + N + K)
    x = torch.randn(M, K, generator=g)
    w = torch.randn(K, N, generator=g) * 0.05
    if dtype == "bf16":
        xt, wt = x.to(torch.bfloat16), w.to(torch.bfloat16)
        x64, w64 = xt.double(), wt.double()
        xb, wb = xt.view(torch.int16).numpy(), wt.view(torch.int16).numpy()
        code = B.CHIMERA_BF16
    else:
        x64, w64 = x.double(), w.double()
        xb, wb = x.numpy(), w.numpy()
        code = B.CHIMERA_F32
    y = np.zeros((M, N), dtype=np.float32)
    B.chimera_debug_gemm(code, xb.ctypes.data, wb.ctypes.data, M, N, K, y.ctypes.data)
    ref = (x64 @ w64).numpy()
    bound = (x64.abs() @ w64.abs()).numpy()
    assert np.all(np.abs(y - ref) <= 2e-5 * bound + 1e-30)
    # one row alone gives the same bits as inside the M-row launch
    r = M // 2
    y1 = np.zeros((1, N), dtype=np.float32)
    xr = np.ascontiguousarray(xb[r:r + 1])
    B.chimera_debug_gemm(code, xr.ctypes.data, wb.ctypes.data, 1, N, K, y1.ctypes.data)
    assert np.array_equal(y1[0].view(np.uint32), y[r].view(np.uint32))


# ---------------------------------------------------------------------------
# Tiny fp32 workload: full independent runs, bit-exact tokens
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def tiny():
    cfg = synth.TINY
    w = synth.make_weights(cfg, device="cpu")
    orc = oracle.Oracle(cfg, synth.weights_to_numpy(w))
    prompt = synth.WORKLOADS["tiny"].prompts()[0]
    return cfg, w, orc, prompt


def test_tiny_full_run_bitexact(tiny):
    cfg, w, orc, prompt = tiny
    log("tiny fp32: T8, 64 tokens, unforced")
    sess = make_session(cfg, w, synth.TREE_T8, max_len=256)
    first = sess.prefill([prompt])
    dec = oracle.Decoder(orc, synth.TREE_T8)
    assert int(first[0]) == dec.prefill(list(prompt))
    ties = TieLog()
    out, worst = [int(first[0])], 0.0
    while len(out) < 64:
        art = gpu_step(sess)
        new, err = check_step(art, 0, dec, tau(cfg), ties)
        out += new
        worst = max(worst, err)
    assert ties.argmax_ties == 0 and ties.list_ties == 0
    assert out[:64] == orc.greedy_ar(list(prompt), 64)
    log(f"tiny worst logit rel err {worst:.2e}")
    sess.close()


@pytest.mark.parametrize("std", [0.06])
def test_tiny_varied_weights_spec_equals_ar(std):
    cfg = synth.TINY
    w = synth.make_weights(cfg, std=std, device="cpu")
    orc = oracle.Oracle(cfg, synth.weights_to_numpy(w))
    prompt = synth.make_prompt(45, cfg.vocab, 21)
    log(f"tiny fp32 std={std}: spec vs AR, 48 tokens")
    spec = make_session(cfg, w, synth.TREE_T8, max_len=256)
    out_s, _ = spec.generate([prompt], 48)
    ar = make_session(cfg, w, (), max_len=256)
    out_a, steps = ar.generate([prompt], 48)
    assert out_s[0] == out_a[0] == orc.greedy_ar(list(prompt), 48)
    assert all(int(n[0]) == 1 for _, n, _ in steps)


def test_tiny_forced_acceptance_closed_form(tiny):
    import torch
    cfg, w, orc, prompt = tiny
    log("tiny fp32: forced p=0.7")
    n0, G = len(prompt), 64
    ar = orc.greedy_ar(list(prompt), G + 8)
    max_len = 256
    stride = max_len + 8
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, n0:n0 + len(ar)] = ar
    ok = synth.force_table(0.7, 3, 0, stride)[None]
    sess = make_session(cfg, w, synth.TREE_T8, max_len=max_len)
    sess.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    out, steps = sess.generate([prompt], G)
    assert out[0] == ar[:G]
    n = n0
    for toks, nn, path in steps:
        run = 0
        while run < 3 and ok[0, n + 1 + run]:
            run += 1
        assert int(nn[0]) == 1 + run
        n += int(nn[0])
    # the oracle along the same forcing takes the same steps
    dec = oracle.Decoder(orc, synth.TREE_T8, oracle.Forcing(ref[0], ok[0]))
    out_o, steps_o = dec.generate(list(prompt), G)
    assert out_o == out[0]
    assert [a["path"] for a in steps_o] == [list(p[0, : int(nn[0])]) for _, nn, p in steps]


def test_tiny_kv_compaction_equals_prefill(tiny):
    cfg, w, orc, prompt = tiny
    log("tiny fp32: KV contents after forced steps (shuffled pages)")
    import torch
    max_len = 256
    stride = max_len + 8
    n0 = len(prompt)
    ar = orc.greedy_ar(list(prompt), 40)
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, n0:n0 + 40] = ar
    ok = np.ones((1, stride), dtype=np.uint8)  # p = 1: every step accepts K + 1
    n_pages = int(np.ceil((max_len + 64) / 16))
    order = np.random.default_rng(0).permutation(n_pages).astype(np.int32)
    sess = make_session(cfg, w, synth.TREE_T8, max_len=max_len, page_order=order)
    sess.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    sess.prefill([prompt])
    for _ in range(5):
        _, nn, path = sess.step()
        assert int(nn[0]) == 4 and list(path[0]) == [0, 1, 4, 7]
    n = int(sess.debug(4)[0])
    seq = list(prompt) + ar[: n - n0]
    _, _, kv = orc.causal_forward(seq)
    for layer in range(cfg.n_layers):
        k, v = sess.kv_read(layer, 0, 0, n)
        np.testing.assert_allclose(k, kv[layer][0], rtol=1e-4, atol=1e-5)
        np.testing.assert_allclose(v, kv[layer][1], rtol=1e-4, atol=1e-5)


def test_tiny_injected_tree_tokens(tiny):
    """Verify/accept/compact on oracle-chosen tree tokens (draft bypassed):
    a tree whose rank-0 chain holds the greedy continuation accepts it."""
    cfg, w, orc, prompt = tiny
    log("tiny fp32: injected tree tokens")
    sess = make_session(cfg, w, synth.TREE_T8, max_len=256)
    dec = oracle.Decoder(orc, synth.TREE_T8)
    sess.prefill([prompt])
    dec.prefill(list(prompt))
    rng = np.random.default_rng(5)
    ties = TieLog()
    for trial in range(4):
        ar = orc.greedy_ar(dec.seq[: dec.n + 1], 3)
        toks = rng.integers(0, cfg.vocab, 7).astype(np.int32)
        if trial % 2 == 0:  # put the greedy chain on nodes 1, 4, 7
            toks[0], toks[3], toks[6] = ar[0], ar[1], ar[2]
        sess.set_tree_tokens(toks[None])
        art = gpu_step(sess)
        assert list(art["tree"][0, 1:]) == list(toks)
        dz = dec.draft()  # keep the oracle's draft state in step
        logits_o, h_o, tkv = dec.verify([dec.pending] + list(toks))
        rngs = logits_o.max(-1) - logits_o.min(-1)
        assert np.max(np.abs(art["logits"][0] - logits_o) / rngs[:, None]) <= tau(cfg)
        path, bonus = dec.accept([dec.pending] + list(toks), list(logits_o.argmax(-1)))
        L = int(art["n"][0])
        assert list(art["path"][0, :L]) == path
        if trial % 2 == 0:
            assert path == [0, 1, 4, 7]
        dec.commit(path, bonus, [dec.pending] + list(toks), h_o, tkv)


# ---------------------------------------------------------------------------
# Small bf16 model with the 7B head size: teacher-forced parity, spec == AR
# ---------------------------------------------------------------------------
SMALL = synth.small_config(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
                           n_draft_heads=4)


@pytest.fixture(scope="module")
def small():
    w = synth.make_weights(SMALL, std=0.06, device="cpu")
    orc = oracle.Oracle(SMALL, synth.weights_to_numpy(w))
    return w, orc


@pytest.mark.parametrize("n0,tree", [(90, "T64"), (600, "T32"), (61, "T64")])
def test_small_bf16_teacher_forced(small, n0, tree):
    w, orc = small
    log(f"small bf16: prompt {n0}, {tree}, teacher-forced steps")
    ranks = synth.TREES[tree]
    prompt = synth.make_prompt(n0, SMALL.vocab, 30 + n0)
    sess = make_session(SMALL, w, ranks, max_len=1024)
    first = sess.prefill([prompt])
    dec = oracle.Decoder(orc, ranks)
    f_o = dec.prefill(list(prompt))
    assert int(first[0]) == f_o
    ties = TieLog()
    for _ in range(10):
        check_step(gpu_step(sess), 0, dec, tau(SMALL), ties)
    log(f"ties: argmax {ties.argmax_ties}, lists {ties.list_ties}")


def test_small_bf16_spec_equals_ar_bitexact(small):
    """GPU speculative decoding reproduces GPU greedy decoding token for
    token: every kernel's per-row arithmetic is independent of the tree."""
    import torch
    w, _ = small
    log("small bf16: GPU spec (forced p=0.7) vs GPU AR, 120 tokens")
    prompt = synth.make_prompt(100, SMALL.vocab, 77)
    G, max_len = 120, 512
    ar_s = make_session(SMALL, w, (), max_len=max_len)
    out_a, _ = ar_s.generate([prompt], G + 8)
    stride = max_len + 8
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, 100:100 + G + 8] = out_a[0]
    ok = synth.force_table(0.7, 3, 0, stride)[None]
    sp = make_session(SMALL, w, synth.TREE_T64, max_len=max_len)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    out_s, steps = sp.generate([prompt], G)
    assert out_s[0] == out_a[0][:G]
    n = 100
    for toks, nn, path in steps:
        run = 0
        while run < 4 and ok[0, n + 1 + run]:
            run += 1
        assert int(nn[0]) == 1 + run
        n += int(nn[0])


def test_small_bf16_batch_ragged(small):
    """Batch of 3 ragged sequences with different forcing rates; each
    sequence equals its own greedy decoding and the oracle's parity holds."""
    import torch
    w, orc = small
    log("small bf16: batch 3 ragged, T32")
    lens = [70, 130, 200]
    prompts = [synth.make_prompt(n, SMALL.vocab, 500 + n) for n in lens]
    max_len, G = 512, 40
    stride = max_len + 8
    ar_s = make_session(SMALL, w, (), max_batch=3, max_len=max_len)
    out_a, _ = ar_s.generate(prompts, G + 8)
    ref = np.full((3, stride), -1, dtype=np.int32)
    oks = []
    for b, n in enumerate(lens):
        ref[b, n:n + G + 8] = out_a[b]
        oks.append(synth.force_table([0.4, 0.7, 0.9][b], 5, b, stride))
    ok = np.stack(oks)
    sp = make_session(SMALL, w, synth.TREE_T32, max_batch=3, max_len=max_len)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    first = sp.prefill(prompts)
    decs = []
    for b in range(3):
        d = oracle.Decoder(orc, synth.TREE_T32, oracle.Forcing(ref[b], ok[b]))
        assert d.prefill(list(prompts[b])) == int(first[b])
        decs.append(d)
    ties = TieLog()
    outs = [[int(f)] for f in first]
    for _ in range(8):
        art = gpu_step(sp)
        for b in range(3):
            new, _ = check_step(art, b, decs[b], tau(SMALL), ties, forced=decs[b].forcing)
            outs[b] += new
    for b in range(3):
        assert outs[b] == out_a[b][: len(outs[b])]


def test_small_bf16_graph_equals_eager(small):
    """The step replayed as a HIP graph gives the same tokens, paths and
    verify logits as launching every kernel individually, step after step
    (host work and synchronisation between the replays)."""
    import torch
    w, _ = small
    log("small bf16: graph replay vs eager launches, 12 steps")
    prompt = synth.make_prompt(80, SMALL.vocab, 91)
    outs = []
    for graph in (False, True):
        sp = make_session(SMALL, w, synth.TREE_T64, max_len=512)
        sp.set_graph(graph)
        sp.prefill([prompt])
        rec = []
        for _ in range(12):
            art = gpu_step(sp)
            rec.append((art["toks"].copy(), art["n"].copy(), art["path"].copy(), art["logits"].copy()))
            torch.cuda.synchronize()
        outs.append(rec)
        sp.close()
    for (ta, na, pa, la), (tb, nb, pb, lb) in zip(*outs):
        assert np.array_equal(ta, tb) and np.array_equal(na, nb) and np.array_equal(pa, pb)
        assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))


def test_small_bf16_pipelined_steps_equal_single_steps(small):
    """chimera_steps (steps enqueued back to back, one synchronisation)
    returns exactly what one chimera_step call per step returns: batch of 3
    ragged sequences, forced acceptance, graph replay and eager launches with
    per-launch events; the committed tokens and the last verify logits
    match bit for bit."""
    import torch
    from paper_2402_15758_amd import binding as B
    w, _ = small
    log("small bf16: pipelined steps vs single steps, batch 3, 14 steps")
    lens = [70, 130, 200]
    prompts = [synth.make_prompt(n, SMALL.vocab, 600 + n) for n in lens]
    max_len = 512
    stride = max_len + 8
    ar_s = make_session(SMALL, w, (), max_batch=3, max_len=max_len)
    out_a, _ = ar_s.generate(prompts, 90)
    ar_s.close()
    ref = np.full((3, stride), -1, dtype=np.int32)
    ok = np.stack([synth.force_table(p, 5, b, stride) for b, p in enumerate([0.5, 0.8, 0.95])])
    for b, n in enumerate(lens):
        ref[b, n:n + 90] = out_a[b]
    runs = {}
    for mode in ("single", "pipelined", "pipelined_eager_profiled"):
        sp = make_session(SMALL, w, synth.TREE_T32, max_batch=3, max_len=max_len)
        sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
        if mode == "pipelined_eager_profiled":
            sp.set_graph(False)
            sp.profile(True)
        sp.prefill(prompts)
        if mode == "single":
            rec = [sp.step() for _ in range(14)]
            toks = np.stack([r[0] for r in rec])
            nn = np.stack([r[1] for r in rec])
            path = np.stack([r[2] for r in rec])
        else:
            a = sp.steps(5)
            b = sp.steps(9)
            toks, nn, path = (np.concatenate([x, y]) for x, y in zip(a, b))
        if mode == "pipelined_eager_profiled":
            pr = sp.profile_read()
            assert pr.steps == 14 and pr.gemm_verify_launches > 0
        runs[mode] = (toks, nn, path, sp.debug(B.DBG_TOKENS), sp.debug(B.DBG_VERIFY_LOGITS))
        sp.close()
    base = runs["single"]
    for mode in ("pipelined", "pipelined_eager_profiled"):
        for x, y in zip(base, runs[mode]):
            assert np.array_equal(np.ascontiguousarray(x).view(np.uint32), np.ascontiguousarray(y).view(np.uint32)), mode
    assert base[1].min() >= 1 and base[1].max() > 1
    # lossless: each sequence's stream is its greedy stream
    for b in range(3):
        got = [int(t) for i in range(14) for t in base[0][i, b, : base[1][i, b]]]
        assert got == out_a[b][1: 1 + len(got)]


def test_pipelined_steps_refuse_bad_counts(small):
    from paper_2402_15758_amd import binding as B
    w, _ = small
    sp = make_session(SMALL, w, synth.TREE_T32, max_len=256)
    sp.prefill([synth.make_prompt(40, SMALL.vocab, 9)])
    for n in (0, B.CHIMERA_MAX_PIPELINED_STEPS + 1):
        with pytest.raises(B.ChimeraError) as e:
            B.chimera_steps(sp.model, sp.kv, sp.ctx, n, np.zeros(8, np.int32), np.zeros(8, np.int32), None,
                            sp.stream())
        assert e.value.status == B.CHIMERA_EINVAL
    with pytest.raises(B.ChimeraError) as e:
        sp.steps(60)  # 60 steps of up to 5 tokens would outgrow the 256-token capacity
    assert e.value.status == B.CHIMERA_ECAPACITY
    toks, nn, _ = sp.step()  # the refused calls changed nothing
    assert nn[0] >= 1
    sp.close()


# ---------------------------------------------------------------------------
# Trigram lookup cache (Sec. 4.1.1): exact memoization of the trigram encoder
# ---------------------------------------------------------------------------
def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


@pytest.mark.parametrize("model,entries,branch", [("tiny", 4096, False), ("tiny", 8, False),
                                                 ("small_bf16", 4096, False), ("small_bf16", 4096, True)])
def test_trigram_cache_is_exact(model, entries, branch):
    """Two passes over one prompt with and without the cache: every step's
    tokens, tree, draft lists, accepted path and verify logits are
    bit-identical.  The second pass repeats the first pass's trigrams, so
    with a large cache its lookups hit; with one 8-way set entries are
    evicted constantly."""
    if model == "tiny":
        cfg, tree = synth.TINY, synth.TREE_T8
    else:
        cfg, tree = synth.small_config(n_layers=2, d_model=512, n_heads=4, head_dim=128, d_ffn=1024, vocab=2048,
                                       n_draft_heads=4, dtype="bf16"), synth.TREE_T32
    log(f"trigram cache: {model}, {entries} entries, {'branch' if branch else 'chain'} drafting, "
        "2 passes x 10 steps")
    w = synth.make_weights(cfg, device="cuda")
    prompt = synth.make_prompt(45, cfg.vocab, 11)
    plain = make_session(cfg, w, tree, max_len=256)
    cached = make_session(cfg, w, tree, max_len=256)
    plain.set_drafting(branch)
    cached.set_drafting(branch)
    cached.trigram_cache(entries)
    per_pass = []
    for rep in range(2):
        f1 = plain.prefill([prompt])
        f2 = cached.prefill([prompt])
        assert list(f1) == list(f2)
        before = cached.trigram_stats()
        for step in range(10):
            a1, a2 = gpu_step(plain), gpu_step(cached)
            for key in a1:
                x1, x2 = a1[key], a2[key]
                if key == "lists":  # slots past a row's candidate count are unused scratch
                    x1, x2 = used_lists(x1, tree, branch), used_lists(x2, tree, branch)
                assert np.array_equal(_bits(x1), _bits(x2)), (rep, step, key)
        after = cached.trigram_stats()
        per_pass.append((after[0] - before[0], after[1] - before[1]))
    log(f"trigram cache: (lookups, hits) per pass {per_pass}")
    assert per_pass[0][0] > 0 and per_pass[1][0] == per_pass[0][0]
    if entries >= 4096:
        assert per_pass[1][1] == per_pass[1][0], "the repeated pass should hit every lookup"
    plain.close()
    cached.close()


# ---------------------------------------------------------------------------
# Typical decoding (Sec. 4.3, Sec. 5.1, T = 1)
# ---------------------------------------------------------------------------
def _sample_margin(z, a, b, seed, pos):
    """Score gap of tokens a and b in the Gumbel-max draw from z."""
    g = lambda v: -np.log(-np.log(co.sample_uniform(seed, 0, pos, v)))
    return abs((z[a] + g(a)) - (z[b] + g(b)))


@pytest.mark.parametrize("tree_name", ["T8", "none"])
def test_tiny_typical_decoding_teacher_forced(tree_name):
    """Each step: the GPU's accepted path and bonus token follow the typical
    rule applied to the GPU's own verify logits exactly (host mirror), and
    the oracle's, computed from its own logits, agree up to near-ties of the
    oracle (margin <= 2 tau * range).  The oracle then commits the GPU's
    choice."""
    cfg = synth.TINY
    tree = synth.TREE_T8 if tree_name == "T8" else ()
    typ = co.Typical(1.0, 0.09, 0.3, seed=1234)
    log(f"typical decoding: tiny, tree {tree_name}, 8 teacher-forced steps")
    w = synth.make_weights(cfg, device="cuda", std=0.06)
    prompt = synth.make_prompt(30, cfg.vocab, 5)
    sess = make_session(cfg, w, tree, max_len=128)
    sess.set_decoding(True, typ.T, typ.eps, typ.delta, typ.seed)
    first = int(sess.prefill([prompt])[0])
    orc = oracle.Oracle(cfg, synth.weights_to_numpy(w))
    dec = oracle.Decoder(orc, tree, typical=typ)
    f_o = dec.prefill(list(prompt))
    t = tau(cfg)
    ties = 0
    if first != f_o:
        logits, _, _ = orc.causal_forward(list(prompt))
        z = logits[-1]
        assert _sample_margin(z, first, f_o, typ.seed, len(prompt)) <= 2 * t * (z.max() - z.min())
        ties += 1
        dec.pending = first
        dec.seq[-1] = first
    ctree = co.Tree(tree)
    lens = []
    for step in range(8):
        art = gpu_step(sess)
        L = int(art["n"][0])
        tree_g = [int(x) for x in art["tree"][0]]
        lg = art["logits"][0].astype(np.float64)
        if dec.K:
            lists_o, dz = dec.draft(chain_tokens=[int(art["lists"][0, k, 0]) for k in range(dec.K)])
            for k in range(dec.K):
                compare_lists(art["lists"][0, k, : dec.s[k]], lists_o[k], dz[k], t, TieLog(), False)
        assert tree_g[0] == dec.pending
        # the kernel against the rule on its own logits
        path_m, bonus_m, _, _ = co.typical_accept(ctree, tree_g, lg, typ, dec.n)
        path_g = [int(x) for x in art["path"][0, :L]]
        bonus_g = int(art["toks"][0, L - 1])
        assert path_g == path_m, (step, path_g, path_m)
        assert bonus_g == bonus_m, (step, bonus_g, bonus_m)
        # the oracle on its own logits
        logits_o, h_o, tkv = dec.verify(tree_g)
        rng = logits_o.max(-1) - logits_o.min(-1)
        assert float(np.max(np.abs(lg - logits_o) / rng[:, None])) <= t
        path_o, bonus_o, ok_o, lp_o = co.typical_accept(ctree, tree_g, logits_o, typ, dec.n)
        if path_o != path_g:
            # admissible only where an oracle pass decision sits on its threshold
            near = False
            for u in range(1, ctree.n):
                _, H = co.log_probs_entropy(logits_o[ctree.parent[u]])
                thr = min(typ.eps, typ.delta * np.exp(-H))
                if abs(lp_o[u] - np.log(thr)) <= 4 * t * rng[ctree.parent[u]]:
                    near = True
            assert near, (step, path_g, path_o)
            ties += 1
        elif bonus_o != bonus_g:
            z = logits_o[path_g[-1]]
            pos = dec.n + ctree.depth[path_g[-1]] + 1
            assert _sample_margin(z, bonus_g, bonus_o, typ.seed, pos) <= 2 * t * (z.max() - z.min())
            ties += 1
        dec.commit(path_g, bonus_g, tree_g, h_o, tkv)
        lens.append(L)
    log(f"typical decoding: accepted lengths {lens}, {ties} near-ties")
    sess.close()


# ---------------------------------------------------------------------------
# Branch-conditioned drafting (tree reading of Sec. 4.4)
# ---------------------------------------------------------------------------
CHAIN3 = [(0,), (0, 0), (0, 0, 0)]
CHAIN4 = [(0,), (0, 0), (0, 0, 0), (0, 0, 0, 0)]
WIDE = [(0,), (1,), (2,), (0, 0), (0, 1), (1, 0), (1, 2), (2, 0), (0, 0, 0), (0, 1, 0), (1, 0, 0), (1, 2, 1)]


@pytest.mark.parametrize("model", ["tiny", "small_bf16"])
def test_branch_drafting_on_a_chain_tree_is_chain_drafting(tiny, small, model):
    """On a chain-shaped tree the drafted nodes are the chain's, and the two
    modes run the same arithmetic in the same order: bit-identical steps."""
    if model == "tiny":
        cfg, w, ranks = tiny[0], tiny[1], CHAIN3
    else:
        cfg, w, ranks = SMALL, small[0], CHAIN4
    log(f"branch drafting: {model}, chain tree, 10 steps in both modes")
    prompt = synth.make_prompt(40, cfg.vocab, 8)
    a = make_session(cfg, w, ranks, max_len=256)
    b = make_session(cfg, w, ranks, max_len=256)
    b.set_drafting(True)
    assert list(a.prefill([prompt])) == list(b.prefill([prompt]))
    for step in range(10):
        x, y = gpu_step(a), gpu_step(b)
        for key in x:
            u, v = x[key], y[key]
            if key == "lists":
                u, v = used_lists(u, ranks, False), used_lists(v, ranks, True)
            assert np.array_equal(_bits(u), _bits(v)), (step, key)
    a.close()
    b.close()


@pytest.mark.parametrize("tree_name", ["T8", "WIDE"])
def test_tiny_branch_drafting_teacher_forced(tiny, tree_name):
    """Every drafted node's list against the oracle's branch-conditioned
    draft along the GPU's tree tokens, then verify and accept as for chain
    drafting; fp32 admits no ties, and the stream is the greedy stream."""
    cfg, w, orc, prompt = tiny
    ranks = synth.TREE_T8 if tree_name == "T8" else WIDE
    log(f"branch drafting: tiny fp32, {tree_name}, teacher-forced until 48 tokens")
    sess = make_session(cfg, w, ranks, max_len=256)
    sess.set_drafting(True)
    first = sess.prefill([prompt])
    dec = oracle.Decoder(orc, ranks, branch=True)
    assert int(first[0]) == dec.prefill(list(prompt))
    ties = TieLog()
    out = [int(first[0])]
    while len(out) < 48:
        new, _ = check_step(gpu_step(sess), 0, dec, tau(cfg), ties)
        out += new
    assert ties.argmax_ties == 0 and ties.list_ties == 0
    assert out[:48] == orc.greedy_ar(list(prompt), 48)
    sess.close()


@pytest.mark.parametrize("n0,tree", [(90, "T64"), (300, "T32")])
def test_small_bf16_branch_drafting_teacher_forced(small, n0, tree):
    w, orc = small
    log(f"branch drafting: small bf16, prompt {n0}, {tree}, 8 teacher-forced steps")
    ranks = synth.TREES[tree]
    prompt = synth.make_prompt(n0, SMALL.vocab, 60 + n0)
    sess = make_session(SMALL, w, ranks, max_len=1024)
    sess.set_drafting(True)
    first = sess.prefill([prompt])
    dec = oracle.Decoder(orc, ranks, branch=True)
    assert int(first[0]) == dec.prefill(list(prompt))
    ties = TieLog()
    for _ in range(8):
        check_step(gpu_step(sess), 0, dec, tau(SMALL), ties)
    log(f"ties: argmax {ties.argmax_ties}, lists {ties.list_ties}")


def test_small_bf16_branch_drafting_batch_forced(small):
    """Batch of 3 ragged sequences, T32, forced acceptance, graph replay:
    each sequence is its own greedy stream, every step accepts 1 +
    (consecutive successes), and the oracle's parity holds per sequence."""
    import torch
    w, orc = small
    log("branch drafting: small bf16, batch 3 ragged, T32, forced")
    lens = [70, 130, 200]
    prompts = [synth.make_prompt(n, SMALL.vocab, 700 + n) for n in lens]
    max_len, G = 512, 40
    stride = max_len + 8
    ar_s = make_session(SMALL, w, (), max_batch=3, max_len=max_len)
    out_a, _ = ar_s.generate(prompts, G + 8)
    ar_s.close()
    ref = np.full((3, stride), -1, dtype=np.int32)
    oks = []
    for b, n in enumerate(lens):
        ref[b, n:n + G + 8] = out_a[b]
        oks.append(synth.force_table([0.5, 0.7, 0.9][b], 6, b, stride))
    ok = np.stack(oks)
    sp = make_session(SMALL, w, synth.TREE_T32, max_batch=3, max_len=max_len)
    sp.set_drafting(True)
    sp.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    first = sp.prefill(prompts)
    decs = []
    for b in range(3):
        d = oracle.Decoder(orc, synth.TREE_T32, oracle.Forcing(ref[b], ok[b]), branch=True)
        assert d.prefill(list(prompts[b])) == int(first[b])
        decs.append(d)
    ties = TieLog()
    outs = [[int(f)] for f in first]
    for _ in range(6):
        art = gpu_step(sp)
        for b in range(3):
            n = decs[b].n
            run = 0
            while run < 4 and ok[b, n + 1 + run]:
                run += 1
            assert int(art["n"][b]) == 1 + run
            new, _ = check_step(art, b, decs[b], tau(SMALL), ties, forced=decs[b].forcing)
            outs[b] += new
    for b in range(3):
        assert outs[b] == out_a[b][: len(outs[b])]
    sp.close()


# ---------------------------------------------------------------------------
# A wide batch: 9 ragged sequences x 32 nodes at 16 heads.  The verify GEMMs
# take 128-row tiles (the last one partly filled); each sequence is checked
# against the oracle.
# ---------------------------------------------------------------------------
WIDE_CFG = synth.small_config(n_layers=1, d_model=2048, n_heads=16, head_dim=128, d_ffn=1024, vocab=2048,
                              n_draft_heads=4)


def test_wide_batch_teacher_forced():
    w = synth.make_weights(WIDE_CFG, std=0.06, device="cpu")
    orc = oracle.Oracle(WIDE_CFG, synth.weights_to_numpy(w))
    lens = [40, 75, 100, 130, 161, 190, 222, 260, 300]
    log(f"wide batch: small bf16 (16 heads), batch {len(lens)} ragged, T32, 4 teacher-forced steps")
    prompts = [synth.make_prompt(n, WIDE_CFG.vocab, 900 + n) for n in lens]
    sp = make_session(WIDE_CFG, w, synth.TREE_T32, max_batch=len(lens), max_len=512)
    first = sp.prefill(prompts)
    decs = []
    ties = TieLog()
    for b, p in enumerate(prompts):
        d = oracle.Decoder(orc, synth.TREE_T32)
        f_o = d.prefill(list(p))
        if int(first[b]) != f_o:  # admissible only as a tie of the oracle's own logits
            logits, _, _ = orc.causal_forward(list(p))
            z = logits[-1]
            assert abs(z[int(first[b])] - z[f_o]) <= 2 * tau(WIDE_CFG) * (z.max() - z.min())
            d.pending = int(first[b])
            d.seq[-1] = int(first[b])
            ties.argmax_ties += 1
        decs.append(d)
    for _ in range(4):
        art = gpu_step(sp)
        for b in range(len(lens)):
            check_step(art, b, decs[b], tau(WIDE_CFG), ties)
    log(f"ties: argmax {ties.argmax_ties}, lists {ties.list_ties}")
    sp.close()


# ---------------------------------------------------------------------------
# bf16 with heads of 64: the library's other 16-bit attention instantiation
# (tree and encoder attention at head_dim 64, whose staged V rows and
# transposed LDS reads use a different row pitch than at head_dim 128)
# ---------------------------------------------------------------------------
HD64_CFG = synth.small_config(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=512, vocab=2048,
                              n_draft_heads=4)


def test_bf16_head_dim_64_teacher_forced():
    """Two ragged sequences, one short and one past position 1024 (so the
    shared pass runs near pairs, far groups of four and a partial last
    chunk), T32 with per-sequence forcing, node by node against the float64
    oracle."""
    w = synth.make_weights(HD64_CFG, std=0.06, device="cpu")
    prompts = [synth.make_prompt(n, HD64_CFG.vocab, 1300 + n) for n in (70, 1109)]
    err, _, lens = teacher_forced_config(HD64_CFG, w, prompts, synth.TREE_T32, [0.6, 0.9], 6,
                                         compute=np.float64, label="bf16 head_dim 64")
    assert err <= tau(HD64_CFG)
    assert max(lens) > 1


# fp32 with heads of 128: the remaining attention instantiation (fp32 V
# staged as V^T), at the float tolerance
F32_HD128_CFG = synth.small_config(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
                                   n_draft_heads=4, dtype="f32")


def test_f32_head_dim_128_teacher_forced():
    w = synth.make_weights(F32_HD128_CFG, std=0.06, device="cpu")
    prompts = [synth.make_prompt(n, F32_HD128_CFG.vocab, 1400 + n) for n in (70, 1109)]
    err, _, lens = teacher_forced_config(F32_HD128_CFG, w, prompts, synth.TREE_T32, [0.6, 0.9], 6,
                                         compute=np.float64, label="f32 head_dim 128")
    assert err <= tau(F32_HD128_CFG)
    assert max(lens) > 1
