"""Edge cases and error paths of the decode step through the C ABI.

* Degenerate inputs: prompts of 1, 2 and 3 tokens (the trigram's zero
  padding reaches the draft and the encoder memory), the first and last
  vocabulary ids, the largest candidate lists (rank 7, s = 8), decoding up
  to the KV capacity.
* Paged KV with page sizes 1, 8, 32 and 256 in shuffled page order; for bf16
  with heads of 128, page sizes 1, 8, 64 and 256 leave every token and every
  committed K/V bit as they are with 16-token pages in order.
* Errors: every invalid call returns its status before any launch and
  leaves the decode state as it was; the following steps equal those of a
  session that never saw the invalid call.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import TieLog, check_step, gpu_step, log, make_session, tau, used_lists

pytestmark = pytest.mark.gpu

CFG = synth.TINY
WIDE8 = [(r,) for r in range(8)] + [(0, 0), (0, 7), (7, 0), (3, 5), (0, 0, 0), (0, 7, 6)]


@pytest.fixture(scope="module")
def tiny():
    w = synth.make_weights(CFG, device="cpu", std=0.06)
    orc = oracle.Oracle(CFG, synth.weights_to_numpy(w))
    return w, orc


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


@pytest.mark.parametrize("branch", [False, True], ids=["chain", "branch"])
@pytest.mark.parametrize("prompt", [[0], [CFG.vocab - 1, 0], [5, CFG.vocab - 1, CFG.vocab - 1]],
                         ids=["len1", "len2", "len3"])
def test_short_prompts_and_vocab_ends(tiny, prompt, branch):
    """Prompts shorter than a trigram, built from the first and last ids:
    each step matches the oracle (fp32: no ties), the stream is greedy."""
    w, orc = tiny
    log(f"edges: prompt {prompt}, {'branch' if branch else 'chain'} drafting, T8, 32 tokens")
    sess = make_session(CFG, w, synth.TREE_T8, max_len=128)
    sess.set_drafting(branch)
    first = sess.prefill([np.array(prompt, dtype=np.int32)])
    dec = oracle.Decoder(orc, synth.TREE_T8, branch=branch)
    assert int(first[0]) == dec.prefill(list(prompt))
    ties = TieLog()
    out = [int(first[0])]
    while len(out) < 32:
        new, _ = check_step(gpu_step(sess), 0, dec, tau(CFG), ties)
        out += new
    assert ties.argmax_ties == 0 and ties.list_ties == 0
    assert out[:32] == orc.greedy_ar(list(prompt), 32)
    sess.close()


@pytest.mark.parametrize("branch", [False, True], ids=["chain", "branch"])
def test_largest_candidate_lists(tiny, branch):
    """A tree using ranks up to 7 (top-8 lists, the kernel's maximum)."""
    w, orc = tiny
    log(f"edges: rank-7 tree, {'branch' if branch else 'chain'} drafting")
    prompt = synth.make_prompt(40, CFG.vocab, 17)
    sess = make_session(CFG, w, WIDE8, max_len=128)
    sess.set_drafting(branch)
    first = sess.prefill([prompt])
    dec = oracle.Decoder(orc, WIDE8, branch=branch)
    assert dec.s[0] == 8 and int(first[0]) == dec.prefill(list(prompt))
    ties = TieLog()
    for _ in range(6):
        check_step(gpu_step(sess), 0, dec, tau(CFG), ties)
    assert ties.argmax_ties == 0 and ties.list_ties == 0
    sess.close()


@pytest.mark.parametrize("page_size", [1, 8, 32, 256])
def test_page_sizes(tiny, page_size):
    """Forced steps (p = 0.7) with shuffled pages of any size: the stream is
    greedy, the accepted lengths follow the seeded successes, and the
    compacted cache equals a fresh causal pass over the committed tokens."""
    import torch
    w, orc = tiny
    log(f"edges: page size {page_size}, shuffled pages, forced p = 0.7")
    prompt = synth.make_prompt(70, CFG.vocab, 23)
    n0, max_len, G = len(prompt), 192, 48
    ar = orc.greedy_ar(list(prompt), G + 8)
    stride = max_len + 8
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, n0:n0 + len(ar)] = ar
    ok = synth.force_table(0.7, 3, 0, stride)[None]
    n_pages = int(np.ceil((max_len + 64) / page_size))
    order = np.random.default_rng(page_size).permutation(n_pages).astype(np.int32)
    from paper_2402_15758_amd import Session
    sess = Session(CFG, w, synth.TREE_T8, max_len=max_len, page_size=page_size, page_order=order)
    sess.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    out, steps = sess.generate([prompt], G)
    assert out[0] == ar[:G]
    n = n0
    for _, nn, _ in steps:
        run = 0
        while run < 3 and ok[0, n + 1 + run]:
            run += 1
        assert int(nn[0]) == 1 + run
        n += int(nn[0])
    n = int(sess.debug(4)[0])
    _, _, kv = orc.causal_forward(list(prompt) + ar[: n - n0])
    for layer in range(CFG.n_layers):
        k, v = sess.kv_read(layer, 0, 0, n)
        np.testing.assert_allclose(k, kv[layer][0], rtol=1e-4, atol=1e-5)
        np.testing.assert_allclose(v, kv[layer][1], rtol=1e-4, atol=1e-5)
    sess.close()


def test_decoding_up_to_capacity(tiny):
    """Steps run until the next one would not fit the KV cache, which is
    refused with CHIMERA_ECAPACITY and leaves the state as it was."""
    from paper_2402_15758_amd import binding as B
    w, orc = tiny
    log("edges: decoding up to the capacity of a 64-position cache")
    prompt = synth.make_prompt(40, CFG.vocab, 29)
    sess = make_session(CFG, w, synth.TREE_T8, max_len=64)
    out = [int(sess.prefill([prompt])[0])]
    with pytest.raises(B.ChimeraError):  # 52 + 8 + 3 + 2 > 64
        sess.prefill([synth.make_prompt(52, CFG.vocab, 1)])
    out = [int(sess.prefill([prompt])[0])]
    while True:
        n_before = int(sess.debug(B.DBG_SEQ_LEN)[0])
        try:
            toks, nn, _ = sess.step()
        except B.ChimeraError as e:
            assert e.status == B.CHIMERA_ECAPACITY
            assert int(sess.debug(B.DBG_SEQ_LEN)[0]) == n_before
            assert n_before + 8 + 3 + 2 > 64
            break
        out += [int(t) for t in toks[0, : nn[0]]]
    assert out == orc.greedy_ar(list(prompt), len(out))
    sess.close()


def test_invalid_calls_change_nothing(tiny):
    """Each invalid call fails with its status; a session that received them
    between its steps produces the same bits as one that did not."""
    from paper_2402_15758_amd import binding as B
    w, _ = tiny
    log("edges: invalid calls between steps")
    prompt = synth.make_prompt(33, CFG.vocab, 31)
    a = make_session(CFG, w, synth.TREE_T8, max_len=128)
    b = make_session(CFG, w, synth.TREE_T8, max_len=128)
    with pytest.raises(B.ChimeraError) as e:
        b.step()
    assert e.value.status == B.CHIMERA_ESTATE

    def expect(status, fn, *args):
        with pytest.raises(B.ChimeraError) as e:
            fn(*args)
        assert e.value.status == status, (fn, e.value)

    import torch
    tri_buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")  # 256-byte aligned, kept alive
    tri_arena = tri_buf.data_ptr()
    assert list(a.prefill([prompt])) == list(b.prefill([prompt]))
    for step in range(6):
        x = gpu_step(a)
        n_before = b.debug(B.DBG_SEQ_LEN).copy()
        expect(B.CHIMERA_EINVAL, b.prefill, [np.zeros(0, dtype=np.int32)])
        expect(B.CHIMERA_EINVAL, b.prefill, [np.array([1, -1, 2], dtype=np.int32)])
        expect(B.CHIMERA_EINVAL, b.prefill, [np.array([CFG.vocab], dtype=np.int32)])
        expect(B.CHIMERA_ECAPACITY, b.prefill, [synth.make_prompt(120, CFG.vocab, 2)])
        expect(B.CHIMERA_EINVAL, B.chimera_set_drafting, b.ctx, 7)
        expect(B.CHIMERA_EINVAL, B.chimera_set_decoding, b.ctx, 1, 0.0, 0.09, 0.3, 0)
        expect(B.CHIMERA_EINVAL, B.chimera_set_tree_tokens, b.ctx, np.zeros(7 * 2, dtype=np.int32), 2)
        expect(B.CHIMERA_EINVAL, B.chimera_set_tree_tokens, b.ctx, np.full(7, CFG.vocab, dtype=np.int32), 1)
        expect(B.CHIMERA_EINVAL, B.chimera_set_trigram_cache, b.ctx, tri_arena, 1 << 20, 12)
        assert np.array_equal(b.debug(B.DBG_SEQ_LEN), n_before)
        y = gpu_step(b)
        for key in x:
            u, v = x[key], y[key]
            if key == "lists":  # slots past a row's candidate count are unused scratch
                u, v = used_lists(u, synth.TREE_T8, False), used_lists(v, synth.TREE_T8, False)
            assert np.array_equal(_bits(u), _bits(v)), (step, key)
    a.close()
    b.close()


# Prompt lengths around the attention decomposition's boundaries: the shared
# MFMA pass takes positions up to P - 16 in 64-position chunks (pairs below
# position 1024, groups of four beyond), the window the last 16.  Prefill runs chains of up to 64 positions,
# whose deep nodes read chain positions >= n through the shared pass.
BOUNDARY_LENS = [12, 13, 16, 17, 47, 48, 62, 63, 64, 65, 77, 78, 79, 80, 81, 125, 126, 127, 128, 129, 143, 144,
                 1023, 1024, 1025, 1039, 1040, 1041, 1295, 1296, 1297, 1535, 1536, 1551, 1552]


def test_attention_boundaries(tiny):
    """For each prompt length: the cache after prefill equals a fresh causal
    pass (every layer, so layer 1 checks layer 0's attention over the
    prompt), and three speculative steps match the oracle node by node."""
    w, orc = tiny
    log(f"edges: attention boundaries, prompts {BOUNDARY_LENS}")
    for n0 in BOUNDARY_LENS:
        prompt = synth.make_prompt(n0, CFG.vocab, 700 + n0)
        sess = make_session(CFG, w, synth.TREE_T8, max_len=max(192, n0 + 64))
        first = sess.prefill([prompt])
        dec = oracle.Decoder(orc, synth.TREE_T8)
        assert int(first[0]) == dec.prefill(list(prompt)), n0
        _, _, kv = orc.causal_forward(list(prompt))
        for layer in range(CFG.n_layers):
            k, v = sess.kv_read(layer, 0, 0, n0)
            np.testing.assert_allclose(k, kv[layer][0], rtol=1e-4, atol=1e-5, err_msg=f"K n0={n0} layer {layer}")
            np.testing.assert_allclose(v, kv[layer][1], rtol=1e-4, atol=1e-5, err_msg=f"V n0={n0} layer {layer}")
        ties = TieLog()
        for _ in range(3):
            check_step(gpu_step(sess), 0, dec, tau(CFG), ties)
        assert ties.argmax_ties == 0 and ties.list_ties == 0, n0
        sess.close()


SMALL_BF16 = synth.small_config(n_layers=2, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=2048,
                                n_draft_heads=4)


@pytest.fixture(scope="module")
def small_bf16_greedy():
    """GPU greedy stream and committed target K/V of one 600-token prompt,
    16-token pages in order."""
    from paper_2402_15758_amd import Session
    w = synth.make_weights(SMALL_BF16, device="cpu", std=0.06)
    prompt = synth.make_prompt(600, SMALL_BF16.vocab, 41)
    ar = Session(SMALL_BF16, w, (), max_len=768)
    out, _ = ar.generate([prompt], 68)
    n = int(ar.debug(4)[0])
    kv = [ar.kv_read(layer, 0, 0, n) for layer in range(SMALL_BF16.n_layers)]
    ar.close()
    return w, prompt, out[0], kv, n


@pytest.mark.parametrize("page_size", [1, 8, 64, 256])
def test_bf16_page_sizes_equal_greedy_bitexact(small_bf16_greedy, page_size):
    """Speculative steps (T64, forced p = 0.7) over shuffled pages of another
    size: the same tokens as greedy decoding, and the same K/V bits at every
    committed position of every layer (paging moves rows, never arithmetic)."""
    import torch
    from paper_2402_15758_amd import Session
    w, prompt, ar_out, ar_kv, ar_n = small_bf16_greedy
    log(f"edges: bf16 page size {page_size}, shuffled pages, forced p = 0.7, against GPU greedy")
    n0, max_len, G = len(prompt), 768, 60
    stride = max_len + 8
    ref = np.full((1, stride), -1, dtype=np.int32)
    ref[0, n0:n0 + len(ar_out)] = ar_out
    ok = synth.force_table(0.7, 3, 0, stride)[None]
    n_pages = int(np.ceil((max_len + 64) / page_size))
    order = np.random.default_rng(100 + page_size).permutation(n_pages).astype(np.int32)
    sess = Session(SMALL_BF16, w, synth.TREE_T64, max_len=max_len, page_size=page_size, page_order=order)
    sess.set_forcing(torch.from_numpy(ref).cuda(), torch.from_numpy(ok).cuda())
    out, steps = sess.generate([prompt], G)
    assert out[0] == list(ar_out[:G])
    assert max(int(nn[0]) for _, nn, _ in steps) > 2
    n = min(int(sess.debug(4)[0]), ar_n)
    for layer in range(SMALL_BF16.n_layers):
        k, v = sess.kv_read(layer, 0, 0, n)
        assert np.array_equal(k, ar_kv[layer][0][:n]) and np.array_equal(v, ar_kv[layer][1][:n]), layer
    sess.close()
