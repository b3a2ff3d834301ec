"""Pins for the CPU oracle: each check ties it to something other than itself
(a library routine, a closed form, an invariant the paper states, or brute
force), chosen so that a dropped term, a wrong sign or index, or a transposed
operand in the oracle fails at least one of them."""
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
import synth
from oracle import dvi
from tests import torch_ref

PIN = synth.ModelShape("pin", n_layers=3, split_k=1, d_model=64, n_heads=4, n_kv_heads=2,
                       head_dim=16, ffn_dim=96, vocab=97, bf16=False, lora_rank=3)


def _model(shape=PIN, seed=0, norms=True, lora_A_std=0.0):
    w = synth.make_weights(shape, seed, lora_A_std=lora_A_std)
    if norms:
        torch_ref.randomize_norms(w, seed)
    return w, oracle.OracleModel(w)


def _drafter(w):
    return dvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), w.shape.lora_gamma)


# ----------------------------------------------------------------------------- generator
def test_splitmix64_reference_value():
    # First output of SplitMix64 from state 0 (Steele, Lea & Flood 2014): mix64(0x9E3779B97F4A7C15).
    assert synth.mix64(0x9E3779B97F4A7C15) == 0xE220A8397B1DCDAF


def test_generator_moments_and_counter_property():
    z = synth.normal(0, 123, 1.0, (1_000_000,), False).astype(np.float64)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    assert abs(scipy.stats.kurtosis(z, fisher=False) - 3.0) < 0.05
    # counter-based: a prefix of a longer draw is the shorter draw
    a = synth.normal(0, 9, 0.02, (1001,), True)
    b = synth.normal(0, 9, 0.02, (5000,), True)
    assert np.array_equal(a, b[:1001])
    u = synth.uniform_int(0, 4, 13, (100000,))
    assert u.min() == 0 and u.max() == 12
    assert np.allclose(np.bincount(u) / u.size, 1 / 13, atol=0.01)


# ----------------------------------------------------------------------------- model pieces
@pytest.mark.parametrize("bf16", [False, True])
def test_forward_matches_library_reference(bf16):
    """Each layer's hidden state equals a float64 reference built from torch.nn.functional
    (rms_norm, linear, scaled_dot_product_attention, silu) with complex-number RoPE and GQA."""
    shape = PIN.replace(bf16=bf16)
    w, m = _model(shape, seed=1)
    T = 11
    toks = synth.uniform_int(1, 77, shape.vocab, (T,))
    ref = torch_ref.forward(w, toks)
    cache = m.new_cache(T)
    h = m.embed(toks)
    for l in range(shape.n_layers):
        h = m.layers(cache, h, 0, l, l + 1)
        r = ref[l].numpy()
        assert np.abs(h - r).max() <= 1e-11 * np.abs(r).max(), l
    z = m.target_logits(m.final_norm(h))
    zr = torch_ref.target_logits(w, ref[-1].numpy())
    assert np.abs(z - zr).max() <= 1e-11 * np.abs(zr).max()


def test_final_norm_is_rms_norm():
    w, m = _model(seed=2)
    x = np.random.default_rng(0).normal(size=(5, PIN.d_model)) * 3.0
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (PIN.d_model,),
                                       weight=torch.from_numpy(w.final_norm.astype(np.float64)),
                                       eps=PIN.rms_eps).numpy()
    assert np.allclose(m.final_norm(x), ref, rtol=1e-13, atol=1e-13)


def test_heads_match_matmul():
    w, m = _model(seed=3, lora_A_std=0.05)
    x = np.random.default_rng(1).normal(size=(4, PIN.d_model))
    W = w.lm_head.astype(np.float64)
    A, B = w.lora_A.astype(np.float64), w.lora_B.astype(np.float64)
    assert np.allclose(m.target_logits(x), x @ W.T, rtol=1e-13, atol=1e-13)
    g = 0.7
    ref = x @ (W + g * A @ B).T          # (W^S + gamma A_s B_s) h, the head as the text writes it
    assert np.allclose(m.draft_logits(x, A, B, g), ref, rtol=1e-12, atol=1e-12)
    # A_s = 0: the draft head is exactly the target head on the same input
    assert np.array_equal(m.draft_logits(x, np.zeros_like(A), B, g), m.target_logits(x))


def test_gqa_equals_mha_with_shared_kv_heads():
    """Grouped heads read kv head h // (H/H_kv): duplicating kv weights into an MHA model
    gives the same outputs bitwise."""
    w, m = _model(seed=4)
    mha_shape = PIN.replace(n_kv_heads=PIN.n_heads)
    w2 = synth.make_weights(mha_shape, 4)
    w2.tok_emb, w2.lm_head, w2.final_norm = w.tok_emb, w.lm_head, w.final_norm
    hd, rep = PIN.head_dim, PIN.n_heads // PIN.n_kv_heads
    for l in range(PIN.n_layers):
        for key in w.layers[l]:
            w2.layers[l][key] = w.layers[l][key]
        for key in ("wk", "wv"):
            blocks = w.layers[l][key].reshape(PIN.n_kv_heads, hd, PIN.d_model)
            w2.layers[l][key] = np.ascontiguousarray(np.repeat(blocks, rep, axis=0).reshape(-1, PIN.d_model))
    m2 = oracle.OracleModel(w2)
    toks = synth.uniform_int(4, 5, PIN.vocab, (9,))
    h1 = m.layers(m.new_cache(9), m.embed(toks), 0, 0, PIN.n_layers)
    h2 = m2.layers(m2.new_cache(9), m2.embed(toks), 0, 0, PIN.n_layers)
    assert np.array_equal(h1, h2)


def test_block_equals_token_by_token():
    """Processing a block at once equals one token at a time, bitwise (row invariance;
    the block is causal by position)."""
    w, m = _model(seed=5)
    toks = synth.uniform_int(5, 6, PIN.vocab, (13,))
    c1, c2 = m.new_cache(13), m.new_cache(13)
    hb = m.layers(c1, m.embed(toks), 0, 0, PIN.n_layers)
    hs = np.concatenate([m.layers(c2, m.embed(toks[i:i + 1]), i, 0, PIN.n_layers) for i in range(13)])
    assert np.array_equal(hb, hs)
    assert np.array_equal(c1[0], c2[0]) and np.array_equal(c1[1], c2[1])
    # split at any layer and continue: layers compose
    c3 = m.new_cache(13)
    hk = m.layers(c3, m.embed(toks), 0, 0, 1)
    assert np.array_equal(m.layers(c3, hk, 0, 1, PIN.n_layers), hb)


def test_attention_row_vs_bruteforce_softmax():
    """One layer with identity-like pieces isolated: the attention output of the last
    position equals scipy softmax(q k^T / sqrt(hd)) v computed from the cache."""
    w, m = _model(seed=6, norms=False)
    T = 7
    toks = synth.uniform_int(6, 7, PIN.vocab, (T,))
    cache = m.new_cache(T)
    m.layers(cache, m.embed(toks), 0, 0, 1)
    K = cache[0][0, :T].reshape(T, PIN.n_kv_heads, PIN.head_dim)
    V = cache[1][0, :T].reshape(T, PIN.n_kv_heads, PIN.head_dim)
    # Rebuild q of the last position with the library reference and compare o via scipy.
    ref = torch_ref
    x = torch.from_numpy(w.tok_emb.astype(np.float64))[torch.as_tensor(toks.astype(np.int64))]
    a = torch.nn.functional.rms_norm(x, (PIN.d_model,), eps=PIN.rms_eps)
    q = torch.nn.functional.linear(a, torch.from_numpy(w.layers[0]["wq"].astype(np.float64)))
    q = ref.rope_complex(q.view(T, PIN.n_heads, PIN.head_dim), torch.arange(T), PIN.rope_theta).numpy()
    o = []
    for hh in range(PIN.n_heads):
        kv = hh // (PIN.n_heads // PIN.n_kv_heads)
        s = K[:, kv] @ q[T - 1, hh] / np.sqrt(PIN.head_dim)
        o.append(scipy.special.softmax(s) @ V[:, kv])
    o = np.concatenate(o)
    h_after = ref.forward(w, toks, n_layers=1)[0].numpy()[T - 1]
    wo = w.layers[0]["wo"].astype(np.float64)
    # the attention half of the block: h + Wo o ; MLP half re-derived from the reference
    x_last = x[T - 1].numpy() + wo @ o
    b = torch.nn.functional.rms_norm(torch.from_numpy(x_last), (PIN.d_model,), eps=PIN.rms_eps)
    g = torch.nn.functional.linear(b, torch.from_numpy(w.layers[0]["w_gate"].astype(np.float64)))
    u = torch.nn.functional.linear(b, torch.from_numpy(w.layers[0]["w_up"].astype(np.float64)))
    mlp = (torch.nn.functional.silu(g) * u).numpy() @ w.layers[0]["w_down"].astype(np.float64).T
    assert np.allclose(x_last + mlp, h_after, rtol=1e-12, atol=1e-12)


def test_rope_position_zero_is_identity_and_keys_rotate():
    """At position 0 the cached key is the unrotated projection; at p>0 its norm is kept."""
    w, m = _model(seed=7, norms=False)
    toks = synth.uniform_int(7, 8, PIN.vocab, (3,))
    cache = m.new_cache(3)
    m.layers(cache, m.embed(toks), 0, 0, 1)
    x = w.tok_emb[toks].astype(np.float64)
    a = x / np.sqrt((x * x).mean(axis=1, keepdims=True) + PIN.rms_eps)
    k_raw = a @ w.layers[0]["wk"].astype(np.float64).T
    assert np.allclose(cache[0][0, 0], k_raw[0], rtol=1e-13, atol=1e-13)
    for p in (1, 2):
        for hh in range(PIN.n_kv_heads):
            sl = slice(hh * PIN.head_dim, (hh + 1) * PIN.head_dim)
            assert np.isclose(np.linalg.norm(cache[0][0, p, sl]), np.linalg.norm(k_raw[p, sl]), rtol=1e-13)
            assert not np.allclose(cache[0][0, p, sl], k_raw[p, sl])


def test_argmax_ties_go_to_lowest_id():
    z = np.array([[0.0, 3.0, 1.0, 3.0], [5.0, 5.0, 5.0, 5.0]])
    assert list(oracle.argmax_lowest(z)) == [1, 0]
    # model level: copy the winning head row to a lower id -> the lower id wins
    w, m = _model(seed=8)
    toks = synth.uniform_int(8, 9, PIN.vocab, (5,))
    h = m.layers(m.new_cache(5), m.embed(toks), 0, 0, PIN.n_layers)
    hn = m.final_norm(h[-1:])
    win = int(oracle.argmax_lowest(m.target_logits(hn))[0])
    lower = (win + 5) % PIN.vocab if win < 5 else 0
    lower = min(lower, win - 1) if win > 0 else None
    if lower is not None:
        w.lm_head[lower] = w.lm_head[win]
        m2 = oracle.OracleModel(w)
        assert int(oracle.argmax_lowest(m2.target_logits(hn))[0]) == lower


def _top2_brute(row):
    """Largest minus second largest entry, by sorting the row's values (repeats kept)."""
    v = sorted((float(x) for x in row), reverse=True)
    return v[0] - v[1]


def test_top2_gap_hand_values_and_ties():
    # a distinct runner-up; a tie for the maximum gives 0; negatives; the maximum anywhere
    z = np.array([[3.0, 1.0, 2.0, 0.5],
                  [5.0, 1.0, 5.0, 4.0],
                  [-1.0, -3.0, -2.0, -1.5],
                  [0.0, 0.0, 0.0, 7.25],
                  [2.0, 2.0, 2.0, 2.0]])
    assert list(oracle.top2_gap(z)) == [1.0, 0.0, 0.5, 7.25, 0.0]


def test_top2_gap_against_sorting_on_batched_rows():
    """Random rows with repeated values, in a [2, 3, V] batch: every row's gap equals the
    sorted-values reference, and the last axis is the one reduced."""
    rng = np.random.default_rng(7)
    z = rng.integers(-6, 7, size=(2, 3, 11)).astype(np.float64) * 0.25
    g = oracle.top2_gap(z)
    assert g.shape == (2, 3)
    for i in range(2):
        for j in range(3):
            assert g[i, j] == _top2_brute(z[i, j])
    # continuous values: the gap is the difference of the two largest
    z = rng.normal(size=(50, 32000))
    ref = np.array([_top2_brute(r) for r in z])
    assert np.array_equal(oracle.top2_gap(z), ref)
    assert np.all(oracle.top2_gap(z) >= 0)


def test_gaps_of_greedy_ar_are_those_of_its_logits():
    """greedy_ar records, for every emitted token, the top-2 gap of the logits row it came from;
    the emitted token is that row's argmax."""
    w, m = _model(seed=16)
    prompt = synth.make_prompts(PIN.vocab, 1, 7, 16)[0]
    ar = dvi.greedy_ar(m, prompt, 12, keep_logits=True)
    for t in range(12):
        assert ar.gaps[t] == _top2_brute(ar.logits[t])
        assert ar.tokens[t] == int(np.argmax(ar.logits[t]))


def test_buffer_prev_id_and_state_come_from_the_same_token():
    """Each logged row holds prev_id = the token whose state drafted it: the pending (last
    committed) token for i = 1, else the draft i-1.  Its h_hat is RMSNorm of h_k computed from
    that token at its position, which a fresh forward over (prompt, committed tokens, earlier
    drafts of the block) reproduces bitwise."""
    k_spec = 4
    w, m, prompt, ar = _ar_and_prompt(seed=17, N=30)
    rng = np.random.default_rng(5)

    def forced(step, pos, out):
        nxt = ar.tokens[len(out):len(out) + k_spec]
        if nxt.size < k_spec:
            return None
        d = nxt.copy()
        j = int(rng.integers(0, k_spec + 1))   # first wrong draft at j (none if j = k_spec)
        if j < k_spec:
            d[j] = (d[j] + 1) % PIN.vocab
        return d

    r = dvi.dvi_generate(m, prompt, 30, k_spec, _drafter(w), forced_drafts=forced)
    assert np.array_equal(r.tokens, ar.tokens)
    P, k = prompt.size, PIN.split_k
    idx, checked = 0, 0
    for s in r.steps:
        rows = r.buffer[idx:idx + min(s.m + 1, k_spec)]
        idx += len(rows)
        committed = ar.tokens[:s.pos - P + 1]          # tokens committed before this step
        for b in rows:
            want_prev = int(committed[-1]) if b.i == 1 else int(s.drafts[b.i - 2])
            assert b.prev_id == want_prev
            seq = np.concatenate([prompt, committed, s.drafts[:b.i - 1]]).astype(np.int32)
            assert seq[-1] == b.prev_id and seq.size == s.pos + b.i
            hk = m.layers(m.new_cache(seq.size), m.embed(seq), 0, 0, k)
            assert np.array_equal(m.final_norm(hk[-1:])[0], b.h_hat)
            checked += 1
    assert checked >= 10 and {b.i for b in r.buffer} >= {1, 2}


# ----------------------------------------------------------------------------- losslessness
def _ar_and_prompt(seed=10, P=9, N=30, shape=PIN):
    w, m = _model(shape, seed=seed)
    prompt = synth.make_prompts(shape.vocab, 1, P, seed)[0]
    return w, m, prompt, dvi.greedy_ar(m, prompt, N)


@pytest.mark.parametrize("k_spec", [1, 2, 4, 8])
def test_dvi_equals_greedy_ar(k_spec):
    w, m, prompt, ar = _ar_and_prompt()
    r = dvi.dvi_generate(m, prompt, 30, k_spec, _drafter(w))
    assert np.array_equal(r.tokens, ar.tokens)
    if k_spec == 1:
        assert all(s.n == 1 for s in r.steps)


def test_dvi_lossless_under_random_lora_and_forced_drafts():
    w, m, prompt, ar = _ar_and_prompt(seed=11)
    rng = np.random.default_rng(0)
    A = rng.normal(0, 0.3, (PIN.vocab, PIN.lora_rank))
    r1 = dvi.dvi_generate(m, prompt, 30, 4, dvi.Drafter(A, w.lora_B.astype(np.float64), 1.0))
    assert np.array_equal(r1.tokens, ar.tokens)
    wrong = lambda step, pos, out: rng.integers(0, PIN.vocab, 4)
    r2 = dvi.dvi_generate(m, prompt, 30, 4, _drafter(w), forced_drafts=wrong)
    assert np.array_equal(r2.tokens, ar.tokens)
    right = lambda step, pos, out: ar.tokens[len(out):len(out) + 4] if len(out) + 4 <= 30 else None
    r3 = dvi.dvi_generate(m, prompt, 30, 4, _drafter(w), forced_drafts=right)
    assert np.array_equal(r3.tokens, ar.tokens)
    assert all(s.m == 4 for s in r3.steps[:-1])


@pytest.mark.parametrize("j", [0, 1, 2, 3, 4])
def test_every_accept_length(j):
    """Drafts = the AR continuation with the first corruption at 0-based index j -> m = j
    (j = k_spec: all correct -> m = k_spec).  Commit count n = min(m+1, k_spec); buffer rows
    min(m+1, k_spec) with rewards 1..1,0."""
    k_spec = 4
    w, m, prompt, ar = _ar_and_prompt(seed=12, N=40)

    def forced(step, pos, out):
        nxt = ar.tokens[len(out):len(out) + k_spec]
        if nxt.size < k_spec:
            return None
        d = nxt.copy()
        if j < k_spec:
            d[j] = (d[j] + 1) % PIN.vocab
        return d

    r = dvi.dvi_generate(m, prompt, 40, k_spec, _drafter(w), forced_drafts=forced)
    assert np.array_equal(r.tokens, ar.tokens)
    first = r.steps[0]
    assert first.m == j
    assert first.n == min(j + 1, k_spec)
    rows = r.buffer[:min(j + 1, k_spec)]
    assert [b.r for b in rows] == [1] * j + ([0] if j < k_spec else [])
    assert [b.i for b in rows] == list(range(1, len(rows) + 1))
    assert all(b.a == first.drafts[b.i - 1] for b in rows)
    # every step that received a full block of forced drafts shows the same m
    P, n_new = 9, 40
    forced_steps = [st for st in r.steps if (1 + st.pos - P) + k_spec <= n_new]
    assert len(forced_steps) > 1 and all(st.m == j for st in forced_steps)


def test_buffer_count_rule_and_no_counterfactual_rows():
    w, m, prompt, ar = _ar_and_prompt(seed=13, N=40)
    r = dvi.dvi_generate(m, prompt, 40, 4, _drafter(w))
    assert len(r.buffer) == sum(min(s.m + 1, 4) for s in r.steps)
    idx = 0
    for s in r.steps:
        rows = r.buffer[idx:idx + min(s.m + 1, 4)]
        idx += len(rows)
        assert all(b.i <= s.m + 1 for b in rows)
        assert [b.r for b in rows] == [1] * min(s.m, 4) + ([0] if s.m < 4 else [])
        for b in rows:   # logged target logits are the verify rows; h_hat are unit-RMS (gain 1 scaled)
            assert np.array_equal(b.logits_phi, s.target_logits[b.i - 1])


def test_agree_prefix_bruteforce():
    rng = np.random.default_rng(3)
    for _ in range(500):
        k = int(rng.integers(1, 9))
        t = rng.integers(0, 3, k)
        d = rng.integers(0, 3, k)
        m = max(i for i in range(k + 1) if all(d[j] == t[j] for j in range(i)))
        assert dvi.agree_prefix(list(d), list(t)) == m


def test_split_at_L_with_zero_lora_accepts_everything():
    """With the split at L (test relaxation of 0<k<L) and A_s = 0 the drafter equals the
    verifier, so every drafted token is accepted."""
    w, m, prompt, ar = _ar_and_prompt(seed=14, N=30)
    r = dvi.dvi_generate(m, prompt, 30, 4, _drafter(w), split_k=PIN.n_layers)
    assert np.array_equal(r.tokens, ar.tokens)
    assert all(s.m == 4 for s in r.steps)


def test_rejected_drafts_leave_committed_cache_untouched():
    """KV[0, len) after a run is the same whichever wrong tokens were drafted (rollback is a
    length reset), and equals the AR cache."""
    w, m, prompt, ar = _ar_and_prompt(seed=15, N=25)
    rng1, rng2 = np.random.default_rng(1), np.random.default_rng(2)
    r1 = dvi.dvi_generate(m, prompt, 25, 4, _drafter(w), forced_drafts=lambda s, p, o: rng1.integers(0, 97, 4),
                          s_max=64)
    r2 = dvi.dvi_generate(m, prompt, 25, 4, _drafter(w), forced_drafts=lambda s, p, o: rng2.integers(0, 97, 4),
                          s_max=64)
    assert r1.length == r2.length
    n = r1.length
    assert np.array_equal(r1.cache[0][:, :n], r2.cache[0][:, :n])
    assert np.array_equal(r1.cache[1][:, :n], r2.cache[1][:, :n])
    # AR cache over the same committed prefix
    c = m.new_cache(64)
    toks = np.concatenate([prompt, ar.tokens])[:n]
    m.layers(c, m.embed(toks), 0, 0, PIN.n_layers)
    assert np.array_equal(c[0][:, :n], r1.cache[0][:, :n])
