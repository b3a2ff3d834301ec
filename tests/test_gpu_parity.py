"""GPU parity: the HIP decode step against the CPU oracle, through the C ABI.

Expected values come from tests/golden/*.npz (written by tests/golden/make_golden.py, which
calls only the oracle) or from the oracle directly for small cases."""
import numpy as np
import pytest

import oracle
import synth
from oracle import dvi as odvi
from oracle import update as oupd
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

SMALL = ["tiny", "1b_L4", "7b_L4", "13b_L4"]
KSPEC = {"tiny": 4, "1b_L4": 5, "7b_L4": 4, "13b_L4": 6}


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", SMALL)
def test_free_running_tokens_match_oracle(name):
    g = gu.golden(name)
    shape = gu.SHAPES[name]
    P, T = g["prompt"].size, g["tokens"].size
    _say("free-running %s P=%d T=%d k_spec=%d" % (name, P, T, KSPEC[name]))
    eng, _ = gu.engine(shape, max_seq=P + T + 16)
    toks, info = eng.generate(g["prompt"][None], T, KSPEC[name])
    agree = gu.compare_free_running(toks[0], g["tokens"], g["gaps"])
    _say("  %d/%d tokens agree before the first (near-tie) divergence; mean m %.2f" % (agree, T, info["m"].mean()))
    assert agree >= 1
    eng.close()


@pytest.mark.parametrize("name", SMALL)
def test_teacher_forced_logits_and_argmax(name):
    """Drafts and commits follow the oracle's sequence: every golden token's verify logits are
    within the storage type's tolerance (row L2 and every element) and its argmax matches
    wherever the oracle is not near a tie."""
    g = gu.golden(name)
    shape = gu.SHAPES[name]
    P, T = g["prompt"].size, g["tokens"].size
    assert g["logits"].shape[0] == T
    _say("teacher-forced %s rows=%d" % (name, T))
    eng, _ = gu.engine(shape, max_seq=P + T + 16)
    rows = gu.teacher_forced(eng, g["prompt"], g["tokens"], KSPEC[name])
    assert [r[0] for r in rows] == list(range(T))
    w2, wm, n = gu.check_teacher_forced(rows, g["logits"][None], g["tokens"][None], g["gaps"][None], shape)
    _say("  %d rows: worst relative L2 error %.3g, worst elementwise error %.3g of max|z|" % (n, w2, wm))
    eng.close()


def _gpu_run(eng, prompt, n_new, k_spec, forced_fn=None):
    """Drive the ABI step by step; returns tokens and the per-step (drafts, targets, m, n)."""
    first = eng.prefill(prompt[None])
    out = [int(first[0])]
    steps = []
    while len(out) < n_new:
        forced = forced_fn(out) if forced_fn else None
        d = eng.draft(k_spec, forced=forced, want=True)
        tg, mv = eng.verify(want=True)
        tok, n, m = eng.commit(max_new=np.array([n_new - len(out)], np.int32))
        assert m[0] == mv[0]
        out.extend(int(t) for t in tok[0, :n[0]])
        steps.append((d[0].copy(), tg[0].copy(), int(m[0]), int(n[0])))
    return np.array(out, np.int32), steps


@pytest.mark.parametrize("name", ["tiny", "7b_L4"])
def test_dvi_equals_gpu_greedy_and_kv_rollback_bitwise(name):
    """(R3) speculative decoding equals plain greedy decoding on the same engine, token for
    token, with bitwise-equal committed keys/values; (R2) two runs that differ only in which
    wrong drafts were proposed end bitwise equal; (R1) a rejected step leaves KV[0, len) as is."""
    shape = gu.SHAPES[name]
    P, T = 70, 30
    prompt = synth.make_prompts(shape.vocab, 1, P, 3)[0]
    eng, w = gu.engine(shape, max_seq=P + T + 16)
    ar, _ = _gpu_run(eng, prompt, T, 1)
    Lc = P + T - 1
    kv_ar = [eng.read_kv(l, 0, 0, Lc) for l in range(shape.n_layers)]
    spec, steps = _gpu_run(eng, prompt, T, 4)
    assert np.array_equal(spec, ar)
    assert eng.lengths()[0] == Lc
    for l in range(shape.n_layers):
        k, v = eng.read_kv(l, 0, 0, Lc)
        assert np.array_equal(k, kv_ar[l][0]) and np.array_equal(v, kv_ar[l][1]), "layer %d" % l
    rng1, rng2 = np.random.default_rng(1), np.random.default_rng(2)
    r1, _ = _gpu_run(eng, prompt, T, 4, lambda out: rng1.integers(0, shape.vocab, (1, 4)))
    kv1 = [eng.read_kv(l, 0, 0, Lc) for l in range(shape.n_layers)]
    r2, _ = _gpu_run(eng, prompt, T, 4, lambda out: rng2.integers(0, shape.vocab, (1, 4)))
    assert np.array_equal(r1, ar) and np.array_equal(r2, ar)
    for l in range(shape.n_layers):
        k, v = eng.read_kv(l, 0, 0, Lc)
        assert np.array_equal(k, kv1[l][0]) and np.array_equal(v, kv1[l][1])
    # R1: one step of all-wrong drafts: KV[0, len) untouched, one token committed
    eng.prefill(prompt[None])
    before = [eng.read_kv(l, 0, 0, P) for l in range(shape.n_layers)]
    wrong = (ar[1:5] + 1) % shape.vocab
    eng.draft(4, forced=wrong[None])
    eng.verify()
    tok, n, m = eng.commit()
    assert m[0] == 0 and n[0] == 1 and tok[0, 0] == ar[1]
    for l in range(shape.n_layers):
        k, v = eng.read_kv(l, 0, 0, P)
        assert np.array_equal(k, before[l][0]) and np.array_equal(v, before[l][1])
    eng.close()


@pytest.mark.parametrize("j", [0, 1, 2, 3, 4])
def test_every_accept_length_and_replay_rows(j):
    shape = gu.SHAPES["tiny"]
    P, T, k = 40, 26, 4
    prompt = synth.make_prompts(shape.vocab, 1, P, 5)[0]
    eng, _ = gu.engine(shape, max_seq=P + T + 16)
    ar, _ = _gpu_run(eng, prompt, T, 1)

    def forced(out):
        nxt = ar[len(out):len(out) + k].copy()
        if nxt.size < k:
            nxt = np.concatenate([nxt, np.zeros(k - nxt.size, np.int32)])
        if j < k:
            nxt[j] = (nxt[j] + 1) % shape.vocab
        return nxt[None]

    toks, steps = _gpu_run(eng, prompt, T, k, forced)
    assert np.array_equal(toks, ar)
    full = [s for s in steps[:-1]]
    assert all(s[2] == j for s in full), [s[2] for s in steps]
    valid, nxt = eng.buffer_info()
    expect_rows = sum(min(s[2] + 1, k) for s in steps)
    assert valid == min(expect_rows, 256)
    buf = eng.read_buffer(0, valid)
    row = 0
    for d, tg, m, n in steps:
        cnt = min(m + 1, k)
        assert list(buf["r"][row:row + cnt]) == [1] * min(m, k) + ([0] if m < k else [])
        assert list(buf["a"][row:row + cnt]) == list(d[:cnt])
        assert list(buf["i"][row:row + cnt]) == list(range(1, cnt + 1))
        assert all(buf["fresh"][row:row + cnt] == 1)
        row += cnt
    eng.close()


def test_replay_ring_smaller_than_one_steps_rows():
    """Four sequences with accept lengths 0..3 log 10 rows per step into a 5-row ring: the ring
    must hold exactly what logging the rows one by one, in sequence order, leaves (Section 3.3
    logging rule; the last writer of a slot wins), with each kept row's verify logits."""
    shape = gu.SHAPES["tiny"]
    B, P, T, k, R = 4, 24, 22, 4, 5
    prompts = synth.make_prompts(shape.vocab, B, P, 11)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, buffer_rows=R)
    first = eng.prefill(prompts)
    ar = [[int(first[b])] for b in range(B)]
    while len(ar[0]) < T:  # each sequence's greedy continuation on the same engine
        eng.draft(1)
        eng.verify()
        tok, n, m = eng.commit()
        for b in range(B):
            ar[b].append(int(tok[b, 0]))
    ar = np.array(ar, np.int32)
    first = eng.prefill(prompts)
    out = [[int(first[b])] for b in range(B)]
    ring, nxt, valid = [None] * R, 0, 0
    for step in range(4):
        forced = np.zeros((B, k), np.int32)
        for b in range(B):
            L = len(out[b])
            forced[b] = ar[b, L:L + k]
            forced[b, b] = (forced[b, b] + 1) % shape.vocab  # sequence b accepts exactly b drafts
        eng.draft(k, forced=forced)
        eng.verify()
        lg = eng.read_logits()
        tok, n, m = eng.commit()
        assert list(m) == list(range(B)), (step, m)
        for b in range(B):
            for i in range(1, min(m[b] + 1, k) + 1):
                prev = out[b][-1] if i == 1 else forced[b, i - 2]
                ring[nxt] = (forced[b, i - 1], int(i <= m[b]), i, prev, lg[b, i - 1].copy())
                nxt, valid = (nxt + 1) % R, min(valid + 1, R)
            out[b].extend(int(t) for t in tok[b, :n[b]])
        assert eng.buffer_info() == (valid, nxt)
        buf = eng.read_buffer(0, valid)
        for sl in range(valid):
            a_, r_, i_, prev_, lgs = ring[sl]
            assert (buf["a"][sl], buf["r"][sl], buf["i"][sl], buf["prev"][sl], buf["fresh"][sl]) == \
                (a_, r_, i_, prev_, 1), (step, sl)
            assert np.array_equal(buf["logits"][sl], lgs), (step, sl)
        ms = (buf["h"].astype(np.float64) ** 2).mean(axis=1)  # RMSNorm(h_k) rows, unit gain
        assert np.allclose(ms, 1.0, atol=1e-4)
    for b in range(B):
        assert np.array_equal(np.array(out[b]), ar[b, :len(out[b])])
    eng.close()


def test_buffer_rows_hold_the_verify_logits_and_normed_states():
    shape = gu.SHAPES["tiny"]
    g = gu.golden("tiny")
    eng, w = gu.engine(shape, max_seq=128)
    eng.prefill(g["prompt"][None])
    eng.draft(4)
    eng.verify()
    lg = eng.read_logits()[0]
    tok, n, m = eng.commit()
    buf = eng.read_buffer(0, min(m[0] + 1, 4))
    for i in range(buf["a"].size):
        assert np.array_equal(buf["logits"][i], lg[i])
    # h rows are RMSNorm(h_k) with unit gain: mean square 1 up to eps
    ms = (buf["h"].astype(np.float64) ** 2).mean(axis=1)
    assert np.allclose(ms, 1.0, atol=1e-4)
    eng.close()


@pytest.mark.parametrize("name,n_rows,r,vocab", [("tiny", 48, 16, None), ("tiny", 100, 16, None), ("tiny", 300, 16, None),
                                                ("1b_L4", 200, 16, None), ("1b_L4", 256, 16, None),
                                                ("tiny", 100, 20, None), ("1b_L4", 200, 40, None),
                                                ("tiny", 300, 64, None), ("tiny", 100, 16, 4112),
                                                ("tiny", 64, 16, 33024)])
def test_drafter_update_gradients_match_oracle(name, n_rows, r, vocab):
    """Row counts cover the update GEMM's 4-, 8- and 16-group variants and more rows than one
    launch takes (300 > 256).  Ranks other than 16 take the large-M logits epilogue through one
    partial pass over the rank (20), two passes (40: 32 + 8) and two full passes (64).  A
    vocabulary of 4112 = 32 * 128 + 16 leaves the gradient pass's last 128-entry block mostly
    empty; one of 33024 = 32 * 1024 + 256 sends the row kernel past the 32 entries per thread it
    holds in registers."""
    shape = gu.SHAPES[name].replace(lora_rank=r)
    if vocab is not None:
        shape = shape.replace(vocab=vocab)
    eng, w = gu.engine(shape, max_seq=64, lora_A_std=0.02, buffer_rows=max(256, n_rows))
    buf = synth.make_buffer(shape.d_model, shape.vocab, n_rows, seed=11)
    eng.prefill(synth.make_prompts(shape.vocab, 1, 8, 1))
    eng.write_buffer(buf.h, buf.a, buf.logits, buf.r, buf.fresh)
    c = oupd.Coeffs(c_kl=0.7, c_ce=0.9, c_pg=0.4, c_ent=0.05, tau=1.3, baseline=0.35)
    st = eng.update_drafter(c.c_kl, c.c_ce, c.c_pg, c.c_ent, c.tau, c.baseline, lr=0.0, grads=True)
    W = w.as_f32(w.lm_head).astype(np.float64)
    ref = oupd.loss_and_grad(W, w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma,
                             buf.h.astype(np.float64), buf.a, buf.logits, buf.r, buf.fresh, c)
    dA = st["grad_A"].cpu().numpy()
    dB = st["grad_B"].cpu().numpy()
    eA, eB = gu.rel_l2(dA, ref.dA), gu.rel_l2(dB, ref.dB)
    _say("update %s rows=%d rank=%d vocab=%d: |dA| rel err %.3g, |dB| rel err %.3g, loss %.6g vs %.6g"
         % (name, n_rows, r, shape.vocab, eA, eB, st["loss"], ref.loss))
    assert eA <= 1e-2 and eB <= 1e-2
    assert st["rows"] == n_rows and st["accepted"] == int(buf.r.sum()) and st["fresh"] == int(buf.fresh.sum())
    for key in ("kl", "ce", "pg", "entropy"):
        assert abs(st[key] - getattr(ref, key)) <= 1e-3 * max(1.0, abs(getattr(ref, key))), key
    # an Adam step with lr > 0 moves A_s, B_s as the oracle's Adam does (same gradient)
    A0, B0 = eng.lora_A.cpu().numpy().copy(), eng.lora_B.cpu().numpy().copy()
    eng.update_drafter(c.c_kl, c.c_ce, c.c_pg, c.c_ent, c.tau, c.baseline, lr=1e-3, opt_step=1)
    A1, B1 = eng.lora_A.cpu().numpy(), eng.lora_B.cpu().numpy()
    # the fresh flags were cleared by the first update: recompute the oracle gradient without them
    ref2 = oupd.loss_and_grad(W, A0.astype(np.float64), B0.astype(np.float64), shape.lora_gamma,
                              buf.h.astype(np.float64), buf.a, buf.logits, buf.r, np.zeros_like(buf.fresh), c)
    z = np.zeros_like(A0, np.float64)
    Ae, _, _ = oupd.adam_step(A0.astype(np.float64), ref2.dA, z, z.copy(), 1, 1e-3)
    zb = np.zeros_like(B0, np.float64)
    Be, _, _ = oupd.adam_step(B0.astype(np.float64), ref2.dB, zb, zb.copy(), 1, 1e-3)
    assert gu.rel_l2(A1 - A0, Ae - A0) <= 5e-2 and gu.rel_l2(B1 - B0, Be - B0) <= 5e-2
    eng.close()


# The paper's objective ablations and drafter variants as coefficient vectors of the one loss.
OBJECTIVES = {
    "kl_only": oupd.Coeffs(c_kl=1.0, c_ce=0.0, c_pg=0.0, c_ent=0.0, tau=1.0, baseline=0.0),
    "ce_only": oupd.Coeffs(c_kl=0.0, c_ce=1.0, c_pg=0.0, c_ent=0.0, tau=1.0, baseline=0.0),
    "pg_only": oupd.Coeffs(c_kl=0.0, c_ce=0.0, c_pg=1.0, c_ent=0.0, tau=1.0, baseline=0.4),
    "entropy_only": oupd.Coeffs(c_kl=0.0, c_ce=0.0, c_pg=0.0, c_ent=0.5, tau=1.0, baseline=0.0),
    "tau_0.5": oupd.Coeffs(c_kl=1.0, c_ce=0.5, c_pg=0.5, c_ent=0.0, tau=0.5, baseline=0.2),
    "tau_2": oupd.Coeffs(c_kl=1.0, c_ce=0.0, c_pg=0.0, c_ent=0.1, tau=2.0, baseline=0.0),
}


@pytest.mark.parametrize("obj", list(OBJECTIVES))
def test_drafter_update_objective_variants(obj):
    """Each objective alone (KL, reward-masked CE, policy gradient, entropy bonus) and
    temperatures other than 1: gradients and loss terms against the oracle."""
    shape = gu.SHAPES["1b_L4"]
    n_rows = 128
    c = OBJECTIVES[obj]
    eng, w = gu.engine(shape, max_seq=64, lora_A_std=0.02, buffer_rows=256)
    buf = synth.make_buffer(shape.d_model, shape.vocab, n_rows, seed=13)
    assert 0 < buf.r.sum() < n_rows
    eng.prefill(synth.make_prompts(shape.vocab, 1, 8, 1))
    eng.write_buffer(buf.h, buf.a, buf.logits, buf.r, buf.fresh)
    st = eng.update_drafter(c.c_kl, c.c_ce, c.c_pg, c.c_ent, c.tau, c.baseline, lr=0.0, grads=True)
    W = w.as_f32(w.lm_head).astype(np.float64)
    ref = oupd.loss_and_grad(W, w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma,
                             buf.h.astype(np.float64), buf.a, buf.logits, buf.r, buf.fresh, c)
    eA = gu.rel_l2(st["grad_A"].cpu().numpy(), ref.dA)
    eB = gu.rel_l2(st["grad_B"].cpu().numpy(), ref.dB)
    _say("objective %s: |dA| rel err %.3g, |dB| rel err %.3g, loss %.6g vs %.6g" % (obj, eA, eB, st["loss"], ref.loss))
    assert eA <= 1e-2 and eB <= 1e-2
    assert abs(st["loss"] - ref.loss) <= 1e-3 * max(1.0, abs(ref.loss))
    for key in ("kl", "ce", "pg", "entropy"):
        assert abs(st[key] - getattr(ref, key)) <= 1e-3 * max(1.0, abs(getattr(ref, key))), key
    eng.close()


@pytest.mark.parametrize("P", [40, 1000])
def test_batched_sequences_are_independent(P):
    """Batch of 4 equals four single-sequence runs, token for token and bitwise in KV.  With
    1000-token prompts the batch's attention grid is large enough to merge in a launch of its
    own, while the single sequences merge inside the attention kernel: both give the same bits."""
    shape = gu.SHAPES["7b_L4"]
    T, B = 20, 4
    prompts = synth.make_prompts(shape.vocab, B, P, 9)
    w = synth.make_weights(shape, 0)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, weights=w)
    toks, info = eng.generate(prompts, T, 4)
    kvb = {l: [eng.read_kv(l, b, 0, P + 5) for b in range(B)] for l in (1, shape.n_layers - 1)}
    eng.close()
    eng1, _ = gu.engine(shape, max_batch=1, max_seq=P + T + 16, weights=w)
    for b in range(B):
        t1, _ = eng1.generate(prompts[b:b + 1], T, 4)
        assert np.array_equal(t1[0], toks[b]), b
        for l, ref in kvb.items():
            k, v = eng1.read_kv(l, 0, 0, P + 5)
            assert np.array_equal(k, ref[b][0]) and np.array_equal(v, ref[b][1]), (l, b)
    eng1.close()


def test_prefill_with_unequal_prompt_lengths():
    """Prompts of different lengths in one batch (some crossing a 64-position block): each
    sequence's first token and its head logits equal the oracle's for its own prompt, and the
    whole run commits, bitwise in keys and values over the sequence's own length, what the
    sequence commits when it runs alone."""
    shape = gu.SHAPES["7b_L4"]
    lens = np.array([70, 57, 31, 66], np.int32)
    B, T, P = lens.size, 16, int(lens.max())
    prompts = synth.make_prompts(shape.vocab, B, P, 21)
    w = synth.make_weights(shape, 0)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, weights=w)
    first = eng.prefill(prompts, lens)
    pre = eng.read_logits()[:, 0].copy()
    om = oracle.OracleModel(w)
    for b in range(B):
        ref = odvi.greedy_ar(om, prompts[b, :lens[b]], 1, keep_logits=True)
        gu.check_close(pre[b], ref.logits[0], shape, "sequence %d prefill logits" % b)
        if ref.gaps[0] > gu.TIE_GAP:
            assert first[b] == ref.tokens[0]
    assert np.array_equal(eng.lengths(), lens)
    toks, info = eng.generate(prompts, T, 4, lens=lens)
    assert np.array_equal(eng.lengths(), lens + T - 1)
    kvb = {l: [eng.read_kv(l, b, 0, int(lens[b]) + T - 1) for b in range(B)] for l in (0, shape.n_layers - 1)}
    eng.close()
    eng1, _ = gu.engine(shape, max_batch=1, max_seq=P + T + 16, weights=w)
    for b in range(B):
        t1, _ = eng1.generate(prompts[b:b + 1, :lens[b]], T, 4)
        assert np.array_equal(t1[0], toks[b]), b
        for l, ref in kvb.items():
            k, v = eng1.read_kv(l, 0, 0, int(lens[b]) + T - 1)
            assert np.array_equal(k, ref[b][0]) and np.array_equal(v, ref[b][1]), (l, b)
    eng1.close()
    _say("unequal prompt lengths %s: %d tokens each, equal to single-sequence runs" % (list(lens), T))


def _tie_partner(t, kind):
    """A lower vocabulary id than t whose logit the head computes in the same summation order
    (a decode-GEMM tile's K chunk order is fixed per group of 12 tiles = 192 ids): same lane
    (t-1, one of a lane's 4 ids), same 16-id tile but another lane, or another tile of the group.
    None when t has no such partner."""
    if kind == "lane":
        return t - 1 if t % 4 else None
    if kind == "tile":
        return t - 4 if t % 16 >= 4 else None
    tile = t // 16
    return t - 16 if tile % 12 else None


@pytest.mark.parametrize("name,kind", [("tiny", "lane"), ("tiny", "tile"), ("tiny", "group"), ("1b_L4", "lane"),
                                       ("1b_L4", "group")])
def test_argmax_ties_go_to_the_lowest_id(name, kind):
    """Greedy choice ties (Section 3.1 greedy argmax; the lowest id wins): a head row W^V[t] (and
    its LoRA row A_s[t]) copied to a lower id t' makes the two logits bitwise equal, so wherever t
    was the argmax, the verify head, the prefill head and the draft head must now choose t'.  The
    three partner kinds reach the tie in the epilogue's own lane, across its lanes, and across tiles
    in the argmax kernel."""
    shape = gu.SHAPES[name]
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    P, k = 21, 4
    _say("argmax ties %s (%s)" % (name, kind))
    eng, _ = gu.engine(shape, max_seq=P + 16, weights=w)
    # a prompt and forced block whose winners (a verify row's, the first draft's) have partners of
    # this kind and are distinct from each other and from the prefill's token
    for seed in range(31, 47):
        prompt = synth.make_prompts(shape.vocab, 1, P, seed)
        forced = synth.uniform_int(seed, 7, shape.vocab, (1, k))
        first = int(eng.prefill(prompt)[0])
        eng.draft(k, forced=forced)
        tg, _ = eng.verify(want=True)
        base = eng.read_logits()[0].copy()
        eng.abort()
        d = eng.draft(2, want=True)[0]           # the draft head's own choices
        eng.abort()
        assert np.array_equal(tg[0], np.argmax(base, axis=1))
        rows = [i for i in range(k) if _tie_partner(int(tg[0, i]), kind) is not None]
        pd = _tie_partner(int(d[0]), kind)
        if rows and pd is not None and d[0] not in tg[0]:
            ids = {int(tg[0, rows[0]]), _tie_partner(int(tg[0, rows[0]]), kind), int(d[0]), pd, first}
            if len(ids) == 5:
                break
    else:
        raise AssertionError("no trajectory with %s partners in 16 prompts" % kind)
    eng.close()
    i = rows[0]
    pairs = [(int(tg[0, i]), _tie_partner(int(tg[0, i]), kind)), (int(d[0]), _tie_partner(int(d[0]), kind))]
    for win, low in pairs:
        w.lm_head[low] = w.lm_head[win]
        w.lora_A[low] = w.lora_A[win]
    eng, _ = gu.engine(shape, max_seq=P + 16, weights=w)
    assert int(eng.prefill(prompt)[0]) == first
    eng.draft(k, forced=forced)
    tg2, _ = eng.verify(want=True)
    lg = eng.read_logits()[0]
    for win, low in pairs:
        assert np.array_equal(lg[:, low], lg[:, win])          # the copies tie bitwise
    assert tg2[0, i] == pairs[0][1], (tg2[0, i], pairs[0])     # verify head: the lower id
    assert np.array_equal(tg2[0], np.argmax(lg, axis=1))       # numpy: first maximum
    eng.abort()
    d2 = eng.draft(2, want=True)[0]
    assert d2[0] == pairs[1][1], (d2[0], pairs[1])            # draft head (LoRA epilogue): the lower id
    dl = eng.read_draft_logits()[0]
    assert int(np.argmax(dl)) == d2[1]
    eng.close()
    # the prefill head (same kernel at another row count): make the first token tie with a lower id
    lowf = _tie_partner(first, kind)
    if lowf is not None:
        w.lm_head[lowf] = w.lm_head[first]
        eng, _ = gu.engine(shape, max_seq=P + 16, weights=w)
        assert int(eng.prefill(prompt)[0]) == lowf
        eng.close()


def test_measure_read_rate():
    """The streaming-read reference the benchmark reports beside the nominal peak: a 512 MiB buffer
    (past the 256 MB last-level cache) reads at a plausible HBM rate, below the 8 TB/s nominal
    peak; arguments it cannot use are refused."""
    import ctypes
    import torch
    from paper_2510_05421_amd._abi import ERR_ARG
    eng, _ = gu.engine(gu.SHAPES["tiny"], max_seq=64)
    rate = eng.read_rate(512 << 20, reps=3)
    _say("streaming read: %.0f GB/s" % rate)
    assert 1000.0 < rate < 8000.0
    buf = torch.empty(4 << 20, dtype=torch.uint8, device=eng.device)
    v = ctypes.c_double()
    for nbytes, reps in ((1000, 3), ((1 << 20) + 8, 3), (4 << 20, 0)):
        assert eng.status_of("dvi_measure_read_rate", buf.data_ptr(), nbytes, reps, ctypes.byref(v)) == ERR_ARG
    del buf
    eng.close()


def test_run_to_run_determinism():
    shape = gu.SHAPES["1b_L4"]
    prompt = synth.make_prompts(shape.vocab, 1, 50, 4)
    eng, _ = gu.engine(shape, max_seq=100)
    a, ia = eng.generate(prompt, 24, 5)
    la = eng.read_logits().copy()
    b, ib = eng.generate(prompt, 24, 5)
    lb = eng.read_logits()
    assert np.array_equal(a, b) and np.array_equal(la, lb)
    assert np.array_equal(ia["m"], ib["m"])
    eng.close()


def test_state_capacity_and_numeric_errors():
    from paper_2510_05421_amd._abi import DVIError, ERR_STATE, ERR_CAPACITY, ERR_ARG, ERR_NUMERIC
    shape = gu.SHAPES["tiny"]
    w = synth.make_weights(shape, 0)
    eng, _ = gu.engine(shape, max_seq=48, max_k_spec=4, weights=w)
    with pytest.raises(DVIError) as e:
        eng.draft(2)
    assert e.value.status == ERR_STATE
    eng.prefill(synth.make_prompts(shape.vocab, 1, 40, 0))
    with pytest.raises(DVIError) as e:
        eng.verify()
    assert e.value.status == ERR_STATE
    with pytest.raises(DVIError) as e:
        eng.draft(5)
    assert e.value.status == ERR_CAPACITY
    with pytest.raises(DVIError) as e:
        eng.draft(4, forced=np.array([[1, 2, 3, shape.vocab]]))
    assert e.value.status == ERR_ARG
    eng.draft(4)
    with pytest.raises(DVIError) as e:   # several steps in one call need READY as well
        eng.decode_steps(4, 1)
    assert e.value.status == ERR_STATE
    eng.abort()                          # back to READY; lengths unchanged
    assert eng.lengths()[0] == 40
    for bad_steps in (0, 65):
        with pytest.raises(DVIError) as e:
            eng.decode_steps(4, bad_steps)
        assert e.value.status == ERR_ARG
    with pytest.raises(DVIError) as e:   # checked up front: 40 + 2 steps x 4 + 4 > 48
        eng.decode_steps(4, 3)
    assert e.value.status == ERR_CAPACITY
    assert eng.lengths()[0] == 40
    tok, n, m = eng.decode_steps(4, 3, max_new=np.array([2], np.int32))  # 40 + 2 + 4 <= 48
    assert int(n.sum()) == 2 and eng.lengths()[0] == 42
    eng.draft(4)
    eng.verify()
    tok, n, m = eng.commit()
    L = 42 + int(n[0])
    while L + 4 <= 48:
        eng.draft(4)
        eng.verify()
        tok, n, m = eng.commit()
        L += int(n[0])
    with pytest.raises(DVIError) as e:   # len + k_spec > max_seq
        eng.draft(4)
    assert e.value.status == ERR_CAPACITY
    eng.close()
    # a NaN in the head makes the head's logits non-finite: the commit refuses, abort recovers
    w.lm_head = w.lm_head.copy()
    w.lm_head[7, 3] = np.nan
    eng, _ = gu.engine(shape, max_seq=64, weights=w)
    with pytest.raises(DVIError) as e:
        eng.prefill(synth.make_prompts(shape.vocab, 1, 8, 0))
    assert e.value.status == ERR_NUMERIC
    eng.draft(2)
    eng.verify()
    with pytest.raises(DVIError) as e:
        eng.commit()
    assert e.value.status == ERR_NUMERIC
    eng.abort()
    with pytest.raises(DVIError) as e:   # several steps: nothing committed from the bad step on
        eng.decode_steps(2, 3)
    assert e.value.status == ERR_NUMERIC
    assert eng.lengths()[0] == 8
    eng.draft(2)                         # the context is READY again
    eng.abort()
    eng.close()


def test_sampling_and_graph_settings_are_checked():
    """dvi_set_sampling rejects negative or non-finite temperatures and changes during a step;
    neither setting leaves the context unusable."""
    from paper_2510_05421_amd._abi import DVIError, ERR_STATE, ERR_ARG
    shape = gu.SHAPES["tiny"]
    eng, _ = gu.engine(shape, max_seq=64)
    for bad in (-1.0, float("nan"), float("inf")):
        with pytest.raises(DVIError) as e:
            eng.set_sampling(bad, 1)
        assert e.value.status == ERR_ARG
    eng.prefill(synth.make_prompts(shape.vocab, 1, 8, 0))
    eng.draft(2)
    with pytest.raises(DVIError) as e:
        eng.set_sampling(1.0, 1)
    assert e.value.status == ERR_STATE
    eng.verify()
    eng.commit()
    eng.set_sampling(0.5, 2)
    eng.set_graphs(False)
    eng.set_graphs(True)
    toks, info = eng.generate(synth.make_prompts(shape.vocab, 1, 8, 0), 12, 4)
    assert toks.shape == (1, 12)
    eng.close()


@pytest.mark.parametrize("tau", [0.0, 1.0])
def test_graph_replay_equals_direct_launches(tau):
    """Draft and verify replayed from captured HIP graphs give the tokens, accept lengths, keys,
    values and drafter updates of direct launches, bitwise.  The prompts end just before a
    256-position attention-grid bucket edge, so generation re-captures there; drafter updates,
    commits and plain-decoding steps run as direct launches between the replays."""
    shape = gu.SHAPES["7b_L4"]
    P, T, B = 236, 48, 2
    prompts = synth.make_prompts(shape.vocab, B, P, 21)
    w = synth.make_weights(shape, 0, lora_A_std=0.02)
    runs = []
    for graphs in (True, False):
        eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, weights=w)
        eng.set_graphs(graphs)
        eng.set_sampling(tau, 5)
        toks, info = eng.generate(prompts, T, 4, update_every=3)
        ar, _ = eng.generate(prompts, 12, 1)
        lens = eng.lengths().copy()
        kv = [eng.read_kv(l, b, 0, int(lens[b])) for l in range(shape.n_layers) for b in range(B)]
        lora = (eng.lora_A.cpu().numpy(), eng.lora_B.cpu().numpy())
        runs.append((toks, info, ar, kv, lora))
        _say("graphs=%s: %d steps, mean m %.2f, %d updates" % (graphs, info["steps"], info["m"].mean(),
                                                              len(info["updates"])))
        eng.close()
    (tg, ig, ag, kg, lg), (td, id_, ad, kd, ld) = runs
    assert np.array_equal(tg, td) and np.array_equal(ag, ad)
    assert np.array_equal(ig["m"], id_["m"]) and np.array_equal(ig["n"], id_["n"])
    for (k1, v1), (k2, v2) in zip(kg, kd):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    assert np.array_equal(lg[0], ld[0]) and np.array_equal(lg[1], ld[1])
    for a, b in zip(ig["updates"], id_["updates"]):
        assert a["loss"] == b["loss"] and a["rows"] == b["rows"]


@pytest.mark.parametrize("name,tau", [("tiny", 1.0), ("tiny", 0.5), ("1b_L4", 1.0)])
def test_sampled_drafts_match_oracle(name, tau):
    """Seeded stochastic drafting: each draft is the oracle's Gumbel-max draw (same generator,
    seed, step and row) wherever the oracle's perturbed scores are not near a tie; commits stay
    greedy decoding's."""
    shape = gu.SHAPES[name]
    k = KSPEC[name]
    P, T, seed = 24, 40, 11
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    prompt = synth.make_prompts(shape.vocab, 1, P, 5)[0]
    drafter = odvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma,
                           sample_tau=tau, seed=seed)
    om = oracle.OracleModel(w)
    ref = odvi.dvi_generate(om, prompt, T, k, drafter)
    ar = odvi.greedy_ar(om, prompt, T)
    assert np.array_equal(ref.tokens, ar.tokens)
    eng, _ = gu.engine(shape, max_seq=P + T + 16, weights=w)
    eng.set_sampling(tau, seed)
    toks, steps = _gpu_run(eng, prompt, T, k)
    agree, differ = 0, 0
    for st, (d, tg, m, n) in zip(ref.steps, steps):
        ok = True
        for j in range(k):
            if st.draft_gaps[j] <= 1e-3:     # a near-tie of the perturbed scores: either draw
                ok = False
                break
            assert d[j] == st.drafts[j], "step drafts %s != oracle %s" % (d, st.drafts)
            agree += 1
        if not ok:
            break
        assert m == st.m and n == st.n
        differ += int(not np.array_equal(st.drafts, st.targets))
    _say("sampled %s tau=%g: %d drafts agree with the oracle before the first near-tie" % (name, tau, agree))
    assert agree >= 2 * k
    gu.compare_free_running(toks, ar.tokens, ar.gaps)
    eng.close()


def test_sampled_drafts_use_each_sequences_own_counter_row():
    """At batch 3, sequence b's draws come from counter row b * 16 + j: its drafts are the
    oracle's draws for sequence index b (wherever the oracle's perturbed scores are not near a
    tie), and every sequence's commits stay greedy decoding's."""
    shape = gu.SHAPES["tiny"]
    B, P, T, k, seed, tau = 3, 24, 30, 4, 17, 1.0
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    prompts = synth.make_prompts(shape.vocab, B, P, 8)
    om = oracle.OracleModel(w)
    refs = [odvi.dvi_generate(om, prompts[b], T, k,
                              odvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma,
                                           sample_tau=tau, seed=seed, seq=b)) for b in range(B)]
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, weights=w)
    eng.set_sampling(tau, seed)
    first = eng.prefill(prompts)
    out = [[int(first[b])] for b in range(B)]
    live = [True] * B
    agree, step = 0, 0
    while min(len(o) for o in out) < T:
        remaining = np.array([T - len(o) for o in out], np.int32)
        d = eng.draft(k, want=True)
        eng.verify()
        tok, n, m = eng.commit(max_new=remaining)
        for b in range(B):
            if remaining[b] > 0 and live[b] and step < len(refs[b].steps):
                st = refs[b].steps[step]
                for j in range(k):
                    if st.draft_gaps[j] <= 1e-3:
                        live[b] = False
                        break
                    assert d[b, j] == st.drafts[j], (b, step, d[b], st.drafts)
                    agree += 1
                if live[b]:
                    assert (m[b], n[b]) == (st.m, st.n), (b, step)
            out[b].extend(int(t) for t in tok[b, :n[b]])
        step += 1
    for b in range(B):
        assert np.array_equal(np.array(out[b]), refs[b].tokens), b
    _say("per-sequence sampled drafts: %d drafts equal to the oracle's draws" % agree)
    assert agree >= 3 * k
    eng.close()


@pytest.mark.parametrize("name,B,k,tau", [("tiny", 3, 4, 0.0), ("1b_L4", 2, 5, 0.0), ("tiny", 2, 4, 1.0),
                                          ("tiny", 2, 1, 0.0)])
def test_decode_steps_equal_separate_calls(name, B, k, tau):
    """Steps queued by dvi_decode_steps (no host synchronisation between them, remaining-token
    limits kept on the device) give the tokens, accept lengths, lengths, caches and replay ring
    of the same steps as separate draft/verify/commit calls, bit for bit, including a sequence
    that reaches its limit in the middle of a call."""
    shape = gu.SHAPES[name]
    P, S = 20, 12
    prompts = synth.make_prompts(shape.vocab, B, P, 13)
    w = synth.make_weights(shape, 0, lora_A_std=0.03)
    limits = np.array([S * k, 5, 17][:B], np.int32)

    def run(multi):
        eng, _ = gu.engine(shape, max_batch=B, max_seq=P + S * k + 16, weights=w, buffer_rows=64)
        if tau > 0:
            eng.set_sampling(tau, 5)
        eng.prefill(prompts)
        left = limits.copy()
        toks, ns, ms = [], [], []
        if multi:
            for cnt in (5, S - 5):
                t, n, m = eng.decode_steps(k, cnt, max_new=left)
                toks += list(t)
                ns += list(n)
                ms += list(m)
                left = left - n.sum(axis=0)
        else:
            for _ in range(S):
                eng.draft(k)
                eng.verify()
                t, n, m = eng.commit(max_new=left)
                toks.append(t)
                ns.append(n)
                ms.append(m)
                left = left - n
        lens = eng.lengths()
        kv = [eng.read_kv(l, b, 0, int(lens[b])) for l in (0, shape.n_layers - 1) for b in range(B)]
        valid, nxt = eng.buffer_info()
        ring = eng.read_buffer(0, valid) if valid else None
        eng.close()
        return np.array(toks), np.array(ns), np.array(ms), lens, kv, (valid, nxt), ring

    a_ = run(False)
    b_ = run(True)
    for x, y in zip(a_[:4], b_[:4]):
        assert np.array_equal(x, y)
    assert np.array_equal(a_[1].sum(axis=0), np.minimum(limits, a_[1].sum(axis=0)))
    assert int(a_[1][:, 1].sum()) == 5  # the second sequence stops at its limit
    for (k1, v1), (k2, v2) in zip(a_[4], b_[4]):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    assert a_[5] == b_[5]
    if a_[6] is not None:
        for key in a_[6]:
            assert np.array_equal(a_[6][key], b_[6][key]), key


def test_sampled_drafting_is_lossless_and_changes_drafts():
    """With sampled drafts, speculative decoding still equals greedy decoding bitwise (tokens
    and keys/values); the accept lengths differ from argmax drafting."""
    shape = gu.SHAPES["7b_L4"]
    P, T, B = 60, 48, 2
    prompts = synth.make_prompts(shape.vocab, B, P, 31)
    w = synth.make_weights(shape, 0, lora_A_std=0.02)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + 16, weights=w)
    greedy_tok, greedy_info = eng.generate(prompts, T, 4)
    eng.set_sampling(1.0, 99)
    samp_tok, samp_info = eng.generate(prompts, T, 4)
    kv_s = [eng.read_kv(l, b, 0, P + T - 1) for l in (1, 3) for b in range(B)]
    eng.set_sampling(0.0)
    ar_tok, _ = eng.generate(prompts, T, 1)
    kv_a = [eng.read_kv(l, b, 0, P + T - 1) for l in (1, 3) for b in range(B)]
    assert np.array_equal(samp_tok, ar_tok) and np.array_equal(greedy_tok, ar_tok)
    for (k1, v1), (k2, v2) in zip(kv_s, kv_a):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    _say("sampled drafting: mean m %.2f vs argmax drafting %.2f" % (samp_info["m"].mean(), greedy_info["m"].mean()))
    assert samp_info["steps"] != greedy_info["steps"] or not np.array_equal(samp_info["m"], greedy_info["m"])
    eng.close()


@pytest.mark.parametrize("B,P,k", [(4, 1, 16), (1, 1, 16), (64, 8, 1), (16, 3, 4)])
def test_edge_shapes_are_lossless(B, P, k):
    """Degenerate and maximum shapes: one-token prompts, the largest k_spec (16), the widest
    block (4 x 16 = 64 rows) and the widest batch (64 sequences): speculative decoding equals
    greedy decoding bitwise, up to the last position of the cache, and sequence 0 agrees with
    the oracle."""
    shape = gu.SHAPES["tiny"]
    T = 40
    prompts = synth.make_prompts(shape.vocab, B, P, 13)
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    max_seq = P + T + k          # a step may write k_spec positions past the last committed token
    eng, _ = gu.engine(shape, max_batch=B, max_seq=max_seq, max_k_spec=k, weights=w)
    spec, info = eng.generate(prompts, T, k)
    lens = eng.lengths().copy()
    kv = [eng.read_kv(l, b, 0, int(lens[b])) for l in (0, shape.n_layers - 1) for b in (0, B - 1)]
    ar, _ = eng.generate(prompts, T, 1)
    assert np.array_equal(spec, ar)
    kv_ar = [eng.read_kv(l, b, 0, int(lens[b])) for l in (0, shape.n_layers - 1) for b in (0, B - 1)]
    for (k1, v1), (k2, v2) in zip(kv, kv_ar):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    ref = odvi.greedy_ar(oracle.OracleModel(w), prompts[0], T)
    agree = gu.compare_free_running(spec[0], ref.tokens, ref.gaps)
    _say("edge B=%d P=%d k_spec=%d: %d steps, mean m %.2f, %d/%d tokens agree with the oracle"
         % (B, P, k, info["steps"], info["m"].mean(), agree, T))
    eng.close()


@pytest.mark.parametrize("name,B,k", [("7b_L4", 5, 8), ("tiny", 3, 13)])
def test_ragged_verify_blocks_are_lossless(name, B, k):
    """Verify blocks of 33-48 rows that fill neither their last 16-row group nor every wave's
    share of rows (5 x 8 = 40 in bf16, 3 x 13 = 39 in fp32): the decode GEMMs' three-group path,
    with its folded-norm partial sums requested several rows at a time, gives the bits of greedy
    decoding's one row per sequence, tokens and cache alike."""
    shape = gu.SHAPES[name]
    T, P = 24, 21
    prompts = synth.make_prompts(shape.vocab, B, P, 17)
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + T + k, max_k_spec=k, weights=w)
    spec, info = eng.generate(prompts, T, k)
    lens = eng.lengths().copy()
    layers = (shape.split_k, shape.n_layers - 1)
    kv = [eng.read_kv(l, b, 0, int(lens[b])) for l in layers for b in (0, B - 1)]
    ar, _ = eng.generate(prompts, T, 1)
    assert np.array_equal(spec, ar)
    kv_ar = [eng.read_kv(l, b, 0, int(lens[b])) for l in layers for b in (0, B - 1)]
    for (k1, v1), (k2, v2) in zip(kv, kv_ar):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    _say("ragged verify %s B=%d k_spec=%d (%d rows): %d steps, mean m %.2f"
         % (name, B, k, B * k, info["steps"], info["m"].mean()))
    eng.close()


@pytest.mark.parametrize("name,r", [("tiny", 4), ("tiny", 6), ("tiny", 24), ("tiny", 64), ("1b_L4", 8),
                                    ("1b_L4", 20)])
def test_draft_head_logits_at_other_lora_ranks(name, r):
    """The draft head's logits W^V h + gamma A_s (B_s h) against the oracle at LoRA ranks other
    than the workloads' 16: multiples of 4 up to 16 take the epilogue's register path, the others
    read A_s and u from memory.  The position checked is the second draft, whose input token is
    forced, so both sides run the same sequence."""
    shape = gu.SHAPES[name].replace(lora_rank=r)
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    P = 12
    prompt = synth.make_prompts(shape.vocab, 1, P, 3)[0]
    _say("draft head %s lora_rank=%d" % (name, r))
    eng, _ = gu.engine(shape, max_seq=P + 8, weights=w)
    first = int(eng.prefill(prompt[None])[0])
    f0 = (first * 7 + 3) % shape.vocab
    eng.draft(2, forced=np.array([[f0, 1]], np.int32))
    got = eng.read_draft_logits()[0]
    eng.close()
    om = oracle.OracleModel(w)
    cache = om.new_cache(P + 4)
    om.layers(cache, om.embed(prompt), 0, 0, shape.n_layers)
    om.layers(cache, om.embed([first]), P, 0, shape.split_k)
    hn = om.final_norm(om.layers(cache, om.embed([f0]), P + 1, 0, shape.split_k))
    A, B = w.lora_A.astype(np.float64), w.lora_B.astype(np.float64)
    ref = om.draft_logits(hn, A, B, shape.lora_gamma)[0]
    plain = om.draft_logits(hn, np.zeros_like(A), B, shape.lora_gamma)[0]
    e, em = gu.check_close(got, ref, shape, "draft logits")
    _say("  relative L2 error %.3g, elementwise %.3g (the LoRA term moves the logits by %.3g)"
         % (e, em, gu.rel_l2(plain, ref)))
    assert gu.rel_l2(plain, ref) > 5 * gu.tol(shape)


@pytest.mark.parametrize("name,P", [("tiny", 70), ("1b_L4", 66), ("7b_L4", 66)])
def test_cache_keys_and_values_match_the_oracle(name, P):
    """The cache's keys (after the rotary embedding) and values at every committed position,
    read back through the ABI, equal the oracle's cache for the same tokens within the storage
    tolerance.  The prompt crosses a 64-position block boundary, and decoding writes on both
    sides of it."""
    shape = gu.SHAPES[name]
    T = 8
    w = synth.make_weights(shape, 0, lora_A_std=0.05)
    prompt = synth.make_prompts(shape.vocab, 1, P, 17)[0]
    eng, _ = gu.engine(shape, max_seq=P + T + 8, weights=w)
    toks, _ = eng.generate(prompt[None], T, KSPEC[name])
    n = int(eng.lengths()[0])            # positions whose keys/values are committed
    assert n == P + T - 1
    got = [eng.read_kv(l, 0, 0, n) for l in range(shape.n_layers)]
    eng.close()
    seq = np.concatenate([prompt, toks[0]])[:n]
    om = oracle.OracleModel(w)
    cache = om.new_cache(n)
    om.layers(cache, om.embed(seq), 0, 0, shape.n_layers)
    worst = worstm = 0.0
    for l, (k, v) in enumerate(got):
        # oracle [n, n_kv * hd] -> [n_kv, n, hd], the ABI's order
        ko = cache[0][l].reshape(n, shape.n_kv_heads, shape.head_dim).transpose(1, 0, 2)
        vo = cache[1][l].reshape(n, shape.n_kv_heads, shape.head_dim).transpose(1, 0, 2)
        for nm, got_x, ref_x in (("keys", k, ko), ("values", v, vo)):
            gx = synth.bf16_bits_to_f32(got_x) if got_x.dtype == np.uint16 else got_x
            # every (kv head, position) row: L2 and elementwise bounds against the oracle row
            for h in range(shape.n_kv_heads):
                e2, em = gu.check_close(gx[h], ref_x[h], shape, "layer %d kv head %d %s" % (l, h, nm))
                worst, worstm = max(worst, e2), max(worstm, em)
                # and each position's vector on its own: a wrong slot in one block shows here
                pe = np.max(np.abs(gx[h].astype(np.float64) - ref_x[h]), axis=1) / np.max(np.abs(ref_x[h]), axis=1)
                assert np.all(pe <= gu.tol(shape)), "layer %d kv head %d %s: position %d error %.3g" % (
                    l, h, nm, int(np.argmax(pe)), float(pe.max()))
    _say("cache %s P=%d: %d positions, worst relative L2 error %.3g, elementwise %.3g" % (name, P, n, worst, worstm))
