"""GPU parity at the full model sizes, in the launch configuration the benchmark times.

The oracle's goldens (tests/golden/{1b,7b,13b,7b_b8_s0..s7}.npz) cover the first 128, 128, 64
and 16 tokens of each workload, with the target-head logits of every one; past them, the
committed output is checked against its definition on the GPU itself: speculative decoding must
commit exactly the tokens of plain greedy decoding (k_spec = 1 on the same engine, whose kernels
give each row the same arithmetic whatever block it sits in) with bitwise-equal keys and values.
The drafter update is checked against the oracle's gradient on a replay ring that the decode
loop itself filled at the 13B shape."""
import dataclasses
import os

import numpy as np
import pytest

import synth
from oracle import update as oupd
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# golden name -> workload k_spec
FULL = {"1b": 5, "7b": 4, "13b": 6}


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def weights_cache():
    cache = {}
    yield cache
    cache.clear()


def _weights(cache, shape):
    key = shape.replace(name="", split_k=1)  # the weights depend on the dimensions only
    if key not in cache:
        cache.clear()
        cache[key] = synth.make_weights(shape, 0)
    return cache[key]


@pytest.mark.parametrize("name", list(FULL))
def test_fullsize_tokens_and_logits_match_oracle(name, weights_cache):
    """Free-running tokens agree with the oracle up to its first near-tie, and teacher-forced
    through every golden token, each verify row's logits are within the bf16 tolerance (row L2
    and every element) with the oracle's argmax away from ties."""
    g = gu.golden(name)
    shape = gu.SHAPES[name]
    P, T = g["prompt"].size, g["tokens"].size
    assert g["logits"].shape[0] == T
    k = FULL[name]
    _say("full-size %s: P=%d, %d oracle tokens, k_spec=%d" % (name, P, T, k))
    eng, _ = gu.engine(shape, max_seq=P + T + 16, weights=_weights(weights_cache, shape))
    toks, info = eng.generate(g["prompt"][None], T, k)
    agree = gu.compare_free_running(toks[0], g["tokens"], g["gaps"])
    _say("  %d/%d tokens agree before the first (near-tie) divergence; mean m %.2f" % (agree, T, info["m"].mean()))
    rows = gu.teacher_forced(eng, g["prompt"], g["tokens"], k)
    assert [r[0] for r in rows] == list(range(T))
    w2, wm, n = gu.check_teacher_forced(rows, g["logits"][None], g["tokens"][None], g["gaps"][None], shape)
    _say("  %d rows: worst relative L2 error %.3g, worst elementwise error %.3g of max|z|" % (n, w2, wm))
    eng.close()


def _kv_layers(shape):
    return sorted({0, shape.split_k - 1, shape.split_k, shape.n_layers - 1})


def _check_lossless(eng, shape, prompts, n_new, k_specs, update_every=0):
    B, P = prompts.shape
    ar, _ = eng.generate(prompts, n_new, 1)
    lens = eng.lengths().copy()
    assert np.all(lens == P + n_new - 1)
    kv_ar = {l: [eng.read_kv(l, b, 0, int(lens[b])) for b in range(B)] for l in _kv_layers(shape)}
    for k in k_specs:
        spec, info = eng.generate(prompts, n_new, k, update_every=update_every)
        same = np.array_equal(spec, ar)
        _say("  k_spec=%d: %d steps, mean m %.2f, tokens/step %.2f, identical to greedy: %s%s"
             % (k, info["steps"], info["m"].mean(), info["n"].sum() / (info["steps"] * B), same,
                ", %d drafter updates" % len(info["updates"]) if info["updates"] else ""))
        if not same:
            b, i = np.argwhere(spec != ar)[0]
            raise AssertionError("k_spec=%d: sequence %d token %d: %d != greedy %d" % (k, b, i, spec[b, i], ar[b, i]))
        assert np.array_equal(eng.lengths(), lens)
        for l, ref in kv_ar.items():
            for b in range(B):
                kk, vv = eng.read_kv(l, b, 0, int(lens[b]))
                assert np.array_equal(kk, ref[b][0]) and np.array_equal(vv, ref[b][1]), (k, l, b)
        for st in info["updates"]:
            assert np.isfinite(st["loss"]) and st["rows"] > 0
    return ar


@pytest.mark.parametrize("wl", ["1b", "7b", "7b_k2", "13b"])
def test_fullsize_speculative_equals_greedy(wl, weights_cache):
    """Every full workload (prompt length, new tokens, k_spec) commits greedy decoding's tokens
    and keys/values bitwise; the 13B workload runs its drafter update every 8 steps.  7b_k2 is
    the 7B model (same weights) split after layer 2: its greedy output is the 7B golden's."""
    W = synth.WORKLOADS[wl]
    shape = W.model
    k_specs = W.k_spec
    prompts = synth.make_prompts(shape.vocab, W.batch, W.prompt_len, 0)
    _say("lossless %s: B=%d P=%d N=%d k_spec %s update_every=%d"
         % (wl, W.batch, W.prompt_len, W.new_tokens, k_specs, W.update_every))
    eng, _ = gu.engine(shape, max_batch=W.batch, max_seq=W.prompt_len + W.new_tokens + 8,
                       weights=_weights(weights_cache, shape))
    ar = _check_lossless(eng, shape, prompts, W.new_tokens, k_specs, update_every=W.update_every)
    gname = {"7b_k2": "7b"}.get(wl, wl)
    if gname in FULL:
        g = gu.golden(gname)
        assert np.array_equal(g["prompt"], prompts[0])
        gu.compare_free_running(ar[0], g["tokens"], g["gaps"])
    eng.close()


def test_fullsize_batch8_long_prompts(weights_cache):
    """7B shape, 8 sequences of 2048 prompt tokens, 256 new tokens, k_spec 8: per-sequence
    accept lengths differ, the committed output is greedy decoding's for every sequence, and
    every sequence agrees with the oracle; teacher-forced through each sequence's 16 golden
    tokens at batch 8, every verify row's logits are within the bf16 tolerance."""
    W = synth.WORKLOADS["7b_b8"]
    shape = W.model
    prompts = synth.make_prompts(shape.vocab, W.batch, W.prompt_len, 0)
    _say("lossless 7b_b8: B=%d P=%d N=%d k_spec=%s" % (W.batch, W.prompt_len, W.new_tokens, W.k_spec))
    eng, _ = gu.engine(shape, max_batch=W.batch, max_seq=W.prompt_len + W.new_tokens + 8,
                       weights=_weights(weights_cache, shape))
    ar = _check_lossless(eng, shape, prompts, W.new_tokens, W.k_spec)
    gs = [gu.golden("7b_b8_s%d" % b) for b in range(W.batch)]
    for b, g in enumerate(gs):
        assert np.array_equal(g["prompt"], prompts[b])
        agree = gu.compare_free_running(ar[b], g["tokens"], g["gaps"])
        _say("  sequence %d: %d/%d oracle tokens agree" % (b, agree, g["tokens"].size))
    T = gs[0]["tokens"].size
    rows = gu.teacher_forced(eng, prompts, np.stack([g["tokens"] for g in gs]), W.k_spec[0])
    assert [r[0] for r in rows] == list(range(T))
    w2, wm, n = gu.check_teacher_forced(rows, [g["logits"] for g in gs], [g["tokens"] for g in gs],
                                        [g["gaps"] for g in gs], shape)
    _say("  teacher-forced at batch 8: %d rows, worst relative L2 %.3g, elementwise %.3g" % (n, w2, wm))
    eng.close()


def _forced_accept_run(eng, prompts, ar, k, V):
    """Decode with every draft block forced to greedy decoding's continuation, the draft at
    index j = (step + sequence) mod (k+1) made wrong (none when j = k): every accept length
    m = 0..k goes through the commit kernel.  Returns (tokens [B, T], accept lengths [steps, B])."""
    B, T = ar.shape
    first = eng.prefill(prompts)
    out = [[int(t)] for t in first]
    ms, step = [], 0
    while min(len(o) for o in out) < T:
        forced = np.zeros((B, k), np.int32)
        for b in range(B):
            c = len(out[b])
            nxt = np.concatenate([ar[b, c:c + k], np.zeros(k, np.int32)])[:k].copy()
            j = (step + b) % (k + 1)
            if j < k:
                nxt[j] = (nxt[j] + 1) % V
            forced[b] = nxt
        eng.draft(k, forced=forced)
        eng.verify()
        tok, n, m = eng.commit(max_new=np.array([T - len(o) for o in out], np.int32))
        for b in range(B):
            out[b].extend(int(t) for t in tok[b, :n[b]])
        ms.append(m.copy())
        step += 1
    return np.array(out, np.int32), np.array(ms)


@pytest.mark.parametrize("wl,n_new", [("7b", 160), ("13b", 120)])
def test_fullsize_every_accept_length_is_lossless(wl, n_new, weights_cache):
    """At the full shapes (not just the random-weight trajectories, whose drafts are rarely
    right), drafts forced to the greedy continuation with one wrong position per step send every
    accept length 0..k_spec through commit and rollback: the output is greedy decoding's and the
    committed keys/values are bitwise those of greedy decoding."""
    W = synth.WORKLOADS[wl]
    shape = W.model
    k = W.k_spec[0]
    prompts = synth.make_prompts(shape.vocab, 1, W.prompt_len, 0)
    _say("forced accept lengths %s: P=%d N=%d k_spec=%d" % (wl, W.prompt_len, n_new, k))
    eng, _ = gu.engine(shape, max_seq=W.prompt_len + n_new + 16, weights=_weights(weights_cache, shape))
    ar, _ = eng.generate(prompts, n_new, 1)
    n_kv = int(eng.lengths()[0])
    kv_ar = {l: eng.read_kv(l, 0, 0, n_kv) for l in _kv_layers(shape)}
    toks, ms = _forced_accept_run(eng, prompts, ar, k, shape.vocab)
    assert np.array_equal(toks, ar)
    seen = set(int(x) for x in ms[:-2, 0])
    _say("  %d steps, accept lengths seen %s" % (len(ms), sorted(seen)))
    assert seen == set(range(k + 1))
    assert int(eng.lengths()[0]) == n_kv
    for l, (k0, v0) in kv_ar.items():
        k1, v1 = eng.read_kv(l, 0, 0, n_kv)
        assert np.array_equal(k1, k0) and np.array_equal(v1, v0), "layer %d" % l
    eng.close()


def test_fullsize_13b_update_on_a_decoded_ring(weights_cache):
    """Drafter update at the 13B shape on a 256-row replay ring filled by the decode loop itself
    (forced drafts give every accept length, so accepted and rejected rows both occur; one update
    in between clears the fresh flags of the older rows): the ring is read back through the ABI
    and the GPU's dA, dB and loss terms match the oracle's on those rows."""
    W = synth.WORKLOADS["13b"]
    shape = W.model
    k = W.k_spec[0]
    base = _weights(weights_cache, shape)
    w = dataclasses.replace(base, lora_A=synth.normal(0, synth.S_LORA_A, 0.02, (shape.vocab, shape.lora_rank), False))
    prompts = synth.make_prompts(shape.vocab, 1, W.prompt_len, 0)
    n_new = 400
    _say("13b update on a decoded ring: P=%d, k_spec=%d" % (W.prompt_len, k))
    eng, _ = gu.engine(shape, max_seq=W.prompt_len + n_new + 16, buffer_rows=256, weights=w)
    ar, _ = eng.generate(prompts, n_new, 1)
    first = eng.prefill(prompts)
    out, step, updated = [int(first[0])], 0, False
    c = oupd.Coeffs(c_kl=0.8, c_ce=0.6, c_pg=0.5, c_ent=0.02, tau=1.0, baseline=0.3)
    while True:
        valid, _ = eng.buffer_info()
        if updated and valid >= 256:
            break
        if not updated and valid >= 100:
            eng.update_drafter(c.c_kl, c.c_ce, c.c_pg, c.c_ent, c.tau, c.baseline, lr=0.0)  # clears fresh
            updated = True
        cpos = len(out)
        assert cpos + k < n_new, "ring not full before the greedy continuation ran out"
        nxt = ar[0, cpos:cpos + k].copy()
        j = step % (k + 1)
        if j < k:
            nxt[j] = (nxt[j] + 1) % shape.vocab
        eng.draft(k, forced=nxt[None])
        eng.verify()
        tok, n, m = eng.commit()
        out.extend(int(t) for t in tok[0, :n[0]])
        step += 1
    assert np.array_equal(np.array(out), ar[0, :len(out)])
    buf = eng.read_buffer(0, 256)
    assert 0 < buf["r"].sum() < 256 and 0 < buf["fresh"].sum() < 256
    st = eng.update_drafter(c.c_kl, c.c_ce, c.c_pg, c.c_ent, c.tau, c.baseline, lr=0.0, grads=True)
    Wv = w.as_f32(w.lm_head).astype(np.float64)
    ref = oupd.loss_and_grad(Wv, w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma,
                             buf["h"].astype(np.float64), buf["a"], buf["logits"], buf["r"], buf["fresh"], c)
    dA, dB = st["grad_A"].cpu().numpy(), st["grad_B"].cpu().numpy()
    eA, eB = gu.rel_l2(dA, ref.dA), gu.rel_l2(dB, ref.dB)
    _say("  %d steps, %d accepted / %d fresh rows: |dA| rel err %.3g, |dB| rel err %.3g, loss %.6g vs %.6g"
         % (step, int(buf["r"].sum()), int(buf["fresh"].sum()), eA, eB, st["loss"], ref.loss))
    assert eA <= 1e-2 and eB <= 1e-2
    assert st["rows"] == 256 and st["accepted"] == int(buf["r"].sum()) and st["fresh"] == int(buf["fresh"].sum())
    for key in ("kl", "ce", "pg", "entropy"):
        assert abs(st[key] - getattr(ref, key)) <= 1e-3 * max(1.0, abs(getattr(ref, key))), key
    eng.close()
