"""GPU parity at the full model sizes, in the launch configuration the benchmark times.

The oracle's goldens (tests/golden/{1b,7b,13b,7b_b8_s0,7b_b8_s7}.npz) cover the first tokens of
each workload; past them, the committed output is checked against its definition on the GPU
itself: speculative decoding must commit exactly the tokens of plain greedy decoding (k_spec = 1
on the same engine, whose kernels give each row the same arithmetic whatever block it sits in)
with bitwise-equal keys and values."""
import os

import numpy as np
import pytest

import synth
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
    g = gu.golden(name)
    shape = gu.SHAPES[name]
    P, T, R = g["prompt"].size, g["tokens"].size, g["logits"].shape[0]
    k = FULL[name]
    _say("full-size %s: P=%d, %d oracle tokens, k_spec=%d" % (name, P, T, k))
    eng, _ = gu.engine(shape, max_seq=P + T + 16, weights=_weights(weights_cache, shape))
    toks, info = eng.generate(g["prompt"][None], T, k)
    agree = gu.compare_free_running(toks[0], g["tokens"], g["gaps"])
    _say("  %d/%d tokens agree before the first (near-tie) divergence; mean m %.2f" % (agree, T, info["m"].mean()))
    rows = gu.teacher_forced(eng, g["prompt"], g["tokens"], k, R)
    worst = 0.0
    for idx, lg, am in rows:
        e = gu.rel_l2(lg, g["logits"][idx])
        worst = max(worst, e)
        assert e <= gu.tol(shape), "row %d: relative L2 error %.3g" % (idx, e)
        if g["gaps"][idx] > gu.TIE_GAP:
            assert am == g["tokens"][idx]
    _say("  worst relative L2 logits error %.3g over %d rows" % (worst, len(rows)))
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
    sequences 0 and 7 agree with the oracle."""
    W = synth.WORKLOADS["7b_b8"]
    shape = W.model
    prompts = synth.make_prompts(shape.vocab, W.batch, W.prompt_len, 0)
    _say("lossless 7b_b8: B=%d P=%d N=%d k_spec=%s" % (W.batch, W.prompt_len, W.new_tokens, W.k_spec))
    eng, _ = gu.engine(shape, max_batch=W.batch, max_seq=W.prompt_len + W.new_tokens + 8,
                       weights=_weights(weights_cache, shape))
    ar = _check_lossless(eng, shape, prompts, W.new_tokens, W.k_spec)
    for b in (0, 7):
        path = os.path.join(gu.GOLDEN, "7b_b8_s%d.npz" % b)
        if not os.path.exists(path):
            continue
        g = gu.golden("7b_b8_s%d" % b)
        assert np.array_equal(g["prompt"], prompts[b])
        agree = gu.compare_free_running(ar[b], g["tokens"], g["gaps"])
        _say("  sequence %d: %d/%d oracle tokens agree" % (b, agree, g["tokens"].size))
    eng.close()
