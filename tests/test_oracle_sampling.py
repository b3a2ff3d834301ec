"""Pins of the oracle's seeded stochastic drafting (oracle/sampling.py): the generator against
numpy's own Philox bit generator, the Gumbel-max draw against softmax(z / tau), and
losslessness of the DVI rollout with sampled drafts."""
import numpy as np
import pytest
from scipy import stats

import oracle
import synth
from oracle import dvi as odvi
from oracle import sampling as sp



@pytest.mark.parametrize("ctr", [(0, 0, 0, 0), (5, 7, 9, 11), (123456789, 42, 3, 0), (2**64 - 2, 1, 0, 2**40)])
@pytest.mark.parametrize("key", [(0, 0), (123, 456), (2**63 + 5, 2**33)])
def test_philox_equals_numpy_bit_generator(ctr, key):
    # numpy's Philox (4 x 64-bit words, 10 rounds) advances its counter before each block:
    # its first block from counter c is the generator's block c + 1
    bg = np.random.Philox(counter=np.array(ctr, dtype=np.uint64), key=np.array(key, dtype=np.uint64))
    raw = [int(x) for x in bg.random_raw(8)]
    value = sum(int(c) << (64 * i) for i, c in enumerate(ctr))   # the 256-bit counter
    for blk in range(2):
        v = (value + 1 + blk) % 2**256
        words = [np.uint64((v >> (64 * i)) & (2**64 - 1)) for i in range(4)]
        mine = sp.philox4x64(*words, *key)
        assert [int(x) for x in mine] == raw[4 * blk:4 * blk + 4]


def test_uniforms_inside_unit_interval_and_distinct_streams():
    u = sp.uniforms(4096, 9, np.arange(8), 3)
    assert u.shape == (8, 4096) and u.min() > 0.0 and u.max() < 1.0
    # different rows, steps and seeds give different streams
    assert not np.array_equal(sp.uniforms(64, 9, 0, 3), sp.uniforms(64, 9, 0, 4))
    assert not np.array_equal(sp.uniforms(64, 9, 0, 3), sp.uniforms(64, 9, 1, 3))
    assert not np.array_equal(sp.uniforms(64, 9, 0, 3), sp.uniforms(64, 10, 0, 3))
    # roughly uniform: Kolmogorov-Smirnov against U(0, 1)
    assert stats.kstest(u.reshape(-1), "uniform").pvalue > 1e-3


@pytest.mark.parametrize("tau", [0.5, 1.0, 2.0])
def test_gumbel_max_draws_from_softmax(tau):
    z = np.array([1.0, -0.5, 0.3, 2.0, 0.0, -1.2])
    n = 40000
    scores = z[None, :] / tau + -np.log(-np.log(sp.uniforms(z.size, 17, np.arange(n), 1)))
    counts = np.bincount(np.argmax(scores, axis=1), minlength=z.size)
    p = np.exp(z / tau - (z / tau).max())
    p /= p.sum()
    assert stats.chisquare(counts, n * p).pvalue > 1e-3
    # the scores of one draft are the same function sample_scores computes
    assert np.array_equal(sp.sample_scores(z, tau, 17, 5, 1), scores[5])


def test_rollout_with_sampled_drafts_is_lossless():
    w = synth.make_weights(synth.TINY, 0, lora_A_std=0.05)
    om = oracle.OracleModel(w)
    prompt = synth.make_prompts(synth.TINY.vocab, 1, 16, 2)[0]
    ar = odvi.greedy_ar(om, prompt, 24)
    greedy = odvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), 1.0)
    sampled = odvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), 1.0, sample_tau=1.0, seed=3)
    rg = odvi.dvi_generate(om, prompt, 24, 4, greedy)
    rs = odvi.dvi_generate(om, prompt, 24, 4, sampled)
    assert np.array_equal(rs.tokens, ar.tokens) and np.array_equal(rg.tokens, ar.tokens)
    # sampling changes the drafts (and so the accept lengths) on some steps
    assert any(not np.array_equal(a.drafts, b.drafts) for a, b in zip(rg.steps, rs.steps))
