"""Helpers shared by the GPU parity tests (engine construction, comparison rules)."""
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TIE_GAP = 5e-2          # oracle top-2 gaps at or below this are near-ties: either token is acceptable
# Logits tolerances (relative), applied twice to every compared row: the row's L2 error over the
# oracle row's L2 norm, and every element's error over the oracle row's largest magnitude.
TOL_FP32 = 1e-4         # fp32 storage
TOL_BF16 = 2e-2         # bf16 storage

SHAPES = {
    "tiny": synth.TINY,
    "1b_L4": synth.shrunk(synth.SHAPE_1B),
    "7b_L4": synth.shrunk(synth.SHAPE_7B),
    "13b_L4": synth.shrunk(synth.SHAPE_13B),
    "1b": synth.SHAPE_1B,
    "7b": synth.SHAPE_7B,
    "13b": synth.SHAPE_13B,
    "7b_b8_s0": synth.SHAPE_7B,
    "7b_b8_s7": synth.SHAPE_7B,
}


def golden(name):
    z = np.load(os.path.join(GOLDEN, name + ".npz"))
    return {k: z[k] for k in z.files}


def tol(shape):
    return TOL_BF16 if shape.bf16 else TOL_FP32


def engine(shape, max_batch=1, max_seq=256, max_k_spec=8, buffer_rows=256, weights=None, lora_A_std=0.0):
    from paper_2510_05421_amd.engine import Engine, EngineConfig
    w = weights if weights is not None else synth.make_weights(shape, 0, lora_A_std=lora_A_std)
    cfg = EngineConfig.from_shape(shape, max_batch=max_batch, max_seq=max_seq, max_k_spec=max_k_spec,
                                  buffer_rows=buffer_rows)
    return Engine(cfg, w, "cuda:0"), w


def compare_free_running(got, ref_tokens, ref_gaps):
    """Tokens must agree until the first disagreement, and that disagreement (if any) must sit
    at an oracle near-tie.  Returns the number of agreeing tokens."""
    n = min(len(got), len(ref_tokens))
    for i in range(n):
        if got[i] != ref_tokens[i]:
            assert ref_gaps[i] <= TIE_GAP, (
                "token %d: GPU %d != oracle %d with oracle top-2 gap %.4g > %.3g"
                % (i, got[i], ref_tokens[i], ref_gaps[i], TIE_GAP))
            return i
    return n


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def rel_max(a, b):
    """Largest elementwise error over the reference's largest magnitude."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


def check_close(got, ref, shape, what):
    """Row-L2 and elementwise bounds (see TOL_*); returns (row L2 error, elementwise error)."""
    t = tol(shape)
    e2, em = rel_l2(got, ref), rel_max(got, ref)
    assert e2 <= t, "%s: relative L2 error %.3g > %.3g" % (what, e2, t)
    assert em <= t, "%s: largest elementwise error %.3g of max|ref| > %.3g" % (what, em, t)
    return e2, em


def teacher_forced(eng, prompts, tokens, k_spec):
    """Follow the oracle's committed sequences (prompts [B, P], tokens [B, T]): drafts and commits
    are forced to them, k_spec at a time (fewer on the last step), so every token's target-head
    logits are computed.  Returns a list of (token index, GPU logits [B, V], GPU argmax [B]), one
    entry per token index 0..T-1 (index 0: the prefill's head)."""
    prompts = np.atleast_2d(prompts)
    tokens = np.atleast_2d(tokens)
    B, T = tokens.shape
    first = eng.prefill(prompts)
    rows = [(0, eng.read_logits()[:, 0].copy(), np.asarray(first).copy())]
    c = 1
    while c < T:
        k = min(k_spec, T - c)
        want = np.ascontiguousarray(tokens[:, c:c + k])
        eng.draft(k, forced=want)
        tg, m = eng.verify(want=True)
        lg = eng.read_logits()
        for i in range(k):
            rows.append((c + i, lg[:, i].copy(), tg[:, i].copy()))
        tok, n, m2 = eng.commit(forced=want)
        assert np.all(n == k) and np.all(m2 == k)
        c += k
    return rows


def check_teacher_forced(rows, ref_logits, ref_tokens, ref_gaps, shape):
    """Every row's logits within the storage tolerance (row L2 and elementwise) and its argmax
    equal to the oracle's wherever the oracle is not near a tie.  ref_* are [B, T, ...]."""
    worst2 = worstm = 0.0
    checked = 0
    for idx, lg, am in rows:
        for b in range(lg.shape[0]):
            e2, em = check_close(lg[b], ref_logits[b][idx], shape, "sequence %d token %d" % (b, idx))
            worst2, worstm = max(worst2, e2), max(worstm, em)
            if ref_gaps[b][idx] > TIE_GAP:
                assert am[b] == ref_tokens[b][idx], "sequence %d token %d: argmax %d != oracle %d" % (
                    b, idx, am[b], ref_tokens[b][idx])
            checked += 1
    return worst2, worstm, checked
