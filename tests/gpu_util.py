"""Helpers shared by the GPU parity tests (engine construction, comparison rules)."""
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TIE_GAP = 5e-2          # oracle top-2 gaps at or below this are near-ties: either token is acceptable
TOL_FP32 = 1e-4         # per-row relative L2 error of logits, fp32 storage
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


def teacher_forced(eng, prompt, tokens, k_spec, n_rows):
    """Follow the oracle's committed sequence: drafts and commits forced to it.  Returns
    (prefill logits row, list of (token index, GPU logits row, GPU argmax))."""
    first = eng.prefill(prompt[None])
    pre = eng.read_logits()[0, 0]
    rows = [(0, pre, int(first[0]))]
    c = 1
    while c < n_rows and c + k_spec <= len(tokens):
        want = tokens[c:c + k_spec]
        eng.draft(k_spec, forced=want[None])
        tg, m = eng.verify(want=True)
        lg = eng.read_logits()[0]
        for i in range(k_spec):
            if c + i < n_rows:
                rows.append((c + i, lg[i], int(tg[0, i])))
        tok, n, m2 = eng.commit(forced=want[None])
        assert n[0] == k_spec and m2[0] == k_spec
        c += k_spec
    return rows
