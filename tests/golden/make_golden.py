"""Write the oracle's expected values for the GPU parity tests.

Calls only the CPU oracle (oracle/) on seeded synthetic inputs (synth/); nothing here reads
GPU output.  Each file holds, for one model shape and prompt:
  tokens  int32 [T]     greedy autoregressive continuation (the committed output DVI must
                         reproduce), the first token from the prefill
  gaps    float64 [T]   top-2 logit gap behind each token (near-ties are exempt)
  logits  [T, V]        target-head logits behind every token (float32 for fp32 shapes,
                         float16 for bf16 shapes, whose tolerance is 2e-2 of the row's largest
                         magnitude)
  prompt  int32 [P]
Usage: python tests/golden/make_golden.py NAME [NAME ...]   (see CASES)
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle import dvi  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))

# name -> (shape, batch index of the prompt, prompt length, tokens)
CASES = {
    "tiny": (synth.TINY, 0, 32, 64),
    "1b_L4": (synth.shrunk(synth.SHAPE_1B), 0, 80, 40),
    "7b_L4": (synth.shrunk(synth.SHAPE_7B), 0, 80, 40),
    "13b_L4": (synth.shrunk(synth.SHAPE_13B), 0, 80, 40),
    "1b": (synth.SHAPE_1B, 0, 256, 128),
    "7b": (synth.SHAPE_7B, 0, 512, 128),
    "13b": (synth.SHAPE_13B, 0, 1024, 64),
}
# the batch-8 long-prompt workload: every sequence of its prompt batch
for _b in range(8):
    CASES["7b_b8_s%d" % _b] = (synth.SHAPE_7B, _b, 2048, 16)
# full-size prompts come from the workload's own prompt stream (batch of 8 for 7b_b8)
PROMPT_BATCH = {"7b_b8_s%d" % _b: 8 for _b in range(8)}


_W = {}


def _weights(shape):
    key = (shape.n_layers, shape.d_model, shape.ffn_dim, shape.vocab, shape.bf16)
    if key not in _W:
        _W.clear()
        _W[key] = synth.make_weights(shape, 0)
    return _W[key]


def make(name):
    shape, b, P, T = CASES[name]
    t0 = time.time()
    w = _weights(shape)
    prompt = synth.make_prompts(shape.vocab, PROMPT_BATCH.get(name, 1), P, 0)[b]
    m = oracle.OracleModel(w)
    ar = dvi.greedy_ar(m, prompt, T, keep_logits=True)
    lg = ar.logits.astype(np.float16 if shape.bf16 else np.float32)
    path = os.path.join(HERE, name + ".npz")
    np.savez_compressed(path, tokens=ar.tokens, gaps=ar.gaps, logits=lg, prompt=prompt)
    print("%s: %d tokens, min gap %.3g, %.0f s -> %s" % (name, T, ar.gaps.min(), time.time() - t0, path),
          flush=True)


if __name__ == "__main__":
    for n in sys.argv[1:] or ["tiny", "1b_L4", "7b_L4", "13b_L4"]:
        make(n)
