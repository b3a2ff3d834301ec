"""Greedy AR decoding and the DVI rollout, on the float64 oracle model.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 3.1: the target path emits y*_{t+1} = argmax p_phi(. | h_{L,t}) (greedy);
committed output must equal plain greedy autoregressive decoding of the frozen
model, token for token, whatever the drafter proposes (lossless speculation).

Section 3.3: at step t the draft path proposes t~_{t+1..t+k_spec} from the
shallow states; the target path maps each shallow state h_{k,t+i-1} through
layers k+1..L to y*_{t+i}; m is the longest prefix on which drafts and
targets agree; the m agreeing tokens are committed and y*_{t+m+1} is emitted;
one replay tuple is logged per drafted position up to and including the first
reject, with reward 1 for accepted positions and 0 for the first reject.

Readings taken where the text is silent (each listed in the design notes):
  * layers are 1-based in the text; here layer index l in 0..L-1 is text
    layer l+1, so the draft path is 0..k-1 and the target path k..L-1;
  * both heads read RMSNorm(h; g_final);
  * drafting is greedy (argmax of p_theta), ties to the lowest id, unless the drafter
    samples (oracle/sampling.py: Gumbel-max over z / tau with Philox4x64-10 noise);
  * when all k_spec drafts agree (m = k_spec) no extra token is produced:
    k_spec tokens are committed and the last one is processed next step, so a
    step commits n = min(m+1, k_spec) tokens;
  * each sequence produces exactly n_new tokens, the first from the prefill.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Optional

import numpy as np

from . import OracleModel, argmax_lowest, top2_gap
from . import sampling


@dataclasses.dataclass
class ARResult:
    tokens: np.ndarray          # int32 [n_new]
    gaps: np.ndarray            # float64 [n_new]: top-2 gap of the logits each token came from
    logits: Optional[np.ndarray] = None   # float64 [n_new, V] if requested


def greedy_ar(model: OracleModel, prompt, n_new: int, keep_logits: bool = False,
              s_max: Optional[int] = None) -> ARResult:
    """Plain greedy decoding of the full model: the definition of DVI's committed output."""
    s = model.shape
    prompt = np.asarray(prompt, dtype=np.int32)
    P = prompt.size
    cache = model.new_cache(s_max or (P + n_new))
    h = model.layers(cache, model.embed(prompt), 0, 0, s.n_layers)
    z = model.target_logits(model.final_norm(h[-1:]))
    toks, gaps, lg = [int(argmax_lowest(z)[0])], [float(top2_gap(z)[0])], [z[0]]
    pos = P
    while len(toks) < n_new:
        h = model.layers(cache, model.embed([toks[-1]]), pos, 0, s.n_layers)
        pos += 1
        z = model.target_logits(model.final_norm(h))
        toks.append(int(argmax_lowest(z)[0]))
        gaps.append(float(top2_gap(z)[0]))
        if keep_logits:
            lg.append(z[0])
    return ARResult(np.array(toks, np.int32), np.array(gaps),
                    np.stack(lg) if keep_logits else None)


@dataclasses.dataclass
class BufferRow:
    h_hat: np.ndarray     # RMSNorm(h_k) of the drafted position's input state, float64 [d]
    a: int                # drafted token t~_{t+i}
    logits_phi: np.ndarray  # target logits at that position, float64 [V]
    r: int                # 1 accepted, 0 first reject
    i: int                # 1-based position within the draft block
    prev_id: int          # token whose state produced the draft
    fresh: int = 1


@dataclasses.dataclass
class StepRecord:
    pos: int                   # cache length before the step
    drafts: np.ndarray         # int32 [k_spec]  t~_{t+1..t+k_spec}
    targets: np.ndarray        # int32 [k_spec]  y*_{t+1..t+k_spec}
    m: int
    n: int
    target_logits: np.ndarray  # float64 [k_spec, V]
    target_gaps: np.ndarray    # float64 [k_spec]
    draft_gaps: Optional[np.ndarray] = None  # float64 [k_spec]: top-2 gap of each draft's scores


@dataclasses.dataclass
class DVIResult:
    tokens: np.ndarray
    steps: List[StepRecord]
    buffer: List[BufferRow]
    cache: tuple
    length: int


def agree_prefix(drafts, targets) -> int:
    """m = max{i in 0..k : drafts[j] == targets[j] for all j < i} (0-based lists)."""
    m = 0
    for d_, t_ in zip(drafts, targets):
        if d_ != t_:
            break
        m += 1
    return m


@dataclasses.dataclass
class Drafter:
    """LoRA draft-head parameters theta = {A_s, B_s} and the scale gamma_s.  sample_tau > 0
    draws each draft from softmax(z / sample_tau) with the seeded Gumbel-max of
    oracle/sampling.py (sequence index seq in the counter); 0 drafts by argmax."""
    A: np.ndarray    # [V, r]
    B: np.ndarray    # [r, d]
    gamma: float
    sample_tau: float = 0.0
    seed: int = 0
    seq: int = 0


def dvi_generate(model: OracleModel, prompt, n_new: int, k_spec: int, drafter: Drafter,
                 forced_drafts: Optional[Callable[[int, int, np.ndarray], Optional[np.ndarray]]] = None,
                 on_step: Optional[Callable[["DVIResult", int], None]] = None,
                 s_max: Optional[int] = None, split_k: Optional[int] = None,
                 max_steps: Optional[int] = None, on_prefill: Optional[Callable[[], None]] = None) -> DVIResult:
    """Run DVI draft -> verify -> commit -> log until n_new tokens are committed.

    forced_drafts(step, pos, committed) may return an int array [k_spec] that
    replaces the drafter's argmax (test hook for exercising every m).
    on_step(result, step) is called after each commit; it may replace
    drafter.A / drafter.B (the online update), read at the next draft.
    max_steps stops after that many decode steps (bounded runs).
    on_prefill() is called once the prompt is processed and the first token chosen (timing).
    """
    s = model.shape
    k = s.split_k if split_k is None else split_k
    L = s.n_layers
    prompt = np.asarray(prompt, dtype=np.int32)
    P = prompt.size
    cache = model.new_cache(s_max or (P + n_new + k_spec))
    h = model.layers(cache, model.embed(prompt), 0, 0, L)
    z = model.target_logits(model.final_norm(h[-1:]))
    out = [int(argmax_lowest(z)[0])]
    if on_prefill is not None:
        on_prefill()
    length = P                   # tokens whose keys/values are in the cache
    res = DVIResult(np.zeros(0, np.int32), [], [], cache, length)
    step = 0
    while len(out) < n_new and (max_steps is None or step < max_steps):
        # ---- draft: k_spec serial single-token passes through layers 1..k
        tau = [out[-1]]
        hk_rows, drafts, dgaps = [], [], []
        forced = forced_drafts(step, length, np.array(out, np.int32)) if forced_drafts else None
        for j in range(k_spec):
            hj = model.layers(cache, model.embed([tau[j]]), length + j, 0, k)
            hk_rows.append(hj[0])
            zt = model.draft_logits(model.final_norm(hj), drafter.A, drafter.B, drafter.gamma)
            if drafter.sample_tau > 0:
                zt = sampling.sample_scores(zt, drafter.sample_tau, drafter.seed, step,
                                            drafter.seq * sampling.ROW_STRIDE + j)[None, :]
            dgaps.append(float(top2_gap(zt)[0]))
            t_next = int(argmax_lowest(zt)[0]) if forced is None else int(forced[j])
            drafts.append(t_next)
            tau.append(t_next)
        # ---- verify: one block pass of layers k+1..L over the k_spec shallow states
        H = np.stack(hk_rows)
        hL = model.layers(cache, H, length, k, L)
        zl = model.target_logits(model.final_norm(hL))
        targets = argmax_lowest(zl)
        # ---- commit
        m = agree_prefix(drafts, targets)
        remaining = n_new - len(out)
        n = min(m + 1, k_spec, remaining)
        out.extend(int(x) for x in targets[:n])
        length += n
        # ---- log tuples up to and including the first reject
        hk_hat = model.final_norm(H)
        for i in range(1, min(m + 1, k_spec) + 1):
            res.buffer.append(BufferRow(hk_hat[i - 1], drafts[i - 1], zl[i - 1],
                                        1 if i <= m else 0, i, tau[i - 1]))
        res.steps.append(StepRecord(length - n, np.array(drafts, np.int32), targets.copy(), m, n,
                                    zl, top2_gap(zl), np.array(dgaps)))
        res.length = length
        if on_step is not None:
            res.tokens = np.array(out, np.int32)
            on_step(res, step)
        step += 1
    res.tokens = np.array(out, np.int32)
    res.length = length
    return res
