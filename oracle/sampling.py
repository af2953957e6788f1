"""Speculative sampling (temperature > 0) for the PARD step, step by step.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

Paper passages followed:
* Sec. 1 and Sec. 2.2: speculative decoding combined with speculative
  sampling (the cited rejection-sampling scheme of Chen et al. 2023 and
  Leviathan et al. 2023) leaves the target model's output distribution
  unchanged.  Restated: a candidate x at position j, drawn from the draft's
  distribution q_j, is kept with probability min(1, p_j(x) / q_j(x)), p_j the
  target's distribution at that position; at the first position whose
  candidate is not kept, the step's last token is drawn from the residual
  distribution proportional to max(0, p_j - q_j); if all K candidates are
  kept, a bonus token is drawn from p_K.  The step emits the kept candidates
  and that last token, exactly as the greedy step emits c_1..c_a and t_a.
* Sec. 3.1 eq. 7: the PARD draft produces its K distributions in one pass;
  candidate c_{j+1} is drawn from its row j (the last real row for j = 0, the
  mask rows after it).  Each row is a fixed distribution given the prefix, so
  it is a valid proposal for position j whatever was drawn before it.

Readings where the paper is silent (each one is listed in the design notes):
* p_j = softmax(target logits / T), q_j = softmax(draft logits / T), one
  temperature T > 0 for both models (T = 0 is the greedy step of
  ``oracle.pard``).
* Drawing from unnormalised weights w with a uniform u in [0, 1): the
  smallest token id x with w_0 + ... + w_x > u * (w_0 + ... + w_{V-1})
  (inverse CDF in token-id order).
* The keep test is u * q_j(x) < p_j(x) (u < p/q without the division).
* Random numbers come from one counter-based generator, SplitMix64 (Steele,
  Lea, Flood 2014): U(seed, slot, draw, j, purpose) is the top 24 bits of
  output 4j + purpose of the stream seeded with output `draw` of the stream
  seeded with output `slot` of the stream seeded with `seed`, scaled by 2^-24.
  `draw` counts the verify steps of the sequence since its prefill; purpose 0
  draws candidate j, 1 is the keep test at position j, 2 draws the last token
  at position j (residual or bonus), 3 draws the first token after the prompt.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from .model import KVCache, Model, forward_cached
from .pard import PardTrace

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
PURPOSE_DRAFT, PURPOSE_KEEP, PURPOSE_LAST, PURPOSE_FIRST = 0, 1, 2, 3


def splitmix64_mix(z: int) -> int:
    """SplitMix64's output function (its published mixing constants and shifts)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64_output(state: int, n: int) -> int:
    """Output n (0-based) of the SplitMix64 stream whose state starts at `state`:
    the state advances by the golden gamma before each output."""
    return splitmix64_mix((state + (n + 1) * GOLDEN_GAMMA) & MASK64)


def uniform(seed: int, slot: int, draw: int, j: int, purpose: int) -> float:
    """The uniform in [0, 1) of (sequence slot, verify step, position, purpose)."""
    if not (0 <= purpose < 4 and j >= 0 and draw >= 0 and slot >= 0):
        raise ValueError("bad random-number coordinates")
    z = splitmix64_output(seed & MASK64, slot)
    z = splitmix64_output(z, draw)
    z = splitmix64_output(z, 4 * j + purpose)
    return float(z >> 40) * 2.0 ** -24


def probs(logits: np.ndarray, temperature: float) -> np.ndarray:
    """softmax(logits / T) per row, in float64."""
    z = np.asarray(logits, np.float64) / float(temperature)
    z = z - z.max(axis=-1, keepdims=True)
    w = np.exp(z)
    return w / w.sum(axis=-1, keepdims=True)


def sample_index(weights: np.ndarray, u: float) -> int:
    """Inverse-CDF draw from unnormalised non-negative weights, token-id order."""
    w = np.asarray(weights, np.float64)
    c = np.cumsum(w)
    x = int(np.searchsorted(c, u * c[-1], side="right"))
    if x >= len(w):                       # only through rounding: the last id with weight
        x = int(np.flatnonzero(w > 0)[-1])
    return x


def keep_decisions(cands: Sequence[int], p_rows: np.ndarray, q_rows: np.ndarray, seed: int, slot: int,
                   draw: int) -> Tuple[int, int]:
    """The speculative-sampling rule on probability rows: (a, last token).

    p_rows: K+1 target distributions (position j scores candidate j+1; row K
    gives the bonus); q_rows: the K draft distributions the candidates were
    drawn from."""
    k = len(cands)
    if p_rows.shape[0] != k + 1 or q_rows.shape[0] < k:
        raise ValueError("need K+1 target rows and K draft rows")
    for j in range(k):
        x = int(cands[j])
        u = uniform(seed, slot, draw, j, PURPOSE_KEEP)
        if not u * q_rows[j, x] < p_rows[j, x]:
            residual = np.maximum(p_rows[j] - q_rows[j], 0.0)
            return j, sample_index(residual, uniform(seed, slot, draw, j, PURPOSE_LAST))
    return k, sample_index(p_rows[k], uniform(seed, slot, draw, k, PURPOSE_LAST))


def prefill_sampled(target: Model, draft: Model, prompt: Sequence[int], temperature: float, seed: int,
                    slot: int = 0):
    """Both caches hold the prompt; the first token is drawn from the target at T."""
    cache_t, cache_d = KVCache(target), KVCache(draft)
    logits = forward_cached(target, cache_t, prompt, logits_rows=[len(prompt) - 1])
    forward_cached(draft, cache_d, prompt, logits_rows=[])
    first = sample_index(probs(logits, temperature)[0], uniform(seed, slot, 0, 0, PURPOSE_FIRST))
    return cache_t, cache_d, first, logits


def draft_step_sampled(draft: Model, cache_d: KVCache, pending: Sequence[int], k: int, mask_id: int,
                       temperature: float, seed: int, slot: int, draw: int):
    """One PARD draft pass (eq. 7) with candidate j+1 drawn from row j at T.

    Returns (candidates, logits); the draft cache keeps the pending tokens."""
    if k < 1 or len(pending) < 1:
        raise ValueError("need k >= 1 and at least one pending token")
    start = cache_d.length
    ids = list(pending) + [mask_id] * (k - 1)
    first = len(pending) - 1
    logits = forward_cached(draft, cache_d, ids, logits_rows=range(first, first + k))
    cache_d.truncate(start + len(pending))
    q = probs(logits, temperature)
    cands = [sample_index(q[j], uniform(seed, slot, draw, j, PURPOSE_DRAFT)) for j in range(k)]
    return cands, logits


def verify_step_sampled(target: Model, cache_t: KVCache, last: int, cands: Sequence[int],
                        draft_logits: np.ndarray, temperature: float, seed: int, slot: int, draw: int):
    """Target pass over [last, c_1..c_K] and the speculative-sampling rule.

    Returns (a, last token, logits); the target cache keeps the a+1 rows whose
    inputs were right (as in the greedy step)."""
    start = cache_t.length
    logits = forward_cached(target, cache_t, [int(last)] + [int(c) for c in cands])
    p = probs(logits, temperature)
    q = probs(draft_logits, temperature) if len(cands) else np.zeros((0, p.shape[1]))
    a, tok = keep_decisions(cands, p, q, seed, slot, draw)
    cache_t.truncate(start + a + 1)
    return a, tok, logits


def generate_sampled(target: Model, draft: Model, prompt: Sequence[int], k: int, n_tokens: int, mask_id: int,
                     temperature: float, seed: int, slot: int = 0) -> PardTrace:
    """The PARD loop with speculative sampling; k = 0 samples the target alone."""
    cache_t, cache_d, first, _ = prefill_sampled(target, draft, prompt, temperature, seed, slot)
    trace = PardTrace(tokens=[first])
    pending = [first]
    draw = 0
    while len(trace.tokens) < n_tokens:
        if k > 0:
            cands, dl = draft_step_sampled(draft, cache_d, pending, k, mask_id, temperature, seed, slot, draw)
        else:
            cands, dl = [], np.zeros((0, target.spec.vocab))
        a, tok, _ = verify_step_sampled(target, cache_t, pending[-1], cands, dl, temperature, seed, slot, draw)
        pending = list(cands[:a]) + [tok]
        trace.tokens += pending
        trace.accepts.append(a)
        trace.candidates.append(list(cands))
        draw += 1
    trace.tokens = trace.tokens[:n_tokens]
    return trace


def sample_ar(target: Model, prompt: Sequence[int], n_tokens: int, temperature: float, seed: int,
              slot: int = 0) -> List[int]:
    """Plain autoregressive sampling from the target at T (the distribution the
    speculative loop must reproduce)."""
    cache = KVCache(target)
    logits = forward_cached(target, cache, prompt, logits_rows=[len(prompt) - 1])
    out = [sample_index(probs(logits, temperature)[0], uniform(seed, slot, 0, 0, PURPOSE_FIRST))]
    draw = 0
    while len(out) < n_tokens:
        logits = forward_cached(target, cache, [out[-1]])
        out.append(sample_index(probs(logits, temperature)[0], uniform(seed, slot, draw, 0, PURPOSE_LAST)))
        draw += 1
    return out
