"""Greedy decoding and the PARD draft / verify / accept loop, step by step.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

Paper passages followed:
* Greedy decoding, Sec. 2.1 eq. 2: the next token is the argmax of the
  model's distribution given all previous tokens.  Ties go to the lowest id.
* Speculative decoding, Sec. 2.2: a drafting stage proposes K candidates
  C = (x'_n .. x'_{n+K-1}); a verification stage scores them with the target
  in one parallel pass.
* Vanilla speculative decoding, Sec. 2.1 eq. 3: the drafting stage is K
  sequential greedy steps of the draft model (its cost K times one draft
  step), each conditioned on the candidates before it.
* PARD drafting, Sec. 3.1 eq. 7 and the PARD-inference figure: the draft runs
  ONE forward over the known prefix followed by shared mask tokens
  m_0 = ... = m_{K-1} (Sec. 4.3, shared mask id), and the k-th candidate
  (k = 0..K-1) is read at the row whose input is m_{k-1} (the last real token
  for k = 0), so it conditions on x_<n and m_0..m_{k-1} only.

Readings where the paper is silent (each one is listed in the design notes):
* K-1 mask rows follow the last real token; the K candidates are the argmax of
  the last real row and of the K-1 mask rows.  Masks sit at consecutive
  positions after the real tokens and attend causally.
* Mask rows are never committed to the draft cache.  Tokens accepted by the
  target are re-fed to the draft as real tokens on the next step (their
  cached K/V came from mask inputs), so a draft pass has a+K rows.
* Verification is greedy: with t_j the target argmax at verify row j (row 0 is
  the pending token, rows 1..K the candidates), a is the largest j such that
  c_i = t_{i-1} for every i <= j; the bonus token is t_a; the step emits
  c_1..c_a followed by the bonus.  The target cache keeps the a+1 rows whose
  inputs were correct (pending token, c_1..c_a).
* The first generated token is the target's argmax after the prompt; it is
  pending (not yet in either cache).  Generation stops after exactly N tokens
  counting that first one; no end-of-sequence token.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

import numpy as np

from .model import KVCache, Model, forward_cached


def argmax_rows(logits: np.ndarray) -> List[int]:
    """Greedy choice per row (eq. 2); numpy's argmax returns the lowest index on ties."""
    return [int(i) for i in np.argmax(logits, axis=-1)]


def greedy_ar(model: Model, prompt: Sequence[int], n_tokens: int) -> List[int]:
    """Plain greedy autoregressive decoding (eq. 2): the first n_tokens after the prompt."""
    cache = KVCache(model)
    logits = forward_cached(model, cache, prompt, logits_rows=[len(prompt) - 1])
    out = argmax_rows(logits)
    while len(out) < n_tokens:
        out += argmax_rows(forward_cached(model, cache, [out[-1]]))
    return out[:n_tokens]


def accept_prefix(cands: Sequence[int], t: Sequence[int]) -> Tuple[int, int]:
    """Greedy acceptance: (a, bonus) with a the longest agreeing prefix, bonus = t[a]."""
    if len(t) != len(cands) + 1:
        raise ValueError("need one more target token than candidates")
    a = 0
    while a < len(cands) and int(cands[a]) == int(t[a]):
        a += 1
    return a, int(t[a])


def prefill(target: Model, draft: Model, prompt: Sequence[int]):
    """Both caches hold the prompt; returns (target cache, draft cache, first token, logits)."""
    cache_t, cache_d = KVCache(target), KVCache(draft)
    logits = forward_cached(target, cache_t, prompt, logits_rows=[len(prompt) - 1])
    forward_cached(draft, cache_d, prompt, logits_rows=[])
    return cache_t, cache_d, argmax_rows(logits)[0], logits


def draft_step(draft: Model, cache_d: KVCache, pending: Sequence[int], k: int,
               mask_id: int) -> Tuple[List[int], np.ndarray]:
    """One PARD draft pass (eq. 7): pending real tokens + (k-1) masks -> k candidates.

    Afterwards the draft cache holds the pending tokens but not the mask rows."""
    if k < 1 or len(pending) < 1:
        raise ValueError("need k >= 1 and at least one pending token")
    start = cache_d.length
    ids = list(pending) + [mask_id] * (k - 1)
    first = len(pending) - 1
    logits = forward_cached(draft, cache_d, ids, logits_rows=range(first, first + k))
    cache_d.truncate(start + len(pending))
    return argmax_rows(logits), logits


def verify_step(target: Model, cache_t: KVCache, last: int, cands: Sequence[int]):
    """Target pass over [last, c_1..c_K]; returns (a, bonus, t, logits).

    The target cache keeps the a+1 rows with correct inputs (rollback)."""
    start = cache_t.length
    logits = forward_cached(target, cache_t, [int(last)] + [int(c) for c in cands])
    t = argmax_rows(logits)
    a, bonus = accept_prefix(cands, t)
    cache_t.truncate(start + a + 1)
    return a, bonus, t, logits


@dataclass
class PardTrace:
    tokens: List[int]
    accepts: List[int] = field(default_factory=list)
    candidates: List[List[int]] = field(default_factory=list)


def pard_generate(target: Model, draft: Model, prompt: Sequence[int], k: int,
                  n_tokens: int, mask_id: int) -> PardTrace:
    """The PARD loop: prefill, then draft (one pass) / verify / accept until n_tokens.

    k = 0 runs plain target steps (no draft), the autoregressive baseline."""
    cache_t, cache_d, first, _ = prefill(target, draft, prompt)
    trace = PardTrace(tokens=[first])
    pending = [first]
    while len(trace.tokens) < n_tokens:
        cands = draft_step(draft, cache_d, pending, k, mask_id)[0] if k > 0 else []
        a, bonus, _, _ = verify_step(target, cache_t, pending[-1], cands)
        pending = list(cands[:a]) + [bonus]
        trace.tokens += pending
        trace.accepts.append(a)
        trace.candidates.append(list(cands))
    trace.tokens = trace.tokens[:n_tokens]
    return trace


def vanilla_draft_step(draft: Model, cache_d: KVCache, pending: Sequence[int],
                       k: int) -> Tuple[List[int], np.ndarray]:
    """Vanilla drafting (Sec. 2.1, eq. 3): k sequential greedy draft steps.

    The first step reads the pending tokens, every later one the candidate
    before it.  Afterwards the draft cache holds the pending tokens and
    c_1..c_{k-1} (c_k is proposed, not read).  Returns the candidates and the
    logits row each was taken from."""
    if k < 1 or len(pending) < 1:
        raise ValueError("need k >= 1 and at least one pending token")
    ids, cands, rows = list(pending), [], []
    for _ in range(k):
        logits = forward_cached(draft, cache_d, ids, logits_rows=[len(ids) - 1])
        c = argmax_rows(logits)[0]
        cands.append(c)
        rows.append(logits[0])
        ids = [c]
    return cands, np.stack(rows)


def vanilla_generate(target: Model, draft: Model, prompt: Sequence[int], k: int,
                     n_tokens: int) -> PardTrace:
    """Vanilla speculative decoding with greedy verification: k sequential
    draft steps, then the same verify / accept as PARD.  After verification
    the draft cache keeps the pending token(s) and the candidates that agree
    with the committed tokens; the tokens after them are pending for the
    next drafting stage."""
    cache_t, cache_d, first, _ = prefill(target, draft, prompt)
    trace = PardTrace(tokens=[first])
    pending = [first]
    while len(trace.tokens) < n_tokens:
        start_d = cache_d.length
        cands, _ = vanilla_draft_step(draft, cache_d, pending, k)
        a, bonus, _, _ = verify_step(target, cache_t, pending[-1], cands)
        keep = min(a, k - 1)
        cache_d.truncate(start_d + len(pending) + keep)
        pending = list(cands[keep:a]) + [bonus]
        trace.tokens += list(cands[:a]) + [bonus]
        trace.accepts.append(a)
        trace.candidates.append(list(cands))
    trace.tokens = trace.tokens[:n_tokens]
    return trace
