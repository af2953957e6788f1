"""GPU checks of vanilla speculative decoding (Sec. 2.1, eq. 3), the baseline
PARD is measured against: K sequential one-row draft passes, then the same
verify pass, on the same kernels (pard_generate_ex, PARD_MODE_VANILLA).

* draft == target: every candidate is the target's greedy token, so a = K on
  every step (the one-row draft passes and the K+1-row verify pass compute the
  same logits: the arithmetic does not depend on the pass's row count);
* lossless: the output equals the target's greedy decoding (eq. 2), for one
  slot and for a batch of slots;
* the fused loop equals the same steps run through the granular calls
  (pard_draft with K = 1, K times, then pard_verify), token for token."""
import numpy as np
import pytest

import oracle
import pard_inputs as pi
from gpu_common import MARGIN, margins, require_gpu, say

pytestmark = pytest.mark.gpu

WL = pi.WORKLOADS["tiny"]
T_SPEC, D_SPEC = pi.with_dtype(WL.target, "bf16"), pi.with_dtype(WL.draft, "bf16")
PROMPT = [int(x) for x in pi.workload_prompts(WL)[0]]


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


@pytest.fixture(scope="module")
def target():
    return oracle.build_model(T_SPEC)


def _check_greedy(toks, target, prompt, what):
    """GPU tokens equal the oracle's greedy tokens up to the first near-tie."""
    cache = oracle.KVCache(target)
    lg = oracle.forward_cached(target, cache, prompt, logits_rows=[len(prompt) - 1])[0]
    for i, g in enumerate(toks):
        ref = int(np.argmax(lg))
        if g != ref:
            assert float(margins(lg)) <= MARGIN, f"{what} token {i}: gpu {g} oracle {ref}"
            return
        lg = oracle.forward_cached(target, cache, [g])[0]


def test_vanilla_self_draft_accepts_every_candidate(B, target):
    eng = B.Engine(T_SPEC, T_SPEC, WL.mask_id, max_ctx=320, max_k=8)
    try:
        for k in (1, 3, 8):
            say(f"[gpu] vanilla, draft == target, K={k}")
            eng.prefill(PROMPT)
            toks, stats = eng.generate(k, 60, mode=B.PARD_MODE_VANILLA)
            hist = list(stats.accept_hist)
            assert hist[k] == stats.steps and sum(hist) == stats.steps, hist[:k + 1]
            _check_greedy(toks, target, PROMPT, f"self-draft K={k}")
    finally:
        eng.close()


@pytest.mark.parametrize("k", [1, 4, 8])
def test_vanilla_is_lossless(B, target, k):
    say(f"[gpu] vanilla, tiny pair, K={k}")
    eng = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=256, max_k=8)
    try:
        eng.prefill(PROMPT)
        toks, stats = eng.generate(k, WL.n_tokens, mode=B.PARD_MODE_VANILLA)
        assert len(toks) == WL.n_tokens == stats.tokens
        _check_greedy(toks, target, PROMPT, f"K={k}")
        committed = sum((a + 1) * n for a, n in enumerate(stats.accept_hist))
        assert eng.kv_len(B.PARD_TARGET) == len(PROMPT) + committed
    finally:
        eng.close()


def test_vanilla_fused_equals_granular(B):
    """The fused vanilla loop and the granular calls run the same passes."""
    k, n = 4, 30
    eng = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=256, max_k=8)
    try:
        first = eng.prefill(PROMPT)
        fused, _ = eng.generate(k, n, mode=B.PARD_MODE_VANILLA)
        eng.prefill(PROMPT)
        hist, out = PROMPT + [first], [first]
        while len(out) < n:
            cands = []
            for _ in range(k):
                cands += eng.draft(hist + cands, 1)
            a, bonus = eng.verify(cands)
            out += cands[:a] + [bonus]
            hist += cands[:a] + [bonus]
        assert fused == out[:n]
    finally:
        eng.close()


def test_vanilla_batched_is_lossless(B, target):
    lens = pi.gen_prompt_lengths(41, 8, 10, 70)
    prompts = [[int(x) for x in pi.gen_prompt(41, T_SPEC.vocab, int(m), b)] for b, m in enumerate(lens)]
    k, n = 4, 24
    eng = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=160, max_k=8, max_batch=8)
    try:
        for b, p in enumerate(prompts):
            eng.prefill(p, seq=b)
        say("[gpu] vanilla, 8 slots in batched passes")
        res, stats = eng.generate_batch(list(range(8)), k, n, mode=B.PARD_MODE_VANILLA)
        assert stats.tokens == 8 * n
        for b, p in enumerate(prompts):
            assert len(res[b]) == n
            _check_greedy(res[b], target, p, f"slot {b}")
    finally:
        eng.close()
