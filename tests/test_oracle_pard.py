"""Pins for the oracle's cached forward and its PARD draft/verify/accept loop.

* cached forward == uncached forward, position by position (brute force);
* one-pass parallel draft == K separate uncached passes over prefix + k masks
  (Sec. 3.1 eq. 7: candidate k conditions on x_<n and m_0..m_{k-1} only);
* lossless greedy speculative decoding: PARD output == plain greedy decoding of
  the target (Sec. 2.1 eq. 2, Sec. 2.2) for K in {1, 2, 4, 8, 12};
* K = 1 reduces to an ordinary draft decode step;
* forced candidates: corrupting the greedy continuation at index j gives a = j;
* draft == target: the first candidate always matches, so a >= 1 every step.
"""
import numpy as np
import pytest

import oracle
import pard_inputs as pi
from oracle import (KVCache, accept_prefix, draft_step, forward_cached, forward_full,
                    greedy_ar, pard_generate, prefill, verify_step)

WL = pi.WORKLOADS["tiny"]


@pytest.fixture(scope="module")
def tiny():
    return oracle.build_model(WL.target), oracle.build_model(WL.draft)


@pytest.fixture(scope="module")
def prompt():
    return [int(x) for x in pi.workload_prompts(WL)[0]]


def test_cached_matches_uncached_position_by_position(tiny, prompt):
    target, _ = tiny
    ids = prompt + [5, 77, 1023, 3]
    cache = KVCache(target)
    rows = []
    for chunk in ([0, 7], [7, 8], [8, 20], [20, len(ids)]):
        rows.append(forward_cached(target, cache, ids[chunk[0]:chunk[1]]))
    cached = np.concatenate(rows)
    for t in range(len(ids)):
        full = forward_full(target, ids[:t + 1])[-1]
        assert np.abs(cached[t] - full).max() < 1e-12


@pytest.mark.parametrize("n_layers", [1, 2])
def test_fill_cache_equals_forward_cached(tiny, prompt, n_layers):
    """The logit-free ingest leaves exactly the cache the full cached forward
    leaves (every layer, every position), so later passes see the same keys."""
    from dataclasses import replace
    target = oracle.build_model(replace(WL.target, n_layers=n_layers))
    a, b = KVCache(target), KVCache(target)
    forward_cached(target, a, prompt[:20])
    forward_cached(target, a, prompt[20:])
    oracle.fill_cache(target, b, prompt[:20])
    oracle.fill_cache(target, b, prompt[20:])
    assert a.length == b.length == len(prompt)
    for l in range(n_layers):
        assert np.array_equal(a.k[l], b.k[l]) and np.array_equal(a.v[l], b.v[l])
    assert np.array_equal(forward_cached(target, a, [9, 1023]), forward_cached(target, b, [9, 1023]))


def test_truncate_then_refeed_reproduces_logits(tiny, prompt):
    target, _ = tiny
    cache = KVCache(target)
    a = forward_cached(target, cache, prompt + [11, 12, 13])
    cache.truncate(len(prompt) + 1)
    b = forward_cached(target, cache, [12, 13])
    assert np.abs(a[-2:] - b).max() < 1e-12
    with pytest.raises(ValueError):
        cache.truncate(cache.length + 1)


@pytest.mark.parametrize("k", [1, 2, 4, 8])
@pytest.mark.parametrize("n_pending", [1, 3])
def test_parallel_draft_equals_separate_masked_passes(tiny, prompt, k, n_pending):
    _, draft = tiny
    prefix = prompt + [101, 202, 303]
    cache = KVCache(draft)
    forward_cached(draft, cache, prefix[:-n_pending], logits_rows=[])
    cands, logits = draft_step(draft, cache, prefix[-n_pending:], k, WL.mask_id)
    assert cache.length == len(prefix)                    # mask rows not committed
    for j in range(k):
        ref = forward_full(draft, prefix + [WL.mask_id] * j)[-1]
        assert np.abs(logits[j] - ref).max() < 1e-12
        assert cands[j] == int(np.argmax(ref))


def test_k1_draft_is_plain_draft_decode(tiny, prompt):
    _, draft = tiny
    cache = KVCache(draft)
    forward_cached(draft, cache, prompt[:-1], logits_rows=[])
    cands, _ = draft_step(draft, cache, prompt[-1:], 1, WL.mask_id)
    assert cands == greedy_ar(draft, prompt, 1)


@pytest.mark.parametrize("k", [0, 1, 2, 4, 8, 12])
def test_pard_is_lossless_vs_greedy(tiny, prompt, k):
    target, draft = tiny
    ref = greedy_ar(target, prompt, WL.n_tokens)
    tr = pard_generate(target, draft, prompt, k, WL.n_tokens, WL.mask_id)
    assert tr.tokens == ref
    assert all(0 <= a <= k for a in tr.accepts)


def test_pard_lossless_qwen_shaped_with_bias():
    t = pi.ModelSpec(n_layers=2, d_model=224, n_heads=14, n_kv_heads=2, head_dim=16,
                     ffn_dim=96, vocab=512, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                     tied=False, dtype="bf16", seed=2, stream=0)
    d = pi.ModelSpec(n_layers=1, d_model=112, n_heads=7, n_kv_heads=1, head_dim=16,
                     ffn_dim=64, vocab=512, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                     tied=True, dtype="bf16", seed=2, stream=1)
    target, draft = oracle.build_model(t), oracle.build_model(d)
    prompt = [int(x) for x in pi.gen_prompt(2, 512, 24)]
    ref = greedy_ar(target, prompt, 40)
    for k in (4, 12):
        assert pard_generate(target, draft, prompt, k, 40, 511).tokens == ref


def test_self_draft_accepts_at_least_one(tiny, prompt):
    target, _ = tiny
    ref = greedy_ar(target, prompt, 40)
    for k in (1, 3, 6):
        tr = pard_generate(target, target, prompt, k, 40, WL.mask_id)
        assert tr.tokens == ref
        assert min(tr.accepts) >= 1
        if k == 1:
            assert set(tr.accepts) == {1}


@pytest.mark.parametrize("k", [1, 4, 8])
def test_forced_candidates_accept_exact_prefix(tiny, prompt, k):
    target, draft = tiny
    greedy = greedy_ar(target, prompt, 2 + k)
    for j in range(k + 1):
        cache_t, _, first, _ = prefill(target, draft, prompt)
        assert first == greedy[0]
        cands = list(greedy[1:1 + k])
        if j < k:
            cands[j] = (cands[j] + 1) % (WL.mask_id)
        a, bonus, t, _ = verify_step(target, cache_t, first, cands)
        assert a == j
        assert bonus == greedy[1 + j]
        assert cache_t.length == len(prompt) + a + 1


def test_accept_prefix_cases():
    assert accept_prefix([], [9]) == (0, 9)
    assert accept_prefix([1, 2, 3], [1, 2, 3, 4]) == (3, 4)
    assert accept_prefix([1, 2, 3], [1, 5, 3, 4]) == (1, 5)
    assert accept_prefix([7, 2], [1, 2, 3]) == (0, 1)
    with pytest.raises(ValueError):
        accept_prefix([1, 2], [1, 2])


# ---- vanilla speculative decoding (Sec. 2.1, eq. 3), the baseline PARD is compared with ----

@pytest.mark.parametrize("k", [1, 3, 6])
def test_vanilla_draft_is_the_drafts_greedy_continuation(tiny, prompt, k):
    """K sequential draft steps propose exactly the draft model's own greedy
    continuation (recomputed from scratch by plain greedy decoding)."""
    _, draft = tiny
    hist = prompt + [17, 400]
    cache = KVCache(draft)
    forward_cached(draft, cache, hist[:-2], logits_rows=[])
    cands, rows = oracle.vanilla_draft_step(draft, cache, hist[-2:], k)
    assert cands == greedy_ar(draft, hist, k)
    assert rows.shape == (k, draft.spec.vocab)
    # the cache holds the pending tokens and c_1..c_{k-1}
    assert cache.length == len(hist) + k - 1


@pytest.mark.parametrize("k", [1, 2, 4, 8])
def test_vanilla_sd_is_lossless_vs_greedy(tiny, prompt, k):
    target, draft = tiny
    n = 40
    trace = oracle.vanilla_generate(target, draft, prompt, k, n)
    assert trace.tokens == greedy_ar(target, prompt, n)
    assert all(0 <= a <= k for a in trace.accepts)


def test_vanilla_sd_self_draft_accepts_everything(tiny, prompt):
    """With the target as its own draft every candidate is the target's greedy
    token: a = K every step, and the rolled-back draft cache stays consistent."""
    target, _ = tiny
    trace = oracle.vanilla_generate(target, target, prompt, 4, 26)
    assert all(a == 4 for a in trace.accepts)
    assert trace.tokens == greedy_ar(target, prompt, 26)


def test_vanilla_sd_draft_cache_matches_fresh_prefill(tiny, prompt):
    """After each step's rollback the draft cache equals a fresh prefill of the
    committed tokens it claims to hold (brute force)."""
    target, draft = tiny
    k = 3
    cache_t, cache_d, first, _ = prefill(target, draft, prompt)
    hist, pending = list(prompt) + [first], [first]
    for _ in range(5):
        start_d = cache_d.length
        cands, _ = oracle.vanilla_draft_step(draft, cache_d, pending, k)
        a, bonus, _, _ = verify_step(target, cache_t, pending[-1], cands)
        keep = min(a, k - 1)
        cache_d.truncate(start_d + len(pending) + keep)
        hist += list(cands[:a]) + [bonus]
        pending = list(cands[keep:a]) + [bonus]
        fresh = KVCache(draft)
        forward_cached(draft, fresh, hist[:cache_d.length], logits_rows=[])
        for l in range(draft.spec.n_layers):
            np.testing.assert_allclose(cache_d.k[l][:cache_d.length], fresh.k[l][:cache_d.length], atol=1e-12)
            np.testing.assert_allclose(cache_d.v[l][:cache_d.length], fresh.v[l][:cache_d.length], atol=1e-12)
        assert cache_d.length + len(pending) == len(hist)
