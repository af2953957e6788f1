"""Pins for the oracle's speculative sampling (oracle/sampling.py).

* The random-number generator against SplitMix64's published outputs, and
  its uniforms against the uniform distribution.
* Inverse-CDF drawing: the set of u that yields token x has measure p(x).
* The keep / residual / bonus rule leaves the target distribution unchanged
  at every position it reaches (the property Sec. 1 and Sec. 2.2 rely on),
  checked by chi-square on synthetic distributions; the draft-equals-target
  case keeps every candidate.
* Whole loop: on a small vocabulary, the tokens of speculative sampling with
  the PARD draft follow the target's autoregressive sampling distribution
  (exact marginals by enumeration); at a vanishing temperature the loop is
  the greedy loop.
"""
import json
import os
from dataclasses import replace

import numpy as np
import pytest
from scipy import stats

import oracle
import pard_inputs as pi
from oracle import sampling as S
from oracle.model import KVCache, forward_cached

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_matches_published_outputs():
    with open(os.path.join(GOLDEN, "splitmix64_state0.json")) as f:
        g = json.load(f)
    got = [f"{S.splitmix64_output(g['state'], n):016x}" for n in range(len(g["outputs_hex"]))]
    assert got == g["outputs_hex"]


def test_uniforms_are_uniform_and_distinct():
    u = np.array([S.uniform(12345, slot, draw, j, p)
                  for slot in range(4) for draw in range(50) for j in range(25) for p in range(4)])
    assert ((u >= 0) & (u < 1)).all()
    assert np.all(u * 2 ** 24 == np.floor(u * 2 ** 24))          # 24-bit grid
    assert abs(u.mean() - 0.5) < 5e-3 and abs(u.var() - 1 / 12) < 3e-3
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    assert len(np.unique(u)) > 0.99 * len(u)                       # coordinates do not collide
    assert S.uniform(1, 0, 0, 0, 0) != S.uniform(2, 0, 0, 0, 0)


def test_sample_index_is_the_inverse_cdf():
    rng = np.random.default_rng(0)
    w = rng.random(7) ** 3
    w[3] = 0.0                                                     # a zero weight is never drawn
    n = 1 << 16
    xs = np.array([S.sample_index(w, (i + 0.5) / n) for i in range(n)])
    assert np.all(np.diff(xs) >= 0)                                # monotone in u
    freq = np.bincount(xs, minlength=7) / n
    assert np.allclose(freq, w / w.sum(), atol=2.0 / n)
    assert freq[3] == 0
    c = np.cumsum(w) / w.sum()
    for x in range(6):
        if w[x] > 0:
            assert S.sample_index(w, c[x] - 1e-9) == x
    assert S.sample_index(w, 0.0) == 0


def _rows(rng, n, v, conc=0.7):
    return rng.dirichlet(np.full(v, conc), size=n)


@pytest.mark.parametrize("k", [1, 3])
def test_keep_rule_reproduces_target_at_every_position(k):
    """Candidates drawn from q_j, the rule applied: the token emitted at
    position j (kept candidate or last token) is distributed as p_j."""
    rng = np.random.default_rng(k)
    v = 6
    p, q = _rows(rng, k + 1, v), _rows(rng, k, v)
    seen = [[] for _ in range(k + 1)]
    for draw in range(30000):
        cands = [S.sample_index(q[j], S.uniform(99, 0, draw, j, S.PURPOSE_DRAFT)) for j in range(k)]
        a, tok = S.keep_decisions(cands, p, q, 99, 0, draw)
        emitted = list(cands[:a]) + [tok]
        for pos, x in enumerate(emitted):
            seen[pos].append(x)
    for pos in range(k + 1):
        counts = np.bincount(seen[pos], minlength=v)
        expected = p[pos] * len(seen[pos])
        assert len(seen[pos]) > 500
        assert stats.chisquare(counts, expected).pvalue > 1e-4, (pos, counts, expected)


def test_keep_rule_cases():
    p = np.array([[0.5, 0.5, 0.0], [0.1, 0.2, 0.7]])
    # a candidate the target gives zero probability is never kept, and the
    # last token then comes from max(0, p - q), here token 0 or 1
    q0 = np.array([[0.0, 0.0, 1.0]])
    for draw in range(50):
        a, tok = S.keep_decisions([2], p, q0, 5, 0, draw)
        assert a == 0 and tok in (0, 1)
    # draft equal to target: every candidate kept, the bonus comes from p_K
    for draw in range(50):
        a, tok = S.keep_decisions([1], p, p[:1], 5, 0, draw)
        assert a == 1
    with pytest.raises(ValueError):
        S.keep_decisions([0, 1], p, q0, 5, 0, 0)


@pytest.fixture(scope="module")
def small_vocab_pair():
    wl = pi.WORKLOADS["tiny"]
    shape = dict(vocab=16, d_model=64, n_heads=2, n_kv_heads=1, head_dim=32, ffn_dim=128, init_std=0.15)
    return oracle.build_model(replace(wl.target, **shape)), oracle.build_model(replace(wl.draft, **shape))


def test_speculative_sampling_follows_target_distribution(small_vocab_pair):
    """Tokens 2 and 3 after the prompt (the first speculative step's output)
    against their exact marginals under autoregressive sampling from the
    target, enumerated over the first token."""
    target, draft = small_vocab_pair
    prompt, v, temp, mask_id = [3, 1, 4, 1, 5, 9, 2, 6], 16, 1.0, 15
    p1 = S.probs(forward_cached(target, KVCache(target), prompt, logits_rows=[len(prompt) - 1]), temp)[0]
    m2, m3 = np.zeros(v), np.zeros(v)
    for y1 in range(v):
        cache = KVCache(target)
        forward_cached(target, cache, prompt, logits_rows=[])
        p2 = S.probs(forward_cached(target, cache, [y1]), temp)[0]
        m2 += p1[y1] * p2
        for y2 in range(v):
            c2 = KVCache(target)
            forward_cached(target, c2, prompt + [y1], logits_rows=[])
            m3 += p1[y1] * p2[y2] * S.probs(forward_cached(target, c2, [y2]), temp)[0]
    toks = np.array([S.generate_sampled(target, draft, prompt, 3, 3, mask_id, temp, seed).tokens
                     for seed in range(3000)])
    for col, m in ((1, m2), (2, m3)):
        counts = np.bincount(toks[:, col], minlength=v)
        keep = m * len(toks) >= 5                  # pool the rare tokens into one bin
        obs = np.append(counts[keep], counts[~keep].sum())
        exp = np.append(m[keep], m[~keep].sum()) * len(toks)
        if exp[-1] == 0:
            obs, exp = obs[:-1], exp[:-1]
        assert stats.chisquare(obs, exp).pvalue > 1e-4, (col, obs, exp)


def test_self_draft_sampling_keeps_every_candidate(small_vocab_pair):
    target, _ = small_vocab_pair
    tr = S.generate_sampled(target, target, [3, 1, 4, 1, 5], 3, 20, 15, 1.0, seed=7)
    # the draft's rows condition on mask tokens, so they differ from the
    # target's beyond the first; the first candidate is always kept
    assert all(a >= 1 for a in tr.accepts)


def test_vanishing_temperature_is_greedy():
    wl = pi.WORKLOADS["tiny"]
    target, draft = oracle.build_model(wl.target), oracle.build_model(wl.draft)
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    greedy = oracle.pard_generate(target, draft, prompt, wl.k, 12, wl.mask_id)
    sampled = S.generate_sampled(target, draft, prompt, wl.k, 12, wl.mask_id, 1e-6, seed=3)
    assert sampled.tokens == greedy.tokens


def test_k0_is_plain_sampling(small_vocab_pair):
    target, draft = small_vocab_pair
    prompt = [2, 7, 1, 8]
    for seed in range(5):
        assert S.generate_sampled(target, draft, prompt, 0, 8, 15, 0.8, seed).tokens == \
            S.sample_ar(target, prompt, 8, 0.8, seed)
