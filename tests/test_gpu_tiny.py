"""GPU parity on the tiny pair (2-layer target, 1-layer tied draft, vocab 1024).

Every call goes through the C ABI; the oracle runs on the same bf16-rounded
weights and the same prompt.  Logits must agree within 3e-2 + 1e-2*|ref|,
token decisions wherever the oracle's top-1/top-2 margin exceeds 0.1, accept
counts and KV lengths exactly.
"""
import numpy as np
import pytest

import oracle
import pard_inputs as pi
from gpu_common import (assert_logits_close, assert_tokens_match, lockstep, margins, require_gpu,
                        say, MARGIN)

pytestmark = pytest.mark.gpu

WL = pi.WORKLOADS["tiny"]
T_SPEC = pi.with_dtype(WL.target, "bf16")
D_SPEC = pi.with_dtype(WL.draft, "bf16")
PROMPT = [int(x) for x in pi.workload_prompts(WL)[0]]


@pytest.fixture(scope="module")
def models():
    return oracle.build_model(T_SPEC), oracle.build_model(D_SPEC)


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


@pytest.fixture(scope="module")
def eng(B):
    say("[gpu] tiny engine: load")
    e = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=512, max_k=16, max_batch=2)
    yield e
    e.close()


def test_weights_match_generator_bitwise(eng, models, B):
    """The device holds each bf16 weight in fp16 encoding: equal to the
    generator's value, except below 2^-14 where fp16 rounds to a subnormal."""
    say("[gpu] tiny: weight readback")
    rng = np.random.default_rng(0)
    for which, model in ((B.PARD_TARGET, models[0]), (B.PARD_DRAFT, models[1])):
        w = model.weights
        spec = model.spec
        cases = [(0, w["embed"])]
        if not spec.tied:
            cases.append((1, w["lm_head"]))
        for l, lw in w["layers"].items():
            for j, name in enumerate(["wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"]):
                cases.append((pi.layer_tensor(l, j), lw[name]))
        for tensor, ref in cases:
            for row in rng.choice(ref.shape[0], size=6, replace=False):
                got = eng.read_weight(which, tensor, int(row), 0, ref.shape[1])
                want = ref[row].astype(np.float16).astype(np.float32)
                assert np.array_equal(got, want), (which, tensor, row)
                big = np.abs(ref[row]) >= 2.0 ** -14
                assert np.array_equal(got[big], ref[row][big].astype(np.float32)), (which, tensor, row)


def test_prefill_logits_and_first_token(eng, models, B):
    say("[gpu] tiny: prefill")
    target, draft = models
    first = eng.prefill(PROMPT)
    _, _, first_o, lg = oracle.prefill(target, draft, PROMPT)
    assert_logits_close(eng.read_logits(B.PARD_TARGET, 1), lg, "prefill")
    assert_tokens_match([first], lg, "first token")
    assert eng.kv_len(B.PARD_TARGET) == eng.kv_len(B.PARD_DRAFT) == len(PROMPT)


@pytest.mark.parametrize("k", [WL.k, 1, 8, 12, 0])
def test_lockstep_draft_verify(eng, models, k):
    say(f"[gpu] tiny: lock-step K={k}")
    target, draft = models
    worst = lockstep(eng, target, draft, PROMPT, k, steps=12, mask_id=WL.mask_id, tag=f"K={k}")
    say(f"    max |logit err| {worst:.3g}")


@pytest.mark.parametrize("k", [16, 24, 32])
def test_large_k_lockstep_and_fused(B, models, k):
    """K past the trained range (the shared mask id extends the draft to any
    K): draft passes of a+K rows up to 64, verify passes of K+1 rows over
    two or three row tiles, the tail's K+1 lm rows; fused loop vs greedy."""
    target, _ = models
    e = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=1024, max_k=32)
    try:
        say(f"[gpu] tiny: large K={k}")
        worst = lockstep(e, target, models[1], PROMPT, k, steps=5, mask_id=WL.mask_id, tag=f"K={k}")
        say(f"    max |logit err| {worst:.3g}")
        e.prefill(PROMPT)
        toks, stats = e.generate(k, 40)
        ref = oracle.greedy_ar(target, PROMPT, 40)
        cache = oracle.KVCache(target)
        lg = oracle.forward_cached(target, cache, PROMPT, logits_rows=[len(PROMPT) - 1])
        for i in range(40):              # equal up to the first near-tie of the oracle
            if margins(lg)[-1] <= MARGIN:
                break
            assert toks[i] == ref[i], f"K={k} token {i}"
            lg = oracle.forward_cached(target, cache, [ref[i]])
    finally:
        e.close()


def test_rope_scaled_pair_lockstep(B):
    """LLaMA-3.1-style rotary scaling (original length 32, so the tiny head's
    frequencies span the kept, blended and divided regimes) on both models."""
    from dataclasses import replace
    scaling = (8.0, 1.0, 4.0, 32)
    t_spec, d_spec = replace(T_SPEC, rope_scaling=scaling), replace(D_SPEC, rope_scaling=scaling)
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    e = B.Engine(t_spec, d_spec, WL.mask_id, max_ctx=512, max_k=8)
    try:
        say("[gpu] tiny: rope-scaled pair, lock-step K=4")
        worst = lockstep(e, target, draft, PROMPT, WL.k, steps=6, mask_id=WL.mask_id, tag="rope-scaled")
        say(f"    max |logit err| {worst:.3g}")
    finally:
        e.close()


@pytest.mark.parametrize("ffn,S", [(14368, 8), (16480, 9)])
def test_wide_gate_up_ragged_last_workgroup_lockstep(B, ffn, S):
    """Gate/up weights of 1796 and 2060 strips: too many for 7 strips per
    workgroup in one round of 256 workgroups, so the plan takes 8 and 9 strips
    per workgroup and the last workgroup holds 4 and 8 strips (the 10-strip
    case runs in the Qwen full-width slices)."""
    from dataclasses import replace
    n_strips = 2 * ffn // 16
    assert n_strips % 7 and -(-n_strips // 7) > 256 and -(-n_strips // S) <= 256 and n_strips % S
    assert S == 8 or -(-n_strips // 8) > 256
    t_spec = replace(T_SPEC, n_layers=1, ffn_dim=ffn)
    target, draft = oracle.build_model(t_spec), oracle.build_model(D_SPEC)
    e = B.Engine(t_spec, D_SPEC, WL.mask_id, max_ctx=512, max_k=8)
    try:
        say(f"[gpu] tiny: target ffn {ffn} ({n_strips} gate/up strips, {S} per workgroup), lock-step K=4")
        worst = lockstep(e, target, draft, PROMPT, WL.k, steps=3, mask_id=WL.mask_id, tag=f"ffn{ffn}")
        say(f"    max |logit err| {worst:.3g}")
    finally:
        e.close()


def test_generate_matches_greedy(eng, models, B):
    say("[gpu] tiny: fused generate vs greedy")
    target, _ = models
    eng.prefill(PROMPT)
    toks, stats = eng.generate(WL.k, WL.n_tokens)
    assert len(toks) == WL.n_tokens == stats.tokens
    assert sum(stats.accept_hist) == stats.steps
    assert sum((a + 1) * n for a, n in enumerate(stats.accept_hist)) >= WL.n_tokens - 1
    # oracle greedy with the margin of every decision
    cache = oracle.KVCache(target)
    lg = oracle.forward_cached(target, cache, PROMPT, logits_rows=[len(PROMPT) - 1])[0]
    ref, marg = [], []
    for i in range(WL.n_tokens):
        ref.append(int(np.argmax(lg)))
        marg.append(float(margins(lg)))
        if toks[i] != ref[i]:
            assert marg[i] <= MARGIN, f"token {i}: gpu {toks[i]} oracle {ref[i]} margin {marg[i]:.3f}"
            break                                   # a genuine near-tie: sequences fork here
        lg = oracle.forward_cached(target, cache, [toks[i]])[0]
    committed = sum((a + 1) * n for a, n in enumerate(stats.accept_hist))
    assert eng.kv_len(B.PARD_TARGET) == len(PROMPT) + committed


@pytest.mark.parametrize("k,mode", [(4, 0), (0, 0), (3, 1)])
def test_generate_phase_times(eng, B, k, mode):
    """pard_stats' phase times come from the device clock at pass boundaries:
    draft + verify + accept cover the timed steps (the gaps between passes are
    a few kernel launches), a plain target step has no draft phase, and the
    step-latency percentiles are ordered and match the mean step."""
    say(f"[gpu] tiny: phase times K={k} mode={mode}")
    eng.prefill(PROMPT)
    toks, st = eng.generate(k, 48, mode=mode)
    assert st.steps >= 8
    phases = st.draft_ms + st.verify_ms + st.accept_ms
    say(f"    steps {st.steps}: elapsed {st.elapsed_ms:.3f} ms, draft {st.draft_ms:.3f} verify {st.verify_ms:.3f} "
        f"accept {st.accept_ms:.3f}, step p50 {st.step_ms_p50:.4f} p90 {st.step_ms_p90:.4f}")
    assert st.verify_ms > 0 and st.accept_ms > 0
    assert (st.draft_ms > 0) == (k > 0)
    assert 0.5 * st.elapsed_ms < phases <= 1.02 * st.elapsed_ms
    assert 0 < st.step_ms_p50 <= st.step_ms_p90
    mean = st.elapsed_ms / st.steps
    assert 0.5 * mean < st.step_ms_p50 < 2.0 * mean


def test_k1_draft_is_plain_draft_decode(eng, models, B):
    say("[gpu] tiny: K=1 draft")
    target, draft = models
    first = eng.prefill(PROMPT)
    prefix = PROMPT + [first]
    cand = eng.draft(prefix, 1)
    cache = oracle.KVCache(draft)
    lg = oracle.forward_cached(draft, cache, prefix, logits_rows=[len(prefix) - 1])
    assert_logits_close(eng.read_logits(B.PARD_DRAFT, 1), lg, "K=1 draft logits")
    assert_tokens_match(cand, lg, "K=1 candidate")


def _decisive_prompt(target, n_follow):
    """First seeded prompt whose greedy continuation has no near-tie for n_follow tokens."""
    for seed in range(100, 400):
        prompt = [int(x) for x in pi.gen_prompt(seed, WL.target.vocab, 32)]
        cache = oracle.KVCache(target)
        lg = oracle.forward_cached(target, cache, prompt, logits_rows=[len(prompt) - 1])[0]
        greedy = []
        for _ in range(n_follow):
            if margins(lg) <= MARGIN:
                break
            greedy.append(int(np.argmax(lg)))
            lg = oracle.forward_cached(target, cache, [greedy[-1]])[0]
        if len(greedy) == n_follow:
            return prompt, greedy
    pytest.skip("no decisive prompt found")


@pytest.mark.parametrize("k", [4, 8])
def test_forced_candidates_accept_exact_prefix(eng, models, k):
    say(f"[gpu] tiny: forced candidates K={k}")
    target, _ = models
    prompt, greedy = _decisive_prompt(target, k + 2)
    for j in range(k + 1):
        first = eng.prefill(prompt)
        assert first == greedy[0]
        cands = list(greedy[1:1 + k])
        if j < k:
            cands[j] = (cands[j] + 1) % WL.mask_id
        a, bonus = eng.verify(cands)
        assert a == j and bonus == greedy[1 + j], (j, a, bonus)


def test_rewind_reproduces_draft_logits(eng, B):
    say("[gpu] tiny: truncate and re-draft")
    first = eng.prefill(PROMPT)
    hist = PROMPT + [first]
    for _ in range(3):
        cands = eng.draft(hist, 4)
        a, bonus = eng.verify(cands)
        hist += cands[:a] + [bonus]
    c1 = eng.draft(hist, 6)
    l1 = eng.read_logits(B.PARD_DRAFT, 6)
    eng.kv_truncate(B.PARD_DRAFT, len(hist) - 4)
    assert eng.kv_len(B.PARD_DRAFT) == len(hist) - 4
    c2 = eng.draft(hist, 6)
    l2 = eng.read_logits(B.PARD_DRAFT, 6)
    assert c1 == c2 and np.array_equal(l1, l2)


def test_runs_are_bitwise_deterministic(eng, B):
    say("[gpu] tiny: determinism")
    outs = []
    for _ in range(2):
        eng.prefill(PROMPT)
        toks, _ = eng.generate(WL.k, 24)
        outs.append((toks, eng.read_logits(B.PARD_TARGET, WL.k + 1).copy()))
    assert outs[0][0] == outs[1][0] and np.array_equal(outs[0][1], outs[1][1])


def test_errors_leave_state_unchanged(eng, B):
    say("[gpu] tiny: error paths")
    with pytest.raises(B.PardError) as e:
        eng.verify([1, 2], seq=1)                       # slot 1 never prefilled
    assert e.value.status == B.PARD_ERR_STATE
    eng.prefill(PROMPT)
    lt, ld = eng.kv_len(B.PARD_TARGET), eng.kv_len(B.PARD_DRAFT)
    for call, code in [(lambda: eng.draft(PROMPT, 17), B.PARD_ERR_ARG),
                       (lambda: eng.verify([1] * 17), B.PARD_ERR_ARG),
                       (lambda: eng.verify([5000]), B.PARD_ERR_ARG),
                       (lambda: eng.kv_truncate(B.PARD_TARGET, lt + 1), B.PARD_ERR_ARG),
                       (lambda: eng.prefill(list(range(500))), B.PARD_ERR_CAPACITY),
                       (lambda: eng.generate(4, 600), B.PARD_ERR_CAPACITY),
                       (lambda: eng.prefill(PROMPT, seq=2), B.PARD_ERR_CAPACITY)]:
        with pytest.raises(B.PardError) as e:
            call()
        assert e.value.status == code
        assert (eng.kv_len(B.PARD_TARGET), eng.kv_len(B.PARD_DRAFT)) == (lt, ld)


def test_fp16_range_overflow_is_reported(B):
    """Activations and the KV cache are fp16: a pass whose values leave fp16's
    range must fail loudly (PARD_ERR_RANGE), not return silently wrong tokens.
    Weights at init_std 5 take the tiny target's residual stream past 65520
    in its first layer (the oracle shows it below), far beyond what the
    benchmark weights do (|x| < 1)."""
    import dataclasses
    from oracle import model as om
    say("[gpu] tiny: fp16 overflow flag")
    t_big = dataclasses.replace(T_SPEC, init_std=5.0)
    m = oracle.build_model(t_big)
    ids = np.asarray(PROMPT)
    x = np.asarray(np.asarray(m.weights["embed"])[ids], np.float64)
    assert np.abs(x).max() < 65520
    empty = np.zeros((0, t_big.n_kv_heads, t_big.head_dim))
    with np.errstate(over="ignore"):
        x1, _, _ = om._layer(t_big, m.weights["layers"][0], x, np.arange(len(ids)), empty, empty)
    assert np.abs(x1).max() >= 65520
    eng = B.Engine(t_big, D_SPEC, WL.mask_id, max_ctx=256, max_k=8)
    try:
        for _ in range(2):                              # reported by every call that overflows
            with pytest.raises(B.PardError) as e:
                eng.prefill(PROMPT)
            assert e.value.status == B.PARD_ERR_RANGE
    finally:
        eng.close()


def test_self_draft_accepts_every_step(B):
    say("[gpu] tiny: draft == target")
    eng = B.Engine(T_SPEC, T_SPEC, WL.mask_id, max_ctx=256, max_k=8)
    try:
        for k in (1, 3):
            eng.prefill(PROMPT)
            toks, stats = eng.generate(k, 40)
            assert stats.accept_hist[0] == 0, list(stats.accept_hist)[:k + 1]
            if k == 1:
                assert stats.accept_hist[1] == stats.steps
    finally:
        eng.close()


QWEN_T = pi.ModelSpec(n_layers=2, d_model=448, n_heads=7, n_kv_heads=1, head_dim=64, ffn_dim=320,
                      vocab=512, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True, tied=False,
                      dtype="bf16", seed=5, stream=0)
QWEN_D = pi.ModelSpec(n_layers=1, d_model=256, n_heads=2, n_kv_heads=1, head_dim=128, ffn_dim=200,
                      vocab=512, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True, tied=True,
                      dtype="bf16", seed=5, stream=1)


def test_qwen_shaped_bias_group7_lockstep(B):
    say("[gpu] qwen-shaped tiny: lock-step with QKV bias, GQA group 7")
    target, draft = oracle.build_model(QWEN_T), oracle.build_model(QWEN_D)
    eng = B.Engine(QWEN_T, QWEN_D, 511, max_ctx=256, max_k=12)
    try:
        prompt = [int(x) for x in pi.gen_prompt(5, 512, 40)]
        for k in (4, 12):
            lockstep(eng, target, draft, prompt, k, steps=6, mask_id=511, tag=f"qwen K={k}")
    finally:
        eng.close()


def test_long_prompt_split_attention_lockstep(models, B):
    say("[gpu] tiny: 2300-token prompt (attention split over 3 key ranges + merge)")
    target, draft = models
    eng = B.Engine(T_SPEC, D_SPEC, WL.mask_id, max_ctx=2400, max_k=8)
    try:
        prompt = [int(x) for x in pi.gen_prompt(11, WL.target.vocab, 2300)]
        worst = lockstep(eng, target, draft, prompt, 6, steps=3, mask_id=WL.mask_id, tag="long")
        say(f"    max |logit err| {worst:.3g}")
        first = eng.prefill(prompt)
        toks, stats = eng.generate(6, 24)
        assert toks[0] == first and len(toks) == 24
    finally:
        eng.close()
