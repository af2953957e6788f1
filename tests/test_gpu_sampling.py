"""GPU parity of speculative sampling (temperature T > 0), through the C ABI.

The device draws with fp32 arithmetic; the oracle with fp64.  Draws are
compared the way argmax decisions are: every GPU decision must equal the rule
applied (in fp64, oracle.sampling) to the GPU's own logits wherever the
uniform is not within rounding distance of a decision boundary, and must equal
the oracle's own decision (from its own logits) wherever the boundary is
further away than the logit tolerance can move it.  The uniforms are the
oracle's independent implementation of the same counter-based generator.

* Lock-step steps on the tiny pair (granular calls) and on the 8B/1B-shaped
  full-width slice.
* The fused loop equals the granular calls token for token (same uniforms,
  same device arithmetic).
* Draft = target: the first candidate is always kept (p_0 == q_0 bitwise).
* Distribution: the first speculative token over 3200 slot/seed draws against
  the target's exact distribution (chi-square), through batched passes of 64
  slots (the row-block lm_head with its per-tile sums).
"""
from dataclasses import replace

import numpy as np
import pytest
from scipy import stats

import oracle
import pard_inputs as pi
from gpu_common import assert_logits_close, require_gpu, say
from oracle import sampling as S
from oracle.model import KVCache, forward_cached

pytestmark = pytest.mark.gpu

SELF_TOL = 1e-4       # CDF / keep-ratio distance within which fp32 and fp64 may decide differently
# A logit error e moves each log-probability by at most 2e/T, so a CDF boundary
# by at most exp(2e/T) - 1 and a keep ratio p/q by a relative exp(4e/T) - 1:
# GPU and oracle decisions are compared where the uniform is further than
# ORACLE_SCALE * e / T (e the step's largest logit error) from the boundary.
ORACLE_SCALE = 5.0


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


def _tiny():
    wl = pi.WORKLOADS["tiny"]
    return wl, pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")


def cdf_margin(prob_row, x, u):
    c = np.cumsum(prob_row)
    lo = c[x - 1] if x > 0 else 0.0
    return min(u - lo, c[x] - u)


def draft_margins(q, cands, seed, slot, draw):
    """Distance of each candidate's uniform from the ends of its CDF interval under q."""
    return [cdf_margin(q[j], cands[j], S.uniform(seed, slot, draw, j, S.PURPOSE_DRAFT)) for j in range(len(cands))]


def verify_margin(cands, p, q, a, tok, seed, slot, draw):
    """Smallest distance of any inspected keep test (u vs p/q) or of the last
    draw from a decision boundary, for the outcome (a, tok)."""
    m = np.inf
    for j in range(min(a + 1, len(cands))):
        x = cands[j]
        u = S.uniform(seed, slot, draw, j, S.PURPOSE_KEEP)
        m = min(m, abs(u * q[j, x] - p[j, x]) / max(p[j, x], u * q[j, x], 1e-30))
    w = np.maximum(p[a] - q[a], 0.0) if a < len(cands) else p[a]
    m = min(m, cdf_margin(w / w.sum(), tok, S.uniform(seed, slot, draw, a, S.PURPOSE_LAST)))
    return m


class SampledLockstep:
    """One slot stepped with sampling on the GPU (granular calls) and checked
    against the rule on its own logits and against the oracle."""

    def __init__(self, eng, target, draft, prompt, k, mask_id, temp, seed, slot=0, tag=""):
        self.eng, self.target, self.draft = eng, target, draft
        self.prompt, self.k, self.mask_id, self.temp, self.seed, self.slot = list(prompt), k, mask_id, temp, seed, slot
        self.tag = tag
        self.draw, self.worst, self.decided, self.compared = 0, 0.0, 0, 0

    def prefill(self):
        from paper_2504_18583_amd.binding import PARD_TARGET
        first = self.eng.prefill(self.prompt, seq=self.slot)
        self.cache_t, self.cache_d, o_first, lg = S.prefill_sampled(self.target, self.draft, self.prompt, self.temp,
                                                                    self.seed, self.slot)
        g = self.eng.read_logits(PARD_TARGET, 1, seq=self.slot)
        err = assert_logits_close(g, lg, f"{self.tag} prefill logits")
        self.worst = max(self.worst, err)
        self.oracle_tol = ORACLE_SCALE * err / self.temp
        u = S.uniform(self.seed, self.slot, 0, 0, S.PURPOSE_FIRST)
        pg = S.probs(g, self.temp)[0]
        mine = S.sample_index(pg, u)
        assert first == mine or cdf_margin(pg, mine, u) < SELF_TOL, f"{self.tag} first token {first} rule {mine}"
        self._compare(first, o_first, cdf_margin(S.probs(lg, self.temp)[0], o_first, u))
        self.pending = [first]
        self.hist = self.prompt + [first]
        return first

    def _compare(self, got, want, margin):
        self.compared += 1
        if margin > self.oracle_tol:
            self.decided += 1
            assert got == want, f"{self.tag}: gpu {got} oracle {want} (margin {margin:.3g})"

    def step(self):
        from paper_2504_18583_amd.binding import PARD_DRAFT, PARD_TARGET
        eng, k, T, seed, slot, draw = self.eng, self.k, self.temp, self.seed, self.slot, self.draw
        cands = eng.draft(self.hist, k, seq=slot)
        g_dl = eng.read_logits(PARD_DRAFT, k, seq=slot)
        o_cands, o_dl = S.draft_step_sampled(self.draft, self.cache_d, self.pending, k, self.mask_id, T, seed, slot,
                                             draw)
        err_d = assert_logits_close(g_dl, o_dl, f"{self.tag} draft logits")
        qg, qo = S.probs(g_dl, T), S.probs(o_dl, T)
        mine = [S.sample_index(qg[j], S.uniform(seed, slot, draw, j, S.PURPOSE_DRAFT)) for j in range(k)]
        for j, m in enumerate(draft_margins(qg, cands, seed, slot, draw)):
            assert cands[j] == mine[j] or m < SELF_TOL, f"{self.tag} candidate {j}: gpu {cands[j]} rule {mine[j]}"
        # the oracle follows the GPU's candidates from here on (a draw near a boundary may differ)
        self.oracle_tol = ORACLE_SCALE * err_d / T
        for j, m in enumerate(draft_margins(qo, o_cands, seed, slot, draw)):
            self._compare(cands[j], o_cands[j], m)
        lt = self.cache_t.length
        a, tok = eng.verify(cands, seq=slot)
        g_vl = eng.read_logits(PARD_TARGET, k + 1, seq=slot)
        o_a, o_tok, o_vl = S.verify_step_sampled(self.target, self.cache_t, self.pending[-1], cands, o_dl, T, seed,
                                                 slot, draw)
        err_v = assert_logits_close(g_vl, o_vl, f"{self.tag} verify logits")
        self.worst = max(self.worst, err_d, err_v)
        self.oracle_tol = ORACLE_SCALE * max(err_d, err_v) / T
        pg = S.probs(g_vl, T)
        ra, rtok = S.keep_decisions(cands, pg, qg, seed, slot, draw)
        if (ra, rtok) != (a, tok):
            assert verify_margin(cands, pg, qg, ra, rtok, seed, slot, draw) < SELF_TOL, \
                f"{self.tag}: gpu {(a, tok)} rule on gpu logits {(ra, rtok)}"
        po = S.probs(o_vl, T)
        self.compared += 1
        if verify_margin(cands, po, qo, o_a, o_tok, seed, slot, draw) > self.oracle_tol:
            self.decided += 1
            assert (a, tok) == (o_a, o_tok), f"{self.tag}: gpu {(a, tok)} oracle {(o_a, o_tok)}"
        if a != o_a:
            self.cache_t.truncate(lt)
            forward_cached(self.target, self.cache_t, [self.pending[-1]] + list(cands[:a]), logits_rows=[])
        assert eng.kv_len(PARD_TARGET, seq=slot) == self.cache_t.length == lt + a + 1
        assert eng.kv_len(PARD_DRAFT, seq=slot) == self.cache_d.length
        self.pending = list(cands[:a]) + [tok]
        self.hist += self.pending
        self.draw += 1
        return a, tok


@pytest.fixture(scope="module")
def tiny_models():
    wl, t_spec, d_spec = _tiny()
    return oracle.build_model(t_spec), oracle.build_model(d_spec)


@pytest.mark.parametrize("temp", [0.1, 0.3])
def test_tiny_sampling_lockstep(B, tiny_models, temp):
    wl, t_spec, d_spec = _tiny()
    target, draft = tiny_models
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=256, max_k=8)
    try:
        eng.set_sampling(temp, seed=2024)
        ls = SampledLockstep(eng, target, draft, prompt, wl.k, wl.mask_id, temp, 2024, tag=f"tiny T={temp}")
        ls.prefill()
        accepts = []
        for step in range(8):
            say(f"[gpu] sampling T={temp}: step {step}")
            accepts.append(ls.step()[0])
        say(f"    accepts {accepts}, oracle-decided {ls.decided}/{ls.compared}, max |logit err| {ls.worst:.3g}")
        assert ls.decided >= ls.compared // 2
    finally:
        eng.close()


def test_fused_sampling_equals_granular(B):
    wl, t_spec, d_spec = _tiny()
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=256, max_k=8)
    try:
        eng.set_sampling(0.2, seed=77)
        first = eng.prefill(prompt)
        toks, stats = eng.generate(wl.k, 40)
        assert len(toks) == 40 and toks[0] == first
        eng.prefill(prompt)                          # the draw counter restarts with the prefill
        hist, out = prompt + [first], [first]
        while len(out) < 40:
            cands = eng.draft(hist, wl.k)
            a, tok = eng.verify(cands)
            out += cands[:a] + [tok]
            hist += cands[:a] + [tok]
        assert toks == out[:40]
        # greedy again after T = 0
        eng.set_sampling(0.0)
        g1 = eng.prefill(prompt)
        g_toks, _ = eng.generate(wl.k, 12)
        eng.prefill(prompt)
        g_toks2, _ = eng.generate(wl.k, 12)
        assert g_toks == g_toks2 and g_toks[0] == g1
    finally:
        eng.close()


def test_self_draft_keeps_first_candidate(B):
    wl, t_spec, _ = _tiny()
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    eng = B.Engine(t_spec, t_spec, wl.mask_id, max_ctx=256, max_k=8)
    try:
        eng.set_sampling(0.5, seed=5)
        first = eng.prefill(prompt)
        hist = prompt + [first]
        for step in range(10):
            cands = eng.draft(hist, 4)
            a, tok = eng.verify(cands)
            assert a >= 1, f"step {step}: first candidate rejected with p == q"
            hist += cands[:a] + [tok]
    finally:
        eng.close()


def test_sampling_errors(B):
    wl, t_spec, d_spec = _tiny()
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=256, max_k=8)
    try:
        for bad in (-1.0, float("nan"), float("inf"), 1e-5):
            with pytest.raises(RuntimeError):
                eng.set_sampling(bad)
        eng.set_sampling(1.0, seed=1)
        first = eng.prefill(prompt)
        with pytest.raises(RuntimeError):            # verify needs this slot's draft of the same K
            eng.verify([1, 2, 3])
        cands = eng.draft(prompt + [first], 3)
        with pytest.raises(RuntimeError):
            eng.verify(cands[:2])
        eng.verify(cands)
        with pytest.raises(RuntimeError):            # vanilla drafting is greedy only
            eng.generate(4, 8, mode=B.PARD_MODE_VANILLA)
    finally:
        eng.close()


def test_first_speculative_token_distribution_batched(B, tiny_models):
    """64 slots per fused call (batched passes), 50 seeds: the first token of
    the first speculative step, after a greedy first token, is distributed as
    the target's p(. | prompt, first) at T."""
    wl, t_spec, d_spec = _tiny()
    target, _ = tiny_models
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    temp, n_slots, n_calls = 0.1, 64, 50
    cache = KVCache(target)
    lg = forward_cached(target, cache, prompt, logits_rows=[len(prompt) - 1])
    first = int(np.argmax(lg))
    p = S.probs(forward_cached(target, cache, [first]), temp)[0]
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=128, max_k=4, max_batch=n_slots)
    got = []
    try:
        for call in range(n_calls):
            eng.set_sampling(0.0)
            for s in range(n_slots):
                assert eng.prefill(prompt, seq=s) == first
            eng.set_sampling(temp, seed=1000 + call)
            res, _ = eng.generate_batch(list(range(n_slots)), 4, 2, max_steps=1)
            got += [r[1] for r in res]
            if call % 10 == 0:
                say(f"[gpu] distribution: call {call}")
    finally:
        eng.close()
    counts = np.bincount(got, minlength=len(p))
    order = np.argsort(-p)
    # bins: the likely tokens one by one (expected >= 10), the rest pooled
    exp_all = p * len(got)
    big = order[exp_all[order] >= 10]
    rest = np.setdiff1d(np.arange(len(p)), big)
    obs = np.append(counts[big], counts[rest].sum())
    exp = np.append(exp_all[big], exp_all[rest].sum())
    say(f"    {len(got)} draws, {len(big)} bins + pooled; top tokens obs {counts[order[:5]]} exp {np.round(exp_all[order[:5]], 1)}")
    assert len(big) >= 3
    assert stats.chisquare(obs, exp).pvalue > 1e-4


@pytest.mark.timeout(900)
def test_llama_8b_1b_full_width_slice_sampling_lockstep(B):
    wl = pi.WORKLOADS["llama8b_1b"]
    t_spec = replace(pi.with_dtype(wl.target, "bf16"), n_layers=2)
    d_spec = replace(pi.with_dtype(wl.draft, "bf16"), n_layers=1)
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]][:96]
    say("[gpu] 8B/1B full-width slice, sampling: oracle build")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=len(prompt) + 64, max_k=wl.k)
    try:
        eng.set_sampling(0.1, seed=31337)
        ls = SampledLockstep(eng, target, draft, prompt, wl.k, wl.mask_id, 0.1, 31337, tag="8B/1B T=0.1")
        ls.prefill()
        for step in range(2):
            say(f"[gpu] 8B/1B full-width slice, sampling: step {step}")
            ls.step()
        say(f"    oracle-decided {ls.decided}/{ls.compared}, max |logit err| {ls.worst:.3g}")
    finally:
        eng.close()


def test_batched_sampling_decisions_per_slot(B):
    """Five slots stepped together with sampling (multi-sequence skinny passes):
    every slot's candidates, keep count and last token equal the rule applied
    in fp64 to that slot's own GPU logits with its own uniforms (slot index),
    away from decision boundaries; KV lengths grow by a + 1."""
    wl, t_spec, d_spec = _tiny()
    temp, seed, k = 0.2, 99, 4
    slots = [1, 3, 4, 6, 7]
    prompts = {s: [int(x) for x in pi.gen_prompt(40 + s, t_spec.vocab, 20 + 7 * s)] for s in slots}
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=256, max_k=8, max_batch=8)
    try:
        eng.set_sampling(temp, seed)
        for s in slots:
            eng.prefill(prompts[s], seq=s)
        for step in range(4):
            lt = {s: eng.kv_len(B.PARD_TARGET, seq=s) for s in slots}
            res, stats = eng.generate_batch(slots, k, 64, max_steps=1)
            say(f"[gpu] batched sampling: step {step}, tokens {[len(r) - 1 for r in res]}")
            for s, toks in zip(slots, res):
                g_dl = eng.read_logits(B.PARD_DRAFT, k, seq=s)
                g_vl = eng.read_logits(B.PARD_TARGET, k + 1, seq=s)
                qg, pg = S.probs(g_dl, temp), S.probs(g_vl, temp)
                cands = [S.sample_index(qg[j], S.uniform(seed, s, step, j, S.PURPOSE_DRAFT)) for j in range(k)]
                margins_ok = all(m >= SELF_TOL for m in draft_margins(qg, cands, seed, s, step))
                a = eng.kv_len(B.PARD_TARGET, seq=s) - lt[s] - 1
                emitted = toks[1:]
                assert len(emitted) == a + 1 and 0 <= a <= k
                if margins_ok:
                    assert emitted[:a] == cands[:a], f"slot {s} step {step}: kept candidates"
                    ra, rtok = S.keep_decisions(cands, pg, qg, seed, s, step)
                    if verify_margin(cands, pg, qg, ra, rtok, seed, s, step) >= SELF_TOL:
                        assert (a, emitted[a]) == (ra, rtok), f"slot {s} step {step}"
    finally:
        eng.close()
