"""GPU parity at the benchmark shapes.

* Full-width slices: the LLaMA3.1-8B / LLaMA3.2-1B-shaped pair and the
  Qwen2.5-7B / 0.5B-shaped pair at their full width, heads and vocabulary but
  with 2 (target) and 1-2 (draft) layers.  Every kernel runs with the grid and
  tile plan of the full models (they depend on widths, heads, vocabulary and
  context, not on depth), on the benchmark's prompt; the fp64 oracle runs the
  same slices in lock-step.
* Full depth (32 / 16 layers): properties that hold at any size -- the accept
  rule against the engine's own logits, KV-length bookkeeping, fused loop ==
  granular calls token for token, bitwise determinism of both models' logits.
* 16k-token context: the attention chunk/merge path at the long-context
  workload's length, on a narrow pair the oracle can follow.
* Long-context plans: one-layer targets with as many KV heads as query heads,
  at contexts where 256-key chunks would give the decode pass's attention
  more than one workgroup per CU, so the plan takes longer chunks (384 and
  640 keys here: not powers of two, several tiles per wavefront, a ragged
  last chunk); and a head_dim-128 case with more than 16 chunks, which the
  many-chunk merge combines (the 16k test covers it at head_dim 64).
"""
from dataclasses import replace

import numpy as np
import pytest

import oracle
import pard_inputs as pi
from gpu_common import lockstep, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


def _slice(spec, n_layers):
    return replace(pi.with_dtype(spec, "bf16"), n_layers=n_layers)


def test_llama_8b_1b_full_width_slice_lockstep(B):
    wl = pi.WORKLOADS["llama8b_1b"]
    t_spec, d_spec = _slice(wl.target, 2), _slice(wl.draft, 1)
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    say(f"[gpu] 8B/1B full-width slice: oracle build (prompt {len(prompt)}, K={wl.k})")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    say("[gpu] 8B/1B full-width slice: engine load")
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=len(prompt) + 64, max_k=wl.k)
    try:
        say("[gpu] 8B/1B full-width slice: lock-step")
        worst = lockstep(eng, target, draft, prompt, wl.k, steps=2, mask_id=wl.mask_id, tag="8B/1B")
        say(f"    max |logit err| {worst:.3g}")
        say("[gpu] 8B/1B full-width slice: fused loop (graph replay) vs granular calls")
        first = eng.prefill(prompt)
        toks, stats = eng.generate(wl.k, 20)
        # granular replay of the same steps
        eng.prefill(prompt)
        hist = prompt + [first]
        out = [first]
        while len(out) < 20:
            cands = eng.draft(hist, wl.k)
            a, bonus = eng.verify(cands)
            out += cands[:a] + [bonus]
            hist += cands[:a] + [bonus]
        assert toks == out[:20]
    finally:
        eng.close()


def test_llama_8b_1b_gate_up_preload_depth_is_bitwise_neutral(B, monkeypatch):
    """The one-launch layer's gate/up tiles take their first iterations from
    LDS (the dynamic area, then the static area shared with the attention
    arrays; QKV workgroups may preload fewer, down to none) and stream the
    rest; where an iteration comes from never changes the arithmetic or its
    order, and the tile's reduction (kept in the preload area) sums in wave
    order.  So every preload split gives bitwise the logits of the default
    plan, at the 8B/1B tile shapes."""
    from paper_2504_18583_amd.binding import PARD_DRAFT, PARD_TARGET
    wl = pi.WORKLOADS["llama8b_1b"]
    t_spec, d_spec = _slice(wl.target, 2), _slice(wl.draft, 1)
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    ref = None
    # (iterations per workgroup, of the QKV workgroups); None: the default plan
    for pre, pre_q in [(None, None), (1, 0), (2, 1), (3, 3), (5, 1), (5, 4)]:
        for name, v in (("PARD_GU_PRE", pre), ("PARD_GU_PRE_Q", pre_q)):
            if v is None:
                monkeypatch.delenv(name, raising=False)
            else:
                monkeypatch.setenv(name, str(v))
        say(f"[gpu] 8B/1B slice: gate/up preload {pre}, QKV workgroups {pre_q}")
        eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=len(prompt) + 64, max_k=wl.k)
        try:
            first = eng.prefill(prompt)
            hist = prompt + [first]
            got = []
            for _ in range(2):
                cands = eng.draft(hist, wl.k)
                dl = eng.read_logits(PARD_DRAFT, wl.k)
                a, bonus = eng.verify(cands)
                vl = eng.read_logits(PARD_TARGET, wl.k + 1)
                got.append((cands, a, bonus, dl, vl))
                hist += cands[:a] + [bonus]
        finally:
            eng.close()
        if ref is None:
            ref = got
            continue
        for (c0, a0, b0, d0, v0), (c1, a1, b1, d1, v1) in zip(ref, got):
            assert (c1, a1, b1) == (c0, a0, b0)
            assert np.array_equal(d1.view(np.uint32), d0.view(np.uint32))
            assert np.array_equal(v1.view(np.uint32), v0.view(np.uint32))


QWEN = pi.WORKLOADS["qwen7b_05b"]
QWEN_T, QWEN_D = _slice(QWEN.target, 2), _slice(QWEN.draft, 2)


@pytest.fixture(scope="module")
def qwen_models(B):
    say("[gpu] Qwen 7B/0.5B full-width slice: oracle build")
    return oracle.build_model(QWEN_T), oracle.build_model(QWEN_D)


@pytest.mark.parametrize("k", QWEN.k_sweep)
def test_qwen_7b_05b_full_width_slice_lockstep(B, qwen_models, k):
    target, draft = qwen_models
    prompt = [int(x) for x in pi.workload_prompts(QWEN)[0]]
    say(f"[gpu] Qwen 7B/0.5B full-width slice: engine load, lock-step K={k} (prompt {len(prompt)})")
    eng = B.Engine(QWEN_T, QWEN_D, QWEN.mask_id, max_ctx=len(prompt) + 64, max_k=max(QWEN.k_sweep))
    try:
        worst = lockstep(eng, target, draft, prompt, k, steps=1, mask_id=QWEN.mask_id, tag=f"qwen K={k}")
        say(f"    max |logit err| {worst:.3g}")
    finally:
        eng.close()


def test_llama_8b_1b_full_depth_properties(B):
    wl = pi.WORKLOADS["llama8b_1b"]
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    say("[gpu] 8B/1B full depth: engine load")
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=len(prompt) + 128, max_k=wl.k)
    try:
        say("[gpu] 8B/1B full depth: granular steps")
        first = eng.prefill(prompt)
        assert eng.kv_len(B.PARD_TARGET) == eng.kv_len(B.PARD_DRAFT) == len(prompt)
        hist = prompt + [first]
        out = [first]
        for step in range(4):
            lt = eng.kv_len(B.PARD_TARGET)
            cands = eng.draft(hist, wl.k)
            dl = eng.read_logits(B.PARD_DRAFT, wl.k)
            assert np.isfinite(dl).all() and cands == [int(i) for i in np.argmax(dl, axis=-1)]
            assert eng.kv_len(B.PARD_DRAFT) == len(hist)
            a, bonus = eng.verify(cands)
            vl = eng.read_logits(B.PARD_TARGET, wl.k + 1)
            assert np.isfinite(vl).all()
            assert (a, bonus) == oracle.accept_prefix(cands, np.argmax(vl, axis=-1)), step
            assert eng.kv_len(B.PARD_TARGET) == lt + a + 1
            out += cands[:a] + [bonus]
            hist += cands[:a] + [bonus]
        say("[gpu] 8B/1B full depth: fused loop twice")
        runs = []
        for _ in range(2):
            assert eng.prefill(prompt) == first
            toks, stats = eng.generate(wl.k, len(out))
            runs.append((toks, eng.read_logits(B.PARD_TARGET, wl.k + 1).copy(),
                         eng.read_logits(B.PARD_DRAFT, wl.k).copy()))
        assert runs[0][0] == out
        # bitwise: fixed reduction orders everywhere, including the draft's
        # down projection, whose input is split over two workgroups per strip
        assert runs[0][0] == runs[1][0] and np.array_equal(runs[0][1], runs[1][1])
        assert np.array_equal(runs[0][2], runs[1][2])
    finally:
        eng.close()


FULL_DEPTH_PROMPT = 64     # tokens of the benchmark prompt the full-depth lock-step uses


@pytest.fixture(scope="module")
def full_depth(B):
    """The 32-layer 8B-shaped target and 16-layer 1B-shaped draft, on the GPU
    and in the oracle (float32 weights held on the host, ~37 GB)."""
    from gpu_common import Lockstep
    wl = pi.WORKLOADS["llama8b_1b"]
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    prompt = [int(x) for x in pi.workload_prompts(wl)[0][:FULL_DEPTH_PROMPT]]
    models = []
    for name, spec in (("target", t_spec), ("draft", d_spec)):
        say(f"[gpu] 8B/1B full depth: oracle {name} weights")
        models.append(oracle.Model(spec, pi.gen_model_weights(spec, progress=lambda m, n=name: say(f"    {n} {m}"))))
    say("[gpu] 8B/1B full depth: engine load")
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=len(prompt) + 64, max_k=wl.k)
    ls = Lockstep(eng, models[0], models[1], prompt, wl.k, wl.mask_id, tag="8B/1B full depth")
    try:
        yield ls
    finally:
        eng.close()


def test_llama_8b_1b_full_depth_prefill_lockstep(full_depth):
    """The headline pair at its full 32/16 layers: prefill logits and first
    token against the float64 oracle at the stated tolerance."""
    say("[gpu] 8B/1B full depth: prefill lock-step")
    full_depth.prefill()
    say(f"    max |logit err| after prefill {full_depth.worst:.4g}")


def test_llama_8b_1b_full_depth_steps_lockstep(full_depth):
    """Two draft/verify steps (K = 8) of the full-depth pair in lock-step: draft
    and verify logits, candidates, accept counts and KV lengths."""
    if not hasattr(full_depth, "cache_t"):
        full_depth.prefill()
    for i in range(2):
        say(f"[gpu] 8B/1B full depth: step {i + 1}")
        full_depth.step()
    say(f"    max |logit err| at full depth {full_depth.worst:.4g}")


def test_16k_context_8b_width_slice_lockstep(B):
    """The long-context workload's attention plan at its real shape: one
    layer of the 8B-shaped target (32 query / 8 KV heads of 128, group 4) and
    of the 1B-shaped draft over a 16 384-token prompt; the decode passes take
    640-key chunks (26 of them, one query group per KV head) combined by the
    many-chunk merge.  The oracle ingests the prompt's keys and values without
    logits (oracle.fill_cache) and runs the last token, then two steps."""
    from gpu_common import Lockstep
    wl = pi.WORKLOADS["llama8b_1b_long"]
    t_spec, d_spec = _slice(wl.target, 1), _slice(wl.draft, 1)
    prompt = [int(x) for x in pi.workload_prompts(wl)[0]]
    n = len(prompt)
    # the verify pass's plan: 8 KV heads x 1 query group, chunks the shortest
    # multiple of 128 keys that keeps the grid within 256 workgroups
    per = 256 // t_spec.n_kv_heads
    chunk = -(-(-(-(n + wl.k + 1) // per)) // 128) * 128
    assert (chunk, -(-(n + wl.k + 1) // chunk)) == (640, 26)
    say(f"[gpu] {n}-token context, 8B/1B width, 1 layer each: oracle build")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=n + 64, max_k=wl.k)
    try:
        ls = Lockstep(eng, target, draft, prompt, wl.k, wl.mask_id, tag="16k 8B width")
        say("[gpu] 16k 8B width: prefill")
        ls.prefill(cache_only_prefix=True)
        for i in range(2):
            say(f"[gpu] 16k 8B width: step {i + 1}")
            ls.step()
        say(f"    max |logit err| {ls.worst:.4g}")
    finally:
        eng.close()


def test_16k_context_chunked_attention_lockstep(B):
    wl = pi.WORKLOADS["tiny"]
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    n = pi.WORKLOADS["llama8b_1b_long"].prompt_len
    prompt = [int(x) for x in pi.gen_prompt(21, t_spec.vocab, n)]
    say(f"[gpu] {n}-token context on the narrow pair: oracle build")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=n + 64, max_k=8)
    try:
        say(f"[gpu] {n}-token context: lock-step K=8")
        worst = lockstep(eng, target, draft, prompt, 8, steps=2, mask_id=wl.mask_id, tag="16k")
        say(f"    max |logit err| {worst:.3g}")
    finally:
        eng.close()


@pytest.mark.parametrize("heads,hd,ctx,chunk", [(16, 128, 4200, 384), (32, 64, 4200, 640), (8, 128, 4200, 256)])
def test_long_key_chunks_lockstep(B, heads, hd, ctx, chunk):
    wl = pi.WORKLOADS["tiny"]
    t_spec = replace(pi.with_dtype(wl.target, "bf16"), n_layers=1, d_model=heads * hd, n_heads=heads,
                     n_kv_heads=heads, head_dim=hd, ffn_dim=512)
    d_spec = pi.with_dtype(wl.draft, "bf16")
    # the plan's chunk for the verify pass: the shortest multiple of 128 keys
    # that keeps KV heads x chunks (one query group) within 256 workgroups
    per = 256 // heads
    assert chunk == max(256, -(-(-(-(ctx + 9) // per)) // 128) * 128) and heads * -(-(ctx + 9) // chunk) <= 256
    if chunk == 256:
        assert -(-(ctx + 9) // chunk) > 16          # the many-chunk merge
    prompt = [int(x) for x in pi.gen_prompt(23, t_spec.vocab, ctx)]
    say(f"[gpu] {heads}x{hd} KV heads, {ctx}-token context ({chunk}-key chunks): oracle build")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=ctx + 64, max_k=8)
    try:
        worst = lockstep(eng, target, draft, prompt, 8, steps=2, mask_id=wl.mask_id, tag=f"chunk{chunk}")
        say(f"    max |logit err| {worst:.3g}")
    finally:
        eng.close()
