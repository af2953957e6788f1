"""GPU parity of multi-sequence passes (the batch-32 workload's regime).

* 32 independent slots with ragged prompt lengths (uniform in [256, 2048], as
  the batch-32 workload draws them), each with its own acceptance and KV
  rollback: stepped one slot at a time (granular calls), and stepped together
  by the fused loop, whose draft and verify passes then hold every slot's
  rows (256-512 and 288 rows at K = 8: the row-block GEMM, split inputs,
  per-sequence attention, tails and next-pass staging).  Each slot is checked
  against its own oracle run every step.
* The same at the full width of the 8B/1B-shaped pair (2 / 1 layers), with
  shorter ragged prompts so that the fp64 oracle keeps up.
* Small batches (skinny GEMMs with several sequences), plain target steps
  (K = 0) over many slots, and whole fused generations against the target's
  greedy decoding (lossless, Sec. 2.1 eq. 2)."""
from dataclasses import replace

import numpy as np
import pytest

import oracle
import pard_inputs as pi
from gpu_common import MARGIN, BatchLockstep, Lockstep, margins, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


def _tiny():
    wl = pi.WORKLOADS["tiny"]
    return wl, pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")


def _ragged_prompts(seed, batch, lo, hi, vocab):
    lens = pi.gen_prompt_lengths(seed, batch, lo, hi)
    return [[int(x) for x in pi.gen_prompt(seed, vocab, int(n), b)] for b, n in enumerate(lens)]


@pytest.fixture(scope="module")
def tiny_models():
    wl, t_spec, d_spec = _tiny()
    return oracle.build_model(t_spec), oracle.build_model(d_spec)


def test_32_ragged_slots_interleaved_lockstep(B, tiny_models):
    wl, t_spec, d_spec = _tiny()
    bw = pi.WORKLOADS["llama8b_1b_batch32"]
    lo, hi = bw.prompt_len_range
    prompts = _ragged_prompts(bw.seed, bw.batch, lo, hi, t_spec.vocab)
    target, draft = tiny_models
    k = bw.k
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=hi + 64, max_k=k, max_batch=bw.batch)
    try:
        slots = [Lockstep(eng, target, draft, p, k, wl.mask_id, seq=b, tag=f"slot {b} (L={len(p)})")
                 for b, p in enumerate(prompts)]
        for b, ls in enumerate(slots):
            if b % 8 == 0:
                say(f"[gpu] batch: prefill slots {b}..{b + 7}")
            ls.prefill()
        for step in range(2):
            say(f"[gpu] batch: step {step} over {len(slots)} slots, one at a time")
            for ls in slots:
                ls.step()
        say(f"    max |logit err| {max(ls.worst for ls in slots):.3g}")
        for b, ls in enumerate(slots):
            assert eng.kv_len(B.PARD_TARGET, seq=b) == ls.cache_t.length
            assert eng.kv_len(B.PARD_DRAFT, seq=b) == ls.cache_d.length
    finally:
        eng.close()


def test_32_ragged_slots_batched_passes_lockstep(B, tiny_models):
    wl, t_spec, d_spec = _tiny()
    bw = pi.WORKLOADS["llama8b_1b_batch32"]
    lo, hi = bw.prompt_len_range
    prompts = _ragged_prompts(bw.seed, bw.batch, lo, hi, t_spec.vocab)
    target, draft = tiny_models
    k = bw.k
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=hi + 128, max_k=k, max_batch=bw.batch)
    try:
        bl = BatchLockstep(eng, target, draft, prompts, k, wl.mask_id, tag="batched")
        say("[gpu] batched passes: prefill 32 slots")
        bl.prefill()
        for step in range(3):
            say(f"[gpu] batched passes: fused step {step} ({len(prompts) * (k + 1)} verify rows)")
            bl.step(n_tokens=64)
        say(f"    max |logit err| {bl.worst:.3g}")
    finally:
        eng.close()


@pytest.mark.parametrize("n_slots,k", [(3, 4), (5, 6)])
def test_small_batches_skinny_path_lockstep(B, tiny_models, n_slots, k):
    wl, t_spec, d_spec = _tiny()
    prompts = _ragged_prompts(11 + n_slots, n_slots, 20, 90, t_spec.vocab)
    target, draft = tiny_models
    # non-contiguous slots, listed out of order
    slots = [2 * i + 1 for i in range(n_slots)][::-1]
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=256, max_k=k, max_batch=2 * n_slots + 2)
    try:
        bl = BatchLockstep(eng, target, draft, prompts, k, wl.mask_id, slots=slots, tag=f"{n_slots} slots")
        bl.prefill()
        for step in range(3):
            say(f"[gpu] {n_slots} slots, K={k}: fused step {step}")
            bl.step(n_tokens=40)
    finally:
        eng.close()


def test_plain_target_steps_over_40_slots(B, tiny_models):
    wl, t_spec, d_spec = _tiny()
    prompts = _ragged_prompts(21, 40, 8, 70, t_spec.vocab)
    target, draft = tiny_models
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=160, max_k=4, max_batch=40)
    try:
        bl = BatchLockstep(eng, target, draft, prompts, 0, wl.mask_id, tag="K=0")
        bl.prefill()
        for step in range(3):
            say(f"[gpu] 40 slots, K=0: fused step {step}")
            bl.step(n_tokens=16)
    finally:
        eng.close()


def test_batched_generation_equals_greedy_decoding(B, tiny_models):
    """Greedy PARD is lossless: every slot's output equals the target's own
    greedy continuation, up to the first near-tie of the oracle."""
    wl, t_spec, d_spec = _tiny()
    prompts = _ragged_prompts(31, 24, 12, 60, t_spec.vocab)
    target, draft = tiny_models
    n_tokens, k = 24, wl.k
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=128, max_k=k, max_batch=24)
    try:
        firsts = [eng.prefill(p, seq=b) for b, p in enumerate(prompts)]
        say("[gpu] 24 slots: one fused batched generation")
        res, stats = eng.generate_batch(list(range(24)), k, n_tokens)
        assert stats.tokens == 24 * n_tokens
        for b, p in enumerate(prompts):
            toks = res[b]
            assert len(toks) == n_tokens and toks[0] == firsts[b]
            ref = oracle.greedy_ar(target, p, n_tokens)
            # compare up to the first position whose oracle margin is small
            cache = oracle.KVCache(target)
            lg = oracle.forward_cached(target, cache, p, logits_rows=[len(p) - 1])
            for i in range(n_tokens):
                if margins(lg)[-1] <= MARGIN:
                    break
                assert toks[i] == ref[i], f"slot {b} token {i}: gpu {toks[i]} oracle {ref[i]}"
                lg = oracle.forward_cached(target, cache, [ref[i]])
            assert eng.kv_len(B.PARD_TARGET, seq=b) >= len(p) + n_tokens - 1
    finally:
        eng.close()


@pytest.mark.timeout(900)
def test_llama_8b_1b_full_width_slice_32_slots_batched(B):
    wl = pi.WORKLOADS["llama8b_1b_batch32"]
    t_spec = replace(pi.with_dtype(wl.target, "bf16"), n_layers=2)
    d_spec = replace(pi.with_dtype(wl.draft, "bf16"), n_layers=1)
    # ragged, but short enough for the fp64 oracle's prefill at full width
    prompts = _ragged_prompts(wl.seed, wl.batch, 16, 80, t_spec.vocab)
    say("[gpu] 8B/1B full-width slice, 32 slots: oracle build")
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
    eng = B.Engine(t_spec, d_spec, wl.mask_id, max_ctx=160, max_k=wl.k, max_batch=wl.batch)
    try:
        bl = BatchLockstep(eng, target, draft, prompts, wl.k, wl.mask_id, tag="8B/1B x32")
        say("[gpu] 8B/1B full-width slice, 32 slots: prefill")
        bl.prefill()
        for step in range(2):
            say(f"[gpu] 8B/1B full-width slice, 32 slots: fused step {step}")
            bl.step(n_tokens=48)
        say(f"    max |logit err| {bl.worst:.3g}")
    finally:
        eng.close()
