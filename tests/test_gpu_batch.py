"""GPU parity for the batched workload's shape of state: 32 independent
sequence slots with ragged prompt lengths (uniform in [256, 2048], as the
batch-32 workload draws them), each with its own acceptance and KV rollback,
stepped in interleaved order so that any state leaking between slots shows.

The narrow pair keeps the oracle fast; the full-width kernels are covered by
the single-sequence slices.  Slots run one pass at a time (this build has no
multi-sequence pass)."""
import pytest

import oracle
import pard_inputs as pi
from gpu_common import Lockstep, require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


def test_32_ragged_slots_interleaved_lockstep(B):
    wl = pi.WORKLOADS["tiny"]
    bw = pi.WORKLOADS["llama8b_1b_batch32"]
    t_spec, d_spec = pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")
    lo, hi = bw.prompt_len_range
    lens = pi.gen_prompt_lengths(bw.seed, bw.batch, lo, hi)
    prompts = [[int(x) for x in pi.gen_prompt(bw.seed, t_spec.vocab, int(n), b)] for b, n in enumerate(lens)]
    target, draft = oracle.build_model(t_spec), oracle.build_model(d_spec)
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
            say(f"[gpu] batch: step {step} over {len(slots)} slots")
            for ls in slots:
                ls.step()
        say(f"    max |logit err| {max(ls.worst for ls in slots):.3g}")
        # every slot kept its own lengths
        for b, ls in enumerate(slots):
            assert eng.kv_len(B.PARD_TARGET, seq=b) == ls.cache_t.length
            assert eng.kv_len(B.PARD_DRAFT, seq=b) == ls.cache_d.length
    finally:
        eng.close()
