"""CPU oracle for the PARD speculative-decode step.

TEST INFRASTRUCTURE.  This package is the slow, plain float64 reference that
the GPU path is checked against.  Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path
(the HIP library ``libpard.so`` and its Python binding) never routes through
it, and it shares no code with that path.  Inputs come from ``pard_inputs``.

Modules:
* ``oracle.model`` -- the decoder (forward with and without a KV cache).
* ``oracle.pard``  -- greedy decoding (eq. 2) and the PARD draft / verify /
  accept loop (Sec. 2.2, Sec. 3.1 eq. 7).
* ``oracle.sampling`` -- speculative sampling at temperature T > 0 (the
  rejection rule Sec. 1 and Sec. 2.2 cite) on the PARD draft, with a
  counter-based SplitMix64 generator.
* ``oracle.cod`` -- conditional drop-token training-data processing (Sec. 3.2,
  Alg. 1, App. B).

Pins (tests marked "not gpu"): the decoder against the independent
Hugging Face Llama/Qwen2 implementations and torch's attention/normalisation
routines; cached vs. uncached forward position by position; the one-pass draft
against K separate uncached passes (eq. 7); lossless greedy speculative
decoding against plain greedy decoding (eq. 2) for K in {1, 2, 4, 8, 12};
forced-candidate acceptance; the draft-equals-target special case.
Sampling: SplitMix64's published outputs; inverse-CDF drawing against the
weights; the keep / residual / bonus rule against the target distribution at
every position (chi-square); the whole sampled loop against enumerated
autoregressive marginals on a small vocabulary; vanishing temperature ==
greedy.  COD: App. B's worked example, the kept-token closed form (App. A's
3.37M), the integrity condition, and packed samples reproducing the eq. 7
draft pass through the decoder.
"""
from .model import (KVCache, Model, attention, fill_cache, forward_cached, forward_full, linear,
                    rms_norm, rope, silu)
from .pard import (PardTrace, accept_prefix, argmax_rows, draft_step, greedy_ar,
                   pard_generate, prefill, vanilla_draft_step, vanilla_generate, verify_step)
from . import cod, sampling


def build_model(spec, layers=None) -> Model:
    """Oracle model with weights generated from ``spec`` by ``pard_inputs``."""
    import pard_inputs
    return Model(spec, pard_inputs.gen_model_weights(spec, layers=layers))
