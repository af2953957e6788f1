"""GPU check of the allocation-free COD entry point (pard_cod_build_noalloc)
against pard_cod_build: two calls in a row on the same GPU, the second with a
smaller batch, every packed output and length bit-exact."""
import numpy as np
import pytest

import pard_inputs as pi
from gpu_common import require_gpu, say

pytestmark = pytest.mark.gpu


def _batch(seed, n, lo, hi, vocab):
    lens = pi.gen_prompt_lengths(seed, n, lo, hi)
    samples = [pi.gen_prompt(seed, vocab, int(L), b) for b, L in enumerate(lens)]
    offs = np.zeros(n + 1, np.int64)
    offs[1:] = np.cumsum(lens)
    return np.concatenate(samples).astype(np.int32), offs


def test_cod_noalloc_matches_workspace_call_twice():
    require_gpu()
    import torch
    from paper_2504_18583_amd import binding as B
    vocab = 1024
    for call, (seed, n, lo, hi) in enumerate(((31, 300, 2, 700), (32, 37, 2, 90))):
        flat, offs = _batch(seed, n, lo, hi, vocab)
        tokens = torch.from_numpy(flat).cuda()
        say(f"[gpu] cod noalloc call {call + 1}: {n} samples, {int(offs[-1])} tokens")
        ref_offs, ref, ref_len = B.cod_build(tokens, offs, 8, 0.7, 0.2, vocab - 1, 5)
        got_offs, got, got_len = B.cod_build_noalloc(tokens, offs, 8, 0.7, 0.2, vocab - 1, 5)
        torch.cuda.synchronize()
        assert np.array_equal(ref_offs, got_offs)
        assert torch.equal(ref_len, got_len)
        lens = ref_len.cpu().numpy()
        for name in ("ids", "labels", "pos", "section", "column"):
            a, g = ref[name].cpu().numpy(), got[name].cpu().numpy()
            for s in range(n):       # packed regions (past each length the outputs are unspecified)
                o = ref_offs[s]
                assert np.array_equal(a[o:o + lens[s]], g[o:o + lens[s]]), (name, s)
