"""GPU parity of COD training-data processing (pard_cod_build) against the
oracle, bit for bit: packed ids, labels, positions, subtask and column of
every sample and its packed length, over ragged batches (2 to 8193 tokens)
and the retention settings of the paper (r = 0.7, r_min = 0.2, K = 8: App. A)
and of App. B's example (r = 0.5)."""
import numpy as np
import pytest

import pard_inputs as pi
from gpu_common import require_gpu, say
from oracle import cod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    require_gpu()
    from paper_2504_18583_amd import binding
    return binding


def _run(B, samples, k, r, r_min, mask_id, seed):
    import torch
    offs = np.zeros(len(samples) + 1, np.int64)
    offs[1:] = np.cumsum([len(x) for x in samples])
    flat = torch.from_numpy(np.concatenate(samples).astype(np.int32)).cuda()
    out_offs, out, out_len = B.cod_build(flat, offs, k, r, r_min, mask_id, seed)
    torch.cuda.synchronize()
    host = {name: v.cpu().numpy() for name, v in out.items()}
    return out_offs, host, out_len.cpu().numpy()


def _check(samples, out_offs, host, lens, k, r, r_min, mask_id, seed):
    for s, toks in enumerate(samples):
        ref = cod.cod_process(toks, k, r, r_min, mask_id, seed, s)
        assert lens[s] == len(ref.ids), f"sample {s}: length {lens[s]} oracle {len(ref.ids)}"
        o = int(out_offs[s])
        for name in ("ids", "labels", "pos", "section", "column"):
            got = host[name][o:o + lens[s]]
            assert np.array_equal(got, np.asarray(getattr(ref, name), np.int32)), f"sample {s} {name}"


@pytest.mark.parametrize("k,r,r_min", [(8, 0.7, 0.2), (3, 0.5, 0.0), (1, 0.7, 0.2), (6, 1.0, 0.0), (5, 0.3, 0.3)])
def test_cod_matches_oracle_ragged_batch(B, k, r, r_min):
    rng = np.random.default_rng(k)
    lens = [2, 3, 5, 64, 65, 1024, 1025] + [int(x) for x in rng.integers(2, 700, size=40)]
    samples = [rng.integers(0, 128256, size=n).astype(np.int64) for n in lens]
    say(f"[gpu] cod: {len(samples)} samples, K={k} r={r} r_min={r_min}")
    out_offs, host, got = _run(B, samples, k, r, r_min, 128255, seed=2504)
    _check(samples, out_offs, host, got, k, r, r_min, 128255, 2504)


def test_cod_longest_samples(B):
    rng = np.random.default_rng(7)
    samples = [rng.integers(0, 1000, size=n).astype(np.int64) for n in (8193, 8192, 4097)]
    say("[gpu] cod: samples of 8193, 8192 and 4097 tokens, K=8")
    out_offs, host, got = _run(B, samples, 8, 0.7, 0.2, 999, seed=1)
    _check(samples, out_offs, host, got, 8, 0.7, 0.2, 999, 1)
    # App. A: about 3.3731 packed tokens per column at r = 0.7, r_min = 0.2, K = 8
    assert abs(got[0] / 8192 - 3.3731) < 1e-3


def test_cod_workload_shapes_spot_check(B):
    """The bench's COD workload (prompt lengths of the batch-32 workload's
    range), every 97th sample against the oracle."""
    wl = pi.WORKLOADS["llama8b_1b_batch32"]
    lo, hi = wl.prompt_len_range
    lens = pi.gen_prompt_lengths(11, 512, lo, hi)
    samples = [pi.gen_prompt(11, wl.target.vocab, int(n), b).astype(np.int64) for b, n in enumerate(lens)]
    out_offs, host, got = _run(B, samples, 8, 0.7, 0.2, wl.mask_id, seed=5)
    for s in range(0, len(samples), 97):
        ref = cod.cod_process(samples[s], 8, 0.7, 0.2, wl.mask_id, 5, s)
        o = int(out_offs[s])
        assert got[s] == len(ref.ids), f"sample {s}"
        for name in ("ids", "labels", "pos", "section", "column"):
            assert np.array_equal(host[name][o:o + got[s]], np.asarray(getattr(ref, name), np.int32)), (s, name)
