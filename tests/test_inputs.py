"""Pins for the shared seeded input generators (SplitMix64 + Box-Muller)."""
import json
import os

import numpy as np
import pytest
import torch
from scipy import stats

import pard_inputs as pi

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_splitmix64_published_outputs():
    g = _golden("splitmix64_state0.json")
    got = pi.uniform_u64(g["state"], 0, len(g["outputs_hex"]))
    assert [f"{int(v):016x}" for v in got] == g["outputs_hex"]


def test_uniform_stream_is_counter_based():
    key = pi.stream_key(7, 1, 33)
    full = pi.uniform_u64(key, 0, 1000)
    assert np.array_equal(pi.uniform_u64(key, 123, 77), full[123:200])


def test_box_muller_is_standard_normal():
    x = pi.normal_f64(pi.stream_key(3, 0, 5), 0, 400_000)
    assert abs(x.mean()) < 5e-3
    assert abs(x.var() - 1.0) < 1e-2
    assert stats.kstest(x, "norm").pvalue > 1e-3
    # the cos and sin halves of each pair are uncorrelated
    assert abs(np.corrcoef(x[0::2], x[1::2])[0, 1]) < 1e-2


def test_normal_subranges_match_full_stream():
    key = pi.stream_key(1, 0, 16)
    full = pi.normal_f64(key, 0, 101)
    for a, b in [(0, 1), (1, 2), (3, 50), (50, 101), (7, 8)]:
        assert np.array_equal(pi.normal_f64(key, a, b - a), full[a:b])


def test_round_bf16_matches_torch_rne():
    x = (pi.normal_f64(pi.stream_key(0, 0, 1), 0, 100_000) * 3.0).astype(np.float32)
    x = np.concatenate([x, np.array([1.00390625, 1.01171875, -1.00390625, 0.0, 65504.0],
                                    np.float32)])
    ours = pi.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_gen_tensor_chunking_and_rounding(monkeypatch):
    spec = pi.WORKLOADS["tiny"].target
    a = pi.gen_tensor(0, 0, 16, (256, 256), 0.02, "bf16")
    monkeypatch.setattr(pi, "_CHUNK", 1000)   # many odd-sized chunks across threads
    b = pi.gen_tensor(0, 0, 16, (256, 256), 0.02, "bf16")
    assert np.array_equal(a, b)
    assert np.array_equal(pi.round_bf16(a), a)
    assert abs(a.std() - 0.02) < 5e-4
    c = pi.gen_tensor(0, 0, 16, (256, 256), 0.02, "fp32")
    assert np.array_equal(pi.round_bf16(c), a)


def test_prompts_exclude_mask_id():
    p = pi.gen_prompt(0, 1024, 20_000)
    assert p.min() >= 0 and p.max() == 1022
    assert p.dtype == np.int32
    lens = pi.gen_prompt_lengths(4, 32, 256, 2048)
    assert lens.min() >= 256 and lens.max() <= 2048
    wl = pi.WORKLOADS["llama8b_1b_batch32"]
    prompts = pi.workload_prompts(wl)
    assert len(prompts) == 32 and [len(x) for x in prompts] == list(lens)


@pytest.mark.parametrize("key,tol", [("llama8b_1b.target", 0.005), ("llama8b_1b.draft", 0.005),
                                     ("qwen7b_05b.target", 0.01), ("qwen7b_05b.draft", 0.005)])
def test_shapes_match_published_model_sizes(key, tol):
    g = _golden("model_sizes.json")
    wl, role = key.split(".")
    spec = getattr(pi.WORKLOADS[wl], role)
    assert abs(spec.n_params() / 1e9 - g[key]) <= tol


def test_layer_subset_generation_is_consistent():
    spec = pi.WORKLOADS["tiny"].target
    full = pi.gen_model_weights(spec)
    part = pi.gen_model_weights(spec, layers=[1])
    assert np.array_equal(full["layers"][1]["w_down"], part["layers"][1]["w_down"])
    assert set(part["layers"]) == {1}
