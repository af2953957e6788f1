"""Pin the step bytes model against the paper's Table 3 (draft-phase traffic)."""
import json
import os

import pard_inputs as pi
from paper_2504_18583_amd import bytes_model as bm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table3_draft_bandwidth.json")


def test_draft_traffic_matches_table3_and_is_flat_in_k():
    with open(GOLDEN) as f:
        g = json.load(f)
    draft = pi.WORKLOADS["llama8b_1b"].draft
    per_k = {}
    for k_str, gb in g["pard"].items():
        k = int(k_str)
        got = bm.draft_pass_bytes(draft, k, n_pending=1, context=512) / 1e9
        assert abs(got - gb) / gb < 0.005, (k, got, gb)
        per_k[k] = got
    assert max(per_k.values()) - min(per_k.values()) < 0.001 * min(per_k.values())


def test_weight_stream_sizes():
    wl = pi.WORKLOADS["llama8b_1b"]
    assert abs(bm.streamed_params(wl.target) / 1e6 - 7504.9) < 0.1
    assert abs(bm.streamed_params(wl.draft) / 1e6 - 1235.8) < 0.1
    assert bm.kv_bytes_per_token(wl.target) == 131072
    assert bm.kv_bytes_per_token(wl.draft) == 32768
