"""Pins for the oracle's COD training-data processing (oracle/cod.py).

* App. B's worked example (r = 0.5, four columns, K = 3): the valid subtask-3
  columns given subtask 2's kept ones, and the attention context of m_{1,2}
  and m_{1,3} as the example states it.
* App. A / eq. 10-11: the kept-token total is N * sum_k max(r^{k-1}, r_min)
  (3.3731 N for r = 0.7, r_min = 0.2, K = 8: the appendix's 3.37M per 1M
  tokens) up to one column per subtask at the sequence end; below N / (1 - r)
  without the floor.
* The COD condition (integrity of prefix key/value states): every kept
  token's whole context is kept.
* Training data meets inference: a packed sample run through the decoder with
  its attention mask and positions gives, at every kept token of subtask k,
  the logits of the one-pass PARD draft (eq. 7) over its real prefix and k-1
  mask tokens -- the conditioning of eq. 8.
"""
import numpy as np
import pytest

import oracle
import pard_inputs as pi
from oracle import cod
from oracle.model import F64, linear, rms_norm, rope, silu


def test_worked_example_structure():
    tokens = [11, 12, 13, 14, 15]                    # "tell me a story about": four columns
    n, seen = 4, 0
    for seed in range(200):
        s = cod.cod_process(tokens, 3, 0.5, 0.0, 99, seed, 0)
        assert len(s.kept[1]) == 2 and len(s.kept[2]) == 1      # 50 % and 25 % of 4
        if s.kept[1] != [1, 2]:
            continue
        seen += 1                                    # the example's subtask-2 choice
        assert s.kept[2][0] in (2, 3)                # m_{1,1} needs the dropped m_{0,0}
    assert seen > 0
    # contexts the example names: m_{1,3} sees [tell, me, m_{0,2}], m_{1,2} sees [tell, m_{0,1}]
    ctx = lambda k, j: [(kb, jb) for kb in (1, 2, 3) for jb in range(n) if cod.attends(k, j, kb, jb)]
    assert ctx(3, 3) == [(1, 0), (1, 1), (2, 2), (3, 3)]
    assert ctx(3, 2) == [(1, 0), (2, 1), (3, 2)]
    # subtask 1 is plain causal
    assert ctx(1, 2) == [(1, 0), (1, 1), (1, 2)]


def test_kept_total_matches_closed_form():
    n = 10_000
    tokens = np.arange(n + 1) % 500
    s = cod.cod_process(tokens, 8, 0.7, 0.2, 499, seed=3, sample=0)
    total = len(s.ids)
    closed = n * (1 + 0.7 + 0.49 + 0.343 + 0.2401 + 0.2 + 0.2 + 0.2)      # 3.3731 n
    assert abs(closed - 3.3731 * n) < 1e-6
    assert closed - 8 <= total <= closed
    assert [len(c) for c in s.kept[:5]] == [n, 7000, 4900, 3430, 2401]
    # without the floor: N (1 - r^K) / (1 - r) < N / (1 - r), each subtask's
    # count rounded to the nearest integer
    s2 = cod.cod_process(tokens, 8, 0.5, 0.0, 499, seed=3, sample=0)
    closed2 = n * (1 - 0.5 ** 8) / 0.5
    assert closed2 - 8 - 4 <= len(s2.ids) <= closed2 + 4 and closed2 < 2 * n


@pytest.mark.parametrize("k_max,r,r_min", [(8, 0.7, 0.2), (4, 0.5, 0.0), (6, 0.9, 0.3), (3, 1.0, 0.0)])
def test_every_kept_token_has_its_whole_context(k_max, r, r_min):
    rng = np.random.default_rng(k_max)
    for sample in range(20):
        tokens = rng.integers(0, 1000, size=int(rng.integers(2, 120)))
        s = cod.cod_process(tokens, k_max, r, r_min, 1000, seed=17, sample=sample)
        kept = [set(c) for c in s.kept]
        n = len(tokens) - 1
        for k in range(2, k_max + 1):
            assert len(kept[k - 1]) == min(cod.keep_target(n, k, r, r_min),
                                           sum(1 for j in range(n) if j >= k - 1 and j - 1 in kept[k - 2]))
            for j in kept[k - 1]:
                assert j - k + 1 >= 0
                for kp in range(2, k):
                    assert (j - k + kp) in kept[kp - 1], (k, j, kp)
        if r == 1.0:                                   # nothing dropped beyond the sequence start
            assert all(len(kept[k - 1]) == n - k + 1 for k in range(1, k_max + 1))
        # packed fields
        assert s.section == sorted(s.section)
        for k, j, i, lab, p in zip(s.section, s.column, s.ids, s.labels, s.pos):
            assert p == j and lab == tokens[j + 1] and i == (tokens[j] if k == 1 else 1000)


def test_selection_is_seeded_and_per_sample():
    tokens = list(range(300))
    a = cod.cod_process(tokens, 5, 0.6, 0.1, 7, seed=1, sample=4)
    assert a.kept == cod.cod_process(tokens, 5, 0.6, 0.1, 7, seed=1, sample=4).kept
    assert a.kept != cod.cod_process(tokens, 5, 0.6, 0.1, 7, seed=1, sample=5).kept
    assert a.kept != cod.cod_process(tokens, 5, 0.6, 0.1, 7, seed=2, sample=4).kept


def _masked_forward(model, ids, pos, mask):
    """The decoder over a packed sample: positions `pos`, row a attends to the
    rows b with mask[a, b] (a plain numpy restatement for this test only)."""
    s, w = model.spec, model.weights
    x = np.asarray(w["embed"], F64)[np.asarray(ids)]
    pos = np.asarray(pos)
    n, hq, hkv, hd = len(ids), s.n_heads, s.n_kv_heads, s.head_dim
    for l in range(s.n_layers):
        lw = w["layers"][l]
        y = rms_norm(x, lw["attn_norm"], s.rms_eps)
        q = rope(linear(y, lw["wq"]).reshape(n, hq, hd), pos, s.rope_theta)
        k = rope(linear(y, lw["wk"]).reshape(n, hkv, hd), pos, s.rope_theta)
        v = linear(y, lw["wv"]).reshape(n, hkv, hd)
        g = hq // hkv
        out = np.zeros((n, hq, hd))
        for h in range(hq):
            sc = q[:, h] @ k[:, h // g].T / np.sqrt(hd)
            sc = np.where(mask, sc, -np.inf)
            p = np.exp(sc - sc.max(axis=1, keepdims=True))
            out[:, h] = (p / p.sum(axis=1, keepdims=True)) @ v[:, h // g]
        hres = x + linear(out.reshape(n, hq * hd), lw["wo"])
        y = rms_norm(hres, lw["mlp_norm"], s.rms_eps)
        x = hres + linear(silu(linear(y, lw["w_gate"])) * linear(y, lw["w_up"]), lw["w_down"])
    return linear(rms_norm(x, w["final_norm"], s.rms_eps), w["lm_head"])


def test_packed_sample_reproduces_the_parallel_draft_pass():
    wl = pi.WORKLOADS["tiny"]
    draft = oracle.build_model(wl.draft)
    tokens = [int(x) for x in pi.gen_prompt(9, wl.draft.vocab, 14)]
    k_max = 4
    s = cod.cod_process(tokens, k_max, 0.7, 0.2, wl.mask_id, seed=5, sample=0)
    logits = _masked_forward(draft, s.ids, s.pos, cod.attention_mask(s))
    checked = 0
    for row, (k, j) in enumerate(zip(s.section, s.column)):
        prefix = tokens[:j - k + 2]                   # real tokens t_0 .. t_{j-k+1}
        cache = oracle.KVCache(draft)
        if len(prefix) > 1:
            oracle.forward_cached(draft, cache, prefix[:-1], logits_rows=[])
        _, dl = oracle.draft_step(draft, cache, [prefix[-1]], k, wl.mask_id)   # eq. 7, one pass
        assert np.allclose(logits[row], dl[k - 1], atol=1e-9, rtol=1e-9), (k, j)
        checked += 1
    assert checked == len(s.ids) and max(s.section) == k_max
