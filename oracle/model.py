"""Plain float64 Llama-style decoder: the oracle's model arithmetic.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
path (the HIP library and its binding) never calls it.

What it computes.  The paper fixes the decoding rule (greedy argmax over the
model's next-token distribution, Sec. 2.1 eq. 2) and says decoding is bound by
reloading weights and the KV cache (Sec. 2.1); the draft and target are
LLaMA3 / Qwen2.5 family decoders (Sec. 4.1).  The block below is the standard
decoder of those families, written out plainly:

    x = E[ids]
    per layer:  h = x + Attn(RMSNorm(x));  x = h + W_down(silu(W_gate y) * W_up y),
                with y = RMSNorm(h)
    logits = RMSNorm(x) @ lm_head^T

* RMSNorm(x) = x / sqrt(mean(x^2) + eps) * g.
* Attention: Q/K/V projections (+ bias for Qwen-shaped models), rotary
  position embedding in the rotate-half layout (dimension i pairs with
  i + head_dim/2, frequency theta^(-2i/head_dim), angle = position * frequency),
  grouped-query heads (query head h reads KV head floor(h * H_kv / H_q)),
  scale 1/sqrt(head_dim), causal over absolute positions, softmax with the
  row maximum subtracted.
* Everything is computed in float64.  Weights are the bf16- or
  fp32-rounded values produced by ``pard_inputs`` (exact in float64).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

F64 = np.float64


@dataclass
class Model:
    """A spec (``pard_inputs.ModelSpec``) plus its canonical weights."""
    spec: object
    weights: dict


def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray] = None) -> np.ndarray:
    """y = x W^T (+ b) for a canonical [out, in] weight, in float64."""
    y = x @ np.asarray(w, dtype=F64).T
    if b is not None:
        y = y + np.asarray(b, dtype=F64)
    return y


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(g, F64)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope_inv_freq(hd: int, theta: float, scaling=None) -> np.ndarray:
    """Rotary frequencies theta^(-2i/hd), i < hd/2.  With LLaMA-3.1-style
    scaling (factor, low_freq_factor, high_freq_factor, original length L):
    a frequency whose wavelength 2 pi / w is shorter than L / high_freq_factor
    is kept, one longer than L / low_freq_factor is divided by factor, and in
    between w is blended as (1 - s) w / factor + s w with
    s = (L / wavelength - low_freq_factor) / (high_freq_factor - low_freq_factor)."""
    inv_freq = float(theta) ** (-(2.0 * np.arange(hd // 2, dtype=F64)) / hd)
    if scaling is None:
        return inv_freq
    factor, low, high, orig = (float(v) for v in scaling)
    wavelen = 2.0 * np.pi / inv_freq
    s = (orig / wavelen - low) / (high - low)
    blended = (1.0 - s) * inv_freq / factor + s * inv_freq
    return np.where(wavelen < orig / high, inv_freq, np.where(wavelen > orig / low, inv_freq / factor, blended))


def rope(x: np.ndarray, pos: np.ndarray, theta: float, scaling=None) -> np.ndarray:
    """Rotate-half rotary embedding of x [n, H, hd] at absolute positions pos [n]."""
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = rope_inv_freq(hd, theta, scaling)
    ang = np.asarray(pos, F64)[:, None] * inv_freq[None, :]          # [n, half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
              q_pos: np.ndarray, k_pos: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention.

    q [n, H_q, hd]; k, v [m, H_kv, hd]; key j is visible to query i iff
    k_pos[j] <= q_pos[i].  Returns [n, H_q, hd].
    """
    n, hq, hd = q.shape
    hkv = k.shape[1]
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty((n, hq, hd), F64)
    for h in range(hq):
        kh = (h * hkv) // hq
        s = (q[:, h, :] @ k[:, kh, :].T) / np.sqrt(F64(hd))
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kh, :]
    return out


class KVCache:
    """Post-RoPE keys and values of every layer, one row per committed position."""

    def __init__(self, model: Model):
        s = model.spec
        self.k: List[np.ndarray] = [np.zeros((0, s.n_kv_heads, s.head_dim), F64)
                                    for _ in range(s.n_layers)]
        self.v: List[np.ndarray] = [np.zeros((0, s.n_kv_heads, s.head_dim), F64)
                                    for _ in range(s.n_layers)]

    @property
    def length(self) -> int:
        return self.k[0].shape[0] if self.k else 0

    def truncate(self, n: int) -> None:
        if n > self.length or n < 0:
            raise ValueError("truncate beyond the cache length")
        self.k = [a[:n] for a in self.k]
        self.v = [a[:n] for a in self.v]


def _layer(spec, lw: dict, x: np.ndarray, pos: np.ndarray,
           k_prev: np.ndarray, v_prev: np.ndarray):
    """One decoder layer over rows x at positions pos, after keys k_prev/v_prev.

    Returns (new x, keys of all positions, values of all positions)."""
    n = x.shape[0]
    hq, hkv, hd = spec.n_heads, spec.n_kv_heads, spec.head_dim
    y = rms_norm(x, lw["attn_norm"], spec.rms_eps)
    q = linear(y, lw["wq"], lw.get("bq")).reshape(n, hq, hd)
    k = linear(y, lw["wk"], lw.get("bk")).reshape(n, hkv, hd)
    v = linear(y, lw["wv"], lw.get("bv")).reshape(n, hkv, hd)
    q = rope(q, pos, spec.rope_theta, spec.rope_scaling)
    k = rope(k, pos, spec.rope_theta, spec.rope_scaling)
    k_all = np.concatenate([k_prev, k], axis=0)
    v_all = np.concatenate([v_prev, v], axis=0)
    k_pos = np.arange(k_all.shape[0])
    a = attention(q, k_all, v_all, pos, k_pos).reshape(n, hq * hd)
    h = x + linear(a, lw["wo"])
    y = rms_norm(h, lw["mlp_norm"], spec.rms_eps)
    m = silu(linear(y, lw["w_gate"])) * linear(y, lw["w_up"])
    return h + linear(m, lw["w_down"]), k_all, v_all


def _head(model: Model, x: np.ndarray) -> np.ndarray:
    s, w = model.spec, model.weights
    return linear(rms_norm(x, w["final_norm"], s.rms_eps), w["lm_head"])


def forward_full(model: Model, ids: Sequence[int]) -> np.ndarray:
    """Logits [n, V] of every position of ``ids``, with no cache (positions 0..n-1)."""
    s, w = model.spec, model.weights
    ids = np.asarray(ids, dtype=np.int64)
    pos = np.arange(len(ids))
    x = np.asarray(np.asarray(w["embed"])[ids], F64)
    empty = np.zeros((0, s.n_kv_heads, s.head_dim), F64)
    for l in range(s.n_layers):
        x, _, _ = _layer(s, w["layers"][l], x, pos, empty, empty)
    return _head(model, x)


def forward_cached(model: Model, cache: KVCache, ids: Sequence[int],
                   logits_rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Run ``ids`` at positions cache.length .. cache.length+n-1 and append their K/V.

    Returns logits of the rows listed in ``logits_rows`` (all rows by default),
    shape [len(logits_rows), V]."""
    s, w = model.spec, model.weights
    ids = np.asarray(ids, dtype=np.int64)
    start = cache.length
    pos = np.arange(start, start + len(ids))
    x = np.asarray(np.asarray(w["embed"])[ids], F64)
    for l in range(s.n_layers):
        x, cache.k[l], cache.v[l] = _layer(s, w["layers"][l], x, pos, cache.k[l], cache.v[l])
    rows = np.arange(len(ids)) if logits_rows is None else np.asarray(list(logits_rows), int)
    if rows.size == 0:
        return np.zeros((0, s.vocab), F64)
    return _head(model, x[rows])


def fill_cache(model: Model, cache: KVCache, ids: Sequence[int]) -> None:
    """Append the K/V of ``ids`` (positions cache.length ..) without any logits.

    The same layer arithmetic as ``forward_cached``, except that in the last
    layer only the keys and values are formed: the attention output and MLP
    of that layer feed nothing the cache holds.  Used to ingest long prompts
    whose outputs are not compared (a 1-layer model then needs no attention
    over the prompt at all)."""
    s, w = model.spec, model.weights
    ids = np.asarray(ids, dtype=np.int64)
    start = cache.length
    pos = np.arange(start, start + len(ids))
    x = np.asarray(np.asarray(w["embed"])[ids], F64)
    last = s.n_layers - 1
    for l in range(last):
        x, cache.k[l], cache.v[l] = _layer(s, w["layers"][l], x, pos, cache.k[l], cache.v[l])
    lw = w["layers"][last]
    n, hkv, hd = x.shape[0], s.n_kv_heads, s.head_dim
    y = rms_norm(x, lw["attn_norm"], s.rms_eps)
    k = rope(linear(y, lw["wk"], lw.get("bk")).reshape(n, hkv, hd), pos, s.rope_theta, s.rope_scaling)
    v = linear(y, lw["wv"], lw.get("bv")).reshape(n, hkv, hd)
    cache.k[last] = np.concatenate([cache.k[last], k], axis=0)
    cache.v[last] = np.concatenate([cache.v[last], v], axis=0)
