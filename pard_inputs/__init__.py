"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module holds the workload definitions (model shapes, seeds, prompt
recipes) and one counter-based random generator.  It contains none of the
method's arithmetic: no transformer maths, no drafting, no verification.
Both sides of the parity tests draw their inputs from here; the HIP library
implements the same generator on the device from the same published
definitions (it does not import this module).

Generator definition (the contract both implementations follow)
----------------------------------------------------------------
* SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014; constants as in Vigna's public-domain
  ``splitmix64.c``).  ``mix64`` is its output function; the i-th output
  (i = 0, 1, ...) of the stream with state ``key`` is
  ``mix64(key + (i + 1) * GAMMA)`` modulo 2**64.
* Stream key of tensor ``t`` of weight stream ``s`` under ``seed``:
  ``mix64(seed * 2**20 + s * 2**16 + t)``.
* Normal deviates by the basic Box-Muller transform (Box & Muller, 1958):
  element i of a tensor (row-major, canonical ``[out, in]`` order) uses the
  outputs z0 = out(2*(i//2)) and z1 = out(2*(i//2) + 1):
  ``u1 = ((z0 >> 11) + 1) * 2**-53`` (in (0, 1]),
  ``u2 = (z1 >> 11) * 2**-53`` (in [0, 1)),
  ``r = sqrt(-2 ln u1)``, ``theta = (2*pi) * u2``;
  even i takes ``r cos theta``, odd i takes ``r sin theta``.
  The value is multiplied by ``init_std`` in float64, rounded to float32
  (round-to-nearest) and, for bf16 weights, rounded float32 -> bf16 with
  round-to-nearest-even.
* Token ids: output i of stream (seed, 15, sequence) taken modulo (V - 1),
  so the last id (the mask id) never appears in a prompt.
* Prompt lengths (batched workload): ``lo + out(b) mod (hi - lo + 1)`` from
  stream (seed, 14, 0).

Tensor ordinals: embedding 0, lm_head 1 (untied models only), and for layer
l: ``16 * (l + 1) + j`` with j = wq 0, wk 1, wv 2, wo 3, w_gate 4, w_up 5,
w_down 6, bq 7, bk 8, bv 9.  RMSNorm gains are 1 and are not drawn.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Tuple

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MIX_C1 = 0xBF58476D1CE4E5B9
MIX_C2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

PROMPT_STREAM = 15
LENGTH_STREAM = 14

T_EMBED, T_LM_HEAD = 0, 1
T_WQ, T_WK, T_WV, T_WO, T_WG, T_WU, T_WD, T_BQ, T_BK, T_BV = range(10)


def layer_tensor(layer: int, j: int) -> int:
    return 16 * (layer + 1) + j


# --------------------------------------------------------------------------
# SplitMix64 (integer-exact, vectorised over numpy uint64)
# --------------------------------------------------------------------------

def mix64_int(z: int) -> int:
    """SplitMix64 output function on a Python int (mod 2**64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX_C1) & MASK64
    z = ((z ^ (z >> 27)) * MIX_C2) & MASK64
    return z ^ (z >> 31)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX_C1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX_C2)
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, stream: int, tensor: int) -> int:
    if not (0 <= seed < (1 << 44) and 0 <= stream < 16 and 0 <= tensor < (1 << 16)):
        raise ValueError("seed/stream/tensor out of range")
    return mix64_int((seed << 20) + (stream << 16) + tensor)


def uniform_u64(key: int, start: int, count: int) -> np.ndarray:
    """Outputs start .. start+count-1 of the SplitMix64 stream with state ``key``."""
    idx = np.arange(start + 1, start + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        state = np.uint64(key) + idx * np.uint64(GAMMA)
        return _mix64_np(state)


def normal_f64(key: int, start: int, count: int) -> np.ndarray:
    """Standard-normal deviates for tensor elements start .. start+count-1."""
    if count == 0:
        return np.zeros(0, np.float64)
    p0 = start // 2
    p1 = (start + count + 1) // 2
    z = uniform_u64(key, 2 * p0, 2 * (p1 - p0))
    z0 = z[0::2]
    z1 = z[1::2]
    scale = np.float64(2.0 ** -53)
    u1 = ((z0 >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * scale
    u2 = (z1 >> np.uint64(11)).astype(np.float64) * scale
    r = np.sqrt(-2.0 * np.log(u1))
    theta = np.float64(2.0 * np.pi) * u2
    out = np.empty(2 * (p1 - p0), np.float64)
    out[0::2] = r * np.cos(theta)
    out[1::2] = r * np.sin(theta)
    off = start - 2 * p0
    return out[off:off + count]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bf16 (ties to even), returned as float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32)


_CHUNK = 1 << 22


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def gen_tensor(seed: int, stream: int, tensor: int, shape: Tuple[int, ...],
               std: float, dtype: str) -> np.ndarray:
    """One weight tensor, canonical row-major layout, values held as float32."""
    n = int(np.prod(shape))
    key = stream_key(seed, stream, tensor)
    out = np.empty(n, np.float32)

    def work(c0: int) -> None:
        c1 = min(n, c0 + _CHUNK)
        v = (normal_f64(key, c0, c1 - c0) * np.float64(std)).astype(np.float32)
        out[c0:c1] = round_bf16(v) if dtype == "bf16" else v

    starts = list(range(0, n, _CHUNK))
    if len(starts) > 1:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(work, starts))
    elif starts:
        work(0)
    return out.reshape(shape)


# --------------------------------------------------------------------------
# Workload definitions
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class ModelSpec:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float
    rope_theta: float
    init_std: float = 0.02
    qkv_bias: bool = False
    tied: bool = False
    dtype: str = "bf16"          # rounding applied to generated weights
    seed: int = 0
    stream: int = 0              # weight stream id (target 0, draft 1)
    # LLaMA-3.1-style rotary frequency scaling: (factor, low_freq_factor,
    # high_freq_factor, original max positions); None = plain RoPE
    rope_scaling: Optional[Tuple[float, float, float, int]] = None

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def n_params(self, with_embedding: bool = True) -> int:
        d, f = self.d_model, self.ffn_dim
        per_layer = (d * self.q_dim + 2 * d * self.kv_dim + self.q_dim * d
                     + 3 * d * f + 2 * d)
        if self.qkv_bias:
            per_layer += self.q_dim + 2 * self.kv_dim
        total = self.n_layers * per_layer + d
        total += self.vocab * d  # embedding (== lm_head when tied)
        if not self.tied:
            total += self.vocab * d
        if not with_embedding:
            total -= self.vocab * d
        return total


@dataclass(frozen=True)
class Workload:
    name: str
    target: ModelSpec
    draft: ModelSpec
    seed: int
    prompt_len: int
    k: int
    n_tokens: int
    batch: int = 1
    k_sweep: Tuple[int, ...] = ()
    prompt_len_range: Optional[Tuple[int, int]] = None

    @property
    def mask_id(self) -> int:
        return self.target.vocab - 1


def _pair(seed: int, tgt: dict, drf: dict) -> Tuple[ModelSpec, ModelSpec]:
    return (ModelSpec(seed=seed, stream=0, **tgt), ModelSpec(seed=seed, stream=1, **drf))


_TINY_T = dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=688,
               vocab=1024, rms_eps=1e-5, rope_theta=1e4, tied=False)
_TINY_D = dict(n_layers=1, d_model=128, n_heads=2, n_kv_heads=1, head_dim=64, ffn_dim=344,
               vocab=1024, rms_eps=1e-5, rope_theta=1e4, tied=True)
_LLAMA8B = dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                ffn_dim=14336, vocab=128256, rms_eps=1e-5, rope_theta=5e5, tied=False)
_LLAMA1B = dict(n_layers=16, d_model=2048, n_heads=32, n_kv_heads=8, head_dim=64,
                ffn_dim=8192, vocab=128256, rms_eps=1e-5, rope_theta=5e5, tied=True)
_QWEN7B = dict(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
               ffn_dim=18944, vocab=152064, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
               tied=False)
_QWEN05B = dict(n_layers=24, d_model=896, n_heads=14, n_kv_heads=2, head_dim=64,
                ffn_dim=4864, vocab=152064, rms_eps=1e-6, rope_theta=1e6, qkv_bias=True,
                tied=True)


def _workloads() -> Dict[str, Workload]:
    w = {}
    t, d = _pair(0, dict(_TINY_T, dtype="fp32"), dict(_TINY_D, dtype="fp32"))
    w["tiny"] = Workload("tiny", t, d, seed=0, prompt_len=32, k=4, n_tokens=64)
    t, d = _pair(1, _LLAMA8B, _LLAMA1B)
    w["llama8b_1b"] = Workload("llama8b_1b", t, d, seed=1, prompt_len=512, k=8, n_tokens=512)
    t, d = _pair(2, _QWEN7B, _QWEN05B)
    w["qwen7b_05b"] = Workload("qwen7b_05b", t, d, seed=2, prompt_len=1024, k=8,
                               n_tokens=256, k_sweep=(4, 8, 12))
    t, d = _pair(3, _LLAMA8B, _LLAMA1B)
    w["llama8b_1b_long"] = Workload("llama8b_1b_long", t, d, seed=3, prompt_len=16384, k=8,
                                    n_tokens=256)
    t, d = _pair(4, _LLAMA8B, _LLAMA1B)
    w["llama8b_1b_batch32"] = Workload("llama8b_1b_batch32", t, d, seed=4, prompt_len=2048,
                                       k=8, n_tokens=256, batch=32,
                                       prompt_len_range=(256, 2048))
    return w


WORKLOADS: Dict[str, Workload] = _workloads()


def with_dtype(spec: ModelSpec, dtype: str) -> ModelSpec:
    return replace(spec, dtype=dtype)


# --------------------------------------------------------------------------
# Model weights (canonical layout) and prompts
# --------------------------------------------------------------------------

def gen_model_weights(spec: ModelSpec, layers: Optional[List[int]] = None,
                      progress=None) -> dict:
    """All weights of one model as float32 arrays in canonical [out, in] layout.

    ``layers`` restricts generation to a subset of layer indices (each layer's
    values do not depend on which other layers are generated).  ``progress``
    (optional) is called with a short message after each generated layer.
    """
    s, d, f = spec, spec.d_model, spec.ffn_dim

    def g(tensor: int, shape: Tuple[int, ...]) -> np.ndarray:
        return gen_tensor(s.seed, s.stream, tensor, shape, s.init_std, s.dtype)

    w = {"embed": g(T_EMBED, (s.vocab, d))}
    w["lm_head"] = w["embed"] if s.tied else g(T_LM_HEAD, (s.vocab, d))
    w["final_norm"] = np.ones(d, np.float32)
    idx = range(s.n_layers) if layers is None else layers
    w["layers"] = {}
    for l in idx:
        lw = {
            "attn_norm": np.ones(d, np.float32),
            "mlp_norm": np.ones(d, np.float32),
            "wq": g(layer_tensor(l, T_WQ), (s.q_dim, d)),
            "wk": g(layer_tensor(l, T_WK), (s.kv_dim, d)),
            "wv": g(layer_tensor(l, T_WV), (s.kv_dim, d)),
            "wo": g(layer_tensor(l, T_WO), (d, s.q_dim)),
            "w_gate": g(layer_tensor(l, T_WG), (f, d)),
            "w_up": g(layer_tensor(l, T_WU), (f, d)),
            "w_down": g(layer_tensor(l, T_WD), (d, f)),
        }
        if s.qkv_bias:
            lw["bq"] = g(layer_tensor(l, T_BQ), (s.q_dim,))
            lw["bk"] = g(layer_tensor(l, T_BK), (s.kv_dim,))
            lw["bv"] = g(layer_tensor(l, T_BV), (s.kv_dim,))
        w["layers"][l] = lw
        if progress is not None:
            progress(f"layer {l + 1}/{s.n_layers}")
    return w


def gen_prompt(seed: int, vocab: int, n: int, sequence: int = 0) -> np.ndarray:
    """n token ids uniform over [0, vocab-2] (the mask id vocab-1 is excluded)."""
    z = uniform_u64(stream_key(seed, PROMPT_STREAM, sequence), 0, n)
    return (z % np.uint64(vocab - 1)).astype(np.int32)


def gen_prompt_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    z = uniform_u64(stream_key(seed, LENGTH_STREAM, 0), 0, batch)
    return (np.uint64(lo) + z % np.uint64(hi - lo + 1)).astype(np.int32)


def workload_prompts(wl: Workload) -> List[np.ndarray]:
    """The prompts of a workload (one per sequence)."""
    if wl.batch == 1:
        return [gen_prompt(wl.seed, wl.target.vocab, wl.prompt_len, 0)]
    lo, hi = wl.prompt_len_range
    lens = gen_prompt_lengths(wl.seed, wl.batch, lo, hi)
    return [gen_prompt(wl.seed, wl.target.vocab, int(n), b) for b, n in enumerate(lens)]
