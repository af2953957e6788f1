"""Algorithmic HBM bytes of the decode step (the roofline numerator).

Decode is bound by reloading the weights and the KV cache (Sec. 2.1), so the
algorithmic traffic of one forward over R rows at committed length L is:

* every streamed weight once, in bf16: all layer matrices, norms and biases,
  the final norm and the lm_head (for tied models the lm_head *is* the
  embedding matrix); the untied embedding contributes only the R gathered rows;
* the KV cache read by attention: 2 (K and V) * H_kv * head_dim * 2 B per layer
  and key position, over the L + R positions a query block sees;
* the KV rows written for the new positions.

Activations, partial sums and logits are excluded (they are small and stay in
cache), which makes the achieved-bandwidth figure conservative.  Table 3 of
the paper prints 2.48 GB of draft-phase traffic for the LLaMA3.2-1B-shaped PARD
draft, constant in k; ``draft_pass_bytes`` reproduces both facts.
"""
from __future__ import annotations

BF16 = 2


def streamed_params(spec) -> int:
    """Parameters read once per forward (everything except untied embedding rows)."""
    n = spec.n_params(with_embedding=True)
    if not spec.tied:
        n -= spec.vocab * spec.d_model
    return n


def kv_bytes_per_token(spec) -> int:
    return 2 * spec.n_layers * spec.n_kv_heads * spec.head_dim * BF16


def forward_bytes(spec, rows: int, context: int) -> int:
    """Algorithmic bytes of one forward over ``rows`` rows after ``context`` cached rows."""
    w = streamed_params(spec) * BF16
    emb = rows * spec.d_model * BF16
    kv_read = kv_bytes_per_token(spec) * (context + rows)
    kv_write = kv_bytes_per_token(spec) * rows
    return w + emb + kv_read + kv_write


def draft_pass_bytes(spec, k: int, n_pending: int, context: int) -> int:
    """One PARD draft pass: n_pending real rows + k-1 mask rows (Sec. 3.1)."""
    return forward_bytes(spec, n_pending + k - 1, context)


def verify_pass_bytes(spec, k: int, context: int) -> int:
    """One target pass over the pending token and k candidates."""
    return forward_bytes(spec, k + 1, context)


def step_bytes(target, draft, k: int, accepted_prev: int, l_t: int, l_d: int) -> int:
    """Draft pass + verify pass of one PARD step."""
    return (draft_pass_bytes(draft, k, accepted_prev + 1, l_d)
            + verify_pass_bytes(target, k, l_t))


def layer_launch_bytes(spec, rows: int, context: int, with_down: bool = False) -> int:
    """One decode layer's launch that carries the QKV GEMM (+ bias), the
    attention, the O-projection, the gate/up GEMM and (with_down) the down
    projection: those weights once, the layer's KV cache read over the context
    + rows positions and its new rows written, the rows' fp16 activations in
    and out (h out, or the next layer's fp16 input with the down projection)."""
    d, hd = spec.d_model, spec.head_dim
    q_dim, kv_dim = spec.n_heads * hd, spec.n_kv_heads * hd
    f_pad = (spec.ffn_dim + 31) // 32 * 32
    w = (d * (q_dim + 2 * kv_dim) + q_dim * d + 2 * f_pad * d + (f_pad * d if with_down else 0)) * BF16
    if spec.qkv_bias:
        w += (q_dim + 2 * kv_dim) * BF16
    kv = 2 * kv_dim * BF16 * (context + rows) + 2 * kv_dim * BF16 * rows
    return w + kv + rows * d * 2 + rows * (d if with_down else f_pad) * 2


def gemm_bytes(n: int, k: int, rows: int, a_bytes: int = 4, out_bytes: int = 4) -> int:
    """One skinny GEMM: bf16 weight [n, k] once, activations in, results out."""
    return n * k * BF16 + rows * k * a_bytes + rows * n * out_bytes


def batch_step_bytes(target, draft, k: int, contexts_t, contexts_d, pending) -> int:
    """One batched step over several sequences: each weight once per pass, and
    each sequence's own embedding rows and KV reads and writes (a forward_bytes
    per sequence without the weights)."""
    total = (streamed_params(target) + streamed_params(draft)) * BF16
    for lt, ld, n_pend in zip(contexts_t, contexts_d, pending):
        total += forward_bytes(target, k + 1, lt) - streamed_params(target) * BF16
        total += forward_bytes(draft, n_pend + k - 1, ld) - streamed_params(draft) * BF16
    return total


def gemm_flops(spec, rows: int) -> int:
    """Multiply-add flops of one forward's weight GEMMs (layers and lm_head) over ``rows`` rows."""
    return 2 * rows * (streamed_params(spec) - spec.n_layers * 2 * spec.d_model - spec.d_model)
